"""Latency calibration curves of the attention path on one MI355X.

    python calibrate.py [--quick] [--json OUT.json] [--md OUT.md]

The paper's optimizer charges every LLM call a latency T_infer taken from
calibrated throughput curves (§4.1, operator profiling: prefill and decode
tokens mapped to latency), and applies a prefix-caching discount: prompt
tokens covered by a cached, shared prefix are not charged as new work
(§4.1, state-conditional estimator). This script measures the attention part
of those curves for this library: the latency of one decode step, and of one
chunked prefill, as a function of the shared prefix length P, the private
suffix (or chunk) length S, the number of requests sharing each prefix G and
the batch size R, on Llama-3-8B-shaped heads (32 query / 8 KV heads, d 128,
bf16).

Each point is a synthetic batch (R / G prefixes of P tokens, each shared by G
requests, every request with S private tokens; pages placed at random in a
pool of 1.25x the need), timed over single calls with HIP events on the
call's stream, the median of the calls taken, inputs rotated over copies
larger than the Infinity Cache so keys stream from HBM.

A model is fitted by least squares on relative error:

    T = c0 + c_row * (query rows x query heads)
        + c_split * (1 if decode rows are split over several work items,
          which adds the merge launch)
        + (A^k + B^k)^(1/k),
    A = c_kv * (distinct K/V bytes) + c_pair_private * (visible (query,
        key) pairs outside shared prefixes x query heads)
    B = c_pair_shared * (visible pairs on shared prefixes x query heads)
        + c_shared * (K/V bytes of prefixes shared by more than one request)

A is the streaming of keys read by one request, B the matrix work of the
grouped prefix pass; the two run side by side in one launch, so they add
when k = 1 and overlap fully as k grows (k is fitted).

in which the prefix-caching discount is explicit: a prefix shared by G
requests contributes its K/V bytes once, not G times. Checks: T grows with S
and with P; at fixed P and S, a larger group is not slower; the fit's
relative error, on the grid and on held-out workloads predicted from their
forests (forest_features works on any batch, e.g. one built from token ids
by halo_prefix_tree_build). One JSON object is printed (and written with
--json).
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MALL_BYTES = 256 << 20
HQ, HKV, D = 32, 8, 128
ELT = 2        # bf16
MONOTONE_TOL = 0.03

DECODE_GRID = dict(requests=[64], group=[1, 4, 16, 64], prefix=[0, 512, 2048, 8192], suffix=[64, 256, 1024])
# large batches in few sharing groups (the regime of serving many replicas of
# one workflow); kept small so the sweep stays within seconds per point
DECODE_GRID_WIDE = dict(requests=[512], group=[8, 64, 512], prefix=[2048, 8192], suffix=[64, 256])
# the largest batches: 1024 requests in 8 groups or one, long suffixes
DECODE_GRID_LARGE = dict(requests=[1024], group=[128, 1024], prefix=[2048, 8192], suffix=[256, 1024, 2048])
PREFILL_GRID = dict(requests=[8, 32], group=["1", "all"], prefix=[0, 1024, 4096], suffix=[128, 512])
QUICK_DECODE = dict(requests=[32], group=[1, 32], prefix=[0, 1024], suffix=[64, 1024])
QUICK_PREFILL = dict(requests=[8], group=["all"], prefix=[0, 1024], suffix=[128, 256])


COEF_NAMES = ("c0_us", "c_kv_us_per_byte", "c_pair_shared_us", "c_pair_private_us", "c_row_us", "c_split_us",
              "c_shared_us_per_byte", "k")
# private keys a decode row reads in one work item before it is split
SPLIT_KEYS = 2048


def features(kind, requests, group, prefix, suffix):
    """Model features of one point: 1, distinct K/V bytes, visible pairs on
    shared prefixes x query heads, the other visible pairs x query heads,
    query rows x query heads (a decode step has one query row per request, a
    prefill chunk `suffix` rows, causal inside the chunk), the split
    indicator (decode rows whose keys span a shared prefix and a suffix, or
    more than SPLIT_KEYS private keys, go through the merge) and the K/V
    bytes of shared prefixes."""
    n_prefixes = requests // group if prefix > 0 else 0
    kv_tokens = n_prefixes * prefix + requests * suffix
    tok_bytes = 2 * HKV * D * ELT
    shared = group > 1 and prefix > 0
    shared_bytes = n_prefixes * prefix * tok_bytes if shared else 0
    if kind == "decode":
        rows = requests
        prefix_pairs, other_pairs = requests * prefix, requests * suffix
        split = 1.0 if shared or prefix + suffix > SPLIT_KEYS else 0.0
    else:
        rows = requests * suffix
        prefix_pairs, other_pairs = requests * suffix * prefix, requests * suffix * (suffix + 1) // 2
        split = 0.0
    pairs_shared = prefix_pairs if shared else 0
    pairs_private = other_pairs + (0 if shared else prefix_pairs)
    return [1.0, float(kv_tokens * tok_bytes), float(pairs_shared * HQ), float(pairs_private * HQ),
            float(rows * HQ), split, float(shared_bytes)]


def forest_features(seg_len, req_paths, q_len=None, num_q_heads=None, num_kv_heads=None, head_dim=None, elt=ELT):
    """The model's features for any batch given as a forest (segment lengths
    and per-request paths, e.g. from halo_prefix_tree_build on token ids;
    q_len for a prefill whose last segment per path is the chunk). Shared
    segments (on more than one path) count once in the K/V bytes: the
    prefix-caching discount of the cost model."""
    num_q_heads = HQ if num_q_heads is None else num_q_heads
    num_kv_heads = HKV if num_kv_heads is None else num_kv_heads
    head_dim = D if head_dim is None else head_dim
    seg_len = [int(x) for x in seg_len]
    tok_bytes = 2 * num_kv_heads * head_dim * elt
    refs = [0] * len(seg_len)
    for path in req_paths:
        for s in path:
            refs[s] += 1
    kv_bytes = sum(seg_len) * tok_bytes
    shared_bytes = sum(n for n, r in zip(seg_len, refs) if r > 1) * tok_bytes
    rows = pairs_shared = pairs_private = 0
    split = 0.0
    for r, path in enumerate(req_paths):
        keys = sum(seg_len[s] for s in path)
        shared_keys = sum(seg_len[s] for s in path if refs[s] > 1)
        if q_len is None:
            rows += 1
            pairs_shared += shared_keys
            pairs_private += keys - shared_keys
            if shared_keys > 0 or keys - shared_keys > SPLIT_KEYS:
                split = 1.0
        else:
            n = int(q_len[r])
            rows += n
            pairs_shared += n * shared_keys
            pairs_private += n * (keys - n - shared_keys) + n * (n + 1) // 2
    return [1.0, float(kv_bytes), float(pairs_shared * num_q_heads), float(pairs_private * num_q_heads),
            float(rows * num_q_heads), split, float(shared_bytes)]


def latency(coef, f):
    """The model's latency (us) for coefficients `coef` (COEF_NAMES order)
    and a feature vector (or an array of them, one per row)."""
    import numpy as np
    F = np.atleast_2d(np.asarray(f, dtype=np.float64))
    c0, ckv, cps, cpp, crow, csplit, cshared, k = coef
    a = ckv * F[:, 1] + cpp * F[:, 3]
    b = cps * F[:, 2] + cshared * F[:, 6]
    t = c0 + crow * F[:, 4] + csplit * F[:, 5] + (a ** k + b ** k) ** (1.0 / k)
    return t if np.ndim(f) > 1 else float(t[0])


def predict_forest(coef, seg_len, req_paths, q_len=None, **shape):
    """Predicted latency (us) of one call on a batch given as a forest."""
    return latency(coef, forest_features(seg_len, req_paths, q_len, **shape))


# starting point of the fit (us, us/byte, us/pair, ...): a few-us launch,
# ~7 TB/s streaming, ~2 PFLOP/s matrix work
_FIT_START = (3.0, 1.4e-7, 5e-7, 1e-9, 1e-3, 5.0, 1e-9)


def fit(points):
    """Least squares of the latency model on relative error over a list of
    (features, latency_us); coefficients are kept positive (fitted in log
    space) and k >= 1. Returns coefficients and relative errors."""
    import numpy as np
    from scipy.optimize import least_squares
    F = np.array([p[0] for p in points], dtype=np.float64)
    y = np.array([p[1] for p in points], dtype=np.float64)

    def coef_of(theta):
        return list(np.exp(theta[:7])) + [1.0 + float(np.exp(theta[7]))]

    x0 = np.append(np.log(_FIT_START), 0.0)
    lo = np.append(np.full(7, -80.0), -10.0)
    hi = np.append(np.full(7, 30.0), 3.0)      # k <= 1 + e^3
    r = least_squares(lambda th: (latency(coef_of(th), F) - y) / y, x0, bounds=(lo, hi), max_nfev=20000)
    coef = [float(c) for c in coef_of(r.x)]
    # a feature that is zero at every point leaves its coefficient undefined
    for j in range(1, 7):
        if not F[:, j].any():
            coef[j] = 0.0
    rel = np.abs(latency(coef, F) - y) / y
    return coef, rel.tolist()


def cross_validate(points):
    """Leave-one-out relative errors of the model on a list of (features,
    latency_us): each point predicted by the fit on all the others."""
    import numpy as np
    errs = []
    for i in range(len(points)):
        coef, _ = fit(points[:i] + points[i + 1:])
        f, y = points[i]
        errs.append(abs(latency(coef, f) - y) / y)
    return errs


def predict(coef, kind, requests, group, prefix, suffix):
    return latency(coef, features(kind, requests, group, prefix, suffix))


def check_monotone(points, tol=MONOTONE_TOL):
    """Violations of the expected orderings among measured points, each
    given by its keys (kind, requests, group, prefix, suffix) -> latency:
    longer suffix or prefix is not faster; a larger sharing group is not
    slower (P > 0)."""
    bad = []
    for (kind, r, g, p, s), t in points.items():
        for (kind2, r2, g2, p2, s2), t2 in points.items():
            if (kind2, r2) != (kind, r):
                continue
            if g2 == g and p2 == p and s2 > s and t2 < t * (1 - tol):
                bad.append(f"{kind} R={r} G={g} P={p}: S {s}->{s2} went {t:.1f}->{t2:.1f} us")
            if g2 == g and s2 == s and p2 > p and t2 < t * (1 - tol):
                bad.append(f"{kind} R={r} G={g} S={s}: P {p}->{p2} went {t:.1f}->{t2:.1f} us")
            if p > 0 and p2 == p and s2 == s and g2 > g and t2 > t * (1 + tol):
                bad.append(f"{kind} R={r} P={p} S={s}: G {g}->{g2} went {t:.1f}->{t2:.1f} us")
    return bad


def _measure(kind, requests, group, prefix, suffix, calls, seed):
    import numpy as np
    import torch
    from paper_2509_02121_amd import halo
    from workloads import build_workload
    n_prefixes = requests // group if prefix > 0 else 0
    seg_len = [prefix] * n_prefixes + [suffix] * requests
    paths = [([r // group] if prefix > 0 else []) + [n_prefixes + r] for r in range(requests)]
    q_len = None if kind == "decode" else np.full(requests, suffix, dtype=np.int32)
    w = build_workload(f"cal_{kind}", seed, HQ, HKV, D, torch.bfloat16, seg_len, paths, q_len,
                       value_scale=0.5, device="cuda")
    return _time_workload(w, calls)


def _time_workload(w, calls):
    """Median of single calls on a workload (inputs rotated past the
    Infinity Cache)."""
    import torch
    from paper_2509_02121_amd import halo
    params = halo.make_params(w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype, w.num_pool_pages, w.scale,
                              w.dtype)
    runner = halo.PrefixAttention(params, w.forest_csr(), "cuda")
    pool_bytes = (w.k_pool.numel() + w.v_pool.numel()) * ELT
    n_rep = max(1, min(16, -(-4 * MALL_BYTES // max(pool_bytes, 1))))
    reps = [(w.q, w.k_pool, w.v_pool)] + [(w.q.clone(), w.k_pool.clone(), w.v_pool.clone())
                                          for _ in range(n_rep - 1)]
    stream = torch.cuda.current_stream()
    outs = [runner.alloc_outputs(w.q) for _ in range(n_rep)]
    fns = [runner.bind(*reps[i], *outs[i], stream) for i in range(n_rep)]
    for i in range(10):
        fns[i % n_rep]()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(calls)]
    for i, (a, b) in enumerate(ev):
        a.record(stream)
        fns[i % n_rep]()
        b.record(stream)
    torch.cuda.synchronize()
    t = sorted(a.elapsed_time(b) * 1e3 for a, b in ev)
    del reps, outs, fns, runner, w
    torch.cuda.empty_cache()
    return t[len(t) // 2]


def run(grids, calls=50, log=print):
    points = {}
    for kind, grid in grids:
        for r in grid["requests"]:
            groups = sorted({r if g == "all" else int(g) for g in grid["group"]} & set(range(1, r + 1)))
            groups = [g for g in groups if r % g == 0]
            for g in groups:
                for p in grid["prefix"]:
                    if p == 0 and g != groups[0]:
                        continue       # without a prefix the group size changes nothing
                    for s in grid["suffix"]:
                        t0 = time.perf_counter()
                        us = _measure(kind, r, g, p, s, calls, seed=1 + len(points))
                        points[(kind, r, g, p, s)] = us
                        log(f"{kind} R={r} G={g} P={p} S={s}: {us:.1f} us "
                            f"({time.perf_counter() - t0:.1f} s)")
    return points


HELD_OUT = ("llama8b_decode", "two_level_tree_decode", "llama70b_batch_decode", "chunked_prefill")


def held_out(summary, calls=50, log=print):
    """Measure the named workloads of the calibrated head shape (forests the
    grid does not contain) and compare with the fitted model's prediction
    from their forests. Curves are per model shape, as the paper keeps them
    per model and hardware configuration."""
    from workloads import make_config
    out = []
    for name in HELD_OUT:
        w = make_config(name, device="cuda")
        if (w.num_q_heads, w.num_kv_heads, w.head_dim) != (HQ, HKV, D):
            del w
            continue                   # curves are per model shape
        kind = "prefill" if w.is_prefill else "decode"
        coef = list(summary[kind]["coef"].values())
        pred = predict_forest(coef, w.seg_len, w.req_paths, w.q_len, num_q_heads=w.num_q_heads,
                              num_kv_heads=w.num_kv_heads, head_dim=w.head_dim)
        us = _time_workload(w, calls)
        out.append(dict(workload=name, kind=kind, us=round(us, 2), predicted_us=round(pred, 2),
                        rel_err=round((pred - us) / us, 4)))
        log(f"held out {name}: {us:.1f} us measured, {pred:.1f} us predicted")
    return out


def summarize(points):
    out = {"model": "T_us = c0 + c_row*rows_x_hq + c_split*split + (A^k + B^k)^(1/k); "
                    "A = c_kv*kv_bytes + c_pair_private*private_pairs_x_hq, "
                    "B = c_pair_shared*shared_pairs_x_hq + c_shared*shared_kv_bytes",
           "shape": {"num_q_heads": HQ, "num_kv_heads": HKV, "head_dim": D, "dtype": "bf16"},
           "points": [dict(kind=k[0], requests=k[1], group=k[2], prefix=k[3], suffix=k[4], us=round(v, 2))
                      for k, v in points.items()]}
    for kind in ("decode", "prefill"):
        pts = [(features(*k), v) for k, v in points.items() if k[0] == kind]
        if len(pts) < 4:
            continue
        coef, rel = fit(pts)
        loo = sorted(cross_validate(pts))
        out[kind] = {"coef": dict(zip(COEF_NAMES, coef)),
                     "effective_kv_tbps": round(1.0 / coef[1] / 1e6, 3) if coef[1] > 0 else None,
                     "max_rel_err": round(max(rel), 4), "median_rel_err": round(sorted(rel)[len(rel) // 2], 4),
                     "loo_median_rel_err": round(loo[len(loo) // 2], 4), "loo_max_rel_err": round(loo[-1], 4)}
    out["monotonicity_violations"] = check_monotone(points)
    return out


def to_markdown(summary, command):
    lines = [f"# Attention latency calibration (decode step and chunked prefill), {HQ}/{HKV} heads", "",
             "Command (repository root, one MI355X):", "", f"    {command}", "",
             f"Heads {HQ}/{HKV}, d {D}, bf16. R requests, G sharing each prefix of P tokens, S private "
             "tokens each (decode) or an S-token causal chunk each (prefill). Median of single calls.", "",
             "| kind | R | G | P | S | us |", "|---|---|---|---|---|---|"]
    for p in summary["points"]:
        lines.append(f"| {p['kind']} | {p['requests']} | {p['group']} | {p['prefix']} | {p['suffix']} | {p['us']} |")
    lines += ["", f"Model: `{summary['model']}` (least squares on relative error, positive coefficients, "
              "k >= 1).", ""]
    for kind in ("decode", "prefill"):
        if kind in summary:
            s = summary[kind]
            lines.append(f"- {kind}: {json.dumps(s['coef'])}; effective K/V streaming rate "
                         f"{s['effective_kv_tbps']} TB/s; relative error max {s['max_rel_err']}, "
                         f"median {s['median_rel_err']}; leave-one-out median {s['loo_median_rel_err']}, "
                         f"max {s['loo_max_rel_err']}.")
    if summary.get("held_out"):
        lines += ["", "Held-out workloads (forests outside the grid), measured and predicted from their forests "
                  "(`forest_features`):", "", "| workload | measured (us) | predicted (us) | error |",
                  "|---|---|---|---|"]
        for h in summary["held_out"]:
            lines.append(f"| {h['workload']} | {h['us']} | {h['predicted_us']} | {h['rel_err']:+.1%} |")
    v = summary["monotonicity_violations"]
    lines += ["", f"Monotonicity violations (tolerance {MONOTONE_TOL:.0%}): " + ("none." if not v else ""), ""]
    lines += [f"- {x}" for x in v]
    return "\n".join(lines) + "\n"


def main():
    global HQ, HKV
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--quick", action="store_true", help="a few points only")
    ap.add_argument("--calls", type=int, default=50)
    ap.add_argument("--json", default=None)
    ap.add_argument("--md", default=None)
    ap.add_argument("--q-heads", type=int, default=HQ)
    ap.add_argument("--kv-heads", type=int, default=HKV)
    args = ap.parse_args()
    HQ, HKV = args.q_heads, args.kv_heads
    import torch
    from paper_2509_02121_amd import halo
    halo.load_library(require_gpu=True)
    torch.cuda.set_device(0)
    grids = [("decode", QUICK_DECODE), ("prefill", QUICK_PREFILL)] if args.quick else \
        [("decode", DECODE_GRID), ("decode", DECODE_GRID_WIDE), ("decode", DECODE_GRID_LARGE),
         ("prefill", PREFILL_GRID)]
    points = run(grids, args.calls, log=lambda m: print(m, flush=True))
    summary = summarize(points)
    if not args.quick:
        summary["held_out"] = held_out(summary, args.calls, log=lambda m: print(m, flush=True))
    if args.json:
        with open(args.json, "w") as f:
            json.dump(summary, f, indent=1)
    if args.md:
        cmd = "python -u calibrate.py" + (" --quick" if args.quick else "") + \
            (f" --q-heads {HQ} --kv-heads {HKV}" if (HQ, HKV) != (32, 8) else "") + \
            (f" --md {args.md}" if args.md else "") + (f" --json {args.json}" if args.json else "")
        with open(args.md, "w") as f:
            f.write(to_markdown(summary, cmd))
    print(json.dumps({k: v for k, v in summary.items() if k != "points"}), flush=True)


if __name__ == "__main__":
    main()
