"""Throughput of the shared-prefix paged-attention path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step = one library call over one batch: the whole decode path (grouped
prefix pass, per-request suffix pass, log-sum-exp merge) or, for the
chunked-prefill workload, the whole prefill. Inputs live in HBM before the
timed region; steps rotate over several copies of the inputs (more bytes
than the 256 MB Infinity Cache) so every step streams its KV pages from HBM.
Prints one JSON line (rank 0, single GPU).
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0        # MI355X HBM3E
BF16_MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
# The largest single-GPU workload: 1024 requests of a 70B-shaped layer (64 q /
# 8 kv heads, d = 128, bf16) in 8 groups of 128 sharing 8192-token prefixes,
# suffixes U{256..2048}.
DEFAULT_WORKLOAD = "llama70b_batch_decode"
# Measured in the same run, after the headline, each with its own roofline.
SECONDARY_WORKLOADS = ("llama8b_decode", "two_level_tree_decode", "chunked_prefill")
MALL_BYTES = 256 << 20


def source_sha256():
    """sha256 over the kernel, planner and shared-header sources: measured
    traffic stays valid only for the code it was measured on."""
    import hashlib
    h = hashlib.sha256()
    for name in ("halo_kernels.hip", "halo_plan.cpp", "halo_internal.h"):
        with open(os.path.join(ROOT, "paper_2509_02121_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def algorithmic_bytes(w, stats):
    """Bytes the method must move once: each segment's K and V, the page-id
    table, Q, O and the LSE."""
    elt = 2 if w.dtype.itemsize == 2 else 4
    kv = int(sum(int(n) for n in w.seg_len)) * 2 * w.num_kv_heads * w.head_dim * elt
    pages = sum(len(p) for p in w.seg_pages) * 4
    rows = w.q.shape[0] * w.num_q_heads
    q = rows * w.head_dim * elt
    o = rows * w.head_dim * elt          # output in the input dtype
    lse = rows * 4
    return kv + pages + q + o + lse


def _cpu_info():
    import os
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:  # pragma: no cover
        pass
    return int(threads), model


def _request_order(w):
    """Requests in the order the CPU baseline samples them: strided over the
    batch (0, R/8, 2R/8, ..., then 1, 1 + R/8, ...), so a bounded sample
    covers every prefix group and the whole suffix-length range."""
    R = w.num_requests
    stride = max(1, R // 8)
    return [r for off in range(stride) for r in range(off, R, stride)]


def cpu_baseline(w, min_seconds=10.0):
    """The fp64 oracle, as it stands, on the host cores: a bounded sample of
    the same workload, one request at a time.

    Each sampled request's segments are upcast to fp64 outside the timed
    region (segments shared by several sampled requests are upcast once, and
    nothing is upcast for requests outside the sample, so host memory stays
    bounded on the largest batch); only the oracle call is timed. Requests are
    taken in a strided order until min_seconds of oracle time have passed.
    The rate is query-tokens per second of oracle time."""
    import numpy as np
    import oracle
    threads, model = _cpu_info()
    refs = {}
    for path in w.req_paths:
        for s in path:
            refs[s] = refs.get(s, 0) + 1
    shared64 = {}

    def kv64(s):
        # segments on several paths are upcast once and kept; private ones
        # are upcast for their one request and dropped after it
        if s in shared64:
            return shared64[s]
        k, v = w.segment_kv(s)
        kv = (k.double().numpy(), v.double().numpy())
        if refs.get(s, 0) > 1:
            shared64[s] = kv
        return kv

    q = w.q.double().cpu().numpy()
    tokens = 0
    done = []
    busy = 0.0
    order = _request_order(w)
    while busy < min_seconds:
        r = order[len(done) % len(order)]
        path = w.req_paths[r]
        seg_k = {s: kv64(s)[0] for s in path}
        seg_v = {s: kv64(s)[1] for s in path}
        a, b = w.q_rows_of_request(r)
        t0 = time.perf_counter()
        if w.is_prefill:
            oracle.prefill(q[a:b], w.q_len[r:r + 1], seg_k, seg_v, [path], w.scale)
        else:
            oracle.decode(q[a:b], seg_k, seg_v, [path], w.scale)
        busy += time.perf_counter() - t0
        tokens += b - a
        done.append(r)
    keys = int(sum(sum(int(w.seg_len[s]) for s in w.req_paths[r]) for r in done))
    sample = (f"{len(done)} of {w.num_requests} requests (strided order), {tokens} query tokens, "
              f"{keys} keys per head group in total; fp64 upcast outside the timed region")
    return {"value": tokens / busy, "unit": "query-tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": sample, "seconds": round(busy, 3),
            "host_cpus": len(os.sched_getaffinity(0)), "os_cpu_count": os.cpu_count(),
            "cpu_model": model, "blas_threads": int(threads)}


def _time_launches(call, steps, warmup, stream):
    """Average GPU time of one launch: HIP events on the launch stream around
    `steps` back-to-back launches."""
    import torch
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / steps


def write_path_bench(args):
    """Paged-KV write path on the workload's own page lists (one JSON line).

    Scatter: every request's last segment (its private suffix, or its prefill
    chunk) is the target; decode appends the segment's last token (start =
    length - 1, count 1), prefill writes the whole chunk; timed per pool and
    for both pools in one call. Copy: one page per
    request, the first page of its last segment, to a distinct free page of
    the pool (the copy of copy-on-write; distinct sources, so that no copy
    reads another's source out of cache). Algorithmic bytes: the
    token bytes read from the input plus the same bytes written to the pool
    (scatter); a page read plus a page written (copy)."""
    import numpy as np
    import torch
    from paper_2509_02121_amd import halo
    from workloads import make_config

    halo.load_library(require_gpu=True)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = make_config(args.workload, device=dev, poison=False)
    params = halo.make_params(w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype, w.num_pool_pages,
                              w.scale, w.dtype)
    R = w.num_requests
    elt = w.k_pool.element_size()
    tok_bytes = w.num_kv_heads * w.head_dim * elt          # one token, one pool
    last = [w.req_paths[r][-1] for r in range(R)]
    lens = np.array([int(w.seg_len[s]) for s in last], np.int64)
    if w.is_prefill:
        start, count = np.zeros(R, np.int32), lens.astype(np.int32)
    else:
        start, count = (lens - 1).astype(np.int32), np.ones(R, np.int32)
    pages = [np.asarray(w.seg_pages[s], np.int32) for s in last]
    indptr = np.zeros(R + 1, np.int32)
    indptr[1:] = np.cumsum([len(p) for p in pages])
    offs = np.zeros(R, np.int64)
    offs[1:] = np.cumsum(count)[:-1]
    n_tok = int(count.sum())
    gen = torch.Generator(device=dev)
    gen.manual_seed(7)
    src = torch.randn((n_tok, w.num_kv_heads, w.head_dim), generator=gen, device=dev).to(w.dtype)
    t = lambda a: torch.as_tensor(a, device=dev)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    sc_args = (t(np.concatenate(pages)), t(indptr), t(start), t(count), t(offs), src, flag, stream)
    used = np.zeros(w.num_pool_pages, bool)
    for p in w.seg_pages:
        used[np.asarray(p, np.int64)] = True
    free = np.nonzero(~used)[0].astype(np.int32)
    if len(free) < R:
        raise SystemExit(f"pool has {len(free)} free pages, {R} needed for the copies")
    cp_src = t(np.array([int(w.seg_pages[s][0]) for s in last], np.int32))
    cp_dst = t(free[:R])
    res = {}
    for name, pool, kind in (("k", w.k_pool, halo.HALO_POOL_K), ("v", w.v_pool, halo.HALO_POOL_V)):
        call = halo.bind_kv_page_scatter(pool, params, kind, *sc_args[:5], src, flag, stream)
        res["scatter_" + name + "_us"] = _time_launches(call, args.steps, args.warmup, stream)
    call = halo.bind_kv_page_scatter_kv(w.k_pool, w.v_pool, params, *sc_args[:5], src, src, flag, stream)
    res["scatter_kv_us"] = _time_launches(call, args.steps, args.warmup, stream)
    call = halo.bind_kv_page_copy(w.k_pool, params, cp_src, cp_dst, flag, stream)
    res["copy_us"] = _time_launches(call, args.steps, args.warmup, stream)
    torch.cuda.synchronize()
    if int(flag.item()):
        raise SystemExit("write path flagged bad input")
    sc_bytes = 2 * n_tok * tok_bytes
    page_bytes = w.num_kv_heads * w.page_size * w.head_dim * elt
    cp_bytes = 2 * R * page_bytes
    gbps = lambda b, us: round(b / (us * 1e-6) / 1e9, 1)
    line = {
        "metric": "paged-KV write path: HBM GB/s per launch",
        "config": {"workload": w.name, "mode": "prefill chunk write" if w.is_prefill else "decode append",
                   "sequences": R, "tokens": n_tok, "copy_pages": R, "steps": args.steps},
        "scatter_bytes": sc_bytes, "copy_bytes": cp_bytes,
    }
    for name in ("k", "v"):
        us = res["scatter_" + name + "_us"]
        line["scatter_" + name] = {"us": round(us, 2), "gbps": gbps(sc_bytes, us),
                                   "frac": round(gbps(sc_bytes, us) / HBM_PEAK_GBPS, 4)}
    us = res["scatter_kv_us"]
    line["scatter_kv_one_call"] = {"us": round(us, 2), "gbps": gbps(2 * sc_bytes, us),
                                   "frac": round(gbps(2 * sc_bytes, us) / HBM_PEAK_GBPS, 4)}
    line["copy"] = {"us": round(res["copy_us"], 2), "gbps": gbps(cp_bytes, res["copy_us"]),
                    "frac": round(gbps(cp_bytes, res["copy_us"]) / HBM_PEAK_GBPS, 4)}
    print(json.dumps(line), flush=True)


def gather_bench(args):
    """Page gather of every segment of the workload (its distinct K/V working
    set), one launch per pool, timed with events on the launch stream (one
    JSON line). Algorithmic bytes: the gathered bytes read plus the same
    bytes written."""
    import numpy as np
    import torch
    from paper_2509_02121_amd import halo
    from workloads import make_config

    halo.load_library(require_gpu=True)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = make_config(args.workload, device=dev, poison=False)
    params = halo.make_params(w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype, w.num_pool_pages,
                              w.scale, w.dtype)
    S = len(w.seg_pages)
    lens = np.asarray(w.seg_len, np.int64)
    indptr = np.zeros(S + 1, np.int32)
    indptr[1:] = np.cumsum([len(p) for p in w.seg_pages])
    offs = np.zeros(S, np.int64)
    offs[1:] = np.cumsum(lens)[:-1]
    n_tok = int(lens.sum())
    t = lambda a: torch.as_tensor(a, device=dev)
    ids = t(np.concatenate(w.seg_pages).astype(np.int32))
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    out = torch.empty((n_tok, w.num_kv_heads, w.head_dim), dtype=w.dtype, device=dev)
    stream = torch.cuda.current_stream()
    res = {}
    lens_d, indptr_d, offs_d = t(lens.astype(np.int32)), t(indptr), t(offs)
    for name, pool, kind in (("k", w.k_pool, halo.HALO_POOL_K), ("v", w.v_pool, halo.HALO_POOL_V)):
        call = halo.bind_kv_page_gather(pool, params, kind, ids, indptr_d, lens_d, offs_d, out, flag, stream)
        res[name] = _time_launches(call, args.steps, args.warmup, stream)
    torch.cuda.synchronize()
    if int(flag.item()):
        raise SystemExit("gather flagged bad input")
    elt = w.k_pool.element_size()
    nbytes = 2 * n_tok * w.num_kv_heads * w.head_dim * elt
    gbps = lambda us: round(nbytes / (us * 1e-6) / 1e9, 1)
    line = {"metric": "paged-KV gather: HBM GB/s per launch",
            "config": {"workload": w.name, "segments": S, "tokens": n_tok, "steps": args.steps},
            "bytes_per_launch": nbytes}
    for name in ("k", "v"):
        line["gather_" + name] = {"us": round(res[name], 2), "gbps": gbps(res[name]),
                                  "frac": round(gbps(res[name]) / HBM_PEAK_GBPS, 4)}
    print(json.dumps(line), flush=True)


def probe_read_bench(args):
    """One tile-read microbenchmark configuration over a pool of
    args.probe_read_bytes bytes (two register stages, two waves per SIMD,
    32 steps of 4 tiles per item, random tile order): the known number of
    bytes every launch reads, for dividing the HBM read counter of a profiled
    run by (one JSON line)."""
    import numpy as np
    import torch
    from paper_2509_02121_amd import probe
    probe.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    n_tiles = args.probe_read_bytes // 4096 // 128 * 128
    pool_bytes = n_tiles * 4096
    pool = torch.empty(pool_bytes, dtype=torch.uint8, device=dev)
    pool.view(torch.int32).fill_(0x3c003c00)
    perm = torch.as_tensor(np.random.Generator(np.random.PCG64(11)).permutation(n_tiles).astype(np.int32),
                           device=dev)
    out = torch.empty(1 << 16, dtype=torch.int32, device=dev)
    nt = 0 if args.probe_plain_loads else 1
    call = probe.bind_stream_read(pool, perm, 32, 2, 2, nt, 256, out, stream)
    steps, warmup = max(1, min(args.steps, 20)), max(1, min(args.warmup, 3))
    us = _time_launches(call, steps, warmup, stream)
    print(json.dumps({"metric": "tile read", "bytes_per_launch": int(pool_bytes), "nontemporal": nt,
                      "launches": steps + warmup, "us": round(us, 1),
                      "gbps": round(pool_bytes / us / 1e3, 1)}), flush=True)


def probe_bench(args):
    """Context microbenchmarks (one JSON line): the HBM read rate of random
    4 KB tiles with the suffix pass's loads, the dense bf16 MFMA rate, and
    the v_exp_f32 rate with and without MFMAs on the same wave. Each figure
    is the mean of `steps` launches timed with HIP events on the launch
    stream after `warmup` launches."""
    import numpy as np
    import torch
    from paper_2509_02121_amd import probe

    probe.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    steps, warmup = max(3, min(args.steps, 20)), max(1, min(args.warmup, 3))
    res = {"metric": "context microbenchmarks (gfx950)", "steps": steps}

    # --- stream read: a 4 GiB pool (16x the Infinity Cache), every tile once
    # per launch, in a seeded random order (or in address order)
    pool_bytes = 4 << 30
    n_tiles = pool_bytes // 4096
    pool = torch.empty(pool_bytes, dtype=torch.uint8, device=dev)
    pool.view(torch.int32).fill_(0x3c003c00)
    rng = np.random.Generator(np.random.PCG64(11))
    perm = torch.as_tensor(rng.permutation(n_tiles).astype(np.int32), device=dev)
    seq = torch.arange(n_tiles, dtype=torch.int32, device=dev)
    out = torch.empty(1 << 16, dtype=torch.int32, device=dev)
    rows = []
    configs = [  # (order, stages, waves per SIMD, non-temporal, steps per item)
        ("random", 2, 2, 1, 32), ("random", 2, 2, 0, 32), ("random", 3, 2, 1, 32), ("random", 2, 1, 1, 32),
        ("random", 3, 1, 1, 32), ("random", 4, 1, 1, 32), ("random", 2, 2, 1, 8), ("random", 3, 2, 1, 8),
        ("address", 2, 2, 1, 32), ("address", 3, 2, 1, 32),
        # independent items (metadata round trip, own pipeline, drain), without
        # and with the per-step MFMA/softmax work
        ("random", 10, 2, 1, 32), ("random", 11, 2, 1, 32), ("random", 10, 2, 1, 16), ("random", 11, 2, 1, 16),
        # the same with the suffix pass's K/V tile access pattern
        ("random", 12, 2, 1, 32), ("random", 13, 2, 1, 32),
        # one item per wave, a workgroup per 8 items (not persistent)
        ("random", 13, 2, 1, -32),
    ]
    for order, stages, wps, nt, spi in configs:
        blocks = 256 if wps == 2 else 512
        if spi < 0:       # one item per wave: as many workgroups as items / 8
            spi = -spi
            blocks = n_tiles // (4 * spi) // 8
        call = probe.bind_stream_read(pool, perm if order == "random" else seq, spi, stages, wps, nt, blocks,
                                      out, stream)
        us = _time_launches(call, steps, warmup, stream)
        gbps = pool_bytes / (us * 1e-6) / 1e9
        mode = {10: "items", 11: "items+compute", 12: "items kv-pattern",
                13: "items+compute kv-pattern"}.get(stages, "stream")
        rows.append({"order": order, "mode": mode, "stages": 2 if stages >= 10 else stages,
                     "waves_per_simd": wps, "nontemporal": nt,
                     "steps_per_item": spi, "blocks": blocks, "bytes_in_flight_per_cu":
                     ((2 if stages >= 10 else stages) - 1) * 16384 * 4 * wps, "us": round(us, 1),
                     "gbps": round(gbps, 1),
                     "frac": round(gbps / HBM_PEAK_GBPS, 4)})
        print(f"stream {rows[-1]}", file=sys.stderr, flush=True)
    res["stream_read"] = {"bytes_per_launch": pool_bytes, "tile_bytes": 4096, "configs": rows}
    del pool, perm, seq
    torch.cuda.empty_cache()

    # --- MFMA: 1024 blocks of 4 waves, 8 independent chains per wave
    fout = torch.empty(1024 * 256, dtype=torch.float32, device=dev)
    mf = {}
    for shape, flop in ((32, 32 * 32 * 16 * 2), (16, 16 * 16 * 32 * 2)):
        iters = 4000
        call = probe.bind_mfma(shape, iters, 1024, fout, stream)
        us = _time_launches(call, steps, warmup, stream)
        tflops = 1024 * 4 * iters * 8 * flop / (us * 1e-6) / 1e12
        mf[f"{shape}x{shape}x{16 if shape == 32 else 32}_bf16"] = {
            "us": round(us, 1), "tflops": round(tflops, 1), "frac_of_2500": round(tflops / BF16_MFMA_PEAK_TFLOPS, 4)}
    res["mfma"] = mf

    # --- v_exp_f32: 16 chains per lane; one 32x32x16 MFMA per M exps
    ex = []
    for blocks in (256, 512):
        for m in (0, 8, 4, 2):
            iters = 4000
            call = probe.bind_exp(m, iters, blocks, fout, stream)
            us = _time_launches(call, steps, warmup, stream)
            cycles = us * 1e-6 * 2.4e9                     # at the 2.4 GHz peak clock
            waves_per_simd = blocks * 4 / 1024
            n_exp = iters * 16 * waves_per_simd            # exps issued per SIMD
            n_mfma = iters * (16 // m if m else 0) * waves_per_simd
            ex.append({"blocks": blocks, "waves_per_simd": waves_per_simd, "exp_per_mfma": m,
                       "us": round(us, 1), "cycles_per_exp": round(cycles / n_exp, 2),
                       "cycles_per_mfma": round(cycles / n_mfma, 2) if m else None})
    res["exp"] = ex

    # --- MFMA beside VALU work on one SIMD: interleaved in each wave, or one
    # wave of each kind per SIMD
    fo = torch.empty(512 * 512, dtype=torch.float32, device=dev)
    ov = []
    for use_exp, ratios in ((0, (2, 4, 8)), (1, (2, 4))):
        for v in ratios:
            for split in (0, 1):
                iters = 2000
                call = probe.bind_overlap(split, v, use_exp, iters, 512, fo, stream)
                us = _time_launches(call, steps, warmup, stream)
                # 512 blocks of 8 waves on 256 CUs: two wave pairs per SIMD, each
                # issuing 16 MFMAs per iteration
                cycles = us * 1e-6 * 2.4e9
                n_mfma = 2 * iters * 16
                ov.append({"valu": "exp" if use_exp else "fma", "valu_per_mfma": v,
                           "split_waves": bool(split), "us": round(us, 1),
                           "cycles_per_mfma_2.4GHz": round(cycles / n_mfma, 2)})
    res["overlap"] = ov
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--replicas", type=int, default=0, help="input copies to rotate over (0: auto)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true",
                    help="time only --workload (no secondary workloads in the line)")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="measured HBM bytes per launch (from rocprofv3 counters), if present")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run a plain device copy of this many bytes (counter calibration; "
                         "also reports its rate as the streaming context)")
    ap.add_argument("--pool-fill", type=float, default=0.0,
                    help="stress variant: grow the page pool to this fraction of the GPU's free "
                         "memory, the needed pages scattered over it (TLB and page-spread effects)")
    ap.add_argument("--write-path", action="store_true",
                    help="only time the paged-KV write path on the workload's page lists: each "
                         "request's newest token appended (decode) or its chunk written (prefill), "
                         "K and V pools, and a copy-on-write page copy per request")
    ap.add_argument("--probe-read-bytes", type=int, default=0,
                    help="only run the tile-read microbenchmark over a pool of this many bytes (every 4 KB tile "
                         "read once per launch, random order), with the suffix pass's non-temporal loads "
                         "(--probe-plain-loads: ordinary loads): a known-size read for scaling HBM counters")
    ap.add_argument("--probe-plain-loads", action="store_true")
    ap.add_argument("--probe", action="store_true",
                    help="only run the context microbenchmarks: random 4 KB tile reads with the suffix "
                         "pass's loads, the bf16 MFMA rate and the v_exp_f32 rate")
    ap.add_argument("--gather", action="store_true",
                    help="only time the page gather of the workload's whole working set (every "
                         "segment, K and V pools) into dense token-major buffers")
    ap.add_argument("--no-decode-loop", action="store_true",
                    help="leave the decode-loop measurement out of the default line")
    ap.add_argument("--decode-loop", action="store_true",
                    help="only time a decode loop: per step one token more per request, the plan "
                         "update and upload, and the attention call (wall clock and GPU time)")
    args = ap.parse_args()
    if args.probe_read_bytes:
        if args.gpus != 1:
            print("bench.py measures one GPU only", file=sys.stderr)
            sys.exit(2)
        probe_read_bench(args)
        return
    if args.probe:
        if args.gpus != 1:
            print("bench.py measures one GPU only", file=sys.stderr)
            sys.exit(2)
        probe_bench(args)
        return
    if args.gather:
        if args.gpus != 1:
            print("bench.py measures one GPU only", file=sys.stderr)
            sys.exit(2)
        gather_bench(args)
        return
    if args.decode_loop:
        if args.gpus != 1:
            print("bench.py measures one GPU only", file=sys.stderr)
            sys.exit(2)
        decode_loop_bench(args)
        return
    if args.write_path:
        if args.gpus != 1:
            print("bench.py measures one GPU only", file=sys.stderr)
            sys.exit(2)
        write_path_bench(args)
        return
    if args.copy_bytes:
        import torch
        n = args.copy_bytes // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)   # the calibration dispatch
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 5
        print(json.dumps({"copy_bytes": n * 4, "copy_us": round(ms * 1e3, 2),
                          "copy_gbps_read_plus_write": round(2 * n * 4 / (ms / 1e3) / 1e9, 1)}), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the library has no multi-GPU path); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2509_02121_amd import halo

    halo.load_library(require_gpu=True)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    head = measure_workload(args.workload, args, dev, pool_fill=args.pool_fill,
                            with_cpu=not args.no_cpu_baseline, percentiles=True)
    secondary = {}
    if not args.no_secondary and not args.pool_fill:
        for name in SECONDARY_WORKLOADS:
            if name != args.workload:
                secondary[name] = measure_workload(name, args, dev, with_cpu=False, percentiles=False)

    w = head.pop("_workload")
    line = {
        "metric": "shared-prefix attention: query-tokens/s + effective HBM GB/s (% roofline)",
        "value": head["value"],
        "unit": "query-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "gpu_ms_per_step": head["gpu_ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic",
        "per_call_us": head["per_call_us"],
        "effective_hbm_gbps": head["effective_hbm_gbps"],
        "hbm_roofline_frac": head["hbm_roofline_frac"],
        "config": head["config"],
        "host_plan": head["host_plan"],
        "roofline": head["roofline"],
        "cpu_baseline": head["cpu_baseline"],
    }
    if head["cpu_baseline"]:
        line["speedup_vs_oracle"] = round(head["value"] / head["cpu_baseline"]["value"], 1)
    if secondary:
        line["secondary"] = {k: {f: v[f] for f in ("value", "unit", "dtype", "ms_per_step", "gpu_ms_per_step",
                                                   "effective_hbm_gbps", "config", "host_plan", "roofline")}
                             for k, v in secondary.items()}
    del w
    if not (args.no_secondary or args.no_decode_loop or args.pool_fill or w_is_prefill(args.workload)):
        # the same batch as a decode loop (a token per request and step, the
        # plan updated in place and uploaded beside the running kernels);
        # last, since its copy stream slows the small secondary calls after it
        secondary.clear()
        torch.cuda.empty_cache()
        line["decode_loop"] = decode_loop_measure(args.workload, 100, 10)
    print(json.dumps(line), flush=True)


def _plan_timing(halo, params, csr, device_meta, stream, repeats=7):
    """Host cost of one batch step's plan: halo_plan_create (median of
    `repeats` runs on this host) and the metadata upload (HIP events on the
    stream around halo_plan_upload from pageable host memory)."""
    import torch
    ts = []
    plan = None
    for _ in range(repeats):
        t0 = time.perf_counter()
        plan = halo.Plan.from_csr(params, csr)
        ts.append((time.perf_counter() - t0) * 1e3)
    ts.sort()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    ups = []
    for _ in range(3):
        torch.cuda.synchronize()
        e0.record(stream)
        plan.upload(device_meta, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ups.append(e0.elapsed_time(e1) * 1e3)
    ups.sort()
    res = {"plan_ms": round(ts[len(ts) // 2], 4), "plan_ms_min": round(ts[0], 4), "repeats": repeats,
           "meta_upload_bytes": int(plan.device_meta_bytes), "upload_us": round(ups[1], 1),
           "workspace_bytes": int(plan.workspace_bytes)}
    if csr.get("q_len") is None:
        # decode-append update: the next step's forest with one token more
        # in every private segment, a fresh page (id 0 stands in) for each
        # segment whose last page is full
        import numpy as np
        refs = np.bincount(csr["req_seg_ids"], minlength=len(csr["seg_len"]))
        grow = (refs == 1).astype(np.int32)
        base = np.asarray(csr["seg_len"], np.int32)
        indptr = np.asarray(csr["seg_page_indptr"], np.int32)
        opens = (base + grow + 15) // 16 > np.diff(indptr)
        nxt = dict(csr)
        nxt["seg_len"] = base + grow
        nxt["seg_page_ids"] = np.insert(np.asarray(csr["seg_page_ids"], np.int32), indptr[1:][opens], 0)
        nxt["seg_page_indptr"] = np.concatenate([[0], np.cumsum(np.diff(indptr) + opens)]).astype(np.int32)
        us = []
        for k in range(repeats):
            # alternately one token more and the plan's own forest again
            t0 = time.perf_counter()
            ok = plan.update_lengths(nxt if k % 2 == 0 else csr)
            us.append((time.perf_counter() - t0) * 1e3)
            assert ok
        us.sort()
        res.update({"update_ms": round(us[len(us) // 2], 4), "update_segments": int(grow.sum()),
                    "update_pages_opened": int(opens.sum()), "private_segments": int((refs == 1).sum())})
    return res


def w_is_prefill(name):
    """Whether the named workload is a prefill batch."""
    import numpy as np
    from workloads import synth
    index = synth.CONFIG_NAMES.index(name)
    return synth._forest(index, np.random.Generator(np.random.PCG64(1000 + index)))[2] is not None


def _decode_loop_pages(name, n_steps):
    """Spare pages a decode loop of n_steps steps needs: every private
    segment opens a page every 16 steps."""
    import numpy as np
    from workloads import synth
    index = synth.CONFIG_NAMES.index(name)
    seg_len, paths, _ = synth._forest(index, np.random.Generator(np.random.PCG64(1000 + index)))
    refs = np.bincount(np.concatenate([np.asarray(p) for p in paths]), minlength=len(seg_len))
    return int((refs == 1).sum()) * (n_steps // 16 + 2)


def decode_loop_bench(args):
    """`--decode-loop`: decode_loop_measure on --workload, one JSON line."""
    import sys as _sys
    d = decode_loop_measure(args.workload, args.steps, args.warmup)
    if d is None:
        _sys.exit(2)
    print(json.dumps({"metric": "decode loop: time per step (plan update + metadata upload + attention call)",
                      "value": d.pop("ms_per_step"), "unit": "ms/step", "higher_is_better": False, "n_gpus": 1,
                      "steps": args.steps, "warmup": args.warmup, **d}), flush=True)


def decode_loop_measure(workload, steps, warmup):
    """A decode loop: each step every request appends one
    token to its private suffix (a spare page of the pool when its last page
    is full), the plan follows (halo_plan_update_lengths, a new plan when
    that refuses), its metadata is uploaded into the buffer the running step
    does not read (a copy stream of its own), and the attention call runs.
    The step forests are built before the timed region: they are the
    serving system's state, not the library's work. Timed: `steps` steps,
    wall clock on the host (update + upload + call, so host work that does
    not overlap the GPU shows) and HIP events on the compute stream. The new
    tokens' K/V are not written (the pool's seeded values stand in; the
    work does not depend on them)."""
    import numpy as np
    import torch
    from paper_2509_02121_amd import halo
    from workloads import make_config

    halo.load_library(require_gpu=True)
    dev = torch.device("cuda", 0)
    n_steps = warmup + steps
    w = make_config(workload, device=dev, poison=False, extra_pages=_decode_loop_pages(workload, n_steps))
    if w.is_prefill:
        print("--decode-loop needs a decode workload", file=sys.stderr)
        return None
    params = halo.make_params(w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype, w.num_pool_pages,
                              w.scale, w.dtype)
    csr0 = w.forest_csr()
    refs = np.bincount(csr0["req_seg_ids"], minlength=len(csr0["seg_len"]))
    grow = (refs == 1).astype(np.int64)
    used = np.zeros(w.num_pool_pages, bool)
    used[csr0["seg_page_ids"]] = True
    free = np.nonzero(~used)[0].astype(np.int32)
    lens = np.asarray(csr0["seg_len"], np.int64)
    ip = np.asarray(csr0["seg_page_indptr"], np.int64)
    ids = np.asarray(csr0["seg_page_ids"], np.int32)
    nf, forests = 0, []
    for _ in range(n_steps):
        opens = (lens + grow + 15) // 16 > np.diff(ip)
        k = int(opens.sum())
        if nf + k > len(free):
            print("--decode-loop: the pool has too few spare pages for that many steps", file=sys.stderr)
            return None
        ids = np.insert(ids, ip[1:][opens], free[nf:nf + k])
        nf += k
        ip = np.concatenate([[0], np.cumsum(np.diff(ip) + opens)])
        lens = lens + grow
        forests.append(dict(csr0, seg_len=lens.astype(np.int32), seg_page_indptr=ip.astype(np.int32),
                            seg_page_ids=ids))
    runner = halo.PrefixAttention(params, csr0, dev)
    o, lse = runner.alloc_outputs(w.q)
    stream = torch.cuda.current_stream()
    host_ms, applied = [], 0

    def step(i):
        t0 = time.perf_counter()
        ok = runner.update(forests[i])
        host_ms.append((time.perf_counter() - t0) * 1e3)
        runner.run(w.q, w.k_pool, w.v_pool, o, lse)
        return ok

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    host_ms.clear()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for i in range(warmup, n_steps):
        applied += int(step(i))
    e1.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    gpu = e0.elapsed_time(e1) / steps
    host_ms.sort()
    # the batch grows by a token per request and step: the attention call
    # alone on the timed region's first and last forest, for reference
    ref = []
    for f in (forests[warmup], forests[-1]):
        pa = halo.PrefixAttention(params, f, dev)
        ref.append(_time_launches(pa.bind(w.q, w.k_pool, w.v_pool, o, lse, stream), 20, 5, stream) / 1e3)
        del pa
    return {"ms_per_step": round(wall, 5), "gpu_ms_per_step": round(gpu, 5),
            "host_update_ms_median": round(host_ms[len(host_ms) // 2], 4),
            "attention_only_ms_first_last": [round(x, 5) for x in ref],
            "overhead_vs_attention_only": round(gpu / (0.5 * (ref[0] + ref[1])) - 1, 4),
            "steps_updated_in_place": applied, "pages_opened": int(nf),
            "dtype": "bf16" if w.dtype.itemsize == 2 else "f32", "data": "synthetic",
            "config": {"workload": w.name, "requests": len(w.req_paths), "steps": steps}}


def measure_workload(name, args, dev, pool_fill=0.0, with_cpu=False, percentiles=False):
    """Time one workload's library call (one step = one call over the whole
    batch) and derive its roofline figures."""
    import torch
    from paper_2509_02121_amd import halo
    from workloads import make_config

    w = make_config(name, device=dev)
    if pool_fill > 0:
        # same forest and values, in a pool of pool_fill x (free memory): the
        # needed pages land at random over the whole pool
        page_bytes = (w.k_pool[0].numel() + w.v_pool[0].numel()) * w.k_pool.element_size()
        have = w.num_pool_pages
        del w
        torch.cuda.empty_cache()
        free = torch.cuda.mem_get_info(dev)[0]
        target = int(pool_fill * free) // page_bytes
        w = make_config(name, device=dev, extra_pages=max(0, target - have))
    params = halo.make_params(w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype, w.num_pool_pages,
                              w.scale, w.dtype)
    csr = w.forest_csr()
    runner = halo.PrefixAttention(params, csr, dev)
    stats = runner.plan.stats()
    stream = torch.cuda.current_stream()
    host_plan = _plan_timing(halo, params, csr, runner.meta, stream)

    pool_bytes = (w.k_pool.numel() + w.v_pool.numel()) * w.k_pool.element_size()
    n_rep = args.replicas or max(1, min(16, -(-4 * MALL_BYTES // max(pool_bytes, 1))))
    reps = [(w.q, w.k_pool, w.v_pool)]
    for _ in range(n_rep - 1):
        reps.append((w.q.clone(), w.k_pool.clone(), w.v_pool.clone()))
    outs = [runner.alloc_outputs(w.q) for _ in range(n_rep)]

    calls = [runner.bind(reps[i][0], reps[i][1], reps[i][2], outs[i][0], outs[i][1], stream)
             for i in range(n_rep)]

    def step(i):
        calls[i % n_rep]()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall_ms = (t1 - t0) * 1e3 / args.steps
    gpu_ms = ev0.elapsed_time(ev1) / args.steps

    per_call_us = None
    if percentiles:
        # spread of single calls (a separate pass, one event pair per call)
        pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                 for _ in range(min(args.steps, 200))]
        for i, (a, b) in enumerate(pairs):
            a.record(stream)
            step(i)
            b.record(stream)
        torch.cuda.synchronize()
        per_call = sorted(a.elapsed_time(b) * 1e3 for a, b in pairs)
        pct = lambda f: round(per_call[min(len(per_call) - 1, int(f * len(per_call)))], 2)
        per_call_us = {"p10": pct(0.1), "median": pct(0.5), "p90": pct(0.9), "calls": len(per_call)}

    q_tokens = w.q.shape[0]
    alg_bytes = algorithmic_bytes(w, stats)
    value = q_tokens / (wall_ms / 1e3)
    eff_gbps = alg_bytes / (wall_ms / 1e3) / 1e9

    # Measured HBM bytes per call (calibrated rocprofv3 FETCH_SIZE + WRITE_SIZE),
    # valid only while the kernel and planner sources are the ones the
    # counters were taken on.
    traffic = None
    try:
        with open(args.traffic_json) as f:
            tr = json.load(f)
        sha = source_sha256()
        if tr.get("_kernel_source_sha256") == sha and w.name in tr and not pool_fill:
            traffic = tr[w.name]["bytes_per_call"]
    except (OSError, ValueError, KeyError):
        traffic = None

    kernels = []
    if stats["num_wide_items"] or stats["num_items"]:
        kernels.append("attn_kernel")
    if stats["num_merge_rows"]:
        kernels.append("merge_kernel")
    kernel_desc = " + ".join(kernels) + (" (one library call; time = all of its kernels)" if len(kernels) > 1 else "")

    if w.is_prefill:
        flops = 4 * w.head_dim * stats["visible_pairs"]
        achieved = flops / (gpu_ms / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": BF16_MFMA_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / BF16_MFMA_PEAK_TFLOPS, 4),
                "traffic": traffic, "kernel": kernel_desc, "algorithmic_flops": flops}
    else:
        achieved = alg_bytes / (gpu_ms / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                "kernel": kernel_desc, "algorithmic_bytes": alg_bytes}

    cpu = cpu_baseline(w, args.cpu_seconds) if with_cpu else None
    res = {
        "value": round(value, 1),
        "unit": "query-tokens/s",
        "dtype": "bf16" if w.dtype == torch.bfloat16 else "f32",
        "ms_per_step": round(wall_ms, 5),
        "gpu_ms_per_step": round(gpu_ms, 5),
        "per_call_us": per_call_us,
        "effective_hbm_gbps": round(eff_gbps, 1),
        "hbm_roofline_frac": round(eff_gbps / HBM_PEAK_GBPS, 4),
        "config": {"workload": w.name, "requests": w.num_requests, "query_tokens": q_tokens,
                   "num_q_heads": w.num_q_heads, "num_kv_heads": w.num_kv_heads,
                   "head_dim": w.head_dim, "page_size": w.page_size,
                   "distinct_kv_tokens": stats["distinct_kv_tokens"], "replicas": n_rep,
                   "work_items": stats["num_items"], "wide_items": stats["num_wide_items"],
                   "merge_rows": stats["num_merge_rows"], "partial_rows": stats["num_partial_rows"],
                   "pool_gb": round(pool_bytes / 1e9, 2), "pool_pages": int(w.num_pool_pages)},
        "host_plan": host_plan,
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    # free the device memory of this workload before the next one
    del calls, outs, reps, runner
    if with_cpu or percentiles:
        res["_workload"] = w
    else:
        del w
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


if __name__ == "__main__":
    main()
