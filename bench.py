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
DEFAULT_WORKLOAD = "llama8b_decode"
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


def cpu_baseline(w, min_seconds=10.0):
    """The fp64 oracle on the host cores over the same batch (decode: the
    whole batch, repeated until min_seconds; prefill: whole requests until
    min_seconds)."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    seg_k, seg_v = {}, {}
    for s in range(len(w.seg_len)):
        k, v = w.segment_kv(s)
        seg_k[s] = k.double().numpy()
        seg_v[s] = v.double().numpy()
    q = w.q.double().cpu().numpy()
    tokens = 0
    passes = 0
    t0 = time.perf_counter()
    if not w.is_prefill:
        while True:
            oracle.decode(q, seg_k, seg_v, w.req_paths, w.scale)
            tokens += w.num_requests
            passes += 1
            if time.perf_counter() - t0 >= min_seconds:
                break
        sample = f"whole {w.num_requests}-request batch x {passes} pass(es)"
    else:
        r = 0
        while True:
            a, b = w.q_rows_of_request(r)
            oracle.prefill(q[a:b], w.q_len[r:r + 1], seg_k, seg_v, [w.req_paths[r]], w.scale)
            tokens += b - a
            passes += 1
            r = (r + 1) % w.num_requests
            if time.perf_counter() - t0 >= min_seconds:
                break
        sample = f"{passes} request(s) of {int(w.q_len[0])} new tokens each"
    dt = time.perf_counter() - t0
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:  # pragma: no cover
        pass
    return {"value": tokens / dt, "unit": "query-tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": sample, "seconds": round(dt, 3),
            "host_cpus": len(os.sched_getaffinity(0)), "os_cpu_count": os.cpu_count(),
            "cpu_model": model, "blas_threads": int(threads)}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--replicas", type=int, default=0, help="input copies to rotate over (0: auto)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="measured HBM bytes per launch (from rocprofv3 counters), if present")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run a plain device copy of this many bytes (counter calibration; "
                         "also reports its rate as the streaming context)")
    ap.add_argument("--pool-fill", type=float, default=0.0,
                    help="stress variant: grow the page pool to this fraction of the GPU's free "
                         "memory, the needed pages scattered over it (TLB and page-spread effects)")
    args = ap.parse_args()
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
        print(f"bench.py measures one GPU only (this build has no multi-GPU path); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2509_02121_amd import halo
    from workloads import make_config

    halo.load_library(require_gpu=True)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = make_config(args.workload, device=dev)
    if args.pool_fill > 0:
        # same forest and values, in a pool of pool_fill x (free memory): the
        # needed pages land at random over the whole pool
        page_bytes = (w.k_pool[0].numel() + w.v_pool[0].numel()) * w.k_pool.element_size()
        have = w.num_pool_pages
        del w
        torch.cuda.empty_cache()
        free = torch.cuda.mem_get_info(dev)[0]
        target = int(args.pool_fill * free) // page_bytes
        w = make_config(args.workload, device=dev, extra_pages=max(0, target - have))
    params = halo.make_params(w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype, w.num_pool_pages,
                              w.scale, w.dtype)
    runner = halo.PrefixAttention(params, w.forest_csr(), dev)
    stats = runner.plan.stats()

    pool_bytes = (w.k_pool.numel() + w.v_pool.numel()) * w.k_pool.element_size()
    n_rep = args.replicas or max(1, min(16, -(-4 * MALL_BYTES // max(pool_bytes, 1))))
    reps = [(w.q, w.k_pool, w.v_pool)]
    for _ in range(n_rep - 1):
        reps.append((w.q.clone(), w.k_pool.clone(), w.v_pool.clone()))
    outs = [runner.alloc_outputs(w.q) for _ in range(n_rep)]
    stream = torch.cuda.current_stream()

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

    # Spread of single calls (a separate pass, one event pair per call).
    per_call = []
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(min(args.steps, 200))]
    for i, (a, b) in enumerate(pairs):
        a.record(stream)
        step(i)
        b.record(stream)
    torch.cuda.synchronize()
    per_call = sorted(a.elapsed_time(b) * 1e3 for a, b in pairs)
    pct = lambda f: round(per_call[min(len(per_call) - 1, int(f * len(per_call)))], 2)

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
        if tr.get("_kernel_source_sha256") == sha and w.name in tr and not args.pool_fill:
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

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args.cpu_seconds)

    line = {
        "metric": "shared-prefix attention: query-tokens/s + effective HBM GB/s (% roofline)",
        "value": round(value, 1),
        "unit": "query-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms, 5),
        "gpu_ms_per_step": round(gpu_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == torch.bfloat16 else "f32",
        "data": "synthetic",
        "per_call_us": {"p10": pct(0.1), "median": pct(0.5), "p90": pct(0.9), "calls": len(per_call)},
        "effective_hbm_gbps": round(eff_gbps, 1),
        "hbm_roofline_frac": round(eff_gbps / HBM_PEAK_GBPS, 4),
        "config": {"workload": w.name, "requests": w.num_requests, "query_tokens": q_tokens,
                   "num_q_heads": w.num_q_heads, "num_kv_heads": w.num_kv_heads,
                   "head_dim": w.head_dim, "page_size": w.page_size,
                   "distinct_kv_tokens": stats["distinct_kv_tokens"], "replicas": n_rep,
                   "work_items": stats["num_items"], "merge_rows": stats["num_merge_rows"],
                   "pool_gb": round(pool_bytes / 1e9, 2), "pool_pages": int(w.num_pool_pages)},
        "roofline": roof,
        "cpu_baseline": cpu,
    }
    if cpu:
        line["speedup_vs_oracle"] = round(value / cpu["value"], 1)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
