"""Shared helpers of the GPU parity tests: run the library through the C ABI
and evaluate the oracle on the same seeded inputs (logical arrays read back
out of the same pools by the generator, never from the library)."""

import numpy as np
import torch

import oracle
from paper_2509_02121_amd import halo

# Tolerances on O (max abs error), from the benchmark spec of the method:
# fp32 inputs 1e-4, bf16 inputs with fp32 accumulation 2e-2. The extra LSE
# and normalized-error bars are derived in the design notes.
TOL = {
    torch.float32: dict(o=1e-4, lse=1e-5, rel=1e-4),
    torch.bfloat16: dict(o=2e-2, lse=1e-3, rel=1e-2),
}


def params_of(w, out_dtype=None):
    return halo.make_params(w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype, w.num_pool_pages,
                            w.scale, out_dtype if out_dtype is not None else w.dtype)


def to_device(w, device="cuda"):
    w.k_pool = w.k_pool.to(device)
    w.v_pool = w.v_pool.to(device)
    w.q = w.q.to(device)
    return w


def run_library(w, out_dtype=None, device="cuda"):
    """The library on w's pools; returns (o float64 numpy, lse numpy, runner)."""
    to_device(w, device)
    pa = halo.PrefixAttention(params_of(w, out_dtype), w.forest_csr(), device)
    o, lse = pa.run(w.q, w.k_pool, w.v_pool)
    torch.cuda.synchronize()
    return o.double().cpu().numpy(), lse.double().cpu().numpy(), pa


def oracle_for(w, requests=None):
    """Oracle outputs for the given requests (default all), in q-row order of
    those requests: (o [rows, H_q, d], lse [rows, H_q], row indices)."""
    if requests is None:
        requests = range(w.num_requests)
    requests = list(requests)
    needed = sorted({s for r in requests for s in w.req_paths[r]})
    seg_k, seg_v = {}, {}
    for s in needed:
        k, v = w.segment_kv(s)
        seg_k[s] = k.double().numpy()
        seg_v[s] = v.double().numpy()
    q_all = w.q
    if not w.is_prefill:
        rows = np.array(requests, dtype=np.int64)
        q = q_all[torch.as_tensor(rows, device=q_all.device)].double().cpu().numpy()
        o, lse = oracle.decode(q, seg_k, seg_v, [w.req_paths[r] for r in requests], w.scale)
        return o, lse, rows
    rows = []
    for r in requests:
        a, b = w.q_rows_of_request(r)
        rows.extend(range(a, b))
    rows = np.array(rows, dtype=np.int64)
    q = q_all[torch.as_tensor(rows, device=q_all.device)].double().cpu().numpy()
    o, lse = oracle.prefill(q, w.q_len[requests], seg_k, seg_v, [w.req_paths[r] for r in requests],
                            w.scale)
    return o, lse, rows


def assert_parity(w, o_gpu, lse_gpu, o_ref, lse_ref, rows, label=""):
    """Element-by-element comparison of the library output rows with the oracle."""
    tol = TOL[w.dtype]
    o = o_gpu[rows]
    lse = lse_gpu[rows]
    assert np.isfinite(o).all(), f"{label}: non-finite output"
    err = np.abs(o - o_ref).max() if o.size else 0.0
    scale = max(np.abs(o_ref).max() if o.size else 0.0, 1e-30)
    assert err <= tol["o"], f"{label}: max abs err {err:.3e} > {tol['o']}"
    assert err / scale <= tol["rel"] or err <= 1e-6, f"{label}: normalized err {err / scale:.3e}"
    fin = np.isfinite(lse_ref)
    assert (np.isneginf(lse[~fin])).all(), f"{label}: rows without keys must have lse = -inf"
    assert (o[~fin] == 0).all(), f"{label}: rows without keys must be 0"
    if fin.any():
        lerr = np.abs(lse[fin] - lse_ref[fin]).max()
        assert lerr <= tol["lse"], f"{label}: lse err {lerr:.3e} > {tol['lse']}"
    return err
