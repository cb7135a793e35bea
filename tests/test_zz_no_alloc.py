"""The no-allocation decode entry point (halo_prefix_attn_decode_noalloc)
against the workspace entry point, through the C ABI, on two calls in a row
(the second on a smaller batch), plus its size limit."""

import numpy as np
import pytest
import torch

from gpu_helpers import assert_parity, oracle_for, params_of, to_device
from paper_2509_02121_amd import halo
from workloads import build_workload, make_config

pytestmark = pytest.mark.gpu


def _both(w):
    """Decode w through the workspace entry point and the no-alloc one; returns
    (o_ws, lse_ws, o_na, lse_na) as CPU tensors, and the plan."""
    to_device(w)
    pa = halo.PrefixAttention(params_of(w), w.forest_csr(), "cuda")
    assert 0 < pa.plan.workspace_bytes <= halo.NOALLOC_SCRATCH_BYTES
    o1, l1 = pa.alloc_outputs(w.q)
    o2, l2 = pa.alloc_outputs(w.q)
    o2.fill_(float("nan"))
    l2.fill_(float("nan"))
    pa.run(w.q, w.k_pool, w.v_pool, o1, l1)
    pa._before_run(None)
    halo.prefix_attn_decode_noalloc(pa.plan, pa.meta, w.q, w.k_pool, w.v_pool, o2, l2)
    torch.cuda.synchronize()
    return o1.cpu(), l1.cpu(), o2.cpu(), l2.cpu(), pa


def _bits(t):
    return t.contiguous().view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).numpy()


def test_noalloc_matches_workspace_decode_twice(gpu_lib):
    """First call: the Llama-8B-shaped decode (64 requests on a 2048-token
    prefix). Second call: a smaller batch (12 requests, other forest) that
    reuses the scratch left by the first. Each equals the workspace entry
    point bit for bit (same plan, same kernels) and meets the oracle bar."""
    print("case: no-alloc decode, llama8b then a 12-request batch", flush=True)
    big = make_config(1)
    o1, l1, o2, l2, _ = _both(big)
    assert np.array_equal(_bits(o1), _bits(o2))
    assert np.array_equal(_bits(l1), _bits(l2))
    ro, rl, rows = oracle_for(big)
    assert_parity(big, o2.double().numpy(), l2.double().numpy(), ro, rl, rows, "noalloc llama8b")

    rng = np.random.default_rng(5)
    seg_len = [700, 300] + [int(x) for x in rng.integers(1, 900, size=12)]
    paths = [[0, 2 + r] if r < 6 else [0, 1, 2 + r] for r in range(12)]
    small = build_workload("noalloc_small", 77, 16, 4, 128, torch.bfloat16, seg_len, paths, value_scale=0.5)
    o1, l1, o2, l2, pa = _both(small)
    assert pa.plan.workspace_bytes < 6 << 20
    assert np.array_equal(_bits(o1), _bits(o2))
    assert np.array_equal(_bits(l1), _bits(l2))
    ro, rl, rows = oracle_for(small)
    assert_parity(small, o2.double().numpy(), l2.double().numpy(), ro, rl, rows, "noalloc small")


def test_noalloc_rejects_a_plan_beyond_its_scratch(gpu_lib):
    """A plan needing more workspace than the scratch holds is refused by the
    C ABI before any launch (the 70B-shaped batch's forest with fp32 output,
    whose partials are fp32; host arrays only, the pointers are never
    dereferenced)."""
    print("case: no-alloc size limit", flush=True)
    rng = np.random.Generator(np.random.PCG64(1004))
    suffix = rng.integers(256, 2048, size=1024, endpoint=True)
    seg_len = np.asarray([8192] * 8 + list(suffix), np.int32)
    n_pages = (seg_len + 15) // 16
    indptr = np.zeros(len(seg_len) + 1, np.int32)
    indptr[1:] = np.cumsum(n_pages)
    csr = dict(seg_len=seg_len, seg_page_indptr=indptr, seg_page_ids=np.arange(indptr[-1], dtype=np.int32),
               req_seg_indptr=np.arange(0, 2049, 2, dtype=np.int32),
               req_seg_ids=np.array([x for r in range(1024) for x in (r // 128, 8 + r)], np.int32), q_len=None)
    plan = halo.Plan.from_csr(halo.make_params(64, 8, 128, torch.bfloat16, int(indptr[-1]), 0.0883883,
                                                torch.float32), csr)
    assert plan.workspace_bytes > halo.NOALLOC_SCRATCH_BYTES
    fake = 1 << 20
    st = halo._LIB.halo_prefix_attn_decode_noalloc(plan._handle, fake, fake, fake, fake, fake, None, None)
    assert st == halo.HALO_ERR_WORKSPACE_TOO_SMALL
    assert b"no-alloc" in halo._LIB.halo_last_error_message()
