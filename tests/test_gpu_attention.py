"""GPU parity of decode and chunked prefill against the fp64 oracle, through
the C ABI, on the seeded workloads (full size, every row or sampled rows),
random forests, edge cases and invariances."""

import numpy as np
import pytest
import torch

from gpu_helpers import assert_parity, oracle_for, params_of, run_library, to_device
from paper_2509_02121_amd import halo
from workloads import build_workload, make_config, random_forest

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def test_tiny_decode_fp32(gpu_lib):
    _say("case: tiny_decode_fp32 (fp32, d 64, 4/4 heads)")
    w = make_config(0)
    o, lse, _ = run_library(w)
    ro, rl, rows = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rows, "tiny")


@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32])
def test_llama8b_decode_full(gpu_lib, out_dtype):
    _say(f"case: llama8b_decode out={out_dtype}")
    w = make_config(1)
    o, lse, pa = run_library(w, out_dtype)
    ro, rl, rows = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rows, "llama8b")
    assert pa.plan.stats()["num_shared_items"] > 0


def test_two_level_tree_decode_full(gpu_lib):
    _say("case: two_level_tree_decode")
    w = make_config(2)
    o, lse, _ = run_library(w)
    ro, rl, rows = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rows, "two-level")


def test_llama70b_batch_decode_sampled(gpu_lib):
    """Full-size 1024-request batch on the GPU; 24 sampled requests (3 per
    prefix group) through the oracle."""
    _say("case: llama70b_batch_decode (full size, sampled rows)")
    w = make_config(4, device="cuda")
    o, lse, _ = run_library(w)
    rng = np.random.default_rng(0)
    sample = sorted(int(g * 128 + x) for g in range(8) for x in rng.choice(128, 3, replace=False))
    ro, rl, rows = oracle_for(w, sample)
    assert_parity(w, o, lse, ro, rl, rows, "70b")
    # every row finite, every lse finite (every request sees keys)
    assert np.isfinite(o).all() and np.isfinite(lse).all()


def test_chunked_prefill_sampled(gpu_lib):
    """Full-size prefill (32 x 512 new tokens over a 4096-token prefix); three
    whole requests through the oracle."""
    _say("case: chunked_prefill (full size, 3 requests)")
    w = make_config(3)
    o, lse, _ = run_library(w)
    ro, rl, rows = oracle_for(w, [0, 13, 31])
    assert_parity(w, o, lse, ro, rl, rows, "prefill")
    assert np.isfinite(o).all()


@pytest.mark.parametrize("seed", range(10))
def test_random_forests(gpu_lib, seed):
    rng = np.random.default_rng(1000 + seed)
    prefill = seed % 3 == 2
    hkv = int(rng.choice([1, 2, 3]))
    group = int(rng.choice([1, 2, 4, 8, 16]))
    d = int(rng.choice([64, 128]))
    dtype = torch.bfloat16 if seed % 2 else torch.float32
    out = torch.float32 if (seed // 2) % 2 else dtype
    seg_len, paths, q_len = random_forest(rng, int(rng.integers(1, 14)), max_len=300,
                                          prefill=prefill, max_q=70)
    _say(f"case: random forest seed={seed} prefill={prefill} hkv={hkv} G={group} d={d} {dtype} "
         f"segs={seg_len}")
    w = build_workload("rf", 2000 + seed, hkv * group, hkv, d, dtype, seg_len, paths, q_len,
                       value_scale=1.0 if dtype == torch.float32 else 0.5)
    o, lse, _ = run_library(w, out)
    ro, rl, rows = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rows, f"rf{seed}")


def test_edge_cases_empty_and_one_token(gpu_lib):
    """Empty segments, a request with no keys, one-token segments, a request
    whose only keys are one shared segment (mixed with requests that have
    suffixes), and ragged page tails."""
    _say("case: edge cases")
    seg_len = [0, 1, 17, 33, 0, 1, 250]
    paths = [[0], [1], [2, 3], [2], [2, 4], [], [2, 5], [6, 1]]
    for dtype in (torch.float32, torch.bfloat16):
        w = build_workload("edge", 5, 8, 2, 128, dtype, seg_len, paths)
        o, lse, _ = run_library(w)
        ro, rl, rows = oracle_for(w)
        assert_parity(w, o, lse, ro, rl, rows, f"edge {dtype}")
        assert (o[0] == 0).all() and np.isneginf(lse[0]).all()
        assert (o[5] == 0).all() and np.isneginf(lse[5]).all()


def test_long_segment_and_wide_batch(gpu_lib):
    """A 20000-token private suffix (many key chunks) and 600 requests on one
    prefix with G = 8 (many stacked row blocks)."""
    _say("case: long segment / wide batch")
    rng = np.random.default_rng(3)
    seg_len = [700] + [20000] + list(rng.integers(1, 40, size=600))
    paths = [[0, 1]] + [[0, 2 + i] for i in range(600)]
    w = build_workload("wide", 9, 16, 2, 128, torch.bfloat16, seg_len, paths, value_scale=0.5)
    o, lse, _ = run_library(w)
    sample = [0, 1, 2, 77, 300, 599, 600]
    ro, rl, rows = oracle_for(w, sample)
    assert_parity(w, o, lse, ro, rl, rows, "wide")


def test_prefill_edge_cases(gpu_lib):
    """Prefill with an empty prefix, a one-token chunk, a chunk shorter than
    a row block, a zero-query request, and a two-level prefix."""
    _say("case: prefill edges")
    seg_len = [100, 3, 1, 40, 0, 64, 5, 200]
    paths = [[0, 1], [2], [0, 3], [4], [0, 5, 6], [7]]
    q_len = [3, 1, 40, 0, 5, 200]
    for dtype, g in ((torch.float32, 4), (torch.bfloat16, 8), (torch.bfloat16, 1)):
        w = build_workload("pedge", 6, 2 * g, 2, 64, dtype, seg_len, paths, q_len)
        o, lse, _ = run_library(w)
        ro, rl, rows = oracle_for(w)
        assert_parity(w, o, lse, ro, rl, rows, f"prefill edge {dtype} G={g}")


def test_structured_inputs_detect_dropped_segments(gpu_lib):
    """Peaked softmax (Q x 8) and a per-segment constant added to V, so a
    dropped or duplicated segment would move O by ~1, far outside tolerance."""
    _say("case: structured inputs")
    w = make_config(1)
    w.q = (w.q.float() * 8).to(torch.bfloat16)
    for s in range(len(w.seg_len)):
        pages = torch.as_tensor(np.asarray(w.seg_pages[s], np.int64))
        w.v_pool[pages] = (w.v_pool[pages].float() + (s % 5) - 2).to(torch.bfloat16)
    o, lse, _ = run_library(w)
    ro, rl, rows = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rows, "structured")


def _flatten(w):
    """The same logical tokens with every request owning private copies of
    its prefix segments (no sharing at all)."""
    seg_len, paths = [], []
    src = []
    for path in w.req_paths:
        p = []
        for s in path:
            seg_len.append(int(w.seg_len[s]))
            src.append(s)
            p.append(len(seg_len) - 1)
        paths.append(p)
    f = build_workload("flat", 1, w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype, seg_len, paths,
                       device=w.k_pool.device)
    for new, old in enumerate(src):
        n = int(w.seg_len[old])
        for t0 in range(0, n, 16):
            po = int(w.seg_pages[old][t0 // 16])
            pn = int(f.seg_pages[new][t0 // 16])
            f.k_pool[pn] = w.k_pool[po]
            f.v_pool[pn] = w.v_pool[po]
    f.q = w.q.clone()
    return f


def test_shared_equals_unshared(gpu_lib):
    """§3 "Scope": sharing must not change the result. The shared-prefix run
    and the fully private (flattened) run agree within the bf16 tolerance,
    and both match the oracle."""
    _say("case: shared == unshared")
    w = to_device(make_config(1))
    o_s, lse_s, pa = run_library(w)
    f = _flatten(w)
    o_u, lse_u, pb = run_library(f)
    assert pb.plan.stats()["num_shared_items"] == 0
    assert np.abs(o_s - o_u).max() <= 2e-2
    assert np.abs(lse_s - lse_u).max() <= 1e-3
    ro, rl, rows = oracle_for(w)
    assert_parity(f, o_u, lse_u, ro, rl, rows, "unshared")


def test_page_placement_and_repeat_are_bitwise(gpu_lib):
    """Moving pages to other pool slots, or running twice, gives bit-identical
    results (the reduction order depends only on logical key positions)."""
    _say("case: placement shuffle / determinism")
    w = to_device(make_config(1))
    o1, l1, pa = run_library(w)
    o1b, l1b = pa.run(w.q, w.k_pool, w.v_pool)
    torch.cuda.synchronize()
    assert np.array_equal(o1, o1b.double().cpu().numpy())
    # permute pool slots
    perm = torch.randperm(w.num_pool_pages, generator=torch.Generator().manual_seed(4))
    inv = torch.empty_like(perm)
    inv[perm] = torch.arange(len(perm))
    k2 = torch.empty_like(w.k_pool)
    v2 = torch.empty_like(w.v_pool)
    k2[perm.to(k2.device)] = w.k_pool
    v2[perm.to(v2.device)] = w.v_pool
    w2 = make_config(1)
    w2.k_pool, w2.v_pool, w2.q = k2, v2, w.q
    w2.seg_pages = [perm[torch.as_tensor(p.astype(np.int64))].numpy().astype(np.int32)
                    for p in w.seg_pages]
    o2, l2, _ = run_library(w2)
    assert np.array_equal(o1, o2) and np.array_equal(np.nan_to_num(l1), np.nan_to_num(l2))


def test_request_permutation(gpu_lib):
    _say("case: request permutation")
    w = to_device(make_config(1))
    o1, l1, _ = run_library(w)
    perm = np.random.default_rng(2).permutation(w.num_requests)
    w.req_paths = [w.req_paths[i] for i in perm]
    w.q = w.q[torch.as_tensor(perm, device=w.q.device)]
    o2, l2, _ = run_library(w)
    assert np.abs(o1[perm] - o2).max() <= 2e-2 and np.abs(l1[perm] - l2).max() <= 1e-3


def test_workspace_too_small_is_rejected(gpu_lib):
    w = to_device(make_config(0))
    pa = halo.PrefixAttention(params_of(w), w.forest_csr())
    o, lse = pa.alloc_outputs(w.q)
    small = torch.empty(pa.plan.workspace_bytes - 256, dtype=torch.uint8, device="cuda")
    # the binding refuses it before the call ...
    with pytest.raises(ValueError, match="workspace has"):
        halo.prefix_attn_decode(pa.plan, pa.meta, w.q, w.k_pool, w.v_pool, o, lse, small)
    # ... and so does the C ABI itself
    st = halo._LIB.halo_prefix_attn_decode(pa.plan._handle, pa.meta.data_ptr(), w.q.data_ptr(),
                                           w.k_pool.data_ptr(), w.v_pool.data_ptr(), o.data_ptr(),
                                           lse.data_ptr(), small.data_ptr(), small.numel(),
                                           halo._stream_handle(None))
    assert st == halo.HALO_ERR_WORKSPACE_TOO_SMALL
