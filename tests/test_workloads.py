"""CPU checks of the seeded workload generator (structure, determinism)."""

import numpy as np
import torch

from workloads import CONFIG_NAMES, make_config, random_forest


def test_tiny_config_structure_and_determinism():
    a = make_config(0)
    b = make_config(0)
    assert a.num_q_heads == 4 and a.num_kv_heads == 4 and a.head_dim == 64
    assert a.dtype == torch.float32
    assert a.seg_len[0] == 256 and len(a.req_paths) == 8
    assert all(16 <= n <= 64 for n in a.seg_len[1:])
    # exact pool: every page used exactly once
    allp = np.concatenate(a.seg_pages)
    assert sorted(allp.tolist()) == list(range(a.num_pool_pages))
    assert torch.equal(a.q, b.q)
    assert torch.equal(torch.nan_to_num(a.k_pool), torch.nan_to_num(b.k_pool))
    c = make_config(0, seed=77)
    assert not torch.equal(a.q, c.q)


def test_llama8b_decode_structure():
    w = make_config(1)
    assert (w.num_q_heads, w.num_kv_heads, w.head_dim) == (32, 8, 128)
    assert w.dtype == torch.bfloat16
    assert w.seg_len[0] == 2048 and len(w.req_paths) == 64
    assert all(64 <= n <= 512 for n in w.seg_len[1:])
    needed = sum(len(p) for p in w.seg_pages)
    assert w.num_pool_pages == int(np.ceil(1.25 * needed))
    allp = np.concatenate(w.seg_pages)
    assert len(set(allp.tolist())) == len(allp)


def test_prefill_structure():
    w = make_config(3)
    assert w.is_prefill and len(w.req_paths) == 32
    assert (w.q_len == 512).all() and w.q.shape == (32 * 512, 32, 128)
    assert all(p[0] == 0 and w.seg_len[p[-1]] == 512 for p in w.req_paths)


def test_forest_csr_roundtrip():
    w = make_config(0)
    csr = w.forest_csr()
    assert csr["seg_page_indptr"][-1] == len(csr["seg_page_ids"])
    for r, p in enumerate(w.req_paths):
        a, b = csr["req_seg_indptr"][r], csr["req_seg_indptr"][r + 1]
        assert csr["req_seg_ids"][a:b].tolist() == p


def test_random_forest_is_valid():
    rng = np.random.default_rng(0)
    for prefill in (False, True):
        seg_len, paths, q_len = random_forest(rng, 20, prefill=prefill)
        for p in paths:
            assert len(set(p)) == len(p)
            assert all(0 <= s < len(seg_len) for s in p)
        if prefill:
            assert all(seg_len[p[-1]] == q_len[i] for i, p in enumerate(paths))
            leaves = [p[-1] for p in paths]
            assert len(set(leaves)) == len(leaves)


def test_names():
    assert len(CONFIG_NAMES) == 5
