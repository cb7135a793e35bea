"""Pins for the fp64 oracle (CPU only).

The paper prints no worked attention example, so each pin comes from the
mathematics: hand-derived cases, a pure-Python brute force, closed forms, a
library special case (torch's fp64 CPU scaled_dot_product_attention), the
exact merge identity behind prefix sharing (shared result == unshared result,
§3 "Scope"), and permutation / page-placement invariances. Each is chosen so
that a plausible slip in the oracle (a dropped scale, a wrong GQA index, a
flipped causal mask, a dropped segment, a transposed operand) fails one of
them.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from workloads import build_workload, make_config, random_forest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_worked.json")


def _brute_attend(q, k, v, scale, visible=None):
    """Pure-Python loops with math.fsum / math.exp (independent of numpy)."""
    n, d = len(q), len(q[0])
    t = len(k)
    outs, lses = [], []
    for i in range(n):
        scores = []
        for j in range(t):
            if visible is not None and not visible[i][j]:
                continue
            scores.append((j, scale * math.fsum(q[i][c] * k[j][c] for c in range(d))))
        if not scores:
            outs.append([0.0] * len(v[0]) if t else [0.0] * d)
            lses.append(-math.inf)
            continue
        m = max(s for _, s in scores)
        w = [(j, math.exp(s - m)) for j, s in scores]
        z = math.fsum(x for _, x in w)
        outs.append([math.fsum(x * v[j][c] for j, x in w) / z for c in range(len(v[0]))])
        lses.append(m + math.log(z))
    return outs, lses


def _brute_forest(q, seg_k, seg_v, paths, scale, q_len=None):
    """Brute-force decode/prefill over a forest, one (row, head) at a time."""
    h_q = len(q[0])
    outs = np.zeros((len(q), h_q, len(q[0][0])))
    lses = np.zeros((len(q), h_q))
    row = 0
    for r, path in enumerate(paths):
        keys = [tok for s in path for tok in seg_k[s]]
        vals = [tok for s in path for tok in seg_v[s]]
        n_q = 1 if q_len is None else int(q_len[r])
        n_prefix = len(keys) - (0 if q_len is None else n_q)
        h_kv = len(keys[0]) if keys else 1
        group = h_q // h_kv
        for i in range(n_q):
            for h in range(h_q):
                g = h // group
                kk = [tok[g] for tok in keys]
                vv = [tok[g] for tok in vals]
                vis = None
                if q_len is not None:
                    vis = [[j < n_prefix or (j - n_prefix) <= i for j in range(len(keys))]]
                o, l = _brute_attend([q[row + i][h]], kk, vv, scale, vis)
                outs[row + i, h] = o[0] if kk else 0.0
                lses[row + i, h] = l[0] if kk else -math.inf
        row += n_q
    return outs, lses


def _np_forest(rng, seg_len, h_kv, d):
    seg_k = [rng.standard_normal((n, h_kv, d)) for n in seg_len]
    seg_v = [rng.standard_normal((n, h_kv, d)) for n in seg_len]
    return seg_k, seg_v


# ---------------------------------------------------------------- hand-worked

def test_hand_worked_golden():
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        vis = None if c["visible"] is None else np.array(c["visible"])
        o, lse = oracle.attend(np.array(c["q"]), np.array(c["k"]), np.array(c["v"]),
                               c["scale"], vis)
        np.testing.assert_allclose(o, np.array(c["o"]), rtol=0, atol=1e-14, err_msg=c["name"])
        np.testing.assert_allclose(lse, np.array(c["lse"]), rtol=0, atol=1e-14, err_msg=c["name"])


# ---------------------------------------------------------------- brute force

@pytest.mark.parametrize("seed", range(6))
def test_attend_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    n, t, d = rng.integers(1, 5), rng.integers(1, 40), rng.integers(1, 9)
    q = rng.standard_normal((n, d))
    k = rng.standard_normal((t, d))
    v = rng.standard_normal((t, d))
    vis = rng.random((n, t)) < 0.7 if seed % 2 else None
    scale = 1.0 / math.sqrt(d)
    o, lse = oracle.attend(q, k, v, scale, vis)
    bo, bl = _brute_attend(q.tolist(), k.tolist(), v.tolist(), scale,
                           None if vis is None else vis.tolist())
    np.testing.assert_allclose(o, np.array(bo), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, np.array(bl), rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed,prefill,h_q,h_kv", [
    (0, False, 2, 1), (1, False, 2, 2), (2, True, 2, 1), (3, True, 4, 2), (4, False, 4, 2)])
def test_forest_matches_brute_force(seed, prefill, h_q, h_kv):
    rng = np.random.default_rng(100 + seed)
    d = 6
    seg_len, paths, q_len = random_forest(rng, 5, max_len=12, prefill=prefill, max_q=6)
    seg_k, seg_v = _np_forest(rng, seg_len, h_kv, d)
    rows = len(paths) if q_len is None else int(q_len.sum())
    q = rng.standard_normal((rows, h_q, d))
    scale = 0.37
    if prefill:
        o, lse = oracle.prefill(q, q_len, seg_k, seg_v, paths, scale)
    else:
        o, lse = oracle.decode(q, seg_k, seg_v, paths, scale)
    bo, bl = _brute_forest(q.tolist(), [x.tolist() for x in seg_k],
                           [x.tolist() for x in seg_v], paths, scale, q_len)
    np.testing.assert_allclose(o, bo, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(np.isinf(lse), np.isinf(bl))
    fin = np.isfinite(bl)
    np.testing.assert_allclose(lse[fin], bl[fin], rtol=0, atol=1e-12)


# ---------------------------------------------------------------- closed forms

def test_closed_form_equal_keys():
    rng = np.random.default_rng(7)
    t, d = 37, 8
    kvec = rng.standard_normal(d)
    k = np.tile(kvec, (t, 1))
    v = rng.standard_normal((t, d))
    q = rng.standard_normal((3, d))
    scale = 0.25
    o, lse = oracle.attend(q, k, v, scale)
    np.testing.assert_allclose(o, np.tile(v.mean(0), (3, 1)), atol=1e-13)
    np.testing.assert_allclose(lse, scale * (q @ kvec) + math.log(t), atol=1e-13)


def test_closed_form_zero_query():
    rng = np.random.default_rng(8)
    k = rng.standard_normal((20, 5))
    v = rng.standard_normal((20, 5))
    o, lse = oracle.attend(np.zeros((1, 5)), k, v, 3.0)
    np.testing.assert_allclose(o[0], v.mean(0), atol=1e-13)
    assert abs(lse[0] - math.log(20)) < 1e-13


def test_closed_form_single_key():
    rng = np.random.default_rng(9)
    q, k, v = rng.standard_normal((2, 4)), rng.standard_normal((1, 4)), rng.standard_normal((1, 4))
    o, lse = oracle.attend(q, k, v, 0.5)
    np.testing.assert_allclose(o, np.tile(v[0], (2, 1)), atol=1e-15)
    np.testing.assert_allclose(lse, 0.5 * (q @ k[0]), atol=1e-14)


def test_closed_form_planted_key():
    rng = np.random.default_rng(10)
    t, d = 50, 4
    k = rng.standard_normal((t, d)) * 0.01
    q = np.zeros((1, d))
    q[0, 0] = 1.0
    k[17] = 0.0
    k[17, 0] = 50.0        # score 50 above ~0 for the rest (scale 1)
    v = rng.standard_normal((t, d))
    o, _ = oracle.attend(q, k, v, 1.0)
    bound = t * math.exp(-49.0) * np.abs(v).max() * 2
    assert np.abs(o[0] - v[17]).max() <= bound


def test_empty_rows_and_requests():
    o, lse = oracle.attend(np.ones((2, 3)), np.zeros((0, 3)), np.zeros((0, 3)), 1.0)
    assert (o == 0).all() and np.isneginf(lse).all()
    vis = np.array([[False, False], [True, False]])
    o, lse = oracle.attend(np.ones((2, 3)), np.ones((2, 3)), np.ones((2, 3)) * 5, 1.0, vis)
    assert (o[0] == 0).all() and np.isneginf(lse[0])
    np.testing.assert_allclose(o[1], 5.0)
    # a request whose segments are all empty
    seg_k = [np.zeros((0, 1, 3)), np.ones((4, 1, 3))]
    seg_v = [np.zeros((0, 1, 3)), np.ones((4, 1, 3))]
    o, lse = oracle.decode(np.ones((2, 2, 3)), seg_k, seg_v, [[0], [0, 1]], 1.0)
    assert (o[0] == 0).all() and np.isneginf(lse[0]).all()
    np.testing.assert_allclose(o[1], 1.0)
    np.testing.assert_allclose(lse[1], 3.0 + math.log(4))


def test_softmax_rows_sum_to_one():
    rng = np.random.default_rng(11)
    q = rng.standard_normal((6, 16)) * 3
    k = rng.standard_normal((300, 16)) * 3
    v = rng.standard_normal((300, 16))
    vis = rng.random((6, 300)) < 0.5
    p = oracle.attention_probs(q, k, 0.25, vis)
    assert np.abs(p.sum(1) - 1).max() <= 1e-12
    assert (p[~vis] == 0).all()
    o, _ = oracle.attend(q, k, v, 0.25, vis)
    np.testing.assert_allclose(o, p @ v, atol=1e-12)


# ------------------------------------------------------ library special case

def _sdpa_reference(q, k, v, scale, g, mask=None):
    """torch fp64 CPU SDPA with K/V repeated to the q heads (h -> h // g)."""
    qt = torch.from_numpy(q).permute(1, 0, 2)                   # [H_q, n, d]
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(g, 0)
    vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(g, 0)
    m = None if mask is None else torch.from_numpy(mask)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=m, scale=scale)
    return o.permute(1, 0, 2).numpy()


@pytest.mark.parametrize("h_q,h_kv", [(4, 2), (8, 2), (3, 3)])
def test_decode_matches_torch_sdpa(h_q, h_kv):
    rng = np.random.default_rng(12 + h_q)
    d = 8
    seg_len, paths, _ = random_forest(rng, 6, max_len=30, allow_empty=False)
    seg_k, seg_v = _np_forest(rng, seg_len, h_kv, d)
    q = rng.standard_normal((len(paths), h_q, d))
    o, _ = oracle.decode(q, seg_k, seg_v, paths, 0.3)
    for r, path in enumerate(paths):
        k = np.concatenate([seg_k[s] for s in path])
        v = np.concatenate([seg_v[s] for s in path])
        ref = _sdpa_reference(q[r:r + 1], k, v, 0.3, h_q // h_kv)
        np.testing.assert_allclose(o[r:r + 1], ref, rtol=0, atol=1e-12)


def test_prefill_matches_torch_sdpa_with_mask():
    rng = np.random.default_rng(13)
    h_q, h_kv, d = 4, 2, 8
    seg_len = [20, 9, 13]
    paths = [[0, 1], [0, 2]]
    q_len = np.array([9, 13], np.int32)
    seg_k, seg_v = _np_forest(rng, seg_len, h_kv, d)
    q = rng.standard_normal((22, h_q, d))
    o, _ = oracle.prefill(q, q_len, seg_k, seg_v, paths, 0.2)
    row = 0
    for r, path in enumerate(paths):
        n = int(q_len[r])
        k = np.concatenate([seg_k[s] for s in path])
        v = np.concatenate([seg_v[s] for s in path])
        t = k.shape[0]
        mask = np.zeros((n, t), dtype=bool)
        for i in range(n):
            mask[i, : t - n + i + 1] = True
        ref = _sdpa_reference(q[row:row + n], k, v, 0.2, 2, mask)
        np.testing.assert_allclose(o[row:row + n], ref, rtol=0, atol=1e-12)
        row += n


def test_prefill_empty_prefix_is_causal_attention():
    rng = np.random.default_rng(14)
    seg_k, seg_v = _np_forest(rng, [11], 2, 8)
    q = rng.standard_normal((11, 2, 8))
    o, _ = oracle.prefill(q, np.array([11]), seg_k, seg_v, [[0]], 0.35)
    qt = torch.from_numpy(q).permute(1, 0, 2)
    kt = torch.from_numpy(seg_k[0]).permute(1, 0, 2)
    vt = torch.from_numpy(seg_v[0]).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True, scale=0.35)
    np.testing.assert_allclose(o, ref.permute(1, 0, 2).numpy(), rtol=0, atol=1e-12)


def test_last_prefill_row_equals_decode():
    rng = np.random.default_rng(15)
    seg_k, seg_v = _np_forest(rng, [40, 7], 2, 8)
    q = rng.standard_normal((7, 4, 8))
    op, lp = oracle.prefill(q, np.array([7]), seg_k, seg_v, [[0, 1]], 0.3)
    od, ld = oracle.decode(q[6:7], seg_k, seg_v, [[0, 1]], 0.3)
    np.testing.assert_allclose(op[6], od[0], atol=1e-12)
    np.testing.assert_allclose(lp[6], ld[0], atol=1e-12)


# --------------------------------------------- shared == unshared (§3 Scope)

def test_segmentwise_merge_equals_concatenated():
    """Attending segment by segment and merging the partials with the exact
    log-sum-exp rule gives the concatenated (unshared) result."""
    rng = np.random.default_rng(16)
    h_q, h_kv, d = 4, 2, 16
    seg_len, paths, _ = random_forest(rng, 8, max_len=50)
    seg_k, seg_v = _np_forest(rng, seg_len, h_kv, d)
    q = rng.standard_normal((len(paths), h_q, d))
    o, lse = oracle.decode(q, seg_k, seg_v, paths, 0.25)
    for r, path in enumerate(paths):
        parts_o, parts_l = [], []
        for s in path:
            po, pl = oracle.decode(q[r:r + 1], seg_k, seg_v, [[s]], 0.25)
            parts_o.append(po[0])
            parts_l.append(pl[0])
        if not path:
            continue
        mo, ml = oracle.merge_partials(np.stack(parts_o), np.stack(parts_l))
        np.testing.assert_allclose(mo, o[r], rtol=0, atol=1e-12)
        fin = np.isfinite(lse[r])
        assert (np.isfinite(ml) == fin).all()
        np.testing.assert_allclose(ml[fin], lse[r][fin], rtol=0, atol=1e-12)


def test_merge_rules():
    o1 = np.array([[[1.0, 2.0]]])
    l1 = np.array([[0.5]])
    mo, ml = oracle.merge_partials(o1, l1)
    assert (mo == o1[0]).all() and (ml == l1[0]).all()
    mo, ml = oracle.merge_partials(np.array([[[1.0, 1.0]], [[9.0, 9.0]]]),
                                   np.array([[0.0], [-np.inf]]))
    np.testing.assert_allclose(mo, [[1.0, 1.0]])
    np.testing.assert_allclose(ml, [0.0])
    mo, ml = oracle.merge_partials(np.ones((2, 1, 2)), np.full((2, 1), -np.inf))
    assert (mo == 0).all() and np.isneginf(ml).all()
    # two parts with equal lse: average, lse + ln 2
    mo, ml = oracle.merge_partials(np.array([[[0.0, 4.0]], [[2.0, 0.0]]]), np.array([[1.0], [1.0]]))
    np.testing.assert_allclose(mo, [[1.0, 2.0]], atol=1e-15)
    np.testing.assert_allclose(ml, [1.0 + math.log(2)], atol=1e-15)


def test_flattened_forest_is_bitwise_identical():
    """Giving every request private copies of its prefix segments (no
    sharing) leaves the oracle output bit-for-bit unchanged."""
    rng = np.random.default_rng(17)
    seg_len, paths, _ = random_forest(rng, 7, max_len=40)
    seg_k, seg_v = _np_forest(rng, seg_len, 2, 8)
    q = rng.standard_normal((len(paths), 4, 8))
    o, lse = oracle.decode(q, seg_k, seg_v, paths, 0.3)
    flat_k, flat_v, flat_paths = [], [], []
    for path in paths:
        p = []
        for s in path:
            flat_k.append(seg_k[s].copy())
            flat_v.append(seg_v[s].copy())
            p.append(len(flat_k) - 1)
        flat_paths.append(p)
    o2, lse2 = oracle.decode(q, flat_k, flat_v, flat_paths, 0.3)
    assert np.array_equal(o, o2) and np.array_equal(lse, lse2)


def test_request_permutation_is_bitwise():
    rng = np.random.default_rng(18)
    seg_len, paths, _ = random_forest(rng, 9, max_len=30)
    seg_k, seg_v = _np_forest(rng, seg_len, 2, 8)
    q = rng.standard_normal((len(paths), 4, 8))
    o, lse = oracle.decode(q, seg_k, seg_v, paths, 0.3)
    perm = rng.permutation(len(paths))
    o2, lse2 = oracle.decode(q[perm], seg_k, seg_v, [paths[i] for i in perm], 0.3)
    assert np.array_equal(o[perm], o2) and np.array_equal(lse[perm], lse2)


def test_key_order_invariance_in_decode():
    rng = np.random.default_rng(19)
    k = rng.standard_normal((64, 1, 8))
    v = rng.standard_normal((64, 1, 8))
    q = rng.standard_normal((1, 2, 8))
    o, lse = oracle.decode(q, [k], [v], [[0]], 0.4)
    perm = rng.permutation(64)
    o2, lse2 = oracle.decode(q, [k[perm]], [v[perm]], [[0]], 0.4)
    np.testing.assert_allclose(o, o2, atol=1e-13)
    np.testing.assert_allclose(lse, lse2, atol=1e-13)


# ------------------------------------------------------ pools and page tables

def test_pool_pages_hold_the_logical_tokens():
    """Reading segments back out of the pools by page id (numpy fancy
    indexing here, independent of the generator's own read-back) gives the
    logical tokens; unused slots are NaN."""
    w = make_config(0)
    kp = w.k_pool.numpy()
    vp = w.v_pool.numpy()

    def vslot(t):   # V rows keep tokens 0-3, 8-11, 4-7, 12-15: bits 2 and 3 swapped
        return (t & 3) | ((t & 4) << 1) | ((t & 8) >> 1)
    for s in range(len(w.seg_len)):
        n = int(w.seg_len[s])
        pages = np.asarray(w.seg_pages[s])
        k_np = np.stack([kp[pages[t // 16], :, :, t % 16, :].reshape(kp.shape[1], -1)
                         for t in range(n)])
        v_np = np.stack([vp[pages[t // 16], :, :, vslot(t % 16)] for t in range(n)])
        k, v = w.segment_kv(s)
        assert np.array_equal(k.numpy(), k_np) and np.array_equal(v.numpy(), v_np)
        assert not np.isnan(k_np).any()
        tail = n % 16
        if tail:
            assert np.isnan(kp[pages[-1], :, :, tail:, :]).all()
            assert np.isnan(vp[pages[-1], :, :, [vslot(t) for t in range(tail, 16)]]).all()
            assert not np.isnan(vp[pages[-1], :, :, [vslot(t) for t in range(tail)]]).any()


def test_page_placement_does_not_change_oracle_output():
    """The same logical tokens laid out in two different page placements
    give bit-identical oracle outputs (the oracle reads logical arrays)."""
    seg_len = [37, 5, 20]
    paths = [[0, 1], [0, 2]]
    a = build_workload("a", 5, 4, 2, 8, torch.float32, seg_len, paths, exact_pool=True)
    b = build_workload("b", 6, 4, 2, 8, torch.float32, seg_len, paths, capacity_factor=3.0)
    def vslot(t):
        return (t & 3) | ((t & 4) << 1) | ((t & 8) >> 1)

    # copy a's logical tokens into b's placement
    for s in range(3):
        k, v = a.segment_kv(s)
        for t in range(seg_len[s]):
            p = int(b.seg_pages[s][t // 16])
            b.k_pool[p, :, :, t % 16, :] = k[t].reshape(b.k_pool.shape[1], -1, b.k_pool.shape[-1])
            b.v_pool[p, :, :, vslot(t % 16)] = v[t]
    for w in (a, b):
        w.q = a.q.clone()
    outs = []
    for w in (a, b):
        ks = [w.segment_kv(s)[0].numpy() for s in range(3)]
        vs = [w.segment_kv(s)[1].numpy() for s in range(3)]
        outs.append(oracle.decode(w.q.numpy(), ks, vs, paths, w.scale))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    assert not np.array_equal(a.seg_pages[0], b.seg_pages[0])


def test_gather_expected_is_concatenation():
    rng = np.random.default_rng(20)
    segs = [rng.standard_normal((n, 2, 4)).astype(np.float32) for n in (3, 0, 5)]
    out = oracle.gather_tokens(segs, [2, 0, 1])
    assert out.shape == (8, 2, 4)
    assert np.array_equal(out[:5], segs[2]) and np.array_equal(out[5:], segs[0])


# ---------------------------------------------------------------- paged KV write path

PAGED_GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paged_kv_layout.json")


def test_paged_kv_golden_offsets():
    """Hand-worked element offsets of both pool layouts."""
    with open(PAGED_GOLDEN) as f:
        cases = json.load(f)["cases"]
    for cs in cases:
        kind = oracle.paged_kv.POOL_K if cs["kind"] == "K" else oracle.paged_kv.POOL_V
        got = oracle.paged_kv.elem_offset(kind, cs["H"], cs["D"], cs["E"], cs["page"], cs["h"], cs["t"], cs["c"])
        assert got == cs["offset"], cs


def test_paged_kv_slot_map_is_the_stated_permutation():
    assert [oracle.paged_kv.v_slot(t) for t in range(16)] == [0, 1, 2, 3, 8, 9, 10, 11, 4, 5, 6, 7, 12, 13, 14, 15]


@pytest.mark.parametrize("dtype,D", [(torch.bfloat16, 128), (torch.float32, 64)])
def test_paged_kv_scatter_agrees_with_generator_readback(dtype, D):
    """Write every segment's tokens with the oracle scatter, then read them
    back with the input generator's tensor read-back (reshape and permute of
    the pool, an independent statement of the same layouts): the logical
    tokens come back. A transposed unit, a wrong slot order or a wrong tile
    base fails this."""
    w = build_workload("wr", 9, 4, 2, D, dtype, [37, 16, 5, 50], [[0, 1], [0, 2], [3]], poison=False)
    ity = torch.int16 if dtype == torch.bfloat16 else torch.int32
    E = 16 // torch.empty(0, dtype=dtype).element_size()
    rng = np.random.default_rng(1)
    info = np.iinfo(np.int16 if ity == torch.int16 else np.int32)
    logical = {s: {kind: rng.integers(info.min, info.max, size=(int(w.seg_len[s]), 2, D), endpoint=True)
                   for kind in (0, 1)} for s in range(4)}
    for kind, pool in ((0, w.k_pool), (1, w.v_pool)):
        flat = pool.view(ity).numpy().ravel()
        segs = range(4)
        src = np.concatenate([logical[s][kind] for s in segs]).astype(flat.dtype)
        offs = np.concatenate([[0], np.cumsum([int(w.seg_len[s]) for s in segs])[:-1]])
        out, flagged = oracle.paged_kv.scatter(flat, kind, 2, D, E, w.num_pool_pages,
                                               [w.seg_pages[s] for s in segs], [0] * 4,
                                               [int(w.seg_len[s]) for s in segs], offs, src)
        assert not flagged
        pool.view(ity).copy_(torch.as_tensor(out).view(pool.shape))
    for s in range(4):
        k, v = w.segment_kv(s)
        assert np.array_equal(k.view(ity).numpy(), logical[s][0])
        assert np.array_equal(v.view(ity).numpy(), logical[s][1])


def test_paged_kv_scatter_rules():
    """Only the written slots change; a range past the page list skips the
    whole sequence, a bad page id skips its page; both are flagged."""
    H, D, E, n_pool = 1, 8, 4, 6
    pool = np.arange(n_pool * H * 16 * D, dtype=np.int64) * -1 - 1
    src = np.arange(40 * H * D, dtype=np.int64).reshape(40, H, D)
    out, flagged = oracle.paged_kv.scatter(pool, 0, H, D, E, n_pool, [[2, 4]], [14], [3], [0], src)
    assert not flagged
    changed = np.nonzero(out != pool)[0]
    want = sorted(oracle.paged_kv.elem_offset(0, H, D, E, pg, 0, t, c)
                  for pg, t in ((2, 14), (2, 15), (4, 0)) for c in range(D))
    assert changed.tolist() == want
    assert out[oracle.paged_kv.elem_offset(0, H, D, E, 4, 0, 0, 5)] == src[2, 0, 5]
    out, flagged = oracle.paged_kv.scatter(pool, 1, H, D, E, n_pool, [[1], [0, 9]], [10, 12], [7, 8], [0, 7], src)
    assert flagged
    changed = set(np.nonzero(out != pool)[0].tolist())
    want = {oracle.paged_kv.elem_offset(1, H, D, E, 0, 0, t, c) for t in range(12, 16) for c in range(D)}
    assert changed == want          # sequence 0 (10 + 7 > 16) skipped; page 9 of sequence 1 skipped
    out, flagged = oracle.paged_kv.page_copy(pool, H * 16 * D, n_pool, [1, 7], [3, 2])
    assert flagged
    pe = H * 16 * D
    assert np.array_equal(out[3 * pe:4 * pe], pool[pe:2 * pe])
    assert np.array_equal(np.delete(out, np.s_[3 * pe:4 * pe]), np.delete(pool, np.s_[3 * pe:4 * pe]))
