"""GPU bit-exactness of the paged-KV write path: halo_kv_page_scatter and
halo_kv_page_scatter_kv (new tokens into their pages, §7 PagedAttention; §2
KV written once and reused) and halo_kv_page_copy (the copy of
copy-on-write), against the oracle's element-by-element scatter and page
copy (oracle.paged_kv)."""

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import assert_parity, oracle_for, params_of, run_library, to_device
from paper_2509_02121_amd import halo
from workloads import build_workload, make_config

pytestmark = pytest.mark.gpu

PAGE = 16


def _random_bits(shape, ity, rng):
    nt = np.int16 if ity == torch.int16 else np.int32
    info = np.iinfo(nt)
    return torch.as_tensor(rng.integers(info.min, info.max, size=shape, endpoint=True, dtype=nt))


def _int_type(dtype):
    return torch.int16 if dtype == torch.bfloat16 else torch.int32


def _scatter(dtype, D, H, n_pool, seqs, kind, rng, flag=None):
    """Scatter random-bit tokens into a random-bit pool on the GPU; returns
    (pool bits after, expected bits from the oracle, pool bits before).
    seqs: list of (page ids, start, count)."""
    ity = _int_type(dtype)
    E = 16 // (2 if dtype == torch.bfloat16 else 4)
    total = sum(c for _, _, c in seqs)
    pool_bits = _random_bits((n_pool * H * PAGE * D,), ity, rng)
    in_bits = _random_bits((max(total, 1), H, D), ity, rng)
    offs = np.concatenate([[0], np.cumsum([c for _, _, c in seqs])[:-1]]).astype(np.int64)
    exp, exp_flag = oracle.paged_kv.scatter(pool_bits.numpy(), kind, H, D, E, n_pool, [p for p, _, _ in seqs],
                                            [st for _, st, _ in seqs], [c for _, _, c in seqs], offs,
                                            in_bits.numpy())
    dev = "cuda"
    pool = pool_bits.to(dev).view(dtype)
    src = in_bits.to(dev).view(dtype)
    indptr = np.zeros(len(seqs) + 1, np.int32)
    indptr[1:] = np.cumsum([len(p) for p, _, _ in seqs])
    ids = np.concatenate([np.asarray(p, np.int32) for p, _, _ in seqs] + [np.zeros(1, np.int32)])
    params = halo.make_params(H, H, D, dtype, n_pool, 0.125, dtype)
    halo.kv_page_scatter(pool, params, kind, torch.as_tensor(ids, device=dev),
                         torch.as_tensor(indptr, device=dev),
                         torch.as_tensor(np.array([s for _, s, _ in seqs], np.int32), device=dev),
                         torch.as_tensor(np.array([c for _, _, c in seqs], np.int32), device=dev),
                         torch.as_tensor(offs, device=dev), src, flag)
    torch.cuda.synchronize()
    if flag is not None:
        assert int(flag.item()) == int(exp_flag)
    return pool.view(ity).cpu().numpy(), exp, pool_bits.numpy()


def _random_seqs(rng, n_pool, n_seqs, max_pages):
    perm = rng.permutation(n_pool)
    seqs, at = [], 0
    for _ in range(n_seqs):
        npg = int(rng.integers(1, max_pages + 1))
        pages = perm[at:at + npg].astype(np.int32)
        at += npg
        cap = npg * PAGE
        start = int(rng.integers(0, cap))
        count = int(rng.integers(0, cap - start + 1))
        seqs.append((pages, start, count))
    return seqs, perm[at:].astype(np.int32)     # and the pages no sequence uses


@pytest.mark.parametrize("dtype,D", [(torch.float32, 64), (torch.bfloat16, 128), (torch.bfloat16, 64)])
@pytest.mark.parametrize("kind", [halo.HALO_POOL_K, halo.HALO_POOL_V])
def test_scatter_bit_exact(gpu_lib, dtype, D, kind):
    """Random ranges (partial pages, page-crossing, empty, whole pages) of
    random-bit tokens (NaN payloads included): every written slot holds the
    input bits and every other pool word is unchanged."""
    print(f"case: scatter {dtype} d{D} kind {kind}", flush=True)
    rng = np.random.default_rng(11 + D + kind)
    H, n_pool = 2, 64
    seqs, spare = _random_seqs(rng, n_pool, 9, 5)
    seqs += [(spare[0:2], 0, 32), (spare[2:3], 15, 1)]   # two whole pages; the last slot only
    got, exp, _ = _scatter(dtype, D, H, n_pool, seqs, kind, rng)
    assert np.array_equal(got, exp)


@pytest.mark.parametrize("dtype,D", [(torch.bfloat16, 128), (torch.float32, 64)])
def test_scatter_kv_equals_two_single_pool_calls(gpu_lib, dtype, D):
    """The two-pool call writes exactly what the two single-pool calls write,
    also with a flagged sequence among the good ones."""
    print(f"case: scatter_kv {dtype} d{D}", flush=True)
    rng = np.random.default_rng(21 + D)
    H, n_pool = 3, 64
    ity = _int_type(dtype)
    seqs, spare = _random_seqs(rng, n_pool, 12, 4)
    seqs.append((spare[:1], 9, 8))                       # 9 + 8 > 16: flagged, skipped
    total = sum(c for _, _, c in seqs)
    dev = "cuda"
    pools = [_random_bits((n_pool * H * PAGE * D,), ity, rng).to(dev).view(dtype) for _ in range(2)]
    ins = [_random_bits((total, H, D), ity, rng).to(dev).view(dtype) for _ in range(2)]
    indptr = np.zeros(len(seqs) + 1, np.int32)
    indptr[1:] = np.cumsum([len(p) for p, _, _ in seqs])
    offs = np.concatenate([[0], np.cumsum([c for _, _, c in seqs])[:-1]]).astype(np.int64)
    lists = (torch.as_tensor(np.concatenate([p for p, _, _ in seqs]), device=dev), torch.as_tensor(indptr, device=dev),
             torch.as_tensor(np.array([st for _, st, _ in seqs], np.int32), device=dev),
             torch.as_tensor(np.array([c for _, _, c in seqs], np.int32), device=dev),
             torch.as_tensor(offs, device=dev))
    params = halo.make_params(H, H, D, dtype, n_pool, 0.125, dtype)
    single = [p.clone() for p in pools]
    flags = torch.zeros(2, dtype=torch.int32, device=dev)
    halo.kv_page_scatter(single[0], params, halo.HALO_POOL_K, *lists, ins[0], flags[0:1])
    halo.kv_page_scatter(single[1], params, halo.HALO_POOL_V, *lists, ins[1], flags[0:1])
    halo.kv_page_scatter_kv(pools[0], pools[1], params, *lists, ins[0], ins[1], flags[1:2])
    torch.cuda.synchronize()
    assert flags.tolist() == [1, 1]
    for a, b in zip(pools, single):
        assert torch.equal(a.view(ity), b.view(ity))


def test_scatter_then_gather_round_trip(gpu_lib):
    """Decode-style appends (one token per sequence at its current length),
    read back with the gather: the appended token is the input, earlier
    tokens are unchanged."""
    print("case: scatter/gather round trip", flush=True)
    w = to_device(build_workload("rt", 5, 4, 2, 128, torch.bfloat16, [37, 16, 5], [[0], [1], [2]],
                                 poison=False))
    params = params_of(w)
    before = [w.segment_kv(s) for s in range(3)]
    dev = "cuda"
    new = torch.randn((3, 2, 128), generator=torch.Generator().manual_seed(3)).to(torch.bfloat16)
    lens = [37, 16, 5]
    pages = [np.asarray(w.seg_pages[s], np.int32) for s in range(3)]
    # room for one more token: sequence 1 is page-full, give it a fresh page
    spare = int(np.setdiff1d(np.arange(w.num_pool_pages), np.concatenate(pages))[0])
    pages[1] = np.append(pages[1], spare).astype(np.int32)
    indptr = np.zeros(4, np.int32)
    indptr[1:] = np.cumsum([len(p) for p in pages])
    ids = torch.as_tensor(np.concatenate(pages), device=dev)
    for kind, pool in ((halo.HALO_POOL_K, w.k_pool), (halo.HALO_POOL_V, w.v_pool)):
        halo.kv_page_scatter(pool, params, kind, ids, torch.as_tensor(indptr, device=dev),
                             torch.as_tensor(np.array(lens, np.int32), device=dev),
                             torch.ones(3, dtype=torch.int32, device=dev),
                             torch.arange(3, dtype=torch.int64, device=dev), new.to(dev))
        out = torch.zeros((sum(lens) + 3, 2, 128), dtype=torch.bfloat16, device=dev)
        offs = np.zeros(3, np.int64)
        offs[1:] = np.cumsum([n + 1 for n in lens])[:-1]
        halo.kv_page_gather(pool, params, kind, ids, torch.as_tensor(indptr, device=dev),
                            torch.as_tensor(np.array(lens, np.int32) + 1, device=dev),
                            torch.as_tensor(offs, device=dev), out)
        torch.cuda.synchronize()
        out = out.cpu()
        for s in range(3):
            old = before[s][0 if kind == halo.HALO_POOL_K else 1]
            seg = out[offs[s]:offs[s] + lens[s] + 1]
            assert torch.equal(seg[:lens[s]].view(torch.int16), old.view(torch.int16))
            assert torch.equal(seg[lens[s]].view(torch.int16), new[s].view(torch.int16))


@pytest.mark.parametrize("dtype,D", [(torch.float32, 64), (torch.bfloat16, 128)])
def test_page_copy_bit_exact(gpu_lib, dtype, D):
    print(f"case: page copy {dtype} d{D}", flush=True)
    rng = np.random.default_rng(7)
    H, n_pool = 3, 40
    ity = _int_type(dtype)
    bits = _random_bits((n_pool * H * PAGE * D,), ity, rng)
    perm = rng.permutation(n_pool)
    src, dst = perm[:9].astype(np.int32), perm[9:18].astype(np.int32)
    exp, _ = oracle.paged_kv.page_copy(bits.numpy(), H * PAGE * D, n_pool, src, dst)
    exp = exp.reshape(n_pool, -1)
    pool = bits.to("cuda").view(dtype)
    halo.kv_page_copy(pool, halo.make_params(H, H, D, dtype, n_pool, 0.125, dtype),
                      torch.as_tensor(src, device="cuda"), torch.as_tensor(dst, device="cuda"))
    torch.cuda.synchronize()
    assert np.array_equal(pool.view(ity).cpu().numpy().reshape(n_pool, -1), exp)


def test_write_path_flags_bad_input(gpu_lib):
    """A page id out of range, or a range past the page list, is skipped and
    flagged; the other sequences are written."""
    print("case: write path bad input", flush=True)
    rng = np.random.default_rng(4)
    H, n_pool, D = 2, 16, 64
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    seqs = [(np.array([3, 4], np.int32), 5, 20),
            (np.array([7, n_pool + 3], np.int32), 10, 12),     # second page out of range
            (np.array([9], np.int32), 10, 7)]                  # 10 + 7 > 16
    got, exp, before = _scatter(torch.float32, D, H, n_pool, seqs, halo.HALO_POOL_K, rng, flag)
    assert int(flag.item()) == 1
    assert np.array_equal(got, exp)
    per = H * PAGE * D
    assert np.array_equal(got.reshape(n_pool, per)[9], before.reshape(n_pool, per)[9])
    assert not np.array_equal(got.reshape(n_pool, per)[7], before.reshape(n_pool, per)[7])
    flag.zero_()
    got, exp, _ = _scatter(torch.float32, D, H, n_pool, seqs[:1], halo.HALO_POOL_K, rng, flag)
    assert int(flag.item()) == 0 and np.array_equal(got, exp)
    pool = torch.zeros(n_pool * per, dtype=torch.float32, device="cuda")
    halo.kv_page_copy(pool, halo.make_params(H, H, D, torch.float32, n_pool, 0.125, torch.float32),
                      torch.tensor([1, n_pool], dtype=torch.int32, device="cuda"),
                      torch.tensor([2, 3], dtype=torch.int32, device="cuda"), flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 1


def test_decode_append_then_attention_matches_oracle(gpu_lib):
    """One decode step end to end: each request's newest token is missing
    (NaN) from the pools, the write path appends it, then the attention over
    the shared-prefix forest matches the oracle on the complete keys."""
    print("case: decode append then attention", flush=True)
    w = to_device(make_config(1))
    dev = "cuda"
    R = w.num_requests
    last = [w.req_paths[r][-1] for r in range(R)]       # each request's private segment
    k_new = torch.stack([w.segment_kv(s)[0][-1] for s in last]).to(dev)
    v_new = torch.stack([w.segment_kv(s)[1][-1] for s in last]).to(dev)
    lens = np.array([int(w.seg_len[s]) for s in last], np.int32)
    pages = [np.asarray(w.seg_pages[s], np.int32) for s in last]
    indptr = np.zeros(R + 1, np.int32)
    indptr[1:] = np.cumsum([len(p) for p in pages])
    ids = torch.as_tensor(np.concatenate(pages), device=dev)
    args = (ids, torch.as_tensor(indptr, device=dev), torch.as_tensor(lens - 1, device=dev),
            torch.ones(R, dtype=torch.int32, device=dev), torch.arange(R, dtype=torch.int64, device=dev))
    params = params_of(w)
    nan = torch.full_like(k_new, float("nan"))
    for kind, pool, new in ((halo.HALO_POOL_K, w.k_pool, k_new), (halo.HALO_POOL_V, w.v_pool, v_new)):
        halo.kv_page_scatter(pool, params, kind, *args, nan)      # the token is not there yet
    torch.cuda.synchronize()
    assert not torch.isfinite(w.segment_kv(last[0])[0][-1]).all()
    halo.kv_page_scatter_kv(w.k_pool, w.v_pool, params, *args, k_new, v_new)   # the decode step writes it
    o, lse, _ = run_library(w)
    o_ref, lse_ref, rows = oracle_for(w)
    assert torch.equal(w.segment_kv(last[0])[0][-1].view(torch.int16).cpu(), k_new[0].view(torch.int16).cpu())
    assert_parity(w, o, lse, o_ref, lse_ref, rows, "decode append")


@pytest.mark.parametrize("prefix_len", [37, 48])
def test_copy_on_write_mid_page_prefix(gpu_lib, prefix_len):
    """A shared prefix that ends inside a page (37 tokens: 2 full pages and 5
    tokens of a third), continued by four requests. Each request copies the
    prefix's partial page to a private page and appends its own tokens there
    and on fresh pages; the shared part of the forest is then the
    page-aligned head of the prefix. Attention over that forest equals the
    oracle's attention over prefix + suffix (the logical keys). prefix_len
    48 is the page-aligned case: the copy list is empty."""
    print(f"case: copy-on-write prefix {prefix_len}", flush=True)
    dev = "cuda"
    dtype, H, HQ, D = torch.bfloat16, 2, 8, 128
    gen = torch.Generator().manual_seed(prefix_len)
    suffix = [5, 20, 11, 1]
    R = len(suffix)
    n_pool = 40
    kp = torch.full((n_pool, H, D // 8, PAGE, 8), float("nan"), dtype=dtype, device=dev)
    vp = torch.full((n_pool, H, D, PAGE), float("nan"), dtype=dtype, device=dev)
    params = halo.make_params(HQ, H, D, dtype, n_pool, float(np.float32(1 / np.sqrt(D))), dtype)
    scale = float(np.float32(1 / np.sqrt(D)))

    def rand_kv(n):
        return ((torch.randn((n, H, D), generator=gen) * 0.5).to(dtype),
                (torch.randn((n, H, D), generator=gen) * 0.5).to(dtype))

    def write(pages, start, count, k, v):
        args = (torch.as_tensor(np.asarray(pages, np.int32), device=dev),
                torch.tensor([0, len(pages)], dtype=torch.int32, device=dev),
                torch.tensor([start], dtype=torch.int32, device=dev),
                torch.tensor([count], dtype=torch.int32, device=dev),
                torch.zeros(1, dtype=torch.int64, device=dev))
        halo.kv_page_scatter(kp, params, halo.HALO_POOL_K, *args, k.to(dev))
        halo.kv_page_scatter(vp, params, halo.HALO_POOL_V, *args, v.to(dev))

    free = list(np.random.default_rng(prefix_len).permutation(n_pool))
    n_pref_pages = (prefix_len + PAGE - 1) // PAGE
    prefix_pages = [int(free.pop()) for _ in range(n_pref_pages)]
    pk, pv = rand_kv(prefix_len)
    write(prefix_pages, 0, prefix_len, pk, pv)
    aligned = prefix_len // PAGE * PAGE
    tail = prefix_len - aligned
    req_pages, src, dst, seg_len = [], [], [], [aligned]
    for r in range(R):
        own = []
        if tail:
            own.append(int(free.pop()))
            src.append(prefix_pages[-1])
            dst.append(own[0])
        while len(own) * PAGE < tail + suffix[r]:
            own.append(int(free.pop()))
        req_pages.append(own)
        seg_len.append(tail + suffix[r])
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    if src:
        for pool in (kp, vp):
            halo.kv_page_copy(pool, params, torch.as_tensor(np.array(src, np.int32), device=dev),
                              torch.as_tensor(np.array(dst, np.int32), device=dev), flag)
    sk, sv = [], []
    for r in range(R):
        k, v = rand_kv(suffix[r])
        sk.append(k)
        sv.append(v)
        write(req_pages[r], tail, suffix[r], k, v)
    torch.cuda.synchronize()
    assert int(flag.item()) == 0
    seg_pages = [np.asarray(prefix_pages[:aligned // PAGE], np.int32)] + \
        [np.asarray(p, np.int32) for p in req_pages]
    seg_page_indptr = np.zeros(R + 2, np.int32)
    seg_page_indptr[1:] = np.cumsum([len(p) for p in seg_pages])
    csr = dict(seg_len=np.asarray(seg_len, np.int32), seg_page_indptr=seg_page_indptr,
               seg_page_ids=np.concatenate(seg_pages).astype(np.int32),
               req_seg_indptr=np.arange(0, 2 * R + 1, 2, dtype=np.int32),
               req_seg_ids=np.array([x for r in range(R) for x in (0, r + 1)], np.int32), q_len=None)
    q = (torch.randn((R, HQ, D), generator=gen) * 0.5).to(dtype)
    pa = halo.PrefixAttention(params, csr, dev)
    o, lse = pa.run(q.to(dev), kp, vp)
    torch.cuda.synchronize()
    seg_k = {0: pk.double().numpy()}
    seg_v = {0: pv.double().numpy()}
    for r in range(R):
        seg_k[r + 1] = sk[r].double().numpy()
        seg_v[r + 1] = sv[r].double().numpy()
    o_ref, lse_ref = oracle.decode(q.double().numpy(), seg_k, seg_v, [[0, r + 1] for r in range(R)], scale)
    err = np.abs(o.double().cpu().numpy() - o_ref).max()
    assert err <= 2e-2, err
    assert np.abs(lse.double().cpu().numpy() - lse_ref).max() <= 1e-3


def test_scatter_and_copy_at_high_page_ids(gpu_lib):
    """Pages past the first 2^31 bytes of a pool (offsets that overflow 32
    bits): a token range written into the last two pages and a page copied
    into the third-to-last one land exactly there, per the oracle."""
    print("case: write path at high page ids", flush=True)
    dev = "cuda"
    H, D, dtype = 1, 128, torch.bfloat16
    page_elems = H * PAGE * D
    n_pool = (3 << 30) // (page_elems * 2)            # 3 GiB of pool
    assert (n_pool - 1) * page_elems * 2 > (1 << 31)
    pool = torch.zeros(n_pool * page_elems, dtype=dtype, device=dev)
    rng = np.random.default_rng(9)
    src_page = _random_bits((page_elems,), torch.int16, rng)
    pool.view(torch.int16)[5 * page_elems:6 * page_elems] = src_page.to(dev)
    toks = _random_bits((20, H, D), torch.int16, rng)
    params = halo.make_params(H, H, D, dtype, n_pool, 0.125, dtype)
    pages = np.array([n_pool - 2, n_pool - 1], np.int32)
    for kind in (halo.HALO_POOL_K, halo.HALO_POOL_V):
        pool.view(torch.int16)[(n_pool - 3) * page_elems:].zero_()
        halo.kv_page_scatter(pool, params, kind, torch.as_tensor(pages, device=dev),
                             torch.tensor([0, 2], dtype=torch.int32, device=dev),
                             torch.tensor([7], dtype=torch.int32, device=dev),
                             torch.tensor([20], dtype=torch.int32, device=dev),
                             torch.zeros(1, dtype=torch.int64, device=dev), toks.to(dev).view(dtype))
        halo.kv_page_copy(pool, params, torch.tensor([5], dtype=torch.int32, device=dev),
                          torch.tensor([n_pool - 3], dtype=torch.int32, device=dev))
        torch.cuda.synchronize()
        tail = pool.view(torch.int16)[(n_pool - 3) * page_elems:].cpu().numpy()
        # the oracle on a 6-page pool whose pages 3, 4, 5 stand for the last three
        small = np.zeros(6 * page_elems, np.int16)
        small[0:page_elems] = src_page.numpy()
        small, _ = oracle.paged_kv.page_copy(small, page_elems, 6, [0], [3])
        small, _ = oracle.paged_kv.scatter(small, kind, H, D, 8, 6, [[4, 5]], [7], [20], [0], toks.numpy())
        assert np.array_equal(tail, small[3 * page_elems:])
    del pool
    torch.cuda.empty_cache()
