"""GPU bit-exactness of halo_kv_page_gather (§7 PagedAttention page tables)."""

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import params_of, to_device
from paper_2509_02121_amd import halo
from workloads import build_workload, make_config

pytestmark = pytest.mark.gpu


def _gather(w, seqs, kind, error_flag=None, pages_override=None):
    pages = [np.asarray(w.seg_pages[s], np.int32) for s in seqs]
    if pages_override is not None:
        pages = pages_override
    indptr = np.zeros(len(seqs) + 1, np.int32)
    indptr[1:] = np.cumsum([len(p) for p in pages])
    lens = np.array([int(w.seg_len[s]) for s in seqs], np.int32)
    offs = np.zeros(len(seqs), np.int64)
    offs[1:] = np.cumsum(lens)[:-1]
    dev = "cuda"
    total = int(lens.sum())
    out = torch.full((total + 3, w.num_kv_heads, w.head_dim), 7.0, dtype=w.dtype, device=dev)
    pool = w.k_pool if kind == halo.HALO_POOL_K else w.v_pool
    ids = torch.as_tensor(np.concatenate(pages) if pages else np.zeros(1, np.int32), device=dev)
    halo.kv_page_gather(pool, params_of(w), kind, ids, torch.as_tensor(indptr, device=dev),
                        torch.as_tensor(lens, device=dev), torch.as_tensor(offs, device=dev), out,
                        error_flag)
    torch.cuda.synchronize()
    return out.cpu()


def _expected(w, seqs, kind):
    """oracle.gather_tokens over the logical per-segment arrays (read back out
    of the pools by the generator's own reshape, not by the library)."""
    which = 0 if kind == halo.HALO_POOL_K else 1
    arrays = {s: w.segment_kv(s)[which] for s in set(seqs)}
    if not seqs:
        return torch.zeros(0)
    exp = oracle.gather_tokens({s: a.numpy() if a.dtype != torch.bfloat16 else a.view(torch.int16).numpy()
                                for s, a in arrays.items()}, seqs)
    t = torch.from_numpy(np.ascontiguousarray(exp))
    return t.view(torch.bfloat16) if w.dtype == torch.bfloat16 else t


def _bits(t):
    return t.contiguous().view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).numpy()


@pytest.mark.parametrize("index", [0, 1])
@pytest.mark.parametrize("kind", [halo.HALO_POOL_K, halo.HALO_POOL_V])
def test_gather_bit_exact(gpu_lib, index, kind):
    print(f"case: gather config {index} kind {kind}", flush=True)
    w = to_device(make_config(index))
    seqs = list(range(len(w.seg_len)))[::-1]       # every segment, reversed order
    out = _gather(w, seqs, kind)
    exp = _expected(w, seqs, kind)
    n = exp.shape[0]
    assert np.array_equal(_bits(out[:n]), _bits(exp))
    assert (out[n:].float() == 7.0).all(), "gather wrote past the last token"


def test_gather_preserves_special_bit_patterns(gpu_lib):
    """NaN payloads, signed zeros, infinities and subnormals move unchanged."""
    print("case: gather special bits", flush=True)
    for dtype, ity, pats in (
            (torch.float32, torch.int32, [0x7fc00001, 0x7f800123, -0x80000000, 0x00000001, 0x7f800000,
                                          -0x00800000, 0xffc0ffee - (1 << 32)]),
            (torch.bfloat16, torch.int16, [0x7fc1, 0x7f81, -0x8000, 0x0001, 0x7f80, -0x0080, -0x3f11])):
        w = build_workload("bits", 3, 2, 2, 64, dtype, [37, 5], [[0, 1]], poison=False)
        for kind, pool in ((halo.HALO_POOL_K, w.k_pool), (halo.HALO_POOL_V, w.v_pool)):
            view = pool.view(ity)
            flat = view.reshape(-1)
            idx = torch.arange(0, flat.numel(), 97)
            flat[idx] = torch.tensor(pats, dtype=ity).repeat(len(idx) // len(pats) + 1)[:len(idx)]
        to_device(w)
        for kind in (halo.HALO_POOL_K, halo.HALO_POOL_V):
            out = _gather(w, [0, 1], kind)
            exp = _expected(w, [0, 1], kind)
            assert np.array_equal(_bits(out[:42]), _bits(exp))


def test_gather_flags_bad_page_ids_and_skips_them(gpu_lib):
    print("case: gather bad page id", flush=True)
    w = to_device(make_config(0))
    pages = [np.asarray(w.seg_pages[s], np.int32).copy() for s in (0, 1)]
    pages[1][0] = w.num_pool_pages + 5          # out of range: must be skipped, not read
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = _gather(w, [0, 1], halo.HALO_POOL_K, flag, pages)
    assert int(flag.item()) == 1
    exp = _expected(w, [0], halo.HALO_POOL_K)
    assert np.array_equal(_bits(out[:256]), _bits(exp))      # the valid sequence is intact
    assert (out[256:256 + 16].float() == 7.0).all()             # the bad page left untouched
    rest = _expected(w, [1], halo.HALO_POOL_K)[16:]
    assert np.array_equal(_bits(out[256 + 16:256 + 16 + rest.shape[0]]), _bits(rest))


@pytest.mark.parametrize("dtype,D", [(torch.bfloat16, 128), (torch.float32, 64), (torch.bfloat16, 64)])
@pytest.mark.parametrize("kind", [halo.HALO_POOL_K, halo.HALO_POOL_V])
def test_gather_skewed_and_empty_sequences(gpu_lib, dtype, D, kind):
    """Empty sequences between others, one long sequence among many short
    ones, lengths ending inside a page: every token lands once, in order, and
    nothing is written past the last token (the work is cut into equal runs
    of tiles, so runs start and end inside sequences)."""
    print(f"case: gather skewed {dtype} d{D} kind {kind}", flush=True)
    rng = np.random.default_rng(D + kind)
    seg_len = [0, 3000, 0, 0, 17, 1, 16, 0, 33] + [int(x) for x in rng.integers(0, 40, size=300)] + [0]
    w = to_device(build_workload("skew", 3, 2, 2, D, dtype, seg_len, [[s] for s in range(len(seg_len))],
                                 poison=False))
    seqs = list(range(len(seg_len)))
    out = _gather(w, seqs, kind)
    exp = _expected(w, seqs, kind)
    n = exp.shape[0]
    assert np.array_equal(_bits(out[:n]), _bits(exp))
    assert (out[n:].float() == 7.0).all(), "gather wrote past the last token"


@pytest.mark.parametrize("kind", [halo.HALO_POOL_K, halo.HALO_POOL_V])
def test_gather_sliced_page_list(gpu_lib, kind):
    """seq_page_indptr need not start at 0: a slice of a larger page list
    (here sequences 3.. of a longer list, indptr and page ids passed as
    views into the full arrays) gathers exactly those sequences."""
    print(f"case: gather sliced page list kind {kind}", flush=True)
    w = to_device(make_config(1))
    seqs = list(range(len(w.seg_len)))
    pages = [np.asarray(w.seg_pages[s], np.int32) for s in seqs]
    indptr = np.zeros(len(seqs) + 1, np.int32)
    indptr[1:] = np.cumsum([len(p) for p in pages])
    lens = np.array([int(w.seg_len[s]) for s in seqs], np.int32)
    sub = seqs[3:]
    offs = np.zeros(len(sub), np.int64)
    offs[1:] = np.cumsum(lens[3:])[:-1]
    dev = "cuda"
    total = int(lens[3:].sum())
    out = torch.full((total + 3, w.num_kv_heads, w.head_dim), 7.0, dtype=w.dtype, device=dev)
    pool = w.k_pool if kind == halo.HALO_POOL_K else w.v_pool
    ids_full = torch.as_tensor(np.concatenate(pages), device=dev)
    indptr_full = torch.as_tensor(indptr, device=dev)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    halo.kv_page_gather(pool, params_of(w), kind, ids_full, indptr_full[3:],
                        torch.as_tensor(lens[3:], device=dev), torch.as_tensor(offs, device=dev), out, flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 0
    out = out.cpu()
    exp = _expected(w, sub, kind)
    assert np.array_equal(_bits(out[:total]), _bits(exp))
    assert (out[total:].float() == 7.0).all(), "gather wrote past the last token"
