"""A decode loop end to end (GPU): prompts as token ids -> prefix forest ->
each segment's K/V written once -> for several steps, every request appends
its new token to its private segment (a fresh page at page boundaries), the
plan is brought up to date in place (new pages included: the plan keeps
room for them), and decode attention is compared with the oracle's
unshared attention over the request's whole token sequence (§3)."""

import types

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import assert_parity
from paper_2509_02121_amd import halo

pytestmark = pytest.mark.gpu

PAGE = 16


def test_decode_loop_over_token_id_forest(gpu_lib):
    print("case: decode loop, 12 steps", flush=True)
    dev = "cuda"
    dtype, H, HQ, D = torch.bfloat16, 2, 8, 128
    rng = np.random.default_rng(17)
    gen = torch.Generator().manual_seed(17)
    sys_a = rng.integers(0, 1000, size=45).tolist()          # shared prefix ending inside a page
    sys_b = rng.integers(0, 1000, size=64).tolist()          # page-aligned shared prefix
    prompts = [sys_a + rng.integers(0, 1000, size=int(n)).tolist() for n in (3, 20, 1, 40)] + \
              [sys_b + rng.integers(0, 1000, size=int(n)).tolist() for n in (16, 5)]
    R = len(prompts)
    tree = halo.PrefixTree(prompts, PAGE)
    paths = tree.paths()
    leaf = [p[-1] for p in paths]
    assert all(tree.seg_refcount[s] == 1 for s in leaf)      # every request owns its last segment
    max_pos = max(len(p) for p in prompts) + 16
    tok_k, tok_v = (torch.randn((1000, H, D), generator=gen) for _ in range(2))
    pos_k, pos_v = (torch.randn((max_pos, H, D), generator=gen) for _ in range(2))

    def kv(tokens, positions):
        t = torch.as_tensor(np.asarray(tokens, np.int64))
        p = torch.as_tensor(np.asarray(positions, np.int64))
        return (0.5 * (tok_k[t] + pos_k[p])).to(dtype), (0.5 * (tok_v[t] + pos_v[p])).to(dtype)

    n_pool = tree.num_pages + 64
    free = list(rng.permutation(n_pool).astype(int))
    seg_pages = [[free.pop() for _ in range(int(n))] for n in tree.pages_per_segment()]
    seg_len = tree.seg_len.astype(np.int64).copy()
    kp = torch.full((n_pool, H, D // 8, PAGE, 8), float("nan"), dtype=dtype, device=dev)
    vp = torch.full((n_pool, H, D, PAGE), float("nan"), dtype=dtype, device=dev)
    scale = float(np.float32(1 / np.sqrt(D)))
    params = halo.make_params(HQ, H, D, dtype, n_pool, scale, dtype)

    def write(segs, starts, counts, k, v):
        indptr = np.zeros(len(segs) + 1, np.int32)
        indptr[1:] = np.cumsum([len(seg_pages[s]) for s in segs])
        offs = np.concatenate([[0], np.cumsum(counts)[:-1]]).astype(np.int64)
        flag = torch.zeros(1, dtype=torch.int32, device=dev)
        halo.kv_page_scatter_kv(kp, vp, params,
                                torch.as_tensor(np.concatenate([seg_pages[s] for s in segs]).astype(np.int32),
                                                device=dev),
                                torch.as_tensor(indptr, device=dev),
                                torch.as_tensor(np.asarray(starts, np.int32), device=dev),
                                torch.as_tensor(np.asarray(counts, np.int32), device=dev),
                                torch.as_tensor(offs, device=dev), k.to(dev), v.to(dev), flag)
        torch.cuda.synchronize()
        assert int(flag.item()) == 0

    # each segment's K/V once, from its source request's tokens
    ks, vs = [], []
    for s in range(tree.num_segments):
        r, o, n = int(tree.seg_src_request[s]), int(tree.seg_src_offset[s]), int(tree.seg_len[s])
        k, v = kv(prompts[r][o:o + n], range(o, o + n))
        ks.append(k)
        vs.append(v)
    write(list(range(tree.num_segments)), [0] * tree.num_segments, [int(x) for x in tree.seg_len],
          torch.cat(ks), torch.cat(vs))

    tokens = [list(p) for p in prompts]
    pa, applied, opened = None, 0, 0
    for step in range(12):
        new = rng.integers(0, 1000, size=R).tolist()
        starts = []
        for r in range(R):
            s = leaf[r]
            if seg_len[s] == len(seg_pages[s]) * PAGE:
                seg_pages[s].append(free.pop())               # a fresh page for the new token
                opened += pa is not None
            starts.append(int(seg_len[s]))
        k, v = kv(new, [len(tokens[r]) for r in range(R)])
        write(leaf, starts, [1] * R, k, v)
        for r in range(R):
            seg_len[leaf[r]] += 1
            tokens[r].append(new[r])
        page_indptr = np.zeros(tree.num_segments + 1, np.int32)
        page_indptr[1:] = np.cumsum([len(p) for p in seg_pages])
        csr = dict(seg_len=seg_len.astype(np.int32), seg_page_indptr=page_indptr,
                   seg_page_ids=np.concatenate(seg_pages).astype(np.int32),
                   req_seg_indptr=tree.req_seg_indptr.copy(), req_seg_ids=tree.req_seg_ids.copy(), q_len=None)
        q = (torch.randn((R, HQ, D), generator=gen) * 0.5).to(dtype)
        if pa is None:
            pa = halo.PrefixAttention(params, csr, dev)
        elif pa.update(csr):
            applied += 1
            if opened == 0:
                # no page opened since planning: byte for byte a fresh plan
                assert pa.plan.image() == halo.Plan.from_csr(params, csr).image()
        o, lse = pa.run(q.to(dev), kp, vp)
        torch.cuda.synchronize()
        seg_k, seg_v = {}, {}
        for r in range(R):
            kk, vv = kv(tokens[r], range(len(tokens[r])))
            seg_k[r], seg_v[r] = kk.double().numpy(), vv.double().numpy()
        o_ref, lse_ref = oracle.decode(q.double().numpy(), seg_k, seg_v, [[r] for r in range(R)], scale)
        assert_parity(types.SimpleNamespace(dtype=dtype), o.double().cpu().numpy(), lse.double().cpu().numpy(),
                      o_ref, lse_ref, np.arange(R), f"decode step {step}")
    # every step after the first updates the plan in place, pages opened too
    print(f"plan updated in place on {applied} of 11 steps, {opened} pages opened", flush=True)
    assert applied == 11 and opened > 0
