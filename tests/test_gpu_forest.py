"""End to end from token ids (GPU): prompts -> prefix forest
(halo_prefix_tree_build) -> pages -> each segment's K/V written once from
its source request (halo_kv_page_scatter_kv) -> decode attention over the
forest; compared with the oracle's unshared attention of every request over
its own whole prompt (§3: sharing must not change the result)."""

import types

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import assert_parity
from paper_2509_02121_amd import halo

pytestmark = pytest.mark.gpu


def _prompts(rng, n, vocab=5000):
    """Prompts grown from earlier ones (unaligned shared lengths, repeats,
    page-aligned prefixes, an empty prompt)."""
    out = []
    for i in range(n):
        u = rng.random()
        if out and u < 0.1:
            out.append(list(out[rng.integers(len(out))]))
        elif out and u < 0.2:
            b = out[rng.integers(len(out))]
            out.append(b[:len(b) // 16 * 16])
        elif i == 3:
            out.append([])
        else:
            b = out[rng.integers(len(out))] if out and u < 0.85 else []
            keep = int(rng.integers(0, len(b) + 1))
            out.append(list(b[:keep]) + rng.integers(0, vocab, size=int(rng.integers(1, 300))).tolist())
    return out


@pytest.mark.parametrize("seed", [0, 1])
def test_decode_over_forest_built_from_token_ids(gpu_lib, seed):
    print(f"case: forest from token ids, seed {seed}", flush=True)
    dev = "cuda"
    rng = np.random.default_rng(seed)
    prompts = _prompts(rng, 40)
    H, HQ, D, dtype = 2, 8, 128, torch.bfloat16
    tree = halo.PrefixTree(prompts, 16)
    assert tree.distinct_tokens < tree.prompt_tokens          # the batch shares prefixes
    # K/V of a token: a function of (token id, position), so equal prefixes have equal K/V
    gen = torch.Generator().manual_seed(seed)
    max_len = max(len(p) for p in prompts)
    tok_k, tok_v = (torch.randn((5000, H, D), generator=gen) for _ in range(2))
    pos_k, pos_v = (torch.randn((max_len, H, D), generator=gen) for _ in range(2))

    def kv(p):
        t = torch.as_tensor(np.asarray(p, np.int64))
        pos = torch.arange(len(p))
        return ((0.5 * (tok_k[t] + pos_k[pos])).to(dtype), (0.5 * (tok_v[t] + pos_v[pos])).to(dtype))

    req_kv = [kv(p) for p in prompts]
    # pages for every segment, placed at random in a pool of 1.25x the need
    n_pool = int(tree.num_pages * 1.25) + 1
    page_ids = rng.permutation(n_pool)[:tree.num_pages].astype(np.int32)
    csr = tree.forest_csr(page_ids)
    kp = torch.full((n_pool, H, D // 8, 16, 8), float("nan"), dtype=dtype, device=dev)
    vp = torch.full((n_pool, H, D, 16), float("nan"), dtype=dtype, device=dev)
    params = halo.make_params(HQ, H, D, dtype, n_pool, float(np.float32(1 / np.sqrt(D))), dtype)
    # one write per segment, from its source request's rows
    starts = np.concatenate([[0], np.cumsum([len(p) for p in prompts])]).astype(np.int64)
    k_all = torch.cat([k for k, _ in req_kv]).to(dev)
    v_all = torch.cat([v for _, v in req_kv]).to(dev)
    offs = (starts[tree.seg_src_request] + tree.seg_src_offset).astype(np.int64)
    S = tree.num_segments
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    halo.kv_page_scatter_kv(kp, vp, params, torch.as_tensor(csr["seg_page_ids"], device=dev),
                            torch.as_tensor(csr["seg_page_indptr"], device=dev),
                            torch.zeros(S, dtype=torch.int32, device=dev),
                            torch.as_tensor(tree.seg_len, device=dev), torch.as_tensor(offs, device=dev),
                            k_all, v_all, flag)
    q = (torch.randn((len(prompts), HQ, D), generator=gen) * 0.5).to(dtype)
    pa = halo.PrefixAttention(params, csr, dev)
    o, lse = pa.run(q.to(dev), kp, vp)
    torch.cuda.synchronize()
    assert int(flag.item()) == 0
    seg_k = {r: req_kv[r][0].double().numpy() for r in range(len(prompts))}
    seg_v = {r: req_kv[r][1].double().numpy() for r in range(len(prompts))}
    o_ref, lse_ref = oracle.decode(q.double().numpy(), seg_k, seg_v, [[r] for r in range(len(prompts))],
                                   float(np.float32(1 / np.sqrt(D))))
    rows = np.arange(len(prompts))
    assert_parity(types.SimpleNamespace(dtype=dtype), o.double().cpu().numpy(), lse.double().cpu().numpy(),
                  o_ref, lse_ref, rows, f"forest seed {seed}")
