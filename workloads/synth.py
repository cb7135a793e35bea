"""Synthetic prefix-forest workloads (structure + seeded values + page pools).

A workload is a *prefix forest*: segments of tokens (a shared system prompt, a
shared template, a per-request suffix, a prefill chunk) and, for each request,
its root-to-leaf path of segment ids. This is the shape of the batched,
replicated agentic workflows of arXiv 2509.02121 §1 and §2 ("Context reuse";
intra-batch prefix sharing), whose KV cache is paged (§7, PagedAttention).

Page pools (the layout the library reads):
  k_pool: [P, H_kv, d/E, page_size, E]  16-byte units of E elements (E = 8
                                        for bf16, 4 for fp32), token-major
                                        inside each unit column
  v_pool: [P, H_kv, d, page_size]       dim-major inside a (page, head) tile;
                                        the 16 slots of a dim row hold tokens
                                        0-3, 8-11, 4-7, 12-15 (V_SLOT_OF_TOKEN)
Unused pages and the tail slots of a segment's last page are NaN when
``poison`` is set, so any read of them shows up in the results.

Structure randomness uses numpy's PCG64; values use a seeded torch generator
on the device the pools live on (fp32 normal, times the value scale, then
rounded to the storage dtype, round-to-nearest-even).
"""

import dataclasses
import math

import numpy as np
import torch

PAGE_SIZE = 16

# Slot of token t inside a V dim row (slots 4-7 and 8-11 swapped, i.e. bits 2
# and 3 of the index exchanged; the map is its own inverse).
V_SLOT_OF_TOKEN = np.array([0, 1, 2, 3, 8, 9, 10, 11, 4, 5, 6, 7, 12, 13, 14, 15], dtype=np.int64)

# Workloads by name, in the order they are numbered (seed = 1000 + index).
CONFIG_NAMES = (
    "tiny_decode_fp32",        # 4/4 heads, d 64, fp32, 8 req on one 256-token prefix
    "llama8b_decode",          # 32/8 heads, d 128, bf16, 64 req on one 2048-token prefix
    "two_level_tree_decode",   # 256 req: 1024-token root, 16 x 1536-token templates
    "chunked_prefill",         # 32 req x 512 new tokens over a cached 4096-token prefix
    "llama70b_batch_decode",   # 64/8 heads, 1024 req in 8 groups on 8192-token prefixes
)


@dataclasses.dataclass
class Workload:
    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: torch.dtype
    page_size: int
    scale: float                 # fp32-rounded 1/sqrt(head_dim), as a Python float
    seg_len: np.ndarray          # [S] int32
    seg_pages: list              # S arrays of int32 page ids
    req_paths: list              # R lists of segment ids, root to leaf
    q_len: object                # None (decode) or [R] int32 (prefill)
    num_pool_pages: int
    k_pool: torch.Tensor
    v_pool: torch.Tensor
    q: torch.Tensor              # [rows, H_q, d]

    @property
    def num_requests(self):
        return len(self.req_paths)

    @property
    def is_prefill(self):
        return self.q_len is not None

    def forest_csr(self):
        """The forest as int32 CSR arrays (the library's host input)."""
        seg_page_indptr = np.zeros(len(self.seg_pages) + 1, dtype=np.int32)
        seg_page_indptr[1:] = np.cumsum([len(p) for p in self.seg_pages])
        seg_page_ids = (np.concatenate(self.seg_pages).astype(np.int32)
                        if self.seg_pages else np.zeros(0, np.int32))
        req_seg_indptr = np.zeros(len(self.req_paths) + 1, dtype=np.int32)
        req_seg_indptr[1:] = np.cumsum([len(p) for p in self.req_paths])
        req_seg_ids = (np.concatenate([np.asarray(p, np.int32) for p in self.req_paths])
                       if self.req_paths else np.zeros(0, np.int32)).astype(np.int32)
        q_len = None if self.q_len is None else np.asarray(self.q_len, np.int32)
        return dict(seg_len=np.asarray(self.seg_len, np.int32),
                    seg_page_indptr=seg_page_indptr, seg_page_ids=seg_page_ids,
                    req_seg_indptr=req_seg_indptr, req_seg_ids=req_seg_ids,
                    q_len=q_len)

    def segment_kv(self, s):
        """Logical K and V of segment s, [L_s, H_kv, d] each, on the CPU.

        Read back out of the pools by page id (a pure copy), so the values
        are exactly the bits the library reads.
        """
        length = int(self.seg_len[s])
        pages = torch.as_tensor(np.asarray(self.seg_pages[s], np.int64))
        kp = self.k_pool[pages.to(self.k_pool.device)].cpu()   # [n, H, d/E, ps, E]
        vp = self.v_pool[pages.to(self.v_pool.device)].cpu()   # [n, H, d, ps]
        vp = vp[..., torch.as_tensor(V_SLOT_OF_TOKEN)]          # slot order -> token order
        k = kp.permute(0, 3, 1, 2, 4).reshape(-1, self.num_kv_heads, self.head_dim)
        v = vp.permute(0, 3, 1, 2).reshape(-1, self.num_kv_heads, self.head_dim)
        return k[:length].contiguous(), v[:length].contiguous()

    def q_rows_of_request(self, r):
        """Row range of request r in q / o (one row per query token)."""
        if self.q_len is None:
            return r, r + 1
        start = int(np.sum(self.q_len[:r]))
        return start, start + int(self.q_len[r])

    def key_bytes(self):
        """Bytes of distinct K+V tokens (each segment once)."""
        elt = torch.finfo(self.dtype).bits // 8
        return int(np.sum(self.seg_len)) * 2 * self.num_kv_heads * self.head_dim * elt


def unit_elems(dtype):
    """Elements per 16-byte unit of the K page layout."""
    return 16 // torch.empty(0, dtype=dtype).element_size()


def _fp32_scale(head_dim):
    return float(np.float32(1.0 / math.sqrt(head_dim)))


def _fill_normal(shape, gen, device, value_scale, dtype, chunk_rows=4096):
    """Seeded N(0,1)*value_scale values rounded to ``dtype``; generated in
    slabs along dim 0 so very large pools never need an fp32 copy."""
    out = torch.empty(shape, dtype=dtype, device=device)
    n = shape[0]
    for a in range(0, n, chunk_rows):
        b = min(n, a + chunk_rows)
        slab = torch.randn((b - a,) + tuple(shape[1:]), generator=gen,
                           device=device, dtype=torch.float32)
        if value_scale != 1.0:
            slab.mul_(value_scale)
        out[a:b].copy_(slab)
    return out


def build_workload(name, seed, num_q_heads, num_kv_heads, head_dim, dtype,
                   seg_len, req_paths, q_len=None, value_scale=1.0,
                   capacity_factor=1.25, exact_pool=False, device="cpu",
                   poison=True, page_size=PAGE_SIZE, extra_pages=0):
    """Lay a forest out in a page pool and fill it with seeded values.

    seg_len: segment lengths in tokens; req_paths: per-request segment ids.
    exact_pool: the pool holds exactly the needed pages, in shuffled order;
    otherwise it holds ceil(capacity_factor * needed) + extra_pages pages
    and the needed pages are placed at random.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    seg_len = np.asarray(seg_len, dtype=np.int32)
    n_pages = [(int(n) + page_size - 1) // page_size for n in seg_len]
    needed = int(sum(n_pages))
    if exact_pool:
        capacity = needed
    else:
        capacity = int(math.ceil(capacity_factor * needed)) + int(extra_pages)
    capacity = max(capacity, 1)
    placement = rng.permutation(capacity)[:needed].astype(np.int32)
    seg_pages = []
    off = 0
    for n in n_pages:
        seg_pages.append(placement[off:off + n].copy())
        off += n

    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    h, d, ps = num_kv_heads, head_dim, page_size
    e = unit_elems(dtype)
    k_pool = _fill_normal((capacity, h, d // e, ps, e), gen, device, value_scale, dtype)
    v_pool = _fill_normal((capacity, h, d, ps), gen, device, value_scale, dtype)
    if q_len is None:
        rows = len(req_paths)
    else:
        q_len = np.asarray(q_len, dtype=np.int32)
        rows = int(q_len.sum())
    q = _fill_normal((rows, num_q_heads, d), gen, device, value_scale, dtype)

    if poison:
        used = np.zeros(capacity, dtype=bool)
        used[placement] = True
        unused = torch.as_tensor(np.nonzero(~used)[0].astype(np.int64), device=device)
        if unused.numel():
            k_pool[unused] = float("nan")
            v_pool[unused] = float("nan")
        for s, n in enumerate(seg_len):
            tail = int(n) % ps
            if tail and n_pages[s]:
                p = int(seg_pages[s][-1])
                k_pool[p, :, :, tail:, :] = float("nan")
                v_pool[p, :, :, torch.as_tensor(V_SLOT_OF_TOKEN[tail:], device=device)] = float("nan")

    return Workload(name=name, seed=int(seed), num_q_heads=num_q_heads,
                    num_kv_heads=num_kv_heads, head_dim=head_dim, dtype=dtype,
                    page_size=page_size, scale=_fp32_scale(head_dim),
                    seg_len=seg_len, seg_pages=seg_pages,
                    req_paths=[list(map(int, p)) for p in req_paths],
                    q_len=q_len, num_pool_pages=capacity,
                    k_pool=k_pool, v_pool=v_pool, q=q)


def _forest(index, rng):
    """Segment lengths, paths and q_len of the numbered workloads."""
    if index == 0:      # tiny decode: one 256-token prefix, 8 requests
        suffix = rng.integers(16, 64, size=8, endpoint=True)
        seg_len = [256] + list(suffix)
        paths = [[0, 1 + r] for r in range(8)]
        return seg_len, paths, None
    if index == 1:      # 64 requests on one 2048-token prefix
        suffix = rng.integers(64, 512, size=64, endpoint=True)
        seg_len = [2048] + list(suffix)
        paths = [[0, 1 + r] for r in range(64)]
        return seg_len, paths, None
    if index == 2:      # two-level tree: 1024 root, 16 templates of 1536
        suffix = rng.integers(128, 1024, size=256, endpoint=True)
        seg_len = [1024] + [1536] * 16 + list(suffix)
        paths = [[0, 1 + r // 16, 17 + r] for r in range(256)]
        return seg_len, paths, None
    if index == 3:      # chunked prefill: 4096 cached + 512 new per request
        seg_len = [4096] + [512] * 32
        paths = [[0, 1 + r] for r in range(32)]
        return seg_len, paths, np.full(32, 512, dtype=np.int32)
    if index == 4:      # 1024 requests in 8 groups of 128 on 8192-token prefixes
        suffix = rng.integers(256, 2048, size=1024, endpoint=True)
        seg_len = [8192] * 8 + list(suffix)
        paths = [[r // 128, 8 + r] for r in range(1024)]
        return seg_len, paths, None
    raise ValueError(index)


def make_config(which, device="cpu", seed=None, poison=True, extra_pages=0):
    """Build one of the numbered workloads (by index 0..4 or by name)."""
    index = CONFIG_NAMES.index(which) if isinstance(which, str) else int(which)
    seed = 1000 + index if seed is None else int(seed)
    rng = np.random.Generator(np.random.PCG64(seed))
    seg_len, paths, q_len = _forest(index, rng)
    if index == 0:
        return build_workload(CONFIG_NAMES[0], seed, 4, 4, 64, torch.float32,
                              seg_len, paths, None, value_scale=1.0,
                              exact_pool=True, device=device, poison=poison)
    hq = 64 if index == 4 else 32
    return build_workload(CONFIG_NAMES[index], seed, hq, 8, 128,
                          torch.bfloat16, seg_len, paths, q_len,
                          value_scale=0.5, capacity_factor=1.25, device=device,
                          poison=poison, extra_pages=extra_pages)


def random_forest(rng, num_requests, max_depth=3, max_len=80, share_prob=0.6,
                  prefill=False, max_q=40, allow_empty=True):
    """A random forest for property tests: shared inner segments of random
    length (possibly 0), private leaves. Returns (seg_len, paths, q_len)."""
    seg_len = []
    paths = []
    open_prefixes = [[]]
    for _ in range(num_requests):
        base = list(open_prefixes[rng.integers(len(open_prefixes))])
        if rng.random() < share_prob and len(base) < max_depth:
            lo = 0 if allow_empty else 1
            seg_len.append(int(rng.integers(lo, max_len + 1)))
            base = base + [len(seg_len) - 1]
            open_prefixes.append(base)
        if prefill:
            n = int(rng.integers(1, max_q + 1))
        else:
            lo = 0 if allow_empty else 1
            n = int(rng.integers(lo, max_len + 1))
        seg_len.append(n)
        paths.append(base + [len(seg_len) - 1])
    q_len = None
    if prefill:
        q_len = np.array([seg_len[p[-1]] for p in paths], dtype=np.int32)
    return seg_len, paths, q_len
