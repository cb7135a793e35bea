"""Paged-KV write path reference (TEST INFRASTRUCTURE ONLY).

Parity status: pinned by ``tests/test_oracle.py`` (hand-worked element
offsets stored in ``tests/golden/paged_kv_layout.json``, agreement with the
input generator's independent tensor read-back of the pools, and the
invariants of a scatter: untouched slots unchanged, flagged input skipped).

What it follows: the paged KV cache of PagedAttention, which the paper cites
(§7) for the KV reuse it relies on (§2: a shared prefix's KV is written once
and read by every request that shares it). New tokens of a sequence are
written into the pages of its page list: token p of a sequence sits in page
``pages[p // 16]``, slot ``p % 16``. A shared page that a request must extend
is first copied to a private page (copy-on-write).

Pool layouts (flat element offsets; E = elements per 16 bytes, 8 for bf16 and
4 for fp32; H = kv heads; D = head dim):
  * K: ``[page][H][D/E][16][E]``: element (page, h, t, c) at
    ``((page*H + h)*16*D) + ((c//E)*16 + t)*E + c%E``;
  * V: ``[page][H][D][16]`` with the 16 slots of a dim row holding tokens
    0-3, 8-11, 4-7, 12-15 (bits 2 and 3 of the token index swapped):
    element (page, h, t, c) at ``((page*H + h)*16*D) + c*16 + slot(t)``.

Everything is plain Python loops over elements on numpy arrays: slow, and
meant for small cases.
"""

import numpy as np

PAGE = 16
POOL_K = 0
POOL_V = 1


def v_slot(t):
    """Slot of token t (0..15) in a V dim row: bits 2 and 3 swapped."""
    return (t & 3) | ((t & 4) << 1) | ((t & 8) >> 1)


def elem_offset(kind, num_kv_heads, head_dim, elems_per_16b, page, h, t, c):
    """Flat offset of (page, head h, token slot t, dim c) in a pool of `kind`."""
    base = (page * num_kv_heads + h) * PAGE * head_dim
    if kind == POOL_K:
        e = elems_per_16b
        return base + ((c // e) * PAGE + t) * e + c % e
    if kind == POOL_V:
        return base + c * PAGE + v_slot(t)
    raise ValueError(kind)


def scatter(pool, kind, num_kv_heads, head_dim, elems_per_16b, num_pool_pages,
            page_lists, starts, counts, in_offsets, src):
    """The pool after writing tokens start .. start+count-1 of each sequence.

    pool: flat array (any dtype; copied, not modified); src: [T, H, D];
    sequence i takes its tokens from rows in_offsets[i] .. + counts[i] - 1.
    A sequence whose range does not fit its page list (start < 0 or
    start + count > 16 * pages) is skipped whole; a page id outside
    [0, num_pool_pages) skips that page's tokens. Returns (pool, flagged)."""
    out = np.array(pool, copy=True)
    flagged = False
    for pages, start, count, off in zip(page_lists, starts, counts, in_offsets):
        start, count, off = int(start), int(count), int(off)
        if count <= 0:
            continue
        if start < 0 or start + count > PAGE * len(pages):
            flagged = True
            continue
        for i in range(count):
            p = start + i
            page = int(pages[p // PAGE])
            if not 0 <= page < num_pool_pages:
                flagged = True
                continue
            for h in range(num_kv_heads):
                for c in range(head_dim):
                    out[elem_offset(kind, num_kv_heads, head_dim, elems_per_16b, page, h, p % PAGE, c)] = \
                        src[off + i, h, c]
    return out, flagged


def page_copy(pool, page_elems, num_pool_pages, src_pages, dst_pages):
    """The pool after page dst_pages[k] became a copy of src_pages[k] (all
    heads), k in order; pairs with an id out of range are skipped and
    flagged. Returns (pool, flagged)."""
    out = np.array(pool, copy=True)
    flagged = False
    for s, d in zip(src_pages, dst_pages):
        s, d = int(s), int(d)
        if not (0 <= s < num_pool_pages and 0 <= d < num_pool_pages):
            flagged = True
            continue
        out[d * page_elems:(d + 1) * page_elems] = pool[s * page_elems:(s + 1) * page_elems]
    return out, flagged
