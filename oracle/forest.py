"""Prefix forest from token ids, by brute force (TEST INFRASTRUCTURE ONLY).

Parity status: pinned by ``tests/test_forest.py`` (a hand-worked forest in
``tests/golden/prefix_forest.json``; every path spells its prompt; the shared
length of every pair of requests is page_size * floor(lcp / page_size), or
the whole prompt for identical prompts, with lcp from a separate character
comparison).

What it follows: §2 (intra-batch prefix sharing: a shared prefix is computed
once and its KV cache reused) and §7 (RadixAttention's prefix tree, on the
paged cache of PagedAttention). The sharing is stated at page granularity,
so every shared boundary falls on a page boundary:
  * chunk k of prompt r is tokens [k*B, min((k+1)*B, len_r)) (B = page size);
  * chunk k of r is shared with s exactly when r and s agree on every token up
    to the end of r's chunk k (their longest common prefix reaches it) and
    their chunks k end at the same position;
  * along r's prompt, a segment is a maximal run of chunks shared with the
    same set of requests; two requests hold the same segment when it covers
    the same chunks for the same set.
Everything below is that definition computed directly from pairwise longest
common prefixes: quadratic in the number of prompts, for small cases only.
"""


def lcp(a, b):
    """Longest common prefix length of two token sequences (plain loop)."""
    n = 0
    while n < len(a) and n < len(b) and a[n] == b[n]:
        n += 1
    return n


def chunk_end(length, k, page_size):
    return min((k + 1) * page_size, length)


def build(prompts, page_size):
    """Returns (segments, paths). segments: list of dicts with keys
    ``members`` (frozenset of requests), ``first_chunk``, ``start`` (token
    offset), ``length``, ``src`` (lowest member), ``parent`` (index or -1),
    in order of first appearance along the prompts in request order.
    paths: per request, its segment indices root first."""
    prompts = [list(p) for p in prompts]
    R = len(prompts)
    L = [[lcp(prompts[r], prompts[s]) for s in range(R)] for r in range(R)]
    segments, index, paths = [], {}, []
    for r in range(R):
        n_chunks = -(-len(prompts[r]) // page_size)
        members = []
        for k in range(n_chunks):
            end = chunk_end(len(prompts[r]), k, page_size)
            members.append(frozenset(s for s in range(R)
                                     if L[r][s] >= end and chunk_end(len(prompts[s]), k, page_size) == end))
        path = []
        k = 0
        while k < n_chunks:
            k1 = k
            while k1 + 1 < n_chunks and members[k1 + 1] == members[k]:
                k1 += 1
            key = (members[k], k)
            if key not in index:
                index[key] = len(segments)
                segments.append(dict(members=members[k], first_chunk=k, start=k * page_size,
                                     length=chunk_end(len(prompts[r]), k1, page_size) - k * page_size,
                                     src=min(members[k]), parent=path[-1] if path else -1))
            path.append(index[key])
            k = k1 + 1
        paths.append(path)
    return segments, paths
