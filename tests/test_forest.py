"""Prefix forest construction from token ids (CPU): the brute-force oracle
against a hand-worked forest and the pairwise longest-common-prefix rule,
then the library's trie builder (halo_prefix_tree_build) against the oracle
on random prompt sets."""

import json
import os
import time

import numpy as np
import pytest

import oracle
from paper_2509_02121_amd import halo

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "prefix_forest.json")


def _canon_oracle(segments, paths):
    keys = [(frozenset(s["members"]), s["start"]) for s in segments]
    table = {k: (s["length"], keys[s["parent"]] if s["parent"] >= 0 else None, len(s["members"]))
             for k, s in zip(keys, segments)}
    return table, [[keys[i] for i in p] for p in paths]


def _canon_library(tree, prompts):
    """Key every segment by (its members, its start offset) after checking
    that the library's own fields agree with its paths and prompts."""
    paths = tree.paths()
    S = tree.num_segments
    members = [set() for _ in range(S)]
    start = [None] * S
    for r, p in enumerate(paths):
        off = 0
        for s in p:
            members[s].add(r)
            assert start[s] in (None, off)
            start[s] = off
            off += int(tree.seg_len[s])
        assert off == len(prompts[r])
    keys = [(frozenset(members[s]), start[s]) for s in range(S)]
    table = {}
    for s in range(S):
        assert members[s], f"segment {s} is on no path"
        assert tree.seg_refcount[s] == len(members[s])
        src, so, n = int(tree.seg_src_request[s]), int(tree.seg_src_offset[s]), int(tree.seg_len[s])
        assert src in members[s] and so == start[s]
        for m in members[s]:
            assert list(prompts[m][start[s]:start[s] + n]) == list(prompts[src][so:so + n])
        par = int(tree.seg_parent[s])
        table[keys[s]] = (n, keys[par] if par >= 0 else None, len(members[s]))
    return table, [[keys[i] for i in p] for p in paths]


def _golden():
    with open(GOLDEN) as f:
        g = json.load(f)
    segs = [dict(members=frozenset(s["members"]), start=s["start"], length=s["length"], parent=s["parent"])
            for s in g["segments"]]
    return g, _canon_oracle(segs, g["paths"])


def test_oracle_matches_hand_worked_forest():
    g, want = _golden()
    segs, paths = oracle.forest.build(g["prompts"], g["page_size"])
    assert _canon_oracle(segs, paths) == want


def _random_prompts(rng, n, page_size, vocab=3):
    """Prompts grown from random earlier prompts (shared prefixes of random,
    often unaligned, length), with exact repeats, page-aligned prefixes of
    others and empty prompts mixed in."""
    prompts = []
    for _ in range(n):
        u = rng.random()
        if prompts and u < 0.15:
            prompts.append(list(prompts[rng.integers(len(prompts))]))
        elif prompts and u < 0.25:
            base = prompts[rng.integers(len(prompts))]
            prompts.append(base[:(len(base) // page_size) * page_size])
        elif u < 0.3:
            prompts.append([])
        else:
            base = prompts[rng.integers(len(prompts))] if prompts else []
            keep = int(rng.integers(0, len(base) + 1))
            tail = rng.integers(0, vocab, size=int(rng.integers(0, 3 * page_size + 2))).tolist()
            prompts.append(list(base[:keep]) + tail)
    return prompts


@pytest.mark.parametrize("page_size", [1, 2, 4, 16])
def test_oracle_pairwise_shared_length(page_size):
    """For every pair, the tokens their paths share are page_size *
    floor(lcp / page_size), or the whole prompt when the prompts are equal
    (lcp by a plain zip, not the oracle's loop); and each path spells its
    prompt."""
    rng = np.random.default_rng(page_size)
    for _ in range(20):
        prompts = _random_prompts(rng, 10, page_size)
        segs, paths = oracle.forest.build(prompts, page_size)
        for r, p in enumerate(paths):
            spelled = []
            for i in p:
                src = prompts[segs[i]["src"]]
                spelled += src[segs[i]["start"]:segs[i]["start"] + segs[i]["length"]]
            assert spelled == prompts[r]
        for r in range(len(prompts)):
            for s in range(len(prompts)):
                n = 0
                for a, b in zip(prompts[r], prompts[s]):
                    if a != b:
                        break
                    n += 1
                want = len(prompts[r]) if prompts[r] == prompts[s] else page_size * (n // page_size)
                shared = sum(segs[i]["length"] for i in set(paths[r]) & set(paths[s]))
                assert shared == want, (r, s)


def test_library_matches_hand_worked_forest():
    g, want = _golden()
    tree = halo.PrefixTree(g["prompts"], g["page_size"])
    assert _canon_library(tree, g["prompts"]) == want
    assert (tree.prompt_tokens, tree.distinct_tokens, tree.num_pages) == (
        g["prompt_tokens"], g["distinct_tokens"], g["num_pages"])


@pytest.mark.parametrize("page_size", [1, 3, 4, 16])
def test_library_matches_oracle_on_random_prompt_sets(page_size):
    rng = np.random.default_rng(100 + page_size)
    for trial in range(40):
        prompts = _random_prompts(rng, int(rng.integers(1, 14)), page_size, vocab=int(rng.integers(2, 5)))
        tree = halo.PrefixTree(prompts, page_size)
        segs, paths = oracle.forest.build(prompts, page_size)
        assert _canon_library(tree, prompts) == _canon_oracle(segs, paths), (trial, prompts)
        assert tree.distinct_tokens == sum(s["length"] for s in segs)
        assert tree.num_pages == sum(-(-s["length"] // page_size) for s in segs)
        # children start on a page boundary; only leaves end inside a page
        parents = set(int(x) for x in tree.seg_parent if x >= 0)
        for s in parents:
            assert tree.seg_len[s] % page_size == 0


def test_library_edge_cases_and_errors():
    assert halo.PrefixTree([]).num_segments == 0
    t = halo.PrefixTree([[], []])
    assert t.num_segments == 0 and t.paths() == [[], []]
    t = halo.PrefixTree([[7] * 33, [7] * 33], page_size=16)     # identical: one shared segment
    assert t.seg_len.tolist() == [33] and t.seg_refcount.tolist() == [2] and t.paths() == [[0], [0]]
    t = halo.PrefixTree([[7] * 33, [7] * 32], page_size=16)     # 32 shared, 1 private
    assert sorted(t.seg_len.tolist()) == [1, 32]
    lib = halo.load_library()
    import ctypes
    h = ctypes.c_void_p()
    bad = np.array([1, 3], np.int32)
    toks = np.zeros(4, np.int32)
    assert lib.halo_prefix_tree_build(halo._ptr(bad), halo._ptr(toks), 1, 16, ctypes.byref(h), None) == \
        halo.HALO_ERR_INVALID_ARGUMENT
    dec = np.array([0, 3, 2], np.int32)
    assert lib.halo_prefix_tree_build(halo._ptr(dec), halo._ptr(toks), 2, 16, ctypes.byref(h), None) == \
        halo.HALO_ERR_INVALID_ARGUMENT
    ok = np.array([0, 3], np.int32)
    assert lib.halo_prefix_tree_build(halo._ptr(ok), halo._ptr(toks), 1, 0, ctypes.byref(h), None) == \
        halo.HALO_ERR_INVALID_ARGUMENT
    assert lib.halo_prefix_tree_build(halo._ptr(ok), None, 1, 16, ctypes.byref(h), None) == \
        halo.HALO_ERR_INVALID_ARGUMENT
    assert lib.halo_prefix_tree_build(halo._ptr(ok), halo._ptr(toks), 1, 16, None, None) == \
        halo.HALO_ERR_INVALID_ARGUMENT
    assert lib.halo_prefix_tree_get(None, None, None, None, None, None, None, None) == \
        halo.HALO_ERR_INVALID_ARGUMENT


def test_library_builds_a_large_batch():
    """The 70B-shaped decode batch as token ids: 1024 prompts in 8 groups of
    128 on 8192-token prefixes plus private suffixes of 256..2048 tokens; the
    forest is 8 shared segments plus 1024 private ones."""
    rng = np.random.default_rng(5)
    prefixes = [rng.integers(0, 32000, size=8192).astype(np.int32) for _ in range(8)]
    prompts = []
    for r in range(1024):
        suffix = rng.integers(0, 32000, size=int(rng.integers(256, 2049))).astype(np.int32)
        suffix[0] = 32000 + r          # private from its first token on
        prompts.append(np.concatenate([prefixes[r // 128], suffix]))
    t0 = time.perf_counter()
    tree = halo.PrefixTree(prompts, 16)
    dt = time.perf_counter() - t0
    total = sum(len(p) for p in prompts)
    print(f"prefix forest of {total} tokens built in {dt * 1e3:.1f} ms (binding included)")
    assert tree.num_segments == 8 + 1024
    assert sorted(tree.seg_refcount.tolist())[-8:] == [128] * 8
    assert tree.distinct_tokens == total - 8 * 127 * 8192
    for r, p in enumerate(tree.paths()):
        assert len(p) == 2 and tree.seg_len[p[0]] == 8192 and tree.seg_refcount[p[0]] == 128
