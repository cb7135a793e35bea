"""The planner's tuning options reach code paths the default plans do not
use: shared rows forced onto wide items or kept off them, other key-chunk
lengths, fewer items per narrow workgroup. Each setting must still give the
oracle's result (GPU, through the C ABI)."""

import numpy as np
import pytest
import torch

from gpu_helpers import assert_parity, oracle_for, params_of, to_device
from paper_2509_02121_amd import halo
from workloads import build_workload, make_config, random_forest

pytestmark = pytest.mark.gpu

OPTIONS = [
    {"wide": 1, "wide_rows": 64, "kc_wide": 256},
    {"wide": 0},
    {"kc_shared": 96, "shared_unit": 1},
    {"kc_private": 64, "items_per_block": 3},
    {"items_per_block": 1},
    {"wide": 1, "wide_min_items": 100000, "kc_private": 1024},
]


def _run(w, options):
    to_device(w)
    pa = halo.PrefixAttention(params_of(w), w.forest_csr(), "cuda", options)
    o, lse = pa.run(w.q, w.k_pool, w.v_pool)
    torch.cuda.synchronize()
    return o.double().cpu().numpy(), lse.double().cpu().numpy()


@pytest.mark.parametrize("opts", OPTIONS, ids=[",".join(f"{k}={v}" for k, v in e.items()) for e in OPTIONS])
def test_option_settings_match_the_oracle(gpu_lib, opts):
    print(f"case: planner options {opts}", flush=True)
    w = make_config(1)                                   # Llama-8B-shaped decode
    o, lse = _run(w, opts)
    ro, rl, rows = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rows, f"llama8b {opts}")
    for seed in range(3):
        rng = np.random.default_rng(77 + seed)
        dtype = torch.bfloat16 if seed != 1 else torch.float32
        seg_len, paths, q_len = random_forest(rng, int(rng.integers(4, 20)), max_len=400,
                                              prefill=seed == 2, max_q=60)
        w = build_workload("knob", 300 + seed, 8, 2, 128 if seed != 1 else 64, dtype, seg_len, paths, q_len,
                           value_scale=0.5 if dtype == torch.bfloat16 else 1.0)
        o, lse = _run(w, opts)
        ro, rl, rows = oracle_for(w)
        assert_parity(w, o, lse, ro, rl, rows, f"forest {seed} {opts}")


@pytest.mark.parametrize("n_req,wide_rows", [(1, 32), (3, 96), (9, 256), (17, 64), (40, 32)])
def test_mixed_wide_and_narrow_launch_cycles(gpu_lib, n_req, wide_rows):
    """Wide and narrow workgroups are launched in whole 4-round cycles; wide
    counts padded to whole cycles and narrow counts that end inside a cycle
    must still cover every item once (oracle parity on decode forests with
    wide items forced)."""
    print(f"case: launch cycles n_req={n_req} wide_rows={wide_rows}", flush=True)
    rng = np.random.default_rng(1000 + n_req)
    seg_len, paths, q_len = random_forest(rng, n_req, max_len=300, share_prob=0.9)
    w = build_workload("cycles", 400 + n_req, 8, 2, 128, torch.bfloat16, seg_len, paths, q_len,
                       value_scale=0.5)
    o, lse = _run(w, {"wide": 1, "wide_rows": wide_rows, "kc_wide": 64})
    ro, rl, rows = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rows, f"cycles {n_req} {wide_rows}")


@pytest.mark.parametrize("dtype,d,opts", [
    (torch.float32, 64, None), (torch.float32, 128, {"kc_private": 4096}),
    (torch.bfloat16, 128, {"kc_private": 4096, "append_reserve": 100}), (torch.bfloat16, 128, None)],
    ids=["f32-d64", "f32-d128-kc4096", "bf16-kc4096-r100", "bf16"])
def test_long_private_spans_and_grown_plans(gpu_lib, dtype, d, opts):
    """Private suffixes of 600-3000 keys: items whose later spans run to
    1024 keys and last spans cut to leave the growth reserve. Oracle parity
    for a fresh plan, and for a plan made for shorter suffixes (up to the
    reserve less, fewer pages) and then brought up to the full forest in
    place, its new page ids included."""
    print(f"case: long private spans {dtype} d={d} {opts}", flush=True)
    rng = np.random.default_rng(4242 + d)
    n_req = 12
    seg_len = [int(rng.integers(100, 700))] + [int(x) for x in rng.integers(600, 3000, size=n_req)]
    paths = [[0, 1 + r] if r % 3 else [1 + r] for r in range(n_req)]
    w = build_workload("long", 500 + d, 8, 2, d, dtype, seg_len, paths, None,
                       value_scale=0.5 if dtype == torch.bfloat16 else 1.0)
    o, lse = _run(w, opts)
    ro, rl, rows = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rows, f"long fresh {dtype} {d}")
    reserve = (opts or {}).get("append_reserve", 256)
    full = w.forest_csr()
    short = {k: (None if v is None else np.array(v)) for k, v in full.items()}
    cut = np.zeros(len(seg_len), np.int64)
    cut[1:] = rng.integers(1, reserve + 1, size=n_req)
    short_len = np.asarray(full["seg_len"], np.int64) - cut
    pages = [list(p[:(int(n) + 15) // 16]) for p, n in zip(w.seg_pages, short_len)]
    short["seg_len"] = short_len.astype(np.int32)
    short["seg_page_indptr"] = np.concatenate([[0], np.cumsum([len(p) for p in pages])]).astype(np.int32)
    short["seg_page_ids"] = np.concatenate(pages).astype(np.int32)
    assert (np.diff(short["seg_page_indptr"]) < np.diff(full["seg_page_indptr"])).any()
    pa = halo.PrefixAttention(params_of(w), short, "cuda", opts)
    assert pa.update(full), "growth within the reserve updates in place"
    o, lse = pa.run(w.q, w.k_pool, w.v_pool)
    torch.cuda.synchronize()
    assert_parity(w, o.double().cpu().numpy(), lse.double().cpu().numpy(), ro, rl, rows,
                  f"long grown {dtype} {d}")


@pytest.mark.parametrize("dtype,opts", [(torch.float32, None), (torch.bfloat16, {"wide": 0})],
                         ids=["f32", "bf16-narrow"])
def test_long_prefixes_in_narrow_prefill_items(gpu_lib, dtype, opts):
    """Prefill chunks over 1500-3000-token cached prefixes in narrow items:
    a first span of at most 512 keys, later spans of up to 1024, and the
    causal chunk span after them (oracle parity)."""
    print(f"case: long prefixes, narrow prefill {dtype} {opts}", flush=True)
    rng = np.random.default_rng(5151)
    n_req = 6
    seg_len = [int(rng.integers(1500, 3000))] + [int(x) for x in rng.integers(1, 100, size=n_req)]
    paths = [[0, 1 + r] for r in range(n_req)]
    q_len = seg_len[1:]
    w = build_workload("longpf", 600, 8, 2, 128, dtype, seg_len, paths, q_len,
                       value_scale=0.5 if dtype == torch.bfloat16 else 1.0)
    plan = halo.Plan.from_csr(params_of(w), w.forest_csr(), opts)
    spans = plan.inspect()["spans"]
    assert (spans[:, 2] - spans[:, 1]).max() > 512, "later spans longer than a first span"
    o, lse = _run(w, opts)
    ro, rl, rows = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rows, f"long prefix prefill {dtype}")


@pytest.mark.parametrize("seed", range(6))
def test_random_long_forests_with_random_options_fresh_and_grown(gpu_lib, seed):
    """Random decode forests with suffixes up to 3000 tokens and random
    options (growth reserve, private and shared chunk lengths, wide items):
    a fresh plan, and a plan made for private segments up to the reserve
    shorter (fewer pages) and then updated in place to the full forest, both
    against the oracle."""
    rng = np.random.default_rng(7000 + seed)
    dtype = torch.bfloat16 if seed % 3 else torch.float32
    d = 128 if seed % 4 else 64
    seg_len, paths, _ = random_forest(rng, int(rng.integers(2, 24)), max_len=int(rng.choice([600, 1500, 3000])))
    opts = {"append_reserve": int(rng.integers(1, 257))}
    if rng.random() < 0.5:
        opts["kc_private"] = int(rng.integers(1, 100)) * 32
    if rng.random() < 0.3:
        opts["kc_shared"] = int(rng.integers(1, 32)) * 32
    if dtype == torch.bfloat16 and rng.random() < 0.3:
        opts["wide"] = 1
    print(f"case: random long forest {seed} {dtype} d={d} {opts}", flush=True)
    w = build_workload("sweep", 9000 + seed, 8, 2, d, dtype, seg_len, paths, None,
                       value_scale=0.5 if dtype == torch.bfloat16 else 1.0)
    o, lse = _run(w, opts)
    ro, rl, rows = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rows, f"random long fresh {seed}")
    full = w.forest_csr()
    refs = np.bincount(full["req_seg_ids"], minlength=len(seg_len))
    cut = np.where((refs == 1) & (np.asarray(seg_len) > 1),
                   rng.integers(0, opts["append_reserve"] + 1, size=len(seg_len)), 0)
    short_len = np.maximum(np.asarray(full["seg_len"], np.int64) - cut, np.minimum(1, np.asarray(full["seg_len"])))
    pages = [list(p[:(int(n) + 15) // 16]) for p, n in zip(w.seg_pages, short_len)]
    short = dict(full, seg_len=short_len.astype(np.int32),
                 seg_page_indptr=np.concatenate([[0], np.cumsum([len(p) for p in pages])]).astype(np.int32),
                 seg_page_ids=np.concatenate([np.asarray(p, np.int32) for p in pages] + [np.zeros(0, np.int32)]))
    pa = halo.PrefixAttention(params_of(w), short, "cuda", opts)
    assert pa.update(full), "growth within the reserve updates in place"
    o, lse = pa.run(w.q, w.k_pool, w.v_pool)
    torch.cuda.synchronize()
    assert_parity(w, o.double().cpu().numpy(), lse.double().cpu().numpy(), ro, rl, rows,
                  f"random long grown {seed}")
