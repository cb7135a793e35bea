"""The planner's tuning knobs reach code paths the default plans do not use:
waves sharing one narrow item and merging in LDS (HALO_SPLIT), shared rows
forced onto wide items or kept off them (HALO_WIDE, HALO_WIDE_ROWS), other
key-chunk lengths and dealing limits. Each setting must still give the
oracle's result (GPU, through the C ABI)."""

import os

import numpy as np
import pytest
import torch

from gpu_helpers import assert_parity, oracle_for, run_library
from workloads import build_workload, make_config, random_forest

pytestmark = pytest.mark.gpu

KNOBS = [
    {"HALO_SPLIT": "2"},
    {"HALO_SPLIT": "8"},
    {"HALO_SPLIT": "4", "HALO_KC_PRIVATE": "64"},
    {"HALO_WIDE": "1", "HALO_WIDE_ROWS": "64", "HALO_KC_WIDE": "256"},
    {"HALO_WIDE": "0"},
    {"HALO_KC_SHARED": "96", "HALO_SHARED_UNIT": "1"},
    {"HALO_ITEMS_PER_BLOCK": "1"},
]


@pytest.fixture
def knobs(request):
    env = request.param
    saved = {k: os.environ.get(k) for k in env}
    os.environ.update(env)
    yield env
    for k, v in saved.items():
        if v is None:
            os.environ.pop(k, None)
        else:
            os.environ[k] = v


@pytest.mark.parametrize("knobs", KNOBS, indirect=True, ids=[",".join(f"{k}={v}" for k, v in e.items())
                                                             for e in KNOBS])
def test_knob_settings_match_the_oracle(gpu_lib, knobs):
    print(f"case: planner knobs {knobs}", flush=True)
    w = make_config(1)                                   # Llama-8B-shaped decode
    o, lse, _ = run_library(w)
    ro, rl, rows = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rows, f"llama8b {knobs}")
    for seed in range(3):
        rng = np.random.default_rng(77 + seed)
        dtype = torch.bfloat16 if seed != 1 else torch.float32
        seg_len, paths, q_len = random_forest(rng, int(rng.integers(4, 20)), max_len=400,
                                              prefill=seed == 2, max_q=60)
        w = build_workload("knob", 300 + seed, 8, 2, 128 if seed != 1 else 64, dtype, seg_len, paths, q_len,
                           value_scale=0.5 if dtype == torch.bfloat16 else 1.0)
        o, lse, _ = run_library(w)
        ro, rl, rows = oracle_for(w)
        assert_parity(w, o, lse, ro, rl, rows, f"forest {seed} {knobs}")
