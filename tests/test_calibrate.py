"""CPU checks of the calibration helpers (calibrate.py): the feature counts
of a point, the fit on synthetic latencies of known coefficients, the
monotonicity check on a planted violation, and the fit quality of the
committed 64/8-head curves."""

import os

import numpy as np

import calibrate
from workloads import CONFIG_NAMES, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_features_count_kv_bytes_pairs_and_rows():
    # 8 requests in 2 groups of 4 on 100-token prefixes, 10 private tokens each
    f = calibrate.features("decode", 8, 4, 100, 10)
    kv_tok = 2 * 100 + 8 * 10
    tok = 2 * 8 * 128 * 2
    assert f == [1.0, kv_tok * tok, 8 * 100 * 32, 8 * 10 * 32, 8 * 32, 1.0, 2 * 100 * tok]
    # one request per prefix: nothing shared, its pairs private, nothing
    # split below SPLIT_KEYS private keys
    f = calibrate.features("decode", 8, 1, 100, 10)
    assert f[2] == 0.0 and f[3] == 8 * 110 * 32 and f[5:] == [0.0, 0.0]
    assert calibrate.features("decode", 8, 1, calibrate.SPLIT_KEYS, 100)[5] == 1.0
    # prefill: 3-token causal chunks see the (shared) prefix and 1, 2, 3 chunk keys
    f = calibrate.features("prefill", 2, 2, 5, 3)
    assert f[2] == 2 * 3 * 5 * 32 and f[3] == 2 * 6 * 32 and f[4] == 2 * 3 * 32
    # no prefix: the group size does not matter
    assert calibrate.features("decode", 8, 1, 0, 10) == calibrate.features("decode", 8, 8, 0, 10)


def test_fit_recovers_known_coefficients():
    """Latencies drawn from the model with known coefficients (1% noise):
    the fit reproduces them, its streaming rate and an unseen point."""
    rng = np.random.default_rng(0)
    true = [3.0, 1.4e-7, 6e-7, 1e-8, 1e-3, 5.0, 5e-8, 2.0]
    pts = []
    for r in (16, 64, 1024):
        for g in (1, 4, 16):
            for p in (0, 512, 4096):
                for s in (64, 1024):
                    f = calibrate.features("decode", r, g, p, s)
                    pts.append((f, calibrate.latency(true, f) * (1 + 0.01 * rng.standard_normal())))
    coef, rel = calibrate.fit(pts)
    assert max(rel) < 0.05
    assert abs(coef[1] - true[1]) / true[1] < 0.1
    pred = calibrate.predict(coef, "decode", 256, 16, 2048, 256)
    want = calibrate.latency(true, calibrate.features("decode", 256, 16, 2048, 256))
    assert abs(pred - want) / want < 0.05


def test_overlap_exponent_spans_sum_and_max():
    """k = 1 adds the streaming and matrix terms; a large k takes their
    maximum."""
    f = [1.0, 1e9, 1e8, 0.0, 0.0, 0.0, 0.0]
    base = [0.0, 1e-7, 1e-6, 0.0, 0.0, 0.0, 0.0]
    assert abs(calibrate.latency(base + [1.0], f) - 200.0) < 1e-6
    assert abs(calibrate.latency(base + [60.0], f) - 100.0) < 2.0


def _stored_calibration(path):
    """Measured points and held-out rows of a committed calibration summary."""
    points, held = {}, {}
    for line in open(path):
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) == 6 and cells[0] in ("decode", "prefill"):
            points[(cells[0], *map(int, cells[1:5]))] = float(cells[5])
        elif len(cells) == 4 and cells[0] in CONFIG_NAMES:
            held[cells[0]] = float(cells[1])
    return points, held


def test_stored_64q_8kv_curves_fit_within_10_percent():
    """The committed 64/8-head calibration: the fitted model predicts each
    stored point from the others (leave-one-out) with a median error of at
    most 10%, decode and prefill, and the held-out 70B-shaped batch (its
    forest is not on the grid) within 10%."""
    points, held = _stored_calibration(os.path.join(ROOT, "profiles", "calibration_curves_64q_8kv.md"))
    saved = calibrate.HQ, calibrate.HKV
    calibrate.HQ, calibrate.HKV = 64, 8
    try:
        s = calibrate.summarize(points)
        assert s["decode"]["loo_median_rel_err"] <= 0.10
        assert s["prefill"]["loo_median_rel_err"] <= 0.10
        rng = np.random.Generator(np.random.PCG64(1004))
        seg_len, paths, _ = synth._forest(4, rng)
        pred = calibrate.predict_forest(list(s["decode"]["coef"].values()), seg_len, paths, None,
                                        num_q_heads=64, num_kv_heads=8, head_dim=128)
        meas = held["llama70b_batch_decode"]
        assert abs(pred - meas) / meas <= 0.10, (pred, meas)
    finally:
        calibrate.HQ, calibrate.HKV = saved


def test_monotonicity_check_flags_planted_violations():
    pts = {("decode", 64, 1, 512, 64): 10.0, ("decode", 64, 1, 512, 256): 14.0,
           ("decode", 64, 4, 512, 64): 9.0, ("decode", 64, 4, 512, 256): 12.0}
    assert calibrate.check_monotone(pts) == []
    pts[("decode", 64, 1, 512, 1024)] = 12.0          # longer suffix, faster: planted
    pts[("decode", 64, 16, 512, 64)] = 11.0           # larger group, slower: planted
    bad = calibrate.check_monotone(pts)
    assert any("S 256->1024" in b for b in bad) and any("G 4->16" in b for b in bad)


def test_forest_features_agree_with_the_grid_features():
    """A uniform forest (R requests, groups of G on P-token prefixes, S
    private tokens) gives the grid point's features, decode and prefill."""
    for (r, g, p, s) in [(8, 4, 100, 10), (8, 1, 100, 10), (8, 8, 0, 10), (6, 3, 1000, 100)]:
        n_pre = r // g if p > 0 else 0
        seg_len = [p] * n_pre + [s] * r
        paths = [([i // g] if p > 0 else []) + [n_pre + i] for i in range(r)]
        assert calibrate.forest_features(seg_len, paths) == calibrate.features("decode", r, g, p, s)
        assert calibrate.forest_features(seg_len, paths, [s] * r)[:5] == \
            calibrate.features("prefill", r, g, p, s)[:5]


def test_forest_prediction_from_token_ids_discounts_shared_prefixes():
    """Through the prefix-tree builder: the same prompts predicted with their
    shared prefix counted once are cheaper than the flattened batch."""
    from paper_2509_02121_amd import halo
    rng = np.random.default_rng(5)
    prefix = rng.integers(0, 1000, size=2048).tolist()
    prompts = [prefix + rng.integers(0, 1000, size=int(n)).tolist() for n in rng.integers(64, 512, size=64)]
    tree = halo.PrefixTree(prompts, 16)
    coef = [3.0, 1.4e-7, 1.3e-6, 1.0e-7, 2.9e-3, 4.6, 2.4e-8, 1.5]
    shared = calibrate.predict_forest(coef, tree.seg_len, tree.paths())
    flat = calibrate.predict_forest(coef, [len(p) for p in prompts], [[r] for r in range(len(prompts))])
    assert tree.distinct_tokens < tree.prompt_tokens and shared < flat
