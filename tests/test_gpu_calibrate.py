"""A tiny calibration sweep on the GPU: the decode latency grows with the
private suffix (64 vs 2048 tokens per request, a 30x difference in streamed
K/V), and the fitted model is produced."""

import pytest

import calibrate

pytestmark = pytest.mark.gpu


def test_tiny_calibration_sweep(gpu_lib):
    print("case: calibration sweep (decode R=16 G=16 P=1024, S 64/2048)", flush=True)
    grid = dict(requests=[16], group=[16], prefix=[1024], suffix=[64, 2048])
    pts = calibrate.run([("decode", grid)], calls=20, log=lambda m: print(m, flush=True))
    short, long_ = pts[("decode", 16, 16, 1024, 64)], pts[("decode", 16, 16, 1024, 2048)]
    assert long_ > short > 0
    assert calibrate.check_monotone(pts) == []
