"""The decode and prefill calls under HIP graph capture (GPU): a call
captured once and replayed several times, with eager work of the program in
between, gives bitwise the eager result each time. The library's launches
record no memset, allocate nothing and read the plan's metadata uploaded
before capture."""

import pytest
import torch

from gpu_helpers import params_of, to_device
from paper_2509_02121_amd import halo
from workloads import make_config

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("index", [1, 3])
def test_captured_call_replays_bitwise(gpu_lib, index):
    print(f"case: graph capture config {index}", flush=True)
    w = to_device(make_config(index))
    pa = halo.PrefixAttention(params_of(w), w.forest_csr(), "cuda")
    o_eager, lse_eager = pa.alloc_outputs(w.q)
    pa.run(w.q, w.k_pool, w.v_pool, o_eager, lse_eager)
    torch.cuda.synchronize()
    o, lse = pa.alloc_outputs(w.q)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        call = pa.bind(w.q, w.k_pool, w.v_pool, o, lse, side)
        call()                          # warm up on the capture stream
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        call()
    for rep in range(4):
        o.fill_(float("nan"))
        lse.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16 if o.dtype == torch.bfloat16 else torch.int32),
                           o_eager.view(torch.int16 if o.dtype == torch.bfloat16 else torch.int32)), rep
        assert torch.equal(lse, lse_eager), rep
        w.q.mul_(1.0)                   # eager work between replays
