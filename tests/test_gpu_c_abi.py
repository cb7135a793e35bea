"""The C ABI from a C++ program with no Python and no torch (GPU): the
driver in tests/abi_driver reads a seeded batch from a file, runs
halo_plan_create, halo_plan_upload and halo_prefix_attn_decode with the HIP
runtime alone, and writes O and LSE back; they match the oracle. In its
loop mode it decodes the batch's last steps, the plan brought up to date in
place each step (halo_plan_update_lengths, halo_plan_upload_update)."""

import os
import subprocess

import numpy as np
import pytest
import torch

from gpu_helpers import assert_parity, oracle_for
from workloads import make_config

pytestmark = pytest.mark.gpu

DRIVER = os.path.join(os.path.dirname(__file__), "abi_driver", "decode")


def _write_input(path, w, out_dtype):
    code = {torch.float32: 0, torch.bfloat16: 1}
    csr = w.forest_csr()
    S, R = len(csr["seg_len"]), len(csr["req_seg_indptr"]) - 1
    ity = np.int16 if w.dtype == torch.bfloat16 else np.int32
    tv = torch.int16 if w.dtype == torch.bfloat16 else torch.int32
    with open(path, "wb") as f:
        np.array([w.num_q_heads, w.num_kv_heads, w.head_dim, code[w.dtype], code[out_dtype],
                  w.num_pool_pages, S, R], np.int32).tofile(f)
        np.array([w.scale], np.float32).tofile(f)
        for k in ("seg_len", "seg_page_indptr", "seg_page_ids", "req_seg_indptr", "req_seg_ids"):
            np.asarray(csr[k], np.int32).tofile(f)
        for t in (w.q, w.k_pool, w.v_pool):
            t.contiguous().view(tv).cpu().numpy().astype(ity).tofile(f)


@pytest.mark.parametrize("index,out_dtype", [(0, torch.float32), (1, torch.bfloat16), (1, torch.float32)])
def test_decode_through_c_driver(gpu_lib, tmp_path, index, out_dtype):
    print(f"case: C driver config {index} out {out_dtype}", flush=True)
    assert os.path.exists(DRIVER), "tests/abi_driver/decode is not built (the library build makes it)"
    w = make_config(index)
    inp, outp = tmp_path / "in.bin", tmp_path / "out.bin"
    _write_input(inp, w, out_dtype)
    r = subprocess.run([DRIVER, str(inp), str(outp)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    rows = w.q.shape[0] * w.num_q_heads
    raw = np.fromfile(outp, np.uint8)
    oel = 2 if out_dtype == torch.bfloat16 else 4
    o_bytes = rows * w.head_dim * oel
    o = torch.from_numpy(raw[:o_bytes].copy()).view(out_dtype).float().numpy().astype(np.float64)
    lse = np.frombuffer(raw[o_bytes:].tobytes(), np.float32).astype(np.float64)
    o = o.reshape(w.q.shape[0], w.num_q_heads, w.head_dim)
    lse = lse.reshape(w.q.shape[0], w.num_q_heads)
    ro, rl, rr = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rr, f"C driver config {index}")


@pytest.mark.parametrize("index,steps", [(1, 40), (2, 24)])
def test_decode_loop_through_c_driver(gpu_lib, tmp_path, index, steps):
    """The driver plans the batch with every private suffix `steps` tokens
    shorter, then appends a token to each per step (pages reopened from the
    batch's own page lists), updating the plan in place and uploading only
    what changed, double-buffered on a copy stream; the last step is the
    batch itself and matches the oracle."""
    print(f"case: C driver decode loop config {index} steps {steps}", flush=True)
    w = make_config(index)
    inp, outp = tmp_path / "in.bin", tmp_path / "out.bin"
    _write_input(inp, w, torch.bfloat16)
    r = subprocess.run([DRIVER, str(inp), str(outp), str(steps)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    print(r.stdout.strip(), flush=True)
    line = next(x for x in r.stdout.splitlines() if x.startswith("loop "))
    fields = line.split()
    assert int(fields[fields.index("in_place") + 1]) == steps, line
    rows = w.q.shape[0] * w.num_q_heads
    raw = np.fromfile(outp, np.uint8)
    o_bytes = rows * w.head_dim * 2
    o = torch.from_numpy(raw[:o_bytes].copy()).view(torch.bfloat16).float().numpy().astype(np.float64)
    lse = np.frombuffer(raw[o_bytes:].tobytes(), np.float32).astype(np.float64)
    o = o.reshape(w.q.shape[0], w.num_q_heads, w.head_dim)
    lse = lse.reshape(w.q.shape[0], w.num_q_heads)
    ro, rl, rr = oracle_for(w)
    assert_parity(w, o, lse, ro, rl, rr, f"C driver loop config {index}")
