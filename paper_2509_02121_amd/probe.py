"""Python binding of libhalo_probe.so, the context microbenchmarks
(measurement only; ctypes argument marshalling). See include/halo_probe.h."""

import ctypes
import os

from .build import PROBE_LIB_PATH

EXPORTED_SYMBOLS = ("halo_probe_stream_read", "halo_probe_mfma", "halo_probe_exp", "halo_probe_overlap",
                    "halo_probe_last_error")

_LIB = None


def load():
    global _LIB
    if _LIB is None:
        if not os.path.exists(PROBE_LIB_PATH):
            raise RuntimeError(f"{PROBE_LIB_PATH} is not built; run `python -m paper_2509_02121_amd.build`")
        lib = ctypes.CDLL(PROBE_LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        lib.halo_probe_stream_read.argtypes = [vp, i64, vp, i64, i32, i32, i32, i32, i32, vp, vp]
        lib.halo_probe_stream_read.restype = ctypes.c_int
        lib.halo_probe_mfma.argtypes = [i32, i32, i32, vp, vp]
        lib.halo_probe_mfma.restype = ctypes.c_int
        lib.halo_probe_exp.argtypes = [i32, i32, i32, vp, vp]
        lib.halo_probe_exp.restype = ctypes.c_int
        lib.halo_probe_overlap.argtypes = [i32, i32, i32, i32, i32, vp, vp]
        lib.halo_probe_overlap.restype = ctypes.c_int
        lib.halo_probe_last_error.argtypes = []
        lib.halo_probe_last_error.restype = ctypes.c_char_p
        _LIB = lib
    return _LIB


def _check(rc):
    if rc != 0:
        raise RuntimeError(f"probe failed ({rc}): {_LIB.halo_probe_last_error().decode()}")


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def bind_stream_read(pool, tiles, steps_per_item, stages, waves_per_simd, nontemporal, blocks, out, stream=None):
    """A zero-argument callable enqueueing one stream-read probe launch."""
    lib = load()
    assert pool.is_cuda and tiles.is_cuda and out.is_cuda and tiles.dtype.itemsize == 4
    waves = blocks * (8 if waves_per_simd == 2 else 4)
    assert out.numel() >= waves
    args = (pool.data_ptr(), pool.numel() * pool.element_size(), tiles.data_ptr(), tiles.numel(),
            int(steps_per_item), int(stages), int(waves_per_simd), int(nontemporal), int(blocks),
            out.data_ptr(), _stream(stream))
    fn = lib.halo_probe_stream_read

    def call():
        _check(fn(*args))
    return call


def bind_mfma(shape, iters, blocks, out, stream=None):
    lib = load()
    assert out.is_cuda and out.numel() >= blocks * 256
    args = (int(shape), int(iters), int(blocks), out.data_ptr(), _stream(stream))

    def call():
        _check(lib.halo_probe_mfma(*args))
    return call


def bind_exp(valu_per_mfma, iters, blocks, out, stream=None):
    lib = load()
    assert out.is_cuda and out.numel() >= blocks * 256
    args = (int(valu_per_mfma), int(iters), int(blocks), out.data_ptr(), _stream(stream))

    def call():
        _check(lib.halo_probe_exp(*args))
    return call


def bind_overlap(split, valu_per_mfma, use_exp, iters, blocks, out, stream=None):
    lib = load()
    assert out.is_cuda and out.numel() >= blocks * 512
    args = (int(split), int(valu_per_mfma), int(use_exp), int(iters), int(blocks), out.data_ptr(), _stream(stream))

    def call():
        _check(lib.halo_probe_overlap(*args))
    return call
