"""Runs decode_windows of the host-built library (tests/emu) on seeded inputs and returns its
logits, for memory checks of the kernels' addressing on the CPU."""
from __future__ import annotations

import ctypes
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
from paper_2601_09921_amd import pwdec, synth  # noqa: E402


def load(path: str) -> ctypes.CDLL:
    lib = pwdec.bind(ctypes.CDLL(path))
    lib.emu_malloc.restype, lib.emu_malloc.argtypes = ctypes.c_void_p, [ctypes.c_size_t]
    lib.emu_free.restype, lib.emu_free.argtypes = None, [ctypes.c_void_p]
    lib.emu_errors.restype, lib.emu_errors.argtypes = ctypes.c_int, []
    return lib


class Buf:
    """A guard-paged "device" buffer of the host build."""

    def __init__(self, lib, arr: np.ndarray):
        self.lib, self.n, self.dtype, self.shape = lib, arr.nbytes, arr.dtype, arr.shape
        self.ptr = lib.emu_malloc(max(arr.nbytes, 1))
        ctypes.memmove(self.ptr, np.ascontiguousarray(arr).ctypes.data, arr.nbytes)

    def get(self) -> np.ndarray:
        out = np.empty(self.shape, self.dtype)
        ctypes.memmove(out.ctypes.data, self.ptr, self.n)
        return out

    def free(self):
        self.lib.emu_free(self.ptr)


def decode(lib, wl, weights: dict, meas_bits: np.ndarray, types: np.ndarray, recurrent: bool = False):
    """decode_windows (or decode_windows_recurrent) through the C ABI of the host build."""
    ts = pwdec.TOKENS_GRID if getattr(wl, "grid", False) else pwdec.TOKENS_STABILIZERS
    emb = pwdec.EMBED_RESNET if "res" in weights else pwdec.EMBED_LINEAR
    dil = tuple(weights["dilations"]) if weights.get("dilations") else (0, 0, 0)
    blob = pwdec.make_blob(wl.d, wl.W, wl.D, wl.L, wl.H, wl.F, wl.dtype, weights, ts)
    n = types.shape[0]
    g = pwdec.geometry(wl.d, wl.W, n)
    m = pwdec.dims(wl.D, wl.L, wl.H, wl.mlp_ratio, wl.dtype, ts, emb, dil)
    h = ctypes.c_void_p()
    buf = ctypes.create_string_buffer(blob, len(blob))
    rc = lib.decoder_create(ctypes.byref(g), ctypes.byref(m), buf, len(blob), ctypes.byref(h))
    if rc != 0:
        raise pwdec.PwdError(rc, lib.decoder_last_error().decode())
    k = wl.d if recurrent else 1
    meas = Buf(lib, synth.pack_bits(meas_bits).view(np.uint32))
    tt = Buf(lib, types.astype(np.uint8))
    logits = Buf(lib, np.full(n * k, np.nan, np.float32))
    bits = Buf(lib, np.full(n * k, 7, np.uint8))
    fn = lib.decode_windows_recurrent if recurrent else lib.decode_windows
    vp = ctypes.c_void_p
    rc = fn(h, vp(meas.ptr), vp(tt.ptr), n, vp(logits.ptr), vp(bits.ptr), None)
    if rc != 0:
        raise pwdec.PwdError(rc, lib.decoder_last_error().decode())
    rc = lib.decoder_sync_status(h, None)
    out = logits.get().reshape(n, k) if recurrent else logits.get(), bits.get(), rc
    lib.decoder_destroy(h)
    for b in (meas, tt, logits, bits):
        b.free()
    return out
