"""Thin ctypes binding of libpwdec.so (include/pwdec.h).

Argument marshalling only: every step of the decoder runs in the library's HIP kernels.
Device buffers are torch tensors on the decoder's GPU; torch supplies memory and streams.
"""
from __future__ import annotations

import ctypes
import os
import re
import struct

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpwdec.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "pwdec.h")

PWD_OK, PWD_EINVAL, PWD_EUNSUPPORTED, PWD_EBLOB, PWD_ENOMEM, PWD_EHIP, PWD_EBATCH, PWD_EDEVICE = (
    0, -1, -2, -3, -4, -5, -6, -7)
DTYPE_F32, DTYPE_BF16, DTYPE_MXFP8 = 0, 1, 2
BLOB_MAGIC = 0x31445750
BLOB_VERSION = 1


class PwdError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"pwdec error {code}: {msg}")
        self.code = code


class Geometry(ctypes.Structure):
    _fields_ = [("distance", ctypes.c_int32), ("window_rounds", ctypes.c_int32),
                ("max_windows", ctypes.c_int32)]


class ModelDims(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("mlp_ratio", ctypes.c_int32), ("dtype", ctypes.c_int32), ("token_set", ctypes.c_int32),
                ("embedder", ctypes.c_int32), ("conv_dilation", ctypes.c_int32 * 3)]


NUM_STAGES = 12
STAGE_NAMES = ["embed_qkv", "attention", "post_qkv", "post_embed_qkv", "post", "readout", "fp32_window",
               "stream_split", "stream_combine", "out_proj", "dilated_conv", "resident"]
SCHEDULE_AUTO, SCHEDULE_LAYERS, SCHEDULE_RESIDENT = 0, 1, 2


class StageTimes(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * NUM_STAGES), ("launches", ctypes.c_int64 * NUM_STAGES)]


_lib = None


def load_library() -> ctypes.CDLL:
    """Loads the in-tree libpwdec.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2601_09921_amd.build.build()")
    _lib = bind(ctypes.CDLL(LIB_PATH))
    return _lib


def bind(lib: ctypes.CDLL) -> ctypes.CDLL:
    """Declares the argument and result types of the include/pwdec.h entry points on `lib`."""
    P, I64, VP = ctypes.POINTER, ctypes.c_int64, ctypes.c_void_p
    sig = {
        "decoder_blob_floats": (ctypes.c_size_t, [P(Geometry), P(ModelDims)]),
        "decoder_validate_config": (ctypes.c_int, [P(Geometry), P(ModelDims)]),
        "decoder_create": (ctypes.c_int, [P(Geometry), P(ModelDims), ctypes.c_void_p, ctypes.c_size_t, P(VP)]),
        "decode_windows": (ctypes.c_int, [VP, VP, VP, I64, VP, VP, VP]),
        "decode_windows_recurrent": (ctypes.c_int, [VP, VP, VP, I64, VP, VP, VP]),
        "decode_windows_noalloc": (ctypes.c_int, [VP, VP, VP, I64, VP, VP, VP]),
        "decoder_detection_events": (ctypes.c_int, [VP, VP, VP, I64, VP, VP]),
        "decode_stream": (ctypes.c_int, [VP, VP, I64, VP, VP, VP, VP, VP, VP]),
        "decoder_sync_status": (ctypes.c_int, [VP, VP]),
        "decoder_last_error": (ctypes.c_char_p, []),
        "decoder_destroy": (ctypes.c_int, [VP]),
        "decoder_profile": (ctypes.c_int, [VP, ctypes.c_int]),
        "decoder_schedule": (ctypes.c_int, [VP, ctypes.c_int]),
        "decoder_profile_read": (ctypes.c_int, [VP, P(StageTimes)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    return lib


def header_functions() -> list[str]:
    """Names of the functions declared in include/pwdec.h."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)


def _check(rc: int):
    if rc != PWD_OK:
        raise PwdError(rc, load_library().decoder_last_error().decode())


def geometry(d: int, W: int, max_windows: int) -> Geometry:
    return Geometry(d, W, max_windows)


TOKENS_STABILIZERS, TOKENS_GRID = 0, 1


EMBED_LINEAR, EMBED_RESNET = 0, 1


def dims(D: int, L: int, H: int, mlp_ratio: int, dtype: int, token_set: int = TOKENS_STABILIZERS,
         embedder: int = EMBED_LINEAR, dilations=(0, 0, 0)) -> ModelDims:
    return ModelDims(D, L, H, mlp_ratio, dtype, token_set, embedder, (ctypes.c_int32 * 3)(*dilations))


def pack_dilations(dil) -> int:
    """Blob header word 13: byte j = dilation of the j-th dilated convolution (0: none)."""
    dil = list(dil) if dil else [0, 0, 0]
    return dil[0] | (dil[1] << 8) | (dil[2] << 16)


def make_blob(d: int, W: int, D: int, L: int, H: int, F: int, dtype: int, weights: dict,
              token_set: int = TOKENS_STABILIZERS) -> bytes:
    """Serializes a weight dict into the library's blob format (header + fp32 tensors)."""
    kappa = np.float32(weights["kappa"])
    eps = np.float32(weights["eps"])
    hdr = [BLOB_MAGIC, BLOB_VERSION, d, W, D, L, H, F, dtype,
           struct.unpack("<I", struct.pack("<f", kappa))[0],
           struct.unpack("<I", struct.pack("<f", eps))[0], token_set,
           EMBED_RESNET if "res" in weights else EMBED_LINEAR, pack_dilations(weights.get("dilations")), 0, 0]
    parts = [weights["w_e"], weights["b_e"]]
    for lw in weights["layers"]:
        parts += [lw[k] for k in ("Wq", "bq", "Wk", "bk", "Wv", "bv", "Wo", "bo", "g1", "be1",
                                  "W1", "b1", "W2", "b2", "g2", "be2")]
    parts += [weights["Wc"], weights["bc"], weights["w_o"], weights["b_o"], weights["beta"]]
    if "res" in weights:
        parts += [weights["res"][k] for k in ("W1", "b1", "W2", "b2")]
    if weights.get("dilations"):
        for lw in weights["layers"]:
            parts += [lw["Wd"], lw["bd"]]
    body = np.concatenate([np.asarray(p, dtype=np.float64).ravel() for p in parts]).astype("<f4")
    return struct.pack("<16I", *hdr) + body.tobytes()


def _dtype_names(t) -> str:
    return str(t.dtype).replace("torch.", "")


def require(t, name: str, dtypes: tuple, device: int, shape: tuple | None = None, min_numel: int | None = None):
    """Checks a device buffer before its pointer crosses the ABI: a CUDA tensor on the decoder's
    device, of one of `dtypes` (names such as "int32"), contiguous, and of exactly `shape` or at
    least `min_numel` elements. The kernels index these buffers with the decoder's geometry, so
    a mismatch would be an out-of-bounds device access; it raises ValueError instead."""
    if t is None:
        raise ValueError(f"{name}: a tensor is required")
    if not getattr(t, "is_cuda", False):
        raise ValueError(f"{name}: must be a CUDA tensor (got device {getattr(t, 'device', '?')})")
    if t.device.index is not None and t.device.index != device:
        raise ValueError(f"{name}: on cuda:{t.device.index}, the decoder is on cuda:{device}")
    if _dtype_names(t) not in dtypes:
        raise ValueError(f"{name}: dtype {_dtype_names(t)}, need one of {', '.join(dtypes)}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, need {tuple(shape)}")
    if min_numel is not None and t.numel() < min_numel:
        raise ValueError(f"{name}: {t.numel()} elements, need at least {min_numel}")


WORDS = ("int32", "uint32")


def _stream_ptr(stream) -> ctypes.c_void_p:
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class Decoder:
    """Owns one pwd_decoder handle."""

    def __init__(self, d: int, W: int, max_windows: int, D: int, L: int, H: int, mlp_ratio: int,
                 dtype: int, blob: bytes, token_set: int = TOKENS_STABILIZERS, embedder: int = EMBED_LINEAR,
                 dilations=(0, 0, 0)):
        import torch
        # torch's HIP runtime starts first: created the other way round (the library's HIP calls
        # before torch initialises its device), torch then finds no GPU in this process
        self.device = torch.cuda.current_device()   # decoder_create uses the current HIP device
        lib = load_library()
        self._lib = lib
        self.d, self.W, self.max_windows = d, W, max_windows
        self.N = d * d - 1
        self.words = (self.N + 31) // 32
        g, m = geometry(d, W, max_windows), dims(D, L, H, mlp_ratio, dtype, token_set, embedder, dilations)
        h = ctypes.c_void_p()
        buf = ctypes.create_string_buffer(blob, len(blob))
        _check(lib.decoder_create(ctypes.byref(g), ctypes.byref(m), buf, len(blob), ctypes.byref(h)))
        self._h = h

    @classmethod
    def from_workload(cls, wl, weights: dict, max_windows: int | None = None) -> "Decoder":
        ts = TOKENS_GRID if getattr(wl, "grid", False) else TOKENS_STABILIZERS
        emb = EMBED_RESNET if "res" in weights else EMBED_LINEAR
        blob = make_blob(wl.d, wl.W, wl.D, wl.L, wl.H, wl.F, wl.dtype, weights, ts)
        dil = tuple(weights["dilations"]) if weights.get("dilations") else (0, 0, 0)
        return cls(wl.d, wl.W, max_windows or wl.B, wl.D, wl.L, wl.H, wl.mlp_ratio, wl.dtype, blob, ts, emb, dil)

    def _windows_in(self, meas, types) -> int:
        require(types, "types", ("uint8",), self.device)
        if types.dim() != 1:
            raise ValueError(f"types: shape {tuple(types.shape)}, need (n,)")
        n = types.shape[0]
        if n > self.max_windows:
            raise ValueError(f"{n} windows, the decoder was created for at most {self.max_windows}")
        require(meas, "meas", WORDS, self.device, shape=(n, self.W + 1, self.words))
        return n

    def decode(self, meas, types, logits, bits, stream=None):
        """meas: int32/uint32 [n][W+1][words] cuda tensor; types: uint8 [n]; outputs float32/uint8 [n]."""
        n = self._windows_in(meas, types)
        require(logits, "logits", ("float32",), self.device, min_numel=n)
        require(bits, "bits", ("uint8",), self.device, min_numel=n)
        _check(self._lib.decode_windows(self._h, ctypes.c_void_p(meas.data_ptr()),
                                        ctypes.c_void_p(types.data_ptr()), n,
                                        ctypes.c_void_p(logits.data_ptr()), ctypes.c_void_p(bits.data_ptr()),
                                        _stream_ptr(stream)))

    def decode_noalloc(self, meas, types, logits, bits, stream=None):
        """As decode, on the library's fixed per-GPU scratch instead of the handle's (no
        allocation; calls on one GPU must not overlap)."""
        n = self._windows_in(meas, types)
        require(logits, "logits", ("float32",), self.device, min_numel=n)
        require(bits, "bits", ("uint8",), self.device, min_numel=n)
        _check(self._lib.decode_windows_noalloc(self._h, ctypes.c_void_p(meas.data_ptr()),
                                                ctypes.c_void_p(types.data_ptr()), n,
                                                ctypes.c_void_p(logits.data_ptr()), ctypes.c_void_p(bits.data_ptr()),
                                                _stream_ptr(stream)))

    def decode_recurrent(self, meas, types, logits, bits, stream=None):
        """As decode, with outputs float32 / uint8 [n][distance]: a readout after each of the
        last `distance` rounds (the recurrent branch of Algorithm 1)."""
        n = self._windows_in(meas, types)
        require(logits, "logits", ("float32",), self.device, min_numel=n * self.d)
        require(bits, "bits", ("uint8",), self.device, min_numel=n * self.d)
        _check(self._lib.decode_windows_recurrent(self._h, ctypes.c_void_p(meas.data_ptr()),
                                                  ctypes.c_void_p(types.data_ptr()), n,
                                                  ctypes.c_void_p(logits.data_ptr()),
                                                  ctypes.c_void_p(bits.data_ptr()), _stream_ptr(stream)))

    def decode_stream(self, rounds, bit, prob=None, window_logits=None, window_bits=None, stream=None,
                      window_probs=None):
        """rounds: int32/uint32 [T][words] cuda tensor of packed measurement rounds; bit: uint8 [1]
        out; prob: float32 [1] out or None; window_logits / window_bits / window_probs: float32 /
        uint8 / float32 [ceil(T/d)] out or None (window_probs: sigmoid of each logit)."""
        ptr = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)
        require(rounds, "rounds", WORDS, self.device)
        if rounds.dim() != 2 or rounds.shape[1] != self.words:
            raise ValueError(f"rounds: shape {tuple(rounds.shape)}, need (T, {self.words})")
        m = -(-rounds.shape[0] // self.d)
        require(bit, "bit", ("uint8",), self.device, min_numel=1)
        if prob is not None:
            require(prob, "prob", ("float32",), self.device, min_numel=1)
        if window_logits is not None:
            require(window_logits, "window_logits", ("float32",), self.device, min_numel=m)
        if window_bits is not None:
            require(window_bits, "window_bits", ("uint8",), self.device, min_numel=m)
        if window_probs is not None:
            require(window_probs, "window_probs", ("float32",), self.device, min_numel=m)
        _check(self._lib.decode_stream(self._h, ptr(rounds), rounds.shape[0], ptr(window_logits),
                                       ptr(window_bits), ptr(window_probs), ptr(bit), ptr(prob),
                                       _stream_ptr(stream)))

    def detection_events(self, meas, types, events, stream=None):
        """events: int32/uint32 [n][W][words] out."""
        n = self._windows_in(meas, types)
        require(events, "events", WORDS, self.device, shape=(n, self.W, self.words))
        _check(self._lib.decoder_detection_events(self._h, ctypes.c_void_p(meas.data_ptr()),
                                                  ctypes.c_void_p(types.data_ptr()), n,
                                                  ctypes.c_void_p(events.data_ptr()), _stream_ptr(stream)))

    def sync_status(self, stream=None) -> int:
        return self._lib.decoder_sync_status(self._h, _stream_ptr(stream))

    def schedule(self, which: int):
        """SCHEDULE_AUTO, SCHEDULE_LAYERS or SCHEDULE_RESIDENT for the following decodes."""
        _check(self._lib.decoder_schedule(self._h, which))

    def profile(self, enable: bool):
        """Per-stage kernel timing with HIP events on the decode stream (on/off)."""
        _check(self._lib.decoder_profile(self._h, 1 if enable else 0))

    def profile_read(self) -> dict:
        """{stage: (total ms, launches)} of the launches recorded since the last read."""
        st = StageTimes()
        _check(self._lib.decoder_profile_read(self._h, ctypes.byref(st)))
        return {STAGE_NAMES[i]: (st.ms[i], st.launches[i]) for i in range(NUM_STAGES) if st.launches[i]}

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            self._lib.decoder_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
