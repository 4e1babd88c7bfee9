"""Host-only checks of the C ABI: the library loads, exports every function the header
declares, and validates configurations and weight blobs without touching a device."""
import ctypes
import dataclasses
import struct

import pytest

from paper_2601_09921_amd import pwdec, synth


@pytest.fixture(scope="module")
def lib():
    return pwdec.load_library()


def test_exports_every_header_function(lib):
    names = pwdec.header_functions()
    assert {"decoder_create", "decode_windows", "decoder_destroy", "decoder_detection_events",
            "decoder_validate_config", "decoder_last_error", "decoder_sync_status"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def validate(lib, d=7, W=14, B=16, D=128, L=3, H=8, r=4, dt=1, ts=0, emb=0, dil=(0, 0, 0)):
    g, m = pwdec.geometry(d, W, B), pwdec.dims(D, L, H, r, dt, ts, emb, dil)
    return lib.decoder_validate_config(ctypes.byref(g), ctypes.byref(m))


@pytest.mark.parametrize("wl", list(synth.WORKLOADS.values()), ids=list(synth.WORKLOADS))
def test_workloads_are_supported(lib, wl):
    assert validate(lib, wl.d, wl.W, wl.B, wl.D, wl.L, wl.H, wl.mlp_ratio, wl.dtype) == pwdec.PWD_OK


@pytest.mark.parametrize("kw", [
    dict(d=4), dict(d=1), dict(d=65), dict(d=37, W=37), dict(d=27, W=27, D=256, H=4),
    dict(W=6), dict(W=22), dict(B=0), dict(r=3), dict(r=6), dict(L=0),
    dict(H=3), dict(D=96, H=6), dict(D=128, H=1), dict(D=256, H=2), dict(dt=3), dict(dt=0, D=256, H=8),
    dict(dt=2, D=64, H=4), dict(dt=2, ts=1, dil=(1, 2, 4)),
    dict(ts=2), dict(ts=-1), dict(ts=1, d=35, W=35), dict(emb=2), dict(emb=-1),
    dict(dil=(1, 2, 4)), dict(ts=1, dil=(1, 0, 2)), dict(ts=1, dil=(1, 2, 8)), dict(ts=1, dil=(-1, 1, 1)),
    dict(dt=0, d=11, W=22, D=64, H=4),
])
def test_rejects_unsupported(lib, kw):
    assert validate(lib, **kw) == pwdec.PWD_EUNSUPPORTED
    assert lib.decoder_last_error()


@pytest.mark.parametrize("kw", [
    dict(D=128, H=2), dict(D=256, H=4), dict(d=25, W=50, D=256, H=4), dict(d=25, W=75, D=128, H=2),
    dict(D=256, H=16), dict(dt=0, d=3, W=6, D=64, H=1),
    dict(d=27, W=54, D=256, H=8), dict(d=35, W=35, D=128, H=8), dict(d=35, W=105, D=256, H=8),
    dict(ts=1), dict(ts=1, d=25, W=50, D=256, H=8), dict(ts=1, d=33, W=33), dict(ts=1, dt=0, d=3, W=6, D=64, H=4),
    dict(r=5), dict(r=5, d=25, W=50, D=256, H=8), dict(r=5, dt=0, d=3, W=6, D=64, H=4),
    dict(emb=1), dict(emb=1, ts=1, d=25, W=50, D=256, H=8), dict(emb=1, dt=0, d=3, W=6, D=64, H=4),
    dict(ts=1, dil=(1, 2, 4)), dict(ts=1, dil=(7, 7, 7)), dict(ts=1, dt=0, d=3, W=6, D=32, H=2, dil=(1, 2, 3)),
    dict(ts=1, D=256, H=8, dil=(1, 2, 4)),
    dict(dt=2), dict(dt=2, d=25, W=50, D=256, H=8), dict(dt=2, r=5), dict(dt=2, emb=1, ts=1, d=11, W=22, D=256, H=8),
])
def test_supported_head_sizes(lib, kw):
    """Head sizes 16, 32 and 64 on the bf16 path (LDS for K and V of one head of 64 at
    d = 25: 2 x 79 KB), 64 on the fp32 path, and distances past 25 while the attention tile
    fits (d = 35, heads of 16 or 32: 155 KB; d = 37 and d = 27 with heads of 64 do not),
    the (d+1)^2 token set, whose tile is counted in grid tokens (d = 33: 1156 tokens fit,
    d = 35: 1296 do not), and feed-forward widths of 4 and 5 times d_model (3 and 6 are
    rejected), and the MXFP8 option (dt=2) on such networks without dilated convolutions."""
    assert validate(lib, **kw) == pwdec.PWD_OK


def test_null_arguments(lib):
    assert lib.decoder_validate_config(None, None) == pwdec.PWD_EINVAL
    h = ctypes.c_void_p()
    g, m = pwdec.geometry(3, 6, 4), pwdec.dims(64, 2, 4, 4, 0)
    assert lib.decoder_create(ctypes.byref(g), ctypes.byref(m), None, 0, ctypes.byref(h)) == pwdec.PWD_EINVAL
    assert lib.decode_windows(None, None, None, 0, None, None, None) == pwdec.PWD_EINVAL
    assert lib.decode_stream(None, None, 0, None, None, None, None, None, None) == pwdec.PWD_EINVAL
    assert lib.decode_windows_recurrent(None, None, None, 0, None, None, None) == pwdec.PWD_EINVAL
    assert lib.decoder_destroy(None) == pwdec.PWD_OK


def blob_for(name):
    wl = synth.WORKLOADS[name]
    return wl, pwdec.make_blob(wl.d, wl.W, wl.D, wl.L, wl.H, wl.F, wl.dtype, synth.make_weights(wl))


@pytest.mark.parametrize("name", ["d3", "d7"])
def test_blob_size_matches_header_formula(lib, name):
    wl, blob = blob_for(name)
    g, m = pwdec.geometry(wl.d, wl.W, 4), pwdec.dims(wl.D, wl.L, wl.H, wl.mlp_ratio, wl.dtype)
    assert len(blob) == 64 + 4 * lib.decoder_blob_floats(ctypes.byref(g), ctypes.byref(m))
    # with the embedder's residual block: two Conv1d(D, D, 3) layers and their biases more
    rw = dataclasses.replace(wl, resnet=True)
    rblob = pwdec.make_blob(rw.d, rw.W, rw.D, rw.L, rw.H, rw.F, rw.dtype, synth.make_weights(rw))
    assert struct.unpack("<I", rblob[48:52])[0] == pwdec.EMBED_RESNET
    m = pwdec.dims(wl.D, wl.L, wl.H, wl.mlp_ratio, wl.dtype, 0, pwdec.EMBED_RESNET)
    assert len(rblob) == 64 + 4 * lib.decoder_blob_floats(ctypes.byref(g), ctypes.byref(m))
    assert len(rblob) - len(blob) == 4 * (6 * wl.D * wl.D + 2 * wl.D)
    # with dilated convolutions (grid token set): per layer three 3x3 Conv2d(D, D) and biases
    cw = dataclasses.replace(wl, grid=True, dil=(1, 2, 3))
    cblob = pwdec.make_blob(cw.d, cw.W, cw.D, cw.L, cw.H, cw.F, cw.dtype, synth.make_weights(cw), 1)
    assert struct.unpack("<I", cblob[52:56])[0] == 0x030201
    m = pwdec.dims(wl.D, wl.L, wl.H, wl.mlp_ratio, wl.dtype, 1, 0, (1, 2, 3))
    assert len(cblob) == 64 + 4 * lib.decoder_blob_floats(ctypes.byref(g), ctypes.byref(m))
    assert len(cblob) - len(blob) == 4 * wl.L * (27 * wl.D * wl.D + 3 * wl.D)


def corrupt(blob, word, value):
    b = bytearray(blob)
    b[4 * word:4 * word + 4] = struct.pack("<I", value)
    return bytes(b)


@pytest.mark.parametrize("how", ["magic", "version", "distance", "layers", "dtype", "token_set", "embedder",
                                 "dilations", "short", "long"])
def test_bad_blobs_rejected_before_device_use(lib, how):
    wl, blob = blob_for("d3")
    bad = {"magic": lambda b: corrupt(b, 0, 0x12345678),
           "version": lambda b: corrupt(b, 1, 9),
           "distance": lambda b: corrupt(b, 2, 5),
           "layers": lambda b: corrupt(b, 5, 3),
           "dtype": lambda b: corrupt(b, 8, 1),
           "token_set": lambda b: corrupt(b, 11, 1),
           "embedder": lambda b: corrupt(b, 12, 1),
           "dilations": lambda b: corrupt(b, 13, 0x010101),
           "short": lambda b: b[:-4],
           "long": lambda b: b + b"\0\0\0\0"}[how](blob)
    g, m = pwdec.geometry(wl.d, wl.W, 4), pwdec.dims(wl.D, wl.L, wl.H, wl.mlp_ratio, wl.dtype)
    h = ctypes.c_void_p()
    buf = ctypes.create_string_buffer(bad, len(bad))
    rc = lib.decoder_create(ctypes.byref(g), ctypes.byref(m), buf, len(bad), ctypes.byref(h))
    assert rc == pwdec.PWD_EBLOB
    assert not h.value
    assert b"blob" in lib.decoder_last_error()


class FakeTensor:
    """Stands in for a torch tensor in the binding's argument checks (no device needed)."""

    def __init__(self, shape, dtype="int32", cuda=True, index=0, contiguous=True):
        self.shape, self._contig = tuple(shape), contiguous
        self.dtype = f"torch.{dtype}"
        self.is_cuda = cuda
        self.device = type("Dev", (), {"index": index})()

    def is_contiguous(self):
        return self._contig

    def numel(self):
        n = 1
        for s in self.shape:
            n *= s
        return n

    def dim(self):
        return len(self.shape)


def test_binding_rejects_buffers_the_kernels_would_overrun():
    """Every device buffer is checked before its pointer crosses the ABI: a mismatch raises
    ValueError instead of an out-of-bounds access on the device."""
    req = pwdec.require
    req(FakeTensor((4, 15, 2)), "meas", pwdec.WORDS, 0, shape=(4, 15, 2))
    req(FakeTensor((4,), "float32"), "logits", ("float32",), 0, min_numel=4)
    bad = [
        (FakeTensor((4, 15, 2), cuda=False), dict(shape=(4, 15, 2))),           # host memory
        (FakeTensor((4, 15, 2), index=1), dict(shape=(4, 15, 2))),              # another GPU
        (FakeTensor((4, 15, 2), "int64"), dict(shape=(4, 15, 2))),              # wrong dtype
        (FakeTensor((4, 15, 2), contiguous=False), dict(shape=(4, 15, 2))),     # a strided view
        (FakeTensor((4, 14, 2)), dict(shape=(4, 15, 2))),                       # W rows, not W + 1
        (FakeTensor((3,)), dict(min_numel=4)),                                  # too few outputs
    ]
    for t, kw in bad:
        with pytest.raises(ValueError):
            req(t, "x", pwdec.WORDS, 0, **kw)
    with pytest.raises(ValueError):
        req(None, "x", pwdec.WORDS, 0)


def test_binding_checks_every_entry_point():
    """The Decoder methods check their buffers against the handle's geometry before calling
    the library: decode's [n] outputs are too small for the recurrent [n][d] outputs, a meas
    tensor of the wrong geometry or a batch above max_windows is refused."""
    dec = object.__new__(pwdec.Decoder)
    dec.d, dec.W, dec.words, dec.max_windows, dec.device = 7, 14, 2, 8, 0
    dec._lib, dec._h = None, None     # never reached: every call below fails its checks
    meas, types = FakeTensor((4, 15, 2)), FakeTensor((4,), "uint8")
    f4, u4 = FakeTensor((4,), "float32"), FakeTensor((4,), "uint8")
    with pytest.raises(ValueError):
        dec.decode_recurrent(meas, types, f4, u4)                      # needs n * d outputs
    with pytest.raises(ValueError):
        dec.decode(FakeTensor((4, 14, 2)), types, f4, u4)              # meas of another window
    with pytest.raises(ValueError):
        dec.decode(FakeTensor((9, 15, 2)), FakeTensor((9,), "uint8"), FakeTensor((9,), "float32"),
                   FakeTensor((9,), "uint8"))                           # above max_windows
    with pytest.raises(ValueError):
        dec.detection_events(meas, types, FakeTensor((4, 15, 2)))      # events have W rows
    with pytest.raises(ValueError):
        dec.decode_stream(FakeTensor((40, 3)), FakeTensor((1,), "uint8"))   # 3 words per round
    with pytest.raises(ValueError):
        dec.decode_stream(FakeTensor((40, 2)), FakeTensor((1,), "uint8"),
                          window_logits=FakeTensor((5,), "float32"))    # 6 windows
