"""Pins of the emulated-MXFP8 reference (oracle/fp8.py) against what the OCP formats fix:
the E4M3 code table, torch's independent float8_e4m3fn conversion, hand-worked blocks under
the MX scale rule, exact results where quantization is the identity, the format's error bound,
and the reduction of the MXFP8 forward pass to the fp64 oracle when quantization is removed."""
import numpy as np
import pytest

from oracle import decoder as O
from oracle import fp8 as MX
from paper_2601_09921_amd import synth


def test_code_table():
    v = MX.e4m3_values()
    assert np.isnan(v[0x7F]) and np.isnan(v[0xFF]) and np.isfinite(v).sum() == 254
    assert v[0x7E] == 448.0 and v[0x08] == 2.0 ** -6 and v[0x01] == 2.0 ** -9 and v[0x38] == 1.0
    assert v[0x80] == 0.0 and np.signbit(v[0x80])
    pos = np.sort(np.unique(np.abs(v[np.isfinite(v)])))
    assert len(pos) == 127          # 0 and 126 positive values
    # every finite value rounds to itself
    fin = v[np.isfinite(v)]
    assert np.array_equal(MX.e4m3_round(fin), fin)


@pytest.mark.parametrize("x,q", [
    (1.0625, 1.0),          # halfway between 1 and 1.125: to the even mantissa (000)
    (1.1875, 1.25),         # halfway between 1.125 and 1.25: to 010
    (0.3, 0.3125),          # quantum 1/32 in [0.25, 0.5): 9.6 quanta -> 10
    (2.0 ** -10, 0.0),      # halfway between 0 and the smallest subnormal: to 0
    (3 * 2.0 ** -10, 2.0 ** -8),   # halfway between 1 and 2 subnormal quanta: to 2
    (240.0, 240.0), (250.0, 256.0), (272.0, 256.0), (304.0, 320.0),
    (447.9, 448.0), (464.0, 448.0), (1e6, 448.0), (-500.0, -448.0), (-0.3, -0.3125), (0.0, 0.0),
])
def test_hand_rounded_values(x, q):
    assert MX.e4m3_round(np.array([x]))[0] == q


def test_agrees_with_torch_float8():
    torch = pytest.importorskip("torch")
    if not hasattr(torch, "float8_e4m3fn"):
        pytest.skip("no float8_e4m3fn in this torch")
    rng = np.random.default_rng(3)
    v = MX.e4m3_values()
    pos = np.sort(np.unique(np.abs(v[np.isfinite(v)])))
    mids = (pos[1:] + pos[:-1]) / 2
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.uniform(-3, 2.3, 20000),
                        mids, -mids, np.nextafter(mids, 0), np.nextafter(mids, 1e9)])
    x = x[np.abs(x) <= 448.0].astype(np.float32)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(MX.e4m3_round(x.astype(np.float64)), ref)


def test_scale_rule():
    e = MX.mx_scale_exponent(np.array([3.0, 1.9, 0.5, 448.0, 512.0, 0.0, 2.0 ** -130, 2.0 ** 130, 2.0 ** 140, 1.0]))
    assert e.tolist() == [-7, -8, -9, 0, 1, -127, -127, 122, 127, -8]


def test_blocks_partition():
    b = MX.mx_blocks(256)
    assert [int(b[f]) for f in (0, 7, 8, 15, 16, 24, 63, 64, 72, 127, 128, 136, 192, 255)] == \
        [0, 0, 1, 1, 0, 1, 1, 2, 3, 3, 4, 5, 6, 7]
    assert np.array_equal(np.bincount(b), np.full(8, 32))


def test_hand_worked_block():
    """One block of 32 features holding i/8, i = 0..31: amax 3.875, X = 2^(1 - 8) = 2^-7, so the
    elements are 16 i. Up to 256 they are exact; from 256 on E4M3 steps by 32 (mantissa m:
    256 + 32 m), so odd i fall halfway and go to the even m: 272 -> 256, 304 -> 320, 336 -> 320,
    368 -> 384, 400 -> 384, 432 -> 448; 464, 480 (no finite code) and 496 clamp to 448."""
    x = np.zeros(128)
    idx = np.nonzero(MX.mx_blocks(128) == 0)[0]
    x[idx] = np.arange(32) / 8
    P, X = MX.mx_quantize(x, axis=0)
    assert np.all(X[idx] == 2.0 ** -7)
    quantized = {17: 256, 19: 320, 21: 320, 23: 384, 25: 384, 27: 448, 29: 448, 30: 448, 31: 448}
    expect = np.array([quantized.get(i, 16 * i) for i in range(32)]) / 128
    assert np.array_equal((P * X)[idx], expect)
    # the other blocks are all zero: scale 2^-127, elements 0
    rest = np.setdiff1d(np.arange(128), idx)
    assert np.all(P[rest] == 0) and np.all(X[rest] == 2.0 ** -127)


def test_block_clamp():
    """amax 1.9: X = 2^-8, 1.9 / X = 486.4 clamps to 448, i.e. 1.75."""
    x = np.full(128, 0.01)
    x[0] = 1.9
    P, X = MX.mx_quantize(x, axis=0)
    assert P[0] == 448.0 and X[0] == 2.0 ** -8 and P[0] * X[0] == 1.75


def test_blocks_are_independent():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 256))
    y = x.copy()
    y[:, MX.mx_blocks(256) == 6] *= 1000.0
    a, b = MX.mx_dequantize(x, -1), MX.mx_dequantize(y, -1)
    keep = MX.mx_blocks(256) != 6
    assert np.array_equal(a[:, keep], b[:, keep]) and not np.array_equal(a, b)


def test_projection_exact_when_representable():
    """Inputs that are already E4M3 values times a block scale that the rule reproduces (each
    block holds an element in [256, 448] X): quantization is the identity and the MX projection
    is the plain product."""
    rng = np.random.default_rng(2)
    v = MX.e4m3_values()
    fin = v[np.isfinite(v)]
    big = fin[(np.abs(fin) >= 256)]

    def representable(shape, axis):
        P = rng.choice(fin, size=shape)
        Pm = np.moveaxis(P, axis, -1)
        blk = MX.mx_blocks(Pm.shape[-1])
        for k in range(blk.max() + 1):
            first = np.nonzero(blk == k)[0][0]
            Pm[..., first] = rng.choice(big, size=Pm.shape[:-1])
        e = rng.integers(-20, 5, size=Pm.shape[:-1] + (blk.max() + 1,))
        return np.moveaxis(Pm * np.exp2(e[..., blk]), -1, axis)

    X = representable((6, 256), -1)
    W = representable((256, 40), 0)
    b = rng.standard_normal(40)
    assert np.array_equal(MX.mx_dequantize(X, -1), X) and np.array_equal(MX.mx_dequantize(W, 0), W)
    assert np.allclose(MX.project_mx(X, W, b), X @ W + b, rtol=1e-15, atol=0)


def test_error_bound():
    """|P X - v| <= half an E4M3 step: 2^-4 |v| for normal elements, X 2^-10 in the subnormal
    range; clamped elements (|v| / X >= 448) are off by at most |v| - 448 X < 64 X."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal((50, 256)) * np.exp2(rng.integers(-12, 12, size=(50, 1)))
    P, X = MX.mx_quantize(x, -1)
    err, r = np.abs(P * X - x), np.abs(x) / X
    normal = (r >= 2.0 ** -6) & (r < 448)
    assert np.all(err[normal] <= 2.0 ** -4 * np.abs(x[normal]) * (1 + 1e-15))
    assert np.all(err[r < 2.0 ** -6] <= X[r < 2.0 ** -6] * 2.0 ** -10)
    assert np.all(err[r >= 448] < 64 * X[r >= 448])
    assert np.all(r < 512)


def test_forward_reduces_to_the_oracle(monkeypatch):
    """With quantization removed, the MXFP8 forward pass is the fp64 oracle's."""
    wl = synth.Workload("t", 3, 6, 5, 0.05, 0.0, 128, 2, 4, 4, synth.DTYPE_MXFP8)
    w = synth.make_weights(wl, seed=9)
    meas, types = synth.make_windows(wl, seed=10, realistic_boundaries=False)
    o, _ = O.forward_windows(meas, types, w, wl.d, wl.H)
    monkeypatch.setattr(MX, "mx_dequantize", lambda x, axis: np.asarray(x, dtype=np.float64))
    e, _ = MX.forward_windows_mx(meas, types, w, wl.d, wl.H)
    assert np.allclose(e, o, rtol=0, atol=1e-12)


def test_forward_quantization_is_visible_but_small():
    wl = synth.Workload("t", 3, 6, 5, 0.05, 0.0, 128, 2, 4, 4, synth.DTYPE_MXFP8)
    w = synth.make_weights(wl, seed=9)
    meas, types = synth.make_windows(wl, seed=10, realistic_boundaries=False)
    o, _ = O.forward_windows(meas, types, w, wl.d, wl.H)
    e, _ = MX.forward_windows_mx(meas, types, w, wl.d, wl.H)
    dev = np.abs(e - o)
    assert 1e-4 < dev.max() < 0.2
