"""Emulated MXFP8 operands for the decoder's low-precision option, on top of the fp64 oracle.

TEST INFRASTRUCTURE ONLY, like oracle/decoder.py: the tests, the smoke check and the benchmark's
CPU baseline may import it; the product path never does.

The paper points to lower-precision arithmetic (quantization) as a route toward its real-time
budget (Sec. 1; Sec. 5, Summary and Outlook) without fixing a format. The MXFP8 option of the
decoder runs four of the matrix products of every Syndrome Transformer layer (App. A.2) on
8-bit operands: the Q, K and V projections and the first feed-forward matrix (d_model -> F).
Everything else is as in the bf16 path. This module defines what that option computes, in
plain numpy, following the OCP Microscaling (MX) format, v1.0:

  * elements are FP8 E4M3: 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits, subnormals
    down to 2^-9, no infinities, largest finite magnitude 448;
  * a block of 32 elements along the reduction axis shares one E8M0 scale X = 2^e with
    e = floor(log2(amax)) - 8 (8 = the exponent of E4M3's largest power of two), clamped to
    E8M0's range [-127, 127]; amax = 0 gives e = -127;
  * each element is stored as E4M3(v / X): rounded to the nearest E4M3 value, ties to even,
    and magnitudes above 448 clamped to 448 (amax / X lies in [256, 512), so clamping only
    touches elements within 12.5 % of amax);
  * a dot product is sum over blocks of X_a X_b sum_i P_a,i P_b,i, accumulated here exactly
    (float64; every product of two E4M3 values and two powers of two is exact).

Blocks. The reduction axis (d_model features) is cut into slices of 128 and each slice into
four blocks of 32: feature f belongs to block 4 (f // 128) + 2 ((f // 64) % 2) + (f // 8) % 2,
i.e. within a 64-feature half of a slice, the runs of 8 features alternate between two blocks.
The partition is a free choice (any fixed partition into blocks of 32 is a valid MX dot
product); this one lets each token's activations be quantized where the matrix core reads them.
Activations take one scale per token and block; weight matrices W [in][out] one per output
feature and block.
"""
from __future__ import annotations

import math

import numpy as np

from . import decoder as O

E4M3_MAX = 448.0
E4M3_EMAX = 8                 # exponent of the largest power of two in E4M3 (256)
E4M3_MIN_NORMAL_EXP = -6      # smallest normal: 2^-6
E4M3_MANTISSA_BITS = 3
MX_BLOCK = 32
E8M0_MIN, E8M0_MAX = -127, 127


def e4m3_round(x) -> np.ndarray:
    """Nearest E4M3 value of each element (ties to even mantissa), magnitudes above 448
    clamped to 448."""
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    e = np.maximum(e, E4M3_MIN_NORMAL_EXP)                 # subnormals share the smallest binade's spacing
    quantum = np.exp2(e - E4M3_MANTISSA_BITS)
    q = np.round(a / quantum) * quantum                    # np.round: halves to even
    q = np.minimum(q, E4M3_MAX)
    return np.where(a > 0, np.copysign(q, x), 0.0)


def e4m3_values() -> np.ndarray:
    """All 256 E4M3 codes decoded from their bit fields (NaN for the two NaN codes)."""
    out = np.empty(256)
    for code in range(256):
        sign = -1.0 if code & 0x80 else 1.0
        exp = (code >> 3) & 0xF
        man = code & 0x7
        if exp == 0xF and man == 0x7:
            out[code] = np.nan
        elif exp == 0:
            out[code] = sign * man * 2.0 ** -9
        else:
            out[code] = sign * (1.0 + man / 8.0) * 2.0 ** (exp - 7)
    return out


def mx_scale_exponent(amax) -> np.ndarray:
    """The shared exponent e of a block from its largest magnitude (OCP MX scale rule)."""
    amax = np.asarray(amax, dtype=np.float64)
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(amax > 0, amax, 1.0))) - E4M3_EMAX
    e = np.where(amax > 0, e, E8M0_MIN)
    return np.clip(e, E8M0_MIN, E8M0_MAX)


def mx_blocks(n: int) -> np.ndarray:
    """Block index of each of n features (n a multiple of 128)."""
    assert n % 128 == 0, n
    f = np.arange(n)
    return 4 * (f // 128) + 2 * ((f // 64) % 2) + (f // 8) % 2


def mx_quantize(x, axis: int):
    """(P, X): E4M3 elements and the per-element block scale, blocks of 32 along `axis`;
    P * X is the value the matrix product uses."""
    x = np.moveaxis(np.asarray(x, dtype=np.float64), axis, -1)
    blk = mx_blocks(x.shape[-1])
    P = np.empty_like(x)
    X = np.empty_like(x)
    for k in range(blk.max() + 1):
        idx = np.nonzero(blk == k)[0]
        assert len(idx) == MX_BLOCK
        v = x[..., idx]
        s = np.exp2(mx_scale_exponent(np.max(np.abs(v), axis=-1, keepdims=True)))
        P[..., idx] = e4m3_round(v / s)
        X[..., idx] = np.broadcast_to(s, v.shape)
    return np.moveaxis(P, -1, axis), np.moveaxis(X, -1, axis)


def mx_dequantize(x, axis: int) -> np.ndarray:
    P, X = mx_quantize(x, axis)
    return P * X


def project_mx(X, W, b):
    """X [..][in] W [in][out] + b with both operands in MXFP8 (X per token, W per output)."""
    return mx_dequantize(X, -1) @ mx_dequantize(W, 0) + b


def attention_mx(X, lw, H):
    """oracle.decoder.attention with the Q, K and V projections in MXFP8."""
    B, N, D = X.shape
    dh = D // H
    Q = project_mx(X, lw["Wq"], lw["bq"])
    K = project_mx(X, lw["Wk"], lw["bk"])
    V = project_mx(X, lw["Wv"], lw["bv"])
    out = np.zeros_like(Q)
    for h in range(H):
        sl = slice(h * dh, (h + 1) * dh)
        scores = Q[:, :, sl] @ np.swapaxes(K[:, :, sl], 1, 2) / math.sqrt(dh)
        out[:, :, sl] = O.softmax(scores) @ V[:, :, sl]
    return out @ lw["Wo"] + lw["bo"]


def feed_forward_mx(X, lw):
    """oracle.decoder.feed_forward with its first matrix in MXFP8."""
    return np.maximum(project_mx(X, lw["W1"], lw["b1"]), 0.0) @ lw["W2"] + lw["b2"]


def forward_windows_mx(meas, types, w, d, H, grid=False):
    """oracle.decoder.forward_windows (Algorithm 1, inference branch; networks without the
    dilated convolutions) with the MXFP8 projections; returns logits and bits."""
    meas = np.asarray(meas, dtype=np.uint8)
    B = meas.shape[0]
    D = w["w_e"].shape[0]
    assert "dilations" not in w
    ev = O.detection_events(meas, types, d)
    pos = np.array([r * (d + 1) + c for r, c in O.token_cells(d, grid)], dtype=np.int64)
    pe = O.positional_encoding((d + 1) ** 2, D)[pos]
    state = np.zeros((B, len(pos), D), dtype=np.float64)
    for n in range(meas.shape[1] - 1):
        X = w["kappa"] * (O.embed_round(ev[:, n, :], w, d, grid, pe) + state)
        for lw in w["layers"]:
            X = O.layer_norm(X + attention_mx(X, lw, H), lw["g1"], lw["be1"], w["eps"])
            X = O.layer_norm(X + feed_forward_mx(X, lw), lw["g2"], lw["be2"], w["eps"])
        state = X
    logits = O.readout(state, types, w, d, grid)
    return logits, (logits > 0).astype(np.uint8)
