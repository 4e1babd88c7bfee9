"""Seeded synthetic inputs for the parallel-window decoder.

This module produces the *inputs* that both the HIP path and the CPU oracle consume:
the workload table, random-init network weights and bit-packed stabilizer-measurement
windows. It holds none of the decoder's arithmetic (no detection events, embedding,
attention, readout); it only draws random numbers and lays them out.

Why synthetic: the paper's networks are trained on Stim circuit-level simulations and on
hardware shots (Sec. 3.3, App. B) and no trained weights are published (App. B, model-size
table), so every input here is random: i.i.d. Bernoulli(p) detection events folded into a
measurement stream, and random-init weights of the stated architecture.
"""
from __future__ import annotations

import dataclasses
import numpy as np

# Window types (Sec. 3.1 and App. A.1.1: initial, bulk and final decoding windows).
WIN_INITIAL, WIN_BULK, WIN_FINAL = 0, 1, 2

DTYPE_F32, DTYPE_BF16, DTYPE_MXFP8 = 0, 1, 2


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shapes of one decoding workload.

    d: code distance; the token set is the d*d-1 stabilizers of the rotated surface code.
    W: rounds per window; the core region is d rounds (Sec. 3.1, b = c = d in the paper;
       here the window is 2d rounds and the buffers split the remaining W-d rounds).
    B: number of windows per batch.
    p: Bernoulli probability of a detection event per (round, stabilizer).
    pair_p: probability per round of one extra correlated flip of a diagonal stabilizer pair.
    D, L, H, mlp_ratio: model width, layers, heads and MLP expansion.
    dtype: DTYPE_F32, DTYPE_BF16 (bf16 weights/activations, fp32 accumulation) or DTYPE_MXFP8
       (as bf16, with the Q/K/V projections and the first feed-forward matrix on MXFP8
       operands; the weights are drawn exactly as for bf16).
    grid: run the network over all (d+1)^2 cells of the stabilizer array instead of the
       d*d-1 stabilizers (inputs stay one bit per stabilizer).
    resnet: add the embedder's residual block of two Conv1d(D, D, kernel 3) over the
       flattened (d+1)^2 array (App. A model table and syndrome-convolution section).
    dil: dilations of the three 3x3 Conv2d(D, D) units each layer runs on the grid between
       attention and feed-forward (model table); empty: none. Needs grid=True.
    """

    name: str
    d: int
    W: int
    B: int
    p: float
    pair_p: float
    D: int
    L: int
    H: int
    mlp_ratio: int
    dtype: int
    grid: bool = False
    resnet: bool = False
    dil: tuple = ()

    @property
    def N(self) -> int:
        return self.d * self.d - 1

    @property
    def F(self) -> int:
        return self.mlp_ratio * self.D

    @property
    def words(self) -> int:
        return (self.N + 31) // 32

    @property
    def b_left(self) -> int:
        return (self.W - self.d) // 2


# The five workloads the throughput study is run on (d = 3 ... 25).
WORKLOADS = {
    "d3": Workload("d3", 3, 6, 64, 0.02, 0.0, 64, 2, 4, 4, DTYPE_F32),
    "d7": Workload("d7", 7, 14, 1024, 0.01, 0.0, 128, 3, 8, 4, DTYPE_BF16),
    "d11": Workload("d11", 11, 22, 4096, 0.005, 0.01, 256, 4, 8, 4, DTYPE_BF16),
    "d17": Workload("d17", 17, 34, 4096, 0.005, 0.0, 256, 4, 8, 4, DTYPE_BF16),
    "d25": Workload("d25", 25, 50, 8192, 0.003, 0.0, 256, 4, 8, 4, DTYPE_BF16),
}

WEIGHT_SEED = 0


def input_seed(d: int) -> int:
    return 1000 + d


def with_batch(wl: Workload, B: int, **kw) -> Workload:
    return dataclasses.replace(wl, B=B, **kw)


def mxfp8(wl: Workload) -> Workload:
    """The same network and inputs with the MXFP8 projections."""
    return dataclasses.replace(wl, name=wl.name + "_mxfp8", dtype=DTYPE_MXFP8)


# ----------------------------------------------------------------------------- weights

def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 value (ties to even), returned as float64."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def make_weights(wl: Workload, seed: int = WEIGHT_SEED, gain: float = 1.0) -> dict:
    """Random-init weights for the decoder of workload `wl`.

    Matrices are stored [in][out] and drawn from N(0, gain^2/fan_in); biases N(0, 0.01^2);
    LayerNorm gains 1+N(0, 0.05^2) and shifts N(0, 0.05^2); the embedding row and bias
    N(0, 1); the readout projection N(0, 1/(d*D)); the per-window-type readout bias
    N(0, 0.25^2). For bf16 workloads every value is rounded to bf16 once, here, so both
    the GPU path and the oracle consume identical numbers.

    The draw order is fixed: embedding, then each layer (q, k, v, o, ln1, mlp1, mlp2, ln2),
    then readout, then (resnet) the embedder's two Conv1d layers, weights [k][in][out]
    N(0, 1/(3D)), then (dil) per layer the three dilated Conv2d layers, weights
    [j][a][e][in][out] N(0, 1/(9D)); each tensor is drawn in one call in row-major order.
    """
    rng = np.random.default_rng(seed)
    D, F, d = wl.D, wl.F, wl.d

    def mat(fan_in, shape):
        return rng.standard_normal(shape) * (gain / np.sqrt(fan_in))

    def bias(n):
        return rng.standard_normal(n) * 0.01

    w = {"w_e": rng.standard_normal(D), "b_e": rng.standard_normal(D), "layers": []}
    for _ in range(wl.L):
        lw = {}
        lw["Wq"], lw["bq"] = mat(D, (D, D)), bias(D)
        lw["Wk"], lw["bk"] = mat(D, (D, D)), bias(D)
        lw["Wv"], lw["bv"] = mat(D, (D, D)), bias(D)
        lw["Wo"], lw["bo"] = mat(D, (D, D)), bias(D)
        lw["g1"] = 1.0 + 0.05 * rng.standard_normal(D)
        lw["be1"] = 0.05 * rng.standard_normal(D)
        lw["W1"], lw["b1"] = mat(D, (D, F)), bias(F)
        lw["W2"], lw["b2"] = mat(F, (F, D)), bias(D)
        lw["g2"] = 1.0 + 0.05 * rng.standard_normal(D)
        lw["be2"] = 0.05 * rng.standard_normal(D)
        w["layers"].append(lw)
    w["Wc"] = mat(4 * D, (2, 2, D, D))
    w["bc"] = bias(D)
    w["w_o"] = rng.standard_normal((d, D)) / np.sqrt(d * D)
    w["b_o"] = np.array([0.01 * rng.standard_normal()])
    w["beta"] = 0.25 * rng.standard_normal(3)
    if wl.resnet:   # drawn last, so the other tensors match the network without it
        w["res"] = {"W1": mat(3 * D, (3, D, D)), "b1": bias(D), "W2": mat(3 * D, (3, D, D)), "b2": bias(D)}
    if wl.dil:      # after that, for the same reason
        assert len(wl.dil) == 3
        w["dilations"] = list(wl.dil)
        for lw in w["layers"]:
            lw["Wd"], lw["bd"] = mat(9 * D, (3, 3, 3, D, D)), bias((3, D))
    w["kappa"] = 0.707
    w["eps"] = 1e-5
    if wl.dtype in (DTYPE_BF16, DTYPE_MXFP8):
        w = map_tensors(w, round_bf16)
    else:
        w = map_tensors(w, lambda a: np.asarray(a, np.float32).astype(np.float64))
    return w


def map_tensors(w: dict, fn) -> dict:
    out = {}
    for k, v in w.items():
        if k == "layers":
            out[k] = [{kk: fn(vv) for kk, vv in lw.items()} for lw in v]
        elif k == "res":
            out[k] = {kk: fn(vv) for kk, vv in v.items()}
        elif isinstance(v, np.ndarray):
            out[k] = fn(v)
        else:
            out[k] = v
    return out


# ----------------------------------------------------------------------------- syndromes

def _stabilizer_cells(d: int):
    """Cells (r, c) of the (d+1)x(d+1) grid that hold a stabilizer, row-major.

    Used here only to place correlated pair flips on the right token indices.
    """
    cells = []
    for r in range(d + 1):
        for c in range(d + 1):
            bulk = 1 <= r <= d - 1 and 1 <= c <= d - 1
            tb = r in (0, d) and 1 <= c <= d - 1 and (r + c) % 2 == 0
            lr = c in (0, d) and 1 <= r <= d - 1 and (r + c) % 2 == 1
            if bulk or tb or lr:
                cells.append((r, c))
    return cells


def diagonal_pairs(d: int):
    """Token-index pairs of same-type stabilizers on diagonal cells (they share one qubit)."""
    cells = _stabilizer_cells(d)
    index = {rc: i for i, rc in enumerate(cells)}
    pairs = []
    for (r, c), i in index.items():
        for dc in (-1, 1):
            j = index.get((r + 1, c + dc))
            if j is not None:
                pairs.append((i, j))
    return np.array(pairs, dtype=np.int64)


def pack_bits(bits: np.ndarray) -> np.ndarray:
    """Pack the last axis of a 0/1 array into uint32 words, LSB first (bit s -> word s//32, bit s%32)."""
    bits = np.asarray(bits, dtype=np.uint8)
    n = bits.shape[-1]
    words = (n + 31) // 32
    pad = np.zeros(bits.shape[:-1] + (words * 32,), dtype=np.uint64)
    pad[..., :n] = bits
    pad = pad.reshape(bits.shape[:-1] + (words, 32))
    shifts = np.arange(32, dtype=np.uint64)
    return (pad << shifts).sum(axis=-1).astype(np.uint32)


def window_types(B: int) -> np.ndarray:
    """Equal mix of the three window types: type[w] = w mod 3."""
    return (np.arange(B) % 3).astype(np.uint8)


def make_windows(wl: Workload, seed: int | None = None, B: int | None = None,
                 realistic_boundaries: bool = True, zero: bool = False):
    """Draw B windows of stabilizer measurements.

    Returns (meas_bits uint8 [B][W+1][N], types uint8 [B]). Row 0 is the round that
    precedes the window's first round. Flips ~ Bernoulli(p) per (round, stabilizer), plus
    for pair_p > 0 one diagonal pair flipped per round with probability pair_p; the
    measurements are M[0] ~ Bernoulli(0.5) and M[t+1] = M[t] xor flips[t].

    Window w draws from its own generator, seeded with (seed, w), so the first k windows
    of a large batch equal a batch of k windows.

    realistic_boundaries: initial windows get all-zero rows 0..b_left (no rounds exist
    before the experiment starts) and final windows hold the last core round's values for
    the rows after the core (no rounds exist after the experiment ends). With False every
    row is random, which exercises the decoder's own boundary masks.
    zero: all-zero measurements (the zero-syndrome invariant input).
    """
    B = wl.B if B is None else B
    seed = input_seed(wl.d) if seed is None else seed
    N, W = wl.N, wl.W
    types = window_types(B)
    meas = np.zeros((B, W + 1, N), np.uint8)
    if zero:
        return meas, types
    pairs = diagonal_pairs(wl.d) if wl.pair_p > 0 else None
    bl = wl.b_left
    rows = np.empty((W + 1, N), np.uint8)
    for w in range(B):
        rng = np.random.default_rng([seed, w])
        rows[0] = rng.random(N) < 0.5
        rows[1:] = rng.random((W, N)) < wl.p
        if pairs is not None:
            hit = np.nonzero(rng.random(W) < wl.pair_p)[0]
            choice = rng.integers(0, len(pairs), size=W)
            for t in hit:
                i, j = pairs[choice[t]]
                rows[1 + t, i] ^= 1
                rows[1 + t, j] ^= 1
        if realistic_boundaries and types[w] == WIN_INITIAL:
            rows[:bl + 1] = 0                 # rows 0..b_left stay zero
        if realistic_boundaries and types[w] == WIN_FINAL:
            rows[bl + 1 + wl.d:] = 0          # rows after the core hold their value
        np.bitwise_xor.accumulate(rows, axis=0, out=meas[w])
    return meas, types


def make_stream(N: int, T: int, p: float, seed: int) -> np.ndarray:
    """A measurement stream R[T][N] of a memory experiment that starts from all zeros."""
    rng = np.random.default_rng(seed)
    flips = (rng.random((T, N)) < p).astype(np.uint8)
    return np.bitwise_xor.accumulate(flips, axis=0).astype(np.uint8)
