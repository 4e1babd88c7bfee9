"""CPU float64 oracle of the parallel-window neural decoder.

TEST INFRASTRUCTURE ONLY. This module is the plain, slow, obviously-correct definition
that the HIP path is checked against. Only the test-suite, the smoke check and the CPU
baseline leg of the benchmark may import it; the product path never does.

It follows the paper's statement of the method step by step:
  * the window decomposition of a syndrome stream (Sec. 3.1, eq. global_xor; App. A.1.1),
  * detection events from consecutive measurement rounds (Sec. 2.2, Sec. 3.2),
  * the stabilizer embedder and sinusoidal positional encoding (App. A.1, model table),
    optionally with its residual block of two Conv1d layers over the flattened stabilizer
    array ahead of the positional encoding (model table; syndrome-convolution section),
  * the recurrent fold D_n = RNNCore((S_n + D_{n-1}) * 0.707) with D_0 = 0
    (Algorithm 1 inference branch; App. A.2 fold equation),
  * Syndrome Transformer layers of multi-head self-attention and feed-forward (App. A.2),
    optionally with the dilated convolutions over the 2-D stabilizer array (model table;
    App. A.2 text: the attention output is scattered onto the grid for them),
  * the readout: 2x2 valid convolution, logical pooling, linear projection (App. A.3),
  * the XOR combination of per-window bits (eq. global_xor).

Readings taken where the paper is silent or ambiguous (each listed in the design notes):
the token set is the d*d-1 real stabilizers by default, with the paper's (d+1)^2 grid as an
option (grid=True); LayerNorm (post-norm, eps from the weights)
replaces BatchNorm; ReLU feed-forward; attention has Q/K/V/O biases and scale 1/sqrt(dh);
the readout convolution is followed by a bias and ReLU, pooling averages over columns;
the embedder's Conv1d layers have kernel 3, zero padding 1, biases and a ReLU between them,
and the block adds its input back (E + Conv2(ReLU(Conv1(E))));
the dilated convolutions sit between the attention block (after LayerNorm 1) and the
feed-forward, need the (d+1)^2 token set (every cell a token), and are three residual units
C = C + ReLU(Conv2d_j(C)), 3x3 kernels with dilations from the weights and zero padding equal
to the dilation (the grid keeps its size);
the window type adds a learned bias to the logit on top of the boundary padding masks.

Everything is float64 numpy. Matrices are stored [in][out] so a projection is X @ W.
"""
from __future__ import annotations

import math
import numpy as np

INITIAL, BULK, FINAL = 0, 1, 2


# ----------------------------------------------------------------------------- geometry

def stabilizer_cells(d: int):
    """Stabilizer cells of the distance-d rotated surface code on the (d+1)x(d+1) grid.

    App. A.1.2 maps every stabilizer to one cell of a (d+1)x(d+1) array. Data qubits sit
    at (i, j), 0 <= i, j < d; the stabilizer at cell (r, c) acts on the data qubits
    (r-1..r, c-1..c) that exist. Interior cells (1 <= r, c <= d-1) are weight-4; a
    boundary cell on the top/bottom row is kept when r+c is even, on the left/right column
    when r+c is odd (weight 2). The stabilizer type is X when r+c is even, else Z.
    Returns a list of (r, c) in row-major order: that is the token order.
    """
    cells = []
    for r in range(d + 1):
        for c in range(d + 1):
            interior = 1 <= r <= d - 1 and 1 <= c <= d - 1
            top_bottom = (r == 0 or r == d) and 1 <= c <= d - 1 and (r + c) % 2 == 0
            left_right = (c == 0 or c == d) and 1 <= r <= d - 1 and (r + c) % 2 == 1
            if interior or top_bottom or left_right:
                cells.append((r, c))
    return cells


def stabilizer_support(d: int, cell):
    r, c = cell
    return [(i, j) for i in (r - 1, r) for j in (c - 1, c) if 0 <= i < d and 0 <= j < d]


def stabilizer_kind(cell) -> str:
    return "X" if (cell[0] + cell[1]) % 2 == 0 else "Z"


def grid_positions(d: int) -> np.ndarray:
    """Flattened grid index r*(d+1)+c of each token (the PE position, App. A.1.2/A.1.4)."""
    return np.array([r * (d + 1) + c for r, c in stabilizer_cells(d)], dtype=np.int64)


def token_cells(d: int, grid: bool = False):
    """Cells that carry a token, row-major. By default the d*d-1 stabilizer cells; with
    grid=True every cell of the (d+1)x(d+1) array, the token set of App. A.1.2 and of
    Algorithm 1's (d+1)^2 x d_model state: a cell without a stabilizer then carries state
    but never receives a detection event."""
    if not grid:
        return stabilizer_cells(d)
    return [(r, c) for r in range(d + 1) for c in range(d + 1)]


def token_events(ev: np.ndarray, d: int, grid: bool = False) -> np.ndarray:
    """Detection events per token: the stabilizer events [..][N] themselves, or (grid) placed
    at their cells of the (d+1)^2 grid with zeros at the other cells."""
    if not grid:
        return ev
    out = np.zeros(ev.shape[:-1] + ((d + 1) ** 2,), dtype=ev.dtype)
    for s, (r, c) in enumerate(stabilizer_cells(d)):
        out[..., r * (d + 1) + c] = ev[..., s]
    return out


# ----------------------------------------------------------------------------- bits

def unpack_bits(words: np.ndarray, n: int) -> np.ndarray:
    """Unpack uint32 words (LSB first) of the last axis into n 0/1 values."""
    words = np.asarray(words, dtype=np.uint32)
    out = np.zeros(words.shape[:-1] + (n,), dtype=np.uint8)
    for s in range(n):
        out[..., s] = (words[..., s // 32] >> np.uint32(s % 32)) & np.uint32(1)
    return out


def pack_bits(bits: np.ndarray) -> np.ndarray:
    """Pack the last axis of 0/1 values into uint32 words, LSB first; spare bits are 0."""
    bits = np.asarray(bits, dtype=np.uint8)
    n = bits.shape[-1]
    nw = (n + 31) // 32
    out = np.zeros(bits.shape[:-1] + (nw,), dtype=np.uint32)
    for s in range(n):
        out[..., s // 32] |= bits[..., s].astype(np.uint32) << np.uint32(s % 32)
    return out


# ----------------------------------------------------------------------------- windows

def window_split(d: int, W: int):
    """Buffer sizes of a window of W rounds with a core of d rounds (Sec. 3.1).

    The paper uses b + c + b rounds with c = d; for a window of W rounds the left buffer is
    floor((W-d)/2) rounds and the right buffer the rest.
    """
    b_left = (W - d) // 2
    return b_left, W - d - b_left


def detection_events(meas: np.ndarray, types: np.ndarray, d: int) -> np.ndarray:
    """Detection events of each window from its measurement rounds.

    meas: 0/1 array [B][W+1][N]; row 0 is the round before the window's first round.
    A detector is the parity of consecutive measurements of one stabilizer (Sec. 2.2):
    E[t] = M[t+1] xor M[t], t = 0..W-1. Boundary padding (App. A.1.1): an initial window
    has no rounds before its core, so its left buffer is zero-filled and its first core
    round is compared with the all-zero initial state; a final window has no rounds after
    its core, so its right buffer is zero-filled.
    """
    meas = np.asarray(meas, dtype=np.uint8)
    B, W1, N = meas.shape
    W = W1 - 1
    b_left, _ = window_split(d, W)
    ev = np.bitwise_xor(meas[:, 1:, :], meas[:, :-1, :])
    for w in range(B):
        if types[w] == INITIAL:
            ev[w, :b_left, :] = 0
            ev[w, b_left, :] = meas[w, b_left + 1, :]
        elif types[w] == FINAL:
            ev[w, b_left + d:, :] = 0
        elif types[w] != BULK:
            raise ValueError(f"window {w}: invalid type {types[w]}")
    return ev


def split_stream(R: np.ndarray, d: int, W: int):
    """Cut a measurement stream R[T][N] into overlapping windows (Sec. 3.1, App. A.1.1).

    The stream is padded to T' = m*d rounds (m = ceil(T/d), Sec. 4.1 pads the syndrome
    data) by holding its last round, so padded rounds carry no detection events. Window i
    has core rounds [i*d, i*d+d) and rows M_i[k] = R[i*d - b_left - 1 + k], k = 0..W;
    rows before the stream read as zeros and rows after it repeat the last round.
    Window 0 is initial, window m-1 final, the rest bulk. Requires m >= 2.
    """
    R = np.asarray(R, dtype=np.uint8)
    T, N = R.shape
    m = -(-T // d)
    if m < 2:
        raise ValueError("a stream needs at least two windows")
    Tp = m * d
    Rp = np.concatenate([R, np.repeat(R[-1:], Tp - T, axis=0)], axis=0)
    b_left, _ = window_split(d, W)
    meas = np.zeros((m, W + 1, N), dtype=np.uint8)
    for i in range(m):
        for k in range(W + 1):
            idx = i * d - b_left - 1 + k
            if idx < 0:
                continue
            meas[i, k] = Rp[min(idx, Tp - 1)]
    types = np.full(m, BULK, dtype=np.uint8)
    types[0], types[-1] = INITIAL, FINAL
    return meas, types


def combine_bits(bits: np.ndarray) -> int:
    """Global logical correction: XOR of the per-window bits (eq. global_xor)."""
    return int(np.bitwise_xor.reduce(np.asarray(bits, dtype=np.uint8)))


def soft_xor(probs: np.ndarray) -> float:
    """Soft-XOR of per-window probabilities (eq. soft_xor): (1 - prod(1 - 2 y_k)) / 2."""
    probs = np.asarray(probs, dtype=np.float64)
    return 0.5 * (1.0 - np.prod(1.0 - 2.0 * probs))


# ----------------------------------------------------------------------------- network

def positional_encoding(num_pos: int, D: int) -> np.ndarray:
    """Sinusoidal encoding of App. A.1.4: PE[t, 2i] = sin(t / 10000^(2i/D)),
    PE[t, 2i+1] = cos(t / 10000^(2i/D)), for i = 0 .. D/2-1 and t = 0 .. num_pos-1."""
    pe = np.zeros((num_pos, D), dtype=np.float64)
    for t in range(num_pos):
        for i in range(D // 2):
            angle = t / (10000.0 ** (2 * i / D))
            pe[t, 2 * i] = math.sin(angle)
            pe[t, 2 * i + 1] = math.cos(angle)
    return pe


def embed(events_t: np.ndarray, w: dict, pe_tokens: np.ndarray) -> np.ndarray:
    """StabilizerEmbedder of one round: Linear(1 -> D) of each stabilizer bit plus PE.

    events_t: [B][N] 0/1; returns S [B][N][D] = E * w_e + b_e + PE[pos(s)].
    """
    e = events_t.astype(np.float64)[:, :, None]
    return e * w["w_e"][None, None, :] + w["b_e"][None, None, :] + pe_tokens[None, :, :]


def conv1d_same(x: np.ndarray, Wk: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Conv1d(D, D) with kernel 3 and zero padding 1 along the sequence axis:
    y[p] = b + sum_{k=0..2} x[p+k-1] @ Wk[k], where x is zero outside the sequence.
    x: [B][L][D]; Wk: [3][D][D] ([k][in][out])."""
    L = x.shape[1]
    y = np.broadcast_to(b, x.shape).astype(np.float64).copy()
    for k in range(3):
        off = k - 1
        # output positions p whose source p + off lies in the sequence
        p0, p1 = max(0, -off), min(L, L - off)
        y[:, p0:p1, :] += x[:, p0 + off:p1 + off, :] @ Wk[k]
    return y


def embed_round(events_t: np.ndarray, w: dict, d: int, grid: bool, pe_tokens: np.ndarray) -> np.ndarray:
    """StabilizerEmbedder of one round with its residual Conv1d block (App. A model table:
    Linear(1 -> D), then 2 x Conv1d(D, D); syndrome-convolution section: the ResNet runs on
    the flattened (d+1)^2 array before PE is added).

    events_t: [B][N] 0/1 stabilizer events. Every cell of the array gets E_lin = e * w_e +
    b_e (e = 0 at a cell without a stabilizer); E_conv = E_lin + Conv2(ReLU(Conv1(E_lin)));
    the tokens take E_conv at their cells plus PE. Without w["res"] this is embed().
    """
    if "res" not in w:
        return embed(token_events(events_t, d, grid), w, pe_tokens)
    e = token_events(events_t, d, True).astype(np.float64)[:, :, None]   # [B][(d+1)^2][1]
    E = e * w["w_e"][None, None, :] + w["b_e"][None, None, :]
    r = w["res"]
    R = conv1d_same(np.maximum(conv1d_same(E, r["W1"], r["b1"]), 0.0), r["W2"], r["b2"])
    cells = np.array([rr * (d + 1) + cc for rr, cc in token_cells(d, grid)], dtype=np.int64)
    return (E + R)[:, cells, :] + pe_tokens[None, :, :]


def layer_norm(y: np.ndarray, gamma: np.ndarray, beta: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm over the last axis with the biased variance."""
    mu = y.mean(axis=-1, keepdims=True)
    var = ((y - mu) ** 2).mean(axis=-1, keepdims=True)
    return gamma * (y - mu) / np.sqrt(var + eps) + beta


def softmax(x: np.ndarray) -> np.ndarray:
    """Row softmax with the row maximum subtracted first."""
    z = x - x.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=-1, keepdims=True)


def attention(X: np.ndarray, lw: dict, H: int) -> np.ndarray:
    """Multi-head self-attention over the stabilizer tokens of each window.

    X: [B][N][D]. Per head h: softmax(Q_h K_h^T / sqrt(dh)) V_h, heads concatenated, then
    the output projection. No mask: every stabilizer attends to every stabilizer.
    """
    B, N, D = X.shape
    dh = D // H
    Q = X @ lw["Wq"] + lw["bq"]
    K = X @ lw["Wk"] + lw["bk"]
    V = X @ lw["Wv"] + lw["bv"]
    out = np.zeros_like(Q)
    for h in range(H):
        sl = slice(h * dh, (h + 1) * dh)
        scores = Q[:, :, sl] @ np.swapaxes(K[:, :, sl], 1, 2) / math.sqrt(dh)
        out[:, :, sl] = softmax(scores) @ V[:, :, sl]
    return out @ lw["Wo"] + lw["bo"]


def feed_forward(X: np.ndarray, lw: dict) -> np.ndarray:
    """Feed-forward block D -> F -> D with ReLU."""
    return np.maximum(X @ lw["W1"] + lw["b1"], 0.0) @ lw["W2"] + lw["b2"]


def conv2d_dilated(G: np.ndarray, Wk: np.ndarray, b: np.ndarray, dil: int) -> np.ndarray:
    """Conv2d(D, D) with a 3x3 kernel, dilation dil and zero padding dil on a square grid:
    y[r][c] = b + sum_{a,e in 0..2} x[r + dil (a-1)][c + dil (e-1)] @ Wk[a][e], where x is
    zero outside the grid. G: [B][S][S][D]; Wk: [3][3][D][D] ([a][e][in][out])."""
    S = G.shape[1]
    y = np.broadcast_to(b, G.shape).astype(np.float64).copy()
    for a in range(3):
        for e in range(3):
            dr, dc = dil * (a - 1), dil * (e - 1)
            # output cells (r, c) whose source (r + dr, c + dc) lies on the grid
            r0, r1 = max(0, -dr), min(S, S - dr)
            c0, c1 = max(0, -dc), min(S, S - dc)
            if r0 < r1 and c0 < c1:
                y[:, r0:r1, c0:c1, :] += G[:, r0 + dr:r1 + dr, c0 + dc:c1 + dc, :] @ Wk[a, e]
    return y


def dilated_block(X: np.ndarray, lw: dict, dilations) -> np.ndarray:
    """The Syndrome Transformer's dilated convolutions (model table: 3 x Conv2d(D, D)) on
    the (d+1) x (d+1) grid of tokens X [B][(d+1)^2][D] (row-major cells): three residual
    units C = C + ReLU(Conv2d_j(C)) with the given dilations."""
    B, N, D = X.shape
    S = int(round(math.sqrt(N)))
    assert S * S == N, "the dilated convolutions need one token per grid cell"
    G = X.reshape(B, S, S, D)
    for j, dil in enumerate(dilations):
        G = G + np.maximum(conv2d_dilated(G, lw["Wd"][j], lw["bd"][j], dil), 0.0)
    return G.reshape(B, N, D)


def transformer_layer(X: np.ndarray, lw: dict, H: int, eps: float, dilations=None) -> np.ndarray:
    """One Syndrome Transformer layer, post-norm: X = LN1(X + MHA(X)); with dilated
    convolutions X = DilatedBlock(X); X = LN2(X + FF(X))."""
    X = layer_norm(X + attention(X, lw, H), lw["g1"], lw["be1"], eps)
    if dilations:
        X = dilated_block(X, lw, dilations)
    return layer_norm(X + feed_forward(X, lw), lw["g2"], lw["be2"], eps)


def rnn_core(X: np.ndarray, w: dict, H: int) -> np.ndarray:
    for lw in w["layers"]:
        X = transformer_layer(X, lw, H, w["eps"], w.get("dilations"))
    return X


def readout(state: np.ndarray, types: np.ndarray, w: dict, d: int, grid: bool = False) -> np.ndarray:
    """Readout of App. A.3 on the final decoder state.

    state: [B][N][D]. The tokens are scattered back onto the (d+1)x(d+1) grid (zeros at
    cells without a token); a 2x2 convolution without padding shrinks it to d x d:
    Y[i, j] = ReLU(b_c + sum_{a,b in {0,1}} G[i+a, j+b] @ Wc[a][b]); logical pooling
    averages over j; a linear map of the d x D features gives the logit, plus the output
    bias and the bias of the window type.
    """
    B, N, D = state.shape
    G = np.zeros((B, d + 1, d + 1, D), dtype=np.float64)
    for s, (r, c) in enumerate(token_cells(d, grid)):
        G[:, r, c, :] = state[:, s, :]
    Y = np.zeros((B, d, d, D), dtype=np.float64)
    for a in (0, 1):
        for b in (0, 1):
            Y += G[:, a:a + d, b:b + d, :] @ w["Wc"][a, b]
    Y = np.maximum(Y + w["bc"], 0.0)
    P = Y.mean(axis=2)                                   # [B][d][D]
    logits = np.einsum("bid,id->b", P, w["w_o"]) + w["b_o"][0]
    return logits + w["beta"][np.asarray(types, dtype=np.int64)]


def forward_windows(meas: np.ndarray, types: np.ndarray, w: dict, d: int, H: int,
                    return_events: bool = False, grid: bool = False):
    """Algorithm 1, inference branch, on a batch of windows.

    meas: 0/1 [B][W+1][N] measurement rounds of the N = d*d-1 stabilizers; types: [B]
    window types. D_0 = 0; for each round n: S_n = Embed(E_n); D_n = RNNCore(kappa * (S_n +
    D_{n-1})); after the last round the readout gives one logit per window; bit = [logit >
    0]. grid=True runs the network over all (d+1)^2 cells (token_cells).
    """
    meas = np.asarray(meas, dtype=np.uint8)
    B = meas.shape[0]
    W1 = meas.shape[1]
    D = w["w_e"].shape[0]
    ev = detection_events(meas, types, d)
    pos = np.array([r * (d + 1) + c for r, c in token_cells(d, grid)], dtype=np.int64)
    pe = positional_encoding((d + 1) ** 2, D)[pos]
    state = np.zeros((B, len(pos), D), dtype=np.float64)
    for n in range(W1 - 1):
        S = embed_round(ev[:, n, :], w, d, grid, pe)
        state = rnn_core(w["kappa"] * (S + state), w, H)
    logits = readout(state, types, w, d, grid)
    bits = (logits > 0).astype(np.uint8)
    if return_events:
        return logits, bits, ev
    return logits, bits


def forward_windows_recurrent(meas: np.ndarray, types: np.ndarray, w: dict, d: int, H: int,
                              grid: bool = False):
    """Algorithm 1, recurrent branch: the same pass over the window's rounds, with a readout
    of the decoder state after every round n > 2b (Sec. recurrent training), i.e. after the
    rounds that complete a window of b left buffer, tau core and b right buffer rounds,
    tau = 1..c. With left and right buffers b_L, b_R (W = b_L + c + b_R) these are the rounds
    n = W - c + 1 .. W. Returns logits [B][c] (column tau-1) and bits; the last column is the
    inference-branch result.
    """
    meas = np.asarray(meas, dtype=np.uint8)
    B, W1 = meas.shape[0], meas.shape[1]
    Wr = W1 - 1
    D = w["w_e"].shape[0]
    ev = detection_events(meas, types, d)
    pos = np.array([r * (d + 1) + c for r, c in token_cells(d, grid)], dtype=np.int64)
    pe = positional_encoding((d + 1) ** 2, D)[pos]
    state = np.zeros((B, len(pos), D), dtype=np.float64)
    logits = np.zeros((B, d), dtype=np.float64)
    for n in range(1, Wr + 1):
        S = embed_round(ev[:, n - 1, :], w, d, grid, pe)
        state = rnn_core(w["kappa"] * (S + state), w, H)
        if n > Wr - d:
            logits[:, n - (Wr - d) - 1] = readout(state, types, w, d, grid)
    return logits, (logits > 0).astype(np.uint8)


def decode_stream(R: np.ndarray, w: dict, d: int, W: int, H: int, grid: bool = False) -> int:
    """Decode a whole memory experiment: split, decode every window, XOR the bits."""
    meas, types = split_stream(R, d, W)
    _, bits = forward_windows(meas, types, w, d, H, grid=grid)
    return combine_bits(bits)
