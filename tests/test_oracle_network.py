"""Pins of the oracle's network (App. A): positional encoding, LayerNorm, attention and
the Syndrome Transformer layer against torch's own float64 modules, the readout against
torch's conv2d, the recurrent fold in closed form, and whole-forward invariants."""
import math

import numpy as np
import pytest
import torch

from oracle import decoder as O
from paper_2601_09921_amd import synth

torch.set_default_dtype(torch.float64)


def tiny_workload(d=3, W=6, D=16, L=2, H=4, B=8, dtype=synth.DTYPE_F32, p=0.2):
    return synth.Workload("tiny", d, W, B, p, 0.0, D, L, H, 4, dtype)


# ----------------------------------------------------------------------------- PE

@pytest.mark.parametrize("D", [16, 64, 256])
def test_positional_encoding_identities(D):
    P = 40
    pe = O.positional_encoding(P, D)
    assert np.array_equal(pe[0], np.tile([0.0, 1.0], D // 2))
    assert np.allclose((pe ** 2).sum(axis=1), D / 2)
    # even/odd pairs rotate: PE(t+k) = R(k w_i) PE(t) with w_0 = 1 and
    # w_{D/2-1} = 10000^{-(D-2)/D}; the frequencies form a geometric progression
    w = np.array([math.atan2(pe[1, 2 * i], pe[1, 2 * i + 1]) for i in range(D // 2)])
    assert w[0] == pytest.approx(1.0)
    assert w[-1] == pytest.approx(10000.0 ** (-(D - 2) / D))
    assert np.allclose(w[1:] / w[:-1], 10000.0 ** (-2.0 / D))
    for t, k in [(3, 5), (17, 11), (0, 39)]:
        s, c = pe[t, 0::2], pe[t, 1::2]
        assert np.allclose(pe[t + k, 0::2], s * np.cos(k * w) + c * np.sin(k * w))
        assert np.allclose(pe[t + k, 1::2], c * np.cos(k * w) - s * np.sin(k * w))


# ----------------------------------------------------------------------------- LN, softmax

def test_layer_norm_properties():
    rng = np.random.default_rng(0)
    y = rng.standard_normal((5, 7, 32)) * 3 + 2
    one, zero = np.ones(32), np.zeros(32)
    z = O.layer_norm(y, one, zero, 0.0)
    assert np.allclose(z.mean(-1), 0) and np.allclose(z.var(-1), 1)
    assert np.allclose(O.layer_norm(5 * y - 7, one, zero, 0.0), z)
    g, b = rng.standard_normal(32), rng.standard_normal(32)
    ref = torch.nn.functional.layer_norm(torch.tensor(y), (32,), torch.tensor(g), torch.tensor(b), 1e-5)
    assert np.allclose(O.layer_norm(y, g, b, 1e-5), ref.numpy(), atol=1e-12)


def test_softmax_properties():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((4, 9)) * 10
    s = O.softmax(x)
    assert np.allclose(s.sum(-1), 1) and (s > 0).all()
    assert np.allclose(O.softmax(x + 123.0), s)
    assert np.allclose(s, torch.softmax(torch.tensor(x), -1).numpy())


# ----------------------------------------------------------------------------- attention

def layer_weights(D, F, seed):
    wl = tiny_workload(D=D)
    w = synth.make_weights(synth.Workload("t", 3, 6, 1, 0.1, 0.0, D, 1, 4, F // D, synth.DTYPE_F32), seed=seed)
    return w["layers"][0]


def torch_mha(lw, D, H):
    m = torch.nn.MultiheadAttention(D, H, bias=True, batch_first=True)
    with torch.no_grad():
        m.in_proj_weight.copy_(torch.tensor(np.concatenate([lw["Wq"].T, lw["Wk"].T, lw["Wv"].T])))
        m.in_proj_bias.copy_(torch.tensor(np.concatenate([lw["bq"], lw["bk"], lw["bv"]])))
        m.out_proj.weight.copy_(torch.tensor(lw["Wo"].T))
        m.out_proj.bias.copy_(torch.tensor(lw["bo"]))
    return m.eval()


@pytest.mark.parametrize("D,H,N", [(16, 4, 8), (32, 2, 13), (64, 8, 48)])
def test_attention_matches_torch_mha(D, H, N):
    lw = layer_weights(D, 4 * D, seed=D + N)
    X = np.random.default_rng(2).standard_normal((3, N, D))
    m = torch_mha(lw, D, H)
    with torch.no_grad():
        ref, _ = m(torch.tensor(X), torch.tensor(X), torch.tensor(X), need_weights=False)
    assert np.allclose(O.attention(X, lw, H), ref.numpy(), atol=1e-12)


def test_attention_special_cases():
    D, H, N = 16, 4, 6
    lw = dict(layer_weights(D, 4 * D, seed=9))
    X = np.random.default_rng(3).standard_normal((2, N, D))
    V = X @ lw["Wv"] + lw["bv"]
    # zero query projection: uniform weights, every token gets the mean of the values
    z = dict(lw, Wq=np.zeros((D, D)), bq=np.zeros(D))
    out = O.attention(X, z, H)
    assert np.allclose(out, (V.mean(axis=1, keepdims=True) @ lw["Wo"] + lw["bo"]).repeat(N, 1))
    # one token attends only to itself
    assert np.allclose(O.attention(X[:, :1], lw, H), V[:, :1] @ lw["Wo"] + lw["bo"])
    # a key bias shifts every score of a query row equally: no effect
    kb = dict(lw, bk=lw["bk"] + 3.0)
    assert np.allclose(O.attention(X, kb, H), O.attention(X, lw, H))
    # no mask, no positions: permuting the tokens permutes the outputs
    perm = np.random.default_rng(4).permutation(N)
    assert np.allclose(O.attention(X[:, perm], lw, H), O.attention(X, lw, H)[:, perm])


@pytest.mark.parametrize("F", [128, 160], ids=["ffn4", "ffn5"])
def test_transformer_layer_matches_torch(F):
    D, H, N = 32, 4, 11
    lw = layer_weights(D, F, seed=21)
    X = np.random.default_rng(5).standard_normal((3, N, D))
    m = torch.nn.TransformerEncoderLayer(D, H, F, dropout=0.0, activation="relu",
                                         layer_norm_eps=1e-5, batch_first=True, norm_first=False)
    with torch.no_grad():
        m.self_attn.load_state_dict(torch_mha(lw, D, H).state_dict())
        m.linear1.weight.copy_(torch.tensor(lw["W1"].T))
        m.linear1.bias.copy_(torch.tensor(lw["b1"]))
        m.linear2.weight.copy_(torch.tensor(lw["W2"].T))
        m.linear2.bias.copy_(torch.tensor(lw["b2"]))
        m.norm1.weight.copy_(torch.tensor(lw["g1"]))
        m.norm1.bias.copy_(torch.tensor(lw["be1"]))
        m.norm2.weight.copy_(torch.tensor(lw["g2"]))
        m.norm2.bias.copy_(torch.tensor(lw["be2"]))
    m.eval()
    with torch.no_grad():
        ref = m(torch.tensor(X))
    assert np.allclose(O.transformer_layer(X, lw, H, 1e-5), ref.numpy(), atol=1e-11)
    # feed-forward with a zero second matrix returns its bias
    assert np.allclose(O.feed_forward(X, dict(lw, W2=np.zeros((F, D)))), np.broadcast_to(lw["b2"], X.shape))


# ----------------------------------------------------------------------------- readout

@pytest.mark.parametrize("d,D", [(3, 16), (5, 8), (7, 4)])
def test_readout_matches_conv2d(d, D):
    wl = synth.Workload("t", d, 2 * d, 4, 0.1, 0.0, D, 1, 2, 4, synth.DTYPE_F32)
    w = synth.make_weights(wl, seed=d)
    B, N = 4, d * d - 1
    state = np.random.default_rng(d).standard_normal((B, N, D))
    types = np.array([0, 1, 2, 1], np.uint8)
    G = torch.zeros(B, D, d + 1, d + 1)
    for s, (r, c) in enumerate(O.stabilizer_cells(d)):
        G[:, :, r, c] = torch.tensor(state[:, s, :])
    weight = torch.tensor(np.transpose(w["Wc"], (3, 2, 0, 1)).copy())      # [out][in][a][b]
    Y = torch.relu(torch.nn.functional.conv2d(G, weight, torch.tensor(w["bc"])))
    P = Y.mean(dim=3)                                                       # pool over columns
    ref = (P * torch.tensor(w["w_o"].T)[None]).sum(dim=(1, 2)) + w["b_o"][0] + torch.tensor(w["beta"][types])
    assert np.allclose(O.readout(state, types, w, d), ref.numpy(), atol=1e-12)
    # zero state: every output cell is ReLU(b_c)
    z = O.readout(np.zeros((3, N, D)), np.array([0, 1, 2]), w, d)
    closed = np.maximum(w["bc"], 0) @ w["w_o"].sum(axis=0) + w["b_o"][0] + w["beta"]
    assert np.allclose(z, closed)


# ----------------------------------------------------------------------------- recurrence

def test_fold_closed_form_without_layers():
    """With no transformer layers D_n = kappa (S_n + D_{n-1}), D_0 = 0, so the final state
    is sum_k kappa^(W-k+1) S_k (App. A.2 fold equation; Algorithm 1 initial state)."""
    wl = tiny_workload(L=0, B=5, W=6)
    w = synth.make_weights(wl, seed=3)
    meas, types = synth.make_windows(wl, seed=7, realistic_boundaries=False)
    logits, _ = O.forward_windows(meas, types, w, wl.d, wl.H)
    ev = O.detection_events(meas, types, wl.d)
    pe = O.positional_encoding((wl.d + 1) ** 2, wl.D)[O.grid_positions(wl.d)]
    kappa = w["kappa"]
    state = sum(kappa ** (wl.W - n) * O.embed(ev[:, n], w, pe) for n in range(wl.W))
    assert np.allclose(logits, O.readout(state, types, w, wl.d))


def torch_model_logits(meas, types, w, wl, grid=False):
    """An independent float64 forward built from torch modules (grid: every cell of the
    (d+1)x(d+1) array is a token, events only at stabilizer cells)."""
    d, D, H, F = wl.d, wl.D, wl.H, wl.F
    layers = []
    for lw in w["layers"]:
        m = torch.nn.TransformerEncoderLayer(D, H, F, dropout=0.0, batch_first=True, layer_norm_eps=w["eps"])
        sd = {
            "self_attn.in_proj_weight": np.concatenate([lw["Wq"].T, lw["Wk"].T, lw["Wv"].T]),
            "self_attn.in_proj_bias": np.concatenate([lw["bq"], lw["bk"], lw["bv"]]),
            "self_attn.out_proj.weight": lw["Wo"].T, "self_attn.out_proj.bias": lw["bo"],
            "linear1.weight": lw["W1"].T, "linear1.bias": lw["b1"],
            "linear2.weight": lw["W2"].T, "linear2.bias": lw["b2"],
            "norm1.weight": lw["g1"], "norm1.bias": lw["be1"],
            "norm2.weight": lw["g2"], "norm2.bias": lw["be2"],
        }
        m.load_state_dict({k: torch.tensor(np.ascontiguousarray(v)) for k, v in sd.items()})
        layers.append(m.eval())
    cells = O.stabilizer_cells(d)
    B = meas.shape[0]
    m_t = torch.tensor(meas.astype(np.float64))
    ev = (m_t[:, 1:] != m_t[:, :-1]).double()
    bl = (wl.W - d) // 2
    for b in range(B):
        if types[b] == 0:
            ev[b, :bl] = 0
            ev[b, bl] = m_t[b, bl + 1]
        if types[b] == 2:
            ev[b, bl + d:] = 0
    # the stabilizer events on the flattened grid (zeros at cells without a stabilizer)
    evg = torch.zeros(B, wl.W, (d + 1) ** 2, dtype=torch.float64)
    for s, (r, c) in enumerate(cells):
        evg[:, :, r * (d + 1) + c] = ev[:, :, s]
    if grid:   # tokens = all cells
        cells = [(r, c) for r in range(d + 1) for c in range(d + 1)]
    cell_idx = [r * (d + 1) + c for r, c in cells]
    convs = None
    if "res" in w:   # the embedder's residual block as two torch Conv1d modules
        convs = []
        for k in ("1", "2"):
            cv = torch.nn.Conv1d(D, D, 3, padding=1).double()
            with torch.no_grad():
                cv.weight.copy_(torch.tensor(np.transpose(w["res"]["W" + k], (2, 1, 0)).copy()))
                cv.bias.copy_(torch.tensor(w["res"]["b" + k]))
            convs.append(cv)
    pos = torch.tensor([r * (d + 1) + c for r, c in cells], dtype=torch.float64)
    freq = 10000.0 ** (-torch.arange(0, D, 2, dtype=torch.float64) / D)
    ang = pos[:, None] * freq[None, :]
    pe = torch.stack([torch.sin(ang), torch.cos(ang)], dim=-1).reshape(len(cells), D)
    state = torch.zeros(B, len(cells), D)
    with torch.no_grad():
        for n in range(wl.W):
            E = evg[:, n, :, None] * torch.tensor(w["w_e"]) + torch.tensor(w["b_e"])   # [B][cells][D]
            if convs is not None:
                Et = E.transpose(1, 2)
                E = (Et + convs[1](torch.relu(convs[0](Et)))).transpose(1, 2)
            S = E[:, cell_idx] + pe
            x = (S + state) * w["kappa"]
            for m in layers:
                x = m(x)
            state = x
        G = torch.zeros(B, D, d + 1, d + 1)
        for s, (r, c) in enumerate(cells):
            G[:, :, r, c] = state[:, s]
        wc = torch.tensor(np.transpose(w["Wc"], (3, 2, 0, 1)).copy())
        Y = torch.relu(torch.nn.functional.conv2d(G, wc, torch.tensor(w["bc"])))
        feat = Y.mean(dim=3).transpose(1, 2).reshape(B, d * D)
        lin = torch.tensor(w["w_o"]).reshape(1, d * D)
        return (feat @ lin.T)[:, 0].numpy() + w["b_o"][0] + w["beta"][types]


@pytest.mark.parametrize("grid", [False, True], ids=["stabilizers", "grid"])
@pytest.mark.parametrize("d,W,D,L,H,r,res", [(3, 6, 16, 2, 4, 4, False), (3, 9, 32, 1, 2, 4, False),
                                             (5, 10, 16, 2, 2, 4, False), (3, 6, 16, 2, 2, 5, False),
                                             (3, 6, 16, 2, 4, 4, True), (5, 10, 16, 1, 2, 5, True)])
def test_forward_matches_torch_model(d, W, D, L, H, r, res, grid):
    wl = synth.Workload("t", d, W, 6, 0.15, 0.0, D, L, H, r, synth.DTYPE_F32, resnet=res)
    w = synth.make_weights(wl, seed=d + W)
    meas, types = synth.make_windows(wl, seed=11, realistic_boundaries=False)
    logits, bits = O.forward_windows(meas, types, w, d, H, grid=grid)
    ref = torch_model_logits(meas, types, w, wl, grid=grid)
    assert np.allclose(logits, ref, atol=1e-10)
    assert np.array_equal(bits, (logits > 0).astype(np.uint8))


def test_forward_invariants():
    wl = tiny_workload(B=9, p=0.3)
    w = synth.make_weights(wl, seed=1)
    meas, types = synth.make_windows(wl, seed=2, realistic_boundaries=False)
    logits, _ = O.forward_windows(meas, types, w, wl.d, wl.H)
    # one window at a time equals the batch
    single = np.array([O.forward_windows(meas[i:i + 1], types[i:i + 1], w, wl.d, wl.H)[0][0] for i in range(9)])
    assert np.allclose(single, logits, atol=1e-13)
    # permuting the windows permutes the outputs
    perm = np.random.default_rng(0).permutation(9)
    assert np.allclose(O.forward_windows(meas[perm], types[perm], w, wl.d, wl.H)[0], logits[perm], atol=1e-13)
    # all-zero syndromes: identical logits within a type, differing across types
    zm, zt = synth.make_windows(wl, zero=True)
    zl, _ = O.forward_windows(zm[:9], zt[:9], w, wl.d, wl.H)
    for t in range(3):
        assert np.ptp(zl[zt[:9] == t]) == 0.0
    assert len(set(np.round(zl[:3], 12))) == 3
    # the recurrence is ordered: a lone event in round t differs from one in round t'
    one = np.zeros((2, wl.W + 1, wl.N), np.uint8)
    one[0, 3:, 2] = 1
    one[1, 4:, 2] = 1
    la, _ = O.forward_windows(one, np.array([1, 1], np.uint8), w, wl.d, wl.H)
    assert abs(la[0] - la[1]) > 1e-6


def test_recurrent_readouts():
    """Algorithm 1's recurrent branch: the last readout is the inference result, and by
    causality the readout after round n of a bulk window (no masks) is the decode of the
    window cut after round n, here from the independent torch model."""
    import dataclasses
    wl = tiny_workload(B=9, W=8, p=0.3)
    w = synth.make_weights(wl, seed=6)
    meas, types = synth.make_windows(wl, seed=8, realistic_boundaries=False)
    rl, rb = O.forward_windows_recurrent(meas, types, w, wl.d, wl.H)
    fl, _ = O.forward_windows(meas, types, w, wl.d, wl.H)
    assert rl.shape == (wl.B, wl.d) and np.array_equal(rb, (rl > 0).astype(np.uint8))
    assert np.array_equal(rl[:, -1], fl)
    bulk = types == O.BULK
    assert bulk.sum() >= 2
    for tau in range(wl.d):
        n = wl.W - wl.d + 1 + tau
        ref = torch_model_logits(meas[bulk, :n + 1], types[bulk], w, dataclasses.replace(wl, W=n))
        assert np.allclose(rl[bulk, tau], ref, atol=1e-10)
    # the readouts move with the rounds they have seen
    assert np.ptp(rl, axis=1).min() > 1e-9


def test_stream_decode_is_xor_of_windows():
    wl = tiny_workload(B=1, W=6)
    w = synth.make_weights(wl, seed=4)
    R = synth.make_stream(wl.N, 17, 0.2, seed=3)
    meas, types = O.split_stream(R, wl.d, wl.W)
    _, bits = O.forward_windows(meas, types, w, wl.d, wl.H)
    assert O.decode_stream(R, w, wl.d, wl.W, wl.H) == int(np.bitwise_xor.reduce(bits))


def test_grid_tokens_fold_and_empty_cells():
    """The (d+1)^2 token set with no transformer layers: the final state of every cell is
    sum_k kappa^(W-k+1) S_k, where a cell without a stabilizer sees only b_e + PE; those cells
    feed the readout, so the logits differ from the stabilizer-only token set."""
    wl = tiny_workload(L=0, B=5, W=6)
    w = synth.make_weights(wl, seed=3)
    meas, types = synth.make_windows(wl, seed=7, realistic_boundaries=False)
    d = wl.d
    ev = O.token_events(O.detection_events(meas, types, d), d, grid=True)
    assert ev.shape[-1] == (d + 1) ** 2 and ev.sum() == O.detection_events(meas, types, d).sum()
    empty = [r * (d + 1) + c for r in range(d + 1) for c in range(d + 1)
             if (r, c) not in set(O.stabilizer_cells(d))]
    assert len(empty) == 2 * d + 2 and not ev[..., empty].any()   # (d+1)^2 - (d^2 - 1) cells
    pe = O.positional_encoding((d + 1) ** 2, wl.D)
    kappa = w["kappa"]
    state = sum(kappa ** (wl.W - n) * O.embed(ev[:, n], w, pe) for n in range(wl.W))
    logits, _ = O.forward_windows(meas, types, w, d, wl.H, grid=True)
    assert np.allclose(logits, O.readout(state, types, w, d, grid=True))
    stab, _ = O.forward_windows(meas, types, w, d, wl.H)
    assert np.abs(logits - stab).max() > 1e-3
