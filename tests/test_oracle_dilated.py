"""Pins of the oracle's dilated convolutions (model table: 3 x Conv2d(D, D) per Syndrome
Transformer; App. A.2: the attention output is scattered onto the 2-D grid for them).
Readings: between LayerNorm 1 and the feed-forward, three residual units C + ReLU(Conv2d(C)),
3x3 kernels, zero padding equal to the dilation; (d+1)^2 token set. Checked against torch's
conv2d, closed forms, the dilated footprint and a torch forward pass built from modules."""
import numpy as np
import pytest

from oracle import decoder as O
from paper_2601_09921_amd import synth

torch = pytest.importorskip("torch")


def torch_conv(G, Wk, b, dil):
    x = torch.tensor(np.transpose(G, (0, 3, 1, 2)).copy())                 # [B][D][S][S]
    wt = torch.tensor(np.transpose(Wk, (3, 2, 0, 1)).copy())               # [out][in][a][e]
    y = torch.nn.functional.conv2d(x, wt, torch.tensor(b), padding=dil, dilation=dil)
    return np.transpose(y.numpy(), (0, 2, 3, 1))


@pytest.mark.parametrize("S,D,dil", [(4, 8, 1), (6, 8, 2), (8, 16, 3), (4, 8, 4)])
def test_conv_matches_torch(S, D, dil):
    rng = np.random.default_rng(S * 10 + dil)
    G = rng.standard_normal((2, S, S, D))
    Wk = rng.standard_normal((3, 3, D, D)) / np.sqrt(9 * D)
    b = rng.standard_normal(D)
    assert np.allclose(O.conv2d_dilated(G, Wk, b, dil), torch_conv(G, Wk, b, dil), atol=1e-12)


def test_footprint_of_one_unit():
    """A single nonzero cell reaches exactly the cells at offsets {-dil, 0, dil}^2 (inside the
    grid) through one unit with zero biases and positive weights."""
    S, D = 9, 4
    for dil in (1, 2, 3):
        lw = {"Wd": np.abs(np.random.default_rng(dil).standard_normal((3, 3, 3, D, D))),
              "bd": np.zeros((3, D))}
        X = np.zeros((1, S * S, D))
        X[0, 4 * S + 4, :] = 1.0
        G = X.reshape(1, S, S, D)
        one = G + np.maximum(O.conv2d_dilated(G, lw["Wd"][0], lw["bd"][0], dil), 0.0)
        changed = {(r, c) for r in range(S) for c in range(S) if np.abs(one[0, r, c] - G[0, r, c]).max() > 0}
        expect = {(4 + dil * a, 4 + dil * e) for a in (-1, 0, 1) for e in (-1, 0, 1)}
        assert changed == expect, (dil, sorted(changed))


def test_zero_weights_add_relu_of_biases():
    rng = np.random.default_rng(3)
    X = rng.standard_normal((2, 25, 8))
    bd = rng.standard_normal((3, 8))
    lw = {"Wd": np.zeros((3, 3, 3, 8, 8)), "bd": bd}
    assert np.allclose(O.dilated_block(X, lw, [1, 2, 4]), X + np.maximum(bd, 0).sum(axis=0), atol=1e-14)


def test_block_needs_grid_tokens():
    with pytest.raises(AssertionError):
        O.dilated_block(np.zeros((1, 8, 4)), {"Wd": np.zeros((3, 3, 3, 4, 4)), "bd": np.zeros((3, 4))}, [1, 1, 1])


def torch_forward(meas, types, w, wl):
    """float64 forward with torch modules: per layer MultiheadAttention, LayerNorm, conv2d on
    the grid, Linear feed-forward; embedding and readout as in the paper."""
    d, D, H = wl.d, wl.D, wl.H
    S = d + 1
    cells = O.stabilizer_cells(d)
    m_t = torch.tensor(meas.astype(np.float64))
    ev = (m_t[:, 1:] != m_t[:, :-1]).double()
    bl = (wl.W - d) // 2
    for b in range(meas.shape[0]):
        if types[b] == 0:
            ev[b, :bl] = 0
            ev[b, bl] = m_t[b, bl + 1]
        if types[b] == 2:
            ev[b, bl + d:] = 0
    evg = torch.zeros(meas.shape[0], wl.W, S * S, dtype=torch.float64)
    for s, (r, c) in enumerate(cells):
        evg[:, :, r * S + c] = ev[:, :, s]
    pos = torch.arange(S * S, dtype=torch.float64)
    freq = 10000.0 ** (-torch.arange(0, D, 2, dtype=torch.float64) / D)
    ang = pos[:, None] * freq[None, :]
    pe = torch.stack([torch.sin(ang), torch.cos(ang)], dim=-1).reshape(S * S, D)
    T = lambda a: torch.tensor(np.ascontiguousarray(a))
    mods = []
    for lw in w["layers"]:
        mha = torch.nn.MultiheadAttention(D, H, batch_first=True).double()
        mha.load_state_dict({"in_proj_weight": T(np.concatenate([lw["Wq"].T, lw["Wk"].T, lw["Wv"].T])),
                             "in_proj_bias": T(np.concatenate([lw["bq"], lw["bk"], lw["bv"]])),
                             "out_proj.weight": T(lw["Wo"].T), "out_proj.bias": T(lw["bo"])})
        mods.append(mha.eval())
    state = torch.zeros(meas.shape[0], S * S, D, dtype=torch.float64)
    ln = torch.nn.functional.layer_norm
    with torch.no_grad():
        for n in range(wl.W):
            x = (evg[:, n, :, None] * T(w["w_e"]) + T(w["b_e"]) + pe + state) * w["kappa"]
            for lw, mha in zip(w["layers"], mods):
                x = ln(x + mha(x, x, x, need_weights=False)[0], (D,), T(lw["g1"]), T(lw["be1"]), w["eps"])
                g = x.transpose(1, 2).reshape(-1, D, S, S)
                for j, dil in enumerate(w["dilations"]):
                    wt = T(np.transpose(lw["Wd"][j], (3, 2, 0, 1)))
                    g = g + torch.relu(torch.nn.functional.conv2d(g, wt, T(lw["bd"][j]), padding=dil, dilation=dil))
                x = g.reshape(-1, D, S * S).transpose(1, 2)
                ff = torch.relu(x @ T(lw["W1"]) + T(lw["b1"])) @ T(lw["W2"]) + T(lw["b2"])
                x = ln(x + ff, (D,), T(lw["g2"]), T(lw["be2"]), w["eps"])
            state = x
        G = state.transpose(1, 2).reshape(-1, D, S, S)
        wc = T(np.transpose(w["Wc"], (3, 2, 0, 1)))
        Y = torch.relu(torch.nn.functional.conv2d(G, wc, T(w["bc"])))
        feat = Y.mean(dim=3).transpose(1, 2).reshape(-1, d * D)
        return (feat @ T(w["w_o"]).reshape(d * D, 1))[:, 0].numpy() + w["b_o"][0] + w["beta"][types]


@pytest.mark.parametrize("d,W,D,L,H,dil", [(3, 6, 16, 2, 2, (1, 2, 4)), (5, 10, 16, 1, 4, (1, 1, 2)),
                                           (3, 9, 8, 2, 2, (2, 1, 3))])
def test_forward_matches_torch(d, W, D, L, H, dil):
    wl = synth.Workload("c", d, W, 5, 0.15, 0.0, D, L, H, 4, synth.DTYPE_F32, grid=True, dil=dil)
    w = synth.make_weights(wl, seed=d + W)
    meas, types = synth.make_windows(wl, seed=13, realistic_boundaries=False)
    logits, bits = O.forward_windows(meas, types, w, d, H, grid=True)
    assert np.allclose(logits, torch_forward(meas, types, w, wl), atol=1e-10)
    # and the block changes the result
    plain = {k: v for k, v in w.items() if k != "dilations"}
    ref, _ = O.forward_windows(meas, types, plain, d, H, grid=True)
    assert np.abs(ref - logits).max() > 1e-3
