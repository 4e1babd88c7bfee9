"""Pins of the oracle's embedder residual block (App. A model table: 2 x Conv1d(D, D) after
Linear(1 -> D); syndrome-convolution section: the block runs on the flattened (d+1)^2 array
ahead of PE). Readings: kernel 3, zero padding 1, biases, ReLU between the two layers, the
input added back. Checked against torch's Conv1d, a closed form and the receptive field."""
import numpy as np
import pytest

from oracle import decoder as O
from paper_2601_09921_amd import synth

torch = pytest.importorskip("torch")


def workload(d=5, D=16, grid=False):
    return synth.Workload("r", d, 2 * d, 4, 0.2, 0.0, D, 1, 2, 4, synth.DTYPE_F32, grid=grid, resnet=True)


def events(wl, seed):
    return (np.random.default_rng(seed).random((wl.B, wl.N)) < 0.3).astype(np.uint8)


@pytest.mark.parametrize("grid", [False, True])
def test_embedding_matches_torch_conv1d(grid):
    wl = workload(grid=grid)
    w = synth.make_weights(wl, seed=5)
    ev = events(wl, 6)
    d, D = wl.d, wl.D
    cells = [r * (d + 1) + c for r, c in O.token_cells(d, grid)]
    pe = O.positional_encoding((d + 1) ** 2, D)[cells]
    got = O.embed_round(ev, w, d, grid, pe)
    evg = np.zeros((wl.B, (d + 1) ** 2))
    for s, (r, c) in enumerate(O.stabilizer_cells(d)):
        evg[:, r * (d + 1) + c] = ev[:, s]
    E = torch.tensor(evg[:, None, :] * w["w_e"][None, :, None] + w["b_e"][None, :, None])   # [B][D][L]
    wt = lambda k: torch.tensor(np.transpose(w["res"]["W" + k], (2, 1, 0)).copy())   # [out][in][k]
    h = torch.relu(torch.nn.functional.conv1d(E, wt("1"), torch.tensor(w["res"]["b1"]), padding=1))
    ref = (E + torch.nn.functional.conv1d(h, wt("2"), torch.tensor(w["res"]["b2"]), padding=1)).numpy()
    ref = np.transpose(ref, (0, 2, 1))[:, cells, :] + pe[None]
    assert np.allclose(got, ref, atol=1e-12)


def test_zero_second_layer_adds_its_bias():
    """With the second Conv1d's weights zero the block adds only that layer's bias: the
    embedding is E * w_e + b_e + b2 + PE."""
    wl = workload()
    w = synth.make_weights(wl, seed=7)
    w["res"]["W2"] = np.zeros_like(w["res"]["W2"])
    ev = events(wl, 8)
    pe = O.positional_encoding((wl.d + 1) ** 2, wl.D)[O.grid_positions(wl.d)]
    plain = dict(w)
    del plain["res"]
    got = O.embed_round(ev, w, wl.d, False, pe)
    assert np.allclose(got, O.embed(ev, plain, pe) + w["res"]["b2"][None, None, :], atol=1e-12)


def test_receptive_field_is_five_cells():
    """Two kernel-3 layers see cells p-2 .. p+2 of the flattened array: flipping the event of
    one stabilizer changes the embedding exactly within that range (the ReLU can hide a
    change, never create one outside it)."""
    wl = workload(d=7, D=32, grid=True)
    w = synth.make_weights(wl, seed=9)
    d = wl.d
    pe = O.positional_encoding((d + 1) ** 2, wl.D)
    ev = np.zeros((1, wl.N), dtype=np.uint8)
    base = O.embed_round(ev, w, d, True, pe)
    for s in (0, 5, wl.N // 2, wl.N - 1):
        r, c = O.stabilizer_cells(d)[s]
        cell = r * (d + 1) + c
        ev1 = ev.copy()
        ev1[0, s] = 1
        diff = np.abs(O.embed_round(ev1, w, d, True, pe) - base).max(axis=-1)[0]
        changed = set(np.flatnonzero(diff > 1e-12).tolist())
        assert cell in changed
        assert changed <= set(range(cell - 2, cell + 3)), (s, cell, sorted(changed))


def test_resnet_changes_the_forward_pass_only_through_the_embedding():
    """The weights without the block are the same draws, so removing "res" gives the plain
    network; with the block the logits move."""
    wl = workload(d=3, D=16)
    w = synth.make_weights(wl, seed=11)
    plain = synth.make_weights(synth.Workload("r", 3, 6, 4, 0.2, 0.0, 16, 1, 2, 4, synth.DTYPE_F32), seed=11)
    assert all(np.array_equal(w[k], plain[k]) for k in ("w_e", "b_e", "Wc", "bc", "w_o", "beta"))
    meas, types = synth.make_windows(wl, seed=12, realistic_boundaries=False)
    a, _ = O.forward_windows(meas, types, w, wl.d, wl.H)
    b, _ = O.forward_windows(meas, types, plain, wl.d, wl.H)
    assert np.abs(a - b).max() > 1e-3
