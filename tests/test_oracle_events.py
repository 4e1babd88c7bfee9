"""Pins of the oracle's bit packing, detection events and window decomposition
(Sec. 2.2 detectors, Sec. 3.1 windows and eq. global_xor, App. A.1.1 boundary padding)."""
import numpy as np
import pytest

from oracle import decoder as O
from paper_2601_09921_amd import synth


@pytest.mark.parametrize("n", [1, 8, 31, 32, 33, 48, 120, 624])
def test_pack_roundtrip_two_implementations(n):
    rng = np.random.default_rng(n)
    bits = (rng.random((3, 5, n)) < 0.5).astype(np.uint8)
    words = synth.pack_bits(bits)
    assert words.shape == (3, 5, (n + 31) // 32)
    assert np.array_equal(O.unpack_bits(words, n), bits)
    assert np.array_equal(O.pack_bits(bits), words)
    # bit s sits in word s//32 at position s%32
    one = np.zeros(n, np.uint8)
    one[n - 1] = 1
    w = synth.pack_bits(one)
    assert w[(n - 1) // 32] == np.uint32(1 << ((n - 1) % 32)) and w.sum() == w[(n - 1) // 32]


def rand_meas(B, W, N, seed):
    rng = np.random.default_rng(seed)
    return (rng.random((B, W + 1, N)) < 0.5).astype(np.uint8)


@pytest.mark.parametrize("d,W", [(3, 6), (3, 9), (5, 10), (5, 5), (7, 14)])
def test_event_telescoping_and_masks(d, W):
    N = d * d - 1
    bl, br = O.window_split(d, W)
    assert bl + d + br == W and bl >= 0 and br >= 0
    meas = rand_meas(3, W, N, d * 100 + W)
    types = np.array([O.INITIAL, O.BULK, O.FINAL], np.uint8)
    ev = O.detection_events(meas, types, d)
    assert ev.shape == (3, W, N) and set(np.unique(ev)) <= {0, 1}
    x = np.bitwise_xor.reduce(ev, axis=1)
    # bulk: events telescope to last xor first measurement
    assert np.array_equal(x[1], meas[1, W] ^ meas[1, 0])
    # initial: nothing in the left padding, reference is the all-zero state
    assert not ev[0, :bl].any()
    assert np.array_equal(x[0], meas[0, W])
    # final: nothing in the right padding
    assert not ev[2, bl + d:].any()
    assert np.array_equal(x[2], meas[2, bl + d] ^ meas[2, 0])


def test_single_faults():
    d, W = 5, 10
    N = d * d - 1
    types = np.array([O.BULK], np.uint8)
    # a data-type error from round k on: one event, at t = k-1
    meas = np.zeros((1, W + 1, N), np.uint8)
    meas[0, 4:, 7] = 1
    ev = O.detection_events(meas, types, d)
    assert ev.sum() == 1 and ev[0, 3, 7] == 1
    # a measurement error in round k only: two events, t = k-1 and t = k
    meas = np.zeros((1, W + 1, N), np.uint8)
    meas[0, 6, 11] = 1
    ev = O.detection_events(meas, types, d)
    assert ev.sum() == 2 and ev[0, 5, 11] == 1 and ev[0, 6, 11] == 1


def test_invalid_type_rejected():
    meas = np.zeros((2, 7, 8), np.uint8)
    with pytest.raises(ValueError):
        O.detection_events(meas, np.array([1, 3], np.uint8), 3)


def stream_events(R):
    prev = np.vstack([np.zeros((1, R.shape[1]), np.uint8), R[:-1]])
    return R ^ prev


@pytest.mark.parametrize("d,W,T", [(3, 6, 20), (3, 9, 9), (5, 10, 23), (5, 15, 50), (7, 14, 14)])
def test_split_stream_cores_partition(d, W, T):
    N = d * d - 1
    R = synth.make_stream(N, T, 0.1, seed=T)
    meas, types = O.split_stream(R, d, W)
    m = meas.shape[0]
    assert m == -(-T // d) and types[0] == O.INITIAL and types[-1] == O.FINAL
    assert (types[1:-1] == O.BULK).all()
    bl, _ = O.window_split(d, W)
    ev = O.detection_events(meas, types, d)
    se = stream_events(R)
    covered = np.zeros(m * d, int)
    for i in range(m):
        for t in range(W):
            tau = i * d - bl + t
            if bl <= t < bl + d:
                covered[tau] += 1
            if 0 <= tau < T:
                assert np.array_equal(ev[i, t], se[tau])        # window sees the stream
            else:
                assert not ev[i, t].any()                      # outside: padding
    assert (covered == 1).all()                                # cores partition the rounds
    # eq. global_xor with the core-event parity as a toy per-window label
    core_par = [int(ev[i, bl:bl + d].sum() % 2) for i in range(m)]
    assert O.combine_bits(np.array(core_par)) == int(se.sum() % 2)


def test_split_stream_needs_two_windows():
    with pytest.raises(ValueError):
        O.split_stream(np.zeros((3, 8), np.uint8), 3, 6)


def test_soft_xor():
    rng = np.random.default_rng(5)
    for m in range(1, 6):
        b = rng.integers(0, 2, m)
        assert O.soft_xor(b.astype(float)) == pytest.approx(O.combine_bits(b))
    p = rng.random(4)
    assert O.soft_xor(p[:1]) == pytest.approx(p[0])
    assert O.soft_xor(p) == pytest.approx(O.soft_xor(p[::-1]))
    assert O.soft_xor(np.array([0.5, 0.1])) == pytest.approx(0.5)


def test_soft_xor_is_the_probability_of_an_odd_count():
    """Brute force over every outcome of m independent bits: P(XOR = 1) = sum of the
    probabilities of the outcomes with an odd number of ones."""
    import itertools
    rng = np.random.default_rng(9)
    for m in range(1, 7):
        p = rng.random(m)
        odd = 0.0
        for bits in itertools.product((0, 1), repeat=m):
            pr = np.prod([pk if b else 1.0 - pk for pk, b in zip(p, bits)])
            if sum(bits) % 2:
                odd += pr
        assert O.soft_xor(p) == pytest.approx(odd, rel=1e-12, abs=1e-15)


def test_synth_windows_follow_boundary_conventions():
    wl = synth.with_batch(synth.WORKLOADS["d7"], 9)
    meas, types = synth.make_windows(wl)
    bl = wl.b_left
    assert meas.shape == (9, wl.W + 1, wl.N)
    assert not meas[types == O.INITIAL, :bl + 1].any()
    fin = meas[types == O.FINAL]
    assert (fin[:, bl + wl.d:] == fin[:, bl + wl.d:bl + wl.d + 1]).all()
    # for such windows the masks change nothing: the raw xor already has zeros there
    ev = O.detection_events(meas, types, wl.d)
    assert np.array_equal(ev[types != O.INITIAL], (meas[:, 1:] ^ meas[:, :-1])[types != O.INITIAL])
