"""GPU parity of the state-resident schedule (one launch for every round and layer, each window's
state, Q, K and V in one wavefront's registers; Algorithm 1's recurrence carried on chip)
against the fp64 oracle, through the C ABI: every window of small batches (all three window
types, ragged last workgroup), the d7 workload's full batch sampled across it, zero syndromes,
batch invariance, and agreement with the layer-phased schedule on the same decoder."""
import numpy as np
import pytest

from gpu_helpers import BF16_ATOL, check_bits, check_logits, gpu_decode, inputs, oracle, say, weights
from oracle import decoder as O
from paper_2601_09921_amd import pwdec, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


# (d, W, B, H, L, grid): 1 to 4 token blocks per window, heads of 16 and 32, 1 to 4 layers,
# batches that leave the last workgroup of four windows partly empty
SHAPES = [
    (3, 6, 7, 8, 1, False),     # 8 tokens, one block
    (5, 10, 9, 4, 2, False),    # 24 tokens, two blocks, heads of 32
    (7, 14, 13, 8, 3, False),   # the d7 network
    (7, 7, 6, 8, 4, True),      # 64 grid tokens, four whole blocks, 4 layers
    (5, 15, 5, 8, 2, True),     # 36 grid tokens, W = 3d
]


def decoder(wl, w, B, schedule):
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=B)
    dec.schedule(schedule)
    return dec


@pytest.mark.parametrize("d,W,B,H,L,grid", SHAPES, ids=[f"d{s[0]}_W{s[1]}_H{s[3]}_L{s[4]}{'_grid' if s[5] else ''}"
                                                       for s in SHAPES])
def test_resident_matches_oracle(d, W, B, H, L, grid):
    wl = synth.Workload(f"r{d}", d, W, B, 0.03, 0.0, 128, L, H, 4, synth.DTYPE_BF16, grid=grid)
    w = synth.make_weights(wl, seed=d + 300)
    meas, types = synth.make_windows(wl, seed=d + 301, realistic_boundaries=False)
    say(f"resident d={d} W={W} B={B} H={H} L={L} grid={grid}")
    dec = decoder(wl, w, B, pwdec.SCHEDULE_RESIDENT)
    logits, bits, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK
    o, _ = O.forward_windows(meas, types, w, d, H, grid=grid)
    err = np.abs(logits - o)
    say(f"  max |gpu - oracle| = {err.max():.3e}")
    assert (err <= BF16_ATOL).all(), (logits, o)
    assert np.array_equal(bits, (logits > 0).astype(np.uint8))
    check_bits(bits, o)
    # batch invariance: a sub-batch starting at window 1 (every window moves to another
    # wavefront and workgroup) gives the same logits bit for bit
    sub, _, _ = gpu_decode(dec, meas[1:], types[1:])
    assert np.array_equal(sub.view(np.uint32), logits[1:].view(np.uint32))
    # the layer-phased schedule of the same decoder agrees within the bf16 tolerance
    dec.schedule(pwdec.SCHEDULE_LAYERS)
    lay, _, _ = gpu_decode(dec, meas, types)
    assert np.abs(lay - logits).max() <= BF16_ATOL
    dec.close()


def test_resident_is_the_default_where_supported():
    """AUTO picks the resident schedule for the d7 network (one resident launch and one readout
    per decode) and the layer-phased one for d25; RESIDENT is refused where it cannot run."""
    wl = synth.WORKLOADS["d7"]
    dec = pwdec.Decoder.from_workload(wl, weights("d7"), max_windows=8)
    meas, types = inputs("d7", 8)
    dec.profile(True)
    gpu_decode(dec, meas, types)
    stages = dec.profile_read()
    dec.profile(False)
    assert stages["resident"][1] == 1 and stages["readout"][1] == 1 and "attention" not in stages
    dec.close()
    big = synth.WORKLOADS["d25"]
    dec = pwdec.Decoder.from_workload(big, weights("d25"), max_windows=4)
    with pytest.raises(pwdec.PwdError) as e:
        dec.schedule(pwdec.SCHEDULE_RESIDENT)
    assert e.value.code == pwdec.PWD_EUNSUPPORTED
    dec.close()


def test_resident_zero_syndromes_equal_within_type():
    wl = synth.WORKLOADS["d7"]
    B = 12
    meas, types = inputs("d7", B, zero=True)
    dec = pwdec.Decoder.from_workload(wl, weights("d7"), max_windows=B)
    logits, _, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK
    for t in range(3):
        sel = logits[types == t]
        assert (sel.view(np.uint32) == sel.view(np.uint32)[0]).all()
    assert len({float(logits[types == t][0]) for t in range(3)}) == 3
    o, _ = O.forward_windows(meas, types, weights("d7"), wl.d, wl.H)
    assert np.abs(logits - o).max() <= BF16_ATOL
    dec.close()


def test_resident_full_d7_batch_sampled():
    """The d7 workload's full batch (1024 windows, 256 workgroups) in the configuration the
    benchmark times: windows spread across the batch -- the first, the last, the whole last
    workgroup and one per 64-window stride -- against the oracle, every other window against a
    decode of that window alone."""
    wl = synth.WORKLOADS["d7"]
    B = wl.B
    meas, types = inputs("d7", B)
    dec = pwdec.Decoder.from_workload(wl, weights("d7"), max_windows=B)
    logits, bits, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK and np.isfinite(logits).all()
    assert np.array_equal(bits, (logits > 0).astype(np.uint8))
    sample = sorted(set([0, 1, 2] + list(range(B - 4, B)) + list(range(63, B, 64))))
    o, _ = O.forward_windows(meas[sample], types[sample], weights("d7"), wl.d, wl.H)
    say(f"  d7 full batch: max |gpu - oracle| over {len(sample)} windows = {np.abs(logits[sample] - o).max():.3e}")
    assert np.abs(logits[sample] - o).max() <= BF16_ATOL
    check_bits(bits[sample], o)
    for wi in (5, 511, 770, B - 1):
        one, _, _ = gpu_decode(dec, meas[wi:wi + 1], types[wi:wi + 1])
        assert one.view(np.uint32)[0] == logits.view(np.uint32)[wi], wi
    dec.close()
