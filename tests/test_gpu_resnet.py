"""GPU parity of the embedder's residual Conv1d block (App. A model table: Linear(1 -> D) then
2 x Conv1d(D, D); syndrome-convolution section: on the flattened (d+1)^2 array ahead of PE)
against the fp64 oracle, which runs the two convolutions directly: fp32 and bf16, both
token sets, the inference and recurrent branches and stream decoding. The library looks the
block's output up by the five event bits around each cell (exact: the block's input is one
bit per cell), so event patterns at the ends of the flattened array and next to empty cells
are what these cases cover."""
import numpy as np
import pytest

from gpu_helpers import BF16_ATOL, FP32_ATOL, FP32_RTOL, check_bits, gpu_decode, gpu_events, say, to_device
from oracle import decoder as O
from paper_2601_09921_amd import pwdec, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BF16, F32 = synth.DTYPE_BF16, synth.DTYPE_F32
# (d, W, B, D, L, H, mlp_ratio, dtype, grid)
SHAPES = [
    (3, 6, 9, 64, 2, 4, 4, F32, False),
    (3, 6, 9, 32, 2, 2, 5, F32, True),
    (5, 10, 7, 128, 2, 8, 4, BF16, False),
    (7, 14, 5, 128, 3, 8, 4, BF16, True),
    (11, 22, 4, 256, 2, 8, 5, BF16, True),
    (13, 26, 3, 256, 1, 4, 4, BF16, False),
    (25, 25, 2, 256, 1, 8, 4, BF16, True),
    (33, 33, 1, 128, 1, 8, 4, BF16, True),     # the largest grid: 1156 cells, 5 position classes
]


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def within(g, o, dtype):
    if dtype == F32:
        return (np.abs(g - o) <= FP32_RTOL * np.abs(o) + FP32_ATOL).all()
    return (np.abs(g - o) <= BF16_ATOL).all()


def workload(d, W, B, D, L, H, r, dtype, grid):
    return synth.Workload(f"r{d}", d, W, B, 0.2, 0.0, D, L, H, r, dtype, grid=grid, resnet=True)


def ids(shapes):
    return [f"d{s[0]}_D{s[3]}_r{s[6]}_{'f32' if s[7] == F32 else 'bf16'}{'_grid' if s[8] else ''}" for s in shapes]


@pytest.mark.parametrize("d,W,B,D,L,H,r,dtype,grid", SHAPES, ids=ids(SHAPES))
def test_resnet_parity(d, W, B, D, L, H, r, dtype, grid):
    wl = workload(d, W, B, D, L, H, r, dtype, grid)
    w = synth.make_weights(wl, seed=d + 900)
    assert "res" in w
    # dense events (p = 0.2) so that most of the 32 patterns around a cell occur
    meas, types = synth.make_windows(wl, seed=d + 901, realistic_boundaries=False)
    say(f"resnet embedder d={d} W={W} B={B} D={D} L={L} H={H} r={r} dtype={dtype} grid={grid}")
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=B)
    o_logits, _, o_ev = O.forward_windows(meas, types, w, d, H, return_events=True, grid=grid)
    if dtype == BF16:
        ev, rc = gpu_events(dec, meas, types, W, wl.words)
        assert rc == pwdec.PWD_OK and np.array_equal(ev, O.pack_bits(o_ev))
    logits, bits, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK
    err = np.abs(logits - o_logits)
    say(f"  max |gpu - oracle| = {err.max():.3e}")
    assert within(logits, o_logits, dtype), (logits, o_logits)
    check_bits(bits, o_logits)
    sub, _, _ = gpu_decode(dec, meas[1:], types[1:])
    assert np.array_equal(sub.view(np.uint32), logits[1:].view(np.uint32))
    dec.close()
    # the block matters: the same draws without it give other logits
    plain = dict(w)
    del plain["res"]
    p_logits, _ = O.forward_windows(meas, types, plain, d, H, grid=grid)
    assert np.abs(p_logits - o_logits).max() > 10 * max(err.max(), 1e-6)


@pytest.mark.parametrize("d,W,B,D,L,H,r,dtype,grid", [SHAPES[0], SHAPES[3], SHAPES[5]],
                         ids=ids([SHAPES[0], SHAPES[3], SHAPES[5]]))
def test_resnet_recurrent(d, W, B, D, L, H, r, dtype, grid):
    wl = workload(d, W, B, D, L, H, r, dtype, grid)
    w = synth.make_weights(wl, seed=d + 902)
    meas, types = synth.make_windows(wl, seed=d + 903, realistic_boundaries=False)
    say(f"resnet embedder recurrent d={d} D={D} dtype={dtype} grid={grid}")
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=B)
    meas_t, types_t = to_device(meas, types)
    logits = torch.full((B, d), float("nan"), dtype=torch.float32, device="cuda")
    bits = torch.full((B, d), 7, dtype=torch.uint8, device="cuda")
    dec.decode_recurrent(meas_t, types_t, logits, bits)
    torch.cuda.synchronize()
    assert dec.sync_status() == pwdec.PWD_OK
    gl = logits.cpu().numpy()
    dec.close()
    ol, _ = O.forward_windows_recurrent(meas, types, w, d, H, grid=grid)
    say(f"  max |gpu - oracle| = {np.abs(gl - ol).max():.3e}")
    assert within(gl, ol, dtype), (gl, ol)
    assert np.array_equal(bits.cpu().numpy(), (gl > 0).astype(np.uint8))


def test_resnet_stream():
    """decode_stream with the block: per-window logits against the oracle's, and the stream
    bit as the XOR of the window bits."""
    wl = workload(7, 14, 1, 128, 2, 8, 4, BF16, False)
    w = synth.make_weights(wl, seed=904)
    T = 6 * wl.d - 3
    m = -(-T // wl.d)
    R = synth.make_stream(wl.N, T, 0.05, seed=905)
    say(f"resnet embedder stream d7 T={T}")
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=m)
    rounds = torch.from_numpy(O.pack_bits(R).view(np.int32)).cuda()
    bit = torch.zeros(1, dtype=torch.uint8, device="cuda")
    wlog = torch.zeros(m, dtype=torch.float32, device="cuda")
    wbits = torch.zeros(m, dtype=torch.uint8, device="cuda")
    dec.decode_stream(rounds, bit, window_logits=wlog, window_bits=wbits)
    torch.cuda.synchronize()
    assert dec.sync_status() == pwdec.PWD_OK
    dec.close()
    meas, types = O.split_stream(R, wl.d, wl.W)
    ol, _ = O.forward_windows(meas, types, w, wl.d, wl.H)
    assert (np.abs(wlog.cpu().numpy() - ol) <= BF16_ATOL).all()
    assert int(bit.item()) == O.combine_bits(wbits.cpu().numpy())
