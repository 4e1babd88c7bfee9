"""GPU parity of the (d+1)^2 token set (App. A.1.2: one token per cell of the stabilizer
array; cells without a stabilizer carry state but receive no detection events) against the
oracle's forward pass with grid=True: fp32 and bf16, the inference and recurrent branches
and stream decoding. Inputs and detection events stay one bit per stabilizer."""
import numpy as np
import pytest

from gpu_helpers import BF16_ATOL, FP32_ATOL, FP32_RTOL, check_bits, gpu_decode, gpu_events, say, to_device
from oracle import decoder as O
from paper_2601_09921_amd import pwdec, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BF16, F32 = synth.DTYPE_BF16, synth.DTYPE_F32
# (d, W, B, D, L, H, dtype)
SHAPES = [
    (3, 6, 9, 64, 2, 4, F32),       # 16 tokens
    (5, 10, 6, 128, 2, 8, BF16),    # 36 tokens
    (7, 14, 5, 128, 3, 8, BF16),    # 64 tokens: four whole blocks
    (11, 22, 3, 256, 2, 8, BF16),   # 144 tokens
    (25, 25, 2, 256, 1, 8, BF16),   # 676 tokens, 43 key blocks
    (33, 33, 1, 128, 1, 8, BF16),   # 1156 tokens, 73 key blocks: the largest grid that fits
]


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def within(g, o, dtype):
    if dtype == F32:
        return (np.abs(g - o) <= FP32_RTOL * np.abs(o) + FP32_ATOL).all()
    return (np.abs(g - o) <= BF16_ATOL).all()


@pytest.mark.parametrize("d,W,B,D,L,H,dtype", SHAPES, ids=[f"d{s[0]}_D{s[3]}" for s in SHAPES])
def test_grid_parity(d, W, B, D, L, H, dtype):
    wl = synth.Workload(f"g{d}", d, W, B, 0.05, 0.0, D, L, H, 4, dtype, grid=True)
    w = synth.make_weights(wl, seed=d + 100)
    meas, types = synth.make_windows(wl, seed=d + 200, realistic_boundaries=False)
    say(f"grid tokens d={d} W={W} B={B} D={D} dtype={dtype}")
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=B)
    o_logits, _, o_ev = O.forward_windows(meas, types, w, d, H, return_events=True, grid=True)
    if dtype == BF16:
        ev, rc = gpu_events(dec, meas, types, W, wl.words)
        assert rc == pwdec.PWD_OK and np.array_equal(ev, O.pack_bits(o_ev))
    logits, bits, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK
    say(f"  max |gpu - oracle| = {np.abs(logits - o_logits).max():.3e}")
    assert within(logits, o_logits, dtype), (logits, o_logits)
    check_bits(bits, o_logits)
    sub, _, _ = gpu_decode(dec, meas[1:], types[1:])
    assert np.array_equal(sub.view(np.uint32), logits[1:].view(np.uint32))
    # the token set matters: the logits are at least twice as close to the grid-token oracle
    # as to the stabilizer-token one
    stab, _ = O.forward_windows(meas, types, w, d, H)
    e_grid, e_stab = np.abs(logits - o_logits).max(), np.abs(logits - stab).max()
    say(f"  vs stabilizer tokens: {e_stab:.3e}")
    assert e_grid < 0.5 * e_stab
    dec.close()


@pytest.mark.parametrize("name,dtype", [("d3", F32), ("d7", BF16)])
def test_grid_recurrent(name, dtype):
    base = synth.WORKLOADS[name]
    wl = synth.Workload("g" + name, base.d, base.W, 4, 0.05, 0.0, base.D, base.L, base.H, 4, dtype, grid=True)
    w = synth.make_weights(wl, seed=7)
    meas, types = synth.make_windows(wl, seed=8, realistic_boundaries=False)
    say(f"grid recurrent {name}")
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=wl.B)
    meas_t, types_t = to_device(meas, types)
    logits = torch.full((wl.B, wl.d), float("nan"), dtype=torch.float32, device="cuda")
    bits = torch.full((wl.B, wl.d), 7, dtype=torch.uint8, device="cuda")
    dec.decode_recurrent(meas_t, types_t, logits, bits)
    torch.cuda.synchronize()
    assert dec.sync_status() == pwdec.PWD_OK
    dec.close()
    ol, _ = O.forward_windows_recurrent(meas, types, w, wl.d, wl.H, grid=True)
    assert within(logits.cpu().numpy(), ol, dtype)


def test_grid_stream():
    base = synth.WORKLOADS["d7"]
    wl = synth.Workload("gs7", base.d, base.W, 1, 0.01, 0.0, base.D, base.L, base.H, 4, BF16, grid=True)
    w = synth.make_weights(wl, seed=9)
    T = 6 * wl.d - 3
    m = -(-T // wl.d)
    R = synth.make_stream(wl.N, T, 0.01, seed=10)
    say(f"grid stream d7 T={T}")
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
    ol, obits = O.forward_windows(meas, types, w, wl.d, wl.H, grid=True)
    assert (np.abs(wlog.cpu().numpy() - ol) <= BF16_ATOL).all()
    assert int(bit.item()) == O.combine_bits(wbits.cpu().numpy())
