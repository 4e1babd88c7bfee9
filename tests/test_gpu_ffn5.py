"""GPU parity of the feed-forward width 5 d_model (App. A model table; mlp_ratio = 5) against
the fp64 oracle, whose feed-forward block takes its width from the weights: fp32 and bf16 at
d_model 128 and 256, both token sets, the inference and recurrent branches. The token kernel
is compiled per width (40 hidden-unit chunks of 32 at d_model 256, 10 of 64 at 128)."""
import numpy as np
import pytest

from gpu_helpers import BF16_ATOL, FP32_ATOL, FP32_RTOL, check_bits, gpu_decode, gpu_events, say, to_device
from oracle import decoder as O
from paper_2601_09921_amd import pwdec, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BF16, F32 = synth.DTYPE_BF16, synth.DTYPE_F32
# (d, W, B, D, L, H, dtype, grid)
SHAPES = [
    (3, 6, 9, 64, 2, 4, F32, False),
    (3, 6, 9, 32, 2, 2, F32, True),
    (5, 10, 7, 128, 2, 8, BF16, False),
    (7, 14, 5, 128, 3, 8, BF16, True),
    (11, 22, 4, 256, 2, 8, BF16, False),
    (13, 26, 3, 256, 1, 4, BF16, True),    # head size 64
    (25, 25, 2, 256, 1, 8, BF16, False),   # the d = 25 network with the model table's width
    (35, 35, 1, 128, 1, 8, BF16, False),   # 1224 tokens, 77 key blocks
]


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def within(g, o, dtype):
    if dtype == F32:
        return (np.abs(g - o) <= FP32_RTOL * np.abs(o) + FP32_ATOL).all()
    return (np.abs(g - o) <= BF16_ATOL).all()


def workload(d, W, B, D, L, H, dtype, grid):
    return synth.Workload(f"f5d{d}", d, W, B, 0.03, 0.0, D, L, H, 5, dtype, grid=grid)


@pytest.mark.parametrize("d,W,B,D,L,H,dtype,grid", SHAPES,
                         ids=[f"d{s[0]}_D{s[3]}_{'f32' if s[6] == F32 else 'bf16'}{'_grid' if s[7] else ''}"
                              for s in SHAPES])
def test_ffn5_parity(d, W, B, D, L, H, dtype, grid):
    wl = workload(d, W, B, D, L, H, dtype, grid)
    assert wl.F == 5 * D
    w = synth.make_weights(wl, seed=d + 500)
    assert w["layers"][0]["W1"].shape == (D, 5 * D)
    meas, types = synth.make_windows(wl, seed=d + 600, realistic_boundaries=False)
    say(f"ffn 5D d={d} W={W} B={B} D={D} L={L} H={H} dtype={dtype} grid={grid}")
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


@pytest.mark.parametrize("d,W,B,D,L,H,dtype,grid", [SHAPES[0], SHAPES[3], SHAPES[4]],
                         ids=["d3_f32", "d7_bf16_grid", "d11_bf16"])
def test_ffn5_recurrent(d, W, B, D, L, H, dtype, grid):
    wl = workload(d, W, B, D, L, H, dtype, grid)
    w = synth.make_weights(wl, seed=d + 700)
    meas, types = synth.make_windows(wl, seed=d + 800, realistic_boundaries=False)
    say(f"ffn 5D recurrent d={d} D={D} dtype={dtype} grid={grid}")
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
