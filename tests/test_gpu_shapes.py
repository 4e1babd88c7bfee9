"""GPU parity beyond the five benchmark workloads: other code distances (token padding to a
multiple of 16 at every size), the paper's window of 3d rounds (b = c = d, Sec. 3.1), and
both head sizes at d_model 128 and 256. Small seeded batches against the fp64 oracle."""
import numpy as np
import pytest

from gpu_helpers import BF16_ATOL, check_bits, gpu_decode, gpu_events, say
from oracle import decoder as O
from paper_2601_09921_amd import pwdec, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BF16 = synth.DTYPE_BF16
# (d, W, B, D, L, H): every odd d not among the benchmark workloads, two window lengths,
# d_model 128 / 256 with head sizes 16 / 32
SHAPES = [
    (5, 10, 7, 128, 2, 8),      # N=24 -> 32 tokens, dh 16
    (5, 15, 5, 256, 1, 8),      # W = 3d
    (9, 18, 5, 128, 2, 4),      # N=80, dh 32
    (13, 26, 4, 256, 2, 8),     # N=168 -> 176
    (15, 45, 3, 128, 1, 8),     # N=224, W = 3d
    (19, 38, 3, 256, 1, 8),     # N=360 -> 368
    (21, 42, 3, 128, 1, 4),     # N=440 -> 448, dh 32
    (23, 23, 3, 256, 1, 8),     # N=528, W = d (no buffers)
    (7, 21, 6, 128, 3, 8),      # d7 network with the paper's W = 3d
]


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("d,W,B,D,L,H", SHAPES, ids=[f"d{s[0]}_W{s[1]}_D{s[3]}_H{s[5]}" for s in SHAPES])
def test_shape_parity(d, W, B, D, L, H):
    wl = synth.Workload(f"d{d}", d, W, B, 0.02, 0.0, D, L, H, 4, BF16)
    w = synth.make_weights(wl, seed=d + W)
    meas, types = synth.make_windows(wl, seed=77 + d, realistic_boundaries=False)
    say(f"shape d={d} W={W} B={B} D={D} L={L} H={H}")
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=B)
    ev, rc = gpu_events(dec, meas, types, W, wl.words)
    assert rc == pwdec.PWD_OK
    o_logits, _, o_ev = O.forward_windows(meas, types, w, d, H, return_events=True)
    assert np.array_equal(ev, O.pack_bits(o_ev))
    logits, bits, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK
    err = np.abs(logits - o_logits)
    say(f"  max |gpu - oracle| = {err.max():.3e}")
    assert (err <= BF16_ATOL).all(), (logits, o_logits)
    check_bits(bits, o_logits)
    # a smaller batch on the same handle gives the same bits for the same windows
    sub, _, _ = gpu_decode(dec, meas[1:], types[1:])
    assert np.array_equal(sub.view(np.uint32), logits[1:].view(np.uint32))
    dec.close()
