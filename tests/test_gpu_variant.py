"""The paper-shaped network exactly as bench.py times it (App. A model table: the (d+1)^2 token
set, the embedder's residual Conv1d block, feed-forward 5 d_model, three dilated convolutions
per layer, 3 layers; d_model 128) on the full d = 25 batch of 8192 windows: one window of each
type against the fp64 oracle, and two windows decoded alone against their rows of the batch,
bit for bit."""
import dataclasses

import numpy as np
import pytest

from gpu_helpers import BF16_ATOL, gpu_decode, say
from oracle import decoder as O
from paper_2601_09921_amd import pwdec, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_paper_variant_full_size_sampled():
    wl = synth.WORKLOADS["d25"]
    vwl = dataclasses.replace(wl, name=wl.name + "_paper", D=128, L=3, H=8, mlp_ratio=5, grid=True,
                              resnet=True, dil=(1, 2, 4))
    w = synth.make_weights(vwl)
    meas, types = synth.make_windows(wl)
    B = wl.B
    say(f"paper-shaped network d25 B={B}")
    dec = pwdec.Decoder.from_workload(vwl, w, max_windows=B)
    logits, bits, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK
    assert np.isfinite(logits).all() and np.array_equal(bits, (logits > 0).astype(np.uint8))
    for w_ in (B // 2 + 3, B - 1):
        one, _, _ = gpu_decode(dec, meas[w_:w_ + 1], types[w_:w_ + 1])
        assert one.view(np.uint32)[0] == logits.view(np.uint32)[w_], f"window {w_}"
    dec.close()
    sample = np.array([int(np.flatnonzero(types == t)[0]) for t in (0, 1, 2)])
    say(f"  oracle on windows {sample.tolist()}")
    ol, _ = O.forward_windows(meas[sample], types[sample], w, wl.d, vwl.H, grid=True)
    err = np.abs(logits[sample] - ol)
    say(f"  max |gpu - oracle| = {err.max():.3e}")
    assert (err <= BF16_ATOL).all(), (logits[sample], ol)
