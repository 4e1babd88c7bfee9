"""decode_windows_noalloc (the entry point for callers that cannot allocate) against
decode_windows on the same decoder, through the C ABI: identical logits and bits, on two
calls in a row with the second batch smaller, for the plain bf16 network, the dilated
convolutions (whose two extra buffers also live in the fixed scratch), the fp32 path, and the
capacity limit at the d=25 network."""

import numpy as np
import pytest

from gpu_helpers import say, to_device
from paper_2601_09921_amd import pwdec, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def run(dec, fn, meas, types):
    meas_t, types_t = to_device(meas, types)
    n = types.shape[0]
    logits = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
    bits = torch.full((n,), 7, dtype=torch.uint8, device="cuda")
    getattr(dec, fn)(meas_t, types_t, logits, bits)
    torch.cuda.synchronize()
    assert dec.sync_status() == pwdec.PWD_OK
    return logits.cpu().numpy(), bits.cpu().numpy()


CASES = [
    # name, workload, batch
    ("d7", synth.WORKLOADS["d7"], 200),
    ("d5_dilated", synth.Workload("c5", 5, 10, 9, 0.05, 0.0, 128, 2, 8, 4, synth.DTYPE_BF16, grid=True,
                                  dil=(1, 2, 4)), 9),
    ("d3_fp32", synth.WORKLOADS["d3"], 64),
    ("d25", synth.WORKLOADS["d25"], 12),
]


@pytest.mark.parametrize("name,wl,B", CASES, ids=[c[0] for c in CASES])
def test_noalloc_equals_decode_windows(name, wl, B):
    w = synth.make_weights(wl, seed=wl.d + 77)
    meas, types = synth.make_windows(wl, B=B, seed=wl.d + 78, realistic_boundaries=False)
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=B)
    for n in (B, max(1, B // 3)):   # two calls in a row, the second smaller
        say(f"noalloc {name} n={n}")
        ref_l, ref_b = run(dec, "decode", meas[:n], types[:n])
        got_l, got_b = run(dec, "decode_noalloc", meas[:n], types[:n])
        assert np.isfinite(got_l).all()
        assert np.array_equal(got_l.view(np.uint32), ref_l.view(np.uint32)), name
        assert np.array_equal(got_b, ref_b)
    dec.close()


def test_noalloc_refuses_batches_beyond_its_scratch():
    """At d=25 (624 tokens, d_model 256) the fixed scratch holds 68 windows: 69 is refused with
    PWD_EBATCH before any launch, and 68 decodes like decode_windows."""
    wl = synth.WORKLOADS["d25"]
    w = synth.make_weights(wl)
    B = 69
    meas, types = synth.make_windows(wl, B=B, seed=5)
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=B)
    meas_t, types_t = to_device(meas, types)
    logits = torch.zeros(B, dtype=torch.float32, device="cuda")
    bits = torch.zeros(B, dtype=torch.uint8, device="cuda")
    with pytest.raises(pwdec.PwdError) as e:
        dec.decode_noalloc(meas_t, types_t, logits, bits)
    assert e.value.code == pwdec.PWD_EBATCH
    say("noalloc d25 68 windows")
    ref_l, _ = run(dec, "decode", meas[:68], types[:68])
    got_l, _ = run(dec, "decode_noalloc", meas[:68], types[:68])
    assert np.array_equal(got_l.view(np.uint32), ref_l.view(np.uint32))
    dec.close()
