"""GPU parity of the HIP decoder against the fp64 oracle, through the C ABI.

Small batches (several token tiles and a ragged tail) compare every window; at the full
batch sizes of each workload, windows the oracle can afford are compared one by one and
the rest are checked through batch invariance and output consistency."""
import copy
import dataclasses
import ctypes
import math
import os

import numpy as np
import pytest

from gpu_helpers import (BF16_ATOL, spread_sample, check_bits, check_logits, decoder, gpu_decode, gpu_events,
                         inputs, oracle, say, weights)
from oracle import decoder as O
from paper_2601_09921_amd import pwdec, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

SMALL = {"d3": 64, "d7": 97, "d11": 13, "d17": 4, "d25": 3}


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pwdec.load_library()


@pytest.mark.parametrize("name", list(SMALL))
@pytest.mark.parametrize("realistic", [True, False])
def test_detection_events_bit_exact(name, realistic):
    wl = synth.WORKLOADS[name]
    B = max(SMALL[name], 6)
    meas, types = inputs(name, B, realistic)
    say(f"events {name} B={B} realistic={realistic}")
    dec = decoder(name, max(B, SMALL[name]))
    ev, rc = gpu_events(dec, meas, types, wl.W, wl.words)
    assert rc == pwdec.PWD_OK
    expect = O.pack_bits(O.detection_events(meas, types, wl.d))
    assert np.array_equal(ev, expect)


@pytest.mark.parametrize("name", list(SMALL))
def test_logits_match_oracle(name):
    B = SMALL[name]
    meas, types = inputs(name, B)
    say(f"decode {name} B={B}")
    logits, bits, rc = gpu_decode(decoder(name, B), meas, types)
    assert rc == pwdec.PWD_OK
    o_logits, o_bits, _ = oracle(name, B)
    check_logits(name, logits, o_logits)
    check_bits(bits, o_logits)
    assert np.array_equal(bits, (logits > 0).astype(np.uint8))


def test_d7_layer_phased_schedule():
    """The d7 network decodes with the state-resident schedule by default; the layer-phased one
    (one launch per layer and round) stays selectable and matches the oracle too, with the
    same batch invariance."""
    wl = synth.WORKLOADS["d7"]
    B = SMALL["d7"]
    meas, types = inputs("d7", B)
    dec = pwdec.Decoder.from_workload(wl, weights("d7"), max_windows=B)
    dec.schedule(pwdec.SCHEDULE_LAYERS)
    say(f"decode d7 B={B} layer-phased")
    logits, bits, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK
    o_logits, _, _ = oracle("d7", B)
    check_logits("d7", logits, o_logits)
    check_bits(bits, o_logits)
    one, _, _ = gpu_decode(dec, meas[B - 1:], types[B - 1:])
    assert one.view(np.uint32)[0] == logits.view(np.uint32)[B - 1]
    dec.close()


@pytest.mark.parametrize("name", ["d3", "d7", "d11"])
def test_masks_reach_the_network(name):
    """Windows whose padded rows hold random measurements decode like the oracle, which
    zeroes those events (App. A.1.1 boundary padding)."""
    B = min(SMALL[name], 12)
    meas, types = inputs(name, B, realistic=False)
    say(f"decode {name} B={B} random padding rows")
    logits, bits, rc = gpu_decode(decoder(name, SMALL[name]), meas, types)
    assert rc == pwdec.PWD_OK
    o_logits, _, _ = oracle(name, B, realistic=False)
    check_logits(name, logits, o_logits)


@pytest.mark.parametrize("name", ["d3", "d7", "d11", "d25"])
def test_batch_invariance_and_repeatability(name):
    B = SMALL[name]
    meas, types = inputs(name, B)
    dec = decoder(name, B)
    say(f"batch invariance {name} B={B}")
    full, fbits, _ = gpu_decode(dec, meas, types)
    again, _, _ = gpu_decode(dec, meas, types)
    assert np.array_equal(full.view(np.uint32), again.view(np.uint32))
    for w in sorted({0, B // 2, B - 1}):
        one, obits, _ = gpu_decode(dec, meas[w:w + 1], types[w:w + 1])
        assert one.view(np.uint32)[0] == full.view(np.uint32)[w], f"window {w}"
        assert obits[0] == fbits[w]
    perm = np.random.default_rng(0).permutation(B)
    pl, _, _ = gpu_decode(dec, meas[perm], types[perm])
    assert np.array_equal(pl.view(np.uint32), full[perm].view(np.uint32))


@pytest.mark.parametrize("name", ["d3", "d7", "d11"])
def test_zero_syndromes(name):
    B = 9
    meas, types = inputs(name, B, zero=True)
    say(f"zero syndromes {name}")
    logits, _, rc = gpu_decode(decoder(name, max(B, SMALL[name])), meas, types)
    assert rc == pwdec.PWD_OK
    for t in range(3):
        sel = logits[types == t]
        assert (sel.view(np.uint32) == sel.view(np.uint32)[0]).all()
    o_logits, _, _ = oracle(name, B, zero=True)
    check_logits(name, logits, o_logits)


DENSE_CASES = [("d3", 0.5), ("d3", 1.0), ("d7", 0.5), ("d7", 1.0), ("d11", 0.5), ("d11", 1.0), ("d25", 1.0)]


@pytest.mark.parametrize("name,p", DENSE_CASES, ids=[f"{n}_p{p}" for n, p in DENSE_CASES])
def test_dense_syndromes(name, p):
    """The other end from zero syndromes: every stabilizer flips with probability 1/2, or in
    every round (detection events in every unmasked position, 83 % of them), so the embedding
    and the recurrent state are far from the sparse regime of the workloads. Against the oracle
    (three windows at d25, one of each type), through the default schedule and, where the
    decoder has another, the layer-phased one."""
    wl = dataclasses.replace(synth.WORKLOADS[name], p=p, pair_p=0.0)
    B = 3 if name == "d25" else 6
    meas, types = synth.make_windows(wl, seed=77, B=B)
    o_logits, _ = O.forward_windows(meas, types, weights(name), wl.d, wl.H)
    dec = decoder(name, max(B, SMALL[name]))
    for schedule in (pwdec.SCHEDULE_AUTO, pwdec.SCHEDULE_LAYERS):
        try:
            dec.schedule(schedule)
        except pwdec.PwdError:
            continue
        say(f"dense syndromes {name} p={p} schedule={schedule}")
        logits, bits, rc = gpu_decode(dec, meas, types)
        assert rc == pwdec.PWD_OK
        check_logits(name, logits, o_logits)
        check_bits(bits, o_logits)
    dec.schedule(pwdec.SCHEDULE_AUTO)


@pytest.mark.parametrize("name", ["d3", "d7"])
def test_invalid_type_and_batch_limits(name):
    B = 6
    meas, types = inputs(name, B)
    dec = decoder(name, SMALL[name])
    bad = types.copy()
    bad[4] = 3
    say(f"invalid type {name}")
    logits, bits, rc = gpu_decode(dec, meas, bad)
    assert rc == pwdec.PWD_EDEVICE
    assert np.isnan(logits[4]) and bits[4] == 0
    good, _, _ = gpu_decode(dec, meas, types)
    ok = np.arange(B) != 4
    assert np.array_equal(logits[ok].view(np.uint32), good[ok].view(np.uint32))
    assert dec.sync_status() == pwdec.PWD_OK
    # n = 0 is a no-op; n > max_windows is refused before any launch, by the binding
    # (ValueError) and by the library itself (PWD_EBATCH through the raw ABI)
    wl = synth.WORKLOADS[name]
    z = torch.zeros(1, dtype=torch.float32, device="cuda")
    zb = torch.zeros(1, dtype=torch.uint8, device="cuda")
    mt = torch.zeros((0, wl.W + 1, wl.words), dtype=torch.int32, device="cuda")
    dec.decode(mt, torch.zeros(0, dtype=torch.uint8, device="cuda"), z, zb)
    big = SMALL[name] + 1
    mb = torch.zeros((big, wl.W + 1, wl.words), dtype=torch.int32, device="cuda")
    tb = torch.zeros(big, dtype=torch.uint8, device="cuda")
    with pytest.raises(ValueError):
        dec.decode(mb, tb, z, zb)
    vp = ctypes.c_void_p
    rc = dec._lib.decode_windows(dec._h, vp(mb.data_ptr()), vp(tb.data_ptr()), big, vp(z.data_ptr()),
                                 vp(zb.data_ptr()), vp(torch.cuda.current_stream().cuda_stream))
    assert rc == pwdec.PWD_EBATCH


def test_spread_sample_covers_xcds_and_the_tail():
    for B, k in ((8192, 3), (4096, 4), (4096, 13), (1024, 97)):
        sample = spread_sample(B, k)
        assert {w % 8 for w in sample} == set(range(8)) and sample[-2:] == [B - 2, B - 1]
        assert min(sample) >= k and max(np.diff(sample)) > B // 16


@pytest.mark.parametrize("name", ["d7", "d11", "d17", "d25"])
def test_full_batch_sampled(name):
    """The full batch of the workload, in the launch configuration the benchmark times: the
    leading windows and windows spread across the batch -- one per XCD residue, the last two
    (the final partial tiles) -- against the oracle; two more against a batch of one."""
    wl = synth.WORKLOADS[name]
    B = wl.B
    meas, types = inputs(name, B)
    dec = decoder(name, B)
    say(f"full batch {name} B={B}")
    logits, bits, rc = gpu_decode(dec, meas, types)
    assert rc == pwdec.PWD_OK
    assert np.isfinite(logits).all()
    assert np.array_equal(bits, (logits > 0).astype(np.uint8))
    k = SMALL[name]
    o_logits, _, _ = oracle(name, k)
    check_logits(name, logits[:k], o_logits)
    check_bits(bits[:k], o_logits)
    spread = spread_sample(B, k)
    say(f"  oracle on {len(spread)} spread windows")
    o_spread, _ = O.forward_windows(meas[spread], types[spread], weights(name), wl.d, wl.H)
    check_logits(name, logits[spread], o_spread)
    check_bits(bits[spread], o_spread)
    for w in (B // 3 + 1, B - 1):
        one, _, _ = gpu_decode(dec, meas[w:w + 1], types[w:w + 1])
        assert one.view(np.uint32)[0] == logits.view(np.uint32)[w], f"window {w}"


def constant_score_weights(wl, w, sign, beta=32.0):
    """Weights under which every attention score of every head is the same number, far outside
    the range the kernel exponentiates directly: Q of a head is the bias beta on the head's
    first feature (zero elsewhere), and K has exactly sign * beta on that feature (its column
    of Wk zeroed), whatever it holds on the others. So q'.k = sign * beta^2 log2(e)/sqrt(dh)
    for every pair (beta = 32: at least 184 log2 units for heads of 16 to 64 features), all
    scores of a row are equal and the softmax is uniform."""
    w = copy.deepcopy(w)
    dh = wl.D // wl.H
    for lw in w["layers"]:
        Wq, Wk, bq, bk = lw["Wq"].copy(), lw["Wk"].copy(), lw["bq"].copy(), lw["bk"].copy()
        for h in range(wl.H):
            f0, head = h * dh, slice(h * dh, (h + 1) * dh)
            Wq[:, head], bq[head] = 0.0, 0.0
            bq[f0] = beta
            Wk[:, f0], bk[f0] = 0.0, sign * beta
        lw["Wq"], lw["Wk"], lw["bq"], lw["bk"] = Wq, Wk, bq, bk
    return w


# (workload, B): heads of 16 (d7), 32 (d11) and 64 (d11 geometry, d_model 128, 2 heads)
RANGE_CASES = {
    "d7": (synth.WORKLOADS["d7"], 5),
    "d11": (synth.WORKLOADS["d11"], 5),
    "d11_dh64": (synth.Workload("d11_dh64", 11, 22, 3, 0.005, 0.0, 128, 2, 2, 4, synth.DTYPE_BF16), 3),
}


@pytest.mark.parametrize("sign", [1.0, -1.0], ids=["overflow", "underflow"])
@pytest.mark.parametrize("name", list(RANGE_CASES))
def test_attention_score_range(name, sign):
    """The attention kernel exponentiates the scores without a shift and recomputes a query
    block with a running maximum when its row sum or output leaves the normal fp32 range.
    With every score equal to +-(at least 184) log2 units, exp2 overflows to inf (sign +1) or
    underflows to 0 (sign -1) for every key: the results can only match the oracle's uniform
    softmax through the running-maximum path (head sizes 16, 32 and 64)."""
    wl, B = RANGE_CASES[name]
    base = weights(name) if name in synth.WORKLOADS else synth.make_weights(wl, seed=5)
    w = constant_score_weights(wl, base, sign)
    meas, types = synth.make_windows(wl, B=B, seed=6)
    # the scores on round 0, layer 0 (X = kappa * Embed(E_0)): one value per head, beyond the
    # exponent range of fp32 (and of bf16) in the direction of sign
    ev = O.detection_events(meas, types, wl.d)
    pe = O.positional_encoding((wl.d + 1) ** 2, wl.D)[O.grid_positions(wl.d)]
    X = w["kappa"] * O.embed(ev[:, 0, :], w, pe)
    lw = w["layers"][0]
    dh = wl.D // wl.H
    Q, K = X @ lw["Wq"] + lw["bq"], X @ lw["Wk"] + lw["bk"]
    for h in range(wl.H):
        sl = slice(h * dh, (h + 1) * dh)
        S = np.einsum("bnd,bmd->bnm", Q[:, :, sl], K[:, :, sl]) * math.log2(math.e) / math.sqrt(dh)
        assert np.all(S == S.flat[0]) and sign * S.flat[0] > 180, (h, S.flat[0])
    o_logits, _ = O.forward_windows(meas, types, w, wl.d, wl.H)
    dec = pwdec.Decoder.from_workload(wl, w, max_windows=B)
    # the layer-phased kernels, and for d7 the state-resident kernel (its own attention) too
    for schedule in [pwdec.SCHEDULE_LAYERS] + ([pwdec.SCHEDULE_RESIDENT] if name == "d7" else []):
        say(f"score range {name} sign={sign:+.0f} B={B} schedule={schedule}")
        dec.schedule(schedule)
        logits, bits, rc = gpu_decode(dec, meas, types)
        assert rc == pwdec.PWD_OK
        assert np.isfinite(logits).all()
        err = np.abs(logits - o_logits)
        say(f"  max |gpu - oracle| = {err.max():.3e}")
        assert (err <= BF16_ATOL).all(), (logits, o_logits)
        check_bits(bits, o_logits)
    dec.close()


def test_decoder_first_in_a_fresh_process():
    """A process whose first GPU work is creating a decoder (before any torch.cuda call) can
    decode: the binding starts torch's HIP runtime before the library's own calls."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("import numpy as np\n"
            "from paper_2601_09921_amd import pwdec, synth\n"
            "wl = synth.with_batch(synth.WORKLOADS['d7'], 4)\n"
            "dec = pwdec.Decoder.from_workload(wl, synth.make_weights(wl))\n"
            "import torch\n"
            "meas, types = synth.make_windows(wl)\n"
            "m = torch.from_numpy(np.ascontiguousarray(synth.pack_bits(meas)).view(np.int32)).cuda()\n"
            "t = torch.from_numpy(types).cuda()\n"
            "lg = torch.empty(4, device='cuda'); bt = torch.empty(4, dtype=torch.uint8, device='cuda')\n"
            "dec.decode(m, t, lg, bt); torch.cuda.synchronize()\n"
            "assert torch.isfinite(lg).all()\n"
            "print('ok')\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=110)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stderr[-2000:]
