"""Host-side pieces of bench.py that need no GPU: the algorithmic FLOP counts the roofline
uses, the keying of the committed HBM-traffic record to the kernel sources, and the refusal
to run on more than one GPU."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2601_09921_amd import synth  # noqa: E402


def test_stage_flops_closed_forms():
    """Per real token and layer: Q/K/V 6 D^2, out-projection 2 D^2, feed-forward 4 D F,
    attention 4 N D (scores and weighted sum); the readout 8 d^2 D^2 + 2 d D per window."""
    wl = synth.WORKLOADS["d25"]
    B, N, D, F, d = 8192, wl.N, wl.D, wl.F, wl.d
    f, total = bench.stage_flops(wl, B)
    assert f["post_qkv"] == B * N * (8 * D * D + 4 * D * F)
    assert f["embed_qkv"] == B * N * 6 * D * D
    assert f["attention"] == B * 4 * N * N * D
    assert f["readout"] == B * (8 * d * d * D * D + 2 * d * D)
    assert total == B * (wl.W * wl.L * N * (8 * D * D + 4 * D * F + 4 * N * D)
                         + 8 * d * d * D * D + 2 * d * D)
    # 24 D^2 per token for post + QKV at F = 4 D: 1.573 MFLOP at D = 256
    assert f["post_qkv"] / (B * N) == 24 * D * D == 1572864


def test_traffic_record_is_keyed_to_the_sources(monkeypatch):
    t = json.load(open(bench.TRAFFIC_FILE))
    assert set(t) >= {"source_hashes", "fetch_scale", "write_scale", "bytes_per_launch"}
    assert set(t["source_hashes"]) == set(bench.STAGE_SOURCES)
    monkeypatch.setattr(bench, "source_hash", lambda stage=None: t["source_hashes"][stage])
    assert bench.load_traffic("post_qkv") == t["bytes_per_launch"].get("post_qkv")
    # another stage's kernel sources changing leaves this stage's record valid
    monkeypatch.setattr(bench, "source_hash",
                        lambda stage=None: t["source_hashes"][stage] if stage == "post_qkv" else "0" * 16)
    assert bench.load_traffic("post_qkv") == t["bytes_per_launch"].get("post_qkv")
    assert bench.load_traffic("attention") is None
    monkeypatch.setattr(bench, "source_hash", lambda stage=None: "0" * 16)
    assert bench.load_traffic("post_qkv") is None
    assert bench.load_traffic("readout") is None


def test_stage_hash_covers_the_kernel_sources(tmp_path, monkeypatch):
    """source_hash(stage) changes with every file of that stage's kernel and with no other."""
    import shutil
    csrc = os.path.join(ROOT, "paper_2601_09921_amd", "csrc")
    root = tmp_path / "r"
    shutil.copytree(csrc, root / "paper_2601_09921_amd" / "csrc")
    monkeypatch.setattr(bench, "ROOT", str(root))
    before = {k: bench.source_hash(k) for k in bench.STAGE_SOURCES}
    with open(root / "paper_2601_09921_amd" / "csrc" / "resident.hip", "a") as f:
        f.write("// edit\n")
    assert {k: bench.source_hash(k) for k in bench.STAGE_SOURCES} == before
    with open(root / "paper_2601_09921_amd" / "csrc" / "attn.hip", "a") as f:
        f.write("// edit\n")
    after = {k: bench.source_hash(k) for k in bench.STAGE_SOURCES}
    assert after["post_qkv"] == before["post_qkv"] and after["attention"] != before["attention"]


def test_attention_bound():
    """Exponentials per launch are one per score (H N^2 per window); the exponential peak is
    1024 SIMDs x 64 lanes per 8 cycles at 2.4 GHz; the two fractions add up."""
    wl = synth.WORKLOADS["d25"]
    st = {"kernel": "attn_kernel<32, 4>", "avg_ms": 4.0, "tflops": 800.0}
    b = bench.attention_bound(st, wl, wl.B, 2500.0)
    assert b["exp_per_launch"] == wl.B * 8 * 624 * 624
    assert abs(b["exp_peak_per_s"] - 19.6608e12) < 1e6
    assert abs(b["exp_frac"] - b["exp_per_launch"] / 4e-3 / 19.6608e12) < 1e-4
    assert b["mfma_frac"] == 0.32 and abs(b["sum"] - (b["mfma_frac"] + b["exp_frac"])) < 1e-4


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert "one GPU" in (r.stdout + r.stderr)
    assert not r.stdout.strip().startswith("{")


def test_transformer_block_fraction():
    """The transformer-block MFMA fraction sums the FLOPs of every launch of those stages over
    their summed time; the readout is not part of it."""
    import bench
    flops = {"attention": 2e12, "post_qkv": 3e12, "readout": 1e12}
    stages = {"attention": (4.0, 2), "post_qkv": (6.0, 2), "readout": (5.0, 1)}   # ms total, launches
    tb = bench.transformer_blocks(stages, flops, steps=1)
    assert tb["stages"] == ["attention", "post_qkv"]
    want = (2 * 2e12 + 2 * 3e12) / 10e-3 / 1e12
    assert abs(tb["tflops"] - want) < 0.1 and abs(tb["frac_of_bf16_peak"] - want / 2500) < 1e-4
