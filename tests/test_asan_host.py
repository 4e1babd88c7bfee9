"""The library's host code under AddressSanitizer (CPU only): configuration checks over a sweep
of geometries and dimensions, the weight-blob parser on a valid blob and on every truncation of
its header (and a spread of truncations of its payload) and on corrupted header words, and the
null-handle checks of every entry point (tests/asan/host_checks.cpp). The host code of
pwdec.cpp is compiled with -fsanitize=address for the host only; the device code is unchanged."""
import os
import shutil
import subprocess

import pytest

from paper_2601_09921_amd import build, pwdec, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("g++ is required")
    try:
        lib = build.build_host_asan()
    except RuntimeError as e:   # no ROCm toolchain
        pytest.skip(str(e))
    out = tmp_path_factory.mktemp("asan")
    exe = str(out / "host_checks")
    libdir = os.path.dirname(lib)
    subprocess.run(["g++", "-O1", "-g", "-fsanitize=address", "-fno-omit-frame-pointer",
                    os.path.join(ROOT, "tests", "asan", "host_checks.cpp"), "-o", exe, f"-L{libdir}",
                    "-lpwdec_asan", f"-Wl,-rpath,{libdir}"], check=True, capture_output=True)
    wl = synth.WORKLOADS["d3"]
    blob = out / "d3.blob"
    blob.write_bytes(pwdec.make_blob(wl.d, wl.W, wl.D, wl.L, wl.H, wl.F, wl.dtype, synth.make_weights(wl)))
    return lib, exe, str(blob)


def run(exe, *args):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0")
    return subprocess.run([exe, *args], capture_output=True, text=True, timeout=300, env=env)


def test_library_host_code_is_instrumented(checker):
    lib, _, _ = checker
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True, check=True).stdout
    assert "__asan_report_load" in syms


def test_host_checks_pass_under_address_sanitizer(checker):
    _, exe, blob = checker
    r = run(exe, blob)
    assert "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    assert r.returncode == 0, r.stdout + r.stderr[-4000:]
    assert "0 failures" in r.stdout
