"""The host half of libleech (csrc/host.cpp: codebook, expansion into the four
layouts, host decode, scale permutation, format-v1 index) built with g++ under
AddressSanitizer and UndefinedBehaviorSanitizer, driven over synthetic blocks
by tests/host_sanitize_driver.cpp: every round trip must hold, every documented
error must come back as its code, and the sanitizers must report nothing
(any report aborts the run)."""
import os
import shutil
import subprocess

import numpy as np
import pytest

from paper_2609_02652_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_02652_amd", "csrc")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not found")
    out = str(tmp_path_factory.mktemp("san") / "driver")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
           os.path.join(CSRC, "host.cpp"), os.path.join(ROOT, "tests", "host_sanitize_driver.cpp"),
           "-o", out, "-lpthread"]
    proc = subprocess.run(cmd, capture_output=True, text=True)
    assert proc.returncode == 0, proc.stderr[-3000:]
    return out


@pytest.mark.parametrize("M,K,seed", [(70, 24 * 33, 1), (257, 500, 2), (1, 24, 3)])
def test_host_entry_points_clean_under_sanitizers(driver, tmp_path, M, K, seed):
    inp = synth.make_gemv_inputs(M, K, seed=seed, name="sanitize")
    path = tmp_path / "blocks.bin"
    with open(path, "wb") as f:
        f.write(np.array([inp.M, inp.Kpad], dtype="<i8").tobytes())
        f.write(np.ascontiguousarray(inp.z, dtype=np.int8).tobytes())
        f.write(np.ascontiguousarray(inp.gain, dtype=np.uint8).tobytes())
        f.write(np.ascontiguousarray(inp.scale).view(np.uint16).tobytes())
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    proc = subprocess.run([driver, str(path)], capture_output=True, text=True, env=env,
                          timeout=300)
    assert proc.returncode == 0 and proc.stdout.startswith("ok"), \
        (proc.stdout[-2000:], proc.stderr[-4000:])
