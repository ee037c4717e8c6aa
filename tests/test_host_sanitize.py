"""CPU-only sanitizer build of the host validators of the C ABI
(paper_2608_22526_amd/csrc/host_check.cpp, the checks behind
rs3_bank_import and rs3_track_import): the validators and a fuzz driver
(tests/host_fuzz.cpp) are compiled with the host compiler under the address
and undefined-behaviour sanitizers and run on malformed snapshots and tracker
states (no GPU, no HIP)."""
import os
import shutil
import subprocess

import pytest

from conftest import ROOT


def _cxx():
    return shutil.which("g++") or shutil.which("c++")


@pytest.mark.parametrize("seed", [1, 2])
def test_host_validators_under_sanitizers(tmp_path, seed):
    cxx = _cxx()
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = tmp_path / "host_fuzz"
    csrc = os.path.join(ROOT, "paper_2608_22526_amd", "csrc")
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-I", csrc, os.path.join(ROOT, "tests", "host_fuzz.cpp"),
           os.path.join(csrc, "host_check.cpp"), "-o", str(exe)]
    subprocess.check_call(cmd)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    p = subprocess.run([str(exe), "20000", str(seed)], stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True,
                       env=env, timeout=300)
    print(p.stdout)
    assert p.returncode == 0, p.stderr[-4000:]
    assert "ok" in p.stdout.split()
