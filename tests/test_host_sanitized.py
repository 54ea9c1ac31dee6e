"""The runtime's host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

tests/host_check.cpp is built with the host compiler together with the library's
host-only source (paper_2605_31464_amd/csrc/host.cpp: configuration checks, the batch
planner, the weight-file parser) and every sanitizer finding aborts it.  It runs the
planner on random batches against a direct restatement, and the weight-file parser on
files written by synth.write_weight_file and on corrupted copies of them.
"""
import os
import shutil
import subprocess

import pytest

from paper_2605_31464_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2605_31464_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs the host C++ compiler")
def test_host_code_is_clean_under_sanitizers(tmp_path):
    exe = tmp_path / "host_check"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
           "-I", CSRC, os.path.join(ROOT, "tests", "host_check.cpp"), os.path.join(CSRC, "host.cpp"),
           "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    files = []
    for name, kw in (("tiny", {}), ("small", {"n_layers": 3, "vocab": 256, "d_ff": 256}),
                     ("7b", {"n_layers": 1, "vocab": 64, "d_ff": 256, "d_model": 256,
                             "n_q_heads": 2, "n_kv_heads": 1})):
        shape = synth.CONFIGS[name].shape.replace(**kw)
        p = tmp_path / f"{name}.surw"
        synth.write_weight_file(p, shape, synth.make_weights(shape))
        files.append(str(p))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe), *files], capture_output=True, text=True, env=env, timeout=600)
    print(r.stdout, r.stderr[-4000:])
    assert r.returncode == 0, r.stderr[-4000:]
    assert "host check ok" in r.stdout
