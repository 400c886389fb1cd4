"""Sanitizer builds on the host (no GPU): the CPU oracle and the C ABI's
host-side validation, each compiled with AddressSanitizer and
UndefinedBehaviorSanitizer (any report aborts) and driven by a small program
under tests/sanitize/ that exercises valid, padded and invalid inputs."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANGXX = "/opt/rocm/llvm/bin/clang++"


def _run(cmd, env=None, timeout=300):
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    return r.returncode, r.stdout + r.stderr


def _clean(out):
    return "AddressSanitizer" not in out and "runtime error" not in out and "LeakSanitizer" not in out


def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_san")
    rc, out = _run(["gcc", "-O1", "-g", "-std=gnu11", "-fopenmp", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                    os.path.join(ROOT, "oracle", "gdn_oracle.c"), os.path.join(SAN, "oracle_driver.c"),
                    "-o", exe, "-lm"])
    assert rc == 0, out
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", OMP_NUM_THREADS="2")
    rc, out = _run([exe], env=env)
    assert rc == 0 and "0 failed checks" in out and _clean(out), out


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANGXX)), reason="needs hipcc")
def test_abi_host_validation_under_asan_ubsan(tmp_path):
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2607_06763_amd", "csrc")]
    # the sanitizers apply to the host pass only
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-Xarch_host", "-fsanitize=address",
             "-Xarch_host", "-fsanitize=undefined"]
    objs = []
    for src, lang in ((os.path.join(ROOT, "paper_2607_06763_amd", "csrc", "gdn_abi.hip"), []),
                      (os.path.join(SAN, "abi_driver.cpp"), ["-x", "hip"])):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        rc, out = _run([HIPCC, *flags, *inc, "-c", *lang, src, "-o", obj])
        assert rc == 0, out
        objs.append(obj)
    exe = str(tmp_path / "abi_san")
    rc, out = _run([CLANGXX, "-fsanitize=address,undefined", *objs, "-L/opt/rocm/lib", "-lamdhip64",
                    "-Wl,-rpath,/opt/rocm/lib", "-o", exe])
    assert rc == 0, out
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    rc, out = _run([exe], env=env)
    assert rc == 0 and "0 failed checks" in out and _clean(out), out
