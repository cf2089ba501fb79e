"""Host sanitizer runs (CPU): AddressSanitizer and UndefinedBehaviorSanitizer over
the C oracle and over the host code of the HIP library.

* The oracle is compiled with gcc and the sanitizers and driven through every
  step of the layer share on small seeded inputs and edge cases
  (`tests/sanitize/oracle_main.c`).
* Every library source is compiled with hipcc, the sanitizers on its host code
  only (the device code is built as usual), and linked with a driver that calls
  every entry point with arguments its validation must refuse and the
  workspace-size functions over a range of shapes (`tests/sanitize/abi_main.cpp`);
  none of those calls reaches the GPU.

A run that touches memory out of bounds, uses freed memory, leaks (oracle) or
performs undefined arithmetic ends with a sanitizer report and a non-zero exit.
"""
import concurrent.futures
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def _run(cmd, env=None, timeout=600):
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    assert r.returncode == 0, "%s\n%s\n%s" % (" ".join(cmd), r.stdout[-3000:], r.stderr[-3000:])
    return r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_address_and_undefined_behavior_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    _run(["gcc", "-O1", "-g", "-std=c99", "-fopenmp", "-fsanitize=address,undefined",
          "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
          os.path.join(ROOT, "oracle", "moe_oracle.c"), os.path.join(HERE, "oracle_main.c"),
          "-o", exe, "-lm"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", OMP_NUM_THREADS="4")
    assert "oracle sanitizer run: OK" in _run([exe], env=env)


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="needs hipcc")
def test_abi_validation_under_host_sanitizers(tmp_path):
    srcs = sorted(glob.glob(os.path.join(ROOT, "paper_2607_08782_amd", "csrc", "*.hip")))
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2607_08782_amd", "csrc")]
    common = [HIPCC, "-O1", "-g", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-Xclang",
              "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wno-pass-failed"] + SAN + inc

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        _run(common + ["-c", src, "-o", obj])
        return obj

    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, srcs + [os.path.join(HERE, "abi_main.cpp")]))
    exe = str(tmp_path / "abi_san")
    _run([HIPCC, "--offload-arch=gfx950"] + SAN + objs + ["-o", exe])
    # the HIP runtime keeps allocations until exit: leak checking is for the oracle run
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0")
    assert "abi sanitizer run: OK" in _run([exe], env=env)
