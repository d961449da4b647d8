"""The CPU oracle and the library's host logic (launch planners, page
allocator, estimator) built with AddressSanitizer and UndefinedBehaviorSanitizer
and run on randomised inputs.  CPU only: the drivers launch no kernel."""
import concurrent.futures
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2504_14489_amd", "csrc")
# host pass only: hipcc takes each -fsanitize option behind -Xarch_host
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def _run(exe, env_extra):
    env = dict(os.environ, **env_extra)
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0 and res.stdout.strip().endswith("ok"), res.stdout[-2000:] + res.stderr[-4000:]


def test_oracle_under_sanitizers(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_driver")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-pthread", "-o", exe,
                           os.path.join(ROOT, "oracle", "mw_oracle.c"), os.path.join(HERE, "oracle_driver.c"),
                           "-lm"])
    _run(exe, {"ASAN_OPTIONS": "detect_leaks=1"})


def test_library_host_logic_under_sanitizers(tmp_path):
    hipcc = "/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else shutil.which("hipcc")
    if not hipcc:
        pytest.skip("hipcc not found")
    from paper_2504_14489_amd import build as hb
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"] + HOST_SAN + inc
    srcs = hb.SOURCES + ["../../tests/sanitize/host_logic.cpp"]

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src).rsplit(".", 1)[0] + ".o"))
        res = subprocess.run([hipcc] + flags + ["-c", os.path.normpath(os.path.join(CSRC, src)), "-o", obj],
                             capture_output=True, text=True)
        assert res.returncode == 0, res.stderr[-3000:]
        return obj

    with concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(compile_one, srcs))
    exe = str(tmp_path / "host_logic")
    res = subprocess.run([hipcc, "--offload-arch=gfx950"] + HOST_SAN + objs + ["-o", exe],
                         capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-3000:]
    # the HIP runtime the library links keeps allocations for the process's
    # lifetime; the drivers' own leaks are covered by the oracle run
    _run(exe, {"ASAN_OPTIONS": "detect_leaks=0"})
