"""The host runtime (validation, segment chains, query expansion, schedule sizing, forest
preprocessing) built with AddressSanitizer and UndefinedBehaviorSanitizer on the host side only,
driven by random valid and malformed inputs (tests/host/sanitize_driver.cpp).  No GPU: every
call stops at its first device allocation, after the host logic has run."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_18954_amd", "csrc")
HIPCC = "/opt/rocm/bin/hipcc"


def test_host_runtime_under_sanitizers(tmp_path):
    if not os.path.exists(HIPCC) or shutil.which("g++") is None:
        pytest.skip("no hipcc")
    exe = tmp_path / "sanitize_driver"
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer"]
    srcs = [os.path.join(CSRC, "api.cpp"), os.path.join(CSRC, "equiv_api.cpp"),
            os.path.join(ROOT, "tests", "host", "sanitize_driver.cpp")]
    objs = []
    for src in srcs:
        obj = tmp_path / (os.path.basename(src) + ".o")
        cmd = [HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", *san,
               "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-c", src, "-o", str(obj)]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-3000:]
        objs.append(str(obj))
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", *san, *objs, "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", HIP_VISIBLE_DEVICES="")
    r = subprocess.run([str(exe), "300"], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and "ok" in r.stdout, (r.stdout + r.stderr)[-4000:]
