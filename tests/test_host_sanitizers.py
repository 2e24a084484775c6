"""The library's host code (plan validation, the storage writer, commit,
chain and reader) under AddressSanitizer and UndefinedBehaviorSanitizer:
tests/native/sanitize_driver.cpp is built with the sanitizers on the host
code only (device code as usual) and run with no GPU visible."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_00455_amd", "csrc")
SOURCES = ["dte_api.hip", "extract.hip", "remap.hip", "store.hip"]
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize-recover=all"]


def hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    return None


@pytest.mark.skipif(hipcc() is None, reason="hipcc not available")
def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    flags = ["--offload-arch=gfx950", "-O1", "-fno-omit-frame-pointer", "-Xclang",
             "-target-feature", "-Xclang", "-packed-fp32-ops", "-I" + CSRC,
             "-I" + os.path.join(ROOT, "include")] + SAN
    objs, procs = [], []
    srcs = [os.path.join(ROOT, "tests", "native", "sanitize_driver.cpp")] + \
        [os.path.join(CSRC, s) for s in SOURCES]
    for src in srcs:
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        objs.append(obj)
        procs.append(subprocess.Popen([hipcc()] + flags + ["-c", src, "-o", obj],
                                      stdout=subprocess.PIPE, stderr=subprocess.STDOUT))
    for p in procs:
        out = p.communicate(timeout=600)[0]
        assert p.returncode == 0, out.decode()[-2000:]
    exe = str(tmp_path / "driver")
    link = subprocess.run([hipcc()] + flags + objs + ["-ldl", "-o", exe],
                          capture_output=True, text=True, timeout=300)
    assert link.returncode == 0, link.stderr[-2000:]
    env = dict(os.environ, HIP_VISIBLE_DEVICES="", ROCR_VISIBLE_DEVICES="",
               ASAN_OPTIONS="detect_leaks=1:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe, str(tmp_path / "store")], capture_output=True, text=True,
                       timeout=300, env=env)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "ok (0 failures)" in r.stdout
