"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the
CPU: the fp64 attention oracle (tests/sanitize/oracle_driver.c linked with
oracle/attn_oracle.c) and the library's C ABI validation and host helpers
(tests/sanitize/abi_driver.c linked with the four library sources, their
host parts instrumented).  Each driver exits non-zero on a failed check, and
a sanitizer report aborts it."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2504_17577_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN_ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr[-4000:]}"
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    run(["gcc", "-std=c11", "-g", "-O1", "-Wall", "-Wextra", "-Werror",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-o", exe,
         os.path.join(HERE, "oracle_driver.c"), os.path.join(ROOT, "oracle", "attn_oracle.c"),
         "-lm", "-lpthread"])
    r = run([exe], env=SAN_ENV, timeout=300)
    assert "all checks passed" in r.stdout


# The driver calls every entry point with fake device addresses and arguments
# that must fail validation; on a machine with a GPU a wrong expectation would
# launch a kernel on those addresses, so it runs only where there is none.
@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="fake-pointer cases run only without a GPU")
@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_abi_validation_under_asan_ubsan(tmp_path):
    # host parts instrumented (every sanitizer flag behind -Xarch_host); the
    # device parts are compiled as usual and never run
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
             "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include"), "-I", CSRC]
    objs, procs = [], []
    for name in ("attn_fwd", "mla_decode", "gemm", "ssd"):
        obj = str(tmp_path / f"{name}.o")
        objs.append(obj)
        procs.append(subprocess.Popen([HIPCC, *flags, "-c", os.path.join(CSRC, f"{name}.hip"),
                                       "-o", obj], stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                                      text=True))
    for p in procs:
        out, err = p.communicate(timeout=900)
        assert p.returncode == 0, err[-4000:]
    drv = str(tmp_path / "abi_driver.o")
    run(["gcc", "-std=c11", "-g", "-O1", "-Wall", "-Werror", "-fsanitize=address,undefined",
         "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"), "-c",
         os.path.join(HERE, "abi_driver.c"), "-o", drv])
    exe = str(tmp_path / "abi_driver")
    run([HIPCC, "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
         "-o", exe, drv, *objs])
    # the HIP runtime's own allocations at load time are not this library's
    env = dict(SAN_ENV, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    r = run([exe], env=env, timeout=300)
    assert "all checks passed" in r.stdout
