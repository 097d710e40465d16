"""CPU sanitizer runs: the oracle and the host side of the C ABI under
AddressSanitizer and UndefinedBehaviorSanitizer.

- The oracle (plain C) is built with gcc and both sanitizers together with
  a driver that calls every oracle entry point on tiny models, each buffer
  allocated at its exact documented size, so any read or write past one is
  reported (tests/sanitize/oracle_driver.c).
- The library's HIP sources are built with the sanitizers on the host side
  only (device code is compiled but never launched: no GPU is used), and a
  driver calls the host paths that never reach the device: validation of
  every entry point, every configuration rejection of buddy_model_create,
  the prior normalisation and the budget helper
  (tests/sanitize/abi_driver.cpp).
Both sanitizers abort the run on the first finding, so a zero exit status
and the driver's last line mean a clean run.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CSRC = os.path.join(ROOT, "paper_2606_09514_amd", "csrc")
HIP_SOURCES = ["api.hip", "k_route.hip", "k_gemv.hip", "k_attn.hip", "k_mfma.hip", "k_gemm.hip",
               "prior.hip"]
# host-side sanitizers on every hipcc line (each flag behind -Xarch_host)
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="abort_on_error=0:halt_on_error=1",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")


def run(cmd, env=None, cwd=None):
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, cwd=cwd)
    assert r.returncode == 0, f"{cmd[0]} exited {r.returncode}:\n{r.stdout}\n{r.stderr[-4000:]}"
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_address_and_ub_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    run(["gcc", "-std=c11", "-g", "-O1", "-fno-omit-frame-pointer", "-ffp-contract=off",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-Wno-unknown-pragmas",
         os.path.join(SAN, "oracle_driver.c"), os.path.join(ROOT, "oracle", "buddy_oracle.c"),
         "-o", exe, "-lm"])
    r = run([exe], env=ENV)
    assert r.stdout.strip().endswith("oracle driver ok"), r.stdout


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_abi_host_code_under_address_and_ub_sanitizers(tmp_path):
    objs, procs = [], []
    for src in HIP_SOURCES:
        obj = str(tmp_path / (src + ".o"))
        objs.append(obj)
        procs.append(subprocess.Popen(
            [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
             "-Xarch_device", "-O0", "-Xarch_device", "-g0", *HOST_SAN,
             "-c", os.path.join(CSRC, src), "-o", obj],
            stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True))
    for p in procs:
        out, _ = p.communicate()
        assert p.returncode == 0, out[-4000:]
    drv = str(tmp_path / "abi_driver.o")
    run([HIPCC, "-O1", "-g", "-std=c++17", *HOST_SAN, "-c",
         os.path.join(SAN, "abi_driver.cpp"), "-o", drv])
    exe = str(tmp_path / "abi_driver")
    run([HIPCC, "--offload-arch=gfx950", *HOST_SAN[:4], *objs, drv, "-o", exe])
    # the HIP runtime's own allocations at exit are not the library's
    env = dict(ENV, ASAN_OPTIONS=ENV["ASAN_OPTIONS"] + ":detect_leaks=0")
    r = run([exe], env=env)
    assert r.stdout.strip().endswith("abi driver ok"), r.stdout
