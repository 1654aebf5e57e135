"""Host AddressSanitizer / UndefinedBehaviorSanitizer builds, run on the CPU:
the fp64 oracle (tests/sanitize/oracle_driver.c calls every oracle function
on small and degenerate shapes) and the library's argument validation
(tests/sanitize/abi_driver.c calls every C entry point with arguments that
must be refused before anything is enqueued, and the size queries over many
shapes).  The library's kernel objects are the ones the regular build made;
only the host code of the ABI sources is rebuilt with the sanitizers, on the
host pass of hipcc (the device code is never instrumented)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2502_10940_amd", "csrc")
BUILD = os.path.join(ROOT, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _check(res):
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert "driver: ok" in res.stdout, out[-4000:]


def test_oracle_under_asan_ubsan(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc missing")
    exe = tmp_path / "oracle_san"
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", *SAN, "-fopenmp", os.path.join(HERE, "oracle_driver.c"),
                    os.path.join(ROOT, "oracle", "cola_oracle.c"), "-o", str(exe), "-lm"], check=True)
    _check(subprocess.run([str(exe)], capture_output=True, text=True, env=ENV, timeout=300))


def test_abi_validation_under_asan_ubsan(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc missing")
    from paper_2502_10940_amd import build as B
    kernels = [s for s in B.SOURCES if s not in ("cola_abi.hip", "block_abi.hip", "gemm_dispatch.hip")]
    objs = [os.path.join(BUILD, os.path.splitext(s)[0] + ".o") for s in kernels]
    if not all(os.path.exists(o) for o in objs):
        B.build()
    host_flags = []
    for f in SAN:
        host_flags += ["-Xarch_host", f]
    san_objs = []
    for src in ("cola_abi.hip", "block_abi.hip", "gemm_dispatch.hip"):
        o = str(tmp_path / (os.path.splitext(src)[0] + ".san.o"))
        subprocess.run([HIPCC, *B.FLAGS, "-O1", "-g", *host_flags, "-c", os.path.join(CSRC, src), "-o", o],
                       check=True, capture_output=True)
        san_objs.append(o)
    drv = str(tmp_path / "abi_driver.o")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", *SAN, "-I", os.path.join(ROOT, "include"), "-c",
                    os.path.join(HERE, "abi_driver.c"), "-o", drv], check=True)
    exe = str(tmp_path / "abi_san")
    subprocess.run([HIPCC, f"--offload-arch={B.ARCH}", *SAN, drv, *san_objs, *objs, "-o", exe], check=True,
                   capture_output=True)
    _check(subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=300))
