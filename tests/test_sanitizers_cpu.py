"""Host AddressSanitizer / UndefinedBehaviorSanitizer builds (CPU only):
the oracle on small inputs through every entry point and option path, and the
HIP library's host code (argument checks, the workspace cap) through its C
ABI.  Device code is compiled as usual; only the host side is instrumented."""
import glob
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")


def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_san")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", *SAN, "-ffp-contract=off",
                           os.path.join(ROOT, "oracle", "mpq_oracle.c"),
                           os.path.join(HERE, "oracle_main.c"), "-o", exe, "-lm"])
    p = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=300)
    assert p.returncode == 0 and "sanitized oracle: ok" in p.stdout, p.stdout + p.stderr


def test_library_host_code_under_asan_ubsan(tmp_path):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    srcs = sorted(glob.glob(os.path.join(ROOT, "paper_2002_09049_amd", "csrc", "*.hip")))
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2002_09049_amd", "csrc")]
    # host-side sanitizers only: each -fsanitize applies to the host pass
    host_san = [f for s in SAN for f in ("-Xarch_host", s)]
    flags = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *host_san, *inc]

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        subprocess.run([hipcc, *flags, "-c", src, "-o", obj], check=True, capture_output=True)
        return obj

    with ThreadPoolExecutor(min(8, len(os.sched_getaffinity(0)))) as ex:
        objs = list(ex.map(compile_one, srcs + [os.path.join(HERE, "abi_main.cpp")]))
    exe = str(tmp_path / "abi_san")
    # objects only on the link line (a source there would make hipcc read
    # every later input as HIP source)
    subprocess.run([hipcc, "--offload-arch=gfx950", *host_san, *objs, "-o", exe], check=True,
                   capture_output=True)
    p = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=300)
    assert p.returncode == 0 and "sanitized ABI checks: ok" in p.stdout, p.stdout + p.stderr
