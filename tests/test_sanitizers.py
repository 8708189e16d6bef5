"""AddressSanitizer and UndefinedBehaviorSanitizer builds (CPU only):

* the oracle (oracle/vecattn_ref.cpp), driven through every entry point by
  tests/sanitize/oracle_main.cpp;
* the library's host code -- the C ABI's argument checks and queries, the
  per-head filter-ratio programme and the launch set-up up to the first HIP
  call -- driven by tests/sanitize/api_main.cpp (no GPU: calls with valid
  arguments must report VECATTN_ERR_DEVICE).

The HIP sources are compiled with the sanitizers on their host side only
(-Xarch_host); the device code is built as usual.  Any invalid access or
undefined operation aborts the driver.
"""
import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_2603_29494_amd.build import SOURCES

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2603_29494_amd", "csrc")
INC = os.path.join(ROOT, "include")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang++")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all"]


def run(cmd, cwd):
    r = subprocess.run(cmd, cwd=cwd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "not a recognized feature" not in l)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{out[-4000:]}"
    return out


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    run(["g++", "-std=c++17", "-O1", "-g", "-fopenmp"] + SAN +
        [os.path.join(ROOT, "tests", "sanitize", "oracle_main.cpp"),
         os.path.join(ROOT, "oracle", "vecattn_ref.cpp"), "-o", exe], str(tmp_path))
    out = run([exe], str(tmp_path))
    assert out.strip().endswith("ok"), out


@pytest.mark.skipif(not (os.path.exists(HIPCC) and os.path.exists(CLANG)),
                    reason="ROCm compilers not available")
def test_host_api_under_sanitizers(tmp_path):
    d = str(tmp_path)
    inc = ["-I" + INC, "-I" + CSRC]
    jobs = []
    for src in ("vecattn_api.cpp", "plan.cpp"):
        jobs.append([CLANG, "-std=c++17", "-O1", "-g", "-D__HIP_PLATFORM_AMD__",
                     "-I" + os.path.join(ROCM, "include")] + inc + SAN +
                    ["-c", os.path.join(CSRC, src), "-o", src + ".o"])
    hip_srcs = [s for s in SOURCES if s.endswith(".hip")]
    for src in hip_srcs:
        jobs.append([HIPCC, "-x", "hip", "--offload-arch=gfx950", "-std=c++17", "-O1", "-g",
                     "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"] + inc +
                    HOST_SAN + ["-c", os.path.join(CSRC, src), "-o", src + ".o"])
    jobs.append([CLANG, "-std=c++17", "-O1", "-g"] + inc + SAN +
                ["-c", os.path.join(ROOT, "tests", "sanitize", "api_main.cpp"), "-o", "api_main.o"])
    with ThreadPoolExecutor(max_workers=8) as ex:
        list(ex.map(lambda c: run(c, d), jobs))
    objs = ["api_main.o", "vecattn_api.cpp.o", "plan.cpp.o"] + [s + ".o" for s in hip_srcs]
    run([HIPCC, "--offload-arch=gfx950"] + HOST_SAN[:4] + objs + ["-o", "api_san"], d)
    out = run([os.path.join(d, "api_san")], d)
    assert out.strip().endswith("ok"), out
