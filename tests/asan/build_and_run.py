"""Build the library's host code with AddressSanitizer against the stand-in
HIP runtime and run the host checks (tests/asan/host_checks.cpp).

Product sources are compiled exactly as shipped, host side only
(``--cuda-host-only``; the sanitizer applies to host code only); the fat
binary symbols the host objects reference are defined empty, since nothing
runs on a device here.  Usage: ``python tests/asan/build_and_run.py OUTDIR``.
Returns the checks' exit status; prints their output.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2607_16074_amd", "csrc")
SOURCES = ["jn_api.cpp", "k_pack.hip", "k_norm.hip", "k_gemm.hip", "k_attn.hip", "k_heads.hip", "k_expert.hip",
           "k_optim.hip"]
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
CLANG = "/opt/rocm/llvm/bin/clang++"
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"{' '.join(cmd)}\n{r.stderr[-4000:]}")
    return r.stdout


def build(out: str) -> str:
    os.makedirs(out, exist_ok=True)
    inc = [f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]

    def product(src):
        obj = os.path.join(out, os.path.splitext(src)[0] + ".o")
        _run([HIPCC, "-x", "hip", "--offload-arch=gfx950", "--cuda-host-only", "-O1", "-g", "-std=c++17",
              "-Wno-unused-result", "-Wno-unused-value"] + SAN + inc + ["-c", os.path.join(CSRC, src), "-o", obj])
        return obj

    def plain(src, extra=()):
        obj = os.path.join(out, os.path.splitext(os.path.basename(src))[0] + ".o")
        _run([CLANG, "-O1", "-g", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include"] + list(extra) +
             ["-fsanitize=address", "-fno-omit-frame-pointer"] + inc + ["-c", src, "-o", obj])
        return obj

    with cf.ThreadPoolExecutor(8) as ex:
        objs = list(ex.map(product, SOURCES))
    objs.append(plain(os.path.join(HERE, "fake_hip_runtime.cpp")))
    objs.append(plain(os.path.join(HERE, "host_checks.cpp")))
    # empty definitions of the fat binaries the host objects name
    undef = _run(["nm", "-u"] + objs)
    fat = sorted(set(re.findall(r"\b(__hip_fatbin_[0-9a-f]+)\b", undef)))
    stub = os.path.join(out, "fatbins.cpp")
    with open(stub, "w") as f:
        f.write("".join(f'extern "C" {{ char {n}[8] = {{0}}; }}\n' for n in fat))
    objs.append(plain(stub))
    exe = os.path.join(out, "host_checks")
    _run([CLANG, "-fsanitize=address", "-o", exe] + objs + ["-lpthread"])
    return exe


def main() -> int:
    out = sys.argv[1] if len(sys.argv) > 1 else os.path.join(ROOT, "_build_asan")
    exe = build(out)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env)
    sys.stdout.write(r.stdout)
    sys.stderr.write(r.stderr[-6000:])
    return r.returncode


if __name__ == "__main__":
    sys.exit(main())
