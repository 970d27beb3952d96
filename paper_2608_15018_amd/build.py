"""Build libs2moe.so for gfx950 with hipcc (in-tree, no JIT cache).

    python -m paper_2608_15018_amd.build                   # the library
    python -m paper_2608_15018_amd.build --host-sanitize   # + ASan/UBSan host layer
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libs2moe.so")
SOURCES = ["api.cpp", "route.hip", "gate.hip", "ffn.hip", "ffn_bf16.hip", "ffn_q4.hip", "combine.hip", "pack.hip", "probe.hip", "expand.hip", "noalloc.hip"]
ARCH = "gfx950"
ROCM_INC = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
# Packed fp32 VALU instructions are switched off for all device code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-I", INCLUDE, "-I", CSRC,
          "-Wall", "-Wno-unused-function"]


def _compile(src: str, objdir: str = OBJDIR, defines=()) -> str:
    out = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *COMMON, *DEVICE_FLAGS, *defines, "-c", os.path.join(CSRC, src), "-o", out]
    if src.endswith(".cpp"):
        cmd = [HIPCC, *COMMON, "-x", "c++", "-D__HIP_PLATFORM_AMD__=1", "-I", ROCM_INC, *defines,
               "-c", os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{msg}")
    if msg.strip():
        print(msg, file=sys.stderr)
    return out


def build(verbose: bool = True, out: str = LIB, objdir: str = OBJDIR, defines=()) -> str:
    """Compile every source and link libs2moe.so; returns its path.  `defines`
    (e.g. ["-DS2MOE_STAGE_STEPS=8"]) override tuning constants."""
    os.makedirs(objdir, exist_ok=True)
    with ThreadPoolExecutor(min(len(SOURCES), os.cpu_count() or 1)) as ex:
        objs = list(ex.map(lambda src: _compile(src, objdir, list(defines)), SOURCES))
    tmp = out + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}{r.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}")
    return out


# Host-side checking build: the C-ABI layer (argument validation, workspace
# arithmetic, struct marshalling) compiled by g++ with AddressSanitizer and
# UndefinedBehaviorSanitizer, linked with the regular device objects.  The
# kernels are not instrumented (no device sanitizer is used).  Load it with
# the ASan runtime first in LD_PRELOAD (host_sanitizer_env) and point
# S2MOE_LIBRARY at it.
SAN_LIB = os.path.join(OBJDIR, "libs2moe_hostsan.so")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
             "-fno-omit-frame-pointer"]


def build_host_sanitized(verbose: bool = True) -> str:
    """Build SAN_LIB (builds the regular objects first if any is missing)."""
    objs = [os.path.join(OBJDIR, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    if not all(os.path.exists(o) for o in objs):
        build(verbose)
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    api_obj = os.path.join(OBJDIR, "api_hostsan.o")
    cc = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", *SAN_FLAGS, "-D__HIP_PLATFORM_AMD__=1",
          "-I", ROCM_INC, "-I", INCLUDE, "-I", CSRC, "-c", os.path.join(CSRC, "api.cpp"),
          "-o", api_obj]
    link = ["g++", "-shared", *SAN_FLAGS, api_obj, *[o for o in objs if not o.endswith("api.o")],
            "-L", os.path.join(rocm, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(rocm, "lib"),
            "-o", SAN_LIB]
    for cmd in (cc, link):
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"sanitized build failed:\n{' '.join(cmd)}\n{r.stdout}{r.stderr}")
    if verbose:
        print(f"built {SAN_LIB}")
    return SAN_LIB


def host_sanitizer_env(env=None) -> dict:
    """Environment that loads SAN_LIB under the ASan runtime.  The runtime is
    put first in LD_PRELOAD, ahead of whatever the environment already
    preloads."""
    env = dict(os.environ if env is None else env)
    asan = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True,
                          text=True, check=True).stdout.strip()
    env["LD_PRELOAD"] = asan + (":" + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    env["S2MOE_LIBRARY"] = SAN_LIB
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    return env


if __name__ == "__main__":
    if "--host-sanitize" in sys.argv[1:]:
        build_host_sanitized()
    else:
        build()
