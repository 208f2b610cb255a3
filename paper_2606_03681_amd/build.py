"""Builds libtfmlayer.so (the C-ABI library of include/tfm_layer.h) for gfx950 with hipcc.

Every source under csrc/ is compiled for gfx950 only; objects go to _build/ at the repository
root and the shared library next to this file.  Always recompiles.

build(sanitize=True) builds a second copy whose host code (argument validation, plans, layouts,
launch sequences) carries AddressSanitizer and UndefinedBehaviorSanitizer checks, for CPU runs
of the host-side tests: _build/san/libtfmlayer_san.so, loaded by the binding when TFM_LIB names
it, in a process that preloads the sanitizer runtime (SAN_RUNTIME).  Device code is built as
usual.
"""

import concurrent.futures
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libtfmlayer.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # packed fp32 VALU forms are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in ordinary VGPRs, so softmax/epilogue arithmetic needs no AGPR copies
    "-mllvm", "-amdgpu-mfma-vgpr-form=1",
    "-Wall", "-Wno-unused-function",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


# attention kernels: no NaN reaches them (padding is never loaded), which lets max chains
# lower to v_max3_f32 without canonicalising moves
EXTRA = {"attn_item.hip": ["-fno-honor-nans"], "attn_item_bwd.hip": ["-fno-honor-nans"],
         "attn_feat.hip": ["-fno-honor-nans"]}


# host-only sanitizer flags (each applies to the host compilation only)
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
SAN_BUILD = os.path.join(BUILD, "san")
SAN_LIB = os.path.join(SAN_BUILD, "libtfmlayer_san.so")
# the clang runtime that the sanitized host code needs (preloaded into the process that loads it)
SAN_RUNTIME = os.path.join(os.path.dirname(os.path.dirname(HIPCC)), "llvm", "lib", "clang")


def san_runtime():
    """Path of the AddressSanitizer runtime (with the UndefinedBehaviorSanitizer handlers) of
    the compiler that builds the sanitized library."""
    found = sorted(glob.glob(os.path.join(SAN_RUNTIME, "*", "lib", "linux",
                                          "libclang_rt.asan-x86_64.so")))
    if not found:
        raise RuntimeError(f"no libclang_rt.asan-x86_64.so under {SAN_RUNTIME}")
    return found[-1]


def _compile(src, sanitize=False):
    out_dir = SAN_BUILD if sanitize else BUILD
    obj = os.path.join(out_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC] + FLAGS + (SAN_FLAGS if sanitize else []) + \
        EXTRA.get(os.path.basename(src), []) + ["-c", src, "-o", obj]
    if src.endswith(".hip"):
        cmd[1:1] = ["-x", "hip"]
    p = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(l for l in (p.stdout + p.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if p.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{msg}")
    return obj, msg


def build(verbose=False, sanitize=False):
    out_dir, lib = (SAN_BUILD, SAN_LIB) if sanitize else (BUILD, LIB)
    os.makedirs(out_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        results = list(ex.map(lambda src: _compile(src, sanitize), srcs))
    for obj, msg in results:
        if verbose and msg.strip():
            print(msg)
    tmp = lib + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + \
          (["-shared-libsan"] + SAN_FLAGS if sanitize else []) + [o for o, _ in results]
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError(f"linking failed:\n{p.stdout}\n{p.stderr}")
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv))
