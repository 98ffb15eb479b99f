"""Compile the gfx950 HIP sources into the in-tree shared library libsaturn.so.

Usage: python -m paper_2309_01226_amd.build   (or call build()).
       python -m paper_2309_01226_amd.build --asan   (host code under AddressSanitizer)
"""

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OUT = os.path.join(PKG, "libsaturn.so")
BUILD_DIR = os.path.join(ROOT, "_build")

SOURCES = ["gemm.hip", "gemm256.hip", "norm.hip", "elementwise.hip", "attention.hip", "attn256.hip", "attn_small.hip", "conv.hip", "ops_abi.cpp", "model.cpp",
           "step.cpp", "resnet.cpp", "abi.cpp", "profile.cpp"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
COMMON = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"), "-Wno-unused-result",
]


# Per-source code-generation options.  The 256-wide attention kernels keep
# their O / dK / dV accumulators and the resident Q / K / V operands live for
# the whole key loop; MFMA results in VGPRs avoid whole-accumulator copies
# between the two register files on every iteration.
EXTRA = {"attn256.hip": ["-mllvm", "--amdgpu-mfma-vgpr-form"]}


def _compile(src):
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [HIPCC] + COMMON + EXTRA.get(src, []) + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {src}\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def _stale(src):
    """True when the object of `src` is older than the source or any header."""
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    if not os.path.exists(obj):
        return True
    deps = [os.path.join(CSRC, src)] + [os.path.join(CSRC, h) for h in os.listdir(CSRC) if h.endswith(".h")]
    deps += [os.path.join(ROOT, "include", h) for h in os.listdir(os.path.join(ROOT, "include"))]
    return max(os.path.getmtime(p) for p in deps) > os.path.getmtime(obj)


def build(verbose=True, incremental=False):
    """Compile every source (incremental=True: only those whose object is
    older than the source or a header) and link libsaturn.so."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    todo = [s for s in SOURCES if _stale(s)] if incremental else SOURCES
    with cf.ThreadPoolExecutor(max_workers=max(1, min(8, len(todo)))) as ex:
        list(ex.map(_compile, todo))
    objs = [os.path.join(BUILD_DIR, os.path.basename(s) + ".o") for s in SOURCES]
    tmp = OUT + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, OUT)
    if verbose:
        print(f"built {OUT}")
    return OUT


# Host translation units (argument checks, arena planning, launch sequences):
# the AddressSanitizer build instruments these for host code only; the
# device code objects of every source are the regular ones.
HOST_SOURCES = [s for s in SOURCES if s.endswith(".cpp")]
ASAN_DIR = os.path.join(BUILD_DIR, "asan")
ASAN_OUT = os.path.join(ASAN_DIR, "libsaturn_asan.so")
ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]


def asan_runtime():
    """Path of the compiler's shared AddressSanitizer runtime (to preload)."""
    r = subprocess.run([HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                       text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


def build_asan(verbose=True):
    """Link ASAN_OUT: the host sources compiled with AddressSanitizer (host
    side only), the .hip sources' regular objects.  Loaded by a process that
    preloads asan_runtime(), for host-only checks of the C ABI."""
    build(verbose=False, incremental=True)
    os.makedirs(ASAN_DIR, exist_ok=True)

    def one(src):
        obj = os.path.join(ASAN_DIR, src + ".o")
        cmd = ([HIPCC] + COMMON + ASAN_FLAGS + EXTRA.get(src, []) +
               ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj])
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"compile failed: {src}\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
        return obj

    with cf.ThreadPoolExecutor(max_workers=max(1, min(8, len(HOST_SOURCES)))) as ex:
        list(ex.map(one, HOST_SOURCES))
    objs = [os.path.join(ASAN_DIR if s in HOST_SOURCES else BUILD_DIR, os.path.basename(s) + ".o")
            for s in SOURCES]
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", "-shared-libasan"] + ASAN_FLAGS[:2] + \
        ["-o", ASAN_OUT] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed\n{r.stdout}\n{r.stderr}")
    if verbose:
        print(f"built {ASAN_OUT}")
    return ASAN_OUT


if __name__ == "__main__":
    if "--asan" in sys.argv:
        build_asan()
    else:
        build(incremental="--incremental" in sys.argv)
    sys.exit(0)
