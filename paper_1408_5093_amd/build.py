"""Build ``libcaffe_conv.so`` (the gfx950 HIP kernels and their C ABI) in-tree.

Every source under ``csrc/`` is compiled by ``hipcc --offload-arch=gfx950``
into ``_build/`` and linked into ``paper_1408_5093_amd/libcaffe_conv.so``.
The library is linked against the HIP runtime that PyTorch loads (when
PyTorch is importable), so that PyTorch's streams and device memory are
valid handles inside the library.

Run ``python -m paper_1408_5093_amd.build`` or call :func:`build`.
"""
import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libcaffe_conv.so")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result",
    # gfx950 packed-fp32 VALU ops are kept out of every kernel
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", CSRC, "-I", INCLUDE,
]


# Per-source extra flags.  The implicit-GEMM kernels keep their MFMA
# accumulators in VGPRs: occupancy counts VGPRs + AGPRs together, and the
# VGPR form avoids a bulk AGPR -> VGPR copy before the fused ReLU epilogue.
EXTRA = {
    "conv_gemm.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
    "conv_wgrad.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
    "conv_bf16.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
}


def _sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))


def _headers():
    return sorted(glob.glob(os.path.join(CSRC, "*.h")) + glob.glob(os.path.join(INCLUDE, "*.h")))


def _torch_lib_dir():
    try:
        import torch  # noqa: F401
    except Exception:
        return None
    d = os.path.join(os.path.dirname(torch.__file__), "lib")
    return d if os.path.exists(os.path.join(d, "libamdhip64.so")) else None


def _compile(src, verbose):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC] + CFLAGS + EXTRA.get(os.path.basename(src), []) + ["-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l and "not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{msg}")
    if msg.strip() and verbose:
        print(msg, flush=True)
    return obj


def build(verbose: bool = False, jobs: int = 8) -> str:
    """Compile every HIP source for gfx950 and link the shared library."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = _sources()
    with cf.ThreadPoolExecutor(max_workers=max(1, min(jobs, len(srcs)))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs))
    tmp = LIB + ".tmp%d" % os.getpid()
    link = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    tdir = _torch_lib_dir()
    if tdir:
        link += ["-L", tdir, "-Wl,-rpath," + tdir]
    link += ["-lamdhip64"]
    if verbose:
        print(" ".join(link), flush=True)
    r = subprocess.run(link, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    return LIB


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(f) > t for f in _sources() + _headers())


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
