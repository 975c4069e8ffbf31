"""Build libtts.so (HIP for gfx950) in-tree.

    python -m paper_2509_00195_amd.build          # or __graft_entry__.build()

Every HIP translation unit is compiled with packed-fp32 instruction
selection disabled (``-target-feature -packed-fp32-ops``) and matrix
instructions in their VGPR form (``-amdgpu-mfma-vgpr-form``).
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libtts.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]

# -amdgpu-mfma-vgpr-form: matrix instructions accumulate in VGPRs. With
# AGPR accumulators the attention kernel's pair loops copied every tile's
# accumulators back into place at each branch join (hundreds of
# v_accvgpr_mov per loop iteration); in VGPR form they accumulate in place.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-mllvm", "-amdgpu-mfma-vgpr-form=1"]

SOURCES_HIP = ["tts_kernels.hip", "tts_kv.hip"]
SOURCES_HOST = ["tts_meta.cpp", "tts_plan.cpp", "tts_alloc.cpp", "tts_sched.cpp", "tts_api.cpp"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd)}")
    return r


def build(verbose: bool = False, out: str = LIB, defines=()) -> str:
    """Compile every source and link libtts.so (or ``out``); returns its path.

    ``defines`` adds preprocessor definitions (tuning builds only)."""
    with tempfile.TemporaryDirectory(prefix="tts_build_") as tmp:
        objs = []
        for src in SOURCES_HIP:
            obj = os.path.join(tmp, src + ".o")
            _run([HIPCC, *COMMON, *[f"-D{d}" for d in defines], *DEVICE, "-c", os.path.join(CSRC, src), "-o", obj])
            objs.append(obj)
        for src in SOURCES_HOST:
            obj = os.path.join(tmp, src + ".o")
            _run([HIPCC, *COMMON, *[f"-D{d}" for d in defines], "-c", os.path.join(CSRC, src), "-o", obj])
            objs.append(obj)
        out_tmp = os.path.join(tmp, "libtts.so")
        _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", out_tmp])
        shutil.copyfile(out_tmp, out + ".tmp")
        os.replace(out + ".tmp", out)
    if verbose:
        print(f"built {out}")
    return out


SANITIZE = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g", "-O1"]


def build_sanitized(out: str, verbose: bool = False) -> str:
    """A CPU-test build of the library: the host sources (metadata, planner,
    scheduler, allocation search, C ABI) compiled by g++ with AddressSanitizer
    and UndefinedBehaviorSanitizer, the HIP sources compiled as usual (their
    kernels are not run by the host tests). Load it with the ASan runtime
    preloaded (``g++ -print-file-name=libasan.so``)."""
    gxx = os.environ.get("CXX_HOST", "g++")
    host_flags = ["-std=c++17", "-fPIC", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                  f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}", *SANITIZE]
    with tempfile.TemporaryDirectory(prefix="tts_san_") as tmp:
        objs = []
        for src in SOURCES_HIP:
            obj = os.path.join(tmp, src + ".o")
            _run([HIPCC, *COMMON, *DEVICE, "-c", os.path.join(CSRC, src), "-o", obj])
            objs.append(obj)
        for src in SOURCES_HOST:
            obj = os.path.join(tmp, src + ".o")
            _run([gxx, *host_flags, "-c", os.path.join(CSRC, src), "-o", obj])
            objs.append(obj)
        out_tmp = os.path.join(tmp, "libtts_san.so")
        _run([gxx, "-shared", "-fPIC", *SANITIZE, *objs, "-L/opt/rocm/lib", "-lamdhip64",
              "-Wl,-rpath,/opt/rocm/lib", "-o", out_tmp])
        shutil.copyfile(out_tmp, out + ".tmp")
        os.replace(out + ".tmp", out)
    if verbose:
        print(f"built {out}")
    return out


if __name__ == "__main__":
    build(verbose=True)
