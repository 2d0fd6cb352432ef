"""Build libsq.so (host library + gfx950 HIP kernels) in-tree with hipcc.

Run ``python -m paper_2602_22603_amd.build_lib`` or call ``build()``.  Every
call compiles from source; the result is ``paper_2602_22603_amd/libsq.so``.
"""

from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys
import tempfile

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_PATH = os.path.join(PKG_DIR, "libsq.so")
SOURCES = ["store.cpp", "kv_kernels.hip", "decode_kernels.hip", "extend_kernels.hip"]
ARCH = "gfx950"

# Packed fp32 VALU instructions are kept out of every HIP object.
HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument", "-I", INCLUDE,
]


def _hipcc():
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found (ROCm toolchain required)")
    return path


# Per-source additions.  The extend kernels' softmax takes maxima of MFMA
# results, which are finite or -inf by construction: with NaN operands not
# honoured, each v_max_f32 needs no canonicalising copy of its inputs.
SOURCE_FLAGS = {"extend_kernels.hip": ["-fno-honor-nans"]}


def _compile(hipcc, src, obj):
    cmd = [hipcc, *HIP_FLAGS, *SOURCE_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    hipcc = _hipcc()
    with tempfile.TemporaryDirectory(prefix="sq_build_") as tmp:
        objs = [os.path.join(tmp, s + ".o") for s in SOURCES]
        with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
            list(ex.map(lambda so: _compile(hipcc, *so), zip(SOURCES, objs)))
        out_tmp = LIB_PATH + ".tmp"
        cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", out_tmp]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
        os.replace(out_tmp, LIB_PATH)
    if verbose:
        print(f"built {LIB_PATH}")
    return LIB_PATH


# Host-side checking build: the host library compiled by g++ with
# AddressSanitizer and UndefinedBehaviorSanitizer (the HIP sources as in the
# product build; no GPU code is sanitized).  Used by the CPU tests, which
# preload the sanitizer runtimes and drive the metadata-only store.
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-fno-sanitize-recover=all"]


def sanitizer_runtimes():
    """Paths of g++'s ASan and UBSan runtimes (for LD_PRELOAD)."""
    out = []
    for name in ("libasan.so", "libubsan.so"):
        res = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True)
        path = res.stdout.strip()
        if res.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
            raise RuntimeError(f"g++ has no {name}")
        out.append(path)
    return out


def build_sanitized(out_dir: str) -> str:
    """Build libsq_san.so in out_dir: store.cpp by g++ with the sanitizers,
    the kernel files by hipcc; returns its path."""
    hipcc = _hipcc()
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(hipcc)))
    objs = []
    for src in SOURCES:
        obj = os.path.join(out_dir, src + ".o")
        if src.endswith(".hip"):
            _compile(hipcc, src, obj)
        else:
            cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-D__HIP_PLATFORM_AMD__",
                   "-I", os.path.join(rocm, "include"), "-I", INCLUDE, *SAN_FLAGS,
                   "-c", os.path.join(CSRC, src), "-o", obj]
            res = subprocess.run(cmd, capture_output=True, text=True)
            if res.returncode != 0:
                raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
        objs.append(obj)
    out = os.path.join(out_dir, "libsq_san.so")
    cmd = ["g++", "-shared", *SAN_FLAGS, *objs, "-L", os.path.join(rocm, "lib"), "-lamdhip64",
           f"-Wl,-rpath,{os.path.join(rocm, 'lib')}", "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return out


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
