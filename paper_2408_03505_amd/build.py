"""Build the HIP library liboptimus_enc.so in-tree for gfx950.

    python -m paper_2408_03505_amd.build
    python -m paper_2408_03505_amd.build --host-sanitized   (host-only check build)

Every .hip file under csrc/ is compiled to an object with hipcc and every
.cpp file (host-only code) with the host C++ compiler, in parallel, and all
are linked into paper_2408_03505_amd/liboptimus_enc.so.  It always
recompiles: the build is the "does it compile" check as well as the product.
"""

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OBJ = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "liboptimus_enc.so")

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
CXX = os.environ.get("CXX", shutil.which("g++") or "c++")
CXXFLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", f"-I{os.path.join(ROOT, 'include')}"]
CFLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # keep the compiler from forming packed fp32 ops (v_pk_*_f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{os.path.join(ROOT, 'include')}",
]


def _compile(src):
    obj = os.path.join(OBJ, os.path.basename(src) + ".o")
    if src.endswith(".cpp"):
        cmd = [CXX, *CXXFLAGS, "-c", src, "-o", obj]
    else:
        cmd = [HIPCC, *CFLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{r.stdout}\n{r.stderr}")
    return obj


# Host-only build of the C-ABI layer under AddressSanitizer and
# UndefinedBehaviorSanitizer: api.hip (host code only) and the kernel packer,
# linked against stand-in launchers (csrc/host_check), with the host compiler
# alone -- no device code is built or run.  Used by the CPU test suite.
SAN_DIR = os.path.join(OBJ, "host_san")
SAN_LIB = os.path.join(SAN_DIR, "liboptimus_enc_host_san.so")
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def build_host_sanitized(verbose=True):
    os.makedirs(SAN_DIR, exist_ok=True)
    srcs = [(os.path.join(CSRC, "api.hip"), ["-x", "c++"]),
            (os.path.join(CSRC, "scheduler.cpp"), []),
            (os.path.join(CSRC, "host_check", "stub_launchers.cpp"), [])]
    inc = ["-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{os.path.join(ROOT, 'include')}"]
    objs = []
    for src, lang in srcs:
        obj = os.path.join(SAN_DIR, os.path.basename(src) + ".o")
        cmd = [CXX, *lang, "-std=c++17", "-fPIC", "-Wall", *inc, *SAN_FLAGS, "-c", src, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"compiling {src} failed:\n{r.stdout}\n{r.stderr}")
        objs.append(obj)
    r = subprocess.run([CXX, "-shared", *SAN_FLAGS, "-o", SAN_LIB, *objs], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    if verbose:
        print(f"built {SAN_LIB}")
    return SAN_LIB


def build(verbose=True):
    os.makedirs(OBJ, exist_ok=True)
    srcs = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    if "--host-sanitized" in sys.argv[1:]:
        build_host_sanitized()
    else:
        build()
    sys.exit(0)
