"""Build the partition's HIP library (libgp.so) in-tree for gfx950.

Each .hip source is compiled to an object with hipcc, in parallel, then all
are linked into paper_1811_06965_amd/_lib/libgp.so; then the C-ABI test
program (tests/host/abi_driver.cpp) is linked against it.  Always recompiles.
"""
import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(HERE, "_lib")
BUILD_DIR = os.path.join(HERE, "_build")
LIB = os.path.join(OUT_DIR, "libgp.so")
ARCH = "gfx950"

FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # keep the compiler from emitting packed fp32 arithmetic
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
]


def hipcc():
    for c in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


# Per-source additions.  The attention kernels post-process every MFMA result
# with vector ALU work (exp, the softmax and dS arithmetic, packing to bf16);
# with the accumulators in AGPRs each value costs a v_accvgpr_read first, so
# their MFMAs write ordinary VGPRs instead (the register file is unified on
# gfx950).
EXTRA_FLAGS = {"attention_mfma.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def _compile(cc, src):
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [cc, *FLAGS, *EXTRA_FLAGS.get(os.path.basename(src), []), "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj, r.stderr


def build(verbose=False):
    cc = hipcc()
    os.makedirs(OUT_DIR, exist_ok=True)
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sources()
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        results = list(ex.map(lambda s: _compile(cc, s), srcs))
    if verbose:
        for _, err in results:
            if err.strip():
                print(err, file=sys.stderr)
    tmp = LIB + ".tmp"
    cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + [o for o, _ in results]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    # A kernel template whose host-side instantiation fails is dropped without a
    # diagnostic, leaving its launch stub undefined in the shared library; catch
    # that here rather than at the first launch.
    nm = shutil.which("nm")
    if nm:
        r = subprocess.run([nm, "-DC", "--undefined-only", tmp], capture_output=True, text=True)
        bad = [l for l in r.stdout.splitlines() if "gp::" in l]
        if bad:
            raise RuntimeError("libgp.so has undefined internal symbols:\n" + "\n".join(bad[:20]))
    os.replace(tmp, LIB)
    build_abi_driver(cc)
    return LIB


# The test program that drives a partition through the C ABI alone (no Python
# in its process); it links the library through a path relative to itself.
DRIVER_SRC = os.path.join(os.path.dirname(HERE), "tests", "host", "abi_driver.cpp")
DRIVER = os.path.join(os.path.dirname(HERE), "tests", "host", "_bin", "abi_driver")


def build_abi_driver(cc=None):
    cc = cc or hipcc()
    os.makedirs(os.path.dirname(DRIVER), exist_ok=True)
    rel = os.path.relpath(OUT_DIR, os.path.dirname(DRIVER))
    cmd = [cc, *FLAGS, DRIVER_SRC, "-o", DRIVER + ".tmp", f"-L{OUT_DIR}", "-lgp", f"-Wl,-rpath,$ORIGIN/{rel}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(DRIVER + ".tmp", DRIVER)
    return DRIVER


if __name__ == "__main__":
    print(build(verbose=True))
