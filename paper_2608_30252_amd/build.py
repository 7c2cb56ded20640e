"""Build libmad.so (HIP, gfx950) in-tree.

    python -m paper_2608_30252_amd.build            # the library
    python -m paper_2608_30252_amd.build --trace    # + libmad_trace.so, the diagnostic phase-trace build

Every translation unit in csrc/ is compiled by hipcc for gfx950 only and
linked into paper_2608_30252_amd/libmad.so.  Packed-fp32 instructions are
disabled for the device code (the compiler still emits ordinary fp32 math).
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libmad.so")
BUILD_DIR = os.path.join(HERE, "_build")
# the same sources with the kernels' phase marks compiled in (MAD_PHASE_TRACE):
# read by paper_2608_30252_amd/phase_trace.py, never by the product path
TRACE_LIB = os.path.join(HERE, "libmad_trace.so")
TRACE_BUILD_DIR = os.path.join(HERE, "_build", "trace")

ARCH = "gfx950"
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def build(verbose: bool = False, out: str = LIB, build_dir: str = BUILD_DIR, defines=()) -> str:
    os.makedirs(build_dir, exist_ok=True)
    cc = hipcc()
    common = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
              "-Wno-unused-function", "-I", os.path.join(HERE, "..", "include")] + DEVICE_FLAGS + \
             [f"-D{d}" for d in defines]

    def compile_one(src):
        obj = os.path.join(build_dir, os.path.basename(src) + ".o")
        cmd = [cc] + common + ["-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{err}")
        if err.strip() and verbose:
            print(err, flush=True)
        return obj

    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, sources()))
    tmp = out + ".tmp"
    cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build_trace(verbose: bool = False) -> str:
    return build(verbose, out=TRACE_LIB, build_dir=TRACE_BUILD_DIR, defines=("MAD_PHASE_TRACE",))


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
    print(LIB)
    if "--trace" in sys.argv:
        build_trace(verbose="-v" in sys.argv)
        print(TRACE_LIB)
