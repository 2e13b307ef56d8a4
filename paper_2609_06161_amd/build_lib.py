"""Build ``libaf1.so`` (HIP kernels + C ABI) and ``libaf1_nabf.so`` (the NABF
building blocks) for gfx950 with hipcc.

Every call recompiles.  Objects go to ``_build/`` beside this file; the
shared library lands in the package directory, where the binding loads it.
"""
import concurrent.futures as cf
import glob
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libaf1.so")
NABF_LIB = os.path.join(HERE, "libaf1_nabf.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# -packed-fp32-ops: no packed fp32 VALU instructions in any kernel.
# kernarg preload: the first 16 argument dwords arrive in SGPRs at wave
# launch, saving a dependent memory round trip in latency-bound kernels.
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-mllvm", "-amdgpu-kernarg-preload-count=16",
         "-Wall", "-fvisibility=hidden", "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    p = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass warns that it does not know the packed-fp32 feature
    err = "\n".join(l for l in p.stderr.splitlines() if "packed-fp32-ops" not in l)
    if p.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip() and verbose:
        print(err)
    return obj


def _link(out: str, objs, libs, verbose: bool) -> None:
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", out + ".tmp", *objs, *libs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)


def build(verbose: bool = False) -> str:
    """Compile every source; link libaf1.so (the layer) and libaf1_nabf.so
    (the offline NABF building blocks, which also need rocBLAS and rocSOLVER
    and reuse the sign-packing kernel).  Returns the path of libaf1.so."""
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = dict(zip(srcs, ex.map(lambda s: _compile(s, verbose), srcs)))
    nabf_src = os.path.join(CSRC, "af1_nabf.hip")
    pack_src = os.path.join(CSRC, "af1_pack.hip")
    _link(LIB, [o for s, o in objs.items() if s != nabf_src], [], verbose)
    _link(NABF_LIB, [objs[nabf_src], objs[pack_src]],
          ["-L/opt/rocm/lib", "-lrocsolver", "-lrocblas"], verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
