"""Build libneo.so (HIP kernels for gfx950 + the C-ABI and planner) in-tree.

    python -m paper_1809_02697_amd.build

Each source is compiled to an object file in parallel, then linked into
``paper_1809_02697_amd/libneo.so``.  Packed-FP32 instructions are disabled
for all device code."""
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libneo.so")
ARCH = "gfx950"
SOURCES = ["conv.hip", "conv_xy.hip", "conv_group.hip", "conv_pair.hip", "layout.hip", "pool.hip", "dense.hip", "api.cpp", "plan.cpp", "tune.cpp",
           "search.cpp", "noalloc.hip", "conv_pool.hip", "conv_stream.hip", "winograd.hip", "conv_int8.hip"]
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function", "-Wno-unused-command-line-argument"]
# Per-source additions.  The integer kernels keep their MFMA accumulators in
# ordinary VGPRs: with the default AGPR form the compiler rotated them through
# accumulator-register copies inside the reduction loop (v_accvgpr_mov).
SOURCE_FLAGS = {"conv_int8.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]}


def _compile(src, objdir):
    obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
    cmd = ["hipcc", "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj] + FLAGS + \
        SOURCE_FLAGS.get(src, [])
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    warn = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l
                     and "not a recognized feature" not in l and l.strip())
    return obj, warn


def build(verbose=True):
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
        res = list(ex.map(lambda s: _compile(s, objdir), SOURCES))
    objs = [o for o, _ in res]
    for _, w in res:
        if w and verbose:
            print(w, file=sys.stderr)
    tmp = OUT + ".tmp%d" % os.getpid()
    cmd = ["hipcc", "-shared", f"--offload-arch={ARCH}", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build())
