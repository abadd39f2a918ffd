"""Compile libfgq.so (all HIP sources under csrc/) for gfx950 with hipcc.

Each source is compiled to an object in parallel, then linked into one
shared library next to this file.  Always recompiles (no timestamp logic).
"""
import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
BUILD_CHECK = os.path.join(HERE, "_build_check")
LIB = os.path.join(HERE, "libfgq.so")
LIB_CHECK = os.path.join(HERE, "libfgq_check.so")
ARCH = "gfx950"

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    # Packed fp32 instructions stay off: some of their forms have given wrong
    # results on this hardware without any error.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


# Per-source flags, by file-name prefix.  The per-group kernels (group*.hip)
# convert every matrix-core result on the vector ALU, so their results must
# be allocated in ordinary VGPRs (otherwise each value is first copied out of
# an accumulation register).
EXTRA = {
    "group": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
}


def extra_flags(src):
    name = os.path.basename(src)
    return [f for prefix, flags in EXTRA.items() if name.startswith(prefix) for f in flags]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _compile(src, verbose, check=False):
    obj = os.path.join(BUILD_CHECK if check else BUILD, os.path.basename(src) + ".o")
    cmd = ["hipcc", *FLAGS, *(["-DFGQ_CHECK"] if check else []), *extra_flags(src), "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    warn = [l for l in (r.stderr or "").splitlines() if "packed-fp32-ops" not in l]
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n" + "\n".join(warn))
    if verbose and warn:
        print("\n".join(warn), flush=True)
    return obj


def _link(objs, check, verbose):
    out = LIB_CHECK if check else LIB
    tmp = out + ".tmp"
    cmd = ["hipcc", f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build_all(verbose=False, jobs=None):
    """Both libraries (libfgq.so and the checking build libfgq_check.so)
    from one pool of compile jobs, the kernel-heavy sources of the slower
    checking build first, so that the cores stay busy to the end."""
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(BUILD_CHECK, exist_ok=True)
    heavy = lambda s: os.path.basename(s).startswith(("fold", "group"))
    srcs = sources()
    order = ([(s, True) for s in srcs if heavy(s)] + [(s, False) for s in srcs if heavy(s)] +
             [(s, True) for s in srcs if not heavy(s)] + [(s, False) for s in srcs if not heavy(s)])
    jobs = jobs or min(len(order), os.cpu_count() or 8)
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda sc: (sc[1], _compile(sc[0], verbose, sc[1])), order))
    return [_link(sorted(o for c, o in objs if c == check), check, verbose) for check in (False, True)]


def build(verbose=False, jobs=None, check=False):
    """Compile libfgq.so; with check=True the checking build
    libfgq_check.so (-DFGQ_CHECK: bounds-checked loads and stores, see
    csrc/bufcheck.h), from the same sources into its own object folder."""
    os.makedirs(BUILD_CHECK if check else BUILD, exist_ok=True)
    # the kernel-heavy sources first, so the parallel compile ends together
    srcs = sorted(sources(), key=lambda s: not os.path.basename(s).startswith(("fold", "group")))
    jobs = jobs or min(len(srcs), 8)
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose, check), srcs))
    return _link(objs, check, verbose)


if __name__ == "__main__":
    if "--all" in sys.argv:
        print(build_all(verbose="-v" in sys.argv))
    else:
        print(build(verbose="-v" in sys.argv, check="--check" in sys.argv))
