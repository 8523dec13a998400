"""Build libflashbob.so (HIP, gfx950 only) in-tree with hipcc.

Usage:  python -m paper_2609_24089_amd.build
"""
import concurrent.futures
import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libflashbob.so")
# Translation units and the extra flags each is compiled with.
SOURCES = [
    ("flashbob.hip", []),
    ("fb_passes_d128.hip", ["-mllvm", "-amdgpu-sched-strategy=iterative-ilp"]),
]

# -packed-fp32-ops keeps hipcc from emitting v_pk_*_f32 (the host pass warns
# that it does not know the feature; that warning is harmless).
HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]

def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (needs ROCm)")


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(line for line in (res.stdout + res.stderr).splitlines()
                    if "is not a recognized feature" not in line)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + out)
    return out


def build_library(verbose=False):
    """Compile every source into libflashbob.so next to this file (always rebuilds)."""
    tmpdir = tempfile.mkdtemp(prefix="flashbob_build_")
    try:
        objs, jobs = [], []
        with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as pool:
            for name, extra in SOURCES:
                obj = os.path.join(tmpdir, name + ".o")
                objs.append(obj)
                cmd = [hipcc()] + HIPCC_FLAGS + extra + ["-c", "-o", obj, os.path.join(CSRC, name)]
                jobs.append(pool.submit(_run, cmd))
            outs = [j.result() for j in jobs]
        tmp = LIB + ".tmp"
        outs.append(_run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs))
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    out = "\n".join(o for o in outs if o.strip())
    if verbose and out.strip():
        print(out)
    os.replace(tmp, LIB)
    return LIB

if __name__ == "__main__":
    print(build_library(verbose="-v" in sys.argv))
