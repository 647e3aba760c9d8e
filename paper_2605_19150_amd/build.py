"""Build libpdssm.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2605_19150_amd.build
"""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libpdssm.so")
# (source, extra flags, object name): the fused kernels are compiled once per
# state size N so that the sizes build in parallel.
SOURCES = [("pdssm_fused.hip", ["-DPDSSM_N=%d" % n], "pdssm_fused_n%d" % n)
           for n in (64, 128, 256, 32, 16, 8)] + [
    ("pdssm_chunked.hip", [], "pdssm_chunked"),
    ("pdssm_ste.hip", [], "pdssm_ste"),
    ("pdssm_decode.hip", [], "pdssm_decode"),
    ("pdssm_select.hip", [], "pdssm_select"),
    ("pdssm_noalloc.hip", [], "pdssm_noalloc"),
    ("pdssm_api.cpp", [], "pdssm_api"),
]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-Wall",
    # keep the compiler from emitting packed fp32 VALU ops (v_pk_*_f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in res.stdout.splitlines()
                    if "packed-fp32-ops" not in l and "--hip-link" not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed (%d):\n%s" % (res.returncode, out))
    if verbose and out.strip():
        print(out)


def build_library(verbose=False):
    """Compile every HIP/C++ source of the library (one hipcc per source, in
    parallel) and link libpdssm.so.  Always recompiles.  Returns the library
    path."""
    from concurrent.futures import ThreadPoolExecutor

    tag = "%d" % os.getpid()
    objdir = os.path.join(PKG, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = [os.path.join(objdir, name + "." + tag + ".o") for _, _, name in SOURCES]
    inc = ["-I", os.path.join(ROOT, "include"), "-I", CSRC]
    compile_flags = [f for f in HIPCC_FLAGS if f != "-shared"]
    jobs = [[hipcc()] + compile_flags + extra + inc + ["-c", os.path.join(CSRC, src), "-o", o]
            for (src, extra, _), o in zip(SOURCES, objs)]
    try:
        with ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 1)) as ex:
            for f in [ex.submit(_run, j, verbose) for j in jobs]:
                f.result()
        tmp = LIB + ".tmp" + tag
        _run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs, verbose)
        os.replace(tmp, LIB)
    finally:
        for o in objs:
            if os.path.exists(o):
                os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose=True))
    sys.exit(0)
