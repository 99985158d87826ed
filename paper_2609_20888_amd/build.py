"""Build libeta.so (the HIP library behind include/eta.h) for gfx950, in-tree.

    python -m paper_2609_20888_amd.build [-v]

hipcc compiles the kernel sources and the host API to objects (in parallel;
the decode kernels' source as three objects, selected by ETA_PART) and links
them into one shared library beside this file.  Packed-fp32
instruction selection is disabled for device code
(`-target-feature -packed-fp32-ops`); the prefill source keeps MFMA
accumulators in the ordinary vector registers (`-amdgpu-mfma-vgpr-form`).
"""
import os
import shutil
import subprocess
import sys
import tempfile
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libeta.so")
SOURCES = [os.path.join(CSRC, f) for f in ("eta_kernels.hip", "eta_prefill.hip", "eta_api.cpp")]
# (source, extra flags, object name): eta_kernels.hip holds split decode on bf16
# caches in part 1, on fp32 caches in part 2, and everything else in part 0
UNITS = [(SOURCES[0], [f"-DETA_PART={p}"], f"eta_kernels.{p}.o") for p in (0, 1, 2)] + \
        [(src, [], os.path.basename(src) + ".o") for src in SOURCES[1:]]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


# MFMA results kept in the ordinary vector registers: for the prefill kernel only
# (no copies between accumulation and arithmetic registers there; the
# calibration kernel is faster with the default register classes)
VGPR_FORM = {"eta_prefill.hip"}


def _flags(src: str):
    extra = ["-mllvm", "-amdgpu-mfma-vgpr-form"] if os.path.basename(src) in VGPR_FORM else []
    return ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *extra,
            "-Wall", "-Wno-unused-function",
            f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]


# hipcc's host pass does not know the packed-fp32 feature and says so; drop that line
_NOISE = "'-packed-fp32-ops' is not a recognized feature"


def _clean(stderr: str) -> str:
    return "\n".join(l for l in stderr.splitlines() if _NOISE not in l)


def build(verbose: bool = False, jobs: int = 5) -> str:
    """Compile every source to an object (in parallel), then link libeta.so."""
    objdir = tempfile.mkdtemp(prefix="eta_build_")
    try:
        cmds = [[hipcc(), *_flags(src), *extra, "-c", src, "-o", os.path.join(objdir, obj)]
                for src, extra, obj in UNITS]
        procs = []
        for cmd in cmds:
            if verbose:
                print(" ".join(cmd), flush=True)
            while len([p for p in procs if p.poll() is None]) >= max(1, jobs):
                time.sleep(0.2)
            procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                                          text=True))
        errs = []
        for cmd, p in zip(cmds, procs):
            _, err = p.communicate()
            err = _clean(err)
            if p.returncode != 0:
                errs.append(f"hipcc failed ({p.returncode}) on {cmd[-3]}:\n{err}")
            elif verbose and err.strip():
                print(err, file=sys.stderr)
        if errs:
            raise RuntimeError("\n".join(errs))
        link = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC",
                *[c[-1] for c in cmds], "-o", OUT + ".tmp"]
        if verbose:
            print(" ".join(link), flush=True)
        r = subprocess.run(link, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed ({r.returncode}):\n{_clean(r.stderr)}")
        os.replace(OUT + ".tmp", OUT)
    finally:
        shutil.rmtree(objdir, ignore_errors=True)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
