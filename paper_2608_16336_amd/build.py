"""Build libmts.so (hipcc, gfx950) in-tree."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "_lib", "libmts.so")
SOURCES = [os.path.join(HERE, "csrc", f)
           for f in ("mts_api.cpp", "mts_tables.cpp", "mts_kernels.hip", "mts_arrivals.hip", "mts_noalloc.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = ["-O3", "--offload-arch=gfx950", "-std=c++17", "-fPIC",
         "-ffp-contract=off",
         # no packed FP32 instructions anywhere
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall"]
# per-source extra flags: the step kernel's floating point never sees a NaN
# (freeness keys are finite or -inf), so its maxima need no NaN quieting
EXTRA = {"mts_kernels.hip": ["-fno-honor-nans"]}


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + out)
    return out


def build(verbose=False):
    os.makedirs(os.path.dirname(LIB), exist_ok=True)
    objdir = os.path.join(os.path.dirname(LIB), "obj")
    os.makedirs(objdir, exist_ok=True)
    outs, objs = [], []
    for src in SOURCES:
        obj = os.path.join(objdir, os.path.basename(src) + ".o")
        outs.append(_run([HIPCC] + FLAGS + EXTRA.get(os.path.basename(src), []) +
                         ["-I", os.path.join(ROOT, "include"), "-c", "-o", obj, src]))
        objs.append(obj)
    tmp = LIB + ".tmp"
    outs.append(_run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs))
    out = "\n".join(o for o in outs if o.strip())
    if verbose and out.strip():
        print(out)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
