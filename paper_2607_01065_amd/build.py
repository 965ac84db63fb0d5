"""Build the GSRQ HIP library (libgsrq.so) for gfx950 in-tree with hipcc."""
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRCS = [os.path.join(HERE, "csrc", f) for f in ("gsrq.hip", "gsrq_wide.hip", "gsrq_weights.hip", "gsrq_attn.hip")]
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libgsrq.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # packed fp32 instructions are kept out of every kernel on purpose
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


# Flags of single translation units.  The attention kernel keeps its MFMA
# accumulators in ordinary VGPRs: with them in AGPRs, the rare rescaling of
# the output sums (VALU work) made the compiler copy all 64 accumulators to
# VGPRs on every token block.  The narrow family's block claims are single-
# lane LDS atomics that the atomic optimizer would wrap in a wave-wide
# count-and-broadcast sequence (six VALU and six SALU instructions per
# block); its few multi-lane same-address atomics reduce over the wave
# themselves.
SRC_FLAGS = {
    "gsrq_attn.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    "gsrq.hip": ["-mllvm", "-amdgpu-atomic-optimizer-strategy=None"],
}


def flags_for(src):
    """hipcc flags of one source (without -shared)."""
    return [f for f in HIPCC_FLAGS if f != "-shared"] + SRC_FLAGS.get(os.path.basename(src), [])


def build(verbose=False, extra=()):
    """Compile every source to an object (in parallel), then link
    libgsrq.so; always recompiles."""
    tmp = LIB + ".tmp"
    objs = [LIB + "." + os.path.basename(src) + ".o" for src in SRCS]
    procs = []
    for src, obj in zip(SRCS, objs):
        cmd = [hipcc(), *flags_for(src), *extra, "-c", "-I", INCLUDE, "-o", obj, src]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE,
                                      text=True))
    failed = False
    for p in procs:
        out, err = p.communicate()
        if p.returncode != 0:
            sys.stderr.write(out + err)
            failed = True
    if not failed:
        cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            failed = True
    for obj in objs:
        if os.path.exists(obj):
            os.remove(obj)
    if failed:
        raise RuntimeError("hipcc failed building libgsrq.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
