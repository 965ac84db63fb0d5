"""Register budget of the hot kernels (CPU only: hipcc cross-compiles).

A kernel whose registers exceed its occupancy target spills to scratch
memory; in the scoring loops that costs 7-10% and it is invisible to the
parity tests.  This compiles both translation units with hipcc's resource
remarks and checks that no kernel on the hot path spills (a few bytes of
fixed stack are allowed).
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

from paper_2607_01065_amd import build as BUILD

HOT = re.compile(r"(assign_accumulate_kernel|encode_kernel|encode_small_kernel|decode_lds_kernel|finalize_kernel|update_kernel|"
                 r"w_score_kernel|w_accumulate_kernel|w_exact_kernel|w_decode|w_encode_fused|"
                 r"wnorm_kernel|wselect_kernel|attn_merge_kernel)")
MAX_SCRATCH = 16   # bytes per lane
# The single-stage narrow encoder runs three waves per SIMD (168 registers)
# and keeps some set-up values of its prologue in scratch: allowed, provided
# that no scratch access lies inside a loop (its block loop reloads nothing).
PROLOGUE_ONLY = re.compile(r"13encode_kernel")
# Kernels allowed to spill outside their innermost loop: the decode-attention
# kernels run two waves per SIMD (256 registers) and spill a few group- or
# pass-level values (reloaded once per 8 token blocks, or once per stage-pair
# pass and group); their per-block loop (loop depth 2) must touch no scratch.
LOOP_CHECKED = re.compile(r"attn_(rq_)?chunk_kernel")


def _remarks(src):
    hipcc = BUILD.hipcc()
    with tempfile.TemporaryDirectory() as tmp:
        cmd = [hipcc, *BUILD.flags_for(src), "-c",
               "-I", BUILD.INCLUDE, "-o", os.path.join(tmp, "x.o"), src,
               "-Rpass-analysis=kernel-resource-usage"]
        res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    out, name = {}, None
    for line in res.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name:
            out[name] = int(m.group(1))
    return out


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
@pytest.mark.parametrize("tu", BUILD.SRCS)
def test_hot_kernels_do_not_spill(tu):
    scratch = _remarks(tu)
    hot = {k: v for k, v in scratch.items() if HOT.search(k) and not PROLOGUE_ONLY.search(k)}
    assert hot, "no hot kernels found in the resource remarks"
    bad = {k: v for k, v in hot.items() if v > MAX_SCRATCH}
    assert not bad, f"kernels spilling to scratch: {bad}"


def _scratch_loop_depths(src):
    """Loop depth of every scratch access, per kernel, from the device
    assembly (LLVM annotates each block label with its loop depth)."""
    hipcc = BUILD.hipcc()
    with tempfile.TemporaryDirectory() as tmp:
        out = os.path.join(tmp, "x.s")
        cmd = [hipcc, *BUILD.flags_for(src), "--cuda-device-only", "-S", "-I", BUILD.INCLUDE,
               "-o", out, src]
        res = subprocess.run(cmd, capture_output=True, text=True)
        assert res.returncode == 0, res.stderr[-2000:]
        lines = open(out).read().splitlines()
    depths, name, depth = {}, None, 0
    for line in lines:
        m = re.match(r"^(_Z\S+):", line)
        if m:
            name, depth = m.group(1), 0
            depths[name] = []
            continue
        if name is None:
            continue
        if line.startswith(".Lfunc_end"):
            name = None
            continue
        if re.match(r"^(\.LBB\d+_\d+:|; %bb\.\d+:)", line):
            m = re.search(r"Depth=(\d+)", line)
            depth = int(m.group(1)) if m else 0
        elif line.lstrip().startswith(";") and "Loop Header" in line:
            m = re.search(r"Depth=(\d+)", line)
            if m:
                depth = int(m.group(1))
        elif re.match(r"\s+scratch_(load|store)", line):
            depths[name].append(depth)
    return depths


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
def test_attention_block_loop_does_not_spill():
    src = [f for f in BUILD.SRCS if f.endswith("gsrq_attn.hip")][0]
    depths = {k: v for k, v in _scratch_loop_depths(src).items() if LOOP_CHECKED.search(k)}
    assert len(depths) == 6, sorted(depths)            # GQ = 1, 2, 4; 1-bit and residual
    bad = {k: max(v) for k, v in depths.items() if v and max(v) >= 2}
    assert not bad, f"scratch accesses inside the token-block loop: {bad}"


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
def test_encoder_scratch_only_in_prologue():
    src = [f for f in BUILD.SRCS if f.endswith("gsrq.hip")][0]
    depths = {k: v for k, v in _scratch_loop_depths(src).items() if PROLOGUE_ONLY.search(k)}
    assert len(depths) >= 4, sorted(depths)            # float16 / float32 rows, both loaders
    bad = {k: max(v) for k, v in depths.items() if v and max(v) >= 1}
    assert not bad, f"scratch accesses inside a loop of the encoder: {bad}"
