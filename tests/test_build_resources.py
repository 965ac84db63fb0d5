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

HOT = re.compile(r"(assign_accumulate_kernel|encode_kernel|decode_lds_kernel|finalize_kernel|update_kernel|"
                 r"w_score_kernel|w_accumulate_kernel|w_exact_kernel|w_decode|w_encode_fused|"
                 r"wnorm_kernel|wselect_kernel|attn_chunk_kernel|attn_merge_kernel)")
MAX_SCRATCH = 16   # bytes per lane


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
    hot = {k: v for k, v in scratch.items() if HOT.search(k)}
    assert hot, "no hot kernels found in the resource remarks"
    bad = {k: v for k, v in hot.items() if v > MAX_SCRATCH}
    assert not bad, f"kernels spilling to scratch: {bad}"
