"""GPU parity of one decoding step of attention over residual-coded caches
(gsrq_attn_decode on the paper's sub-1-bit layout: one subspace per head,
d = 128, K = 256, M stages; 0.75 bit at M = 12, the setting of the decoding
latency analysis, Appendix C) against the float64 oracle, through the C ABI.

Inputs come from synth.attn_case_rq (seeded codebooks with stage gains
falling as in a residual cascade, uniform codes, queries).  The oracle
unpacks the codes itself and sums the stages' codewords in float64 (keys:
float16 codewords, values: float32 codewords, the inputs the library
declares), then takes attn_weights.  Tolerance: tests/attn_rq_bound.py,
whose CPU checks (tests/test_attn_rq_tolerance.py) show that it admits the
kernel's declared roundings and rejects a dropped block or keys turned one
position off.  The value weights are summed as 64-bit integers, so repeated
calls agree bit for bit.
"""
import numpy as np
import pytest

import synth
from tests import attn_rq_bound as AB
from tests.gpu_util import say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2607_01065_amd import gsrq as B  # noqa: E402

BASE = 500000.0


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _tensors(case):
    return {k: _dev(case[k]) for k in ("k_codes", "v_codes", "lens", "k_gain", "k_shape",
                                       "v_gain", "v_shape", "q")}


def _run(t, **kw):
    out = B.attn_decode(t["k_codes"], t["v_codes"], t["lens"], t["k_gain"], t["k_shape"],
                        t["v_gain"], t["v_shape"], t["q"], rope_base=BASE, **kw)
    torch.cuda.synchronize()
    return out


def _check(case, out, pairs=None, what=""):
    """pairs: [(b, [query heads])] to compare, default every head of every
    sequence."""
    Bn, Hq = out.shape[0], out.shape[1]
    pairs = [(b, None) for b in range(Bn)] if pairs is None else pairs
    worst = 0.0
    for b, heads in pairs:
        ref, tol = AB.reference(case, b, heads, BASE)
        for h in (range(Hq) if heads is None else heads):
            err = np.abs(out[b, h] - ref[h])
            assert np.all(err <= tol[h]), (
                f"{what} b{b} h{h}: err {err.max():.3g} > tol {tol[h][err.argmax()]:.3g} "
                f"(ref {ref[h][err.argmax()]:.4g})")
            worst = max(worst, float(np.max(err / tol[h])))
    say(what, "worst err / tolerance", f"{worst:.3g}")
    return worst


@pytest.mark.parametrize("Bn,cap,lens,Hkv,GQ,M,qdt", [
    (1, 40, [37], 1, 4, 12, "float32"),             # one partial block, 0.75 bit
    (3, 5000, [5000, 1, 0], 2, 4, 12, "float32"),   # ragged: two chunks, one token, empty
    (2, 3000, [2999, 1025], 3, 2, 16, "float16"),   # 1 bit, GQ = 2, float16 queries
    (2, 4100, [4097, 64], 2, 1, 3, "float32"),      # odd M: a single-stage last pass; GQ = 1
    (1, 700, [700], 1, 4, 1, "float32"),            # one stage
    (2, 9000, [9000, 8191], 8, 4, 12, "float16"),   # 8 heads, three chunks
    (2, 700, [900, -3], 1, 4, 12, "float32"),       # lengths clamped to [0, cap]
    (1, 266300, [266300], 1, 1, 2, "float32"),      # 66 chunks: the value merge in two rounds
])
def test_attn_rq_parity(Bn, cap, lens, Hkv, GQ, M, qdt):
    say("attn rq parity", Bn, cap, lens, Hkv, GQ, M, qdt)
    case = synth.attn_case_rq(Bn, cap, lens, Hkv, GQ, M=M, seed=41, q_dtype=qdt)
    out = _run(_tensors(case)).cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(out))
    _check(case, out, what=f"attn rq {Bn}x{cap} GQ{GQ} M{M}")
    for b, L in enumerate(lens):
        if L <= 0:
            assert np.all(out[b] == 0.0)


def test_attn_rq_peaked_scores():
    """Peaked softmax (queries x 3) and key codewords of one stage scaled up
    in the later part of the cache, so that a few tokens dominate."""
    case = synth.attn_case_rq(2, 6000, [6000, 5300], 2, 4, M=12, seed=42, q_scale=3.0)
    case["k_gain"][0, :, 255] *= 3.0
    kb = case["k_codes"].view(np.uint8).reshape(2, 6000, -1)
    M, Hkv = case["M"], case["Hkv"]
    for h in range(Hkv):
        col = kb[:, :2500, h]                        # stage 0 of head h
        col[col == 255] = 0
        kb[:, 2500::7, h] = 255
    say("attn rq peaked")
    out = _run(_tensors(case)).cpu().numpy().astype(np.float64)
    _check(case, out, what="attn rq peaked")


def test_attn_rq_full_size_sampled():
    """The benchmark's shape: 8 sequences x 32768 tokens, 8 key/value heads,
    32 query heads, 12 stages; a few (sequence, head) pairs against the
    oracle, and the call repeated: the outputs agree bit for bit."""
    Bn, cap, Hkv, GQ = 8, 32768, 8, 4
    lens = [32768, 32768, 30001, 32768, 17, 32768, 32767, 1]
    case = synth.attn_case_rq(Bn, cap, lens, Hkv, GQ, M=12, seed=43, q_dtype="float16")
    say("attn rq full size sampled")
    t = _tensors(case)
    out = _run(t)
    again = _run(t)
    assert torch.equal(out, again), "integer weight sums: repeated calls must agree"
    out = out.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(out))
    _check(case, out, pairs=[(0, [0, 3]), (2, [13]), (4, [31]), (7, [8]), (6, [20])],
           what="attn rq full size")


def test_attn_rq_tables_ready_and_tag():
    """A second call that reuses the workspace's tables (GSRQ_ATTN_TABLES_READY)
    gives the same output bit for bit; with codebooks of another case (a
    different codebook array) the device-checked tag gives NaN outputs."""
    case = synth.attn_case_rq(2, 3000, [2999, 1500], 2, 4, M=12, seed=44)
    t = _tensors(case)
    n = B.attn_workspace_bytes(2, 3000, 8, 2, d=128, M=12)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    first = _run(t, workspace=ws)
    reused = _run(t, workspace=ws, tables_ready=True)
    assert torch.equal(first, reused)
    other = synth.attn_case_rq(2, 3000, [2999, 1500], 2, 4, M=12, seed=45)
    t2 = _tensors(other)
    bad = _run(t2, workspace=ws, tables_ready=True)
    assert torch.isnan(bad).all()
    # a workspace holding 1-bit tables does not pass for residual-coded ones
    one = synth.attn_case(2, 3000, [2999, 1500], 2, 4, seed=46)
    t1 = _tensors(one)
    n1 = max(n, B.attn_workspace_bytes(2, 3000, 8, 2))
    ws1 = torch.empty(n1, dtype=torch.uint8, device="cuda")
    _run(t1, workspace=ws1)
    bad = _run(t, workspace=ws1, tables_ready=True)
    assert torch.isnan(bad).all()


def test_attn_rq_more_than_16_stages_unsupported():
    case = synth.attn_case_rq(1, 64, [64], 1, 4, M=17, seed=47)
    with pytest.raises(B.GsrqError) as e:
        _run(_tensors(case))
    assert e.value.status == B.GSRQ_E_UNSUPPORTED
