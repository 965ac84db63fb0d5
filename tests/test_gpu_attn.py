"""GPU parity of one decoding step of attention over coded caches
(gsrq_attn_decode, the fused unpack + dequantise + RoPE + attention kernel
of Appendix C) against the float64 oracle, through the C ABI.

Inputs come from synth.attn_case (seeded codebooks, codes and queries).  The
oracle decodes the codes itself (unpack_codes, then g * s), takes the float16
decode of keys and values (g * s rounded to float32, then float16: the values
the library declares it reads) and computes the attention in float64
(attn_weights).

Tolerance: tests/attn_bound.py, a statistical bound from the realised
operands (8 standard deviations of the first-order output error under the
probabilistic model of every rounding the kernel declares: float16 query
per 32-token block, float16 RoPE of the keys with float16 cosines/sines,
float16 weights in the value product, float32 sums) plus the deterministic
subnormal and store terms.  tests/test_attn_tolerance.py shows on the CPU
that it admits those roundings and rejects an output with a 32-token block
left out or with the key positions shifted by one.
The test also reports the worst observed error relative to that bound.
"""
import numpy as np
import pytest

import synth
from tests import attn_bound as AB
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


def _run(case, base=BASE):
    t = {k: _dev(case[k]) for k in ("k_codes", "v_codes", "lens", "k_gain", "k_shape",
                                    "v_gain", "v_shape")}
    q = _dev(case["q"])
    out = B.attn_decode(t["k_codes"], t["v_codes"], t["lens"], t["k_gain"], t["k_shape"],
                        t["v_gain"], t["v_shape"], q, rope_base=base)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def _reference(case, b, heads=None, base=BASE):
    """Oracle output [Hq, 128] and per-element tolerance for sequence b."""
    return AB.reference(case, b, heads, base)


def _check(case, out, heads=None, what=""):
    worst = 0.0
    for b in range(out.shape[0]):
        ref, tol = _reference(case, b, heads)
        hs = range(out.shape[1]) if heads is None else heads
        for h in hs:
            err = np.abs(out[b, h] - ref[h])
            assert np.all(err <= tol[h]), (
                f"{what} b{b} h{h}: err {err.max():.3g} > tol {tol[h][err.argmax()]:.3g} "
                f"(ref {ref[h][err.argmax()]:.4g})")
            worst = max(worst, float(np.max(err / tol[h])))
    say(what, "worst err / tolerance", f"{worst:.3g}")
    return worst


@pytest.mark.parametrize("Bn,cap,lens,Hkv,GQ,qdt", [
    (1, 40, [37], 1, 4, "float32"),                # one partial block pair
    (3, 5000, [5000, 1, 0], 2, 4, "float32"),      # ragged: full, one token, empty
    (2, 3000, [2999, 1025], 3, 2, "float16"),      # GQ = 2, float16 queries
    (2, 4100, [4097, 64], 2, 1, "float32"),        # GQ = 1 (32 blocks per wave group)
    (2, 2048, [2048, 2000], 8, 4, "float16"),      # 8 heads: 1024-wide rows
    (2, 700, [900, -3], 1, 4, "float32"),          # lengths clamped to [0, cap]
])
def test_attn_decode_parity(Bn, cap, lens, Hkv, GQ, qdt):
    say("attn parity", Bn, cap, lens, Hkv, GQ, qdt)
    case = synth.attn_case(Bn, cap, lens, Hkv, GQ, seed=41, q_dtype=qdt)
    out = _run(case)
    assert np.all(np.isfinite(out))
    _check(case, out, what=f"attn {Bn}x{cap} GQ{GQ}")
    for b, L in enumerate(lens):
        if L <= 0:
            assert np.all(out[b] == 0.0)


def test_attn_decode_peaked_and_rising_scores():
    """Peaked softmax (queries x 3), and keys whose scores jump in the later
    blocks of a chunk (large-gain codewords used only after token 2500), so
    the running reference maximum is raised and the partial sums rescaled."""
    case = synth.attn_case(2, 6000, [6000, 5300], 2, 4, seed=42, q_scale=3.0)
    G = case["k_gain"].shape[1]
    case["k_gain"][0, :, 255] *= 4.0
    kb = case["k_codes"].view(np.uint8).reshape(2, 6000, G)
    kb[:, :2500][kb[:, :2500] == 255] = 0
    kb[:, 2500::7, :] = 255
    say("attn peaked / rising")
    out = _run(case)
    _check(case, out, what="attn rising")


def test_attn_decode_full_size_sampled():
    """The benchmark's shape: 8 sequences x 32768 tokens, 8 key/value heads,
    32 query heads, one chunking of the launch; a few (sequence, head) pairs
    against the oracle."""
    Bn, cap, Hkv, GQ = 8, 32768, 8, 4
    lens = [32768, 32768, 30001, 32768, 17, 32768, 32767, 1]
    case = synth.attn_case(Bn, cap, lens, Hkv, GQ, seed=43, q_dtype="float16")
    say("attn full size sampled")
    out = _run(case)
    assert np.all(np.isfinite(out))
    for b in (0, 2, 4, 6, 7):
        heads = [0, 13, 31] if b != 2 else [5, 22]
        ref, tol = _reference(case, b, heads)
        for h in heads:
            err = np.abs(out[b, h] - ref[h])
            assert np.all(err <= tol[h]), f"b{b} h{h}: {err.max():.3g} > {tol[h][err.argmax()]:.3g}"



def test_attn_decode_tables_ready_reuses_workspace():
    """A second call on the same workspace with GSRQ_ATTN_TABLES_READY (same
    codebooks, new queries and lengths) skips the table build and gives the
    output of a call that builds them, bit for bit, and the oracle's."""
    case = synth.attn_case(3, 3000, [3000, 1700, 5], 2, 4, seed=7, q_dtype="float16")
    t = {k: _dev(case[k]) for k in ("k_codes", "v_codes", "lens", "k_gain", "k_shape",
                                    "v_gain", "v_shape", "q")}
    ws = torch.empty(B.attn_workspace_bytes(3, 3000, 8, 2), dtype=torch.uint8, device="cuda")
    args = [t[k] for k in ("k_codes", "v_codes")]
    cb = [t[k] for k in ("k_gain", "k_shape", "v_gain", "v_shape")]
    B.attn_decode(*args, t["lens"], *cb, t["q"], workspace=ws)
    rng = np.random.default_rng(8)
    case["q"] = rng.standard_normal(case["q"].shape).astype(np.float16)
    case["lens"] = np.array([2999, 3000, 1], np.int32)
    q2, lens2 = _dev(case["q"]), _dev(case["lens"])
    say("attn tables ready")
    ready = B.attn_decode(*args, lens2, *cb, q2, workspace=ws, tables_ready=True)
    fresh = B.attn_decode(*args, lens2, *cb, q2)
    torch.cuda.synchronize()
    assert torch.equal(ready, fresh)
    _check(case, ready.cpu().numpy().astype(np.float64), what="attn tables ready")
