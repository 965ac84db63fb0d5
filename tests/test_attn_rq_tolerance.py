"""CPU checks of the parity tolerance for decode attention over residual-coded
caches (tests/attn_rq_bound.py): it admits an output computed with the
roundings the kernel declares (float16 query per 32-token block; per pass of
two stages, the float16 sum of the two codeword pieces turned by R_t in
float16 arithmetic with float16 cosines and sines; float32 weights truncated
to 64-bit fixed point), and it rejects the oracle's output with one 32-token
block left out or with the keys turned at positions shifted by one
(mistakes planted in the oracle's output, on the CPU)."""
import math

import numpy as np
import pytest

import synth
from oracle import gsrq_oracle as O
from tests import attn_rq_bound as AB

BASE = 500000.0


def _f16(x):
    return np.asarray(x, np.float64).astype(np.float16).astype(np.float64)


def emulate_rounded(q_h, parts_f16, v, base):
    """One head's attention with the kernel's declared roundings, in numpy.
    parts_f16 [P, 2, L, hd]: each pass's two stage codewords (float16
    values; a single-stage pass has zeros in its second slot)."""
    _, _, L, hd = parts_f16.shape
    half = hd // 2
    scale = 1.0 / math.sqrt(hd) * math.log2(math.e)
    theta = O.rope_theta(hd, base)
    t = np.arange(L) % 32
    ang = t[:, None] * theta[None, :]
    c = np.cos(ang).astype(np.float32).astype(np.float16).astype(np.float64)
    s = np.sin(ang).astype(np.float32).astype(np.float16).astype(np.float64)
    blk = np.arange(L) // 32
    nblk = blk.max() + 1
    qrot = O.rope((scale * q_h)[None, None, :].repeat(nblk, axis=1),
                  (L - 1) - 32 * np.arange(nblk), base)[0]
    qrot = _f16(qrot)
    sc = np.zeros(L)
    for P in range(parts_f16.shape[0]):
        kp = _f16(parts_f16[P, 0] + parts_f16[P, 1])          # float16 pair sum
        x, y = kp[:, :half], kp[:, half:]
        xr = _f16(x * c - _f16(y * s))
        yr = _f16(x * s + _f16(y * c))
        sc += np.sum(qrot[blk] * np.concatenate([xr, yr], axis=1), axis=1)
    m = float(np.max(sc))
    pv = np.exp2(sc - m).astype(np.float32).astype(np.float64)
    pq = np.floor(pv * 2.0 ** 32) * 2.0 ** -32                # 64-bit fixed point
    return (pq @ v) / np.sum(pv)


def _parts(case, b, hk):
    """Per pass the two stage codewords of every token (float16 values)."""
    kt, _ = AB.tables(case)
    M, Hkv = case["M"], case["Hkv"]
    L = AB.seq_len(case, b)
    kc = O.unpack_codes(case["k_codes"][b, :L], M, Hkv, 256)[:, :, hk]
    P = (M + 1) // 2
    out = np.zeros((P, 2, L, AB.HD))
    for m in range(M):
        out[m // 2, m % 2] = kt[m, hk][kc[:, m]]
    return out


@pytest.fixture(scope="module")
def case4096():
    case = synth.attn_case_rq(1, 4096, [4096], 1, 4, M=12, seed=41)
    ref, tol = AB.reference(case, 0)
    return case, ref, tol


def test_rounded_computation_within_tolerance(case4096):
    case, ref, tol = case4096
    _, v, _, _ = AB.head_caches(case, 0, 0)
    parts = _parts(case, 0, 0)
    q = case["q"][0].astype(np.float64)
    worst = 0.0
    for h in range(q.shape[0]):
        o = emulate_rounded(q[h], parts, v, BASE)
        worst = max(worst, float((np.abs(o - ref[h]) / tol[h]).max()))
    print("emulated roundings: worst err / tolerance", worst)
    assert worst <= 1.0
    assert worst >= 0.02          # the tolerance is not vacuous


@pytest.mark.parametrize("L,GQ,M,q_scale", [(37, 4, 12, 1.0), (1, 1, 3, 1.0), (700, 2, 16, 3.0),
                                            (300, 4, 1, 1.0)])
def test_rounded_computation_within_tolerance_small(L, GQ, M, q_scale):
    case = synth.attn_case_rq(1, L, [L], 1, GQ, M=M, seed=5, q_scale=q_scale)
    ref, tol = AB.reference(case, 0)
    _, v, _, _ = AB.head_caches(case, 0, 0)
    parts = _parts(case, 0, 0)
    q = case["q"][0].astype(np.float64)
    for h in range(q.shape[0]):
        o = emulate_rounded(q[h], parts, v, BASE)
        assert np.all(np.abs(o - ref[h]) <= tol[h])


@pytest.mark.parametrize("blk", [0, 17, 127])
def test_dropped_block_is_rejected(case4096, blk):
    case, ref, tol = case4096
    drop, _ = AB.reference(case, 0, drop_block=blk)
    bad = np.abs(drop - ref) > tol
    print(f"block {blk} left out: {int(bad.sum())} of {bad.size} elements outside")
    assert bad.any(axis=1).all(), "every head must see the missing block"


def test_positions_shifted_by_one_are_rejected(case4096):
    case, ref, tol = case4096
    k, _, _, _ = AB.head_caches(case, 0, 0)
    L = k.shape[0]
    k1 = O.rope(k[None], np.ones(L), BASE)[0]               # turned at positions 1 .. L
    shifted, _ = AB.reference(case, 0, keys={0: k1})
    bad = np.abs(shifted - ref) > tol
    assert bad.any(axis=1).all()


def test_tolerance_is_a_small_fraction_of_the_output(case4096):
    case, ref, tol = case4096
    assert np.median(tol / np.maximum(np.abs(ref), 1e-12)) < 0.1
