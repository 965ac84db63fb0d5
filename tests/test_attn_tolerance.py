"""CPU checks of the decode-attention parity tolerance (tests/attn_bound.py):
it admits an output computed with the roundings the kernel declares
(float16 query per 32-token block, keys turned in float16 arithmetic with
float16 cosines and sines, float16 softmax weights in the value product),
and it rejects the oracle's output with one 32-token block left out or with
the keys turned at positions shifted by one (mistakes planted in the
oracle's output, on the CPU)."""
import math

import numpy as np
import pytest

import synth
from oracle import gsrq_oracle as O
from tests import attn_bound as AB

BASE = 500000.0


def _f16(x):
    return np.asarray(x, np.float64).astype(np.float16).astype(np.float64)


def emulate_rounded(q_h, k, v, base):
    """One head's attention computed with the operand roundings of the
    decode-attention kernel's declared precision, in numpy: query turned
    by R_{L-1-32b} for block b and rounded to float16; key pair (x, y)
    turned by R_t, t = i mod 32, in float16 arithmetic (x' = fl(x c -
    fl(y s)), y' = fl(x s + fl(y c))) with c, s = fp16(fp32(cos / sin));
    scores from the rounded operands in log2 units; weights 2^(s - m + 15)
    rounded to float16 in the value sum, unrounded in the softmax sum."""
    L = k.shape[0]
    hd = k.shape[1]
    half = hd // 2
    scale = 1.0 / math.sqrt(hd) * math.log2(math.e)
    theta = O.rope_theta(hd, base)
    t = np.arange(L) % 32
    ang = t[:, None] * theta[None, :]
    c = np.cos(ang).astype(np.float32).astype(np.float16).astype(np.float64)
    s = np.sin(ang).astype(np.float32).astype(np.float16).astype(np.float64)
    x, y = k[:, :half], k[:, half:]
    xr = _f16(x * c - _f16(y * s))
    yr = _f16(x * s + _f16(y * c))
    kr = np.concatenate([xr, yr], axis=1)
    blk = np.arange(L) // 32
    nblk = blk.max() + 1
    qrot = O.rope((scale * q_h)[None, None, :].repeat(nblk, axis=1),
                  (L - 1) - 32 * np.arange(nblk), base)[0]            # [nblk, hd]
    qrot = _f16(qrot)
    sc = np.sum(qrot[blk] * kr, axis=1)
    m = float(np.max(sc)) + 8.0
    pv = np.exp2(sc - m + 15.0)
    return (_f16(pv) @ v) / np.sum(pv)


@pytest.fixture(scope="module")
def case4096():
    case = synth.attn_case(1, 4096, [4096], 1, 4, seed=41)
    q, k16, v16 = AB.case_sequence(case, 0)
    ref, tol = AB.reference(case, 0)
    return case, q, k16, v16, ref, tol


def test_rounded_computation_within_tolerance(case4096):
    case, q, k16, v16, ref, tol = case4096
    worst = 0.0
    for h in range(q.shape[0]):
        o = emulate_rounded(q[h], k16[:, 0], v16[:, 0], BASE)
        r = np.abs(o - ref[h]) / tol[h]
        worst = max(worst, float(r.max()))
    print("emulated roundings: worst err / tolerance", worst)
    assert worst <= 1.0
    # the tolerance is not vacuous: the emulated error is a visible part of it
    assert worst >= 0.02


@pytest.mark.parametrize("L,GQ,q_scale", [(37, 4, 1.0), (1, 1, 1.0), (700, 2, 3.0)])
def test_rounded_computation_within_tolerance_small(L, GQ, q_scale):
    case = synth.attn_case(1, L, [L], 1, GQ, seed=5, q_scale=q_scale)
    q, k16, v16 = AB.case_sequence(case, 0)
    ref, tol = AB.reference(case, 0)
    for h in range(q.shape[0]):
        o = emulate_rounded(q[h], k16[:, 0], v16[:, 0], BASE)
        assert np.all(np.abs(o - ref[h]) <= tol[h])


@pytest.mark.parametrize("blk", [0, 17, 127])
def test_dropped_block_is_rejected(case4096, blk):
    case, q, k16, v16, ref, tol = case4096
    drop, _ = AB.reference(case, 0, drop_block=blk)
    bad = np.abs(drop - ref) > tol
    print(f"block {blk} left out: {int(bad.sum())} of {bad.size} elements outside")
    assert bad.any(axis=1).all(), "every head must see the missing block"


def test_positions_shifted_by_one_are_rejected(case4096):
    case, q, k16, v16, ref, tol = case4096
    L = k16.shape[0]
    # keys turned at positions 1 .. L instead of 0 .. L-1
    k1 = O.rope(np.transpose(k16, (1, 0, 2)), np.ones(L), BASE).transpose(1, 0, 2)
    shifted, _ = AB.reference(case, 0, keys=k1)
    bad = np.abs(shifted - ref) > tol
    assert bad.any(axis=1).all()


def test_tolerance_is_far_below_the_worst_case_bound(case4096):
    """The statistical bound is orders of magnitude below the old
    Cauchy-Schwarz form scale (6 2^-11) |q| max|k| propagated through
    exp: the median tolerance is a small fraction of |output|."""
    case, q, k16, v16, ref, tol = case4096
    assert np.median(tol / np.maximum(np.abs(ref), 1e-12)) < 0.1
