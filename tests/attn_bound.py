"""Oracle outputs and parity tolerance for one decoding step of attention over
coded caches (the fused decoding kernel of Appendix C: unpack, dequantise,
RoPE, attention), shared by the GPU parity test and its CPU checks.

The reference is the float64 oracle (attn_weights) on the float16 decode of
the codes, fp16(fp32(g * s)), the values the library declares it reads.

Tolerance.  The kernel rounds at known points; each rounding error is at
most half an ulp and is modelled, as in the standard probabilistic model of
floating-point error, as an independent zero-mean variable, uniform on its
interval (variance (half ulp)^2 / 3).  The output error is then, to first
order, a sum of many independent terms whose variance is computed from the
realised operands of the case (not from Cauchy-Schwarz worst cases), and
the tolerance is Z = 8 standard deviations plus the few deterministic
terms.  With at most 21 effective terms 8 sigma is above the worst case
of their sum (8 sqrt(n/3) >= n), and with more the sum is close to Gaussian,
whose 8-sigma tail is ~1e-15.  Scores are in natural units below (the
kernel's log2 units scale every term alike).  For query head h of length L,
softmax weights p_i, decoded values v_i, output o, pair norms
Pq_j = |(q_j, q_{j+64})| of the scaled query and Pk_ij of key i (both
invariant under the rotations):

  * query operand: per block b of 32 tokens the kernel rounds the query
    turned by R_{L-1-32b} to float16 (after float32 arithmetic):
    dq_bj has variance vq_j = (2^-11 + 4u)^2 Pq_j^2 / 3, shared by the
    block's tokens, which see the query against their keys turned by
    R_{i mod 32} (k''_i).  First-order output change
      do_n = sum_i p_i ds_i (v_in - o_n)        (the mean score change drops
                                                 out since sum_i p_i (v_in - o_n) = 0)
    so Var_Q(n) = sum_b sum_j vq_j A_bjn^2, A_bjn = sum_{i in b} p_i k''_ij (v_in - o_n);
  * key operand: each element of a key pair (x, y), turned in float16
    arithmetic with float16 cosines/sines (each within 2^-12), takes three
    roundings: variance <= (2^-24 / 3 + 2 2^-22 / 3) Pk^2 = 3 2^-24 Pk^2;
    with the float32 score sum (128 exact products) added per token:
    Var_K(n) = sum_i p_i^2 (v_in - o_n)^2 [sum_j Pq_j^2 3 2^-24 Pk_ij^2
               + 128 (u sum_j Pq_j Pk_ij)^2 / 3];
  * weights: the value product takes the weights rounded to float16
    (2^-11), the softmax sum their float32 value; exp2 and the float32
    subtraction of the reference add a few u times (|s| + |m| + 24):
    Var_W(n) = sum_i p_i^2 v_in^2 vw_i;
  * float32 accumulation of the value sums and of the softmax sum (at most
    L / 16 additions each, each within u of the running sum, bounded by
    sum p |v| and by 1): Var_S(n) = (L / 16) u^2 ((sum_i p_i |v_in|)^2 + o_n^2) / 3;
  * deterministic: float16 subnormal weights (below 2^-14, absolute error
    2^-25 against a largest weight of at least 2^7, so 2^-32 of the sum per
    token): L 2^-32 max|v|; the float32 output store u |o_n|.

  tol_n = 8 sqrt(Var_Q + Var_K + Var_W + Var_S) + L 2^-32 max|v| + u |o_n| + 1e-30.

A kernel that skips or repeats a 32-token block, or turns the keys at a
position off by one, is caught (tests/test_attn_tolerance.py plants both in
the oracle's output and checks).
"""
from __future__ import annotations

import math

import numpy as np

from oracle import gsrq_oracle as O

U = 2.0 ** -24
Z = 8.0
HD = 128


def decode_rows(codes_rows, gain, shape):
    """Decoded rows in float32 arithmetic, (float32 g * s) per codeword,
    from the oracle's own unpacking; [L, D] float32."""
    G = gain.shape[1]
    idx = O.unpack_codes(codes_rows, 1, G, gain.shape[2])[:, 0, :]
    cw = gain[0][np.arange(G)[None, :], idx][..., None] * shape[0][np.arange(G)[None, :], idx]
    return cw.astype(np.float32).reshape(codes_rows.shape[0], G * shape.shape[-1])


def case_sequence(case, b):
    """(q [Hq, hd] float64, k16 [L, Hkv, hd], v16 [L, Hkv, hd]) of sequence b:
    the float16 decode of its codes, widened exactly."""
    Hkv = case["Hkv"]
    cap = case["k_codes"].shape[1]
    L = int(min(max(int(case["lens"][b]), 0), cap))
    q = case["q"][b].astype(np.float64)
    k16 = decode_rows(case["k_codes"][b, :L], case["k_gain"], case["k_shape"])
    v16 = decode_rows(case["v_codes"][b, :L], case["v_gain"], case["v_shape"])
    k16 = k16.astype(np.float16).astype(np.float64).reshape(L, Hkv, HD)
    v16 = v16.astype(np.float16).astype(np.float64).reshape(L, Hkv, HD)
    return q, k16, v16


def _pair_norms(x):
    """|(x_j, x_{j+64})| for every element j of the last axis."""
    h = x.shape[-1] // 2
    pn = np.sqrt(x[..., :h] ** 2 + x[..., h:] ** 2)
    return np.concatenate([pn, pn], axis=-1)


def head_tolerance(q_h, k, v, p, s, o, base, scale):
    """Tolerance [hd] of one query head.  q_h [hd] query before RoPE; k, v
    [L, hd] the head's float16-decoded keys / values; p, s [L] the oracle's
    weights and natural-unit scores; o [hd] the oracle output."""
    L = k.shape[0]
    if L == 0:
        return np.full(HD, 1e-30)
    qs = scale * q_h
    Pq2 = _pair_norms(qs) ** 2                                  # [hd]
    Pk = _pair_norms(k)                                         # [L, hd]
    dv = v - o[None, :]                                         # [L, hd]
    # query operand, one rounding per 32-token block
    vq = (2.0 ** -11 + 4 * U) ** 2 * Pq2 / 3.0
    kr = O.rope(k[None], np.arange(L) % 32, base)[0]            # k''_i = R_{i mod 32} k_i
    nb = (L + 31) // 32
    pad = nb * 32 - L
    kp = np.pad(kr * p[:, None], ((0, pad), (0, 0))).reshape(nb, 32, HD)
    dvp = np.pad(dv, ((0, pad), (0, 0))).reshape(nb, 32, HD)
    var_q = np.zeros(HD)
    for c0 in range(0, nb, 64):
        A = np.matmul(kp[c0:c0 + 64].transpose(0, 2, 1), dvp[c0:c0 + 64])   # [blocks, j, n]
        var_q += np.einsum("j,bjn->n", vq, A * A)
    # key operands and the float32 score sums, per token
    vk_i = 3.0 * 2.0 ** -24 * (Pk ** 2 @ Pq2) + 128.0 * (U * (Pk @ np.sqrt(Pq2))) ** 2 / 3.0
    var_k = (p ** 2 * vk_i) @ (dv ** 2)
    # weights: float16 rounding in the value product, exp2 and the reference
    s2 = np.abs(s) * math.log2(math.e)
    m2 = float(np.max(s2)) + 8.0 + 15.0
    vw_i = (2.0 ** -22 + (4 * U * (s2 + m2 + 24.0) * math.log(2.0)) ** 2 + (2 * U) ** 2) / 3.0
    var_w = (p ** 2 * vw_i) @ (v ** 2)
    # float32 accumulation of value sums and softmax sum
    spv = p @ np.abs(v)
    var_s = (L / 16.0) * U * U * (spv ** 2 + o ** 2) / 3.0
    sigma = np.sqrt(var_q + var_k + var_w + var_s)
    return Z * sigma + L * 2.0 ** -32 * float(np.max(np.abs(v))) + U * np.abs(o) + 1e-30


def reference(case, b, heads=None, base=500000.0, keys=None, values=None, drop_block=None):
    """Oracle output [Hq, hd] and tolerance [Hq, hd] for sequence b.

    keys / values replace the case's decoded caches (CPU checks);
    drop_block = j leaves tokens 32 j .. 32 j + 31 out of the softmax (the
    output of a kernel that skipped that block), the tolerance staying that
    of the true case."""
    Hkv, GQ = case["Hkv"], case["GQ"]
    Hq = Hkv * GQ
    q, k16, v16 = case_sequence(case, b)
    if keys is not None:
        k16 = keys
    if values is not None:
        v16 = values
    L = k16.shape[0]
    ref = np.zeros((Hq, HD))
    tol = np.full((Hq, HD), 1e-30)
    if L == 0:
        return ref, tol
    scale = 1.0 / math.sqrt(HD)
    p, s = O.attn_weights(q, k16, base)
    for h in range(Hq) if heads is None else heads:
        kv = h // GQ
        o = p[h] @ v16[:, kv]
        tol[h] = head_tolerance(q[h], k16[:, kv], v16[:, kv], p[h], s[h], o, base, scale)
        if drop_block is not None:
            keep = np.ones(L, bool)
            keep[32 * drop_block:32 * drop_block + 32] = False
            o = (p[h][keep] @ v16[keep, kv]) / np.sum(p[h][keep])
        ref[h] = o
    return ref, tol
