"""Oracle outputs and parity tolerance for one decoding step of attention over
residual-coded caches (one subspace per head: d = head_dim = 128, K = 256, M
stages; the paper's 0.75-bit setting is M = 12), the layout of the decoding
kernel of Appendix C at its measured rate.

The reference is the float64 oracle (attn_weights) on the caches the library
declares it reads: a key row is the exact sum of its stages' float16
codewords fp16(fp32(g s)), a value row the exact sum of its stages' float32
codewords fl(g s).

Tolerance, as for the 1-bit layout (tests/attn_bound.py): every rounding
the kernel declares is modelled as an independent zero-mean error of at most
half an ulp (variance (half ulp)^2 / 3), the output error to first order is
a sum of such terms whose variance comes from the realised operands, and
the tolerance is Z = 8 standard deviations plus the deterministic terms.
Per query head (length L, weights p_i, scaled query pair norms Pq_j):

  * query operand: per 32-token block the query turned by R_{L-1-32b},
    rounded to float16, shared by all passes: as the 1-bit form with the
    full key k''_i = R_{i mod 32} k_i;
  * key operands, per pass P over stages 2P, 2P + 1: the two stages'
    float16 codeword pieces summed in float16 (one rounding, variance
    2^-22 / 3 of the pair's squared norm Pk_P^2), then turned by R_t in
    float16 arithmetic (3 2^-24 Pk_P^2, as the 1-bit form), with the
    float32 score sums over all passes:
      vk_i = sum_P (3 2^-24 + 2^-22 / 3) sum_j Pq_j^2 Pk_Pij^2
             + 128 P (u sum_P sum_j Pq_j Pk_Pij)^2 / 3;
  * weights: float32 exp2 and the float32 subtraction of the reference
    (no float16 rounding on this path);
  * bins: the chunk's per-stage, per-codeword weight sums are exact in 64-bit
    fixed point and stored as float32: with W_mk the weight of codeword k of
    stage m (bounded by the total over chunks), Var_B(n) = sum_m sum_k
    (u W_mk c_mkn)^2 / 3;
  * the float32 softmax sum: (L / 16) u^2 o_n^2 / 3;
  * deterministic: the fixed-point weights are truncated to 2^-32 (of the
    chunk's reference, at most that of the normalised weight), once per
    token and stage: L M 2^-32 max|c|; the float32 output store u |o_n|.

A kernel that skips a 32-token block or turns the keys one position off is
caught (tests/test_attn_rq_tolerance.py plants both in the oracle's output).
"""
from __future__ import annotations

import math

import numpy as np

from oracle import gsrq_oracle as O

U = 2.0 ** -24
Z = 8.0
HD = 128


def _f16(x):
    return np.asarray(x, np.float64).astype(np.float16).astype(np.float64)


def tables(case):
    """Float16 key codewords and float32 value codewords, as float64
    [M, Hkv, K, hd]."""
    kt = (case["k_gain"][..., None] * case["k_shape"]).astype(np.float32)
    vt = (case["v_gain"][..., None] * case["v_shape"]).astype(np.float32)
    return _f16(kt), vt.astype(np.float64)


def seq_len(case, b):
    return int(min(max(int(case["lens"][b]), 0), case["k_codes"].shape[1]))


def head_caches(case, b, hk, kt=None, vt=None):
    """Decoded caches of key/value head hk of sequence b, from the oracle's
    own unpacking: keys [L, hd], values [L, hd], the key's pass partials
    [P, L, hd] (stages 2P and 2P + 1 summed exactly), value codes [L, M]."""
    M, Hkv = case["M"], case["Hkv"]
    if kt is None:
        kt, vt = tables(case)
    L = seq_len(case, b)
    kc = O.unpack_codes(case["k_codes"][b, :L], M, Hkv, 256)[:, :, hk]      # [L, M]
    vc = O.unpack_codes(case["v_codes"][b, :L], M, Hkv, 256)[:, :, hk]
    P = (M + 1) // 2
    parts = np.zeros((P, L, HD))
    v = np.zeros((L, HD))
    for m in range(M):
        parts[m // 2] += kt[m, hk][kc[:, m]]
        v += vt[m, hk][vc[:, m]]
    return parts.sum(axis=0), v, parts, vc


def _pair_norms(x):
    h = x.shape[-1] // 2
    pn = np.sqrt(x[..., :h] ** 2 + x[..., h:] ** 2)
    return np.concatenate([pn, pn], axis=-1)


def head_tolerance(q_h, k, v, parts, vcodes, vt_h, p, s, o, base, scale):
    """Tolerance [hd] of one query head.  q_h [hd] query before RoPE; k, v
    [L, hd] the head's decoded keys / values; parts [P, L, hd] the key's pass
    partials; vcodes [L, M] the value codes; vt_h [M, K, hd] the head's
    float32 value codewords; p, s [L] the oracle's weights and natural-unit
    scores; o [hd] the oracle output."""
    L = k.shape[0]
    if L == 0:
        return np.full(HD, 1e-30)
    M = vcodes.shape[1]
    npass = parts.shape[0]
    qs = scale * q_h
    Pq2 = _pair_norms(qs) ** 2                                  # [hd]
    dv = v - o[None, :]
    # query operand, one rounding per 32-token block
    vq = (2.0 ** -11 + 4 * U) ** 2 * Pq2 / 3.0
    kr = O.rope(k[None], np.arange(L) % 32, base)[0]
    nb = (L + 31) // 32
    pad = nb * 32 - L
    kp = np.pad(kr * p[:, None], ((0, pad), (0, 0))).reshape(nb, 32, HD)
    dvp = np.pad(dv, ((0, pad), (0, 0))).reshape(nb, 32, HD)
    var_q = np.zeros(HD)
    for c0 in range(0, nb, 64):
        A = np.matmul(kp[c0:c0 + 64].transpose(0, 2, 1), dvp[c0:c0 + 64])
        var_q += np.einsum("j,bjn->n", vq, A * A)
    # key operands per pass, and the float32 score sums over the passes
    vk_i = np.zeros(L)
    lin = np.zeros(L)
    for P in range(npass):
        Pk = _pair_norms(parts[P])
        vk_i += (3.0 * 2.0 ** -24 + 2.0 ** -22 / 3.0) * (Pk ** 2 @ Pq2)
        lin += Pk @ np.sqrt(Pq2)
    vk_i += 128.0 * npass * (U * lin) ** 2 / 3.0
    var_k = (p ** 2 * vk_i) @ (dv ** 2)
    # weights: float32 exp2 and the reference subtraction
    s2 = np.abs(s) * math.log2(math.e)
    m2 = float(np.max(s2)) + 8.0
    vw_i = ((4 * U * (s2 + m2 + 24.0) * math.log(2.0)) ** 2 + (2 * U) ** 2) / 3.0
    var_w = (p ** 2 * vw_i) @ (v ** 2)
    # bins stored as float32
    var_b = np.zeros(HD)
    for m in range(M):
        W = np.bincount(vcodes[:, m], weights=p, minlength=vt_h.shape[1])        # [K]
        var_b += (U * U / 3.0) * ((W ** 2) @ (vt_h[m] ** 2))
    # float32 softmax sum
    var_s = (L / 16.0) * U * U * o ** 2 / 3.0
    sigma = np.sqrt(var_q + var_k + var_w + var_b + var_s)
    det = L * M * 2.0 ** -32 * float(np.max(np.abs(vt_h)))
    return Z * sigma + det + U * np.abs(o) + 1e-30


def reference(case, b, heads=None, base=500000.0, keys=None, values=None, drop_block=None):
    """Oracle output [Hq, hd] and tolerance [Hq, hd] for sequence b (only the
    query heads in `heads`, default all; other rows stay zero).

    keys / values: {hk: [L, hd]} replacing decoded caches (CPU checks);
    drop_block = j leaves tokens 32 j .. 32 j + 31 out of the softmax, the
    tolerance staying that of the true case."""
    Hkv, GQ = case["Hkv"], case["GQ"]
    Hq = Hkv * GQ
    q = case["q"][b].astype(np.float64)
    ref = np.zeros((Hq, HD))
    tol = np.full((Hq, HD), 1e-30)
    L = seq_len(case, b)
    if L == 0:
        return ref, tol
    kt, vt = tables(case)
    scale = 1.0 / math.sqrt(HD)
    hs = list(range(Hq)) if heads is None else list(heads)
    for hk in sorted({h // GQ for h in hs}):
        k, v, parts, vc = head_caches(case, b, hk, kt, vt)
        k_true = k
        if keys is not None and hk in keys:
            k = keys[hk]
        if values is not None and hk in values:
            v = values[hk]
        qh = q[hk * GQ:(hk + 1) * GQ]
        p, s = O.attn_weights(qh, k[:, None, :], base)
        pt, st = (p, s) if k is k_true else O.attn_weights(qh, k_true[:, None, :], base)
        for g in range(GQ):
            h = hk * GQ + g
            if h not in hs:
                continue
            o_true = pt[g] @ v
            tol[h] = head_tolerance(q[h], k_true, v, parts, vc, vt[:, hk], pt[g], st[g], o_true,
                                    base, scale)
            o = p[g] @ v
            if drop_block is not None:
                keep = np.ones(L, bool)
                keep[32 * drop_block:32 * drop_block + 32] = False
                o = (p[g][keep] @ v[keep]) / np.sum(p[g][keep])
            ref[h] = o
    return ref, tol
