"""Plain float64 CPU oracle of GSKM, GSRQ and decode attention over a coded cache.

TEST INFRASTRUCTURE ONLY.  This module is the parity reference for the HIP
path.  Only the test suite, the smoke check of the graft entry point and the
CPU-baseline leg of the benchmark may import it; the library and its Python
binding never do, and this module shares no code with them.

Everything is written from the paper (arXiv 2607.01065, "GSRQ: Gain-Shape
Residual Quantization for Sub-1-bit KV Cache"), in the paper's order and
notation, in float64, with no blocking, fusion or reordering beyond what the
definitions state.  Inputs given in float16 or float32 are widened to float64
exactly.

Notation (paper symbol -> name used here):
  subspace dimension (Sec. 6.2 "D", implied D/M in Sec. 3)   -> d
  number of subspaces / codebooks per stage (Sec. 3 "M")      -> G = D_full / d
  number of residual stages (Sec. 3 "L", Sec. 6.2 "R")        -> M
  codebook size                                               -> K
  maximum GSKM iterations (Alg. 1 "T")                        -> T
  per-sample weight (Sec. 5.3, eq. 9 "w_i")                   -> w

Readings taken where the paper is silent (each is listed in the design notes):
  * equal-gain initial assignment before the first gain update (Alg. 1 asks
    for gains "by (8)" before any assignment exists);
  * an empty (or zero-weight) cluster keeps its gain and shape (Sec. 5.2,
    implementation details); at initialisation such a cluster takes the
    norm of its seed row as gain;
  * epsilon of the per-sample normalisation is 1e-8;
  * a mean direction is "numerically close to zero" when
    ||sum_i w_i y_i|| <= 1e-6 * sum_i w_i; the previous shape is kept;
  * weighted GSKM: every mean in eqs. (7) and (8) becomes a w-weighted mean
    (Sec. 5.1 / 5.3); the assignment itself is unweighted;
  * ties in every argmax go to the lowest codeword index;
  * the stop test of Alg. 1 is per subspace; at t = 1 it compares with the
    initial assignment;
  * the next-stage residual is the residual of re-encoding the stage input
    with the stage's final codebook;
  * encode and decode use each codeword's own gain g_k (the gain-shape pair
    is one implicit codebook, Sec. 5.2, eq. 3), not a per-vector gain.
"""
from __future__ import annotations

import numpy as np

EPS = 1e-8              # epsilon of y_i = x_i / (||x_i|| + eps)  (Sec. 5.2)
SHAPE_KEEP_REL = 1e-6   # mean direction treated as zero below this (reading)


# ----------------------------------------------------------------------------
# Gain-shape K-means (Sec. 5.2, eqs. 3-8, Algorithm 1)
# ----------------------------------------------------------------------------

def gskm_scores(X, gain, shape):
    """Assignment scores of eq. (5): S[i, k] = 2 g_k x_i^T s_k - g_k^2.

    X: [N, d]; gain: [K]; shape: [K, d].  Maximising S over k is the same as
    minimising ||x_i - g_k s_k||^2 of eq. (4), the constant ||x_i||^2 dropped.
    """
    X = np.asarray(X, dtype=np.float64)
    gain = np.asarray(gain, dtype=np.float64)
    shape = np.asarray(shape, dtype=np.float64)
    proj = X @ shape.T                              # x_i^T s_k
    return 2.0 * gain[None, :] * proj - gain[None, :] ** 2


def gskm_assign(X, gain, shape):
    """Eq. (5): k_i = argmax_k (2 g_k x_i^T s_k - g_k^2), lowest k on ties."""
    S = gskm_scores(X, gain, shape)
    return np.argmax(S, axis=1).astype(np.int64)


def assignment_margin(X, gain, shape):
    """Relative top-2 margin of the eq. (5) scores of every row.

    margin_i = (S_(1) - S_(2)) / max(||x_i||^2, 1e-30): the gap in squared
    distortion between the best and second-best codeword, relative to the
    row's energy (S = ||x||^2 - ||x - g s||^2).  For K = 1 the margin is +inf.
    """
    X = np.asarray(X, dtype=np.float64)
    S = gskm_scores(X, gain, shape)
    if S.shape[1] == 1:
        return np.full(S.shape[0], np.inf)
    top2 = -np.partition(-S, 1, axis=1)[:, :2]
    energy = np.maximum(np.sum(X * X, axis=1), 1e-30)
    return (top2[:, 0] - top2[:, 1]) / energy


def normalize_rows(X, eps=EPS):
    """Eq. (6) with the safeguard of Sec. 5.2: y_i = x_i / (||x_i|| + eps)."""
    X = np.asarray(X, dtype=np.float64)
    return X / (np.linalg.norm(X, axis=1, keepdims=True) + eps)


def weighted_distortion(X, w, gain, shape, assign):
    """J = sum_i w_i ||x_i - g_{k_i} s_{k_i}||^2 (the l2 objective, eq. 4)."""
    X = np.asarray(X, dtype=np.float64)
    C = np.asarray(gain, np.float64)[:, None] * np.asarray(shape, np.float64)
    R = X - C[assign]
    return float(np.sum(np.asarray(w, np.float64) * np.sum(R * R, axis=1)))


def gskm_update(X, w, assign, gain, shape):
    """One update step of Algorithm 1 (eqs. 6, 7, 8), weighted.

    For every cluster k with W_k = sum_{i in I_k} w_i > 0:
      shape (eq. 7): s_k = m_k / ||m_k||,  m_k = sum_{i in I_k} w_i y_i,
                     kept when ||m_k|| <= 1e-6 W_k (mean direction ~ 0);
      gain  (eq. 8): g_k = max(0, sum_{i in I_k} w_i x_i^T s_k / W_k),
                     with the (possibly kept) new shape, summed per sample.
    Clusters with W_k = 0 keep (g_k, s_k).  Returns new (gain, shape).
    """
    X = np.asarray(X, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    gain = np.array(gain, dtype=np.float64, copy=True)
    shape = np.array(shape, dtype=np.float64, copy=True)
    Y = normalize_rows(X)
    K = gain.shape[0]
    for k in range(K):
        members = np.nonzero(assign == k)[0]
        if members.size == 0:
            continue
        Wk = np.sum(w[members])
        if not Wk > 0.0:
            continue
        m = np.sum(w[members, None] * Y[members], axis=0)
        mnorm = np.linalg.norm(m)
        if mnorm > SHAPE_KEEP_REL * Wk:
            shape[k] = m / mnorm
        proj = X[members] @ shape[k]
        gain[k] = max(0.0, float(np.sum(w[members] * proj) / Wk))
    return gain, shape


def gskm_init(X, w, init_rows, assign0=None):
    """Initialisation of Algorithm 1 from K seed rows.

    Shapes are the normalised seed rows (points on the unit sphere).  Gains
    follow eq. (8) over an equal-gain assignment k_i = argmax_k x_i^T s_k
    (lowest k on ties); a cluster that receives no weight takes the norm of
    its seed row.  Passing assign0 uses that assignment instead of the
    equal-gain one (teacher forcing in the parity tests).
    Returns (gain, shape, initial assignment).
    """
    X = np.asarray(X, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    init_rows = np.asarray(init_rows, dtype=np.int64)
    seeds = X[init_rows]
    norms = np.linalg.norm(seeds, axis=1)
    if np.any(norms == 0.0):
        raise ValueError("GSKM initialisation needs nonzero seed rows")
    shape = seeds / (norms[:, None] + EPS)
    if assign0 is None:
        assign0 = np.argmax(X @ shape.T, axis=1).astype(np.int64)
    else:
        assign0 = np.asarray(assign0, np.int64)
    K = shape.shape[0]
    gain = np.empty(K, dtype=np.float64)
    for k in range(K):
        members = np.nonzero(assign0 == k)[0]
        Wk = np.sum(w[members]) if members.size else 0.0
        if Wk > 0.0:
            proj = X[members] @ shape[k]
            gain[k] = max(0.0, float(np.sum(w[members] * proj) / Wk))
        else:
            gain[k] = norms[k]
    return gain, shape, assign0


def gskm(X, w, K, T, init_rows, *, gain=None, shape=None, prev_assign=None):
    """Algorithm 1 (weighted GSKM) on one subspace.

    X: [N, d] data, w: [N] weights (None = all ones), K codewords, at most T
    iterations, init_rows: [K] distinct seed row indices.  Passing gain and
    shape resumes from that codebook instead (then prev_assign, if given, is
    the assignment the stop test compares against at t = 1).

    Returns dict(gain [K], shape [K, d], iters_run, assign [N],
    trace [iters_run]) where trace[t-1] is the weighted distortion of the
    iteration-t assignment measured against the codebook it was made with.
    """
    X = np.asarray(X, dtype=np.float64)
    N = X.shape[0]
    w = np.ones(N) if w is None else np.asarray(w, dtype=np.float64)
    if gain is None:
        gain, shape, prev = gskm_init(X, w, init_rows)
    else:
        gain = np.asarray(gain, np.float64).copy()
        shape = np.asarray(shape, np.float64).copy()
        prev = None if prev_assign is None else np.asarray(prev_assign, np.int64)
    assert gain.shape[0] == K
    trace = []
    iters_run = 0
    assign = prev
    for t in range(1, T + 1):
        assign = gskm_assign(X, gain, shape)
        trace.append(weighted_distortion(X, w, gain, shape, assign))
        gain, shape = gskm_update(X, w, assign, gain, shape)
        iters_run = t
        if prev is not None and np.array_equal(assign, prev):
            break
        prev = assign
    return dict(gain=gain, shape=shape, iters_run=iters_run, assign=assign,
                trace=np.asarray(trace))


# ----------------------------------------------------------------------------
# Gain-shape residual quantisation (Sec. 3, Sec. 5.1): PQ subspaces x RQ stages
# ----------------------------------------------------------------------------

def split_groups(D, d):
    if d <= 0 or D % d != 0:
        raise ValueError("subvector dimension must divide the vector dimension")
    return D // d


def gsrq_encode(X, gains, shapes):
    """Greedy residual encoding with gain-shape codebooks (Sec. 3, 5.1).

    X: [N, D]; gains: [M, G, K]; shapes: [M, G, K, d].  For every subspace g
    and stage m in order: k = argmax_k (2 g_k r^T s_k - g_k^2) on the current
    residual r, then r <- r - g_k s_k.
    Returns (codes [N, M, G] int64, residual [N, D] float64).
    """
    R = np.array(X, dtype=np.float64, copy=True)
    gains = np.asarray(gains, np.float64)
    shapes = np.asarray(shapes, np.float64)
    M, G, K, d = shapes.shape
    N = R.shape[0]
    assert R.shape[1] == G * d
    codes = np.zeros((N, M, G), dtype=np.int64)
    for m in range(M):
        for g in range(G):
            cols = slice(g * d, (g + 1) * d)
            k = gskm_assign(R[:, cols], gains[m, g], shapes[m, g])
            codes[:, m, g] = k
            R[:, cols] -= gains[m, g][k, None] * shapes[m, g][k]
    return codes, R


def gsrq_decode(codes, gains, shapes, M_use=None):
    """Reconstruction as the sum over stages of g s (Sec. 3): a prefix of
    M_use stages may be decoded (Sec. 1).  Returns [N, D] float64."""
    gains = np.asarray(gains, np.float64)
    shapes = np.asarray(shapes, np.float64)
    M, G, K, d = shapes.shape
    M_use = M if M_use is None else int(M_use)
    if not 1 <= M_use <= M:
        raise ValueError("M_use out of range")
    codes = np.asarray(codes, np.int64)
    N = codes.shape[0]
    Xhat = np.zeros((N, G * d), dtype=np.float64)
    for m in range(M_use):
        for g in range(G):
            k = codes[:, m, g]
            Xhat[:, g * d:(g + 1) * d] += gains[m, g][k, None] * shapes[m, g][k]
    return Xhat


def gsrq_train(X, w, d, K, M, T, init_rows):
    """GSRQ calibration (Sec. 5.1): weighted GSKM in every (stage, subspace).

    X: [N, D]; w: [N] (None = ones), shared by every subspace and stage
    (Sec. 5.3); init_rows: [M, G, K] seed rows per stage and subspace, taken
    from that stage's residual.  Stage m trains on the residual left by
    re-encoding stage m-1's input with its final codebook.
    Returns dict(gains [M,G,K], shapes [M,G,K,d], iters_run [M,G]).
    """
    R = np.array(X, dtype=np.float64, copy=True)
    N, D = R.shape
    G = split_groups(D, d)
    gains = np.zeros((M, G, K))
    shapes = np.zeros((M, G, K, d))
    iters = np.zeros((M, G), dtype=np.int64)
    for m in range(M):
        for g in range(G):
            cols = slice(g * d, (g + 1) * d)
            out = gskm(R[:, cols], w, K, T, init_rows[m][g])
            gains[m, g] = out["gain"]
            shapes[m, g] = out["shape"]
            iters[m, g] = out["iters_run"]
        _, R = gsrq_encode(R, gains[m:m + 1], shapes[m:m + 1])
    return dict(gains=gains, shapes=shapes, iters_run=iters)


# ----------------------------------------------------------------------------
# Rate and bit packing
# ----------------------------------------------------------------------------

def bits_per_element(d, K, M):
    """Average bits per element, M log2(K) / d (Sec. 6.2, configurations)."""
    return M * np.log2(K) / d


def code_bits(K):
    b = int(round(np.log2(K)))
    if K < 2 or (1 << b) != K:
        raise ValueError("K must be a power of two >= 2")
    return b


def words_per_row(M, G, K):
    return (M * G * code_bits(K) + 31) // 32


def pack_codes(codes, K):
    """Bit-pack codes [N, M, G] into uint32 rows.

    Code t = m*G + g of a row occupies bits [t*b, t*b + b) of that row's bit
    string, least significant bit first, where bit p lives in word p // 32 at
    position p % 32, and b = log2 K.  Written bit by bit.
    """
    codes = np.asarray(codes, np.int64)
    N, M, G = codes.shape
    b = code_bits(K)
    W = words_per_row(M, G, K)
    out = np.zeros((N, W), dtype=np.uint64)
    flat = codes.reshape(N, M * G)
    for t in range(M * G):
        for u in range(b):
            p = t * b + u
            bit = (flat[:, t] >> u) & 1
            out[:, p // 32] |= bit.astype(np.uint64) << np.uint64(p % 32)
    return out.astype(np.uint32)


def unpack_codes(words, M, G, K):
    words = np.asarray(words, np.uint32).astype(np.uint64)
    N = words.shape[0]
    b = code_bits(K)
    flat = np.zeros((N, M * G), dtype=np.int64)
    for t in range(M * G):
        for u in range(b):
            p = t * b + u
            bit = (words[:, p // 32] >> np.uint64(p % 32)) & np.uint64(1)
            flat[:, t] |= bit.astype(np.int64) << u
    return flat.reshape(N, M, G)


# ----------------------------------------------------------------------------
# Metrics (Sec. 6.1) and the gradient log-weight (Sec. 5.3, Appendix B)
# ----------------------------------------------------------------------------

def metrics(X, Xhat):
    """MSE E||x - xhat||^2, gain error E| ||x|| - ||xhat|| |, cosine E cos(x, xhat)
    over the rows of X (Sec. 6.1).  cos is taken as 0 when either norm is 0."""
    X = np.asarray(X, np.float64)
    Xhat = np.asarray(Xhat, np.float64)
    diff = X - Xhat
    mse = float(np.mean(np.sum(diff * diff, axis=1)))
    nx = np.linalg.norm(X, axis=1)
    nh = np.linalg.norm(Xhat, axis=1)
    gain_err = float(np.mean(np.abs(nx - nh)))
    dots = np.sum(X * Xhat, axis=1)
    denom = nx * nh
    cos = np.where(denom > 0, dots / np.where(denom > 0, denom, 1.0), 0.0)
    return dict(mse=mse, gain_err=gain_err, cos=float(np.mean(cos)))


def log_weight(norms, tau=1.0, eps=1e-8):
    """Appendix B: w = log(1 + lambda * ||grad||), lambda = tau / (median + eps)."""
    norms = np.asarray(norms, np.float64)
    lam = tau / (np.median(norms) + eps)
    return np.log1p(lam * norms)


# ----------------------------------------------------------------------------
# Standard l2 K-means, the baseline GSKM replaces (Sec. 4, Sec. 6.1)
# ----------------------------------------------------------------------------

def kmeans_assign(X, C):
    """Nearest centroid by squared l2 distance, lowest index on ties."""
    X = np.asarray(X, np.float64)
    C = np.asarray(C, np.float64)
    d2 = np.sum((X[:, None, :] - C[None, :, :]) ** 2, axis=2)
    return np.argmin(d2, axis=1).astype(np.int64)


def kmeans_update(X, w, assign, C):
    """Centroid of every cluster with weight = weighted mean of its members;
    clusters without weight keep their centroid.  Returns the new [K, d]."""
    X = np.asarray(X, np.float64)
    w = np.asarray(w, np.float64)
    C = np.array(C, dtype=np.float64, copy=True)
    for k in range(C.shape[0]):
        members = np.nonzero(assign == k)[0]
        Wk = np.sum(w[members]) if members.size else 0.0
        if Wk > 0.0:
            C[k] = np.sum(w[members, None] * X[members], axis=0) / Wk
    return C


def kmeans(X, w, K, T, init_rows, *, centroids=None, prev_assign=None):
    """Weighted Lloyd K-means from seed rows: assign to the nearest centroid
    (lowest index on ties), centroid = weighted mean of its members, empty
    clusters keep their centroid, stop when the assignment repeats.
    Passing centroids resumes from them (prev_assign, if given, is what the
    stop test compares against at t = 1).
    Returns dict(centroids [K, d], iters_run, assign, trace) where trace[t-1]
    is the weighted distortion after the iteration-t update."""
    X = np.asarray(X, np.float64)
    N = X.shape[0]
    w = np.ones(N) if w is None else np.asarray(w, np.float64)
    if centroids is None:
        C = X[np.asarray(init_rows, np.int64)].copy()
        prev = None
    else:
        C = np.array(centroids, dtype=np.float64, copy=True)
        prev = None if prev_assign is None else np.asarray(prev_assign, np.int64)
    assert C.shape[0] == K
    trace = []
    iters_run = 0
    assign = None
    for t in range(1, T + 1):
        assign = kmeans_assign(X, C)
        C = kmeans_update(X, w, assign, C)
        R = X - C[assign]
        trace.append(float(np.sum(w * np.sum(R * R, axis=1))))
        iters_run = t
        if prev is not None and np.array_equal(assign, prev):
            break
        prev = assign
    return dict(centroids=C, iters_run=iters_run, assign=assign,
                trace=np.asarray(trace))


# ----------------------------------------------------------------------------
# One decoding step of attention over a coded KV cache (Appendix C: the
# decoding kernel unpacks the codes, dequantises, applies RoPE and computes
# attention).  Readings (the paper names the steps only):
#   * keys are quantised before RoPE, so RoPE is applied to each dequantised
#     key at its position;
#   * RoPE in the rotate-half form of the LLaMA family: for a head of hd
#     elements, element j < hd/2 and element j + hd/2 form a pair rotated by
#     the angle p * theta_j, theta_j = base^(-2j/hd), p the token position;
#   * the cached tokens of a sequence sit at positions 0 .. L-1 and the query
#     is the newest token, at position L-1 (its own key is in the cache);
#   * grouped-query attention: query head h reads key/value head h // (Hq/Hkv);
#   * softmax scale 1/sqrt(hd); an empty cache (L = 0) gives a zero output.
# ----------------------------------------------------------------------------

def rope_theta(hd, base):
    """theta_j = base^(-2j/hd) for j = 0 .. hd/2 - 1 (float64)."""
    j = np.arange(hd // 2, dtype=np.float64)
    return np.power(float(base), -2.0 * j / hd)


def rope(x, positions, base):
    """Rotate-half RoPE of the last axis of x [..., P, hd] at integer
    positions [P]: pair (j, j + hd/2) is rotated by positions * theta_j."""
    x = np.asarray(x, np.float64)
    hd = x.shape[-1]
    ang = np.asarray(positions, np.float64)[:, None] * rope_theta(hd, base)[None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :hd // 2], x[..., hd // 2:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def attn_weights(q, K, base, scale=None, *, operands_f16=False):
    """Softmax weights of one query token over one sequence's cache:
    p[h, i] = softmax_i(scale * RoPE(q_h, L-1) . RoPE(K[i, h // (Hq/Hkv)], i)).

    q [Hq, hd] before RoPE; K [L, Hkv, hd] dequantised keys before RoPE.
    operands_f16 rounds the rotated query and the rotated keys to float16
    (round to nearest even) before their dot products: the operand precision
    of a float16 matrix-core kernel, not part of the method.
    Returns (p [Hq, L], s [Hq, L] scaled scores), float64."""
    q = np.asarray(q, np.float64)
    K = np.asarray(K, np.float64)
    Hq, hd = q.shape
    L, Hkv = K.shape[0], K.shape[1]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    scale = 1.0 / np.sqrt(hd) if scale is None else float(scale)
    p = np.zeros((Hq, L), dtype=np.float64)
    sc = np.zeros((Hq, L), dtype=np.float64)
    if L == 0:
        return p, sc
    # RoPE of the query at position L-1 (same rotation for every head)
    qr = rope(q[:, None, :], np.array([L - 1]), base)[:, 0, :]
    kr = rope(np.transpose(K, (1, 0, 2)), np.arange(L), base)   # [Hkv, L, hd]
    if operands_f16:
        qr = qr.astype(np.float16).astype(np.float64)
        kr = kr.astype(np.float16).astype(np.float64)
    group = Hq // Hkv
    for h in range(Hq):
        s = (kr[h // group] @ qr[h]) * scale
        e = np.exp(s - np.max(s))
        p[h] = e / np.sum(e)
        sc[h] = s
    return p, sc


def attn_decode(q, K, V, base, scale=None, *, operands_f16=False):
    """Attention of one query token over one sequence's decoded cache.

    q  [Hq, hd]        the newest token's query, before RoPE;
    K  [L, Hkv, hd]    dequantised keys before RoPE, token i at position i;
    V  [L, Hkv, hd]    dequantised values.
    Returns [Hq, hd] float64: o_h = sum_i p[h, i] V[i, h // (Hq/Hkv)] with the
    weights of attn_weights (zero for an empty cache)."""
    q = np.asarray(q, np.float64)
    V = np.asarray(V, np.float64)
    Hq, hd = q.shape
    Hkv = np.asarray(K).shape[1]
    p, _ = attn_weights(q, K, base, scale, operands_f16=operands_f16)
    out = np.zeros((Hq, hd), dtype=np.float64)
    group = Hq // Hkv
    for h in range(Hq):
        out[h] = p[h] @ V[:, h // group, :]
    return out
