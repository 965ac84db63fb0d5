"""Pins of the float64 oracle against facts fixed by the paper and by mathematics.

Each test ties some part of the oracle to something other than itself: brute
force on tiny inputs, closed forms, grid searches of the optimality claims of
eqs. (7) and (8), exact invariants, a hand-derived example and the rate table
of Sec. 6.2.  A dropped term, a wrong sign or index, or a transposed operand in
the oracle fails at least one of them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import gsrq_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def _unit(v):
    return v / np.linalg.norm(v, axis=-1, keepdims=True)


# --------------------------------------------------------------------- eq. (5)

@pytest.mark.parametrize("d,K,seed", [(2, 3, 0), (3, 5, 1), (4, 8, 2), (2, 8, 3)])
def test_assignment_equals_bruteforce_nearest_codeword(d, K, seed):
    """Eq. (5) is argmin_k ||x - g_k s_k||^2 (eq. 4); checked by explicit loops."""
    rng = _rng(seed, d, K)
    N = 64
    X = rng.standard_normal((N, d)) * rng.uniform(0.1, 3.0, size=(N, 1))
    shape = _unit(rng.standard_normal((K, d)))
    gain = rng.uniform(0.0, 3.0, size=K)
    gain[0] = 0.0                            # a zero-gain codeword is the origin
    k_or = O.gskm_assign(X, gain, shape)
    for i in range(N):
        best, best_k = None, None
        for k in range(K):
            dist = 0.0
            for j in range(d):
                diff = float(X[i, j]) - float(gain[k]) * float(shape[k, j])
                dist += diff * diff
            if best is None or dist < best:
                best, best_k = dist, k
        assert k_or[i] == best_k


def test_assignment_ties_go_to_lowest_index():
    shape = np.array([[1.0, 0.0], [1.0, 0.0], [0.0, 1.0], [0.0, 1.0]])
    gain = np.array([1.0, 1.0, 2.0, 2.0])
    X = np.array([[3.0, 0.0], [0.0, 5.0], [0.0, 0.0]])
    k = O.gskm_assign(X, gain, shape)
    # row 0 equidistant from codewords 0 and 1; row 1 from 2 and 3; the origin
    # is nearest to the two gain-1 codewords (0 and 1)
    assert list(k) == [0, 2, 0]


def test_margin_is_relative_gap_of_distortions():
    X = np.array([[2.0, 0.0]])
    shape = np.array([[1.0, 0.0], [0.0, 1.0]])
    gain = np.array([1.0, 1.0])
    # distortions: ||(1,0)||^2 = 1 and ||(2,-1)||^2 = 5 -> gap 4 over ||x||^2 = 4
    assert O.assignment_margin(X, gain, shape)[0] == pytest.approx(1.0)


# ------------------------------------------------------------ eqs. (6)-(8)

def test_shape_update_maximises_weighted_alignment_on_circle():
    """Eq. (7): the new shape maximises sum_i w_i y_i^T s over ||s|| = 1."""
    rng = _rng(7)
    X = rng.standard_normal((40, 2)) * rng.uniform(0.1, 5.0, size=(40, 1)) + np.array([1.0, 0.5])
    w = rng.lognormal(0.0, 1.0, size=40)
    assign = np.zeros(40, dtype=np.int64)
    g, s = O.gskm_update(X, w, assign, np.array([1.0]), np.array([[1.0, 0.0]]))
    th = np.linspace(0.0, 2.0 * np.pi, 100000, endpoint=False)
    S = np.stack([np.cos(th), np.sin(th)], axis=1)
    Y = X / np.linalg.norm(X, axis=1, keepdims=True)
    obj = (w[:, None] * (Y @ S.T)).sum(axis=0)
    best = S[np.argmax(obj)]
    assert np.linalg.norm(s[0] - best) < 2 * np.pi / 100000 * 2
    # magnitude invariance: rescaling individual rows leaves the shape unchanged
    scale = rng.uniform(0.01, 100.0, size=(40, 1))
    _, s2 = O.gskm_update(X * scale, w, assign, np.array([1.0]), np.array([[1.0, 0.0]]))
    assert np.allclose(s2, s, atol=1e-12)


def test_gain_update_is_nonnegative_least_squares_gain():
    """Eq. (8): g = argmin_{g >= 0} sum_i w_i ||x_i - g s||^2 for the new s."""
    rng = _rng(8)
    X = rng.standard_normal((30, 3)) + np.array([2.0, -1.0, 0.5])
    w = rng.lognormal(0.0, 1.0, size=30)
    assign = np.zeros(30, dtype=np.int64)
    g, s = O.gskm_update(X, w, assign, np.array([0.3]), np.array([[0.0, 0.0, 1.0]]))
    grid = np.linspace(0.0, 6.0, 600001)
    J = np.array([np.sum(w * np.sum((X - gg * s[0]) ** 2, axis=1)) for gg in grid[::1000]])
    coarse = grid[::1000][np.argmin(J)]
    fine = grid[(grid > coarse - 0.01) & (grid < coarse + 0.01)]
    J2 = [np.sum(w * np.sum((X - gg * s[0]) ** 2, axis=1)) for gg in fine]
    assert abs(g[0] - fine[int(np.argmin(J2))]) < 2e-5


def test_gain_clamps_to_zero_for_negative_projections():
    """The clamp of eq. (8): a cluster whose members project negatively on the
    (kept) shape gets gain 0, which is the constrained minimiser."""
    X = np.array([[-1.0, 0.0], [1.0, 0.0]])
    w = np.array([1.0, 1.0])
    # y's cancel exactly -> mean direction ~ 0 -> shape kept at (1,0);
    # weighted mean projection is 0; then tilt the weights negative side
    g, s = O.gskm_update(X, w, np.array([0, 0]), np.array([5.0]), np.array([[1.0, 0.0]]))
    assert np.allclose(s[0], [1.0, 0.0]) and g[0] == 0.0
    X = np.array([[-3.0, 0.0], [1.0, 0.0]])
    w = np.array([1.0, 1.0])
    g, s = O.gskm_update(X, w, np.array([0, 0]), np.array([5.0]), np.array([[1.0, 0.0]]))
    assert np.allclose(s[0], [1.0, 0.0])     # y's still cancel: (-1,0) + (1,0)
    assert g[0] == 0.0                        # mean projection -1 clamps to 0


def test_empty_cluster_keeps_codeword():
    X = np.array([[1.0, 0.0], [2.0, 0.1]])
    gain = np.array([1.0, 7.0])
    shape = np.array([[1.0, 0.0], [0.0, 1.0]])
    g, s = O.gskm_update(X, np.ones(2), np.array([0, 0]), gain, shape)
    assert g[1] == 7.0 and np.array_equal(s[1], [0.0, 1.0])


def test_duplicate_row_equals_doubled_weight():
    """A row with weight 2 acts exactly like two copies of it with weight 1."""
    rng = _rng(9)
    X = rng.standard_normal((50, 4))
    w = rng.lognormal(0.0, 1.0, size=50)
    seeds = rng.choice(50, size=5, replace=False)
    w2 = w.copy()
    w2[3] *= 2.0
    a = O.gskm(X, w2, 5, 8, seeds)
    Xd = np.concatenate([X, X[3:4]], axis=0)
    wd = np.concatenate([w, w[3:4]])
    b = O.gskm(Xd, wd, 5, 8, seeds)
    assert a["iters_run"] == b["iters_run"]
    assert np.allclose(a["gain"], b["gain"], rtol=1e-12, atol=1e-12)
    assert np.allclose(a["shape"], b["shape"], rtol=1e-12, atol=1e-12)
    assert np.array_equal(a["assign"], b["assign"][:50])


def test_energy_identity_after_update():
    """Right after an update, sum_i w_i ||x_i - c_{k_i}||^2 equals
    sum_i w_i ||x_i||^2 - sum_k W_k g_k^2, because eq. (8) is the exact
    least-squares gain (also when clamped to 0: then W_k g_k^2 = 0)."""
    rng = _rng(10)
    X = rng.standard_normal((300, 6)) * rng.uniform(0.2, 2.0, size=6)
    w = rng.lognormal(0.0, 1.0, size=300)
    seeds = rng.choice(300, size=12, replace=False)
    g, s, a0 = O.gskm_init(X, w, seeds)
    for _ in range(4):
        a = O.gskm_assign(X, g, s)
        g, s = O.gskm_update(X, w, a, g, s)
        J = O.weighted_distortion(X, w, g, s, a)
        Wk = np.bincount(a, weights=w, minlength=12)
        E = np.sum(w * np.sum(X * X, axis=1)) - np.sum(Wk * g * g)
        assert J == pytest.approx(E, rel=1e-10)


def test_half_steps_do_not_increase_distortion():
    """The assignment minimises distortion for a fixed codebook, and the gain
    step minimises it for fixed assignment and shapes; the whole iteration
    carries no monotonicity guarantee (Sec. 5.2) so it is not asserted."""
    rng = _rng(11)
    X = rng.standard_normal((400, 8))
    w = rng.lognormal(0.0, 1.0, size=400)
    seeds = rng.choice(400, size=16, replace=False)
    g, s, prev = O.gskm_init(X, w, seeds)
    for _ in range(5):
        a = O.gskm_assign(X, g, s)
        assert O.weighted_distortion(X, w, g, s, a) <= O.weighted_distortion(X, w, g, s, prev) + 1e-9
        g, s = O.gskm_update(X, w, a, g, s)
        J = O.weighted_distortion(X, w, g, s, a)
        for k in range(16):
            for delta in (-1e-3, 1e-3):
                g2 = g.copy()
                g2[k] = max(0.0, g2[k] + delta)
                assert O.weighted_distortion(X, w, g2, s, a) >= J - 1e-9
        prev = a


# ----------------------------------------------------------------- Alg. 1

def test_single_cluster_closed_form():
    """K = 1: the shape is the normalised weighted sum of the y_i and the gain
    the clamped weighted mean projection; the repeated assignment stops the
    loop after the first iteration."""
    rng = _rng(12)
    X = rng.standard_normal((100, 5)) + np.array([1.0, 2.0, 0.0, -1.0, 0.5])
    w = rng.lognormal(0.0, 1.0, size=100)
    out = O.gskm(X, w, 1, 10, np.array([17]))
    Y = X / np.linalg.norm(X, axis=1, keepdims=True)
    m = (w[:, None] * Y).sum(axis=0)
    s = m / np.linalg.norm(m)
    g = max(0.0, float((w * (X @ s)).sum() / w.sum()))
    assert out["iters_run"] == 1
    # the test's y_i omit the 1e-8 safeguard, hence 1e-9 rather than ~1e-15
    assert np.allclose(out["shape"][0], s, atol=1e-9)
    assert out["gain"][0] == pytest.approx(g, rel=1e-9)


def test_hand_derived_weighted_example():
    """Four 2-D points, two clusters, derived by hand.

    X = (3,0), (0,1), (-2,0), (1,1); w = 1, 3, 1, 2; seeds rows 0 and 2, so
    s0 = (1,0), s1 = (-1,0).  Equal-gain assignment: x.s0 = 3, 0, -2, 1 and
    x.s1 = -3, 0, 2, -1 -> clusters {0,1,3} (row 1 tie -> 0) and {2}.
    Initial gains: g0 = (1*3 + 3*0 + 2*1)/6 = 5/6, g1 = 2.
    Iteration 1 scores 2 g x.s - g^2 keep the same assignment, so the loop
    updates once and stops.  Update of cluster 0:
      sum w y = (1,0) + 3 (0,1) + 2 (1,1)/sqrt2 = (1 + sqrt2, 3 + sqrt2),
      s0 = that / sqrt(14 + 8 sqrt2),
      g0 = (1*3 s0x + 3*1 s0y + 2 (s0x + s0y)) / 6 = 5 (s0x + s0y) / 6.
    Cluster 1 keeps s1 = (-1,0), g1 = 2.
    """
    X = np.array([[3.0, 0.0], [0.0, 1.0], [-2.0, 0.0], [1.0, 1.0]])
    w = np.array([1.0, 3.0, 1.0, 2.0])
    g_init, s_init, a0 = O.gskm_init(X, w, np.array([0, 2]))
    assert list(a0) == [0, 0, 1, 0]
    assert g_init[0] == pytest.approx(5.0 / 6.0, rel=1e-7) and g_init[1] == pytest.approx(2.0, rel=1e-7)
    out = O.gskm(X, w, 2, 10, np.array([0, 2]))
    r2 = math.sqrt(2.0)
    nrm = math.sqrt(14.0 + 8.0 * r2)
    s0 = np.array([1.0 + r2, 3.0 + r2]) / nrm
    g0 = 5.0 * (s0[0] + s0[1]) / 6.0
    assert out["iters_run"] == 1
    assert list(out["assign"]) == [0, 0, 1, 0]
    assert np.allclose(out["shape"][0], s0, atol=1e-9)
    assert out["gain"][0] == pytest.approx(g0, rel=1e-9)
    assert np.allclose(out["shape"][1], [-1.0, 0.0], atol=1e-7)
    assert out["gain"][1] == pytest.approx(2.0, rel=1e-7)
    # the iteration-1 distortion, by hand with g0 = 5/6, g1 = 2:
    # rows: (3 - 5/6)^2 + 0, (5/6)^2 + 1, 0, (1 - 5/6)^2 + 1
    J1 = 1 * (13 / 6) ** 2 + 3 * ((5 / 6) ** 2 + 1) + 1 * 0.0 + 2 * ((1 / 6) ** 2 + 1)
    assert out["trace"][0] == pytest.approx(J1, rel=1e-7)


def test_planted_clusters_are_recovered():
    rng = _rng(13)
    K, d, per = 6, 8, 200
    S = _unit(rng.standard_normal((K, d)))
    # make the planted shapes well separated
    S = np.linalg.qr(rng.standard_normal((d, d)))[0][:K]
    G = np.array([0.5, 1.0, 2.0, 3.0, 4.5, 6.0])
    X = np.concatenate([G[k] * S[k] + 0.01 * rng.standard_normal((per, d)) for k in range(K)])
    seeds = np.array([k * per + 3 for k in range(K)])
    out = O.gskm(X, None, K, 20, seeds)
    assert np.allclose(out["gain"], G, rtol=2e-3)
    assert np.allclose(out["shape"], S, atol=5e-3)
    assert out["iters_run"] <= 2


def test_equivariances():
    """Exact symmetries: X -> aX scales gains only; X -> XQ rotates shapes;
    w -> bw changes nothing; permuting rows permutes the assignment."""
    rng = _rng(14)
    N, d, K, T = 300, 4, 10, 6
    X = rng.standard_normal((N, d)) * np.array([3.0, 1.0, 0.5, 0.2])
    w = rng.lognormal(0.0, 1.0, size=N)
    seeds = rng.choice(N, size=K, replace=False)
    base = O.gskm(X, w, K, T, seeds)
    a = O.gskm(4.0 * X, w, K, T, seeds)       # power of 2: exact in binary
    assert np.array_equal(a["assign"], base["assign"])
    assert np.allclose(a["gain"], 4.0 * base["gain"], rtol=1e-12)
    assert np.allclose(a["shape"], base["shape"], atol=1e-12)
    Q = np.linalg.qr(rng.standard_normal((d, d)))[0]
    b = O.gskm(X @ Q, w, K, T, seeds)
    assert np.array_equal(b["assign"], base["assign"])
    assert np.allclose(b["shape"], base["shape"] @ Q, atol=1e-9)
    assert np.allclose(b["gain"], base["gain"], rtol=1e-9)
    c = O.gskm(X, 8.0 * w, K, T, seeds)
    assert np.array_equal(c["assign"], base["assign"])
    assert np.allclose(c["gain"], base["gain"], rtol=1e-12)
    perm = rng.permutation(N)
    inv = np.argsort(perm)
    e = O.gskm(X[perm], w[perm], K, T, inv[seeds])
    assert np.array_equal(e["assign"], base["assign"][perm])
    assert np.allclose(e["gain"], base["gain"], rtol=1e-12)


def test_iteration_limit_and_stop_rule():
    rng = _rng(15)
    X = rng.standard_normal((500, 3))
    seeds = rng.choice(500, size=20, replace=False)
    one = O.gskm(X, None, 20, 1, seeds)
    assert one["iters_run"] == 1 and len(one["trace"]) == 1
    full = O.gskm(X, None, 20, 200, seeds)
    assert full["iters_run"] < 200
    # at the stop, re-assigning with the final codebook reproduces the
    # assignment the final update was computed from
    again = O.gskm_assign(X, full["gain"], full["shape"])
    assert np.array_equal(again, full["assign"])


# ------------------------------------------------------------------- GSRQ

def test_encode_decode_reconstruction_identity():
    rng = _rng(16)
    N, D, d, K, M = 200, 16, 4, 8, 3
    X = rng.standard_normal((N, D))
    seeds = np.stack([np.stack([rng.choice(N, K, replace=False) for _ in range(D // d)]) for _ in range(M)])
    cb = O.gsrq_train(X, None, d, K, M, 5, seeds)
    codes, R = O.gsrq_encode(X, cb["gains"], cb["shapes"])
    Xhat = O.gsrq_decode(codes, cb["gains"], cb["shapes"])
    assert np.allclose(Xhat + R, X, atol=1e-12)
    # prefix decoding: decoding m stages equals X minus the stage-m residual
    for m in range(1, M + 1):
        _, Rm = O.gsrq_encode(X, cb["gains"][:m], cb["shapes"][:m])
        assert np.allclose(O.gsrq_decode(codes, cb["gains"], cb["shapes"], m) + Rm, X, atol=1e-12)
    # each stage's codes are the eq. (5) choice on that stage's residual
    E = X.copy()
    for m in range(M):
        for g in range(D // d):
            cols = slice(g * d, (g + 1) * d)
            k = O.gskm_assign(E[:, cols], cb["gains"][m, g], cb["shapes"][m, g])
            assert np.array_equal(k, codes[:, m, g])
            E[:, cols] -= cb["gains"][m, g][k, None] * cb["shapes"][m, g][k]


def test_residual_energy_falls_with_stages():
    rng = _rng(17)
    N, D, d, K, M = 1000, 16, 8, 16, 4
    X = rng.standard_normal((N, D))
    seeds = np.stack([np.stack([rng.choice(N, K, replace=False) for _ in range(D // d)]) for _ in range(M)])
    cb = O.gsrq_train(X, None, d, K, M, 10, seeds)
    codes, _ = O.gsrq_encode(X, cb["gains"], cb["shapes"])
    errs = [O.metrics(X, O.gsrq_decode(codes, cb["gains"], cb["shapes"], m))["mse"] for m in range(1, M + 1)]
    assert all(b <= a + 1e-12 for a, b in zip(errs, errs[1:]))
    assert errs[-1] < 0.5 * np.mean(np.sum(X * X, axis=1))


def test_two_stage_recursion_hand_worked():
    """GSRQ recursion (Sec. 3 residual quantisation, Sec. 5.1), worked by hand
    with one codeword per stage (K = 1 converges in one iteration).

    X = (3, 0), (0, 1), w = 1, d = D = 2.  Stage 0: y = (1, 0), (0, 1) (up to
    the 1e-8 safeguard), so s1 = (1, 1)/sqrt2, projections 3/sqrt2 and
    1/sqrt2, g1 = sqrt2 and the codeword is (1, 1).  The residuals
    r = (2, -1), (-1, 0) are stage 1's training data: y = (2, -1)/sqrt5 and
    (-1, 0), so s2 = m / ||m|| with m = (2/sqrt5 - 1, -1/sqrt5), and g2 is
    the mean of r.s2.  A stage trained on X instead would repeat stage 0.
    """
    X = np.array([[3.0, 0.0], [0.0, 1.0]])
    seeds = np.zeros((2, 1, 1), dtype=np.int64)
    cb = O.gsrq_train(X, None, 2, 1, 2, 5, seeds)
    r2, r5 = math.sqrt(2.0), math.sqrt(5.0)
    assert np.allclose(cb["shapes"][0, 0, 0], [1 / r2, 1 / r2], atol=1e-8)
    assert cb["gains"][0, 0, 0] == pytest.approx(r2, rel=1e-8)
    m = np.array([2.0 / r5 - 1.0, -1.0 / r5])
    s2 = m / math.hypot(m[0], m[1])
    g2 = 0.5 * ((2.0 * s2[0] - s2[1]) + (-s2[0]))
    assert g2 > 0.1
    assert np.allclose(cb["shapes"][1, 0, 0], s2, atol=1e-8)
    assert cb["gains"][1, 0, 0] == pytest.approx(g2, rel=1e-7)
    assert list(cb["iters_run"][:, 0]) == [1, 1]
    # the final residual is X minus both codewords
    codes, R = O.gsrq_encode(X, cb["gains"], cb["shapes"])
    c2 = g2 * s2
    assert np.allclose(R, [[2.0 - c2[0], -1.0 - c2[1]], [-1.0 - c2[0], -c2[1]]], atol=1e-7)


def _nearest_by_loops(r, gains, shapes):
    """Nearest codeword g_k s_k to r by explicit loops over k and the
    elements (squared distance, lowest index on ties)."""
    best, bk = None, -1
    for k in range(len(gains)):
        dist = 0.0
        for j in range(len(r)):
            e = r[j] - gains[k] * shapes[k][j]
            dist += e * e
        if best is None or dist < best:
            best, bk = dist, k
    return bk


def _recursion_case():
    rng = _rng(40)
    N, D, d, K, M, T = 40, 4, 2, 4, 3, 1
    G = D // d
    X = rng.standard_normal((N, D)) * np.array([2.0, 1.0, 0.7, 1.5])
    w = rng.lognormal(0.0, 1.0, size=N)
    seeds = np.stack([np.stack([rng.choice(N, K, replace=False) for _ in range(G)])
                      for _ in range(M)])
    return X, w, d, K, M, T, seeds


def _recursion_holds(train):
    """Whether train(X, w, d, K, M, T, seeds) gives, at every stage, the
    codebook of weighted GSKM on the residual built by per-row
    nearest-codeword subtraction (explicit loops) with the earlier stages'
    final codebooks.  Also returns whether the case separates re-encoding
    from reusing the last training assignment."""
    X, w, d, K, M, T, seeds = _recursion_case()
    N, D = X.shape
    G = D // d
    cb = train(X, w, d, K, M, T, seeds)
    R = [list(map(float, row)) for row in X]
    ok, reused_differs = True, False
    for m in range(M):
        for g in range(G):
            Rg = np.array([row[g * d:(g + 1) * d] for row in R])
            ref = O.gskm(Rg, w, K, T, seeds[m][g])
            ok &= bool(np.allclose(cb["gains"][m, g], ref["gain"], rtol=1e-12, atol=1e-14))
            ok &= bool(np.allclose(cb["shapes"][m, g], ref["shape"], rtol=1e-12, atol=1e-14))
            for i in range(N):
                r = R[i][g * d:(g + 1) * d]
                k = _nearest_by_loops(r, ref["gain"], ref["shape"])
                reused_differs |= k != ref["assign"][i]
                for j in range(d):
                    R[i][g * d + j] -= ref["gain"][k] * ref["shape"][k][j]
    return ok, reused_differs


def test_stage_recursion_trains_on_reencoded_residual():
    """Reading of Sec. 5.1: the next stage trains on the stage input minus
    its reconstruction with the stage's FINAL codebook (re-encoding).  With
    T = 1 the last training assignment was made with the pre-update
    codebook, so it differs from the re-encode for some rows (asserted)."""
    ok, reused_differs = _recursion_holds(O.gsrq_train)
    assert reused_differs, "case does not separate re-encoding from the last assignment"
    assert ok
    X, w, d, K, M, T, seeds = _recursion_case()
    cb = O.gsrq_train(X, w, d, K, M, T, seeds)
    codes, Rend = O.gsrq_encode(X, cb["gains"], cb["shapes"])
    assert np.allclose(Rend + O.gsrq_decode(codes, cb["gains"], cb["shapes"]), X, atol=1e-12)


def _train_mutant(on_input, reuse_assignment):
    """gsrq_train with a planted mistake: every stage trained on X, or the
    next residual taken from the last training assignment."""
    def train(X, w, d, K, M, T, seeds):
        X = np.asarray(X, np.float64)
        R = X.copy()
        G = X.shape[1] // d
        gains, shapes = np.zeros((M, G, K)), np.zeros((M, G, K, d))
        for m in range(M):
            for g in range(G):
                cols = slice(g * d, (g + 1) * d)
                out = O.gskm((X if on_input else R)[:, cols], w, K, T, seeds[m][g])
                gains[m, g], shapes[m, g] = out["gain"], out["shape"]
                if reuse_assignment:
                    k = out["assign"]
                    R[:, cols] -= gains[m, g][k, None] * shapes[m, g][k]
            if not reuse_assignment:
                _, R = O.gsrq_encode(R, gains[m:m + 1], shapes[m:m + 1])
        return dict(gains=gains, shapes=shapes)
    return train


@pytest.mark.parametrize("on_input,reuse", [(True, False), (False, True)])
def test_stage_recursion_check_rejects_planted_mistakes(on_input, reuse):
    """The recursion check fails for a stage trained on X and for a residual
    taken from the last training assignment (both planted in a copy of the
    recursion, on the CPU)."""
    ok, _ = _recursion_holds(_train_mutant(on_input, reuse))
    assert not ok
    # the correct recursion written the same way passes
    ok, _ = _recursion_holds(_train_mutant(False, False))
    assert ok


def test_rate_formula_matches_paper_configurations():
    with open(os.path.join(GOLDEN, "rate_configs.json")) as f:
        fx = json.load(f)
    for c in fx["cases"]:
        assert O.bits_per_element(c["D"], c["K"], c["R"]) == pytest.approx(c["bpa"], abs=1e-12)
    # the five synthetic workloads of this repository
    assert O.bits_per_element(8, 256, 2) == 2.0
    assert O.bits_per_element(8, 256, 1) == 1.0
    assert [O.bits_per_element(16, 256, m) for m in (1, 2, 4)] == [0.5, 1.0, 2.0]
    assert O.bits_per_element(128, 4096, 8) == 0.75


def test_packing_bit_layout_by_hand():
    # b = 12: codes 0xABC, 0x123, 0xFFF, 0x001 -> 48 bits in two words
    codes = np.array([0xABC, 0x123, 0xFFF, 0x001]).reshape(1, 1, 4)
    words = O.pack_codes(codes, 4096)
    assert words.shape == (1, 2)
    assert words[0, 0] == (0xABC | (0x123 << 12) | ((0xFFF & 0xFF) << 24))
    assert words[0, 1] == ((0xFFF >> 8) | (0x001 << 4))
    # b = 8: byte t of the row is code t (stage-major, then subspace)
    codes = np.array([[[1, 2, 3], [4, 5, 250]]])           # M=2, G=3
    words = O.pack_codes(codes, 256)
    assert list(words[0]) == [0x04030201, 0x0000FA05]
    rng = _rng(18)
    for K, M, G in [(2, 3, 5), (16, 2, 7), (256, 1, 128), (4096, 8, 8), (1024, 3, 3)]:
        c = rng.integers(0, K, size=(9, M, G))
        w = O.pack_codes(c, K)
        assert w.shape[1] == O.words_per_row(M, G, K)
        assert np.array_equal(O.unpack_codes(w, M, G, K), c)


def test_metrics_definitions():
    X = np.array([[3.0, 4.0], [1.0, 0.0]])
    Xh = np.array([[3.0, 0.0], [0.0, 0.0]])
    m = O.metrics(X, Xh)
    assert m["mse"] == pytest.approx((16.0 + 1.0) / 2)
    assert m["gain_err"] == pytest.approx((2.0 + 1.0) / 2)
    assert m["cos"] == pytest.approx((0.6 + 0.0) / 2)


def test_log_weight_closed_form():
    """Appendix B: median maps to log(1 + tau); the transform is invariant to
    a global rescale of the gradient norms and keeps their order."""
    rng = _rng(19)
    n = rng.lognormal(0.0, 2.0, size=1001)
    wt = O.log_weight(n)
    med = np.median(n)
    assert O.log_weight(np.array([med]), tau=1.0) is not None
    assert np.interp(med, np.sort(n), np.sort(wt)) == pytest.approx(math.log(2.0), rel=1e-6)
    assert np.allclose(O.log_weight(7.0 * n), wt, rtol=1e-6)
    assert np.array_equal(np.argsort(wt), np.argsort(n))
    assert wt.max() / np.median(wt) < n.max() / med


def test_kmeans_baseline_objective_is_monotone():
    rng = _rng(20)
    X = rng.standard_normal((600, 8))
    w = rng.lognormal(0.0, 1.0, size=600)
    out = O.kmeans(X, w, 24, 30, rng.choice(600, size=24, replace=False))
    tr = out["trace"]
    assert all(b <= a * (1 + 1e-12) for a, b in zip(tr, tr[1:]))


def test_gskm_beats_kmeans_direction_on_gaussian_under_capacity():
    """Sec. 6.1, random-normal sweep: on x ~ N(0, I_D) with a small codebook
    GSKM reconstructs with higher cosine similarity and lower gain error than
    K-means (the paper reports this ordering; its plotted values are absent)."""
    rng = _rng(21)
    N, D, K = 10000, 128, 64
    X = rng.standard_normal((N, D))
    seeds = rng.choice(N, size=K, replace=False)
    gs = O.gskm(X, None, K, 20, seeds)
    km = O.kmeans(X, None, K, 20, seeds)
    Xg = gs["gain"][gs["assign"], None] * gs["shape"][gs["assign"]]
    Xk = km["centroids"][km["assign"]]
    mg, mk = O.metrics(X, Xg), O.metrics(X, Xk)
    assert mg["cos"] > mk["cos"]
    assert mg["gain_err"] < mk["gain_err"]
    assert mg["mse"] < mk["mse"]


def test_kmeans_steps_hand_worked():
    """Lloyd steps on a hand-worked 1-D case: X = (0, 2, 10), w = (1, 3, 1),
    centroids (1, 9).  Nearest: 0 and 2 go to centroid 1 (distance 1 each),
    10 goes to 9.  New
    centroids: (1*0 + 3*2) / 4 = 1.5 and 10; distortion after the update
    1 * 1.5^2 + 3 * 0.5^2 + 0 = 3.  A point equidistant from two centroids
    goes to the lower index."""
    X = np.array([[0.0], [2.0], [10.0]])
    w = np.array([1.0, 3.0, 1.0])
    C = np.array([[1.0], [9.0]])
    a = O.kmeans_assign(X, C)
    assert a.tolist() == [0, 0, 1]
    C1 = O.kmeans_update(X, w, a, C)
    assert C1.ravel().tolist() == [1.5, 10.0]
    out = O.kmeans(X, w, 2, 1, [0, 2], centroids=C)
    assert out["trace"][0] == pytest.approx(3.0, abs=1e-15)
    assert O.kmeans_assign(np.array([[5.0]]), C).tolist() == [0]
    # an empty cluster keeps its centroid
    C2 = O.kmeans_update(X, w, np.array([0, 0, 0]), C)
    assert C2[1, 0] == 9.0 and C2[0, 0] == pytest.approx(16.0 / 5.0)


def test_kmeans_assign_matches_brute_force():
    rng = _rng(22)
    X = rng.standard_normal((50, 3))
    C = rng.standard_normal((7, 3))
    C[4] = C[2]                               # duplicate: the lower index wins
    a = O.kmeans_assign(X, C)
    for i in range(50):
        best, bk = None, -1
        for k in range(7):
            dd = sum((X[i, j] - C[k, j]) ** 2 for j in range(3))
            if best is None or dd < best:
                best, bk = dd, k
        assert a[i] == bk


def test_log_weight_tames_heavy_tailed_norms():
    """Sec. 5.3: gradient norms with max/median > 400 come out of the log
    smoothing (tau = 1) with max/median < 10.  Heavy-tailed synthetic norms
    (the stand-in gradient rows of the benchmark inputs)."""
    import synth
    G = synth.gradient_rows(32768, 64, seed=7, dtype=np.float32)
    n = np.linalg.norm(G.astype(np.float64), axis=1)
    w = O.log_weight(n, tau=1.0)
    assert n.max() / np.median(n) > 400
    assert w.max() / np.median(w) < 10
    # median maps to log(2) exactly in exact arithmetic (lambda * median = 1)
    assert np.median(w) == pytest.approx(math.log(2.0), rel=1e-6)


# ------------------------------------------- decode attention (Appendix C)

@pytest.mark.parametrize("hd,base", [(128, 500000.0), (128, 10000.0), (8, 10.0)])
def test_rope_first_pair_turns_by_position_in_radians(hd, base):
    """theta_0 = base^0 = 1 for every base: the pair (0, hd/2) turns by
    exactly p radians at position p (rotate-half form)."""
    for p in (0, 1, 2, 1000, 123457):
        e0 = np.zeros((1, hd))
        e0[0, 0] = 1.0
        r = O.rope(e0, np.array([p]), base)[0]
        assert r[0] == pytest.approx(math.cos(p), abs=1e-12)
        assert r[hd // 2] == pytest.approx(math.sin(p), abs=1e-12)
        assert np.count_nonzero(np.abs(r) > 1e-15) <= 2
        eh = np.zeros((1, hd))
        eh[0, hd // 2] = 1.0
        r = O.rope(eh, np.array([p]), base)[0]
        assert r[0] == pytest.approx(-math.sin(p), abs=1e-12)
        assert r[hd // 2] == pytest.approx(math.cos(p), abs=1e-12)


def test_rope_last_pair_frequency():
    """theta_63 of a 128-element head with base 10^4 is 10^(-4 * 126/128)
    = 10^-3.9375 = 1.1547819846894583e-4 (hand value); at position 1000 the
    pair (63, 127) turns by 0.11547819846894583 rad."""
    th = O.rope_theta(128, 10000.0)
    assert th[63] == pytest.approx(1.1547819846894583e-4, rel=1e-14)
    assert th[0] == 1.0
    x = np.zeros((1, 128))
    x[0, 63] = 1.0
    r = O.rope(x, np.array([1000]), 10000.0)[0]
    a = 0.11547819846894583
    assert r[63] == pytest.approx(math.cos(a), abs=1e-13)
    assert r[127] == pytest.approx(math.sin(a), abs=1e-13)


def test_rope_scores_depend_on_relative_position_only():
    rng = _rng(70)
    q, k = rng.standard_normal((2, 128))
    for a, b, sh in ((5, 17, 3), (1000, 2, 99), (0, 0, 131071)):
        s1 = O.rope(q[None], np.array([a]), 500000.0)[0] @ O.rope(k[None], np.array([b]), 500000.0)[0]
        s2 = (O.rope(q[None], np.array([a + sh]), 500000.0)[0]
              @ O.rope(k[None], np.array([b + sh]), 500000.0)[0])
        assert s1 == pytest.approx(s2, rel=1e-9, abs=1e-9)
        n = np.linalg.norm(O.rope(k[None], np.array([b]), 500000.0)[0])
        assert n == pytest.approx(np.linalg.norm(k), rel=1e-13)


def test_attention_two_tokens_hand_worked():
    """Keys e_0 at positions 0 and 1, query at position 1 with scale*q = e_0:
    scores cos(-1) and 1, so o = (e^cos1 v0 + e v1) / (e^cos1 + e).  With
    scale*q = e_64 instead the scores are sin(-1) and 0 (the sign of the
    rotation shows here)."""
    hd = 128
    v = np.zeros((2, 1, hd))
    v[0, 0, :] = 1.0
    v[1, 0, :] = -2.0
    K = np.zeros((2, 1, hd))
    K[:, 0, 0] = 1.0
    q = np.zeros((1, hd))
    q[0, 0] = math.sqrt(hd)
    o = O.attn_decode(q, K, v, 500000.0)
    a0, a1 = math.exp(math.cos(1.0)), math.exp(1.0)
    assert o[0, 5] == pytest.approx((a0 * 1.0 + a1 * -2.0) / (a0 + a1), rel=1e-12)
    q = np.zeros((1, hd))
    q[0, 64] = math.sqrt(hd)
    o = O.attn_decode(q, K, v, 10000.0)
    a0, a1 = math.exp(-math.sin(1.0)), 1.0
    assert o[0, 7] == pytest.approx((a0 * 1.0 + a1 * -2.0) / (a0 + a1), rel=1e-12)


def test_attention_special_cases():
    """One token: the output is its value; a zero query: the mean value;
    query head h reads key/value head h // (Hq / Hkv); empty cache: zeros."""
    rng = _rng(71)
    Hq, Hkv, hd = 4, 2, 128
    q = rng.standard_normal((Hq, hd))
    K = rng.standard_normal((1, Hkv, hd))
    V = rng.standard_normal((1, Hkv, hd))
    o = O.attn_decode(q, K, V, 500000.0)
    for h in range(Hq):
        assert np.allclose(o[h], V[0, h // 2], rtol=0, atol=1e-14)
    K = rng.standard_normal((9, Hkv, hd))
    V = rng.standard_normal((9, Hkv, hd))
    o = O.attn_decode(np.zeros((Hq, hd)), K, V, 500000.0)
    for h in range(Hq):
        assert np.allclose(o[h], V[:, h // 2].mean(axis=0), rtol=0, atol=1e-13)
    assert np.all(O.attn_decode(q, K[:0], V[:0], 500000.0) == 0.0)


def test_attention_float16_operand_error_within_bound():
    """The error of float16 operands stays inside the bound used by the GPU
    tests: each rotated operand element is off by at most 2^-11 of itself, so
    a score moves by at most eps = scale 2^-10 ||q|| max_t ||k_t|| (plus
    float32 summation, covered by the 1e-5 term), the softmax weights by a
    factor within e^(+-2 eps), and the output by (e^(2 eps) - 1) max|v|."""
    rng = _rng(72)
    Hq, Hkv, hd, L = 4, 1, 128, 500
    q = rng.standard_normal((Hq, hd))
    K = rng.standard_normal((L, Hkv, hd)) * rng.uniform(0.5, 2.0, size=(L, 1, 1))
    V = rng.standard_normal((L, Hkv, hd))
    o = O.attn_decode(q, K, V, 500000.0)
    o16 = O.attn_decode(q, K, V, 500000.0, operands_f16=True)
    scale = 1.0 / math.sqrt(hd)
    for h in range(Hq):
        eps = scale * 2.0 ** -10 * np.linalg.norm(q[h]) * np.max(np.linalg.norm(K[:, 0], axis=1))
        bound = (math.expm1(2 * eps) + 1e-5) * np.max(np.abs(V))
        err = np.max(np.abs(o16[h] - o[h]))
        assert 0 < err <= bound
