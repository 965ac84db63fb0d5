"""GPU parity of the HIP path against the float64 oracle, through the C ABI.

Inputs are seeded and synthetic (synth.py); every expected value comes from
oracle/ on the same inputs.  Index parity follows the margin rule (equal
wherever the relative top-2 margin exceeds 1e-4; below it the GPU's choice
must be within the margin); codebooks and reconstructions agree to 1e-5
relative (float32 path), updates compared teacher-forced (the oracle's update
applied to the GPU's own assignment and previous codebook).
"""
import numpy as np
import pytest

import synth
from oracle import gsrq_oracle as O
from tests.gpu_util import CB_RTOL, MARGIN, check_assignment, rel_err, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2607_01065_amd import gsrq as B  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


def _rng(*k):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(k))))


def random_codebook(X, M, G, K, d, seed, zero_gain=True, dup=True):
    """Codebooks for encode tests: unit shapes, gains near the data norms."""
    rng = _rng(seed, M, G, K, d)
    sh = rng.standard_normal((M, G, K, d))
    sh /= np.linalg.norm(sh, axis=-1, keepdims=True)
    Xg = np.asarray(X, np.float64).reshape(X.shape[0], G, d)
    typ = np.median(np.linalg.norm(Xg, axis=-1), axis=0)          # [G]
    gain = typ[None, :, None] * rng.uniform(0.3, 1.6, size=(M, G, K)) / (1 + np.arange(M))[:, None, None]
    if zero_gain:
        gain[:, :, 1] = 0.0
    if dup and K >= 4:
        sh[:, :, 3] = sh[:, :, 2]
        gain[:, :, 3] = gain[:, :, 2]
    return gain.astype(np.float32), sh.astype(np.float32)


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def unpack(codes_t, M, G, K):
    return O.unpack_codes(codes_t.cpu().numpy().view(np.uint32), M, G, K)


@pytest.mark.parametrize("dtype", [np.float16, np.float32])
@pytest.mark.parametrize("N,D,d,K", [(1000, 64, 8, 256), (777, 24, 4, 16), (129, 16, 8, 2)])
def test_encode_single_stage(dtype, N, D, d, K):
    say("encode single stage", dtype.__name__, N, D, d, K)
    X, _, _ = synth.small_case(N, D, d, K, 1, seed=11, dtype=dtype)
    G = D // d
    gain, shape = random_codebook(X, 1, G, K, d, seed=5)
    codes, res = B.encode(to_dev(X), to_dev(gain), to_dev(shape), residual=True)
    torch.cuda.synchronize()
    k = unpack(codes, 1, G, K)
    R = res.cpu().numpy().astype(np.float64)
    X64 = X.astype(np.float64)
    below = 0
    for g in range(G):
        cols = slice(g * d, (g + 1) * d)
        _, nb, _ = check_assignment(X64[:, cols], gain[0, g], shape[0, g], k[:, 0, g], f"g{g}")
        below += nb
        ref = X64[:, cols] - gain[0, g].astype(np.float64)[k[:, 0, g], None] * shape[0, g].astype(np.float64)[k[:, 0, g]]
        scale = np.maximum(np.abs(X64[:, cols]).max(), 1e-3)
        assert np.allclose(R[:, cols], ref, rtol=CB_RTOL, atol=1e-6 * scale)
    say("below-margin index differences:", below, "of", N * G)


@pytest.mark.parametrize("M,K,d,D", [(3, 16, 4, 24), (2, 256, 8, 32), (4, 8, 2, 6)])
def test_encode_multi_stage_teacher_forced(M, K, d, D):
    say("encode multi stage", M, K, d, D)
    N = 613
    X, w, seeds = synth.small_case(N, D, d, K, M, seed=12, dtype=np.float32)
    G = D // d
    cb = O.gsrq_train(X, w, d, K, M, 4, seeds)
    gain = cb["gains"].astype(np.float32)
    shape = cb["shapes"].astype(np.float32)
    codes, res = B.encode(to_dev(X), to_dev(gain), to_dev(shape), residual=True)
    torch.cuda.synchronize()
    k = unpack(codes, M, G, K)
    R = X.astype(np.float64)
    for m in range(M):
        for g in range(G):
            cols = slice(g * d, (g + 1) * d)
            check_assignment(R[:, cols], gain[m, g], shape[m, g], k[:, m, g], f"m{m} g{g}")
            kk = k[:, m, g]
            R[:, cols] -= gain[m, g].astype(np.float64)[kk, None] * shape[m, g].astype(np.float64)[kk]
    Rg = res.cpu().numpy().astype(np.float64)
    scale = np.abs(X).max()
    assert np.allclose(Rg, R, rtol=1e-5, atol=1e-6 * scale)


@pytest.mark.parametrize("M,K,d,D,N", [(1, 256, 8, 64, 1000), (3, 16, 4, 24, 333), (2, 4096 // 16, 8, 16, 50),
                                        (3, 8, 2, 6, 2000), (2, 32, 4, 40, 5000), (1, 256, 8, 1024, 4100),
                                        (12, 256, 8, 32, 300)])
def test_decode(M, K, d, D, N):
    say("decode", M, K, d, D, N)
    G = D // d
    rng = _rng(13, M, K, d, D, N)
    codes = rng.integers(0, K, size=(N, M, G))
    words = O.pack_codes(codes, K).view(np.int32)
    gain = rng.uniform(0.0, 5.0, size=(M, G, K)).astype(np.float32)
    sh = rng.standard_normal((M, G, K, d))
    shape = (sh / np.linalg.norm(sh, axis=-1, keepdims=True)).astype(np.float32)
    for M_use in range(1, M + 1):
        ref = O.gsrq_decode(codes, gain, shape, M_use)
        out32 = B.decode(to_dev(words), to_dev(gain), to_dev(shape), D, M_use, out_dtype=torch.float32)
        out16 = B.decode(to_dev(words), to_dev(gain), to_dev(shape), D, M_use, out_dtype=torch.float16)
        torch.cuda.synchronize()
        o32 = out32.cpu().numpy().astype(np.float64)
        assert np.allclose(o32, ref, rtol=1e-6, atol=1e-6 * np.abs(ref).max())
        # bit for bit against the decode contract: each codeword rounded to
        # float32, stages summed in float32 in order
        acc = np.zeros((N, D), np.float32)
        for m in range(M_use):
            for g in range(G):
                kk = codes[:, m, g]
                acc[:, g * d:(g + 1) * d] += gain[m, g][kk, None] * shape[m, g][kk]
        assert np.array_equal(out32.cpu().numpy(), acc)
        o16 = out16.cpu().numpy().astype(np.float64)
        ulp = np.spacing(np.abs(ref).astype(np.float16)).astype(np.float64)
        assert np.all(np.abs(o16 - ref) <= ulp + 1e-6 * np.abs(ref).max())


def _teacher_forced_update_check(Xg, w, k_gpu, g_prev, s_prev, g_gpu, s_gpu, what):
    g_ref, s_ref = O.gskm_update(Xg, w, k_gpu, g_prev, s_prev)
    scale = max(float(np.max(g_ref)), 1e-6)
    eg = np.abs(g_gpu.astype(np.float64) - g_ref) / np.maximum(g_ref, 1e-3 * scale)
    es = np.linalg.norm(s_gpu.astype(np.float64) - s_ref, axis=1)
    assert eg.max() <= CB_RTOL, f"{what}: gain rel err {eg.max():.3g} at k={eg.argmax()}"
    assert es.max() <= CB_RTOL, f"{what}: shape err {es.max():.3g} at k={es.argmax()}"
    return eg.max(), es.max()


@pytest.mark.parametrize("dtype,N,D,d,K,weighted", [
    (np.float32, 1500, 32, 8, 64, True),
    (np.float16, 2100, 64, 8, 256, True),
    (np.float32, 300, 12, 3, 8, False),
])
def test_train_teacher_forced(dtype, N, D, d, K, weighted):
    say("train teacher forced", dtype.__name__, N, D, d, K, weighted)
    X, w, seeds = synth.small_case(N, D, d, K, 1, seed=14, dtype=dtype, weights=weighted)
    G = D // d
    X64 = X.astype(np.float64)
    w64 = w.astype(np.float64)
    Xd = to_dev(X)
    wd = to_dev(w) if weighted else None
    ww = w64 if weighted else np.ones(N)
    # initialisation only (T = 0): equal-gain assignment and eq. (8) gains
    r = B.train_stage(Xd, d, K, 0, seed_rows=seeds[0], w=wd)
    torch.cuda.synchronize()
    gain = r.gain.cpu().numpy()
    shape = r.shape.cpu().numpy()
    assign = r.assign.cpu().numpy().view(np.uint16).astype(np.int64)
    assert np.all(r.iters.cpu().numpy() == 0)
    for g in range(G):
        Xg = X64[:, g * d:(g + 1) * d]
        _, s0, _ = O.gskm_init(Xg, ww, seeds[0, g])
        check_assignment(Xg, np.ones(K), s0, assign[g], f"init g{g}")
        g0, s0, _ = O.gskm_init(Xg, ww, seeds[0, g], assign0=assign[g])
        assert np.all(np.linalg.norm(shape[g] - s0, axis=1) <= CB_RTOL)
        assert np.all(rel_err(gain[g], g0, 1e-3 * g0.max()) <= CB_RTOL)
    # iterations resumed one at a time from the GPU's own state
    for t in range(1, 6):
        gp, sp, ap = r.gain.clone(), r.shape.clone(), r.assign.clone()
        gp_np, sp_np = gp.cpu().numpy(), sp.cpu().numpy()
        prev = ap.cpu().numpy().view(np.uint16).astype(np.int64)
        r = B.train_stage(Xd, d, K, 1, w=wd, gain=gp, shape=sp, assign=ap, resume=True,
                          assign_in=True)
        torch.cuda.synchronize()
        gain = r.gain.cpu().numpy()
        shape = r.shape.cpu().numpy()
        assign = r.assign.cpu().numpy().view(np.uint16).astype(np.int64)
        trace = r.trace.cpu().numpy()
        assert np.all(r.iters.cpu().numpy() == 1)
        for g in range(G):
            Xg = X64[:, g * d:(g + 1) * d]
            check_assignment(Xg, gp_np[g], sp_np[g], assign[g], f"it{t} g{g}")
            _teacher_forced_update_check(Xg, ww, assign[g], gp_np[g].astype(np.float64),
                                         sp_np[g].astype(np.float64), gain[g], shape[g],
                                         f"it{t} g{g}")
            J = O.weighted_distortion(Xg, ww, gp_np[g], sp_np[g], assign[g])
            assert trace[g, 0] == pytest.approx(J, rel=1e-5)


def test_train_stop_rule_and_residual():
    """Planted clusters converge: the stop test ends every subspace early, the
    iteration count and the trace agree with the oracle's run, and R_next is
    the re-encoding residual."""
    say("train stop rule / residual")
    rng = _rng(15)
    N, d, K, G = 1024, 8, 16, 4
    S = np.linalg.qr(rng.standard_normal((d, d)))[0]
    cent = np.concatenate([S, -S])[:K]                        # 16 well-separated directions
    gains = rng.uniform(1.0, 4.0, size=(G, K))
    lab = rng.integers(0, K, size=(N, G))
    X = np.concatenate([gains[g][lab[:, g], None] * cent[lab[:, g]] for g in range(G)], axis=1)
    X = (X + 0.02 * rng.standard_normal(X.shape)).astype(np.float32)
    seeds = np.stack([np.array([np.nonzero(lab[:, g] == k)[0][0] for k in range(K)]) for g in range(G)])
    w = rng.lognormal(0.0, 1.0, size=N).astype(np.float32)
    r = B.train_stage(to_dev(X), d, K, 20, seed_rows=seeds, w=to_dev(w), residual=True)
    torch.cuda.synchronize()
    iters = r.iters.cpu().numpy()
    for g in range(G):
        ref = O.gskm(X[:, g * d:(g + 1) * d].astype(np.float64), w.astype(np.float64), K, 20, seeds[g])
        assert iters[g] == ref["iters_run"] < 20
        assert np.allclose(r.trace.cpu().numpy()[g, :iters[g]], ref["trace"], rtol=1e-5)
        assert np.all(r.trace.cpu().numpy()[g, iters[g]:] == 0)
        assert np.allclose(r.gain.cpu().numpy()[g], ref["gain"], rtol=1e-5)
        assert np.allclose(r.shape.cpu().numpy()[g], ref["shape"], atol=1e-5)
        cols = slice(g * d, (g + 1) * d)
        kk = ref["assign"]
        res_ref = X[:, cols].astype(np.float64) - ref["gain"][kk, None] * ref["shape"][kk]
        assert np.allclose(r.residual.cpu().numpy()[:, cols], res_ref, atol=1e-5)
    # NO_EARLY_STOP runs every iteration
    r2 = B.train_stage(to_dev(X), d, K, 7, seed_rows=seeds, w=to_dev(w), no_early_stop=True)
    torch.cuda.synchronize()
    assert np.all(r2.iters.cpu().numpy() == 7)


def test_decode_row_cap_sampled():
    """1-bit layer shape with more tokens than one workgroup can stage codes
    for (140000 rows x 128 subspaces: the row range per workgroup is capped
    and the grid grows): sampled rows, including the ragged tail, against
    the oracle's decode of the same codes."""
    say("decode row cap")
    N, D, d, K = 140000, 1024, 8, 256
    G = D // d
    rng = _rng(16)
    codes = rng.integers(0, K, size=(N, 1, G))
    words = O.pack_codes(codes, K).view(np.int32)
    gain = rng.uniform(0.0, 5.0, size=(1, G, K)).astype(np.float32)
    sh = rng.standard_normal((1, G, K, d))
    shape = (sh / np.linalg.norm(sh, axis=-1, keepdims=True)).astype(np.float32)
    out = B.decode(to_dev(words), to_dev(gain), to_dev(shape), D, out_dtype=torch.float16)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([rng.choice(N, size=3000, replace=False), np.arange(N - 300, N),
                                     np.arange(0, 300)]))
    ref = O.gsrq_decode(codes[rows], gain, shape)
    got = out.cpu().numpy()[rows].astype(np.float64)
    ulp = np.spacing(np.abs(ref).astype(np.float16)).astype(np.float64)
    assert np.all(np.abs(got - ref) <= ulp + 1e-6 * np.abs(ref).max())
