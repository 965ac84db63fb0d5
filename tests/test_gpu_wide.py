"""GPU parity of the wide-subspace path (d in {16, ..., 128}, or K > 256)
against the float64 oracle, through the C ABI.

Same rules as the narrow path: indices follow the margin rule, codebooks and
reconstructions agree to 1e-5 relative, updates are compared teacher-forced.
Shapes cover the resident and streamed fragment tables, float16 and float32
stage inputs, every template width (d = 8 with K > 256 up to d = 128), and
ragged row counts.
"""
import numpy as np
import pytest

import synth
from oracle import gsrq_oracle as O
from tests.gpu_util import CB_RTOL, check_assignment, rel_err, say
from tests.test_gpu_parity import (_rng, _teacher_forced_update_check, random_codebook, to_dev,
                                   unpack)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2607_01065_amd import gsrq as B  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


@pytest.mark.parametrize("dtype", [np.float16, np.float32])
@pytest.mark.parametrize("N,D,d,K", [
    (1000, 64, 16, 256),     # resident table, two pairs per row
    (257, 64, 32, 64),       # resident, four groups
    (700, 256, 128, 512),    # streamed, d = 128
    (1300, 32, 8, 1024),     # streamed, one group (d = 8, K > 256)
    (130, 128, 64, 32),      # one tile
    (400, 512, 256, 256),    # streamed, d = 256 (two heads per subvector)
    (3000, 256, 128, 1024),  # single float16 pass (d >= 64, K >= 1024) + listed rows
    (2500, 128, 64, 2048),   # single pass, d = 64
])
def test_wide_encode_single_stage(dtype, N, D, d, K):
    say("wide encode single stage", dtype.__name__, N, D, d, K)
    X, _, _ = synth.small_case(N, D, d, K, 1, seed=21, dtype=dtype)
    G = D // d
    gain, shape = random_codebook(X, 1, G, K, d, seed=6)
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
        kk = k[:, 0, g]
        ref = X64[:, cols] - gain[0, g].astype(np.float64)[kk, None] * shape[0, g].astype(np.float64)[kk]
        scale = np.maximum(np.abs(X64[:, cols]).max(), 1e-3)
        assert np.allclose(R[:, cols], ref, rtol=CB_RTOL, atol=1e-6 * scale)
    say("below-margin index differences:", below, "of", N * G)


@pytest.mark.parametrize("dtype,M,K,d,D,N,exact_rows", [
    (np.float32, 3, 64, 16, 48, 613, False),     # stage-fused kernel (d <= 16)
    (np.float16, 4, 256, 16, 128, 2000, False),  # stage-fused, the rate-sweep shape
    (np.float32, 3, 512, 8, 32, 700, None),      # stage-fused, d = 8 with K > 256
    (np.float16, 3, 256, 16, 64, 900, True),     # stage-fused, rows re-scored in float64
    (np.float16, 2, 256, 128, 256, 400, False),  # stage-fused, d = 128 (residual in registers)
    (np.float32, 3, 256, 128, 256, 613, False),  # stage-fused d = 128, float32 rows, ragged N
    (np.float16, 3, 256, 128, 128, 700, True),   # stage-fused d = 128, rows re-scored in float64
    (np.float16, 3, 512, 64, 128, 700, None),    # stage-fused d = 64, table at the LDS limit
    (np.float32, 4, 32, 64, 192, 333, None),     # stage-fused d = 64, one tile (odd tile count)
    (np.float16, 4, 16, 32, 64, 301, False),     # one launch per stage (d = 32)
    (np.float32, 3, 128, 256, 512, 300, False),  # one launch per stage (d = 256)
    (np.float32, 2, 1024, 128, 128, 2200, None), # single pass + listed rows, per stage
])
def test_wide_encode_multi_stage_teacher_forced(dtype, M, K, d, D, N, exact_rows):
    """Stage m is checked on the residual the GPU's own earlier choices leave.
    exact_rows: a quarter of the rows are set to stage-0 codewords, so their
    stage-1 residual is zero (or float32 noise) and the key cannot decide
    them: the float64 re-scoring path.  None: random codebooks instead of the
    oracle's training (K > N / 2 leaves exactly coded rows whose zero
    residuals cannot seed the next stage)."""
    say("wide encode multi stage", dtype.__name__, M, K, d, D, N, exact_rows)
    X, w, seeds = synth.small_case(N, D, d, K, M, seed=22, dtype=dtype)
    G = D // d
    if exact_rows is None:
        gain, shape = random_codebook(X, M, G, K, d, seed=28)
    else:
        cb = O.gsrq_train(X.astype(np.float64), w, d, K, M, 3, seeds)
        gain = cb["gains"].astype(np.float32)
        shape = cb["shapes"].astype(np.float32)
    if exact_rows:
        rng = _rng(27, N)
        pick = rng.choice(N, size=N // 4, replace=False)
        for g in range(G):
            k = rng.integers(0, K, size=pick.size)
            X[pick, g * d:(g + 1) * d] = (gain[0, g][k, None] * shape[0, g][k]).astype(dtype)
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
    assert np.allclose(Rg, R, rtol=1e-5, atol=1e-6 * np.abs(X.astype(np.float64)).max())


@pytest.mark.parametrize("M,K,d,D,N,prefixes", [
    (32, 256, 128, 256, 600, (12, 16, 32)),   # 2 bit; prefixes 0.75 / 1 / 2 bit
    (12, 256, 256, 512, 400, (4, 12)),        # 0.375 bit (d = 256: two heads)
])
def test_paper_rate_deep_stages(M, K, d, D, N, prefixes):
    """The paper's own rate configurations (Sec. 6.2 / Appendix A): K = 256
    with d = 128 and M = 32 stages (2 bits per element; its prefixes of 12
    and 16 stages are the 0.75- and 1-bit configurations), and d = 256 with
    M = 12 (0.375 bit).  Codebooks from the oracle's GSRQ training; the
    encode is checked stage by stage on the residual the GPU's own earlier
    choices leave (margin rule), the residual output against that, and the
    prefix decodes bit for bit against a float32 emulation of the decode
    contract (each codeword rounded to float32, stages summed in float32 in
    order)."""
    say("paper rate deep stages", M, K, d, D, N)
    X, w, seeds = synth.small_case(N, D, d, K, M, seed=26, dtype=np.float16)
    G = D // d
    cb = O.gsrq_train(X.astype(np.float64), w, d, K, M, 2, seeds)
    gain = cb["gains"].astype(np.float32)
    shape = cb["shapes"].astype(np.float32)
    Xd, gd, sd = to_dev(X), to_dev(gain), to_dev(shape)
    codes, res = B.encode(Xd, gd, sd, residual=True)
    torch.cuda.synchronize()
    k = unpack(codes, M, G, K)
    R = X.astype(np.float64)
    for m in range(M):
        for g in range(G):
            cols = slice(g * d, (g + 1) * d)
            check_assignment(R[:, cols], gain[m, g], shape[m, g], k[:, m, g], f"m{m} g{g}")
            kk = k[:, m, g]
            R[:, cols] -= gain[m, g].astype(np.float64)[kk, None] * shape[m, g].astype(np.float64)[kk]
    assert np.allclose(res.cpu().numpy().astype(np.float64), R, rtol=1e-5,
                       atol=1e-6 * np.abs(X.astype(np.float64)).max())
    for M_use in prefixes:
        out = B.decode(codes, gd, sd, D, M_use, out_dtype=torch.float32)
        torch.cuda.synchronize()
        acc = np.zeros((N, D), np.float32)
        for m in range(M_use):
            for g in range(G):
                kk = k[:, m, g]
                acc[:, g * d:(g + 1) * d] += gain[m, g][kk, None] * shape[m, g][kk]
        assert np.array_equal(out.cpu().numpy(), acc), f"decode prefix {M_use}"
        assert B.bits_per_element(d, K, M_use) == pytest.approx(M_use * 8 / d)


@pytest.mark.parametrize("M,K,d,D,N", [
    (2, 256, 16, 64, 1000),     # LDS table, 16-element entries
    (1, 1024, 8, 32, 333),      # LDS table, K > 256
    (3, 4096, 128, 256, 77),    # gather from global memory, 12-bit codes
    (2, 64, 64, 128, 50),       # gather, d = 64
    (2, 256, 256, 512, 60),     # gather, d = 256
])
def test_wide_decode(M, K, d, D, N):
    say("wide decode", M, K, d, D, N)
    G = D // d
    rng = _rng(23, M, K, d, D, N)
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
        # bit for bit against the decode contract (float32 codewords, summed
        # in float32 in stage order)
        acc = np.zeros((N, D), np.float32)
        for m in range(M_use):
            for g in range(G):
                kk = codes[:, m, g]
                acc[:, g * d:(g + 1) * d] += gain[m, g][kk, None] * shape[m, g][kk]
        assert np.array_equal(out32.cpu().numpy(), acc)
        o16 = out16.cpu().numpy().astype(np.float64)
        ulp = np.spacing(np.abs(ref).astype(np.float16)).astype(np.float64)
        assert np.all(np.abs(o16 - ref) <= ulp + 1e-6 * np.abs(ref).max())


@pytest.mark.parametrize("dtype,N,D,d,K,weighted", [
    (np.float16, 3000, 64, 16, 64, True),
    (np.float32, 2000, 256, 128, 128, True),
    (np.float16, 4100, 16, 8, 512, False),
    (np.float32, 1500, 64, 32, 32, True),
    (np.float16, 1200, 512, 256, 128, True),
    (np.float32, 3000, 128, 128, 1024, True),   # single pass + listed rows
    (np.float16, 2600, 128, 64, 1024, False),   # single pass, d = 64
])
def test_wide_train_teacher_forced(dtype, N, D, d, K, weighted):
    say("wide train teacher forced", dtype.__name__, N, D, d, K, weighted)
    X, w, seeds = synth.small_case(N, D, d, K, 1, seed=24, dtype=dtype, weights=weighted)
    G = D // d
    X64 = X.astype(np.float64)
    Xd = to_dev(X)
    wd = to_dev(w) if weighted else None
    ww = w.astype(np.float64) if weighted else np.ones(N)
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
    for t in range(1, 4):
        gp, sp, ap = r.gain.clone(), r.shape.clone(), r.assign.clone()
        gp_np, sp_np = gp.cpu().numpy(), sp.cpu().numpy()
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


def test_wide_train_stop_rule_and_residual():
    """Planted clusters in d = 16: every subspace stops early with the
    oracle's iteration count, trace and codebook; R_next is the re-encoding
    residual."""
    say("wide train stop rule / residual")
    rng = _rng(25)
    N, d, K, G = 2048, 16, 32, 3
    S = np.linalg.qr(rng.standard_normal((d, d)))[0]
    cent = np.concatenate([S, -S])[:K]
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
    r2 = B.train_stage(to_dev(X), d, K, 5, seed_rows=seeds, w=to_dev(w), no_early_stop=True)
    torch.cuda.synchronize()
    assert np.all(r2.iters.cpu().numpy() == 5)


@pytest.mark.parametrize("N,D,d,K", [(700, 32, 8, 256), (700, 64, 16, 256), (300, 256, 128, 512),
                                     (300, 256, 128, 2048)])
def test_rows_far_below_codebook_scale(N, D, d, K):
    """Float32 rows (residuals) 1e3 to 1e5 times smaller than the largest
    gains, as late residual stages produce: indices follow the margin rule
    and the residual output is exact (both kernel families)."""
    say("tiny rows", N, D, d, K)
    rng = _rng(26, N, D, d, K)
    G = D // d
    scale = np.where(rng.random(N) < 0.5, 1e-3, 1e-5)[:, None]
    X = (rng.standard_normal((N, D)) * scale).astype(np.float32)
    sh = rng.standard_normal((1, G, K, d))
    sh /= np.linalg.norm(sh, axis=-1, keepdims=True)
    gain = rng.uniform(50.0, 150.0, size=(1, G, K))
    gain[:, :, :K // 8] = rng.uniform(0.0, 2e-3, size=(1, G, K // 8))   # small codewords
    gain[:, :, K // 8 + 1] = gain[:, :, K // 8]                            # equal gains
    gain, shape = gain.astype(np.float32), sh.astype(np.float32)
    codes, res = B.encode(to_dev(X), to_dev(gain), to_dev(shape), residual=True)
    torch.cuda.synchronize()
    k = unpack(codes, 1, G, K)
    X64 = X.astype(np.float64)
    R = res.cpu().numpy().astype(np.float64)
    for g in range(G):
        cols = slice(g * d, (g + 1) * d)
        check_assignment(X64[:, cols], gain[0, g], shape[0, g], k[:, 0, g], f"g{g}")
        kk = k[:, 0, g]
        ref = X64[:, cols] - gain[0, g].astype(np.float64)[kk, None] * shape[0, g].astype(np.float64)[kk]
        assert np.allclose(R[:, cols], ref, rtol=1e-5, atol=1e-6 * np.abs(ref).max())
