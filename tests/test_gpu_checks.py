"""GPU tests of the boundary's checks, repeatability and small-batch encode,
through the C ABI.

* GSRQ_CHECK_INPUTS: a negative or non-finite weight, a non-finite element
  of X, or a zero seed subvector under GSKM seeding (Alg. 1 starts from
  shapes on the unit sphere; the oracle refuses such a seed) return
  GSRQ_E_ARG with every output untouched; valid inputs give the unchecked
  call's results.
* GSRQ_ATTN_TABLES_READY on a workspace whose tag does not match the call
  (no tables, or tables of other codebook arrays) gives NaN outputs.
* Repeatability (run twice, compare bit for bit): codes, assignments,
  decodes, attention outputs and per-token weights are bitwise repeatable;
  trained codebooks are reduced in a fixed order from float64 sums that LDS
  atomics add in a varying order, so an element may differ in its last
  float32 bit (reported, bounded by one ulp).
* Encode of 1, 8 and 64 appended tokens (the per-step append of decoding)
  against the oracle under the margin rule, narrow and wide families.
* Per-token weights at N = 65536 (above the LDS selection size).
"""
import numpy as np
import pytest

import synth
from oracle import gsrq_oracle as O
from tests.gpu_util import CB_RTOL, check_assignment, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2607_01065_amd import gsrq as B  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _case(N, D, d, K, dtype, seed):
    X, w, seeds = synth.small_case(N, D, d, K, 1, seed=seed, dtype=dtype)
    return X, w, seeds[0]


def _train_args(X, w, seeds, K, d, **kw):
    G = X.shape[1] // d
    gain = torch.full((G, K), 7.0, dtype=torch.float32, device="cuda")
    shape = torch.full((G, K, d), 7.0, dtype=torch.float32, device="cuda")
    return dict(seed_rows=seeds, w=w, gain=gain, shape=shape, **kw)


@pytest.mark.parametrize("N,D,d,K,dtype", [(600, 32, 8, 16, np.float32),
                                           (600, 32, 8, 16, np.float16),
                                           (1200, 64, 16, 512, np.float16)])
def test_check_inputs_rejects_bad_inputs(N, D, d, K, dtype):
    say("check inputs", N, D, d, K, dtype.__name__)
    X, w, seeds = _case(N, D, d, K, dtype, seed=11)
    cases = {}
    wb = w.copy(); wb[17] = -0.5
    cases["negative weight"] = (X, wb)
    wb = w.copy(); wb[3] = np.nan
    cases["NaN weight"] = (X, wb)
    wb = w.copy(); wb[N - 1] = np.inf
    cases["infinite weight"] = (X, wb)
    Xb = X.copy(); Xb[5, D - 1] = np.inf
    cases["infinite element"] = (Xb, w)
    Xb = X.copy(); Xb[N // 2, 3] = np.nan
    cases["NaN element"] = (Xb, w)
    Xb = X.copy(); g = 1; Xb[seeds[g, 2], g * d:(g + 1) * d] = 0
    cases["zero seed subvector"] = (Xb, w)
    for what, (Xc, wc) in cases.items():
        a = _train_args(_dev(Xc), _dev(wc), seeds, K, d, check_inputs=True)
        with pytest.raises(B.GsrqError) as e:
            B.train_stage(_dev(Xc), d, K, 3, **a)
        assert e.value.status == B.GSRQ_E_ARG, what
        torch.cuda.synchronize()
        assert torch.all(a["gain"] == 7.0) and torch.all(a["shape"] == 7.0), what
    # K-means seeding takes a zero seed row as a centroid: accepted
    Xz = cases["zero seed subvector"][0]
    a = _train_args(_dev(Xz), _dev(w), seeds, K, d, check_inputs=True, kmeans=True)
    B.train_stage(_dev(Xz), d, K, 2, **a)
    torch.cuda.synchronize()
    assert torch.all(torch.isfinite(a["gain"]))


@pytest.mark.parametrize("N,D,d,K,dtype", [(2048, 64, 8, 64, np.float16),
                                           (2048, 64, 16, 256, np.float32)])
def test_check_inputs_valid_matches_unchecked(N, D, d, K, dtype):
    X, w, seeds = _case(N, D, d, K, dtype, seed=12)
    Xd, wd = _dev(X), _dev(w)
    r1 = B.train_stage(Xd, d, K, 4, seeds, wd, check_inputs=True, no_early_stop=True)
    r2 = B.train_stage(Xd, d, K, 4, seeds, wd, no_early_stop=True)
    torch.cuda.synchronize()
    assert torch.equal(r1.assign, r2.assign)
    assert torch.allclose(r1.gain, r2.gain, rtol=1e-6, atol=0)
    assert torch.allclose(r1.shape, r2.shape, rtol=0, atol=1e-6)


def test_zero_seed_without_check_gives_zero_shape():
    """Without the check a zero seed subvector is the caller's mistake; the
    initial shape of that codeword is the zero vector (y = x / (||x|| + eps)
    of a zero row), and the outputs stay finite."""
    N, D, d, K = 600, 32, 8, 16
    X, w, seeds = _case(N, D, d, K, np.float32, seed=13)
    g, k = 2, 5
    X[seeds[g, k], g * d:(g + 1) * d] = 0
    r = B.train_stage(_dev(X), d, K, 0, seeds, _dev(w))
    torch.cuda.synchronize()
    assert torch.all(r.shape[g, k] == 0)
    assert torch.all(torch.isfinite(r.gain)) and torch.all(torch.isfinite(r.shape))


def test_attn_tables_tag_mismatch_gives_nan():
    case = synth.attn_case(2, 700, [700, 300], 2, 4, seed=9, q_dtype="float16")
    t = {k: _dev(case[k]) for k in ("k_codes", "v_codes", "lens", "k_gain", "k_shape",
                                    "v_gain", "v_shape", "q")}
    codes = [t["k_codes"], t["v_codes"]]
    cb = [t["k_gain"], t["k_shape"], t["v_gain"], t["v_shape"]]
    n = B.attn_workspace_bytes(2, 700, 8, 2)
    say("attn tag")
    # a workspace that never held tables
    ws = torch.zeros(n, dtype=torch.uint8, device="cuda")
    out = B.attn_decode(*codes, t["lens"], *cb, t["q"], workspace=ws, tables_ready=True)
    torch.cuda.synchronize()
    assert torch.all(torch.isnan(out))
    # tables built for these codebooks, then reused: finite and equal to a rebuild
    B.attn_decode(*codes, t["lens"], *cb, t["q"], workspace=ws)
    ok = B.attn_decode(*codes, t["lens"], *cb, t["q"], workspace=ws, tables_ready=True)
    fresh = B.attn_decode(*codes, t["lens"], *cb, t["q"])
    torch.cuda.synchronize()
    assert torch.equal(ok, fresh)
    # the same values in other arrays: the tag names the arrays, so NaN
    cb2 = [c.clone() for c in cb]
    bad = B.attn_decode(*codes, t["lens"], *cb2, t["q"], workspace=ws, tables_ready=True)
    torch.cuda.synchronize()
    assert torch.all(torch.isnan(bad))
    # another RoPE base than the tables were built with
    bad = B.attn_decode(*codes, t["lens"], *cb, t["q"], workspace=ws, tables_ready=True,
                        rope_base=10000.0)
    torch.cuda.synchronize()
    assert torch.all(torch.isnan(bad))


def _ulp_diff(a, b):
    """Per element distance in float32 ulps (same-sign finite values)."""
    ai = a.contiguous().view(torch.int32).to(torch.int64)
    bi = b.contiguous().view(torch.int32).to(torch.int64)
    return (ai - bi).abs()


@pytest.mark.parametrize("N,D,d,K,M,dtype", [(16384, 256, 8, 256, 2, np.float16),
                                             (8192, 256, 16, 256, 2, np.float16),
                                             (4096, 256, 128, 512, 2, np.float32)])
def test_repeat_runs_are_bitwise_repeatable(N, D, d, K, M, dtype):
    say("repeatability", N, D, d, K, M, dtype.__name__)
    X, w, seeds = synth.small_case(N, D, d, K, M, seed=21, dtype=dtype)
    Xd, wd = _dev(X), _dev(w)

    def run():
        R = Xd
        gains, shapes, assigns = [], [], []
        for m in range(M):
            r = B.train_stage(R, d, K, 6, seeds[m], wd, no_early_stop=True, residual=True)
            gains.append(r.gain)
            shapes.append(r.shape)
            assigns.append(r.assign)
            R = r.residual
        gain, shape = torch.stack(gains), torch.stack(shapes)
        codes, res = B.encode(Xd, gain, shape, residual=True)
        xh = B.decode(codes, gain, shape, D, out_dtype=torch.float32)
        torch.cuda.synchronize()
        return gain, shape, assigns, codes, res, xh

    a, b = run(), run()
    gdiff = _ulp_diff(a[0], b[0])
    sdiff = _ulp_diff(a[1], b[1])
    say("codebook elements differing between runs", int((gdiff > 0).sum()),
        int((sdiff > 0).sum()), "of", gdiff.numel() + sdiff.numel())
    assert int(gdiff.max()) <= 1 and int(sdiff.max()) <= 1
    if int(gdiff.max()) == 0 and int(sdiff.max()) == 0:
        # same codebooks: everything downstream is bitwise the same
        for x, y in zip(a[2], b[2]):
            assert torch.equal(x, y)
        assert torch.equal(a[3], b[3])
        assert torch.equal(a[4], b[4])
        assert torch.equal(a[5], b[5])
    # encode / decode with fixed codebooks are bitwise repeatable
    c1, r1 = B.encode(Xd, a[0], a[1], residual=True)
    c2, r2 = B.encode(Xd, a[0], a[1], residual=True)
    x1 = B.decode(c1, a[0], a[1], D, out_dtype=torch.float16)
    x2 = B.decode(c1, a[0], a[1], D, out_dtype=torch.float16)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2) and torch.equal(r1, r2) and torch.equal(x1, x2)


def test_attention_and_weights_are_bitwise_repeatable():
    case = synth.attn_case(3, 5000, [5000, 4097, 33], 2, 4, seed=22, q_dtype="float16")
    t = {k: _dev(case[k]) for k in ("k_codes", "v_codes", "lens", "k_gain", "k_shape",
                                    "v_gain", "v_shape", "q")}
    args = [t[k] for k in ("k_codes", "v_codes", "lens", "k_gain", "k_shape", "v_gain",
                           "v_shape", "q")]
    o1 = B.attn_decode(*args)
    o2 = B.attn_decode(*args)
    G = _dev(synth.gradient_rows(20000, 512, seed=3))
    w1, _, s1 = B.row_weights(G)
    w2, _, s2 = B.row_weights(G)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)
    assert torch.equal(w1, w2) and torch.equal(s1, s2)


@pytest.mark.parametrize("D,d,K,M,dtype", [(1024, 8, 256, 1, np.float16),
                                           (1024, 16, 256, 2, np.float16),
                                           (1024, 128, 256, 4, np.float32)])
def test_append_encode_small_batches(D, d, K, M, dtype):
    """Encode of 1, 8 and 64 new tokens with a trained codebook (the append
    step of autoregressive decoding) against the oracle, stage by stage on
    the GPU's own residuals (margin rule), plus the residual output."""
    G = D // d
    X, w, _ = synth.small_case(4096, D, d, K, M, seed=23, dtype=dtype)
    seeds = synth.draw_seed_rows(np.random.default_rng(23), 2048, K, M, G)
    cb = O.gsrq_train(X[:2048].astype(np.float64), w[:2048], d, K, M, 3, seeds)
    gain = cb["gains"].astype(np.float32)
    shape = cb["shapes"].astype(np.float32)
    gd, sd = _dev(gain), _dev(shape)
    for n in (1, 8, 64):
        say("append encode", n, D, d, K, M)
        Xn = X[3000:3000 + n]
        codes, res = B.encode(_dev(Xn), gd, sd, residual=True)
        torch.cuda.synchronize()
        k = O.unpack_codes(codes.cpu().numpy().view(np.uint32), M, G, K)
        R = Xn.astype(np.float64)
        for m in range(M):
            for g in range(G):
                cols = slice(g * d, (g + 1) * d)
                check_assignment(R[:, cols], gain[m, g], shape[m, g], k[:, m, g],
                                 what=f"append n={n} m={m} g={g}")
                R[:, cols] -= gain[m, g][k[:, m, g], None].astype(np.float64) * \
                    shape[m, g][k[:, m, g]].astype(np.float64)
        scale = max(float(np.abs(Xn.astype(np.float64)).max()), 1e-30)
        assert np.max(np.abs(res.cpu().numpy() - R)) <= CB_RTOL * scale


def test_row_weights_above_lds_selection_size():
    """N = 65536 norms take the selection path that does not stage the norms
    in LDS; the median is exact and the weights match the oracle's."""
    N, D = 65536, 256
    G = synth.gradient_rows(N, D, seed=8, dtype=np.float16)
    w, norms, stats = B.row_weights(_dev(G), tau=1.0)
    torch.cuda.synchronize()
    n_gpu = norms.cpu().numpy()
    n_ref = np.linalg.norm(G.astype(np.float64), axis=1)
    assert np.all(np.abs(n_gpu - n_ref) <= 1e-6 * n_ref + 1e-30)
    med = stats.cpu().numpy()[0]
    assert med == np.median(n_gpu.astype(np.float64))
    ref = O.log_weight(n_gpu.astype(np.float64), tau=1.0)
    assert np.all(np.abs(w.cpu().numpy() - ref) <= 1e-6 * np.abs(ref) + 1e-30)
    for N2 in (65537, 100001):
        n2 = torch.rand(N2, device="cuda", dtype=torch.float32)
        _, _, st = B.row_weights(norms=n2, tau=1.0)
        torch.cuda.synchronize()
        assert st.cpu().numpy()[0] == np.median(n2.cpu().numpy().astype(np.float64))


def test_attn_workspace_contents_do_not_leak_into_outputs():
    """A sequence shorter than the cache leaves chunks without tokens, which
    write only their (reference, sum) record; a workspace filled with NaN
    bits beforehand must still give the output of a fresh one."""
    case = synth.attn_case(3, 6000, [6000, 700, 0], 2, 4, seed=24, q_dtype="float16")
    t = {k: _dev(case[k]) for k in ("k_codes", "v_codes", "lens", "k_gain", "k_shape",
                                    "v_gain", "v_shape", "q")}
    args = [t[k] for k in ("k_codes", "v_codes", "lens", "k_gain", "k_shape", "v_gain",
                           "v_shape", "q")]
    n = B.attn_workspace_bytes(3, 6000, 8, 2)
    ws = torch.full((n,), 0xFF, dtype=torch.uint8, device="cuda")     # NaN float bits
    dirty = B.attn_decode(*args, workspace=ws)
    clean = B.attn_decode(*args, workspace=torch.zeros(n, dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    assert torch.all(torch.isfinite(dirty))
    assert torch.equal(dirty, clean)


@pytest.mark.parametrize("N,D,d,K,M,dtype", [(1, 1024, 8, 256, 1, np.float16),
                                             (8, 1024, 8, 256, 1, np.float16),
                                             (64, 1024, 8, 256, 2, np.float32),
                                             (256, 1024, 8, 256, 1, np.float16),
                                             (257, 1024, 8, 256, 1, np.float16),
                                             (33, 24, 4, 16, 3, np.float32),
                                             (2049, 256, 8, 256, 3, np.float16),
                                             (777, 24, 4, 16, 2, np.float32)])
def test_prepared_encode_matches_encode(N, D, d, K, M, dtype):
    """gsrq_encode_prepared gives gsrq_encode's codes and residual bit for
    bit (the same operand tables, built once), including the append sizes
    1, 8 and 64: up to 256 rows it runs the latency kernel (one wave per
    row block and subspace), above that the stage-fused encoder; 4-bit codes
    (K = 16) are OR'd into zeroed words."""
    say("prepared encode", N, D, d, K, M, dtype.__name__)
    X, w, seeds = synth.small_case(max(N, 2 * K), D, d, K, M, seed=31, dtype=dtype)
    G = D // d
    rng = np.random.default_rng(31)
    sh = rng.standard_normal((M, G, K, d))
    sh /= np.linalg.norm(sh, axis=-1, keepdims=True)
    gain = (np.median(np.linalg.norm(X.astype(np.float64).reshape(-1, G, d), axis=-1))
            * rng.uniform(0.3, 1.5, size=(M, G, K)) / (1 + np.arange(M))[:, None, None])
    gd, sd = _dev(gain.astype(np.float32)), _dev(sh.astype(np.float32))
    prep = B.prepare_codebook(gd, sd)
    Xd = _dev(X[:N])
    c1, r1 = B.encode(Xd, gd, sd, residual=True)
    c2, r2 = B.encode_prepared(Xd, prep, residual=True)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2) and torch.equal(r1, r2)
    k = O.unpack_codes(c2.cpu().numpy().view(np.uint32), M, G, K)
    R = X[:N].astype(np.float64)
    for m in range(M):
        for g in range(G):
            cols = slice(g * d, (g + 1) * d)
            check_assignment(R[:, cols], gain[m, g].astype(np.float32), sh[m, g].astype(np.float32),
                             k[:, m, g], what=f"prepared m={m} g={g}")
            kk = k[:, m, g]
            R[:, cols] -= gain[m, g].astype(np.float32)[kk, None].astype(np.float64) * \
                sh[m, g].astype(np.float32)[kk].astype(np.float64)


def test_prepared_encode_checks_its_header():
    """A buffer prepared for another shape, or never prepared, gives all-ones
    code fields and a NaN residual instead of plausible codes."""
    import ctypes
    N, D, d, K = 100, 64, 8, 256
    X, _, _ = synth.small_case(2 * K, D, d, K, 1, seed=32, dtype=np.float16)
    rng = np.random.default_rng(32)
    sh = rng.standard_normal((1, D // d, K, d))
    sh /= np.linalg.norm(sh, axis=-1, keepdims=True)
    gd = _dev(np.full((1, D // d, K), 2.0, np.float32))
    sd = _dev(sh.astype(np.float32))
    prep = B.prepare_codebook(gd, sd)
    lib = B.load_library()
    Xd = _dev(X[:N])
    for what, buf, K2 in (("other K", prep.buf, 128),
                          ("never prepared", torch.zeros_like(prep.buf), K)):
        s = B.make_shape(N, D, d, K2, 1)
        W = B.code_words(N, D, d, K2, 1)
        codes = torch.zeros((N, W), dtype=torch.int32, device="cuda")
        res = torch.zeros((N, D), dtype=torch.float32, device="cuda")
        st = lib.gsrq_encode_prepared(ctypes.byref(s), Xd.data_ptr(), B.GSRQ_F16, D,
                                      buf.data_ptr(), codes.data_ptr(), res.data_ptr(), None)
        assert st == B.GSRQ_OK, what
        torch.cuda.synchronize()
        k = O.unpack_codes(codes.cpu().numpy().view(np.uint32), 1, D // d, K2)
        assert np.all(k == K2 - 1), what            # every code field all ones
        assert torch.all(torch.isnan(res)), what
