"""GPU parity at the workloads' real sizes and on degenerate inputs.

The 1-bit LLaMA-3-8B layer workload runs in the launch configuration the
benchmark times (32768 x 1024 float16, d=8, K=256, weighted); the oracle checks
sampled subspaces one by one (teacher-forced).  The tiny workload runs end to
end (two stages).  Degenerate inputs: zero rows, zero weights, identical rows,
d = 1, K = 2, empty and oversized arguments.
"""
import numpy as np
import pytest

import synth
from oracle import gsrq_oracle as O
from tests.gpu_util import CB_RTOL, check_assignment, rel_err, say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2607_01065_amd import gsrq as B  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _update_check(Xg, w, k, g_prev, s_prev, g_gpu, s_gpu, what):
    g_ref, s_ref = O.gskm_update(Xg, w, k, g_prev, s_prev)
    scale = max(float(np.max(g_ref)), 1e-6)
    eg = np.abs(g_gpu.astype(np.float64) - g_ref) / np.maximum(g_ref, 1e-3 * scale)
    es = np.linalg.norm(s_gpu.astype(np.float64) - s_ref, axis=1)
    assert eg.max() <= CB_RTOL, f"{what}: gain rel err {eg.max():.3g}"
    assert es.max() <= CB_RTOL, f"{what}: shape err {es.max():.3g}"


@pytest.fixture(scope="module")
def layer_1bit():
    wl = synth.WORKLOADS["llama3_8b_layer_1bit"]
    return wl, synth.make_kv(wl, layer=0, seed=0)


@pytest.mark.parametrize("cache", ["keys", "values"])
def test_llama3_layer_1bit_training_sampled(layer_1bit, cache):
    """Initialisation and two resumed iterations at full size; subspaces 0, 37,
    64 and 127 checked against the oracle (margin rule, teacher-forced update,
    trace)."""
    wl, kv = layer_1bit
    X = kv.keys if cache == "keys" else kv.values
    w = kv.w_keys if cache == "keys" else kv.w_values
    seeds = kv.seeds_keys if cache == "keys" else kv.seeds_values
    N, D, d, K = wl.N, wl.D, wl.d, wl.K
    say("layer 1-bit training", cache, N, D, d, K)
    Xd, wd = to_dev(X), to_dev(w)
    r = B.train_stage(Xd, d, K, 0, seed_rows=seeds[0], w=wd)
    torch.cuda.synchronize()
    X64 = X.astype(np.float64)
    w64 = w.astype(np.float64)
    groups = [0, 37, 64, 127]
    gain = r.gain.cpu().numpy()
    shape = r.shape.cpu().numpy()
    assign = r.assign.cpu().numpy().view(np.uint16).astype(np.int64)
    for g in groups:
        Xg = X64[:, g * d:(g + 1) * d]
        _, s0, _ = O.gskm_init(Xg, w64, seeds[0, g])
        check_assignment(Xg, np.ones(K), s0, assign[g], f"init g{g}")
        g0, s0, _ = O.gskm_init(Xg, w64, seeds[0, g], assign0=assign[g])
        assert np.all(np.linalg.norm(shape[g] - s0, axis=1) <= CB_RTOL)
        assert np.all(rel_err(gain[g], g0, 1e-3 * g0.max()) <= CB_RTOL)
    for t in (1, 2):
        gp, sp, ap = r.gain.clone(), r.shape.clone(), r.assign.clone()
        gp_np, sp_np = gp.cpu().numpy(), sp.cpu().numpy()
        r = B.train_stage(Xd, d, K, 1, w=wd, gain=gp, shape=sp, assign=ap, resume=True,
                          assign_in=True)
        torch.cuda.synchronize()
        gain = r.gain.cpu().numpy()
        shape = r.shape.cpu().numpy()
        assign = r.assign.cpu().numpy().view(np.uint16).astype(np.int64)
        trace = r.trace.cpu().numpy()
        for g in groups:
            Xg = X64[:, g * d:(g + 1) * d]
            check_assignment(Xg, gp_np[g], sp_np[g], assign[g], f"it{t} g{g}")
            _update_check(Xg, w64, assign[g], gp_np[g].astype(np.float64),
                          sp_np[g].astype(np.float64), gain[g], shape[g], f"it{t} g{g}")
            J = O.weighted_distortion(Xg, w64, gp_np[g], sp_np[g], assign[g])
            assert trace[g, 0] == pytest.approx(J, rel=1e-5)


def test_llama3_layer_1bit_encode_decode_sampled(layer_1bit):
    """Full-size training (T=20, as benchmarked), then encode and decode of all
    rows; codes of sampled subspaces against the oracle's eq. (5) choice on the
    GPU's codebook (margin rule), decoded rows and reconstruction MSE exact."""
    wl, kv = layer_1bit
    N, D, d, K = wl.N, wl.D, wl.d, wl.K
    say("layer 1-bit encode/decode", N, D, d, K)
    Xd, wd = to_dev(kv.keys), to_dev(kv.w_keys)
    r = B.train_stage(Xd, d, K, wl.T, seed_rows=kv.seeds_keys[0], w=wd, trace=False)
    gain, shape = r.gain[None].contiguous(), r.shape[None].contiguous()
    codes, _ = B.encode(Xd, gain, shape)
    xh16 = B.decode(codes, gain, shape, D)
    xh32 = B.decode(codes, gain, shape, D, out_dtype=torch.float32)
    torch.cuda.synchronize()
    g_np, s_np = gain.cpu().numpy(), shape.cpu().numpy()
    k = O.unpack_codes(codes.cpu().numpy().view(np.uint32), 1, wl.G, K)
    X64 = kv.keys.astype(np.float64)
    for g in [0, 5, 64, 100, 127]:
        Xg = X64[:, g * d:(g + 1) * d]
        check_assignment(Xg, g_np[0, g], s_np[0, g], k[:, 0, g], f"enc g{g}")
    rows = np.random.default_rng(1).choice(N, 512, replace=False)
    ref = O.gsrq_decode(k[rows], g_np, s_np)
    assert np.array_equal(xh32.cpu().numpy()[rows], ref.astype(np.float32))
    o16 = xh16.cpu().numpy()[rows].astype(np.float64)
    ulp = np.spacing(np.abs(ref).astype(np.float16)).astype(np.float64)
    assert np.all(np.abs(o16 - ref) <= ulp)
    # reconstruction MSE of the sampled rows, GPU decode vs oracle decode
    m_gpu = O.metrics(X64[rows], xh32.cpu().numpy()[rows])["mse"]
    m_ref = O.metrics(X64[rows], ref)["mse"]
    assert m_gpu == pytest.approx(m_ref, rel=1e-5)


def test_tiny_workload_two_stages_end_to_end():
    """The tiny workload (4096 x 128 fp32, d=8, K=256, M=2, T=10) trained stage
    by stage on the GPU; every stage's codes follow the margin rule on the
    GPU's codebook, R_next is the re-encoding residual, and the stage-fused
    encode of both stages equals the per-stage chain."""
    wl = synth.WORKLOADS["tiny"]
    kv = synth.make_kv(wl)
    N, D, d, K, M, T = wl.N, wl.D, wl.d, wl.K, wl.M, wl.T
    say("tiny workload end to end", N, D, d, K, M, T)
    X = kv.keys
    w = kv.w_keys
    Xd, wd = to_dev(X), to_dev(w)
    gains, shapes = [], []
    R = Xd
    R64 = X.astype(np.float64)
    for m in range(M):
        r = B.train_stage(R, d, K, T, seed_rows=kv.seeds_keys[m], w=wd, residual=True)
        torch.cuda.synchronize()
        g_np, s_np = r.gain.cpu().numpy(), r.shape.cpu().numpy()
        assert np.all((r.iters.cpu().numpy() >= 1) & (r.iters.cpu().numpy() <= T))
        Rn = r.residual.cpu().numpy().astype(np.float64)
        for g in range(wl.G):
            cols = slice(g * d, (g + 1) * d)
            k_ref = O.gskm_assign(R64[:, cols], g_np[g], s_np[g])
            res = R64[:, cols] - g_np[g].astype(np.float64)[k_ref, None] * s_np[g].astype(np.float64)[k_ref]
            # R_next follows the oracle's choice wherever the margin is clear
            marg = O.assignment_margin(R64[:, cols], g_np[g], s_np[g])
            ok = marg > 1e-4
            assert np.allclose(Rn[ok, cols], res[ok], rtol=1e-5, atol=1e-6 * np.abs(R64).max())
        gains.append(r.gain)
        shapes.append(r.shape)
        R = r.residual
        R64 = Rn
    gain = torch.stack(gains).contiguous()
    shape = torch.stack(shapes).contiguous()
    codes, res = B.encode(Xd, gain, shape, residual=True)
    torch.cuda.synchronize()
    assert np.allclose(res.cpu().numpy(), R64, rtol=1e-5, atol=1e-6 * np.abs(X).max())
    k = O.unpack_codes(codes.cpu().numpy().view(np.uint32), M, wl.G, K)
    xh = B.decode(codes, gain, shape, D, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = O.gsrq_decode(k, gain.cpu().numpy(), shape.cpu().numpy())
    assert np.allclose(xh.cpu().numpy(), ref, rtol=1e-6, atol=1e-6 * np.abs(ref).max())
    mse_gpu = O.metrics(X, xh.cpu().numpy())["mse"]
    mse_ref = O.metrics(X, ref)["mse"]
    assert mse_gpu == pytest.approx(mse_ref, rel=1e-5)
    assert mse_gpu < 0.5 * O.metrics(X, np.zeros_like(X))["mse"]


def test_degenerate_inputs():
    """Zero rows, zero-weight rows, identical rows (ties everywhere), d = 1
    and K = 2: initialisation and one iteration match the oracle."""
    rng = np.random.default_rng(5)
    N, d, K = 777, 1, 2
    X = rng.standard_normal((N, 4)).astype(np.float32)
    X[::7] = 0.0                                  # zero rows
    X[100:140] = X[99]                            # identical rows
    w = rng.lognormal(0.0, 1.0, size=N).astype(np.float32)
    w[::5] = 0.0                                  # zero weights
    seeds = np.stack([rng.choice(np.nonzero(np.abs(X[:, g]) > 0)[0], K, replace=False)
                      for g in range(4)])
    say("degenerate inputs", N, d, K)
    Xd, wd = to_dev(X), to_dev(w)
    r = B.train_stage(Xd, d, K, 0, seed_rows=seeds, w=wd)
    torch.cuda.synchronize()
    X64 = X.astype(np.float64)
    w64 = w.astype(np.float64)
    gain0 = r.gain.cpu().numpy()
    shape0 = r.shape.cpu().numpy()
    assign0 = r.assign.cpu().numpy().view(np.uint16).astype(np.int64)
    for g in range(4):
        Xg = X64[:, g:g + 1]
        g0, s0, _ = O.gskm_init(Xg, w64, seeds[g], assign0=assign0[g])
        check_assignment(Xg, np.ones(K), s0, assign0[g], f"init g{g}")
        assert np.allclose(shape0[g], s0, atol=1e-6)
        assert np.allclose(gain0[g], g0, rtol=1e-5, atol=1e-6)
    r1 = B.train_stage(Xd, d, K, 1, w=wd, gain=r.gain.clone(), shape=r.shape.clone(),
                       assign=r.assign.clone(), resume=True, assign_in=True)
    torch.cuda.synchronize()
    a1 = r1.assign.cpu().numpy().view(np.uint16).astype(np.int64)
    for g in range(4):
        Xg = X64[:, g:g + 1]
        check_assignment(Xg, gain0[g], shape0[g], a1[g], f"it1 g{g}")
        _update_check(Xg, w64, a1[g], gain0[g].astype(np.float64),
                      shape0[g].astype(np.float64), r1.gain.cpu().numpy()[g],
                      r1.shape.cpu().numpy()[g], f"it1 g{g}")


def test_argument_errors_on_device():
    X = torch.zeros((10, 16), dtype=torch.float16, device="cuda")
    with pytest.raises(B.GsrqError) as e:
        B.train_stage(X, 8, 16, 1, seed_rows=np.zeros((2, 16), np.int32))   # N < K
    assert e.value.status == B.GSRQ_E_ARG
    gain = torch.ones((1, 4, 512), device="cuda")
    shape = torch.ones((1, 4, 512, 4), device="cuda")
    with pytest.raises(B.GsrqError) as e:
        B.encode(X, gain, shape)                                   # d = 4 with K > 256
    assert e.value.status == B.GSRQ_E_UNSUPPORTED
    empty = torch.zeros((0, 16), dtype=torch.float16, device="cuda")
    with pytest.raises(B.GsrqError) as e:
        B.encode(empty, torch.ones((1, 2, 16), device="cuda"),
                 torch.ones((1, 2, 16, 8), device="cuda"))                     # N = 0
    assert e.value.status == B.GSRQ_E_ARG


@pytest.mark.parametrize("layer", [0, 31])
def test_full_cache_layer_sampled(layer):
    """Full-model cache workload, one layer at full size: K and V codebooks
    trained on the layer's 4096-token calibration draw, then all 131072 tokens
    encoded and decoded; sampled subspaces follow the margin rule on the GPU's
    codebook, sampled decoded rows are exact."""
    wl = synth.WORKLOADS["llama3_8b_cache_1bit"]
    N, D, d, K = wl.N, wl.D, wl.d, wl.K
    say("full cache layer", layer, N, D, d, K)
    cal = synth.make_calibration(wl, layer, seed=0, N=4096, M=1)
    keys, values, _, _ = synth.make_kv_device(wl, layer, seed=0)
    rows = np.sort(np.random.default_rng(layer).choice(N, 4096, replace=False))
    for name, X, Xc, wc, seeds in (("keys", keys, cal.keys, cal.w_keys, cal.seeds_keys),
                                   ("values", values, cal.values, cal.w_values, cal.seeds_values)):
        r = B.train_stage(to_dev(Xc), d, K, wl.T, seed_rows=seeds[0], w=to_dev(wc), trace=False)
        gain, shape = r.gain[None].contiguous(), r.shape[None].contiguous()
        codes, _ = B.encode(X, gain, shape)
        xh = B.decode(codes, gain, shape, D, out_dtype=torch.float32)
        torch.cuda.synchronize()
        g_np, s_np = gain.cpu().numpy(), shape.cpu().numpy()
        k = O.unpack_codes(codes.cpu().numpy().view(np.uint32)[rows], 1, wl.G, K)
        Xs = X[torch.from_numpy(rows).cuda()].cpu().numpy().astype(np.float64)
        for g in [0, 17, 64, 127]:
            check_assignment(Xs[:, g * d:(g + 1) * d], g_np[0, g], s_np[0, g], k[:, 0, g],
                             f"{name} layer {layer} g{g}")
        ref = O.gsrq_decode(k, g_np, s_np)
        assert np.array_equal(xh.cpu().numpy()[rows], ref.astype(np.float32))
