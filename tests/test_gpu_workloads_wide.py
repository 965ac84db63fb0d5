"""GPU parity at the real sizes of the wide-subspace workloads.

Rate sweep: 65536 tokens x 8 heads x 128 float16, d = 16, K = 256 (0.5 bit per
stage).  Large codebook: the same rows with d = 128, K = 4096 (12-bit codes).
The paper's lowest rate: 32768 tokens, d = 256 (two heads), K = 256.
Both run in the launch configuration the benchmark uses, for two stages (the
second trains on the first stage's float32 residual); the oracle checks
sampled subspaces (and, at K = 4096, sampled rows for the index rule) with the
GPU's own previous state as input (teacher forcing).
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


def _stage_checks(R, w, seeds, d, K, groups, rows, what):
    """Initialisation and one resumed iteration of one stage on device input
    R; returns the stage's final GPU state."""
    R64 = R.cpu().numpy().astype(np.float64)
    w64 = w.cpu().numpy().astype(np.float64)
    r = B.train_stage(R, d, K, 0, seed_rows=seeds, w=w)
    torch.cuda.synchronize()
    gain = r.gain.cpu().numpy()
    shape = r.shape.cpu().numpy()
    assign = r.assign.cpu().numpy().view(np.uint16).astype(np.int64)
    for g in groups:
        Xg = R64[:, g * d:(g + 1) * d]
        _, s0, _ = O.gskm_init(Xg, w64, seeds[g])
        check_assignment(Xg[rows], np.ones(K), s0, assign[g][rows], f"{what} init g{g}")
        g0, s0, _ = O.gskm_init(Xg, w64, seeds[g], assign0=assign[g])
        assert np.all(np.linalg.norm(shape[g] - s0, axis=1) <= CB_RTOL)
        assert np.all(rel_err(gain[g], g0, 1e-3 * g0.max()) <= CB_RTOL)
    gp, sp, ap = r.gain.clone(), r.shape.clone(), r.assign.clone()
    gp_np, sp_np = gp.cpu().numpy(), sp.cpu().numpy()
    r = B.train_stage(R, d, K, 1, w=w, gain=gp, shape=sp, assign=ap, resume=True,
                      assign_in=True, residual=True)
    torch.cuda.synchronize()
    gain = r.gain.cpu().numpy()
    shape = r.shape.cpu().numpy()
    assign = r.assign.cpu().numpy().view(np.uint16).astype(np.int64)
    trace = r.trace.cpu().numpy()
    for g in groups:
        Xg = R64[:, g * d:(g + 1) * d]
        check_assignment(Xg[rows], gp_np[g], sp_np[g], assign[g][rows], f"{what} it1 g{g}")
        _update_check(Xg, w64, assign[g], gp_np[g].astype(np.float64),
                      sp_np[g].astype(np.float64), gain[g], shape[g], f"{what} it1 g{g}")
        J = O.weighted_distortion(Xg, w64, gp_np[g], sp_np[g], assign[g])
        assert trace[g, 0] == pytest.approx(J, rel=1e-5)
    return r


@pytest.mark.parametrize("name,groups", [("rate_sweep_d16", [0, 21, 63]),
                                         ("large_codebook_d128", [0, 5]),
                                         ("paper_rates_d256", [0, 3])])
def test_wide_workload_two_stages_sampled(name, groups):
    """Two stages of training at full size (stage 1 on stage 0's float32
    residual), then the two-stage encode and decode of every row."""
    wl = synth.WORKLOADS[name]
    kv = synth.make_kv(wl, layer=0, seed=0, M=2)
    N, D, d, K = wl.N, wl.D, wl.d, wl.K
    G = D // d
    say("wide workload", name, N, D, d, K)
    rows = np.sort(np.random.default_rng(2).choice(N, 4096 if K > 256 else N, replace=False))
    X, w = to_dev(kv.keys), to_dev(kv.w_keys)
    r0 = _stage_checks(X, w, kv.seeds_keys[0], d, K, groups, rows, "stage0")
    R1 = r0.residual
    r1 = _stage_checks(R1, w, kv.seeds_keys[1], d, K, groups, rows, "stage1")
    gain = torch.stack([r0.gain, r1.gain]).contiguous()
    shape = torch.stack([r0.shape, r1.shape]).contiguous()
    codes, res = B.encode(X, gain, shape, residual=True)
    xh = B.decode(codes, gain, shape, D, out_dtype=torch.float32)
    xh1 = B.decode(codes, gain, shape, D, 1, out_dtype=torch.float32)
    torch.cuda.synchronize()
    g_np, s_np = gain.cpu().numpy(), shape.cpu().numpy()
    k = O.unpack_codes(codes.cpu().numpy().view(np.uint32), 2, G, K)
    R = kv.keys.astype(np.float64)[rows]
    for m in range(2):
        for g in groups:
            cols = slice(g * d, (g + 1) * d)
            check_assignment(R[:, cols], g_np[m, g], s_np[m, g], k[rows, m, g], f"enc m{m} g{g}")
            kk = k[rows, m, g]
            R[:, cols] -= g_np[m, g].astype(np.float64)[kk, None] * s_np[m, g].astype(np.float64)[kk]
    # decode: sums of the coded codewords (prefixes too); residual output
    sub = rows[:512]
    ref = O.gsrq_decode(k[sub], g_np, s_np)
    ref1 = O.gsrq_decode(k[sub], g_np, s_np, 1)
    assert np.allclose(xh.cpu().numpy()[sub], ref, rtol=1e-6, atol=1e-6 * np.abs(ref).max())
    assert np.array_equal(xh1.cpu().numpy()[sub], ref1.astype(np.float32))
    Xs = kv.keys.astype(np.float64)[sub]
    assert np.allclose(res.cpu().numpy()[sub], Xs - ref, rtol=1e-5,
                       atol=1e-5 * np.abs(Xs).max())
    m_gpu = O.metrics(Xs, xh.cpu().numpy()[sub])["mse"]
    m_ref = O.metrics(Xs, ref)["mse"]
    assert m_gpu == pytest.approx(m_ref, rel=1e-5)
