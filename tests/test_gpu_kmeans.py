"""GPU parity of the K-means baseline (GSRQ_KMEANS) against the float64
oracle's Lloyd K-means, through the C ABI, for both kernel families.

K-means is the baseline GSKM replaces (Sec. 4, Sec. 6.1).  The library runs it
with the GSKM kernels, holding centroid c_k as gain ||c_k|| and shape
c_k / ||c_k||, so the comparison is on c = gain * shape.  Same rules as the
GSKM tests: indices follow the margin rule, updates are compared
teacher-forced (the oracle's update applied to the GPU's own assignment and
previous centroids) to 1e-5 relative, and a free-running comparison is made
only on planted clusters, where no near-tie can flip the trajectory.  The
last tests check the ordering the paper reports on x ~ N(0, I) (GSKM above
K-means in cosine, below it in gain error), computed from the GPU's own
codebooks, encodings and reconstructions.
"""
import numpy as np
import pytest

import synth
from oracle import gsrq_oracle as O
from tests.gpu_util import CB_RTOL, check_assignment, say
from tests.test_gpu_parity import _rng, to_dev

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2607_01065_amd import gsrq as B  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


def _centroids(gain, shape):
    return gain.astype(np.float64)[..., None] * shape.astype(np.float64)


def _check_centroids(C_gpu, C_ref, what):
    scale = max(float(np.max(np.linalg.norm(C_ref, axis=-1))), 1e-6)
    err = np.linalg.norm(C_gpu - C_ref, axis=-1) / np.maximum(np.linalg.norm(C_ref, axis=-1),
                                                             1e-3 * scale)
    assert err.max() <= CB_RTOL, f"{what}: centroid rel err {err.max():.3g} at k={err.argmax()}"


@pytest.mark.parametrize("dtype,N,D,d,K,weighted", [
    (np.float32, 1500, 32, 8, 64, True),      # narrow family
    (np.float16, 2100, 64, 8, 256, True),
    (np.float32, 300, 12, 3, 8, False),
    (np.float16, 3000, 64, 16, 64, True),     # wide family
    (np.float32, 2000, 256, 128, 128, True),
    (np.float16, 4100, 16, 8, 512, False),
])
def test_kmeans_teacher_forced(dtype, N, D, d, K, weighted):
    say("kmeans teacher forced", dtype.__name__, N, D, d, K, weighted)
    X, w, seeds = synth.small_case(N, D, d, K, 1, seed=31, dtype=dtype, weights=weighted)
    G = D // d
    # a zero seed row is allowed for K-means: its centroid is 0
    X[seeds[0, 0, 1], 0:d] = 0
    X64 = X.astype(np.float64)
    Xd = to_dev(X)
    wd = to_dev(w) if weighted else None
    ww = w.astype(np.float64) if weighted else np.ones(N)
    # seeding only (T = 0): the centroids are the seed rows
    r = B.train_stage(Xd, d, K, 0, seed_rows=seeds[0], w=wd, kmeans=True)
    torch.cuda.synchronize()
    C = _centroids(r.gain.cpu().numpy(), r.shape.cpu().numpy())
    assert np.all(r.iters.cpu().numpy() == 0)
    for g in range(G):
        Xg = X64[:, g * d:(g + 1) * d]
        _check_centroids(C[g], Xg[seeds[0, g]], f"seed g{g}")
    assert np.all(C[0, 1] == 0.0)
    # iterations one at a time from the GPU's own state; the first has no
    # previous assignment
    for t in range(1, 5):
        gp, sp, ap = r.gain.clone(), r.shape.clone(), r.assign.clone()
        gp_np, sp_np = gp.cpu().numpy(), sp.cpu().numpy()
        C_prev = _centroids(gp_np, sp_np)
        r = B.train_stage(Xd, d, K, 1, w=wd, gain=gp, shape=sp, assign=ap, resume=True,
                          assign_in=t > 1, kmeans=True)
        torch.cuda.synchronize()
        C = _centroids(r.gain.cpu().numpy(), r.shape.cpu().numpy())
        assign = r.assign.cpu().numpy().view(np.uint16).astype(np.int64)
        trace = r.trace.cpu().numpy()
        assert np.all(r.iters.cpu().numpy() == 1)
        for g in range(G):
            Xg = X64[:, g * d:(g + 1) * d]
            # nearest centroid = eq. (5) with gain ||c|| and unit shape
            check_assignment(Xg, gp_np[g], sp_np[g], assign[g], f"km it{t} g{g}")
            C_ref = O.kmeans_update(Xg, ww, assign[g], C_prev[g])
            _check_centroids(C[g], C_ref, f"km it{t} g{g}")
            R = Xg - C_ref[assign[g]]
            J = float(np.sum(ww * np.sum(R * R, axis=1)))
            assert trace[g, 0] == pytest.approx(J, rel=1e-5), f"km it{t} g{g} trace"


@pytest.mark.parametrize("d,K,G", [(8, 16, 4), (16, 32, 3)])
def test_kmeans_free_running_planted(d, K, G):
    """Planted clusters (arbitrary centres, not on a sphere): the GPU's
    K-means stops at the oracle's iteration with its trace, centroids and
    next-stage residual; the trace never increases."""
    say("kmeans planted", d, K, G)
    rng = _rng(32, d)
    N = 2048
    centres = rng.standard_normal((G, K, d)) * 3.0
    lab = rng.integers(0, K, size=(N, G))
    X = np.concatenate([centres[g][lab[:, g]] for g in range(G)], axis=1)
    X = (X + 0.05 * rng.standard_normal(X.shape)).astype(np.float32)
    seeds = np.stack([np.array([np.nonzero(lab[:, g] == k)[0][0] for k in range(K)])
                      for g in range(G)])
    w = rng.lognormal(0.0, 1.0, size=N).astype(np.float32)
    r = B.train_stage(to_dev(X), d, K, 20, seed_rows=seeds, w=to_dev(w), residual=True,
                      kmeans=True)
    torch.cuda.synchronize()
    iters = r.iters.cpu().numpy()
    trace = r.trace.cpu().numpy()
    C = _centroids(r.gain.cpu().numpy(), r.shape.cpu().numpy())
    res = r.residual.cpu().numpy()
    for g in range(G):
        cols = slice(g * d, (g + 1) * d)
        Xg = X[:, cols].astype(np.float64)
        ref = O.kmeans(Xg, w.astype(np.float64), K, 20, seeds[g])
        assert iters[g] == ref["iters_run"] < 20
        assert np.allclose(trace[g, :iters[g]], ref["trace"], rtol=1e-5)
        assert np.all(trace[g, iters[g]:] == 0)
        # non-increasing up to the float32 per-row distortion of the wide
        # family (each row's ||x - c||^2 is formed in float32)
        assert np.all(np.diff(trace[g, :iters[g]]) <= 1e-6 * trace[g, 0])
        _check_centroids(C[g], ref["centroids"], f"planted g{g}")
        res_ref = Xg - ref["centroids"][ref["assign"]]
        assert np.allclose(res[:, cols], res_ref, atol=1e-5)


def _gaussian_metrics(d, K, seed=0):
    """Sec. 6.1 metrics of K-means and GSKM on N = 10,000 samples of
    N(0, I_d) (synth.gaussian_case), both trained (T = 100, stop rule),
    encoded and decoded on the GPU from the same seed rows."""
    X, seeds = synth.gaussian_case(10000, d, K, seed=seed)
    Xd = to_dev(X)
    out = {}
    for name, km in (("gskm", False), ("kmeans", True)):
        r = B.train_stage(Xd, d, K, 100, seed_rows=seeds[None].astype(np.int32), kmeans=km)
        gain, shape = r.gain[None].contiguous(), r.shape[None].contiguous()
        codes, _ = B.encode(Xd, gain, shape)
        xh = B.decode(codes, gain, shape, d, out_dtype=torch.float32)
        torch.cuda.synchronize()
        out[name] = O.metrics(X.astype(np.float64), xh.cpu().numpy().astype(np.float64))
    return out


@pytest.mark.parametrize("d,K,gap", [(128, 256, 0.04), (256, 1024, 0.10), (64, 2048, 0.03)])
def test_gskm_vs_kmeans_ordering_on_gaussian(d, K, gap):
    """Sec. 6.1, random-normal sweeps: where a codeword serves a few to a
    few tens of samples, GSKM's reconstruction has clearly higher cosine
    similarity and lower gain error than K-means'.  The full sweep (D at
    K = 2048, K at D = 256, three seeds, with float64-oracle spot checks)
    is tests/sweep_gaussian.py; its cosine gaps at (256, 1024) and
    (64, 2048) are +14.5% (+14.2 .. +15.1 over seeds) and +5.6%
    (+5.2 .. +5.9); at (128, 256) the float64 oracle gives +6.1% on this
    seed (cosine 0.3320 against 0.3128).  The asserted gaps sit below the
    measured ones by more than their spread over seeds."""
    out = _gaussian_metrics(d, K)
    say("fig4", d, K, out)
    g, k = out["gskm"], out["kmeans"]
    assert g["cos"] > (1.0 + gap) * k["cos"]
    assert g["gain_err"] < k["gain_err"]
    assert g["mse"] < k["mse"]


def test_gskm_and_kmeans_tie_at_small_k_on_gaussian():
    """The capacity sweep's other end (D = 256, K = 8, about 1,250 samples
    per codeword): the two methods are within 1% of each other in every
    metric, in either direction, which is this reading's departure from the
    paper's largest gap at small K (each centroid then averages so many
    isotropic samples that its direction is equally poor for both)."""
    out = _gaussian_metrics(256, 8)
    say("fig4 tie", out)
    for key in ("mse", "gain_err", "cos"):
        a, b = out["gskm"][key], out["kmeans"][key]
        assert abs(a - b) <= 0.01 * abs(b), key
