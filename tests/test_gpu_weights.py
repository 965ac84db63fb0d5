"""GPU parity of the per-token weights (Sec. 5.3, Appendix B) against the
float64 oracle, through the C ABI.

The device computes w_i = ||g_i||_2 from gradient rows, the exact median of
the float32 norms, and w~ = log(1 + lambda w), lambda = tau / (median + eps).
Norms agree with float64 norms of the same rows to 1e-6 relative; the median
is compared exactly with numpy's median of the GPU's own float32 norms (a
selection, so no rounding is involved); the smoothed weights agree with the
oracle's log_weight of those norms to 1e-6 relative (float32 output).
Inputs are synthetic heavy-tailed gradient rows (synth.gradient_rows).
"""
import numpy as np
import pytest

import synth
from oracle import gsrq_oracle as O
from tests.gpu_util import say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

from paper_2607_01065_amd import gsrq as B  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load_library()


@pytest.mark.parametrize("N,D,dtype,pad,tau", [
    (32768, 1024, np.float16, 0, 1.0),     # one 1-bit layer's tokens, all heads
    (1001, 128, np.float32, 8, 1.0),       # odd N, padded rows
    (4096, 100, np.float16, 0, 0.1),       # row length not a multiple of 8 (scalar loads)
    (2, 64, np.float32, 0, 10.0),
    (1, 32, np.float16, 0, 1.0),
])
def test_row_weights_from_gradients(N, D, dtype, pad, tau):
    say("row weights", N, D, dtype.__name__, pad, tau)
    G = synth.gradient_rows(N, D + pad, seed=5, dtype=dtype)
    Gd = torch.from_numpy(G).cuda()[:, :D]
    w, norms, stats = B.row_weights(Gd, tau=tau)
    torch.cuda.synchronize()
    n_gpu = norms.cpu().numpy()
    n_ref = np.linalg.norm(G[:, :D].astype(np.float64), axis=1)
    assert np.all(np.abs(n_gpu - n_ref) <= 1e-6 * n_ref + 1e-30)
    med, lam = stats.cpu().numpy()
    assert med == np.median(n_gpu.astype(np.float64))
    tau32 = float(np.float32(tau))           # the ABI takes tau as float32
    assert lam == pytest.approx(tau32 / (med + 1e-8), rel=1e-15)
    ref = O.log_weight(n_gpu.astype(np.float64), tau=tau32)
    assert np.all(np.abs(w.cpu().numpy() - ref) <= 1e-6 * np.abs(ref) + 1e-30)


def test_row_weights_from_norms_ties_and_zeros():
    """Norms given directly (no gradient rows): many equal values and zeros;
    the exact median, for odd and even N."""
    rng = np.random.default_rng(6)
    for N in (999, 1000):
        n = rng.choice(np.array([0.0, 0.5, 2.0, 2.0, 2.0, 3.25, 1e-20, 7.0], np.float32), size=N)
        nd = torch.from_numpy(n).cuda()
        w, _, stats = B.row_weights(norms=nd, tau=1.0)
        torch.cuda.synchronize()
        assert stats.cpu().numpy()[0] == np.median(n.astype(np.float64))
        ref = O.log_weight(n.astype(np.float64), tau=1.0)
        assert np.all(np.abs(w.cpu().numpy() - ref) <= 1e-6 * np.abs(ref) + 1e-30)


def test_row_weights_tame_heavy_tail():
    """Sec. 5.3: raw gradient norms are heavy-tailed (max/median > 400 on
    this synthetic draw) and the log smoothing brings the ratio below 10."""
    G = torch.from_numpy(synth.gradient_rows(32768, 1024, seed=7)).cuda()
    w, norms, _ = B.row_weights(G, tau=1.0)
    torch.cuda.synchronize()
    n, wt = norms.cpu().numpy().astype(np.float64), w.cpu().numpy().astype(np.float64)
    say("heavy tail", n.max() / np.median(n), wt.max() / np.median(wt))
    assert n.max() / np.median(n) > 400
    assert wt.max() / np.median(wt) < 10
