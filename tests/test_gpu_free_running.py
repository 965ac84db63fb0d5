"""Free-running GSKM on the tiny configuration (4096 tokens x 1 head x 128,
float32, d = 8, K = 256, T = 10, weighted; first stage of the key cache):
the GPU and the float64 oracle each run Algorithm 1 from the same seed rows
with no teacher forcing, for 0 (the initialisation: an equal-gain
assignment and eq. (8) gains for the seed shapes), 1, 2, ..., T iterations,
and the report gives per subspace the first iteration at which the two
assignments differ, the codebook deltas before it, both iteration counts
(the stop rule) and the final objectives.

The GPU scores rows to about 22 significant bits and the oracle in float64,
so their assignments can only differ at near ties, and the trajectories
can only part there.  Checked:
  1. before a subspace's first differing iteration its codebooks agree to
     CB_RTOL (relative to the codebook's largest codeword norm);
  2. at that iteration the GPU's assignment passes the margin rule against
     the oracle's codebook of the previous iteration, or for the
     initialisation against unit gains and the seed shapes (every differing
     row is a near tie, and the GPU's choice lies within the margin);
  3. the final weighted objectives of the two sides agree to 1%.
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


def test_free_running_tiny_report():
    wl = synth.WORKLOADS["tiny"]
    kv = synth.make_kv(wl, layer=0, seed=0)
    X = kv.keys.astype(np.float32)
    w = kv.w_keys.astype(np.float32)
    d, K, T, G = wl.d, wl.K, wl.T, wl.G
    seeds = np.ascontiguousarray(kv.seeds_keys[0], dtype=np.int32)   # [G, K]
    Xd = torch.from_numpy(X).cuda()
    wd = torch.from_numpy(w).cuda()
    X64, w64 = X.astype(np.float64), w.astype(np.float64)

    # GPU: fresh runs of t = 0 .. T iterations
    gpu = []
    for t in range(0, T + 1):
        r = B.train_stage(Xd, d, K, t, seed_rows=seeds, w=wd, trace=False)
        torch.cuda.synchronize()
        gpu.append(dict(gain=r.gain.cpu().numpy().astype(np.float64),
                        shape=r.shape.cpu().numpy().astype(np.float64),
                        assign=r.assign.cpu().numpy().view(np.uint16).astype(np.int64),
                        iters=r.iters.cpu().numpy().astype(np.int64)))

    report = []
    for g in range(G):
        Xg = X64[:, g * d:(g + 1) * d]
        init_gain, init_shape, init_assign = O.gskm_init(Xg, w64, seeds[g])
        # the equal-gain assignment is made with unit gains and the seed shapes
        prev = (np.ones(K), init_shape)
        first = None
        delta_before = 0.0
        orc = None
        for t in range(0, T + 1):
            if t == 0:
                orc = dict(gain=init_gain, shape=init_shape, assign=init_assign, iters_run=0)
            else:
                orc = O.gskm(Xg, w64, K, t, seeds[g])
            ga, ka = gpu[t], orc
            if first is None:
                if np.array_equal(ga["assign"][g], ka["assign"]):
                    Cg = ga["gain"][g][:, None] * ga["shape"][g]
                    Co = ka["gain"][:, None] * ka["shape"]
                    scale = max(float(np.linalg.norm(Co, axis=1).max()), 1e-30)
                    dlt = float(np.abs(Cg - Co).max()) / scale
                    delta_before = max(delta_before, dlt)
                    assert dlt <= CB_RTOL, f"g{g} t{t}: codebook delta {dlt:.2e} before any flip"
                else:
                    first = t
                    # the assignment of iteration t was made with the codebook of t - 1
                    check_assignment(Xg, prev[0], prev[1], ga["assign"][g], f"g{g} t{t}")
            prev = (orc["gain"], orc["shape"])
        last = gpu[-1]
        Jg = O.weighted_distortion(Xg, w64, last["gain"][g], last["shape"][g], last["assign"][g])
        Jo = O.weighted_distortion(Xg, w64, orc["gain"], orc["shape"], orc["assign"])
        report.append((g, first, delta_before, int(last["iters"][g]), int(orc["iters_run"]),
                       Jg / Jo))
        assert abs(Jg / Jo - 1.0) <= 0.01, f"g{g}: final objective ratio {Jg / Jo:.4f}"
    say("free-running tiny (subspace, first differing iteration, max codebook delta before it, "
        "iterations GPU / oracle, final objective ratio GPU / oracle):")
    for g, first, dlt, ig, io, ratio in report:
        say(f"  g{g:2d} first flip {'-' if first is None else first:>2} delta {dlt:.1e} "
            f"iters {ig}/{io} J ratio {ratio:.6f}")
    flips = sum(1 for r in report if r[1] is not None)
    say(f"{flips} of {G} subspaces part at a near tie within {T} iterations")
