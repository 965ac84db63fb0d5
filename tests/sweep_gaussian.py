"""Random-normal sweeps of Sec. 6.1 (K-means against GSKM) on the GPU path.

For x ~ N(0, I_D) and N = 10,000 samples, both methods train one codebook
of K codewords from the same K seed rows, for at most T iterations with the
library's stop rule (an assignment that repeats), on the GPU through the C
ABI (GSRQ_KMEANS for the baseline); the samples are then encoded and decoded
on the GPU with the trained codebook, and the three metrics of Sec. 6.1
(MSE E||x - x_hat||^2, gain error E| ||x|| - ||x_hat|| |, cosine similarity
E cos(x, x_hat)) are taken from the oracle's metric definitions on the
float32 reconstruction.

  * dimension sweep: D in 8 .. 256 with K = 2048 (Fig. random analysis a-c);
  * capacity sweep: K in 2 .. 8192 with D = 256 (Fig. random analysis d-f).

Each point is averaged over --seeds draws (synth.gaussian_case); the
relative cosine gap (GSKM - KM) / KM is given with its range over the seeds.

Oracle spot checks: at a few points the float64 oracle trains both methods
(GSKM alone where its K-means would not fit in memory) free-running from
the same seeds and the same T; its metrics must
agree with the GPU's to --spot-rtol (the two trajectories can part after a
near-tie, so the check is on the metrics, not on the codebooks).

Usage (needs the built library and a GPU):
  python tests/sweep_gaussian.py [--seeds 3] [--iters 100] > sweep.md
Progress goes to stderr, the markdown tables to stdout.
"""
from __future__ import annotations

import argparse
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import synth  # noqa: E402
from oracle import gsrq_oracle as O  # noqa: E402

N = 10000
D_SWEEP = (8, 16, 32, 64, 128, 256)                 # at K = 2048
K_SWEEP = tuple(2 ** e for e in range(1, 14))       # 2 .. 8192 at D = 256
# (D, K, methods) checked against the oracle; the oracle's K-means forms
# every distance from an [N, K, D] difference, so it runs at small K * D only
SPOT = ((256, 2, "km gskm"), (256, 8, "km gskm"), (256, 32, "km gskm"),
        (8, 2048, "km gskm"), (256, 1024, "gskm"), (256, 2048, "gskm"))
METRICS = ("mse", "gain_err", "cos")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gpu_point(X, seeds, D, K, T, kmeans):
    import torch
    from paper_2607_01065_amd import gsrq as B
    Xd = torch.from_numpy(X).cuda()
    r = B.train_stage(Xd, D, K, T, seed_rows=seeds[None].astype(np.int32),
                      kmeans=kmeans, trace=False)
    gain, shape = r.gain[None].contiguous(), r.shape[None].contiguous()
    codes, _ = B.encode(Xd, gain, shape)
    xh = B.decode(codes, gain, shape, D, out_dtype=torch.float32)
    torch.cuda.synchronize()
    m = O.metrics(X.astype(np.float64), xh.cpu().numpy().astype(np.float64))
    m["iters"] = int(r.iters[0].item())
    return m


def oracle_point(X, seeds, K, T, kmeans):
    X64 = X.astype(np.float64)
    if kmeans:
        r = O.kmeans(X64, None, K, T, seeds)
        C = r["centroids"]
        xh = C[O.kmeans_assign(X64, C)]
    else:
        r = O.gskm(X64, None, K, T, seeds)
        a = O.gskm_assign(X64, r["gain"], r["shape"])
        xh = r["gain"][a, None] * r["shape"][a]
    m = O.metrics(X64, xh)
    m["iters"] = int(r["iters_run"])
    return m


def sweep(points, nseeds, T):
    rows = []
    for D, K in points:
        per = {"km": [], "gs": []}
        t0 = time.time()
        for s in range(nseeds):
            X, seeds = synth.gaussian_case(N, D, K, seed=s)
            per["km"].append(gpu_point(X, seeds, D, K, T, True))
            per["gs"].append(gpu_point(X, seeds, D, K, T, False))
        gaps = [(g["cos"] - k["cos"]) / k["cos"] for g, k in zip(per["gs"], per["km"])]
        row = dict(D=D, K=K, gap=float(np.mean(gaps)), gap_lo=float(min(gaps)),
                   gap_hi=float(max(gaps)))
        for side in ("km", "gs"):
            for k in METRICS + ("iters",):
                row[f"{side}_{k}"] = float(np.mean([m[k] for m in per[side]]))
        rows.append(row)
        log(f"D={D} K={K}: cos KM {row['km_cos']:.4f} GSKM {row['gs_cos']:.4f} "
            f"gap {100 * row['gap']:+.2f}% ({time.time() - t0:.1f} s)")
    return rows


def table(title, rows):
    out = [f"### {title}", "",
           "| D | K | MSE KM | MSE GSKM | gain err KM | gain err GSKM | cos KM | cos GSKM "
           "| cos gap (range) | iters KM / GSKM |",
           "|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for r in rows:
        out.append(
            f"| {r['D']} | {r['K']} | {r['km_mse']:.4g} | {r['gs_mse']:.4g} | "
            f"{r['km_gain_err']:.4g} | {r['gs_gain_err']:.4g} | {r['km_cos']:.4f} | "
            f"{r['gs_cos']:.4f} | {100 * r['gap']:+.2f}% "
            f"({100 * r['gap_lo']:+.2f} .. {100 * r['gap_hi']:+.2f}) | "
            f"{r['km_iters']:.0f} / {r['gs_iters']:.0f} |")
    return "\n".join(out) + "\n"


def spot_checks(T, rtol):
    out = ["### Oracle spot checks (seed 0, free-running, float64 oracle)", "",
           "| D | K | method | metric | GPU | oracle | rel. diff |",
           "|---:|---:|---|---|---:|---:|---:|"]
    worst = 0.0
    for D, K, which in SPOT:
        X, seeds = synth.gaussian_case(N, D, K, seed=0)
        for name, km in (("KM", True), ("GSKM", False)):
            if name.lower() not in which.split():
                continue
            t0 = time.time()
            g = gpu_point(X, seeds, D, K, T, km)
            o = oracle_point(X, seeds, K, T, km)
            for k in METRICS:
                rel = abs(g[k] - o[k]) / abs(o[k])
                worst = max(worst, rel)
                out.append(f"| {D} | {K} | {name} | {k} | {g[k]:.5g} | {o[k]:.5g} | {rel:.2e} |")
            out.append(f"| {D} | {K} | {name} | iters | {g['iters']} | {o['iters']} | |")
            log(f"spot D={D} K={K} {name}: oracle {time.time() - t0:.1f} s")
    return "\n".join(out) + "\n", worst


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--seeds", type=int, default=3)
    ap.add_argument("--iters", type=int, default=100, help="T, the iteration cap")
    ap.add_argument("--spot-rtol", type=float, default=0.02)
    ap.add_argument("--no-spot", action="store_true", help="skip the oracle spot checks")
    a = ap.parse_args(argv)
    import torch
    from paper_2607_01065_amd import gsrq as B
    if not torch.cuda.is_available():
        sys.exit("the sweep runs on the GPU path; no GPU is visible")
    B.load_library()
    print(f"N = {N}, x ~ N(0, I_D), T = {a.iters} (stop when an assignment repeats), "
          f"{a.seeds} seeds per point; metrics of Sec. 6.1 on the GPU's float32 "
          "reconstruction; cos gap = (cos GSKM - cos KM) / cos KM, mean and range over seeds.\n")
    print(table("Dimension sweep (K = 2048)", sweep([(D, 2048) for D in D_SWEEP], a.seeds, a.iters)))
    print(table("Capacity sweep (D = 256)", sweep([(256, K) for K in K_SWEEP], a.seeds, a.iters)))
    if not a.no_spot:
        text, worst = spot_checks(a.iters, a.spot_rtol)
        print(text)
        print(f"worst relative metric difference GPU vs oracle: {worst:.2e} (limit {a.spot_rtol})")
        if worst > a.spot_rtol:
            sys.exit(1)
    sys.stdout.flush()


if __name__ == "__main__":
    main()
