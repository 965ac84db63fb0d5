"""Helpers shared by the GPU parity tests (comparison rules, not arithmetic of
the method: expected values always come from the oracle)."""
import sys

import numpy as np

from oracle import gsrq_oracle as O

MARGIN = 1e-4          # relative top-2 margin above which indices must agree
CB_RTOL = 1e-5         # codebook / reconstruction tolerance (float32 path)


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


def check_assignment(X, gain, shape, k_gpu, what=""):
    """Margin rule: indices equal the oracle's wherever the relative top-2
    margin exceeds MARGIN; below it the GPU choice must still be within the
    margin of the best score.  Returns (n_above_mismatch, n_below, n_rows)."""
    X = np.asarray(X, np.float64)
    k_gpu = np.asarray(k_gpu, np.int64)
    S = O.gskm_scores(X, gain, shape)
    k_ref = np.argmax(S, axis=1)
    marg = O.assignment_margin(X, gain, shape)
    energy = np.maximum(np.sum(X * X, axis=1), 1e-30)
    above = marg > MARGIN
    bad = np.nonzero(above & (k_gpu != k_ref))[0]
    assert bad.size == 0, (f"{what}: {bad.size} index mismatches above the margin, first rows "
                           f"{bad[:5]}, gpu {k_gpu[bad[:5]]} ref {k_ref[bad[:5]]} margin {marg[bad[:5]]}")
    assert np.all((k_gpu >= 0) & (k_gpu < S.shape[1])), what
    rows = np.arange(X.shape[0])
    slack = (S[rows, k_ref] - S[rows, k_gpu]) / energy
    assert np.all(slack <= MARGIN), f"{what}: below-margin choice worse than the margin"
    return int(bad.size), int(np.sum(~above & (k_gpu != k_ref))), X.shape[0]


def rel_err(a, b, floor):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.abs(a - b) / np.maximum(np.abs(b), floor)
