"""Whole-workload parity: the oracle over every matrix of a full-size
workload, and a summary per workload (largest relative Frobenius error, its
ratio to the band, and the fraction of matrices within the band).

The oracle runs on the host in a pool of single-threaded workers (one matrix
per task); numpy's LAPACK releases the interpreter lock, so the pool scales
with the host cores given to the run (at most 16 are used)."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle.shampoo_oracle as O
from tests.gpu_util import rel, say


def band(kappa):
    """Root tolerance for a damped condition number: 1e-3 up to 1e6, 5e-3
    above (to 1e8)."""
    return 1e-3 if kappa <= 1e6 else 5e-3


def pool_map(fn, items):
    from threadpoolctl import threadpool_limits
    items = list(items)
    with threadpool_limits(1), ThreadPoolExecutor(max(1, min(16, os.cpu_count() or 4))) as ex:
        return list(ex.map(fn, items))


def summarize(name, errs, bands):
    """Prints and returns (max error, max error / band, fraction within band)."""
    errs, bands = np.asarray(errs, dtype=np.float64), np.asarray(bands, dtype=np.float64)
    ratio = errs / bands
    frac = float(np.mean(ratio <= 1.0))
    say(f"{name}: {len(errs)} matrices, max rel err {errs.max():.3e}, max err/band {ratio.max():.3f}, "
        f"within band {frac:.4f}")
    return float(errs.max()), float(ratio.max()), frac


def root_parity(A, X, p, eps, eps_relative=False, lam_max=None, eig=None):
    """One GPU root X (host array) against the oracle's root of the same fp32
    input A: (relative error, damped condition number, band)."""
    eig = O.sym_eig(A) if eig is None else eig
    Xo, st, _ = O.inv_root(A, p, eps, eps_relative, lam_max, eig=eig)
    assert st == O.CONVERGED, "oracle: damped matrix not positive definite"
    kappa = O.cond_damped(A, eps, eps_relative, lam_max, eig=eig)
    return rel(X, Xo), kappa, band(kappa)
