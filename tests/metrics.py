"""Comparison metrics shared by the tests (fp64, no assumptions of orthonormality)."""
import numpy as np


def proj_dist(P, Pref, block=1024):
    """||P P^T - Pref Pref^T||_F, formed explicitly one row block at a time (the
    Gram-based shortcut cancels catastrophically near zero)."""
    P = np.asarray(P, dtype=np.float64)
    Pref = np.asarray(Pref, dtype=np.float64)
    s = P.shape[0]
    tot = 0.0
    for i in range(0, s, block):
        d = P[i:i + block] @ P.T - Pref[i:i + block] @ Pref.T
        tot += float(np.sum(d * d))
    return float(np.sqrt(tot))


def orth_err(P):
    P = np.asarray(P, dtype=np.float64)
    return float(np.abs(P.T @ P - np.eye(P.shape[1])).max())


def max_rel_violation(x, ref, rtol, atol):
    """max over elements of |x - ref| / (atol + rtol |ref|); <= 1 means within tolerance."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(x - ref) / (atol + rtol * np.abs(ref)))) if x.size else 0.0
