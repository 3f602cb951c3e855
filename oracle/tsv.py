"""TSV-Merge of App. F, float64 (test infrastructure).

For one 2-D matrix with base W_0 and deltas Delta_i (i = 1..K):
  1. Delta_i ~ U_i^(r) Sigma_i^(r) V_i^(r)T, the exact top-r singular triplets
     (full LAPACK SVD, truncated);
  2. U = [U_1^(r) | ... | U_K^(r)], V likewise, Sigma = blockdiag(Sigma_i^(r));
  3. orthogonalisation in the Procrustes form: U_perp = P_U Q_U^T from the
     thin SVD U = P_U D_U Q_U^T (equal to U (U^T U)^{-1/2} at full rank), same
     for V;
  4. Delta_hat = U_perp Sigma V_perp^T and W = W_0 + alpha * Delta_hat.

The top-r truncation is only well defined when sigma_r > sigma_{r+1}; tests
plant a spectral gap for that reason.
"""
import numpy as np

from .numerics import from_f64, to_f64


def truncated_svd(d, r):
    u, s, vt = np.linalg.svd(np.asarray(d, dtype=np.float64), full_matrices=False)
    return u[:, :r], s[:r], vt[:r].T


def procrustes(x):
    """P Q^T from the thin SVD X = P D Q^T."""
    p, _, qt = np.linalg.svd(x, full_matrices=False)
    return p @ qt


def tsv_delta(deltas, r, factors=None):
    """Delta_hat for one matrix.  ``factors`` = list of (U_i, s_i, V_i) to skip step 1."""
    if factors is None:
        factors = [truncated_svd(d, r) for d in deltas]
    u = np.concatenate([f[0] for f in factors], axis=1)
    s = np.concatenate([f[1] for f in factors])
    v = np.concatenate([f[2] for f in factors], axis=1)
    if u.shape[1] > min(u.shape[0], v.shape[0]):
        raise ValueError("K*r exceeds min(rows, cols)")
    up = procrustes(u)
    vp = procrustes(v)
    return (up * s) @ vp.T, dict(u=u, s=s, v=v, u_perp=up, v_perp=vp)


def tsv_merge(base, deltas, r, alpha=1.0, dtype="bf16", shape=None, factors=None):
    """W_TSV = W_0 + alpha * Delta_hat rounded once to the storage format."""
    w0 = to_f64(base, dtype).reshape(shape)
    ds = [to_f64(d, dtype).reshape(shape) for d in deltas]
    dh, info = tsv_delta(ds, r, factors)
    out = from_f64(w0 + np.float64(alpha) * dh, dtype)
    return out.reshape(shape), dh, info
