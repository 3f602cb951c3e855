"""OrthoMerge-G-TIES (App. F, the geometry-aware baseline), float64 (test infrastructure).

One 2-D weight matrix W_0 (m x n, m >= n) and K experts W_i = W_0 + tau_i.  The steps follow
App. F in its order:

  1. one-sided orthogonal Procrustes per expert: R_i = argmin_{R in O(n)} |W_0 R - W_i|_F,
     R_i = U V^T from the SVD W_0^T W_i = U S V^T                       (rotation on the input side)
  2. inverse Cayley map A_i = (R_i + I)^{-1} (R_i - I)                (skew-symmetric)
  3. magnitude-corrected mean A = (mean_i |A_i|_F) * sum_i A_i / |sum_i A_i|_F
  4. forward Cayley map R = (I - A)^{-1} (I + A), W_rot = W_0 R
  5. residuals delta_i = W_i - W_0 R_i, merged by the TIES rule (TopKMask with count k,
     sign election, disjoint mean)
  6. W_OM = W_rot + lambda * tau_TIES(delta)

Readings (the paper is silent on them): the residuals enter TIES as binary32 (the official
implementation's precision), so the TopKMask ranks binary32 magnitudes with the flat-index tie
rule of the other TIES paths; the merged residual update u = lambda * t is carried as binary32,
and W_OM = W_rot + u is rounded once to the storage type.  A skew sum that cancels to rounding
level (|sum A_i|_F <= 1e-12 sum |A_i|_F) gives A = 0 (no rotation).  The Procrustes rotation
is unique only when W_0^T W_i is nonsingular, which needs m >= n (a wide W_0 has rank < n); wide
matrices are outside this operator.  The SVD, the
linear solves and the TIES steps use library primitives and oracle/ties.py.
"""
import numpy as np

from oracle import numerics as nm
from oracle import ties


def procrustes(w0, wi):
    """R = U V^T for W_0^T W_i = U S V^T (App. F, one-sided Procrustes)."""
    u, s, vt = np.linalg.svd(np.asarray(w0, dtype=np.float64).T @ np.asarray(wi, dtype=np.float64))
    if s[-1] == 0.0:
        raise np.linalg.LinAlgError("W_0^T W_i is singular: the Procrustes rotation is not unique")
    return u @ vt


def inverse_cayley(r):
    """A = (R + I)^{-1} (R - I)."""
    n = r.shape[0]
    eye = np.eye(n)
    return np.linalg.solve(r + eye, r - eye)


def forward_cayley(a):
    """R = (I - A)^{-1} (I + A)."""
    n = a.shape[0]
    eye = np.eye(n)
    return np.linalg.solve(eye - a, eye + a)


# |sum A_i|_F at or below this fraction of sum |A_i|_F counts as a cancelled sum
CANCEL_REL = 1e-12


def merged_skew(skews):
    """(1/K sum |A_i|_F) * sum A_i / |sum A_i|_F.  The direction sum / |sum| is undefined when the
    skews cancel and is rounding noise when they cancel to rounding level: a sum of norm at most
    CANCEL_REL * sum |A_i|_F gives A = 0 (no rotation)."""
    total = sum(skews)
    norm = np.linalg.norm(total)
    norms = sum(np.linalg.norm(a) for a in skews)
    if norm <= CANCEL_REL * norms:
        return np.zeros_like(total)
    return (norms / len(skews) / norm) * total


def rotation_part(w0, ws):
    """Steps 1-4: the experts' rotations R_i, their skews A_i, the merged A and R, and W_rot."""
    w0 = np.asarray(w0, dtype=np.float64)
    rs = [procrustes(w0, wi) for wi in ws]
    skews = [inverse_cayley(r) for r in rs]
    a = merged_skew(skews)
    r = forward_cayley(a)
    return dict(rotations=rs, skews=skews, a=a, r=r, w_rot=w0 @ r)


def orthomerge_ties(w0, deltas, k, lam=1.0, dtype="bf16"):
    """OrthoMerge-G-TIES for one matrix.  w0 and deltas are storage arrays (m x n); k is the
    TopKMask count of each residual.  Returns dict(out=storage array of W_OM, w_rot, residuals
    (binary32), masks, u32 (the merged residual update), parts of rotation_part)."""
    m, n = np.shape(w0)
    if m < n:
        raise ValueError("OrthoMerge's Procrustes rotation needs rows >= cols")
    w0f = nm.to_f64(np.asarray(w0).ravel(), dtype).reshape(m, n)
    ws = [w0f + nm.to_f64(np.asarray(d).ravel(), dtype).reshape(m, n) for d in deltas]
    rot = rotation_part(w0f, ws)
    res = [(wi - w0f @ ri).astype(np.float32) for wi, ri in zip(ws, rot["rotations"])]
    masks = [ties.topk_mask(d.ravel(), k, "f32") for d in res]
    t, gamma = ties.ties_merge([d.ravel() for d in res], masks, "f32")
    u32 = ties.merged_update(t, lam).astype(np.float32)
    out = nm.from_f64(rot["w_rot"].ravel() + u32.astype(np.float64), dtype)
    return dict(out=out, residuals=res, masks=masks, u32=u32, gamma=gamma, **rot)
