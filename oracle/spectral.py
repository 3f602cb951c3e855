"""ISO-Merger (Sec. 4.2; App. E; Algorithm 1), float64 (test infrastructure).

One 2-D weight matrix at a time: base W_0 and K expert matrices
W_i = W_0 + Delta_i.  The steps follow App. E in its order:

  1. thin SVDs W_0 = U_0 Sigma_0 V_0^T and W_i = U_i Sigma_i V_i^T   (App. E Setup)
  2. joint sign canonicalisation s_ik = sign(<u_0k, u_ik>), sign(0) := 1
     applied to u_ik and v_ik                                        (App. E, gauge)
  3. frame displacements Delta U_i = U_i - U_0, Delta V_i = V_i - V_0 and
     tangent projection Pi_U0(D) = D - U_0 sym(U_0^T D)              (App. E, tangent)
  4. D_keep keeps the leading k_keep = round(rho_keep q) modes       (App. E, eq. of D_keep)
  5. proxies g_i = xi~_U,i Sigma_0 V_0^T + U_0 Sigma_0 xi~_V,i^T and
     Gram Gamma_ij = <g_i, g_j>_F                                    (App. E, retention)
  6. drop zero-norm proxies, solve (Gamma + lambda_ridge I) c = diag Gamma,
     clip c to [c_min, c_max]                                        (App. E, retention)
  7. xi_* = Pi(sum_i c_i xi~_i), U_* = polar(U_0 + xi_U*),
     V_* = polar(V_0 + xi_V*), W_* = U_* Sigma_0 V_*^T                (App. E, retraction)

The SVD is LAPACK's (numpy.linalg.svd, a library primitive); polar(X) is
P Q^T from the thin SVD X = P S Q^T, as the paper defines it.  The Gram
system is solved by Cholesky (the paper names no solver; the matrix is SPD).
"""
import math

import numpy as np


def thin_svd(w):
    """W = U diag(s) V^T with s nonincreasing; returns (U, s, V)."""
    u, s, vt = np.linalg.svd(np.asarray(w, dtype=np.float64), full_matrices=False)
    return u, s, vt.T


def sym(a):
    return 0.5 * (a + a.T)


def tangent_project(anchor, d):
    """Pi_{U_0}(D) = D - U_0 sym(U_0^T D): orthogonal projection onto T_{U_0} St."""
    return d - anchor @ sym(anchor.T @ d)


def polar(x):
    """polar(X) = P Q^T for the thin SVD X = P S Q^T."""
    p, _, qt = np.linalg.svd(x, full_matrices=False)
    return p @ qt


def k_keep_of(rho_keep, q):
    """k_keep = round(rho_keep * q), halves rounded up, formed in float64."""
    return int(math.floor(rho_keep * q + 0.5))


def canonicalize(u0, u, v):
    """Joint sign canonicalisation against the base (App. E): sign(0) := 1."""
    s = np.sign(np.sum(u0 * u, axis=0))
    s[s == 0] = 1.0
    return u * s, v * s


def iso_merge_factors(u0, s0, v0, experts, rho_keep=0.9, ridge=1e-12, c_min=0.0, c_max=1.5):
    """Algorithm 1 body from precomputed SVDs.

    ``experts`` is a list of (U_i, s_i, V_i).  Returns a dict with W_star,
    U_star, V_star, coefficients c (K,), Gram, the masked tangents and the
    aggregate tangents xi_U, xi_V.
    """
    q = s0.size
    kk = k_keep_of(rho_keep, q)
    keep = (np.arange(q) < kk).astype(np.float64)            # D_keep, modes 1..k_keep
    S0 = np.diag(s0)
    xu_t, xv_t, g = [], [], []
    for (u, s, v) in experts:
        u, v = canonicalize(u0, u, v)
        xu = tangent_project(u0, u - u0) * keep              # xi~_U,i = Pi(Delta U_i) D_keep
        xv = tangent_project(v0, v - v0) * keep
        xu_t.append(xu)
        xv_t.append(xv)
        g.append(xu @ S0 @ v0.T + u0 @ S0 @ xv.T)
    K = len(experts)
    nz = [i for i in range(K) if np.linalg.norm(g[i]) > 0]
    c = np.zeros(K)
    gram = np.zeros((K, K))
    for i in range(K):
        for j in range(K):
            gram[i, j] = np.sum(g[i] * g[j])
    if nz:
        gam = gram[np.ix_(nz, nz)]
        b = np.diag(gam).copy()
        chol = np.linalg.cholesky(gam + ridge * np.eye(len(nz)))
        y = np.linalg.solve(chol, b)
        cbar = np.linalg.solve(chol.T, y)
        c[nz] = np.clip(cbar, c_min, c_max)
    agg_u = sum(c[i] * xu_t[i] for i in range(K))
    agg_v = sum(c[i] * xv_t[i] for i in range(K))
    xi_u = tangent_project(u0, agg_u)
    xi_v = tangent_project(v0, agg_v)
    u_star = polar(u0 + xi_u)
    v_star = polar(v0 + xi_v)
    w_star = u_star @ S0 @ v_star.T
    return dict(w_star=w_star, u_star=u_star, v_star=v_star, c=c, gram=gram,
                xi_u=xi_u, xi_v=xi_v, xu_masked=xu_t, xv_masked=xv_t, k_keep=kk)


def iso_merge(w0, deltas, rho_keep=0.9, ridge=1e-12, c_min=0.0, c_max=1.5):
    """Algorithm 1 for one matrix: W_i = W_0 + Delta_i (raw expert deltas)."""
    w0 = np.asarray(w0, dtype=np.float64)
    u0, s0, v0 = thin_svd(w0)
    experts = [thin_svd(w0 + np.asarray(d, dtype=np.float64)) for d in deltas]
    res = iso_merge_factors(u0, s0, v0, experts, rho_keep, ridge, c_min, c_max)
    res["s0"] = s0
    return res


def average_1d(w0, experts):
    """1-D parameters: w_* = w_0 + (1/K) sum_i (w_i - w_0) (App. E, scope)."""
    w0 = np.asarray(w0, dtype=np.float64)
    return w0 + sum(np.asarray(w, dtype=np.float64) - w0 for w in experts) / len(experts)


def spectral_diagnostics(w0, w1):
    """Spectral drift of one matrix from W_0 to W_1 = W_0 + Delta W (Sec. 3):
    delta_Sigma = |sigma(W_1) - sigma(W_0)|_2 / |W_0|_F,
    rho_Sigma = |sigma(W_1) - sigma(W_0)|_2 / |Delta W|_F,
    kappa_spec = (d_out d_in / q) |diag(U_0^T Delta W V_0)|_2^2 / |Delta W|_F^2."""
    w0 = np.asarray(w0, dtype=np.float64)
    w1 = np.asarray(w1, dtype=np.float64)
    dw = w1 - w0
    u0, s0, v0 = thin_svd(w0)
    s1 = np.linalg.svd(w1, compute_uv=False)
    d = np.linalg.norm(s1 - s0)
    ndw = np.linalg.norm(dw)
    diag = np.einsum("ik,ij,jk->k", u0, dw, v0)
    m, n = w0.shape
    return dict(delta_sigma=d / np.linalg.norm(w0), rho_sigma=d / ndw,
                kappa_spec=(m * n / min(m, n)) * np.sum(diag ** 2) / ndw ** 2)


def spectrum_interpolate(w0, w_rl, alpha):
    """W~(alpha) = U_RL [(1 - alpha) Sigma_0 + alpha Sigma_RL] V_RL^T (Sec. 3, base spectrum restored
    at alpha = 0 with the trained frames kept)."""
    s0 = np.linalg.svd(np.asarray(w0, dtype=np.float64), compute_uv=False)
    u, s, v = thin_svd(w_rl)
    return (u * ((1.0 - alpha) * s0 + alpha * s)) @ v.T


def truncation_rank(q, rank_frac):
    """r = max(1, floor(rank_frac q)), the integer truncation rank of the rank-sensitivity study."""
    return max(1, int(math.floor(rank_frac * q)))


def transport_ratios(w_in, w_end, rank_frac=0.9):
    """Unexplained-update ratios of one transition W_j -> W_i (Sec. 3, Prop. 3.1), with W_j = w_in the
    incoming checkpoint and W_i = w_end the learned endpoint, both truncated to their top-r SVD:
      W_mix = P_j W_i^(r) Q_j,  W_L = P_j W_i^(r),  W_R = W_i^(r) Q_j,  W_iso = U_i^(r) Sigma_j^(r) V_i^(r)T,
      u_h = |W_i^(r) - W_h|_F / |W_i^(r) - W_j^(r)|_F   (NaN when the denominator is zero),
    with P_j = U_j^(r) U_j^(r)T and Q_j = V_j^(r) V_j^(r)T.  Also returns the rank-r boundary gap,
    min over both endpoints of sigma_r - sigma_{r+1} (sigma_{q+1} := 0): the transition is admissible
    when it is positive."""
    w_in = np.asarray(w_in, dtype=np.float64)
    w_end = np.asarray(w_end, dtype=np.float64)
    q = min(w_in.shape)
    r = truncation_rank(q, rank_frac)
    uj, sj, vj = thin_svd(w_in)
    ui, si, vi = thin_svd(w_end)
    wi = (ui[:, :r] * si[:r]) @ vi[:, :r].T
    wj = (uj[:, :r] * sj[:r]) @ vj[:, :r].T
    p = uj[:, :r] @ uj[:, :r].T
    qm = vj[:, :r] @ vj[:, :r].T
    recon = {
        "mix": p @ wi @ qm,
        "L": p @ wi,
        "R": wi @ qm,
        "iso": (ui[:, :r] * sj[:r]) @ vi[:, :r].T,
    }
    den = np.linalg.norm(wi - wj)
    u = {h: (np.linalg.norm(wi - x) / den if den > 0 else math.nan) for h, x in recon.items()}

    def gap(s):
        return s[r - 1] - (s[r] if r < q else 0.0)

    u["gap"] = min(gap(sj), gap(si))
    u["rank"] = r
    return u


def svd_reconstruction(w0):
    """W_rec = U Sigma V^T from the thin SVD of W_0 (App. G, the reconstruction whose spectrum the
    precision study compares with W_0's)."""
    u, s, v = thin_svd(w0)
    return (u * s) @ v.T


def spectral_error(w0, w_rec):
    """Mean squared spectral error of App. G: eps_sigma = (1/q) |sigma(W_rec) - sigma(W_0)|_2^2,
    q = min(d_out, d_in), both spectra sorted nonincreasing."""
    w0 = np.asarray(w0, dtype=np.float64)
    s0 = np.linalg.svd(w0, compute_uv=False)
    s1 = np.linalg.svd(np.asarray(w_rec, dtype=np.float64), compute_uv=False)
    return float(np.sum((s1 - s0) ** 2) / min(w0.shape))
