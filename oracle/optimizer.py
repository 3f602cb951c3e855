"""ISO-Optimizer step with AdamW or Muon as the base rule (ISO-AdamW, ISO-Muon; Sec. 4.3), float64.

Test infrastructure: only the tests, the smoke check and the CPU baseline use it.  One weight
matrix W = U Sigma_0 V^T trained through its frame variables with Sigma_0 fixed, in the order
of Sec. 4.3:

  1. factor gradients G_U = G_W V Sigma_0, G_V = G_W^T U Sigma_0     (chain rule of W = U S V^T)
  2. the base rule (AdamW or Muon, decoupled weight decay) on U and on V with their own state
  3. polar retraction U+ = polar(U~), V+ = polar(V~), polar(X) = P Q^T for X = P D Q^T
  4. W+ = U+ Sigma_0 V+^T

AdamW, per entry, with t the step being taken:
  m <- b1 m + (1 - b1) g;  v <- b2 v + (1 - b2) g^2;
  x <- x - lr ((m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps) + wd x).

Muon (the paper names the rule without restating it; this is its usual form), per matrix x of
shape rows x q with momentum buffer b:
  b <- mu b + g;  d = g + mu b (Nesterov) or d = b;  o = polar(d);
  x <- x - lr (sqrt(max(1, rows / q)) o + wd x).
Muon approximates polar(d) with a few quintic Newton-Schulz steps; here o is the polar factor
itself.  The zero direction (a zero gradient on a zero momentum buffer) has no polar factor: it
takes o = 0, as the sign of zero is zero, so x only decays by lr wd x.
"""
import numpy as np

from .spectral import polar


def factor_gradients(g_w, u, v, s):
    """G_U = G_W V Sigma_0 and G_V = G_W^T U Sigma_0 (Sec. 4.3, factor gradients)."""
    return g_w @ (v * s), g_w.T @ (u * s)


def adamw(x, g, m, v, t, lr, b1, b2, eps, wd):
    """One AdamW update of x; returns (x, m, v), all new arrays."""
    m = b1 * m + (1.0 - b1) * g
    v = b2 * v + (1.0 - b2) * (g * g)
    bc1 = 1.0 - b1 ** t
    bc2 = 1.0 - b2 ** t
    x = x - lr * ((m / bc1) / (np.sqrt(v / bc2) + eps) + wd * x)
    return x, m, v


def iso_adamw_step(u, v, s, g_w, state, t, lr, b1=0.9, b2=0.999, eps=1e-8, wd=0.0):
    """One ISO-AdamW step.  state = (m_u, v_u, m_v, v_v).  Returns (U+, V+, W+, new state)."""
    m_u, v_u, m_v, v_v = state
    g_u, g_v = factor_gradients(g_w, u, v, s)
    u_t, m_u, v_u = adamw(u, g_u, m_u, v_u, t, lr, b1, b2, eps, wd)
    v_t, m_v, v_v = adamw(v, g_v, m_v, v_v, t, lr, b1, b2, eps, wd)
    u_p = polar(u_t)
    v_p = polar(v_t)
    return u_p, v_p, (u_p * s) @ v_p.T, (m_u, v_u, m_v, v_v)


def muon(x, g, b, lr, mu, wd, nesterov=True):
    """One Muon update of x (rows x q) with momentum buffer b; returns (x, b), new arrays."""
    b = mu * b + g
    d = g + mu * b if nesterov else b
    o = polar(d) if d.any() else np.zeros_like(d)
    scale = np.sqrt(max(1.0, x.shape[0] / x.shape[1]))
    return x - lr * (scale * o + wd * x), b


def iso_muon_step(u, v, s, g_w, state, lr, mu=0.95, wd=0.0, nesterov=True):
    """One ISO-Muon step.  state = (b_u, b_v).  Returns (U+, V+, W+, new state)."""
    b_u, b_v = state
    g_u, g_v = factor_gradients(g_w, u, v, s)
    u_t, b_u = muon(u, g_u, b_u, lr, mu, wd, nesterov)
    v_t, b_v = muon(v, g_v, b_v, lr, mu, wd, nesterov)
    u_p = polar(u_t)
    v_p = polar(v_t)
    return u_p, v_p, (u_p * s) @ v_p.T, (b_u, b_v)
