"""Element-wise data-free merges of App. F, restated in float64 (test infrastructure).

Notation follows the paper's App. F: base theta_0 (here ``base``), task vectors
tau_i = theta_i - theta_0 (here ``deltas[i]``), and the merged model
theta_0 + tau_merge.  All inputs are storage arrays (bf16 as uint16 bit
patterns, fp32 as float32) of one select unit, flattened row-major.

Readings where the paper is silent (each is also listed in the design doc):
  * TopKMask ties at the threshold go to the lower flat index, so exactly k
    entries are kept; k itself comes from the density by round-half-up.
  * sign(.) in the election is the sign of the exact real sum; sign 0 leaves
    the agreeing set empty, so the merged coordinate is 0.
  * Every merged sum is formed in float64 from +0.0 adding the terms in
    expert order; the mean divides that sum by the count in float64; then
    u = lambda * t, v = w0 + u, and v is rounded once to the output format.
"""
import numpy as np

from .numerics import (exact_sum_sign, from_f64, magnitude_key, sequential_sum, to_f64)

NO_SELECT_KEY = 0xFFFFFFFF


def _check_finite(vals, what):
    if not np.all(np.isfinite(vals)):
        raise FloatingPointError(f"non-finite value in {what}")


def topk_mask(delta, k, dtype):
    """TopKMask(|tau_i|, rho) of App. F (TIES "Trim"), brute-force form.

    Entry p is kept iff it is among the first k entries of the order
    (|tau| descending, flat index ascending).  Full sort of all entries.
    """
    x = to_f64(delta, dtype).ravel()
    _check_finite(x, "delta")
    n = x.size
    if not 0 <= k <= n:
        raise ValueError("k out of range")
    order = np.lexsort((np.arange(n), -np.abs(x)))
    m = np.zeros(n, dtype=bool)
    m[order[:k]] = True
    return m


def topk_mask_joint(deltas, k, dtype):
    """TopKMask of one delta held in pieces (App. F, TIES "Trim" with tau_i the whole-model
    delta): the mask of the pieces concatenated in order, split back into one mask per piece."""
    flat = np.concatenate([np.asarray(d).ravel() for d in deltas])
    m = topk_mask(flat, k, dtype)
    out, o = [], 0
    for d in deltas:
        n = np.asarray(d).size
        out.append(m[o:o + n])
        o += n
    return out


def topk_descriptor(delta, k, dtype):
    """Threshold description of the same TopKMask, found by partial selection.

    Returns (T_key, n_above, tie_quota, tie_cutoff) where T_key is the storage
    bit pattern of the k-th largest magnitude, n_above = #{|tau| > T},
    tie_quota = k - n_above and tie_cutoff is N when every entry with
    |tau| == T is kept, else one past the flat index of the tie_quota-th entry
    with |tau| == T.  Entry p is kept iff key_p > T_key or (key_p == T_key and
    p < tie_cutoff).  For k = 0: (0xFFFFFFFF, 0, 0, 0).
    """
    x = to_f64(delta, dtype).ravel()
    _check_finite(x, "delta")
    n = x.size
    if not 0 <= k <= n:
        raise ValueError("k out of range")
    if k == 0:
        return (NO_SELECT_KEY, 0, 0, 0)
    a = np.abs(x)
    t = np.partition(a, n - k)[n - k]           # k-th largest magnitude
    n_above = int(np.count_nonzero(a > t))
    quota = k - n_above
    ties = np.flatnonzero(a == t)
    cutoff = n if quota == ties.size else int(ties[quota - 1]) + 1
    t_key = int(magnitude_key(from_f64(np.array([t]), dtype), dtype)[0])
    return (t_key, n_above, quota, cutoff)


def topk_descriptor_counting(delta, k, dtype="bf16"):
    """The same threshold description as ``topk_descriptor``, found by counting (bf16 only).

    The bf16 magnitude key (the bit pattern of |tau|, 15 bits) is monotone in
    |tau|, so the k-th largest magnitude is the largest key T whose count of
    keys >= T reaches k.  n_above counts the keys > T; the tie cutoff is one
    past the flat index of the quota-th entry with key T (N when all of them
    are kept).  Linear in N, for the 10^8-10^9-entry tensors of the
    whole-stack parity checks.
    """
    if dtype != "bf16":
        raise ValueError("counting form is for 15-bit bf16 keys")
    b = np.asarray(delta, dtype=np.uint16).ravel()
    n = b.size
    if not 0 <= k <= n:
        raise ValueError("k out of range")
    key = b & np.uint16(0x7FFF)
    hist = np.bincount(key, minlength=1 << 15).astype(np.int64)
    if np.any(hist[0x7F80:]):
        raise FloatingPointError("non-finite value in delta")
    if k == 0:
        return (NO_SELECT_KEY, 0, 0, 0)
    at_or_above = np.cumsum(hist[::-1])[::-1]          # at_or_above[c] = #{key >= c}
    t_key = int(np.flatnonzero(at_or_above >= k)[-1])
    n_above = int(at_or_above[t_key] - hist[t_key])
    quota = k - n_above
    if quota == hist[t_key]:
        cutoff = n
    else:
        ties = np.flatnonzero(key == np.uint16(t_key))
        cutoff = int(ties[quota - 1]) + 1
    return (t_key, n_above, quota, cutoff)


def mask_from_descriptor(delta, desc, dtype):
    t_key, _, _, cutoff = desc
    key = magnitude_key(np.asarray(delta).ravel(), dtype).astype(np.int64)
    idx = np.arange(key.size)
    return (key > t_key) | ((key == t_key) & (idx < cutoff))


def elect_sign(terms):
    """gamma^p = sign(sum_i tilde tau_i^p), exact (App. F, TIES "Elect")."""
    return exact_sum_sign(terms)


def ties_merge(deltas, masks, dtype):
    """tau_TIES of App. F: mean over A_p = {i : tilde tau_i != 0, sign = gamma}.

    Returns (t, gamma) with t the float64 disjoint mean (0 where A_p is empty).
    """
    xs = [to_f64(d, dtype).ravel() for d in deltas]
    for x in xs:
        _check_finite(x, "delta")
    tt = [np.where(m, x, 0.0) for x, m in zip(xs, masks)]      # tilde tau = m (.) tau
    gamma = elect_sign(tt)
    agree = [(t != 0) & (np.sign(t).astype(np.int8) == gamma) for t in tt]
    total = sequential_sum(tt, agree)
    count = np.sum(np.stack(agree), axis=0)
    t = np.where(count > 0, total / np.maximum(count, 1), 0.0)
    return t, gamma


def ta_merge(deltas, dtype):
    """Task Arithmetic of App. F before scaling: sum_i tau_i."""
    xs = [to_f64(d, dtype).ravel() for d in deltas]
    for x in xs:
        _check_finite(x, "delta")
    return sequential_sum(xs)


def ram_merge(deltas, eps, dtype):
    """RAM of App. F: mean over A_p = {i : |tau_i^p| > eps}, 0 if A_p is empty.

    (c^p = 1 gives tau_j itself, which is the same mean.)
    """
    xs = [to_f64(d, dtype).ravel() for d in deltas]
    for x in xs:
        _check_finite(x, "delta")
    act = [np.abs(x) > eps for x in xs]
    total = sequential_sum(xs, act)
    count = np.sum(np.stack(act), axis=0)
    return np.where(count > 0, total / np.maximum(count, 1), 0.0)


def merged_update(t, lam):
    """u = lambda * t: the merged task vector tau_merge (App. F) in float64."""
    return np.float64(lam) * t


def apply_update(base, u, dtype):
    """theta_merge = theta_0 + tau_merge, rounded once to the storage format."""
    w = to_f64(base, dtype).ravel()
    _check_finite(w, "base")
    return from_f64(w + u, dtype)


def merge_unit(base, deltas, dtype, mode, k=None, lam=1.0, eps=1e-5, masks=None):
    """Whole element-wise path for one select unit.

    mode "ties": Trim (TopKMask with count k) -> Elect -> disjoint Merge ->
    theta_0 + lambda*tau; "ta": theta_0 + lambda*sum tau_i; "ram": RAM mean
    (lambda kept as a plain factor, 1 by default as in the paper).
    Returns dict(out=storage array, tau=float32 merged update, u=float64,
    gamma=int8 or None, masks=list or None).
    """
    gamma = None
    if mode == "ties":
        if masks is None:
            masks = [topk_mask(d, k, dtype) for d in deltas]
        t, gamma = ties_merge(deltas, masks, dtype)
    elif mode == "ta":
        t = ta_merge(deltas, dtype)
    elif mode == "ram":
        t = ram_merge(deltas, eps, dtype)
    else:
        raise ValueError(mode)
    u = merged_update(t, lam)
    return dict(out=apply_update(base, u, dtype), tau=u.astype(np.float32), u=u, gamma=gamma, masks=masks)


def merge_at(base_vals, delta_vals, mode, descs=None, idx=None, dtype="bf16", lam=1.0, eps=1e-5):
    """Merged outputs at sampled coordinates only.

    ``base_vals`` (n,) and ``delta_vals`` (K, n) are the storage values at flat
    indices ``idx`` of a unit whose TopKMask thresholds are ``descs`` (one
    descriptor per delta, from topk_descriptor).  Used for parity at sizes
    where the whole tensor would not fit the oracle's time budget.
    """
    K = len(delta_vals)
    if mode == "ties":
        masks = []
        for i in range(K):
            t_key, _, _, cutoff = descs[i]
            key = magnitude_key(delta_vals[i], dtype).astype(np.int64)
            masks.append((key > t_key) | ((key == t_key) & (np.asarray(idx) < cutoff)))
        t, gamma = ties_merge(list(delta_vals), masks, dtype)
    elif mode == "ta":
        t, gamma = ta_merge(list(delta_vals), dtype), None
    else:
        t, gamma = ram_merge(list(delta_vals), eps, dtype), None
    u = merged_update(t, lam)
    return dict(out=apply_update(base_vals, u, dtype), tau=u.astype(np.float32), gamma=gamma)
