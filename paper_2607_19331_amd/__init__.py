"""MI355X (gfx950) merge/update hot path of ISO and the App. F merges.

Thin Python binding over libiso.so (include/iso.h): functions carry the C names and only
turn torch tensors into pointers and tables.  Every step of the path runs in the HIP
library; there is no CPU or PyTorch fallback, and a missing library raises.
"""
import ctypes
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

from . import _lib
from ._lib import (BF16, F32, MERGE_RAM, MERGE_TA, MERGE_TIES, OP_BLOCKDIAG, OP_MERGE, OP_SIGN, OP_TOPK,
                   OP_UPDATE_APPLY, OP_UPDATE_FUSED, OP_UPDATE_FUSED_SELECT, OP_UPDATE_ORTHO, OP_UPDATE_SPECTRAL,
                   UPDATE_APPLY, UPDATE_FUSED, UPDATE_ORTHO, UPDATE_SPECTRAL, IsoSelectDesc)

DESC_BYTES = ctypes.sizeof(IsoSelectDesc)


class IsoError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {_lib.load().iso_status_string(status).decode()} (status {status})")


@dataclass
class Entry:
    """One row of the tensor table: device tensors of one weight matrix."""
    rows: int
    cols: int
    base: Optional[object] = None
    deltas: List[object] = field(default_factory=list)
    out: Optional[object] = None
    k: int = 0
    group: int = 0          # select_group: 0 alone, > 0 joint TopKMask with the same id


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _table(entries: Sequence[Entry]):
    arr = (_lib.IsoTensor * max(1, len(entries)))()
    for j, e in enumerate(entries):
        if len(e.deltas) > _lib.MAX_K:
            raise ValueError(f"at most {_lib.MAX_K} deltas per tensor")
        arr[j].base = _ptr(e.base)
        for i, d in enumerate(e.deltas):
            arr[j].deltas[i] = _ptr(d)
        arr[j].out = _ptr(e.out)
        arr[j].rows = e.rows
        arr[j].cols = e.cols
        arr[j].k = e.k
        arr[j].select_group = e.group
    return arr


def _ptr_array(xs):
    if xs is None:
        return None
    arr = (ctypes.c_void_p * max(1, len(xs)))()
    for i, x in enumerate(xs):
        arr[i] = _ptr(x)
    return arr


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def _check(rc, where):
    if rc != 0:
        raise IsoError(rc, where)


def _ws(ws):
    return (_ptr(ws), ws.numel() * ws.element_size()) if ws is not None else (None, 0)


def iso_workspace_size(op, entries, K, dtype):
    return _lib.load().iso_workspace_size(op, _table(entries), len(entries), K, dtype)


def iso_workspace_size_tsv(entries, K, dtype, rank):
    return _lib.load().iso_workspace_size_tsv(_table(entries), len(entries), K, dtype, rank)


def workspace(op, entries, K, dtype, device="cuda", rank=None):
    """Allocate a workspace tensor of the size the library asks for (caller-owned)."""
    import torch
    n = iso_workspace_size_tsv(entries, K, dtype, rank) if op == OP_BLOCKDIAG else iso_workspace_size(op, entries, K, dtype)
    ws = torch.empty(max(n, 256) + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + max(n, 256)]


def iso_topk_mask(entries, K, dtype, desc, mask_bits=None, ws=None, stream=None):
    wp, wb = _ws(ws)
    rc = _lib.load().iso_topk_mask(_table(entries), len(entries), K, dtype, _ptr(desc), _ptr_array(mask_bits), wp, wb,
                                   _stream(stream))
    _check(rc, "iso_topk_mask")


def iso_sign_elect(entries, K, dtype, desc, sign_out, ws=None, stream=None):
    wp, wb = _ws(ws)
    rc = _lib.load().iso_sign_elect(_table(entries), len(entries), K, dtype, _ptr(desc), _ptr_array(sign_out), wp, wb,
                                    _stream(stream))
    _check(rc, "iso_sign_elect")


def iso_merge(entries, K, dtype, mode, desc, lam, eps, tau_out, ws=None, stream=None):
    wp, wb = _ws(ws)
    rc = _lib.load().iso_merge(_table(entries), len(entries), K, dtype, mode, _ptr(desc), float(lam), float(eps),
                               _ptr_array(tau_out), wp, wb, _stream(stream))
    _check(rc, "iso_merge")


def iso_update(entries, K, dtype, mode, merge=MERGE_TIES, lam=1.0, eps=1e-5, desc=None, tau_in=None, sign_out=None,
               rho_keep=0.9, ridge=1e-12, c_min=0.0, c_max=1.5, coef_out=None, ws=None, stream=None):
    a = _lib.IsoUpdateArgs()
    a.mode, a.merge, a.lambda_, a.eps_act = mode, merge, float(lam), float(eps)
    keep = [_ptr_array(tau_in), _ptr_array(sign_out)]
    a.desc = _ptr(desc)
    a.tau_in = ctypes.cast(keep[0], ctypes.c_void_p).value if keep[0] is not None else None
    a.sign_out = ctypes.cast(keep[1], ctypes.c_void_p).value if keep[1] is not None else None
    a.rho_keep, a.ridge, a.c_min, a.c_max = float(rho_keep), float(ridge), float(c_min), float(c_max)
    a.coef_out = _ptr(coef_out)
    wp, wb = _ws(ws)
    rc = _lib.load().iso_update(_table(entries), len(entries), K, dtype, ctypes.byref(a), wp, wb, _stream(stream))
    _check(rc, "iso_update")


def iso_update_noalloc(entries, K, dtype, mode, merge=MERGE_TIES, lam=1.0, eps=1e-5, desc=None, tau_in=None,
                       sign_out=None, rho_keep=0.9, ridge=1e-12, c_min=0.0, c_max=1.5, coef_out=None, stream=None):
    """iso_update on the library's fixed per-device scratch block (no workspace argument); returns the
    block's device address, to be passed as ``ws`` to iso_read_device_status / iso_read_fallback_count."""
    a = _lib.IsoUpdateArgs()
    a.mode, a.merge, a.lambda_, a.eps_act = mode, merge, float(lam), float(eps)
    keep = [_ptr_array(tau_in), _ptr_array(sign_out)]
    a.desc = _ptr(desc)
    a.tau_in = ctypes.cast(keep[0], ctypes.c_void_p).value if keep[0] is not None else None
    a.sign_out = ctypes.cast(keep[1], ctypes.c_void_p).value if keep[1] is not None else None
    a.rho_keep, a.ridge, a.c_min, a.c_max = float(rho_keep), float(ridge), float(c_min), float(c_max)
    a.coef_out = _ptr(coef_out)
    scratch = ctypes.c_void_p()
    rc = _lib.load().iso_update_noalloc(_table(entries), len(entries), K, dtype, ctypes.byref(a),
                                        ctypes.byref(scratch), _stream(stream))
    _check(rc, "iso_update_noalloc")
    return scratch.value


def iso_blockdiag_project(entries, K, dtype, rank, alpha, delta_hat=None, ws=None, stream=None):
    wp, wb = _ws(ws)
    rc = _lib.load().iso_blockdiag_project(_table(entries), len(entries), K, dtype, int(rank), float(alpha),
                                           _ptr_array(delta_hat), wp, wb, _stream(stream))
    _check(rc, "iso_blockdiag_project")


def iso_blockdiag_project_factors(entries, K, dtype, rank, alpha, factors, delta_hat=None, ws=None, stream=None):
    """factors[j * K + i] = (U, s, V) device float64 tensors of delta i of tensor j (U rows x rank and
    V cols x rank row-major, s of length rank)."""
    arr = (_lib.IsoFactors * max(1, len(factors)))()
    for q, (u, s_, v) in enumerate(factors):
        arr[q].u, arr[q].s, arr[q].v = _ptr(u), _ptr(s_), _ptr(v)
    wp, wb = _ws(ws)
    rc = _lib.load().iso_blockdiag_project_factors(_table(entries), len(entries), K, dtype, int(rank), float(alpha),
                                                   arr, _ptr_array(delta_hat), wp, wb, _stream(stream))
    _check(rc, "iso_blockdiag_project_factors")


@dataclass
class Frame:
    """One matrix trained by ISO-AdamW or ISO-Muon: float64 device tensors (column-major frames and
    optimizer state; ISO-Muon uses m_u and m_v as its momentum buffers and takes v_u = v_v = None)."""
    u: object
    v: object
    sigma: object
    m_u: object
    v_u: object
    m_v: object
    v_v: object
    grad: object
    w_out: object
    rows: int
    cols: int
    rank: int


def _frames(frames):
    arr = (_lib.IsoFrame * max(1, len(frames)))()
    for q, f in enumerate(frames):
        for name in ("u", "v", "sigma", "m_u", "v_u", "m_v", "v_v", "grad", "w_out"):
            setattr(arr[q], name, _ptr(getattr(f, name)))
        arr[q].rows, arr[q].cols, arr[q].rank = f.rows, f.cols, f.rank
    return arr


def optimizer_workspace(frames, device="cuda"):
    import torch
    n = _lib.load().iso_workspace_size_optimizer(_frames(frames), len(frames))
    if n == 0:
        raise ValueError("bad frame table")
    return torch.empty((n + 7) // 8, dtype=torch.float64, device=device)


def iso_optimizer_step(frames, dtype, lr, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, step=1, ws=None,
                       stream=None):
    o = _lib.IsoAdamW(lr, beta1, beta2, eps, weight_decay, step)
    wp, wb = _ws(ws)
    rc = _lib.load().iso_optimizer_step(_frames(frames), len(frames), dtype, ctypes.byref(o), wp, wb, _stream(stream))
    _check(rc, "iso_optimizer_step")


def iso_optimizer_step_muon(frames, dtype, lr, momentum=0.95, weight_decay=0.0, nesterov=True, ws=None, stream=None):
    o = _lib.IsoMuon(lr, momentum, weight_decay, 1 if nesterov else 0)
    wp, wb = _ws(ws)
    rc = _lib.load().iso_optimizer_step_muon(_frames(frames), len(frames), dtype, ctypes.byref(o), wp, wb,
                                             _stream(stream))
    _check(rc, "iso_optimizer_step_muon")


def iso_spectral_diagnostics(entries, dtype, out, ws=None, stream=None):
    """out: device float64 tensor of 3 * len(entries): {delta_Sigma, rho_Sigma, kappa_spec} per tensor."""
    wp, wb = _ws(ws)
    rc = _lib.load().iso_spectral_diagnostics(_table(entries), len(entries), dtype, _ptr(out), wp, wb, _stream(stream))
    _check(rc, "iso_spectral_diagnostics")


def iso_spectral_error(entries, dtype, out, self_recon=False, ws=None, stream=None):
    """out: device float64 tensor of len(entries): eps_sigma per tensor, W_0 = base and W_rec = deltas[0]
    (a whole matrix), or with self_recon the reconstruction from the library's own SVD of the base."""
    wp, wb = _ws(ws)
    rc = _lib.load().iso_spectral_error(_table(entries), len(entries), dtype, 1 if self_recon else 0, _ptr(out), wp,
                                        wb, _stream(stream))
    _check(rc, "iso_spectral_error")


def iso_spectrum_interpolate(entries, dtype, alpha, ws=None, stream=None):
    wp, wb = _ws(ws)
    rc = _lib.load().iso_spectrum_interpolate(_table(entries), len(entries), dtype, float(alpha), wp, wb,
                                              _stream(stream))
    _check(rc, "iso_spectrum_interpolate")


def iso_transport_ratios(entries, dtype, rank_frac, out, ws=None, stream=None):
    """rank_frac: one fraction or a sequence of them.  out: device float64 tensor of
    5 * len(rank_frac) * len(entries): {u_mix, u_L, u_R, u_iso, gap} per tensor and fraction (tensor
    major), for the transition base -> base + deltas[0] truncated to rank max(1, floor(f q))."""
    fr = [float(rank_frac)] if isinstance(rank_frac, (int, float)) else [float(f) for f in rank_frac]
    arr = (ctypes.c_double * max(1, len(fr)))(*fr)
    wp, wb = _ws(ws)
    rc = _lib.load().iso_transport_ratios(_table(entries), len(entries), dtype, arr, len(fr), _ptr(out), wp, wb,
                                          _stream(stream))
    _check(rc, "iso_transport_ratios")


def iso_k_from_density(n, num, den):
    return _lib.load().iso_k_from_density(n, num, den)


def iso_read_device_status(ws, stream=None):
    return _lib.load().iso_read_device_status(_ptr(ws), _stream(stream))


def iso_read_fallback_count(ws, stream=None):
    """Tensors that the last single-read fused TIES call on ws sent to the two-pass path."""
    import ctypes
    c = ctypes.c_int32(0)
    st = _lib.load().iso_read_fallback_count(_ptr(ws), _stream(stream), ctypes.byref(c))
    if st != 0:
        raise IsoError(st, "iso_read_fallback_count")
    return c.value


def iso_profile_begin():
    st = _lib.load().iso_profile_begin()
    if st != 0:
        raise IsoError(st, "iso_profile_begin")


def iso_profile_flops():
    """Binary64 flops the optimizer steps' timed Newton-Schulz iterations performed since
    iso_profile_begin."""
    import ctypes
    f = ctypes.c_double(0.0)
    st = _lib.load().iso_profile_flops(ctypes.byref(f))
    if st != 0:
        raise IsoError(st, "iso_profile_flops")
    return f.value


def iso_profile_end():
    """(total milliseconds, launches) of the main kernels timed since iso_profile_begin."""
    import ctypes
    ms, n = ctypes.c_double(0.0), ctypes.c_int32(0)
    st = _lib.load().iso_profile_end(ctypes.byref(ms), ctypes.byref(n))
    if st != 0:
        raise IsoError(st, "iso_profile_end")
    return ms.value, n.value


def iso_status_string(s):
    return _lib.load().iso_status_string(s).decode()


def desc_tensor(n, device="cuda"):
    """Device buffer for n select descriptors (32 bytes each)."""
    import torch
    return torch.empty(n * DESC_BYTES // 8, dtype=torch.int64, device=device)


def decode_desc(t):
    """Host view of descriptors: list of (t_key, key_max, n_above, tie_quota, tie_cutoff)."""
    import numpy as np
    a = t.detach().cpu().numpy().view(np.uint8).reshape(-1, DESC_BYTES)
    out = []
    for row in a:
        u32 = row[:8].view(np.uint32)
        i64 = row[8:].view(np.int64)
        out.append((int(u32[0]), int(u32[1]), int(i64[0]), int(i64[1]), int(i64[2])))
    return out
