"""Helpers for the GPU parity tests: upload storage arrays, run the C ABI, fetch results."""
import os
import sys

import numpy as np

import paper_2607_19331_amd as iso


_PROGRESS = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "gpurun_out",
                         "gpu_case_progress.log")


def say(msg):
    """Progress line: printed (seen with -s) and appended to gpurun_out/gpu_case_progress.log, so that
    a long case shows progress even when pytest captures its output."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()
    try:
        os.makedirs(os.path.dirname(_PROGRESS), exist_ok=True)
        with open(_PROGRESS, "a") as f:
            f.write(f"[gpu-case] {msg}\n")
    except OSError:
        pass


def dt_code(dtype):
    return iso.BF16 if dtype == "bf16" else iso.F32


def to_dev(a, dev="cuda"):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(dev)
    return torch.from_numpy(a.view(np.int32)).to(dev)


def empty_like_storage(n, dtype, dev="cuda"):
    import torch
    return torch.empty(max(n, 1), dtype=torch.int16 if dtype == "bf16" else torch.int32, device=dev)


def from_dev(t, n, dtype):
    a = t.detach().cpu().numpy()[:n]
    return a.view(np.uint16) if dtype == "bf16" else a.view(np.float32)


class Unit:
    """One tensor with its base and K deltas as host storage arrays and device copies."""

    def __init__(self, rows, cols, base, deltas, dtype, k=0, dev="cuda"):
        self.rows, self.cols, self.dtype, self.k = rows, cols, dtype, k
        self.n = rows * cols
        self.base, self.deltas = base, deltas
        self.dbase = to_dev(base, dev) if self.n else empty_like_storage(0, dtype, dev)
        self.ddeltas = [to_dev(d, dev) if self.n else empty_like_storage(0, dtype, dev) for d in deltas]
        self.dout = empty_like_storage(self.n, dtype, dev)

    def entry(self):
        return iso.Entry(self.rows, self.cols, base=self.dbase, deltas=self.ddeltas, out=self.dout, k=self.k)


def run_topk(units, K, dtype, with_bits=False, dev="cuda"):
    import torch
    es = [u.entry() for u in units]
    ws = iso.workspace(iso.OP_TOPK, es, K, dt_code(dtype), dev)
    desc = iso.desc_tensor(len(es) * K, dev)
    bits = None
    if with_bits:
        bits = [torch.empty(max(1, (u.n + 31) // 32), dtype=torch.int32, device=dev) for u in units for _ in range(K)]
    iso.iso_topk_mask(es, K, dt_code(dtype), desc, mask_bits=bits, ws=ws)
    st = iso.iso_read_device_status(ws)
    d = iso.decode_desc(desc)
    b = None
    if with_bits:
        b = [x.cpu().numpy().view(np.uint32) for x in bits]
    return d, b, st, desc


def bits_to_mask(words, n):
    w = np.asarray(words, dtype=np.uint32)
    m = ((w[:, None] >> np.arange(32, dtype=np.uint32)) & 1).astype(bool).ravel()
    return m[:n]


def run_fused(units, K, dtype, merge, desc=None, lam=1.0, eps=1e-5, want_sign=False, dev="cuda"):
    import torch
    es = [u.entry() for u in units]
    op = iso.OP_UPDATE_FUSED_SELECT if (merge == iso.MERGE_TIES and desc is None) else iso.OP_UPDATE_FUSED
    ws = iso.workspace(op, es, K, dt_code(dtype), dev)
    signs = [torch.empty(max(u.n, 16), dtype=torch.int8, device=dev) for u in units] if want_sign else None
    iso.iso_update(es, K, dt_code(dtype), iso.UPDATE_FUSED, merge=merge, lam=lam, eps=eps, desc=desc,
                   sign_out=signs, ws=ws)
    st = iso.iso_read_device_status(ws)
    outs = [from_dev(u.dout, u.n, dtype) for u in units]
    sg = [s.cpu().numpy()[:u.n] for s, u in zip(signs, units)] if want_sign else None
    return outs, sg, st


def run_merge(units, K, dtype, mode, desc, lam=1.0, eps=1e-5, dev="cuda"):
    import torch
    es = [u.entry() for u in units]
    ws = iso.workspace(iso.OP_MERGE, es, K, dt_code(dtype), dev)
    taus = [torch.empty(max(u.n, 4), dtype=torch.float32, device=dev) for u in units]
    iso.iso_merge(es, K, dt_code(dtype), mode, desc, lam, eps, taus, ws=ws)
    st = iso.iso_read_device_status(ws)
    return [t.cpu().numpy()[:u.n] for t, u in zip(taus, units)], st


def run_sign(units, K, dtype, desc, dev="cuda"):
    import torch
    es = [u.entry() for u in units]
    ws = iso.workspace(iso.OP_SIGN, es, K, dt_code(dtype), dev)
    signs = [torch.empty(max(u.n, 16), dtype=torch.int8, device=dev) for u in units]
    iso.iso_sign_elect(es, K, dt_code(dtype), desc, signs, ws=ws)
    st = iso.iso_read_device_status(ws)
    return [s.cpu().numpy()[:u.n] for s, u in zip(signs, units)], st


def run_apply(units, dtype, taus_host, lam=1.0, dev="cuda"):
    import torch
    es = [u.entry() for u in units]
    ws = iso.workspace(iso.OP_UPDATE_APPLY, es, 1, dt_code(dtype), dev)
    taus = [torch.from_numpy(np.ascontiguousarray(t, dtype=np.float32)).to(dev) if u.n else
            torch.empty(4, dtype=torch.float32, device=dev) for t, u in zip(taus_host, units)]
    iso.iso_update(es, 1, dt_code(dtype), iso.UPDATE_APPLY, lam=lam, tau_in=taus, ws=ws)
    st = iso.iso_read_device_status(ws)
    return [from_dev(u.dout, u.n, dtype) for u in units], st
