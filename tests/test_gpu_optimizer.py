"""GPU ISO-AdamW and ISO-Muon steps (iso_optimizer_step, iso_optimizer_step_muon) against the float64 oracle.

Frames, moments and Sigma_0 are binary64 on both sides; the GPU's products sum in another
order and its polar factor comes from Newton-Schulz instead of an SVD, so frames and moments
agree to 1e-10 (entries of order 0.1), fp32 weights within 1e-6 * max(|ref|, 2^-10 max|ref|)
and bf16 weights within one ulp, over three consecutive steps.
"""
import numpy as np
import pytest

from oracle import numerics as nm
from oracle import optimizer as op

import paper_2607_19331_amd as iso
from tests.gpu_helpers import say, to_dev, from_dev

pytestmark = pytest.mark.gpu


def _colmajor(a):
    import torch
    return torch.tensor(np.asfortranarray(a).ravel(order="F"), dtype=torch.float64, device="cuda")


def _back(t, rows, cols):
    return t.cpu().numpy().reshape(cols, rows).T


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_three_steps_match_the_oracle(dtype):
    import torch
    rng = np.random.default_rng(11 if dtype == "f32" else 12)
    shapes = [(96, 64, 64), (80, 120, 80), (256, 200, 150)]
    frames, ref = [], []
    for m, n, q in shapes:
        u, _ = np.linalg.qr(rng.standard_normal((m, q)))
        v, _ = np.linalg.qr(rng.standard_normal((n, q)))
        s = np.sort(rng.uniform(0.5, 2.0, q))[::-1].copy()
        g_store = nm.from_f64(rng.standard_normal(m * n) * 0.1, dtype)
        g = nm.to_f64(g_store, dtype).reshape(m, n)
        z = [np.zeros((m, q)), np.zeros((m, q)), np.zeros((n, q)), np.zeros((n, q))]
        dev = dict(u=_colmajor(u), v=_colmajor(v), sigma=torch.tensor(s, device="cuda"),
                   m_u=_colmajor(z[0]), v_u=_colmajor(z[1]), m_v=_colmajor(z[2]), v_v=_colmajor(z[3]),
                   grad=to_dev(g_store),
                   w_out=torch.empty(m * n, dtype=torch.int16 if dtype == "bf16" else torch.int32, device="cuda"))
        frames.append(iso.Frame(rows=m, cols=n, rank=q, **dev))
        ref.append(dict(u=u, v=v, s=s, g=g, st=tuple(z)))
    ws = iso.optimizer_workspace(frames)
    dt = iso.BF16 if dtype == "bf16" else iso.F32
    hp = dict(lr=0.02, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)
    for t in (1, 2, 3):
        say(f"iso-adamw {dtype} step {t}: {shapes}")
        iso.iso_optimizer_step(frames, dt, step=t, ws=ws, **hp)
        assert iso.iso_read_device_status(ws) == 0
        for F, R in zip(frames, ref):
            R["u"], R["v"], w_ref, R["st"] = op.iso_adamw_step(R["u"], R["v"], R["s"], R["g"], R["st"], t, hp["lr"],
                                                               hp["beta1"], hp["beta2"], hp["eps"], hp["weight_decay"])
            m, n, q = F.rows, F.cols, F.rank
            assert np.abs(_back(F.u, m, q) - R["u"]).max() <= 1e-10
            assert np.abs(_back(F.v, n, q) - R["v"]).max() <= 1e-10
            for name, a, rows in (("m_u", R["st"][0], m), ("v_u", R["st"][1], m), ("m_v", R["st"][2], n),
                                  ("v_v", R["st"][3], n)):
                got = _back(getattr(F, name), rows, q)
                assert np.abs(got - a).max() <= 1e-10 * max(1.0, np.abs(a).max()), name
            w = from_dev(F.w_out, m * n, dtype)
            if dtype == "f32":
                ref_w = w_ref.ravel()
                scale = np.maximum(np.abs(ref_w), 2.0 ** -10 * np.abs(ref_w).max())
                assert np.max(np.abs(w.astype(np.float64) - ref_w) / scale) <= 1e-6
            else:
                want = nm.f64_to_bf16(w_ref.ravel()).astype(np.int32)
                assert np.max(np.abs(w.astype(np.int32) - want)) <= 1


@pytest.mark.parametrize("dtype,nesterov", [("f32", True), ("bf16", False)])
def test_muon_three_steps_match_the_oracle(dtype, nesterov):
    """ISO-Muon (iso_optimizer_step_muon): frames, momentum buffers and weights over three steps, to the
    bars of the ISO-AdamW test; the direction's polar factor is Newton-Schulz on the GPU, an SVD in the
    oracle."""
    import torch
    rng = np.random.default_rng(31 if nesterov else 32)
    shapes = [(96, 64, 64), (80, 120, 80), (256, 200, 150)]
    frames, ref = [], []
    for m, n, q in shapes:
        u, _ = np.linalg.qr(rng.standard_normal((m, q)))
        v, _ = np.linalg.qr(rng.standard_normal((n, q)))
        s = np.sort(rng.uniform(0.5, 2.0, q))[::-1].copy()
        g_store = nm.from_f64(rng.standard_normal(m * n) * 0.1, dtype)
        g = nm.to_f64(g_store, dtype).reshape(m, n)
        z = (np.zeros((m, q)), np.zeros((n, q)))
        dev = dict(u=_colmajor(u), v=_colmajor(v), sigma=torch.tensor(s, device="cuda"),
                   m_u=_colmajor(z[0]), v_u=None, m_v=_colmajor(z[1]), v_v=None, grad=to_dev(g_store),
                   w_out=torch.empty(m * n, dtype=torch.int16 if dtype == "bf16" else torch.int32, device="cuda"))
        frames.append(iso.Frame(rows=m, cols=n, rank=q, **dev))
        ref.append(dict(u=u, v=v, s=s, g=g, st=z))
    ws = iso.optimizer_workspace(frames)
    dt = iso.BF16 if dtype == "bf16" else iso.F32
    hp = dict(lr=0.02, momentum=0.9, weight_decay=0.01)
    for t in (1, 2, 3):
        say(f"iso-muon {dtype} nesterov={nesterov} step {t}: {shapes}")
        iso.iso_optimizer_step_muon(frames, dt, nesterov=nesterov, ws=ws, **hp)
        assert iso.iso_read_device_status(ws) == 0
        for F, R in zip(frames, ref):
            R["u"], R["v"], w_ref, R["st"] = op.iso_muon_step(R["u"], R["v"], R["s"], R["g"], R["st"], hp["lr"],
                                                              hp["momentum"], hp["weight_decay"], nesterov)
            m, n, q = F.rows, F.cols, F.rank
            assert np.abs(_back(F.u, m, q) - R["u"]).max() <= 1e-10
            assert np.abs(_back(F.v, n, q) - R["v"]).max() <= 1e-10
            for name, a, rows in (("m_u", R["st"][0], m), ("m_v", R["st"][1], n)):
                got = _back(getattr(F, name), rows, q)
                assert np.abs(got - a).max() <= 1e-10 * max(1.0, np.abs(a).max()), name
            w = from_dev(F.w_out, m * n, dtype)
            if dtype == "f32":
                ref_w = w_ref.ravel()
                scale = np.maximum(np.abs(ref_w), 2.0 ** -10 * np.abs(ref_w).max())
                assert np.max(np.abs(w.astype(np.float64) - ref_w) / scale) <= 1e-6
            else:
                want = nm.f64_to_bf16(w_ref.ravel()).astype(np.int32)
                assert np.max(np.abs(w.astype(np.int32) - want)) <= 1


def test_muon_zero_and_ill_conditioned_directions():
    """Three frames in one ISO-Muon call: a zero gradient (both directions zero: o = 0, the frames
    only decay and are retracted back), a gradient whose U-side direction has condition number
    ~1e8 (singular values 1 .. 1e-8 before the storage rounding; the scaled iteration needs ~35
    of its 48 steps), and a Gaussian one.  Status OK and the oracle's frames and weights to the bars
    above; lr 1e-3 keeps the ill-conditioned polar factor's rounding-level differences (~eps cond)
    far below the frame bar."""
    import torch
    rng = np.random.default_rng(33)
    dtype = "f32"
    specs = [("zero", 64, 48, 48), ("illcond", 96, 64, 64), ("gauss", 80, 72, 72)]
    frames, ref = [], []
    for kind, m, n, q in specs:
        u, _ = np.linalg.qr(rng.standard_normal((m, q)))
        v, _ = np.linalg.qr(rng.standard_normal((n, q)))
        s = np.sort(rng.uniform(0.5, 2.0, q))[::-1].copy()
        if kind == "zero":
            g = np.zeros((m, n))
        elif kind == "illcond":
            # G_W V Sigma_0 = U D Q^T with D from 1 down to 1e-8 (n = q: V is square orthogonal)
            qq, _ = np.linalg.qr(rng.standard_normal((q, q)))
            a = (u * np.logspace(0, -8, q)) @ qq.T
            g = (a / s) @ v.T
        else:
            g = rng.standard_normal((m, n)) * 0.1
        g_store = nm.from_f64(g.ravel(), dtype)
        g = nm.to_f64(g_store, dtype).reshape(m, n)
        z = (np.zeros((m, q)), np.zeros((n, q)))
        dev = dict(u=_colmajor(u), v=_colmajor(v), sigma=torch.tensor(s, device="cuda"),
                   m_u=_colmajor(z[0]), v_u=None, m_v=_colmajor(z[1]), v_v=None, grad=to_dev(g_store),
                   w_out=torch.empty(m * n, dtype=torch.int32, device="cuda"))
        frames.append(iso.Frame(rows=m, cols=n, rank=q, **dev))
        ref.append(dict(u=u, v=v, s=s, g=g, st=z))
    gu = ref[1]["g"] @ ref[1]["v"] * ref[1]["s"]
    sv = np.linalg.svd(gu, compute_uv=False)
    say(f"iso-muon zero / ill-conditioned (cond {sv[0] / sv[-1]:.2e}) / gaussian directions")
    ws = iso.optimizer_workspace(frames)
    hp = dict(lr=1e-3, momentum=0.9, weight_decay=0.01)
    for t in (1, 2):
        iso.iso_profile_begin()
        iso.iso_optimizer_step_muon(frames, iso.F32, nesterov=True, ws=ws, **hp)
        flops = iso.iso_profile_flops()
        ms, regions = iso.iso_profile_end()
        assert iso.iso_read_device_status(ws) == 0
        # two timed polar iterations (directions, retraction), every job at least one step of
        # 4 m q^2 flops in each
        unit = sum(4.0 * r * q * q for _, m, n, q in specs for r in (m, n))
        assert regions == 2 and ms > 0.0 and flops >= 2 * unit
        for (kind, *_), F, R in zip(specs, frames, ref):
            R["u"], R["v"], w_ref, R["st"] = op.iso_muon_step(R["u"], R["v"], R["s"], R["g"], R["st"], hp["lr"],
                                                              hp["momentum"], hp["weight_decay"], True)
            m, n, q = F.rows, F.cols, F.rank
            assert np.abs(_back(F.u, m, q) - R["u"]).max() <= 1e-10, (kind, t)
            assert np.abs(_back(F.v, n, q) - R["v"]).max() <= 1e-10, (kind, t)
            if kind == "zero":
                assert not _back(F.m_u, m, q).any() and not _back(F.m_v, n, q).any()
            w = from_dev(F.w_out, m * n, dtype)
            ref_w = w_ref.ravel()
            scale = np.maximum(np.abs(ref_w), 2.0 ** -10 * np.abs(ref_w).max())
            assert np.max(np.abs(w.astype(np.float64) - ref_w) / scale) <= 1e-6, (kind, t)
