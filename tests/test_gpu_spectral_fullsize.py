"""ISO-Merger (Algorithm 1, SPECTRAL mode of iso_update) at the 7B stack's full matrix shapes, in
bf16 with the stack's seeded deltas (the inputs bench.py's full-layer record uses).

* Layer 0's gate_proj (18944 x 3584) and down_proj (3584 x 18944), K = 4: the merged weights at
  32768 seeded coordinates and the last 1024 entries against the oracle's, stored by
  tests/golden/make_iso_merge_7b.py (which runs only the oracle), to one bf16 ulp as at small
  sizes; c* to 1e-8 relative (the two sides' SVDs are different algorithms, and at this size the
  singular vectors of the closest of the 3584 singular values, which the tangent displacements
  and hence c* depend on, are determined only to eps sigma_1 / gap: 2e-9 is measured on gate_proj,
  2e-10 on down_proj, against 1e-11 and below at the small sizes).
* embed_tokens (152064 x 3584), beyond what the oracle finishes inside a test, is checked by
  properties that hold at any size:
  - the coefficients are finite and inside [c_min, c_max];
  - W_* keeps the base spectrum: sigma(U_* Sigma_0 V_*^T) = sigma_0, so after the single rounding
    to bf16 (relative error at most u = 2^-8 per entry) Mirsky's inequality bounds the App. G
    spectral error: eps_sigma(W_0, W_*) <= |W_* - fl(W_*)|_F^2 / q <= u^2 |W_*|_F^2 / q;
  - duplicating an expert changes nothing: with tau_1 = tau_2 = tau the ridge system gives
    c_1 = c_2 = a / (2a + lambda), so c_1 + c_2 equals the single expert's a / (a + lambda) up to
    lambda / (2a), and the aggregate tangent -- hence W_* -- is the single expert's (one ulp).
    Only the sum is checked: the system is singular but for the ridge along (1, -1), so the split
    between the two copies carries the solve's rounding amplified by 2a / lambda.
"""
import os
import sys

import numpy as np
import pytest

from oracle import numerics as nm

import paper_2607_19331_amd as iso
import synth
from tests.gpu_helpers import say

sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden"))
import make_iso_merge_7b as golden  # noqa: E402

pytestmark = pytest.mark.gpu


def _inputs(wl, t, K, dup=False):
    import torch
    spec = wl.tensors[t]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    base = torch.empty(spec.numel, dtype=torch.int16, device=dev)
    synth.fill_device(base.data_ptr(), spec.numel, wl, t, 0, stream)
    ds = []
    for i in range(K):
        if dup and i > 0:
            ds.append(ds[0])
            continue
        d = torch.empty(spec.numel, dtype=torch.int16, device=dev)
        synth.fill_device(d.data_ptr(), spec.numel, wl, t, 1 + i, stream)
        ds.append(d)
    return spec, base, ds


def _merge(spec, base, ds, K):
    import torch
    out = torch.empty(spec.numel, dtype=torch.int16, device="cuda")
    es = [iso.Entry(spec.rows, spec.cols, base=base, deltas=ds[:K], out=out, k=0)]
    ws = iso.workspace(iso.OP_UPDATE_SPECTRAL, es, K, iso.BF16)
    coef = torch.zeros(K, dtype=torch.float64, device="cuda")
    iso.iso_update(es, K, iso.BF16, iso.UPDATE_SPECTRAL, coef_out=coef, ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    del ws
    torch.cuda.empty_cache()
    return out, coef.cpu().numpy()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["gate", "down"])
def test_full_shape_against_oracle(name):
    ref = np.load(golden.PATH)
    wl = synth.workload("7b")
    t = golden.TENSORS[name]
    spec, base, ds = _inputs(wl, t, wl.K)
    say(f"ISO-Merger full shape {spec.name} {spec.rows}x{spec.cols} K={wl.K}")
    out, coef = _merge(spec, base, ds, wl.K)
    rel = np.max(np.abs(coef / ref[f"{name}_c"] - 1.0))
    idx = golden.sample_idx(spec.numel)
    have = out.cpu().numpy().view(np.uint16)[idx].astype(np.int32)
    want = nm.f64_to_bf16(ref[f"{name}_w"]).astype(np.int32)
    hw = nm.to_f64(have.astype(np.uint16), "bf16")
    wrel = np.abs(hw - ref[f"{name}_w"]) / np.abs(ref[f"{name}_w"]).max()
    say(f"{spec.name}: c rel diff {rel:.3e}, max |W - W_ref| / max|W_ref| {wrel.max():.3e}, "
        f"ulps off {np.bincount(np.minimum(np.abs(have - want), 3))}")
    assert rel <= 1e-8, (coef, ref[f"{name}_c"])
    bad = np.flatnonzero(np.abs(have - want) > 1)
    assert bad.size == 0, (idx[bad[:8]], have[bad[:8]], want[bad[:8]])


@pytest.mark.timeout(900)
def test_embedding_shape_properties():
    import torch
    wl = synth.workload("7b")
    t = 196
    spec, base, ds = _inputs(wl, t, wl.K)
    assert spec.name == "embed_tokens" and (spec.rows, spec.cols) == (152064, 3584)
    say(f"ISO-Merger full shape {spec.name} {spec.rows}x{spec.cols} K={wl.K}")
    out, coef = _merge(spec, base, ds, wl.K)
    assert np.all(np.isfinite(coef)) and np.all((coef >= 0.0) & (coef <= 1.5)), coef
    q = min(spec.rows, spec.cols)
    w = out.cpu().numpy().view(np.uint16)
    fro2 = float(np.sum(nm.to_f64(w, "bf16") ** 2))
    say(f"{spec.name}: spectral error of W_* against W_0")
    e = [iso.Entry(spec.rows, spec.cols, base=base, deltas=[out], out=None, k=0)]
    ws = iso.workspace(iso.OP_UPDATE_SPECTRAL, e, 1, iso.BF16)
    err = torch.zeros(1, dtype=torch.float64, device="cuda")
    iso.iso_spectral_error(e, iso.BF16, err, ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    del ws
    eps = float(err.cpu()[0])
    say(f"{spec.name}: eps_sigma {eps:.3e}, bound {2.0 ** -16 * fro2 / q:.3e}")
    assert 0.0 <= eps <= 2.0 ** -16 * fro2 / q
    del ds, out, w
    torch.cuda.empty_cache()
    # tau_1 = tau_2 against the single expert
    spec, base, ds = _inputs(wl, t, 2, dup=True)
    say(f"{spec.name}: one expert, then the same expert twice")
    out1, c1 = _merge(spec, base, ds, 1)
    out2, c2 = _merge(spec, base, ds, 2)
    say(f"{spec.name}: c single {c1}, c twice {c2}")
    assert np.isclose(c2.sum(), c1[0], rtol=1e-8, atol=0), (c1, c2)
    a = out1.cpu().numpy().view(np.uint16).astype(np.int32)
    b = out2.cpu().numpy().view(np.uint16).astype(np.int32)
    say(f"{spec.name}: ulps between the two merges {np.bincount(np.minimum(np.abs(a - b), 3))}")
    assert np.max(np.abs(a - b)) <= 1
