"""Launch-geometry independence of the streaming path (TopKMask, sign election, disjoint mean and
update): the same tensors merged (a) in one call, (b) one call per tensor, (c) in one call in
reverse order, and (d) by the two-pass route (iso_topk_mask descriptors, then FUSED with them)
give bit-identical merged weights and elected signs.  Grouping changes the grids, the
tile-to-tensor map, which tensors share the sampled bracket launches and the workspace layout;
(d) replaces the single-read kernels by the exact select and merge kernels altogether.  Each
result is also checked against the oracle once, so that four equal wrong answers cannot pass.
"""
import numpy as np
import pytest

from oracle import numerics as nm
from oracle import ties

import paper_2607_19331_amd as iso
from tests.gpu_helpers import Unit, from_dev, say

pytestmark = pytest.mark.gpu

SHAPES = [(300, 257), (64, 4096), (1, 10007), (1024, 1100), (5, 5), (2048, 1536)]


def _units(rng, K):
    us = []
    for rows, cols in SHAPES:
        n = rows * cols
        base = nm.from_f64(rng.standard_normal(n) * 0.02, "bf16")
        ds = []
        for _ in range(K):
            # coarse values give many equal magnitudes, so the flat-index tie rule decides
            v = np.round(rng.standard_normal(n) * 8.0) / 8192.0
            v[rng.random(n) < 0.5] = 0.0
            ds.append(nm.from_f64(v, "bf16"))
        us.append(Unit(rows, cols, base, ds, "bf16", nm.k_from_density(n, 0.15)))
    return us


def _fused(units, K, desc=None):
    import torch
    es = [u.entry() for u in units]
    op = iso.OP_UPDATE_FUSED_SELECT if desc is None else iso.OP_UPDATE_FUSED
    ws = iso.workspace(op, es, K, iso.BF16)
    signs = [torch.empty(max(u.n, 16), dtype=torch.int8, device="cuda") for u in units]
    iso.iso_update(es, K, iso.BF16, iso.UPDATE_FUSED, merge=iso.MERGE_TIES, lam=1.0, desc=desc, sign_out=signs,
                   ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    return [from_dev(u.dout, u.n, "bf16").copy() for u in units], [s.cpu().numpy()[:u.n].copy()
                                                                   for s, u in zip(signs, units)]


@pytest.mark.parametrize("K", [2, 4])
def test_grouping_and_route_do_not_change_results(K):
    rng = np.random.default_rng(2600 + K)
    units = _units(rng, K)
    say(f"geometry K={K}: one call")
    out_a, sg_a = _fused(units, K)
    say(f"geometry K={K}: one call per tensor")
    out_b, sg_b = [], []
    for u in units:
        o, g = _fused([u], K)
        out_b += o
        sg_b += g
    say(f"geometry K={K}: reverse order")
    o, g = _fused(units[::-1], K)
    out_c, sg_c = o[::-1], g[::-1]
    say(f"geometry K={K}: two-pass route")
    es = [u.entry() for u in units]
    wsel = iso.workspace(iso.OP_TOPK, es, K, iso.BF16)
    desc = iso.desc_tensor(len(es) * K)
    iso.iso_topk_mask(es, K, iso.BF16, desc, ws=wsel)
    assert iso.iso_read_device_status(wsel) == 0
    out_d, sg_d = _fused(units, K, desc=desc)
    for j, u in enumerate(units):
        for name, o, g in (("per tensor", out_b, sg_b), ("reversed", out_c, sg_c), ("two-pass", out_d, sg_d)):
            assert np.array_equal(out_a[j], o[j]), (name, SHAPES[j])
            assert np.array_equal(sg_a[j], g[j]), (name, SHAPES[j])
        r = ties.merge_unit(u.base, u.deltas, "bf16", "ties", k=u.k, lam=1.0)
        assert np.array_equal(out_a[j], r["out"]), SHAPES[j]
        assert np.array_equal(sg_a[j], r["gamma"]), SHAPES[j]
