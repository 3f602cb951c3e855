"""Joint TopKMask selection (select_group) on the GPU against the oracle.

Tensors sharing a select_group id are selected together per delta, as the concatenation of
their deltas in table order (App. F's TopKMask of a whole-model delta).  The descriptors stay per
tensor: each must describe exactly that tensor's part of the oracle's joint mask, and the merged
weights of iso_update (TIES, selection inside the call) must equal the oracle's bit for bit.
Magnitudes are drawn from a small set so that the threshold code is shared across tensors.
"""
import numpy as np
import pytest

from oracle import numerics as nm
from oracle import ties

import paper_2607_19331_amd as iso
from tests.gpu_helpers import Unit, from_dev, say

pytestmark = pytest.mark.gpu


def tied_unit(rng, rows, cols, K, k):
    n = rows * cols
    base = nm.from_f64(rng.standard_normal(n) * 0.02, "bf16")
    mags = np.array([0.0, 1e-4, 2e-4, 5e-4, 1e-3])
    ds = [nm.from_f64(rng.choice(mags, size=n, p=[0.4, 0.3, 0.15, 0.1, 0.05]) * rng.choice([-1.0, 1.0], size=n),
                      "bf16") for _ in range(K)]
    return Unit(rows, cols, base, ds, "bf16", k)


# (rows, cols, group, k): group 1 puts its whole count on its first member, group 2 spreads it;
# the empty tensor and the tensor alone sit between members
SHAPES = [(64, 48, 1, 2000), (40, 40, 2, 300), (0, 0, 1, 0), (100, 37, 1, 0), (30, 70, 0, 500),
          (33, 33, 2, 250), (17, 9, 1, 0)]


def _entries(units):
    es = []
    for u, (_, _, g, _) in zip(units, SHAPES):
        e = u.entry()
        e.group = g
        es.append(e)
    return es


def _oracle_masks(units, K):
    """Per tensor, per delta: the oracle's mask of that tensor under the joint selection."""
    masks = [[None] * K for _ in units]
    for g in sorted({s[2] for s in SHAPES}):
        idx = [j for j, s in enumerate(SHAPES) if s[2] == g]
        for i in range(K):
            if g == 0:
                for j in idx:
                    masks[j][i] = ties.topk_mask(units[j].deltas[i], units[j].k, "bf16")
            else:
                kg = sum(units[j].k for j in idx)
                parts = ties.topk_mask_joint([units[j].deltas[i] for j in idx], kg, "bf16")
                for j, m in zip(idx, parts):
                    masks[j][i] = m
    return masks


def test_joint_selection_descriptors_and_merge():
    import torch
    rng = np.random.default_rng(17)
    K = 2
    units = [tied_unit(rng, r, c, K, k) if r * c else Unit(0, 0, np.zeros(0, np.uint16),
                                                           [np.zeros(0, np.uint16)] * K, "bf16", 0)
             for r, c, _, k in SHAPES]
    es = _entries(units)
    want = _oracle_masks(units, K)
    say("groups: iso_topk_mask over 7 tensors in 2 groups")
    ws = iso.workspace(iso.OP_TOPK, es, K, iso.BF16)
    desc = iso.desc_tensor(len(es) * K)
    iso.iso_topk_mask(es, K, iso.BF16, desc, ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    d = iso.decode_desc(desc)
    for j, u in enumerate(units):
        for i in range(K):
            t_key, key_max, n_above, quota, cutoff = d[j * K + i]
            if u.n == 0:
                continue
            got = ties.mask_from_descriptor(u.deltas[i], (t_key, n_above, quota, cutoff), "bf16")
            assert np.array_equal(got, want[j][i]), (j, i)
            assert n_above + quota == int(want[j][i].sum()), (j, i)
    say("groups: iso_update FUSED TIES, selection inside the call")
    wsu = iso.workspace(iso.OP_UPDATE_FUSED_SELECT, es, K, iso.BF16)
    iso.iso_update(es, K, iso.BF16, iso.UPDATE_FUSED, merge=iso.MERGE_TIES, lam=1.0, desc=None, ws=wsu)
    assert iso.iso_read_device_status(wsu) == 0
    torch.cuda.synchronize()
    for j, u in enumerate(units):
        if u.n == 0:
            continue
        ref = ties.merge_unit(u.base, u.deltas, "bf16", "ties", masks=want[j])["out"]
        assert np.array_equal(from_dev(u.dout, u.n, "bf16"), ref), j


def test_whole_layer_as_one_group():
    """The single-layer workload (seven bf16 matrices, K = 2) selected as one whole-model delta with
    density 0.1 of the layer: per delta the members' shares add up to the group's count, and the
    descriptors of q_proj and down_proj (first and last member) give exactly the oracle's joint
    masks; the merged weights of down_proj match the oracle bit for bit."""
    import torch
    import synth
    wl = synth.workload("layer")
    K = wl.K
    n_all = sum(s.numel for s in wl.tensors)
    k_all = iso.iso_k_from_density(n_all, wl.density.numerator, wl.density.denominator)
    units = []
    for t, spec in enumerate(wl.tensors):
        base = synth.fill_host(wl, t, 0)
        ds = [synth.fill_host(wl, t, 1 + i) for i in range(K)]
        units.append(Unit(spec.rows, spec.cols, base, ds, "bf16", k_all if t == 0 else 0))
    es = []
    for u in units:
        e = u.entry()
        e.group = 7
        es.append(e)
    say(f"groups: whole layer as one group, k = {k_all} of {n_all}")
    ws = iso.workspace(iso.OP_TOPK, es, K, iso.BF16)
    desc = iso.desc_tensor(len(es) * K)
    iso.iso_topk_mask(es, K, iso.BF16, desc, ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    d = iso.decode_desc(desc)
    for i in range(K):
        assert sum(d[j * K + i][2] + d[j * K + i][3] for j in range(len(es))) == k_all
        want = ties.topk_mask_joint([u.deltas[i] for u in units], k_all, "bf16")
        for j in (0, len(units) - 1):
            t_key, _, n_above, quota, cutoff = d[j * K + i]
            got = ties.mask_from_descriptor(units[j].deltas[i], (t_key, n_above, quota, cutoff), "bf16")
            assert np.array_equal(got, want[j]), (j, i)
        if i == 0:
            masks_last = [None] * K
        masks_last[i] = want[-1]
        del want
    wsu = iso.workspace(iso.OP_UPDATE_FUSED_SELECT, es, K, iso.BF16)
    iso.iso_update(es, K, iso.BF16, iso.UPDATE_FUSED, merge=iso.MERGE_TIES, lam=1.0, desc=None, ws=wsu)
    assert iso.iso_read_device_status(wsu) == 0
    torch.cuda.synchronize()
    u = units[-1]
    ref = ties.merge_unit(u.base, u.deltas, "bf16", "ties", masks=masks_last)["out"]
    assert np.array_equal(from_dev(u.dout, u.n, "bf16"), ref)
