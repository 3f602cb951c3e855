"""iso_update_noalloc (iso_update on the library's fixed per-device scratch block) against iso_update
with a caller workspace: the same kernels on the same inputs, so the outputs must agree bit for bit.
Two calls in a row on the shared block, the second with a smaller input (the block keeps the first
call's contents), then a call too large for the block, which is refused before anything runs."""
import numpy as np
import pytest

from oracle import numerics as nm

import paper_2607_19331_amd as iso
from tests.gpu_helpers import Unit, dt_code, from_dev, say

pytestmark = pytest.mark.gpu


def _units(rng, shapes, K, dtype, p_zero=0.6):
    us = []
    for r, c in shapes:
        n = r * c
        base = nm.from_f64(rng.standard_normal(n) * 0.02, dtype)
        ds = []
        for _ in range(K):
            v = rng.standard_normal(n) * 5e-5
            v[rng.random(n) < p_zero] = 0.0
            ds.append(nm.from_f64(v, dtype))
        us.append(Unit(r, c, base, ds, dtype, k=int(round(0.1 * n))))
    return us


def _both(units, K, dtype, **kw):
    import torch
    es = [u.entry() for u in units]
    scratch = iso.iso_update_noalloc(es, K, dt_code(dtype), iso.UPDATE_FUSED, **kw)
    assert scratch and scratch % 256 == 0
    assert iso.iso_read_device_status(scratch) == 0
    fb = iso.iso_read_fallback_count(scratch) if dtype == "bf16" else 0
    got = [from_dev(u.dout, u.n, dtype).copy() for u in units]
    for u in units:
        u.dout.fill_(0x5A5A)
    op = iso.OP_UPDATE_FUSED_SELECT if kw.get("desc") is None and kw.get("merge", iso.MERGE_TIES) == iso.MERGE_TIES \
        else iso.OP_UPDATE_FUSED
    ws = iso.workspace(op, es, K, dt_code(dtype))
    iso.iso_update(es, K, dt_code(dtype), iso.UPDATE_FUSED, ws=ws, **kw)
    assert iso.iso_read_device_status(ws) == 0
    want = [from_dev(u.dout, u.n, dtype) for u in units]
    torch.cuda.synchronize()
    return got, want, fb


def test_noalloc_matches_iso_update_twice_then_refuses_a_large_call():
    rng = np.random.default_rng(77)
    first = _units(rng, [(1024, 2048), (333, 777), (0, 0), (1500, 1000)], 4, "bf16")
    say("noalloc: fused TIES select, bf16 K=4, 3.9M entries")
    got, want, fb = _both(first, 4, "bf16", merge=iso.MERGE_TIES, lam=1.0)
    assert fb == 0
    for g, w in zip(got, want):
        assert np.array_equal(g, w)
    second = _units(rng, [(100, 300), (7, 5)], 2, "bf16")
    say("noalloc: second, smaller call, bf16 K=2, lambda 0.7")
    got, want, _ = _both(second, 2, "bf16", merge=iso.MERGE_TIES, lam=0.7)
    for g, w in zip(got, want):
        assert np.array_equal(g, w)
    third = _units(rng, [(256, 192)], 3, "f32")
    say("noalloc: fp32 two-pass select, K=3")
    got, want, _ = _both(third, 3, "f32", merge=iso.MERGE_TIES, lam=1.0)
    assert np.array_equal(got[0].view(np.uint32), want[0].view(np.uint32))
    n = 4096 * 4096                                  # real buffers: nothing may run on them anyway
    big = Unit(4096, 4096, np.zeros(n, np.uint16), [np.zeros(n, np.uint16)] * 4, "bf16", k=1000)
    es = [big.entry()]
    assert iso.iso_workspace_size(iso.OP_UPDATE_FUSED_SELECT, es, 4, iso.BF16) > (64 << 20)
    say("noalloc: a call beyond the block is refused")
    with pytest.raises(iso.IsoError) as e:
        iso.iso_update_noalloc(es, 4, iso.BF16, iso.UPDATE_FUSED, merge=iso.MERGE_TIES)
    assert e.value.status == 6                      # ISO_ERR_UNSUPPORTED
