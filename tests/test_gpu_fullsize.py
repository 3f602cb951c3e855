"""Parity at the full workload sizes, in the launch configuration bench.py times.

Each workload's whole stack is generated on the device by the seeded generator and merged by
one iso_update call (FUSED, TIES, lambda 1, the selection inside the call: the single-read path
for bf16, the two-pass path for fp32), as bench.py times it; iso_topk_mask is also run over the
whole stack.  Every tensor's descriptors (the 545M-entry embeddings included) must satisfy what
holds at any size: n_above + tie_quota = k, a cutoff inside the tensor, the threshold key at most
the largest key.  Sampled tensors are then checked against the oracle: their base and K deltas
are regenerated on the host, the oracle's TopKMask descriptors are computed over the whole delta,
the GPU descriptors must equal them, and the merged weights must equal the
oracle's bit for bit -- on every coordinate for the Tiny and single-layer workloads, and for the
1.5B and 7B stacks on a million random coordinates per tensor, a window around every delta's tie
cutoff and the ragged tail.  The sampled tensors are one of each shape class (GQA k, attention
square, both MLP orientations) and, for the 1.5B and 7B stacks, the 10^8-entry embedding and
unembedding matrices; bf16 descriptors come from the oracle's linear-time counting form (pinned
against brute force and partial selection), fp32 ones from partial selection.
"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

from oracle import ties

import paper_2607_19331_amd as iso
import synth
from tests.gpu_helpers import say

pytestmark = pytest.mark.gpu

# workload, sampled tensor indices, "all" (every coordinate) or "sample"
CASES = [
    ("tiny", [0], "all"),
    ("layer", [1, 4, 6], "all"),
    ("1.5b", [1, 3, 4, 6, 196], "sample"),
    ("7b", [1, 3, 4, 6, 196, 197], "sample"),
]


def _stack(wl):
    import torch
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    st = torch.int16 if wl.dtype == "bf16" else torch.int32
    entries = []
    for t, spec in enumerate(wl.tensors):
        n = spec.numel
        base = torch.empty(n, dtype=st, device=dev)
        synth.fill_device(base.data_ptr(), n, wl, t, 0, stream)
        ds = []
        for i in range(wl.K):
            d = torch.empty(n, dtype=st, device=dev)
            synth.fill_device(d.data_ptr(), n, wl, t, 1 + i, stream)
            ds.append(d)
        out = torch.empty(n, dtype=st, device=dev)
        k = iso.iso_k_from_density(n, wl.density.numerator, wl.density.denominator)
        entries.append(iso.Entry(spec.rows, spec.cols, base=base, deltas=ds, out=out, k=k))
    return entries


def _sample_idx(rng, n, descs):
    parts = [rng.integers(0, n, size=min(n, 1 << 20)), np.arange(max(0, n - 4096), n)]
    for d in descs:
        c = int(d[3])
        parts.append(np.arange(max(0, c - 2048), min(n, c + 2048)))
    return np.unique(np.concatenate(parts))


def _descriptor(d, k, sdt):
    if sdt == "bf16":
        return ties.topk_descriptor_counting(d, k)
    return ties.topk_descriptor(d, k, sdt)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,picks,how", CASES, ids=[c[0] for c in CASES])
def test_full_workload(name, picks, how):
    import torch
    wl = synth.workload(name)
    dt = iso.BF16 if wl.dtype == "bf16" else iso.F32
    say(f"full-size {name}: {len(wl.tensors)} tensors, {wl.numel} params, K={wl.K}")
    entries = _stack(wl)
    ws = iso.workspace(iso.OP_UPDATE_FUSED_SELECT, entries, wl.K, dt)
    iso.iso_update(entries, wl.K, dt, iso.UPDATE_FUSED, merge=iso.MERGE_TIES, lam=1.0, desc=None, ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    if dt == iso.BF16:
        say(f"full-size {name}: tensors sent to the two-pass path: {iso.iso_read_fallback_count(ws)}")
    wsel = iso.workspace(iso.OP_TOPK, entries, wl.K, dt)
    desc = iso.desc_tensor(len(entries) * wl.K)
    iso.iso_topk_mask(entries, wl.K, dt, desc, ws=wsel)
    assert iso.iso_read_device_status(wsel) == 0
    gdesc = iso.decode_desc(desc)
    del wsel
    torch.cuda.synchronize()
    for t, e in enumerate(entries):
        for i in range(wl.K):
            t_key, key_max, n_above, quota, cutoff = gdesc[t * wl.K + i]
            assert n_above + quota == e.k and 0 <= quota, (t, i)
            assert 0 <= cutoff <= wl.tensors[t].numel, (t, i)
            assert e.k == 0 or t_key <= key_max, (t, i)
    rng = np.random.default_rng(7)
    sdt = "bf16" if wl.dtype == "bf16" else "f32"
    for t in picks:
        spec, e = wl.tensors[t], entries[t]
        say(f"full-size {name}: {spec.name} {spec.rows}x{spec.cols}")
        base = synth.fill_host(wl, t, 0, threads=8)
        ds = [synth.fill_host(wl, t, 1 + i, threads=8) for i in range(wl.K)]
        with ThreadPoolExecutor(wl.K) as ex:
            want = list(ex.map(lambda d: _descriptor(d, e.k, sdt), ds))
        for i in range(wl.K):
            g = gdesc[t * wl.K + i]
            assert (g[0], g[2], g[3], g[4]) == want[i], (spec.name, i)
        out = e.out.cpu().numpy()
        out = out.view(np.uint16) if sdt == "bf16" else out.view(np.float32)
        if how == "all":
            masks = [ties.mask_from_descriptor(d, w, sdt) for d, w in zip(ds, want)]
            ref = ties.merge_unit(base, ds, sdt, "ties", masks=masks)["out"]
            assert np.array_equal(out, ref), spec.name
        else:
            idx = _sample_idx(rng, spec.numel, want)
            r = ties.merge_at(base[idx], np.stack([d[idx] for d in ds]), "ties", descs=want, idx=idx, dtype=sdt)
            bad = np.flatnonzero(out[idx] != r["out"])
            assert bad.size == 0, (spec.name, idx[bad[:8]])
        del base, ds, out
    del entries
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
def test_whole_model_group_7b():
    """TopKMask of the whole-model task vector (App. F, TIES "Trim" with tau_i spanning the model):
    all 198 tensors of the 7B stack in one select_group, 7.6e9 entries per delta, k the sum of the
    per-tensor counts at density 0.1.  The joint threshold is checked against a whole-model key
    histogram counted independently on the device (PyTorch bincount of the 15-bit magnitude keys):
    a member's n_above is its own count of keys above the joint threshold key T,
    the tie quota goes to the tied entries in table order, and each member's cutoff keeps exactly
    its quota of them (a member left with none of the threshold entries describes the same mask
    by its own smallest key above T, kept whole).  The merged weights of the same selection inside iso_update are then
    compared with the oracle's merge at a million sampled coordinates of four tensors, given
    those descriptors."""
    import time

    import torch
    wl = synth.workload("7b")
    K = wl.K
    entries = _stack(wl)
    for e in entries:
        e.group = 1
    kg = sum(e.k for e in entries)
    say(f"whole-model group: {len(entries)} tensors, {wl.numel} entries per delta, k = {kg}")
    ws = iso.workspace(iso.OP_TOPK, entries, K, iso.BF16)
    desc = iso.desc_tensor(len(entries) * K)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    iso.iso_topk_mask(entries, K, iso.BF16, desc, ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    say(f"whole-model group: iso_topk_mask {1e3 * (time.perf_counter() - t0):.1f} ms")
    del ws
    g = iso.decode_desc(desc)
    for i in range(K):
        hist = torch.zeros(1 << 15, dtype=torch.int64, device="cuda")
        for e in entries:
            for piece in e.deltas[i].split(1 << 28):
                hist += torch.bincount((piece & 0x7FFF).to(torch.int32), minlength=1 << 15)
        at_or_above = hist.flip(0).cumsum(0).flip(0)
        T = int(torch.nonzero(at_or_above >= kg).max())
        quota = kg - (int(at_or_above[T]) - int(hist[T]))
        say(f"whole-model group: delta {i}: T = {T:#06x}, quota {quota} of {int(hist[T])} tied")
        left = quota
        for j, e in enumerate(entries):
            if j % 50 == 0:
                say(f"whole-model group: delta {i}: member {j}")
            t_key, key_max, n_above, q, cutoff = g[j * K + i]
            k16 = e.deltas[i] & 0x7FFF
            tied = torch.nonzero(k16 == T).flatten()
            take = min(left, int(tied.numel()))
            left -= take
            if t_key == T:
                # the member keeps its entries above T and the first `take` of its T entries
                assert n_above == int((k16 > T).sum()), (j, i)
                assert q == take and int((tied < cutoff).sum()) == take, (j, i)
            else:
                # no T entry is left for this member: its own TopKMask of that count then has the
                # smallest key above T that it holds as threshold, all of whose entries it keeps --
                # the same mask
                assert t_key > T and take == 0, (j, i, t_key)
                assert int(((k16 > T) & (k16 < t_key)).sum()) == 0, (j, i)
                assert n_above == int((k16 > t_key).sum()), (j, i)
                assert q == int((k16 == t_key).sum()) and cutoff == e.rows * e.cols, (j, i)
            del k16, tied
        assert left == 0
    say("whole-model group: merge with the selection inside the call")
    ws = iso.workspace(iso.OP_UPDATE_FUSED_SELECT, entries, K, iso.BF16)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    iso.iso_update(entries, K, iso.BF16, iso.UPDATE_FUSED, merge=iso.MERGE_TIES, lam=1.0, desc=None, ws=ws)
    assert iso.iso_read_device_status(ws) == 0
    say(f"whole-model group: iso_update {1e3 * (time.perf_counter() - t0):.1f} ms")
    del ws
    rng = np.random.default_rng(11)
    for t in (1, 4, 6, 196):
        spec, e = wl.tensors[t], entries[t]
        say(f"whole-model group: oracle merge at sampled coordinates of {spec.name}")
        want = [tuple(g[t * K + i][j] for j in (0, 2, 3, 4)) for i in range(K)]
        idx = np.unique(np.concatenate([rng.integers(0, spec.numel, size=1 << 20),
                                        np.arange(max(0, spec.numel - 4096), spec.numel)]))
        base = synth.fill_host(wl, t, 0, threads=8)[idx]
        ds = np.stack([synth.fill_host(wl, t, 1 + i, threads=8)[idx] for i in range(K)])
        r = ties.merge_at(base, ds, "ties", descs=want, idx=idx, dtype="bf16")
        out = e.out.cpu().numpy().view(np.uint16)[idx]
        bad = np.flatnonzero(out != r["out"])
        assert bad.size == 0, (spec.name, idx[bad[:8]])
    del entries
    torch.cuda.empty_cache()
