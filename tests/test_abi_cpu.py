"""C ABI checks that need no GPU: the library loads, exports what include/iso.h declares,
and rejects bad arguments on the host before anything is queued."""
import ctypes
import os
import re

import pytest

import paper_2607_19331_amd as iso
from paper_2607_19331_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "iso.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:iso_status|size_t|int64_t|const char\*)\s+(iso_\w+)\s*\(", src, re.M)))


def test_library_exports_every_declared_symbol():
    L = _lib.load()
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(_lib.SYMBOLS)


FAKE = 0x100000     # never dereferenced: every call below fails validation first


def entry(rows=16, cols=16, k=10, K=2, misalign=False, out=True):
    d = [FAKE + 0x1000 * (i + 1) + (8 if (misalign and i == 1) else 0) for i in range(K)]
    return iso.Entry(rows, cols, base=FAKE, deltas=d, out=FAKE + 0x100 if out else None, k=k)


def call_topk(es, K, ws_bytes=1 << 30, ws=FAKE * 16, desc=FAKE * 8):
    L = _lib.load()
    return L.iso_topk_mask(iso._table(es), len(es), K, iso.BF16, desc, None, ws, ws_bytes, None)


def test_host_validation_errors():
    L = _lib.load()
    assert call_topk([entry()], 0) == _lib.ERR_INVALID_ARG
    assert call_topk([entry(K=8)], 9) == _lib.ERR_INVALID_ARG
    assert call_topk([entry(k=257)], 2) == _lib.ERR_INVALID_ARG
    assert call_topk([entry(k=-1)], 2) == _lib.ERR_INVALID_ARG
    assert call_topk([entry(misalign=True)], 2) == _lib.ERR_ALIGNMENT
    assert call_topk([entry()], 2, ws_bytes=100) == _lib.ERR_WORKSPACE
    assert call_topk([entry()], 2, ws=FAKE * 16 + 64) == _lib.ERR_ALIGNMENT
    assert call_topk([entry()], 2, desc=None) == _lib.ERR_INVALID_ARG
    assert call_topk([entry(rows=1 << 17, cols=1 << 16)], 2) == _lib.ERR_UNSUPPORTED
    assert call_topk([], 2) == _lib.OK
    bad = iso.Entry(-1, 3, base=FAKE, deltas=[FAKE, FAKE], out=FAKE)
    assert call_topk([bad], 2) == _lib.ERR_INVALID_ARG
    # iso_merge: TIES needs descriptors, eps must be >= 0, lambda finite
    es = [entry()]
    tau = (ctypes.c_void_p * 1)(FAKE)
    assert L.iso_merge(iso._table(es), 1, 2, iso.BF16, 1, None, 1.0, 0.0, tau, FAKE * 16, 1 << 30, None) == 1
    assert L.iso_merge(iso._table(es), 1, 2, iso.BF16, 0, None, float("nan"), 0.0, tau, FAKE * 16, 1 << 30, None) == 1
    assert L.iso_merge(iso._table(es), 1, 2, iso.BF16, 2, None, 1.0, -1.0, tau, FAKE * 16, 1 << 30, None) == 1
    assert L.iso_merge(iso._table(es), 1, 2, iso.BF16, 7, None, 1.0, 0.0, tau, FAKE * 16, 1 << 30, None) == 1
    # iso_update: missing output, bad mode, spectral size limit
    a = _lib.IsoUpdateArgs()
    a.mode, a.merge, a.lambda_, a.eps_act = 1, 0, 1.0, 0.0
    noout = [entry(out=False)]
    assert L.iso_update(iso._table(noout), 1, 2, iso.BF16, ctypes.byref(a), FAKE * 16, 1 << 30, None) == 1
    a.mode = 9
    assert L.iso_update(iso._table(es), 1, 2, iso.BF16, ctypes.byref(a), FAKE * 16, 1 << 30, None) == 1
    a.mode, a.rho_keep, a.ridge, a.c_min, a.c_max = 2, 0.9, 1e-12, 0.0, 1.5
    big = [entry(rows=16385, cols=16385, k=0)]           # the limit is on min(rows, cols)
    assert L.iso_update(iso._table(big), 1, 2, iso.BF16, ctypes.byref(a), FAKE * 16, 1 << 30, None) == \
        _lib.ERR_UNSUPPORTED
    tall = [entry(rows=152064, cols=64, k=0)]             # a long side alone is accepted
    assert L.iso_update(iso._table(tall), 1, 2, iso.BF16, ctypes.byref(a), FAKE * 16, 100, None) == \
        _lib.ERR_WORKSPACE
    a.rho_keep = 0.0
    assert L.iso_update(iso._table(es), 1, 2, iso.BF16, ctypes.byref(a), FAKE * 16, 1 << 30, None) == 1
    assert L.iso_update(iso._table(es), 1, 2, iso.BF16, None, FAKE * 16, 1 << 30, None) == 1
    assert L.iso_read_device_status(None, None) == 1


def test_group_validation():
    """Joint selection: negative ids and a group count above the group's size are invalid, an
    fp32 call with a group is unsupported; a member's own k may exceed its size."""
    L = _lib.load()
    a, b = entry(rows=16, cols=16, k=300), entry(rows=16, cols=16, k=0)
    a.group = b.group = 3
    assert call_topk([a, b], 2, ws_bytes=100) == _lib.ERR_WORKSPACE    # 300 <= 512: passes validation
    a.k = 600
    assert call_topk([a, b], 2) == _lib.ERR_INVALID_ARG
    a.k, a.group = 10, -1
    assert call_topk([a, b], 2) == _lib.ERR_INVALID_ARG
    a.group = 3
    es = [a, b]
    assert L.iso_topk_mask(iso._table(es), 2, 2, iso.F32, FAKE * 8, None, FAKE * 16, 1 << 30, None) == \
        _lib.ERR_UNSUPPORTED
    n_alone = iso.iso_workspace_size(iso.OP_TOPK, [entry(), entry()], 2, iso.BF16)
    assert iso.iso_workspace_size(iso.OP_TOPK, es, 2, iso.BF16) >= n_alone + 2 * 32768 * 8


def test_group_beyond_32_bits():
    """A joint selection over more than 2^32 entries (a whole-model delta at 7B scale): three
    members of 2^31 entries, group count 2^32 + 5.  The planner accepts it (64-bit group bins)
    and sizes its workspace; a count above the group's size is still rejected, and so is an
    overflowing sum of member counts."""
    es = [entry(rows=1 << 16, cols=1 << 15, k=0) for _ in range(3)]
    for e in es:
        e.group = 1
    es[0].k = (1 << 32) + 5
    assert call_topk(es, 2, ws_bytes=100) == _lib.ERR_WORKSPACE
    need = iso.iso_workspace_size(iso.OP_TOPK, es, 2, iso.BF16)
    assert need >= 2 * 32768 * 8
    es[1].k = 3 * (1 << 31) - es[0].k + 1
    assert call_topk(es, 2, ws_bytes=100) == _lib.ERR_INVALID_ARG
    es[1].k = (1 << 63) - 1                                     # the member sum saturates
    assert call_topk(es, 2, ws_bytes=100) == _lib.ERR_INVALID_ARG


def test_workspace_sizes():
    es = [entry(rows=2048, cols=5632, k=1153434, K=2), entry(rows=7, cols=9, k=3, K=2)]
    n_sel = iso.iso_workspace_size(iso.OP_TOPK, es, 2, iso.BF16)
    n_fused = iso.iso_workspace_size(iso.OP_UPDATE_FUSED, es, 2, iso.BF16)
    n_fs = iso.iso_workspace_size(iso.OP_UPDATE_FUSED_SELECT, es, 2, iso.BF16)
    assert n_sel >= 4 * 32768 * 4 and n_fused < n_sel <= n_fs
    assert n_sel % 256 == 0 and n_fused % 256 == 0
    assert iso.iso_workspace_size(99, es, 2, iso.BF16) == 0
    assert iso.iso_workspace_size(iso.OP_TOPK, es, 0, iso.BF16) == 0


@pytest.mark.parametrize("n,num,den,k", [(65536, 1, 5, 13107), (11534336, 1, 10, 1153434), (5, 1, 10, 1),
                                         (15, 1, 10, 2), (10, 0, 1, 0), (7, 1, 1, 7),
                                         (545009664, 1, 10, 54500966)])
def test_k_from_density_matches_oracle(n, num, den, k):
    from fractions import Fraction
    from oracle.numerics import k_from_density
    assert iso.iso_k_from_density(n, num, den) == k == k_from_density(n, Fraction(num, den))


def test_status_strings():
    for s in range(8):
        assert iso.iso_status_string(s)
    assert "unknown" in iso.iso_status_string(42)


def test_optimizer_validation():
    L = _lib.load()
    f = (_lib.IsoFrame * 1)()
    for i, name in enumerate(("u", "v", "sigma", "m_u", "v_u", "m_v", "v_v", "grad", "w_out")):
        setattr(f[0], name, FAKE + 0x1000 * i)
    f[0].rows, f[0].cols, f[0].rank = 64, 48, 48
    o = _lib.IsoAdamW(1e-3, 0.9, 0.999, 1e-8, 0.0, 1)
    assert L.iso_workspace_size_optimizer(f, 1) > 0
    f[0].rank = 49
    assert L.iso_optimizer_step(f, 1, iso.F32, ctypes.byref(o), FAKE * 16, 1 << 30, None) == _lib.ERR_INVALID_ARG
    assert L.iso_workspace_size_optimizer(f, 1) == 0
    f[0].rank = 48
    o.beta2 = 1.0
    assert L.iso_optimizer_step(f, 1, iso.F32, ctypes.byref(o), FAKE * 16, 1 << 30, None) == _lib.ERR_INVALID_ARG
    o.beta2, o.step = 0.999, 0
    assert L.iso_optimizer_step(f, 1, iso.F32, ctypes.byref(o), FAKE * 16, 1 << 30, None) == _lib.ERR_INVALID_ARG
    o.step = 1
    f[0].u = FAKE + 4
    assert L.iso_optimizer_step(f, 1, iso.F32, ctypes.byref(o), FAKE * 16, 1 << 30, None) == _lib.ERR_ALIGNMENT
    f[0].u = None
    assert L.iso_optimizer_step(f, 1, iso.F32, ctypes.byref(o), FAKE * 16, 1 << 30, None) == _lib.ERR_INVALID_ARG


def test_transport_ratio_validation():
    L = _lib.load()
    es = [entry(K=1, out=False)]
    t = iso._table(es)

    def fr(*xs):
        return (ctypes.c_double * max(1, len(xs)))(*xs)

    def call(fracs, n, out=FAKE * 8, table=t, n_t=1, ws_bytes=1 << 30):
        return L.iso_transport_ratios(table, n_t, iso.F32, fracs, n, out, FAKE * 16, ws_bytes, None)

    for frac in (0.0, -0.5, 1.5, float("nan")):
        assert call(fr(0.9, frac), 2) == _lib.ERR_INVALID_ARG, frac
    assert call(fr(0.9), 0) == _lib.ERR_INVALID_ARG
    assert call(fr(*([0.5] * 17)), 17) == _lib.ERR_INVALID_ARG
    assert call(None, 1) == _lib.ERR_INVALID_ARG
    assert call(fr(0.9), 1, out=None) == _lib.ERR_INVALID_ARG
    assert call(fr(0.9), 1, out=FAKE * 8 + 4) == _lib.ERR_ALIGNMENT
    big = [iso.Entry(16385, 16385, base=FAKE, deltas=[FAKE + 0x1000], out=None, k=0)]
    assert call(fr(0.9), 1, table=iso._table(big)) == _lib.ERR_UNSUPPORTED
    tall = [iso.Entry(16385, 8, base=FAKE, deltas=[FAKE + 0x1000], out=None, k=0)]
    assert call(fr(0.9), 1, table=iso._table(tall), ws_bytes=100) == _lib.ERR_WORKSPACE
    assert call(fr(0.2, 0.9), 2, ws_bytes=100) == _lib.ERR_WORKSPACE
    assert call(fr(*([0.5] * 16)), 16, n_t=0) == _lib.OK


def test_muon_validation():
    L = _lib.load()
    f = (_lib.IsoFrame * 1)()
    for i, name in enumerate(("u", "v", "sigma", "m_u", "v_u", "m_v", "v_v", "grad", "w_out")):
        setattr(f[0], name, FAKE + 0x1000 * i)
    f[0].rows, f[0].cols, f[0].rank = 64, 48, 48
    f[0].v_u = None                     # Muon keeps no second moments
    f[0].v_v = None
    o = _lib.IsoMuon(0.02, 0.95, 0.0, 1)
    assert L.iso_workspace_size_optimizer(f, 1) > 0
    assert L.iso_optimizer_step_muon(f, 1, iso.F32, ctypes.byref(o), FAKE * 16, 100, None) == _lib.ERR_WORKSPACE
    adam = _lib.IsoAdamW(1e-3, 0.9, 0.999, 1e-8, 0.0, 1)
    assert L.iso_optimizer_step(f, 1, iso.F32, ctypes.byref(adam), FAKE * 16, 1 << 30, None) == _lib.ERR_INVALID_ARG
    for bad in (1.0, -0.1, float("nan")):
        o.momentum = bad
        assert L.iso_optimizer_step_muon(f, 1, iso.F32, ctypes.byref(o), FAKE * 16, 1 << 30, None) == \
            _lib.ERR_INVALID_ARG, bad
    o.momentum, o.lr = 0.95, float("inf")
    assert L.iso_optimizer_step_muon(f, 1, iso.F32, ctypes.byref(o), FAKE * 16, 1 << 30, None) == _lib.ERR_INVALID_ARG
    o.lr = 0.02
    assert L.iso_optimizer_step_muon(f, 1, iso.F32, None, FAKE * 16, 1 << 30, None) == _lib.ERR_INVALID_ARG
    f[0].m_u = None
    assert L.iso_optimizer_step_muon(f, 1, iso.F32, ctypes.byref(o), FAKE * 16, 1 << 30, None) == _lib.ERR_INVALID_ARG
    f[0].m_u = FAKE + 0x3000 + 4
    assert L.iso_optimizer_step_muon(f, 1, iso.F32, ctypes.byref(o), FAKE * 16, 1 << 30, None) == _lib.ERR_ALIGNMENT


def test_spectral_error_validation():
    L = _lib.load()
    t = iso._table([entry(K=1, out=False)])

    def call(self_recon=0, out=FAKE * 8, table=t, n_t=1, ws_bytes=1 << 30):
        return L.iso_spectral_error(table, n_t, iso.F32, self_recon, out, FAKE * 16, ws_bytes, None)

    assert call(self_recon=2) == _lib.ERR_INVALID_ARG
    assert call(self_recon=-1) == _lib.ERR_INVALID_ARG
    assert call(out=None) == _lib.ERR_INVALID_ARG
    assert call(out=FAKE * 8 + 4) == _lib.ERR_ALIGNMENT
    assert call(ws_bytes=100) == _lib.ERR_WORKSPACE
    assert call(n_t=0) == _lib.OK
    nodelta = iso._table([iso.Entry(16, 16, base=FAKE, deltas=[None], out=None, k=0)])
    assert call(table=nodelta) == _lib.ERR_INVALID_ARG          # W_rec is required unless self_recon
    assert call(self_recon=1, table=nodelta, ws_bytes=100) == _lib.ERR_WORKSPACE
    big = iso._table([iso.Entry(16385, 16385, base=FAKE, deltas=[FAKE + 0x1000], out=None, k=0)])
    assert call(table=big) == _lib.ERR_UNSUPPORTED
    tall = iso._table([iso.Entry(8, 16385, base=FAKE, deltas=[FAKE + 0x1000], out=None, k=0)])
    assert call(table=tall, ws_bytes=100) == _lib.ERR_WORKSPACE


def test_noalloc_validation():
    """iso_update_noalloc checks its arguments as iso_update does and refuses, before anything is
    queued, a call whose workspace exceeds the fixed block."""
    L = _lib.load()
    a = _lib.IsoUpdateArgs()
    a.mode, a.merge, a.lambda_, a.eps_act = iso.UPDATE_FUSED, iso.MERGE_TIES, 1.0, 1e-5
    t = iso._table([entry(rows=16, cols=16, k=10, K=2)])
    assert L.iso_update_noalloc(t, 1, 2, iso.BF16, None, None, None) == _lib.ERR_INVALID_ARG
    assert L.iso_update_noalloc(t, 1, 9, iso.BF16, ctypes.byref(a), None, None) == _lib.ERR_INVALID_ARG
    assert L.iso_update_noalloc(iso._table([entry(misalign=True)]), 1, 2, iso.BF16, ctypes.byref(a), None,
                                None) == _lib.ERR_ALIGNMENT
    big = iso._table([entry(rows=4096, cols=4096, k=10, K=4)])
    assert L.iso_update_noalloc(big, 1, 4, iso.BF16, ctypes.byref(a), None, None) == _lib.ERR_UNSUPPORTED
    assert L.iso_update_noalloc(t, 0, 2, iso.BF16, ctypes.byref(a), None, None) == _lib.OK


def test_calibration_library_exports_its_declaration():
    src = open(os.path.join(ROOT, "include", "iso_calibrate.h")).read()
    names = re.findall(r"^\s*int\s+(iso_\w+)\s*\(", src, re.M)
    assert names == ["iso_calibrate_stream"]
    L = ctypes.CDLL(os.path.join(ROOT, "paper_2607_19331_amd", "libiso_calibrate.so"))
    f = L.iso_calibrate_stream
    f.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p]
    ptrs = (ctypes.c_void_p * 8)(*([FAKE] * 8))
    assert f(None, 5, FAKE, 16, 1, None) == 1                # bad arguments return before any launch
    assert f(ptrs, 0, FAKE, 16, 1, None) == 1
    assert f(ptrs, 9, FAKE, 16, 1, None) == 1
    assert f(ptrs, 5, None, 16, 1, None) == 1
    assert f(ptrs, 5, FAKE, 0, 1, None) == 1


def test_orthomerge_validation():
    """iso_update ORTHO refuses, before anything is queued, wide matrices (the Procrustes rotation
    of a wide W_0 is not unique), a non-finite lambda, joint-selection groups, k above the tensor
    size and a workspace below iso_workspace_size(ISO_OP_UPDATE_ORTHO)."""
    import math
    L = _lib.load()
    a = _lib.IsoUpdateArgs()
    a.mode, a.merge, a.lambda_, a.eps_act = 3, 1, 1.0, 0.0

    def call(es, ws_bytes=1 << 40):
        return L.iso_update(iso._table(es), len(es), 2, iso.BF16, ctypes.byref(a), FAKE * 16, ws_bytes, None)

    assert call([entry(rows=8, cols=16, k=10)]) == _lib.ERR_UNSUPPORTED
    assert call([entry(rows=16385, cols=16385, k=10)]) == _lib.ERR_UNSUPPORTED
    g = entry(rows=16, cols=8, k=10)
    g.group = 1
    assert call([g]) == _lib.ERR_UNSUPPORTED
    assert call([entry(rows=16, cols=8, k=129)]) == _lib.ERR_INVALID_ARG
    assert call([entry(rows=16, cols=8, k=10)], ws_bytes=100) == _lib.ERR_WORKSPACE
    a.lambda_ = math.inf
    assert call([entry(rows=16, cols=8, k=10)]) == _lib.ERR_INVALID_ARG
    a.lambda_ = 1.0
    assert call([]) == _lib.OK
    es = [entry(rows=300, cols=128, k=10)]
    assert L.iso_workspace_size(iso.OP_UPDATE_ORTHO, iso._table(es), 1, 2, iso.BF16) > 0


def test_profile_flops_counter_without_a_gpu():
    """iso_profile_flops: a NULL output is refused; after iso_profile_begin the counter reads 0 and
    iso_profile_end with nothing timed returns no regions (no HIP call is made)."""
    L = _lib.load()
    assert L.iso_profile_flops(None) == _lib.ERR_INVALID_ARG
    iso.iso_profile_begin()
    assert iso.iso_profile_flops() == 0.0
    assert iso.iso_profile_end() == (0.0, 0)
