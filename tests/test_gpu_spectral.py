"""GPU ISO-Merger (Algorithm 1, SPECTRAL mode of iso_update) against the float64 oracle.

The two sides use different SVD algorithms (one-sided Jacobi on the GPU, LAPACK gesdd in
the oracle), so the merged matrix agrees to rounding, not bit for bit: fp32 outputs within
1e-6 * max(|ref|, 2^-10 max|ref|), bf16 outputs within one unit in the last place.  The
coefficients c* agree to 1e-9 relative.
"""
import numpy as np
import pytest

from oracle import numerics as nm
from oracle import spectral as sp

import paper_2607_19331_amd as iso
import synth
from tests.gpu_helpers import Unit, dt_code, from_dev, say

pytestmark = pytest.mark.gpu


def run_spectral(units, K, dtype, rho_keep=0.9, ridge=1e-12, c_min=0.0, c_max=1.5):
    import torch
    es = [u.entry() for u in units]
    ws = iso.workspace(iso.OP_UPDATE_SPECTRAL, es, K, dt_code(dtype))
    coef = torch.zeros(len(units) * K, dtype=torch.float64, device="cuda")
    iso.iso_update(es, K, dt_code(dtype), iso.UPDATE_SPECTRAL, rho_keep=rho_keep, ridge=ridge, c_min=c_min,
                   c_max=c_max, coef_out=coef, ws=ws)
    st = iso.iso_read_device_status(ws)
    return [from_dev(u.dout, u.n, dtype) for u in units], coef.cpu().numpy().reshape(len(units), K), st


def _ref(u, K, dtype, **kw):
    w0 = nm.to_f64(u.base, dtype).reshape(u.rows, u.cols)
    ds = [nm.to_f64(d, dtype).reshape(u.rows, u.cols) for d in u.deltas]
    return sp.iso_merge(w0, ds, **kw)


def _close(got, dtype, ref_f64):
    ref = ref_f64.ravel()
    if dtype == "f32":
        g = got.astype(np.float64)
        scale = np.maximum(np.abs(ref), 2.0 ** -10 * np.abs(ref).max())
        return np.max(np.abs(g - ref) / scale) <= 1e-6
    want = nm.f64_to_bf16(ref).astype(np.int32)
    have = got.astype(np.int32)
    return np.max(np.abs(have - want)) <= 1           # same-sign neighbours: 1 ulp apart in the bit pattern


def _unit(rng, rows, cols, K, dtype, scale=1e-3, p_nz=0.3):
    n = rows * cols
    base = nm.from_f64(rng.standard_normal(n) * 0.02, dtype)
    ds = []
    for _ in range(K):
        v = rng.standard_normal(n) * scale
        v[rng.random(n) > p_nz] = 0.0
        ds.append(nm.from_f64(v, dtype))
    return Unit(rows, cols, base, ds, dtype)


def test_tiny_workload():
    wl = synth.tiny()
    spec = wl.tensors[0]
    say("spectral tiny 256x256 K=3 fp32")
    base = synth.fill_host(wl, 0, 0)
    ds = [synth.fill_host(wl, 0, 1 + i) for i in range(wl.K)]
    u = Unit(spec.rows, spec.cols, base, ds, "f32")
    outs, coef, st = run_spectral([u], wl.K, "f32")
    assert st == 0
    ref = _ref(u, wl.K, "f32")
    assert _close(outs[0], "f32", ref["w_star"])
    assert np.allclose(coef[0], ref["c"], rtol=1e-9, atol=1e-12)
    s = np.linalg.svd(outs[0].astype(np.float64).reshape(256, 256), compute_uv=False)
    assert np.allclose(s, ref["s0"], rtol=1e-5)


# the small shapes have one column block (q <= 16 on the LDS path, q <= 32 on the Gram path for the
# 1500-long columns): its pairs are swept by the block paired with the phantom block
@pytest.mark.parametrize("rows,cols,K,dtype", [(96, 64, 2, "f32"), (48, 80, 3, "f32"), (64, 64, 1, "bf16"),
                                               (130, 65, 4, "bf16"), (33, 17, 2, "f32"), (12, 8, 2, "f32"),
                                               (16, 16, 3, "bf16"), (5, 3, 2, "f32"), (9, 1, 2, "f32"),
                                               (1500, 24, 2, "f32"), (20, 1500, 2, "f32")])
def test_shapes(rows, cols, K, dtype):
    rng = np.random.default_rng(rows * 1000 + cols)
    u = _unit(rng, rows, cols, K, dtype)
    say(f"spectral {rows}x{cols} K={K} {dtype}")
    outs, coef, st = run_spectral([u], K, dtype)
    assert st == 0
    ref = _ref(u, K, dtype)
    assert _close(outs[0], dtype, ref["w_star"])
    assert np.allclose(coef[0], ref["c"], rtol=1e-9, atol=1e-12)


def test_zero_deltas_return_base_and_table_of_two():
    rng = np.random.default_rng(3)
    u0 = _unit(rng, 40, 40, 2, "f32", scale=0.0)
    u1 = _unit(rng, 72, 56, 2, "f32")
    say("spectral zero deltas + second tensor")
    outs, coef, st = run_spectral([u0, u1], 2, "f32")
    assert st == 0
    assert np.array_equal(outs[0], u0.base)
    assert np.all(coef[0] == 0)
    ref = _ref(u1, 2, "f32")
    assert _close(outs[1], "f32", ref["w_star"])


def test_keep_ratio_and_clip_range():
    rng = np.random.default_rng(4)
    u = _unit(rng, 64, 48, 3, "f32")
    say("spectral rho_keep 0.5, clip [0.2, 0.9]")
    outs, coef, st = run_spectral([u], 3, "f32", rho_keep=0.5, c_min=0.2, c_max=0.9)
    assert st == 0
    ref = _ref(u, 3, "f32", rho_keep=0.5, c_min=0.2, c_max=0.9)
    assert _close(outs[0], "f32", ref["w_star"])
    assert np.allclose(coef[0], ref["c"], rtol=1e-9)


# one call over several matrices: they run as one batch of Jacobi jobs of different shapes.  The
# first set's longest columns (700) take the Gram-based block Jacobi for the whole batch, the
# second set fits LDS; an empty matrix sits between the others
MIXED = {
    "gram_path": [(300, 200), (200, 300), (0, 0), (96, 700), (64, 64)],
    "lds_path": [(120, 80), (80, 120), (0, 0), (64, 64), (17, 33)],
}


@pytest.mark.parametrize("name", list(MIXED))
def test_batched_mixed_shapes(name):
    rng = np.random.default_rng(len(name))
    K = 3
    units = [_unit(rng, r, c, K, "f32") if r * c else Unit(0, 0, np.zeros(0, np.float32),
                                                          [np.zeros(0, np.float32)] * K, "f32")
             for r, c in MIXED[name]]
    say(f"spectral batch {name}: {MIXED[name]} K={K}")
    outs, coef, st = run_spectral(units, K, "f32")
    assert st == 0
    for u, o, c in zip(units, outs, coef):
        if u.n == 0:
            continue
        ref = _ref(u, K, "f32")
        assert _close(o, "f32", ref["w_star"]), (u.rows, u.cols)
        assert np.allclose(c, ref["c"], rtol=1e-9, atol=1e-12), (u.rows, u.cols)


@pytest.mark.parametrize("t_idx", [0, 4], ids=["q_proj_2048x2048", "gate_proj_2048x5632"])
def test_single_layer_shapes(t_idx):
    """Algorithm 1 at the single-layer workload's shapes (bf16, K = 2), from the seeded generator."""
    import time
    wl = synth.workload("layer")
    spec = wl.tensors[t_idx]
    base = synth.fill_host(wl, t_idx, 0)
    ds = [synth.fill_host(wl, t_idx, 1 + i) for i in range(wl.K)]
    u = Unit(spec.rows, spec.cols, base, ds, "bf16")
    say(f"spectral layer {spec.name} {spec.rows}x{spec.cols} K={wl.K}")
    t0 = time.perf_counter()
    outs, coef, st = run_spectral([u], wl.K, "bf16")
    say(f"spectral layer {spec.name}: {time.perf_counter() - t0:.2f} s on the GPU")
    assert st == 0
    ref = _ref(u, wl.K, "bf16")
    assert _close(outs[0], "bf16", ref["w_star"])
    assert np.allclose(coef[0], ref["c"], rtol=1e-9, atol=1e-12)


def test_warm_started_batch_lds_path():
    """Eight 256 x 256 matrices with K = 4 in one call: their Jacobi workgroups outnumber what the
    chip holds at once, so the experts' SVDs start from the base's right factor."""
    rng = np.random.default_rng(41)
    K = 4
    units = [_unit(rng, 256, 256, K, "f32") for _ in range(8)]
    say("spectral warm-started batch 8 x 256x256 K=4")
    outs, coef, st = run_spectral(units, K, "f32")
    assert st == 0
    for u, o, c in zip(units, outs, coef):
        ref = _ref(u, K, "f32")
        assert _close(o, "f32", ref["w_star"])
        assert np.allclose(c, ref["c"], rtol=1e-9, atol=1e-12)


def test_whole_layer_one_call():
    """The single-layer workload's seven matrices in one call (the warm-started Gram path, as
    bench.py times it); q_proj and gate_proj checked against the oracle."""
    import time
    wl = synth.workload("layer")
    units = []
    for t, spec in enumerate(wl.tensors):
        base = synth.fill_host(wl, t, 0)
        ds = [synth.fill_host(wl, t, 1 + i) for i in range(wl.K)]
        units.append(Unit(spec.rows, spec.cols, base, ds, "bf16"))
    say(f"spectral whole layer, {len(units)} matrices, K={wl.K}")
    t0 = time.perf_counter()
    outs, coef, st = run_spectral(units, wl.K, "bf16")
    say(f"spectral whole layer: {time.perf_counter() - t0:.2f} s on the GPU")
    assert st == 0
    for t in (0, 4):
        ref = _ref(units[t], wl.K, "bf16")
        assert _close(outs[t], "bf16", ref["w_star"]), wl.tensors[t].name
        assert np.allclose(coef[t], ref["c"], rtol=1e-9, atol=1e-12), wl.tensors[t].name
    assert np.all((coef >= 0.0) & (coef <= 1.5))



def test_sign_zero_inner_product():
    """sign(0) := 1 in the joint canonicalisation (App. E).  W_0 = [diag(8..1); 0] (12 x 8) and an
    expert W_1 = R W_0 with R turning the planes (e_1, e_2) and (e_3, e_10) by pi/2: its columns
    8 e_2, -7 e_1, 6 e_10, 5 e_4, ... are mutually orthogonal, so one-sided Jacobi rotates nothing
    and its factors are the normalised columns U_1 = [e_2, -e_1, e_10, e_4 .. e_8], V_1 = I -- the
    gauge the canonicalisation sees.  Modes 1-3 then have <u_0k, u_1k> = 0 exactly and must be
    kept as they are.  A second, generic expert makes the Gram system 2 x 2.  The results of
    zeroing those modes (sign(0) = 0) or flipping them (sign(0) = -1) are far from the answer."""
    m, n = 12, 8
    s0 = np.arange(n, 0, -1).astype(np.float64)
    w0 = np.zeros((m, n))
    w0[:n, :n] = np.diag(s0)
    rmat = np.eye(m)
    for a, b in ((0, 1), (2, 9)):
        rmat[:, [a, b]] = 0.0
        rmat[b, a], rmat[a, b] = 1.0, -1.0
    w1 = rmat @ w0
    rng = np.random.default_rng(12)
    d2 = (rng.standard_normal((m, n)) * 0.05).astype(np.float32).astype(np.float64)
    base = w0.astype(np.float32).ravel()
    ds = [(w1 - w0).astype(np.float32).ravel(), d2.astype(np.float32).ravel()]
    u = Unit(m, n, base, ds, "f32")
    say("spectral sign(0) := 1, 12x8 K=2")
    outs, coef, st = run_spectral([u], 2, "f32")
    assert st == 0
    u0 = np.eye(m)[:, :n]
    u1 = w1 / s0                                        # normalised columns
    assert np.all(np.sum(u0[:, :3] * u1[:, :3], axis=0) == 0.0)
    e2 = sp.thin_svd(w0 + d2)

    def cand(scale):
        uu, vv = u1.copy(), np.eye(n)
        uu[:, :3] *= scale
        vv[:, :3] *= scale
        return sp.iso_merge_factors(u0, s0, np.eye(n), [(uu, s0, vv), e2])

    ref = cand(1.0)
    assert _close(outs[0], "f32", ref["w_star"])
    assert np.allclose(coef[0], ref["c"], rtol=1e-9, atol=1e-12)
    got = outs[0].astype(np.float64).reshape(m, n)
    for wrong in (cand(0.0), cand(-1.0)):
        assert np.max(np.abs(got - wrong["w_star"])) > 0.1


def test_tall_matrices_on_the_cholesky_factor():
    """Tall and wide matrices (longer side >= 1024 and >= twice the shorter) run their Jacobi on the
    Cholesky factor R of A^T A and form U as A V S^{-1}; one call with two of them (fp32 tall
    2048 x 256, and 200 x 1100 with 64-column panels and a ragged last panel) beside a square one,
    K = 3, against the oracle to the usual bars."""
    rng = np.random.default_rng(77)
    K = 3
    units = [_unit(rng, 2048, 256, K, "f32"), _unit(rng, 200, 1100, K, "f32"), _unit(rng, 160, 160, K, "f32")]
    say("spectral cholesky-preconditioned batch: 2048x256, 200x1100, 160x160, K=3")
    outs, coef, st = run_spectral(units, K, "f32")
    assert st == 0
    for u, o, c in zip(units, outs, coef):
        ref = _ref(u, K, "f32")
        assert _close(o, "f32", ref["w_star"]), (u.rows, u.cols)
        assert np.allclose(c, ref["c"], rtol=1e-9, atol=1e-12), (u.rows, u.cols)


def test_ill_conditioned_tall_matrix_falls_back_to_plain_jacobi():
    """A tall fp32 base with singular values from 1 down to 1e-5: the Gram route would lose up to
    eps cond^2 of its small singular values, so the guard (condition number above 1e3) sends that
    matrix back to plain Jacobi on A, while a well-conditioned tall matrix of the same call keeps
    the Cholesky route; both against the oracle to the usual bars."""
    rng = np.random.default_rng(78)
    K = 2
    m, n = 1536, 128
    p, _ = np.linalg.qr(rng.standard_normal((m, n)))
    qq, _ = np.linalg.qr(rng.standard_normal((n, n)))
    w0 = (p * np.logspace(0, -5, n)) @ qq.T * 0.05
    ds = []
    for _ in range(K):
        v = rng.standard_normal(m * n) * 1e-4
        v[rng.random(m * n) > 0.3] = 0.0
        ds.append(nm.from_f64(v, "f32"))
    bad = Unit(m, n, nm.from_f64(w0.ravel(), "f32"), ds, "f32")
    good = _unit(rng, 1280, 96, K, "f32")
    s = np.linalg.svd(nm.to_f64(bad.base, "f32").reshape(m, n), compute_uv=False)
    say(f"spectral ill-conditioned tall {m}x{n} (cond {s[0] / s[-1]:.1e}) beside a well-conditioned 1280x96, K={K}")
    outs, coef, st = run_spectral([bad, good], K, "f32")
    assert st == 0
    for u, o, c in zip((bad, good), outs, coef):
        ref = _ref(u, K, "f32")
        assert _close(o, "f32", ref["w_star"]), (u.rows, u.cols)
        assert np.allclose(c, ref["c"], rtol=1e-9, atol=1e-12), (u.rows, u.cols)


def test_repeat_calls_bit_identical():
    """Six matrices of mixed shapes (three tall enough for the Cholesky route) in one call, twice on
    the same workspace: the Jacobi job sets run as concurrent groups on several streams and the
    per-matrix steps are spread over them, so a race between them would show as a difference
    between the two calls.  Outputs and coefficients must be bit-identical, and one matrix of each
    route still matches the oracle."""
    import torch
    rng = np.random.default_rng(77)
    shapes = [(512, 512), (1536, 384), (1024, 256), (640, 640), (300, 700), (1200, 400)]
    K = 2
    units = [_unit(rng, r, c, K, "f32") for r, c in shapes]
    es = [u.entry() for u in units]
    ws = iso.workspace(iso.OP_UPDATE_SPECTRAL, es, K, dt_code("f32"))
    runs = []
    for rep in range(2):
        say(f"spectral repeat call {rep}: {len(units)} matrices {shapes}")
        coef = torch.zeros(len(units) * K, dtype=torch.float64, device="cuda")
        iso.iso_update(es, K, dt_code("f32"), iso.UPDATE_SPECTRAL, rho_keep=0.9, ridge=1e-12, c_min=0.0,
                       c_max=1.5, coef_out=coef, ws=ws)
        assert iso.iso_read_device_status(ws) == 0
        runs.append(([from_dev(u.dout, u.n, "f32").copy() for u in units], coef.cpu().numpy().copy()))
    for t in range(len(units)):
        assert np.array_equal(runs[0][0][t].view(np.uint32), runs[1][0][t].view(np.uint32)), shapes[t]
    assert np.array_equal(runs[0][1].view(np.uint64), runs[1][1].view(np.uint64))
    for t in (0, 1):
        ref = _ref(units[t], K, "f32")
        assert _close(runs[1][0][t], "f32", ref["w_star"]), shapes[t]
