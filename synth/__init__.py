"""Seeded synthetic workloads (inputs only; no merge arithmetic).

The element recipe lives in ``philox.h``; ``libsynth_host.so`` (gcc) and
``libsynth_dev.so`` (hipcc) are two builds of it that produce identical bits,
so a tensor generated in HBM can be checked element by element against
values regenerated on the host.

Workloads are the five shapes the hot path is measured on: weights stand in
for the paper's checkpoints (Qwen2.5-7B-Instruct with RL experts; a
DeepSeek-R1-Distill-Qwen-1.5B pair) which are not available; deltas are
modelled as i.i.d. sparse perturbations of the stated distributions.
"""
import ctypes
import os
from dataclasses import dataclass, field
from fractions import Fraction
from typing import List

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))

NORMAL, LAPLACE, ZERO = 0, 1, 2
F32, BF16 = 0, 1


class Recipe(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint32), ("stream", ctypes.c_uint32), ("dist", ctypes.c_uint32),
                ("zero_thresh", ctypes.c_uint32), ("scale", ctypes.c_double)]


@dataclass(frozen=True)
class Dist:
    kind: int            # NORMAL / LAPLACE / ZERO
    scale: float         # sigma or b
    p_zero: Fraction = Fraction(0)

    @property
    def zero_thresh(self):
        return int(min(self.p_zero * 2 ** 32 + Fraction(1, 2), 2 ** 32 - 1) // 1)


@dataclass(frozen=True)
class TensorSpec:
    name: str
    rows: int
    cols: int

    @property
    def numel(self):
        return self.rows * self.cols


@dataclass
class Workload:
    name: str
    dtype: str                      # "f32" | "bf16"
    K: int
    tensors: List[TensorSpec]
    base: Dist
    delta: Dist
    density: Fraction
    seed: int = 0
    tsv_rank: int = 0               # >0: MLP matrices go through the blockdiag/SVD projection
    tsv_names: tuple = field(default_factory=tuple)

    @property
    def numel(self):
        return sum(t.numel for t in self.tensors)

    def recipe(self, t_idx, role):
        """role 0 = base, 1..K = delta i."""
        d = self.base if role == 0 else self.delta
        return Recipe(self.seed, ((t_idx & 0xFFFFFF) << 8) | role, d.kind, d.zero_thresh, d.scale)

    @property
    def sdtype(self):
        return BF16 if self.dtype == "bf16" else F32

    def np_dtype(self):
        return np.uint16 if self.dtype == "bf16" else np.float32


def _layers(n_layers, hidden, inter, kv):
    out = []
    for layer in range(n_layers):
        p = f"layers.{layer}."
        out += [TensorSpec(p + "q_proj", hidden, hidden), TensorSpec(p + "k_proj", kv, hidden),
                TensorSpec(p + "v_proj", kv, hidden), TensorSpec(p + "o_proj", hidden, hidden),
                TensorSpec(p + "gate_proj", inter, hidden), TensorSpec(p + "up_proj", inter, hidden),
                TensorSpec(p + "down_proj", hidden, inter)]
    return out


def tiny():
    """One fp32 256x256 matrix, K=3, nonzero prob 0.3, density 0.2, seed 0."""
    return Workload("tiny", "f32", 3, [TensorSpec("w", 256, 256)], Dist(NORMAL, 0.02),
                    Dist(NORMAL, 1e-3, Fraction(7, 10)), Fraction(1, 5))


def layer():
    """One 2048-hidden layer in bf16 (shapes as rows x cols), K=2, 50% zeros, density 0.1."""
    t = [TensorSpec(n, 2048, 2048) for n in ("q_proj", "k_proj", "v_proj", "o_proj")]
    t += [TensorSpec("gate_proj", 2048, 5632), TensorSpec("up_proj", 2048, 5632),
          TensorSpec("down_proj", 5632, 2048)]
    return Workload("layer", "bf16", 2, t, Dist(NORMAL, 0.02), Dist(NORMAL, 1e-4, Fraction(1, 2)),
                    Fraction(1, 10))


def stack_1p5b():
    """28 layers, hidden 1536, intermediate 8960, kv 256 (2 heads x 128), tied 151936 x 1536 embedding."""
    t = _layers(28, 1536, 8960, 256) + [TensorSpec("embed_tokens", 151936, 1536)]
    return Workload("1.5b", "bf16", 4, t, Dist(NORMAL, 0.02), Dist(LAPLACE, 5e-5, Fraction(7, 10)),
                    Fraction(1, 20))


def stack_7b():
    """28 layers, hidden 3584, intermediate 18944, GQA kv 512, untied 152064 x 3584 embed and lm_head."""
    t = _layers(28, 3584, 18944, 512) + [TensorSpec("embed_tokens", 152064, 3584),
                                          TensorSpec("lm_head", 152064, 3584)]
    return Workload("7b", "bf16", 4, t, Dist(NORMAL, 0.02), Dist(NORMAL, 5e-5, Fraction(4, 5)),
                    Fraction(1, 10))


def stack_7b_tsv():
    w = stack_7b()
    w.name = "7b-tsv"
    w.tsv_rank = 64
    w.tsv_names = ("gate_proj", "up_proj", "down_proj")
    return w


WORKLOADS = {"tiny": tiny, "layer": layer, "1.5b": stack_1p5b, "7b": stack_7b, "7b-tsv": stack_7b_tsv}


def workload(name):
    return WORKLOADS[name]()


# ---- library loading -----------------------------------------------------------------------------

_host = None
_dev = None


def host_lib():
    global _host
    if _host is None:
        path = os.path.join(HERE, "libsynth_host.so")
        if not os.path.exists(path):
            raise RuntimeError("libsynth_host.so is not built; run __graft_entry__.build()")
        _host = ctypes.CDLL(path)
        _host.synth_fill_host.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                          ctypes.POINTER(Recipe), ctypes.c_int64]
        _host.synth_gather_host.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                            ctypes.POINTER(Recipe)]
    return _host


def dev_lib():
    global _dev
    if _dev is None:
        path = os.path.join(HERE, "libsynth_dev.so")
        if not os.path.exists(path):
            raise RuntimeError("libsynth_dev.so is not built; run __graft_entry__.build()")
        _dev = ctypes.CDLL(path)
        _dev.synth_fill_device.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int,
                                           ctypes.POINTER(Recipe), ctypes.c_int64, ctypes.c_void_p]
        _dev.synth_fill_device.restype = ctypes.c_int
    return _dev


def fill_host(wl, t_idx, role, first=0, n=None, threads=1):
    """Storage array (uint16 bf16 bits or float32) for elements [first, first+n) of a tensor.

    With threads > 1 the range is split into that many contiguous pieces filled
    concurrently (each element depends only on its own counter, so the bits are
    the same)."""
    spec = wl.tensors[t_idx]
    if n is None:
        n = spec.numel - first
    out = np.empty(n, dtype=wl.np_dtype())
    r = wl.recipe(t_idx, role)
    lib = host_lib()
    parts = max(1, min(int(threads), n // (1 << 20)))
    if parts == 1:
        lib.synth_fill_host(out.ctypes.data, n, wl.sdtype, ctypes.byref(r), first)
        return out
    from concurrent.futures import ThreadPoolExecutor
    edges = [n * p // parts for p in range(parts + 1)]

    def piece(p):
        a, b = edges[p], edges[p + 1]
        lib.synth_fill_host(out[a:].ctypes.data, b - a, wl.sdtype, ctypes.byref(r), first + a)

    with ThreadPoolExecutor(parts) as ex:
        list(ex.map(piece, range(parts)))
    return out


def gather_host(wl, t_idx, role, idx):
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, dtype=wl.np_dtype())
    r = wl.recipe(t_idx, role)
    host_lib().synth_gather_host(out.ctypes.data, idx.ctypes.data, idx.size, wl.sdtype, ctypes.byref(r))
    return out


def fill_device(ptr, n, wl, t_idx, role, stream=0, first=0):
    """Generate elements [first, first+n) of (tensor, role) into device memory at ``ptr``."""
    r = wl.recipe(t_idx, role)
    rc = dev_lib().synth_fill_device(ctypes.c_void_p(ptr), n, wl.sdtype, ctypes.byref(r), first,
                                     ctypes.c_void_p(stream))
    if rc != 0:
        raise RuntimeError(f"synth_fill_device failed ({rc})")


def build(verbose=False):
    """Compile both builds of the generator in-tree."""
    import subprocess
    cmds = [
        ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-o",
         os.path.join(HERE, "libsynth_host.so"), os.path.join(HERE, "host.c")],
        ["hipcc", "--offload-arch=gfx950", "-O3", "-ffp-contract=off", "-fPIC", "-shared",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-o", os.path.join(HERE, "libsynth_dev.so"), os.path.join(HERE, "device.hip")],
    ]
    for c in cmds:
        if verbose:
            print(" ".join(c))
        subprocess.run(c, check=True)
