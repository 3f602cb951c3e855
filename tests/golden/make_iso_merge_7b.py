"""Writes iso_merge_7b.npz: the oracle's ISO-Merger (Algorithm 1, App. E) on two full-size matrices
of the 7B stack -- layer 0's gate_proj (18944 x 3584, tall) and down_proj (3584 x 18944, wide) --
with the stack's K = 4 bf16 expert deltas from the seeded generator, at the default parameters
(rho_keep 0.9, ridge 1e-12, c in [0, 1.5]).  Stored per matrix: the coefficients c (K) and W_*
in binary64 at the coordinates sample_idx(rows * cols) (32768 seeded positions and the last
1024 entries).  Only the oracle and the seeded input generator run here.

    python tests/golden/make_iso_merge_7b.py        # about 15 minutes on 8 cores
"""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import numerics as nm  # noqa: E402
from oracle import spectral as sp  # noqa: E402
import synth  # noqa: E402

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "iso_merge_7b.npz")
TENSORS = {"gate": 4, "down": 6}            # indices in the 7B stack (layer 0)
SAMPLE_SEED = 2607


def sample_idx(n):
    rng = np.random.default_rng(SAMPLE_SEED)
    return np.unique(np.concatenate([rng.integers(0, n, size=32768), np.arange(max(0, n - 1024), n)]))


def main():
    wl = synth.workload("7b")
    out = {}
    for name, t in TENSORS.items():
        spec = wl.tensors[t]
        t0 = time.time()
        w0 = nm.to_f64(synth.fill_host(wl, t, 0, threads=8), "bf16").reshape(spec.rows, spec.cols)
        ds = [nm.to_f64(synth.fill_host(wl, t, 1 + i, threads=8), "bf16").reshape(spec.rows, spec.cols)
              for i in range(wl.K)]
        res = sp.iso_merge(w0, ds)
        out[f"{name}_c"] = res["c"]
        out[f"{name}_w"] = res["w_star"].ravel()[sample_idx(spec.numel)]
        print(f"{spec.name} {spec.rows}x{spec.cols}: c = {res['c']}, {time.time() - t0:.0f} s", flush=True)
        del w0, ds, res
    np.savez_compressed(PATH, **out)
    print("wrote", PATH)


if __name__ == "__main__":
    main()
