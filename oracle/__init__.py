"""CPU oracle for the ISO merge/update hot path.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, float64 restatement
of what the paper defines, written so that it can be checked against the paper
by eye.  Only the test suite, the smoke check and the benchmark's CPU-baseline
leg may import it.  The product path (the HIP library and its Python binding)
never imports, calls or links anything here, and the oracle shares no code with
it: the two meet only through the seeded input generator in ``synth``.

Modules
-------
numerics  storage-format conversions, single rounding float64 -> bf16/fp32,
          exact sign of a float sum (Shewchuk grow-expansion), density -> k.
ties      TopKMask (App. F, TIES "Trim"), sign election, TIES disjoint mean,
          Task Arithmetic, RAM, and the final theta_0 + lambda*tau.
spectral  ISO-Merger (Sec. 4.2, App. E, Algorithm 1) in float64.
tsv       TSV-Merge (App. F): per-delta truncated SVD, concatenation,
          Procrustes orthogonalisation, reconstruction.

Every function with no independent pin says "parity unpinned" in its
docstring; the pins live in tests/test_oracle_*.py.
"""
