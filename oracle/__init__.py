"""NOVA-KV test oracle -- plain, slow, fp64 CPU implementation.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()``
and the benchmark's CPU-baseline leg may import or run anything in this
package.  The GPU library (``paper_2608_04074_amd``) never imports it, and it
shares no code, header, table or helper with the GPU path; the only module
both sides use is the seeded input generator ``synth``, which holds none of the
method's arithmetic.

Contents (each function cites the passage of the paper it follows):
  calibration  statistics, Theorem 1 key transform, Corollary 1 value
               transform, volume-equalizing grouping fold, codebooks
  vq           exhaustive nearest-codeword encoder (plain C helper
               ``vq_ref.c``), Lloyd k-means, codeword lookup
  codec        append-time encode of keys and values; the key-scale format
               (per-token bf16 scale), the scalar value arm (per-token
               affine INT2 in a rotation basis), bf16 storage of band rows
  attention    plain-form decode attention (reconstruct, then textbook
               softmax attention with an optional sink), with the key scale,
               the sink-plus-recent band and the scalar value arm; a fast
               split form used only to check the plain one
  fp8          fp8 E4M3 snapping of the codebooks
  grouping     Theorem 2 volumes, rate allocation and distortions
  accounting   cache byte and parameter counts

Parity status: every function is pinned by tests in ``tests/test_oracle_*.py``
except Lloyd training beyond its invariants (monotone distortion, lossless on
<= k distinct points, determinism) -- "parity unpinned" for the exact
codebook values, which are inputs to the GPU path, not outputs it must match.
"""

from . import accounting, attention, calibration, codec, fp8, grouping, vq  # noqa: F401
