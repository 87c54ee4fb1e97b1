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

Parity status: every function is pinned by tests in ``tests/test_oracle_*.py``.
Lloyd training is pinned by its invariants (monotone distortion, lossless on
<= k distinct points, determinism), by scikit-learn's Lloyd from the same
start when no cluster empties, by a start that must be k distinct training
points, and by a hand-built case whose empty clusters must be refilled from
the worst-fit points, farthest first.  The value grouping is pinned by a
distribution on which the variance order, its reverse, the eigenvalue order
of M_o and the raw-coordinate order all differ.  The pins of these steps are
also run against planted mistakes, which they must catch.
"""

from . import accounting, attention, calibration, codec, fp8, grouping, vq  # noqa: F401
