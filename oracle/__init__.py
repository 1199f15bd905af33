"""CPU oracle for DynaCalKV compressed-KV decode attention.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check of the entry
module and the CPU-baseline leg of the benchmark may import this package.  The
GPU library never calls it, and it shares no code, tables or constants with
the HIP path: it is a plain, slow, fp64 restatement of what the method
computes, written so that each step can be checked against the paper by eye.

Modules
  bf16        round-to-nearest-even from fp64 directly to bfloat16
  bookkeeping head/group partition, offsets (Sec. III-C column-wise grouping)
  params      parameter counts of the key factors (Sec. III-C equations)
  layout      the paged latent-cache layout (a stated reading: the paper
              fixes no cache layout)
  append      latent write z = x L (Sec. III-A), rounded to the storage type
  attention   decode: rebuild K = Z_g R_g and V = Z_v R_v per head
              (Sec. III-A, III-C, III-D), then textbook two-pass softmax
              attention in fp64
  dense       uncompressed paged K/V decode (the comparison baseline)
  rope        decode with rotary position embedding on the rebuilt keys (a
              reading: the paper never mentions positional encodings)
  compress    offline key compression, Algorithm 1: CKA head similarity,
              agglomerative clustering, energy ranks, greedy budget
              adjustment, per-group SVD, the cluster-count objective
              (Sec. III-A, III-C)
  calibrate   value calibration refinement: calibration error and the two
              closed-form factor updates (Sec. III-D)

Parity status: every function here is pinned by the `-m "not gpu"` tests
(closed forms, full-rank equivalence with uncompressed attention computed by
a library routine, printed Table 1 figures, exhaustive/brute-force checks;
the rotary reading by RoFormer's complex form and hand-worked rotations).
"""

from . import bf16, bookkeeping, params, layout, append, attention, dense  # noqa: F401
from . import compress, calibrate, rope  # noqa: F401
