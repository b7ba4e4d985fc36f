"""Float64 CPU oracle for bucket-level gradient-conflict resolution.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this package: it exists so that tests, the smoke check and the
benchmark's CPU-baseline leg can check the HIP library against a plain,
slow, obviously correct restatement of the paper's method.  It shares no
code with the HIP library (no kernels, headers, helpers or constants).

Parity status of each function (what pins it is listed in its docstring):

* gram, combine, bf16 rounding ........ pinned (definitions; library routines,
  brute force, torch's RNE cast)
* mgda_fw ............................. pinned for K=2 (closed form) and by the
  exact solver's optimum it approaches; for K>=3 after 20 iterations its
  distance to the optimum is a diagnostic, not a claim
* mgda_exact .......................... pinned (simplex grid search, KKT)
* pcgrad .............................. pinned (vector-form projection on
  tiny buckets, no-conflict and K=2 closed forms)
* cagrad_fw / cagrad_exact ............ pinned (primal feasibility, zero
  duality gap, random-direction search, c=0 reduction, descent bound)
* slice_offsets, gram_reduce ........... pinned (partition of every bucket,
  additivity of inner products over slices, exact on integer data)
* conflicts ........................... pinned (cosines and conflict counts
  from the vectors, closed-form configurations, invariances)
"""

from .reference import (  # noqa: F401
    bf16_bits_to_f64,
    cagrad_exact,
    cagrad_fw,
    combine,
    conflicts,
    decode_rows,
    f64_to_bf16_bits,
    gram,
    gram_reduce,
    mgda_exact,
    mgda_fw,
    pair_min_norm,
    pcgrad,
    resolve,
    round_to_dtype,
    slice_offsets,
    solve,
)
