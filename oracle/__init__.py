"""CPU oracle for the guarded decode-op path -- TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package. The product library never calls it, and it shares no
code with the GPU library: no kernels, headers, tables, constants or
helpers. Both sides take their inputs from the seeded generators in
`workloads`, which hold no arithmetic of the ops.

Contents
--------
numerics   exact double -> bfloat16 / float32 round-to-nearest-even and the
           exact bf16 -> double upcast.
ops        RMSNorm, residual-add + RMSNorm, RoPE on Q and K, SwiGLU and the
           decode chain, evaluated in float64 from their plain definitions
           and rounded once to the output dtype.
selection  the guarded specialization cache as a step-by-step model of
           ordered dispatch (Algorithm 1 of the paper, Sec. 3.2) and of the
           miss / install / error paths (Sec. 3.5): key packing, guard
           flags, the install policy table, version order and statistics.

Every function is pinned by tests under `-m "not gpu"` against closed
forms, library routines and brute force; nothing here is "parity unpinned".
"""
from . import numerics, ops, selection  # noqa: F401
