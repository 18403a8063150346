"""Plain fp64 CPU oracle for the ReLU-sparse FFN hot path. TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check in `__graft_entry__` and the benchmark's
CPU-baseline leg may import this package. The library (`paper_2603_23198_amd`)
never calls it, and this package shares no code with the HIP kernels: it
re-derives the TwELL layout, the row classification and the bf16 rounding from
the paper on its own.

Contents (paper sections are those of "Sparser, Faster, Lighter Transformer
Language Models"):

* `bf16`   - round-to-nearest-even to bf16, written from the IEEE definition.
* `twell`  - Alg. 1's TwELL extraction (per row and column tile, ascending
             scan, strict > 0), the hybrid row classification of Sec. 3.4
             and the row-ELL of the hybrid format.
* `ffn`    - the gated FFN (eq. sec2:eq:gated-mlp), the non-gated FFN
             (eq. secC:eq:non-gated-mlp), the sparse formulations of
             Alg. 2 / eq. sec3:eq:twell_to_dense_fused_matmul and Alg. 3,
             the L1 term of eq. l1 and the gradients of
             eq. sec3:eq:all_other_gradients.
* `sizing` - the binomial tail behind the TwELL compression-factor choice
             (Appendix A, TwELL matmul discussion).
* `training` - the dead-unit record (a unit is dead for a training step when it
             was never active in it) and the targeted re-initialisation of dead
             units' gate-projection columns (appendix on training modifications).

Everything is computed in float64 on the *stored* inputs (bf16 bit patterns
or float32 values widened exactly). Pins: every function is checked by the
`-m "not gpu"` tests against brute force, exact rational arithmetic, closed
forms, finite differences or library routines; none is "parity unpinned".
"""
