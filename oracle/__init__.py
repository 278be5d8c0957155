"""Plain, slow float64 CPU oracle of the APEX MoE-decode hot path.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it.  It shares no code with the HIP path (no
kernels, headers, helpers or constants); the only module both sides use is the seeded
input generator, which holds none of the method's arithmetic.

Every function follows a passage of the paper (APEX: Adaptive Expert Prefetching for
Memory-Efficient Edge MoE Inference) and cites it by section, equation or algorithm:

* ``routing``    prefetch router, ranked list, adaptive prefetch-set selection
                 (Sec. IV-A, IV-B Eq. 1, IV-C Eq. 8-9, IV-D)
* ``gating``     original-router top-k, correctness-preserving and stall-free
                 selection (Sec. III-A, IV-E, Algorithm 1)
* ``ffn``        SwiGLU experts and their gated sum (Sec. III-A, IV-E)
* ``residency``  per-layer HBM cache of expert slots (replaces the per-layer buffer of
                 Sec. V-C; rule stated in the module)
* ``metrics``    oracle budget delta*, overlap, full coverage (Sec. IV-B Eq. 2-3, V-C)
* ``decode``     one decode step through all layers, composing the above

Pins: every function is checked in ``tests/test_oracle_*.py`` against brute force,
closed forms, library routines on special cases and invariants the paper states.
"""
