"""CPU oracle for the ZO-Act forward-only step.  TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct NumPy implementation of what the hot path
computes, written from the paper (ZO-Act, arXiv 2607.01125): Algorithm 1
(one-shot activation basis), the adapted linear of Section 3, and the body of
Algorithm 2 in the two-sided form (one +/- pair per step) followed by Adam.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this package.  It shares no code with the HIP library: it reads the synthetic
inputs from `synth` as data and nothing else.

Floating point: fp32-mode quantities are computed in float64; bf16-mode
quantities are computed in float32/float64 with every bf16 storage rounding
emulated bit-exactly (round-to-nearest-even).  The Gaussian perturbation is
computed in float32 exactly as specified in `oracle.rng`.

Parity status of each function is stated in its module header; every function
is pinned by a CPU test under tests/ (closed forms, brute force, invariants),
except where a header says "parity unpinned".
"""
