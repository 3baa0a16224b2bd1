"""CPU oracle for refusal-gated decoding (test infrastructure only).

A plain, slow, float64 numpy reference for everything the GPU path computes:
Philox4x32-10 draws, greedy argmax, temperature-scaled min-p and p-less
sampling with an inverse-CDF draw, grouped-query attention over a shared prompt KV plus a
per-row tail, a Llama-style decoder step and prefill, the refusal-prefix
compatibility predicate, the greedy probe with early exit and the gate of
Algorithm 1 (Section 3).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It shares no code with the HIP library and never imports
it; the HIP library never imports or calls anything here.

Parity status: every function is pinned by the CPU tests (closed forms,
brute-force loops, library routines, invariants, published known-answer
vectors), except where a module header says "parity unpinned".
"""
