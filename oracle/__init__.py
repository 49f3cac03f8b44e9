"""CPU oracle for the XShare batch-level MoE layer -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct re-statement of what the paper's method
computes, used to check the HIP path.  Only the tests, the package's smoke
check and the benchmark's CPU-baseline leg may import it; the product path
never calls it, and it shares no code, constants or helpers with the HIP
sources.

Modules:
* ``numerics`` -- the fp32 exponential and the ranked softmax used by the gates
  (Section 2.2), with every rounding step spelled out;
* ``route``    -- vanilla top-k gating (Section 2.2), Algorithm 2 (warm-up,
  fixed-budget greedy of Algorithm 1, refinement; Section 3.4), and
  Algorithms 3 + 4 (per-request then batch selection; Section 4.1);
* ``ffn``      -- the MoE layer output of Section 2.1 with SwiGLU experts,
  in float64.

Parity status: every function here is pinned by the CPU tests (closed form
of Section 1, brute-force optimum of Eq. (2) per Corollary 3.2, invariants,
special-case reductions, an independent library ranking, a float64 softmax,
a closed-form FFN); no function is "parity unpinned".
"""
