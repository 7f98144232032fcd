"""CPU oracle for the DriveCache cache-aware denoising step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library, its
Python binding, the sampler) may import, call or link anything here; only the
tests, the smoke check and the CPU-baseline leg of the benchmark do.  The
oracle shares no code with the HIP path: it consumes the same seeded inputs
(`paper_2608_16354_amd.inputs`, which holds no method arithmetic) and
re-derives everything else from the paper.

Precision: the generator arithmetic is float64 NumPy; the planner is float64
Python scalars, one IEEE operation at a time (no fused multiply-add); schedule
costs are exact integers.

Modules
  planner  motion statistics, support gate, motion intensity, scene tables
           (Sec. 3.1, Eq. 2-4, Eq. 8-9)
  dp       exact schedule DP with backtracking (Sec. 3.2, Eq. 10-11) and an
           independent brute-force enumeration of reuse placements
  budget   the response-budget rule (Sec. 4.1 protocol, Sec. 3.2)
  dit      the spatiotemporal DiT generator, its cache boundary (Eq. 1) and
           the Euler flow-matching sampler
  runtime  the causal controller: drift check, veto, charge and suffix
           replanning (Sec. 3.2, Eq. 12), and the uncached sampler

Pins (what fixes each part independently of this code) live in
tests/test_oracle_*.py.  Parity unpinned: the full-scale bf16 generator
numerics are checked only against this oracle; the paper prints no tables,
weights or worked example to compare with.
"""
