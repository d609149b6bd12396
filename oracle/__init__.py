"""CPU oracle for the GCPSL hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow reimplementation of what the path computes, written from the
paper ("Concurrent Split Learning Through Stable Client Clustering") and the
readings of it listed in the design notes: static client clustering
(Alg. 1), cluster-local GPSL sampling (Eq. 1, Eq. 3), the split forward and
backward pass, the SGD update, sample-weighted fusion (Eq. 5) and direct data
participation (Sec. V-E, Eq. 7), and the epoch-barrier round schedule
(Sec. III-A, Eq. 6).  Floating point is fp64 throughout; for the
bf16 workloads the oracle rounds to bf16 (round-to-nearest-even) at the same
points the GPU path does.

Only tests/, the smoke check and the cpu_baseline leg of the benchmark may
import this package.  It shares no code with the HIP path; both take their
inputs from gcpsl_inputs, which holds no arithmetic of the method.

Parity status of each part (pins live in tests/test_oracle_*.py):
  rng, assign, sampler, participation  pinned (published test vectors,
                                        brute force, hand-built cases)
  model layers, split step, SGD        pinned (textbook loops, finite
                                        differences, torch.autograd)
  fusion                               pinned (identity, worked example)
  epoch-barrier schedule (Eq. 6)       pinned (worked example, waiting
                                        clusters untouched, equal lengths
                                        reduce to the lockstep schedule)
  multi-step end-to-end values         pinned (per-replica torch autograd +
                                        torch.optim.SGD training loops fused
                                        by numpy's weighted average, across
                                        fusions, fp32 and bf16)
"""
