"""CPU oracle for the WeightBridge resharding hot path (test infrastructure only).

This package is a plain, slow, obviously correct statement of what the
plan-driven resharding copy computes. It exists to check the HIP path; only the
test suite, the smoke check and the CPU-baseline leg of the benchmark import
it. It shares no code with ``paper_2609_25442_amd`` (the C++ planner and the
HIP kernels) and never imports it; the two meet only in the seeded synthetic
checkpoint generator, which holds no resharding arithmetic.

Modules and the passages they follow (WeightBridge, arXiv 2609.25442):

* ``catalog``  -- the checkpoint index space that bridges trainer and rollout
  layouts (Sec. 3.1, "the checkpoint of the full model can be used as a bridge").
* ``layout``   -- source maps as slice-copies, each optionally transposed
  (Sec. 3.1 and App. B), generated for FSDP flat shards, Megatron-style TP/EP
  and serving-style TP/EP layouts.
* ``plan``     -- correspondence by overlapping source maps, trainer-replica
  de-duplication and balanced assignment (Sec. 3.2, "Generating an efficient
  routing plan"), plus the coalesced per-receiver wire format (Sec. 3.2,
  packing kernel).
* ``casts``    -- fp32 -> bf16 and -> fp8 e4m3 rounding written from the IEEE 754
  and OCP OFP8 definitions, and the 128x128 blockwise scale (not in the paper,
  which leaves precision conversion to future work in Sec. 5).
* ``transfer`` -- pack (Sec. 3.2, packing kernel), unpack (Sec. 3.2, assembly
  kernel) and the plan-independent expected rollout tensors.

Pins (tests/test_oracle_*.py) tie each function to something other than
itself: published parameter counts, brute-force enumeration on tiny layouts,
independent torch slicing, torch's own dtype conversions, and values fixed by
the IEEE/OCP formats.
"""
