"""CPU oracle for the pruned, mixed-precision, block-quantized MoE layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute anything in this package; only the test suite, the smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the HIP library.

Plain, slow, obviously correct numpy in float64, one function per step of the
layer forward of "Collaborative Compression for Large-Scale MoE Deployment on
Edge" (arXiv 2509.25689):

* ``quant``  -- the block-32 symmetric weight format (quantize, dequantize,
  canonical bit packing).  Section 3.3 keeps most tensors at a low bit width
  and gives each tensor its own width; the block format is the concrete
  encoding this library uses in place of llama.cpp's codebooks.
* ``router`` -- sigmoid scores, experts removed by pruning masked out,
  group-limited top-k, normalisation and scaling (Sections 3.1 and 3.2; the
  DeepSeek-V3 routing the paper's model uses).
* ``bucket`` -- token-to-expert bucketing as a stable sort.
* ``moe``    -- the SwiGLU experts, the weighted combine and the shared expert
  (Fig. 1, middle), accumulated in float64, plus the error metric.
* ``planner`` -- the bit-allocation arithmetic of Section 3.3.

Pins: every function is checked in ``tests/test_oracle_*.py`` against closed
forms, brute force on tiny inputs, special cases that reduce to a textbook
routine, and invariants.  The whole-layer output has no worked example in the
paper: parity unpinned against the paper; pinned by those properties only.
"""
