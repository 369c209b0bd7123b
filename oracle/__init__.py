"""CPU oracle for the single-device pipeline-stage training path.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute anything in this package: only the tests, the smoke check and the
benchmark's CPU-baseline leg use it. It shares no code with the HIP library
(no kernels, headers, helpers, tables or pre/post-processing); the only
common module is `synth`, which generates seeded inputs and holds none of
the method's arithmetic.

The oracle computes plain definitions in float64 with numpy (matrix products
are library calls; everything else is written out), except where the method
itself is defined in float32 (gradient accumulation and the AdamW step over
fp32 master parameters, with the bf16 cast), which are evaluated in float32
one IEEE operation at a time.

Modules
  stage   -- decoder-stage Chunk forward/backward (dense and top-2 MoE),
             the microbatch Order runner and gradient accumulation
  optim   -- fp32 gradient accumulation, AdamW and the bf16 RNE cast
  order   -- 1F1B / GPipe Order generation and the Order validity rules

Every function that has no independent pin says "parity unpinned" in its
docstring; all others are pinned by tests under tests/test_oracle_*.py.
"""
