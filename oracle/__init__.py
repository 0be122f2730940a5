"""Plain, slow fp64 CPU oracle of pipelined gradient coding (PGC).

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import, call or execute anything in this package. The
product path (the HIP library and its Python binding) never imports it, and
the two share no code: no kernels, headers, helpers or table generators.

Modules:
  rng         -- SplitMix64 and the straggler-mask / encoding-matrix draws,
                 written from the generator's published definition, and the
                 simulated cluster step with exponential worker delays.
  pgc_oracle  -- placement, schedule, coded gradients, decoding and the
                 update, step by step in the paper's order and notation.

Parity unpinned (no value in the paper to check against; see the module
docstrings for what is pinned instead):
  * the particular real-valued encoding matrix B of the naive cyclic scheme
    (the paper cites its construction but does not print one);
  * the bf16-input MLP gradient beyond the 2e-2 tolerance of its path.
"""
