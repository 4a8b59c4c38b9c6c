"""CPU reference for the shared-stage hot path.  TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, float64 NumPy statement of what the hot path
computes.  It shares no code with the HIP library and imports nothing from
it.  Only the test suite, the smoke check and the benchmark's CPU-baseline leg
may import it; the product path never calls it.

Modules
-------
``layer``      decoder-layer forward (prefill with optional cached prefix,
               and decode as the single-row case), stack forward.
``partition``  the integer side: packed-batch metadata and the complementary
               CU-mask partition.

Every layer formula here is silent in the paper (it keeps the model execution
of its base runtime unchanged, §5); the paper only fixes that prefill reads
the whole context and builds the key/value cache, and that decode re-reads the
weights and the cache for each new token (§2.1, "Autoregressive
transformers").  The layer composition is the standard pre-norm decoder layer
(RMSNorm, RoPE, grouped-query causal attention, SwiGLU FFN) and each reading
of an unstated detail is listed at the top of the module that takes it.
"""
