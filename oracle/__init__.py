"""CPU oracle for one mixed scheduler step's attention over a paged KV cache, and for
the other prefill operation the paper profiles (the fused gate-up projection).

TEST INFRASTRUCTURE. Only the tests, the package entry's smoke check and the
benchmark's CPU-baseline leg may import or run anything here; the product path
never does. It shares no code with the HIP path: inputs arrive as bf16 bit
patterns and integer descriptors, and everything else (bf16 decoding, the cache
semantics, masking, softmax, page addressing) is written out again here, slowly
and in float64.

Modules:
  attention -- the attention of a mixed step (chunked prefill rows and decode rows)
  kv_cache  -- where kv_append puts a step's new keys and values in the page pools
  policy    -- the P-PAS per-iteration prefill budget (Algorithm 1)
  rope      -- rotary position embedding of a step's new Q and K rows before the append
  gemm      -- the fused gate-up projection of a decoder block's MLP (the other profiled prefill op)
"""
