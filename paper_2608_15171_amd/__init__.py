"""MI355X-native attention for one mixed scheduler step over a paged KV cache.

The compute lives in the HIP library ``libppas.so`` (C ABI declared in
``include/ppas.h``); ``paper_2608_15171_amd.ppas`` is its thin Python binding.
``inputs`` draws seeded synthetic steps, ``ppas_trace`` composes the steps of a
multi-request trace under the P-PAS policy, and ``metrics`` holds the
algorithmic FLOP/byte accounting used for roofline fractions.

Importing this package loads nothing native; importing ``.ppas`` does, and fails
loudly when the library has not been built.
"""
