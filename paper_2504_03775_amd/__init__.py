"""MI355X-native KV-cache transfer hot path of FlowKV (arXiv 2504.03775).

Contiguity-aware block allocation, bidirectional segment alignment and a
one-launch segment-coalesced copy for gfx950, behind the C ABI in
``include/flowkv.h``.  ``paper_2504_03775_amd.flowkv`` is the binding (it
loads ``libflowkv.so`` and fails if it is not built);
``paper_2504_03775_amd.build`` builds it.
"""
