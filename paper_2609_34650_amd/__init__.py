"""MI355X-native fused hybrid causal-attention layer (Selective Attention
Freezing): ordinary softmax heads and fixed-pattern heads in one kernel.

The compute lives in ``libsaf.so`` (hand-written HIP for gfx950, C ABI
declared in ``include/saf.h``).  ``paper_2609_34650_amd.binding`` marshals
torch tensors into that ABI.  Importing this package loads nothing, so the
seeded input generators in ``paper_2609_34650_amd.inputs`` stay usable
without a GPU.
"""
