"""MI355X-native Partial FC classifier-head step (arXiv 2010.05222) on one class shard.

The step (sampling, remap, gather + normalise, cosine contraction, margin
softmax cross-entropy, backward and the sparse momentum update) runs in
libpfc.so, hand-written HIP for gfx950 behind the C ABI of include/pfc.h.
``paper_2010_05222_amd.pfc`` is the ctypes binding with the same names,
``paper_2010_05222_amd.head.PfcShard`` a torch-facing wrapper that owns the
step's buffers, and ``paper_2010_05222_amd.build`` compiles the library.
"""

__all__ = ["build", "pfc", "head"]
