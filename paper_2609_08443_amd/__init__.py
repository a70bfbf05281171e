"""MI355X (gfx950) implementation of SequenceO1's Sketch Attention sketching step.

The computation lives in libsa_sketch.so (HIP kernels behind the C ABI of
include/sa_sketch.h); ``sa_sketch`` is its Python binding and ``workloads``
draws the paper-shaped synthetic inputs.
"""

__all__ = ["sa_sketch", "workloads"]
