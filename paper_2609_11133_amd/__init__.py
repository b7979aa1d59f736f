"""MI355X-native MoE decode layer.

The hot path (router logits, top-k softmax, token grouping, grouped FP8/MXFP4
SwiGLU experts, weighted combine) runs in hand-written HIP kernels for gfx950
behind the C ABI declared in ``include/moe_decode.h``.  ``binding`` is a thin ctypes
layer over that library; importing it fails loudly when the library is not built.
"""
__all__ = ["configs", "synth"]
