"""Memory-efficient exact attention for MI355X (gfx950).

Dense softmax attention computed over key/value tiles with the lazy softmax
and a running maximum (arXiv 2112.05682, Sections 2-4), plus a backward that
recomputes tile scores instead of storing them (Section 5.2).  The kernels are
hand-written HIP for gfx950 behind the C ABI in ``include/mea.h``; this package
is the thin Python binding.
"""
from .attention import (MemoryEfficientAttention, PackedQKVAttention, attention, attention_bwd,
                        attention_fwd, attention_packed, bwd_workspace_bytes, fwd_workspace_bytes)
from .nn import MultiheadAttention, TransformerBlock, TransformerLM

__all__ = ["attention", "attention_fwd", "attention_bwd", "attention_packed", "MemoryEfficientAttention",
           "PackedQKVAttention",
           "fwd_workspace_bytes", "bwd_workspace_bytes", "MultiheadAttention", "TransformerBlock",
           "TransformerLM"]
