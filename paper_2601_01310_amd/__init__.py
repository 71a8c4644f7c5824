"""Tarragon expert-worker forward on MI355X (gfx950).

The expert-worker (EW) side of Tarragon (arXiv 2601.01310) computes, for one
batch of token embeddings and one MoE layer: top-k gating, the logical-expert
to physical-slot remap through the expert routing table (ERT) that masks
failed slots (§4.2, §5.1, §5.3), the per-slot token permutation, the SwiGLU
expert FFN and the gate-weighted combine (§2.1).

The compute runs in hand-written HIP kernels behind the C-ABI library
``libtg.so`` (declared in ``include/tg.h``); :mod:`.tg` is its ctypes binding.
"""

__all__ = ["tg", "synth"]
