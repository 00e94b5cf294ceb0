"""FlashForward per-stage renderer attention on MI355X (gfx950).

The compute path is the HIP library libff (paper_2609_32540_amd/csrc, C ABI in
include/ff.h); `paper_2609_32540_amd.ff` is its Python binding.
"""
from .ff import FFError, RendererCache, lib  # noqa: F401
