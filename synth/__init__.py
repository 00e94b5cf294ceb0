"""Seeded synthetic inputs for the FlashForward renderer-attention path.

This module is shared by the CPU oracle's tests and by the GPU path's tests and
benchmark.  It holds the workload shapes and the random-number recipe only: no
step of the method (no RoPE, no attention, no cache bookkeeping) lives here.

Workloads
---------
The five workloads follow the paper's settings: Wan2.1-T2V backbones (1.3B:
12 heads x 128, 30 layers; 14B: 40 heads x 128, 40 layers), three-latent
renderer chunks (Sec. 3, notation paragraph: B_R = 3), S = 4 denoising stages,
and latent grids of 30x52 (480p) and 45x80 (720p).  The history ring holds W
chunks per (stage, layer), the paper's H (Sec. 3.1, Eq. step-update) with the
value each workload states.

Recipe
------
Every tensor is drawn as standard normal values from numpy's Philox
bit generator keyed by ``SeedSequence([seed, workload_id, a, b, c, tensor_id,
block])``: ``(a, b, c)`` is ``(chunk, stage, layer)`` for chunk tensors and
``(frame, 0, layer)`` for anchor frames, and ``block`` numbers consecutive runs
of ``ROWS_PER_BLOCK`` tokens so that blocks can be drawn in parallel.  Values
are drawn in float32, multiplied by the workload's ``input_scale`` and rounded
once (round-to-nearest-even, by torch) to the storage dtype.  The oracle then
upcasts these exact stored values to float64.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

ROWS_PER_BLOCK = 1024

# tensor ids of the recipe
T_Q, T_K, T_V, T_ANCHOR_K, T_ANCHOR_V = 0, 1, 2, 3, 4


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    wid: int                      # workload id used in the seed key
    dtype: str                    # "f32" or "bf16"
    heads: int
    head_dim: int
    grid_h: int
    grid_w: int
    frames_per_chunk: int         # B_R
    ring_chunks: int              # W
    stages: int                   # S
    layers: int
    n_chunks: int                 # chunks generated in sequence
    input_scale: float
    # which anchor frames each chunk reads, by name only (the rule itself is
    # the method's, not this module's): "none", "fixed:<f0>,<f1>,...",
    # "gamma:<delta>" (the window Gamma(i)) or "flank:<delta>" (the first
    # anchor and the two partition entries flanking the chunk)
    anchor_rule: str
    max_anchor_frames: int

    @property
    def tokens_per_frame(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def chunk_tokens(self) -> int:
        return self.frames_per_chunk * self.tokens_per_frame

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def rope_theta(self) -> float:
        return 10000.0

    @property
    def latent_frames(self) -> int:
        return self.n_chunks * self.frames_per_chunk


WORKLOADS: Dict[str, Workload] = {
    # tiny CPU-checkable case
    "tiny-f32": Workload("tiny-f32", 1, "f32", 2, 64, 8, 8, 3, 2, 4, 1, 6, 1.0,
                         "fixed:0,15", 2),
    # 1.3B-shaped, 480p
    "1.3b-480p": Workload("1.3b-480p", 2, "bf16", 12, 128, 30, 52, 3, 4, 4, 30, 27,
                          1.0 / math.sqrt(128.0), "gamma:10", 3),
    # 1.3B-shaped, 480p, long horizon (87 chunks = 261 latent frames)
    "1.3b-480p-long": Workload("1.3b-480p-long", 3, "bf16", 12, 128, 30, 52, 3, 4, 4, 30, 87,
                               1.0 / math.sqrt(128.0), "flank:24", 3),
    # 14B-shaped, 480p
    "14b-480p": Workload("14b-480p", 4, "bf16", 40, 128, 30, 52, 3, 4, 4, 40, 27, 1.0,
                         "gamma:10", 3),
    # 14B-shaped, 720p
    "14b-720p": Workload("14b-720p", 5, "bf16", 40, 128, 45, 80, 3, 4, 4, 40, 27, 1.0,
                         "gamma:10", 3),
}


def small_workload(name: str, *, dtype: str = "bf16", heads: int = 2, head_dim: int = 128,
                   grid_h: int = 6, grid_w: int = 11, ring_chunks: int = 2, stages: int = 2,
                   layers: int = 2, n_chunks: int = 5, input_scale: float = 1.0,
                   anchor_rule: str = "fixed:0,7", max_anchor_frames: int = 3,
                   frames_per_chunk: int = 3, wid: int = 100) -> Workload:
    """A reduced workload for tests that must also run the oracle in full."""
    return Workload(name, wid, dtype, heads, head_dim, grid_h, grid_w, frames_per_chunk,
                    ring_chunks, stages, layers, n_chunks, input_scale, anchor_rule,
                    max_anchor_frames)


def _block_values(seed_key: Sequence[int], n_rows: int, row_elems: int, block: int) -> np.ndarray:
    r0 = block * ROWS_PER_BLOCK
    r1 = min(n_rows, r0 + ROWS_PER_BLOCK)
    g = np.random.Generator(np.random.Philox(np.random.SeedSequence(list(seed_key) + [block])))
    return g.standard_normal((r1 - r0) * row_elems, dtype=np.float32)


def normal_rows(seed_key: Sequence[int], n_rows: int, row_elems: int, scale: float,
                dtype: torch.dtype) -> torch.Tensor:
    """[n_rows, row_elems] standard normal values (times ``scale``), stored in ``dtype``."""
    n_blocks = (n_rows + ROWS_PER_BLOCK - 1) // ROWS_PER_BLOCK
    out = np.empty(n_rows * row_elems, dtype=np.float32)
    workers = max(1, min(16, os.cpu_count() or 1, n_blocks))

    def fill(b: int) -> None:
        v = _block_values(seed_key, n_rows, row_elems, b)
        s = b * ROWS_PER_BLOCK * row_elems
        out[s:s + v.size] = v

    if workers == 1:
        for b in range(n_blocks):
            fill(b)
    else:
        with ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill, range(n_blocks)))
    if scale != 1.0:
        out *= np.float32(scale)
    t = torch.from_numpy(out.reshape(n_rows, row_elems))
    return t.to(dtype) if dtype != torch.float32 else t


def chunk_tensor(w: Workload, tensor_id: int, chunk: int, stage: int, layer: int,
                 seed: int = 0) -> torch.Tensor:
    """Q, K or V of one chunk at (stage, layer): [chunk_tokens, heads, head_dim]."""
    t = normal_rows([seed, w.wid, chunk, stage, layer, tensor_id], w.chunk_tokens,
                    w.heads * w.head_dim, w.input_scale, w.torch_dtype)
    return t.view(w.chunk_tokens, w.heads, w.head_dim)


def anchor_frame_tensor(w: Workload, tensor_id: int, frame: int, layer: int,
                        seed: int = 0) -> torch.Tensor:
    """Pre-RoPE anchor K (tensor_id 3) or V (4) of one latent frame: [G, heads, head_dim]."""
    t = normal_rows([seed, w.wid, frame, 0, layer, tensor_id], w.tokens_per_frame,
                    w.heads * w.head_dim, w.input_scale, w.torch_dtype)
    return t.view(w.tokens_per_frame, w.heads, w.head_dim)


def anchor_tensors(w: Workload, frames: Sequence[int], layer: int,
                   seed: int = 0) -> Tuple[torch.Tensor, torch.Tensor]:
    """Stacked pre-RoPE anchor K and V for ``frames``: [len(frames)*G, heads, head_dim]."""
    ks = [anchor_frame_tensor(w, T_ANCHOR_K, f, layer, seed) for f in frames]
    vs = [anchor_frame_tensor(w, T_ANCHOR_V, f, layer, seed) for f in frames]
    return torch.cat(ks, 0), torch.cat(vs, 0)
