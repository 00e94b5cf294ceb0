"""Shared helpers of the GPU parity tests: build the library's cache and the
oracle's cache for one workload, move seeded inputs, compare results."""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

import synth
from oracle import ff_oracle as fo
from paper_2609_32540_amd import ff

BF16_MAX_ABS = 2e-2
BF16_REL_L2 = 5e-3
F32_MAX_ABS = 1e-5
F32_REL_L2 = 1e-5


def anchor_frames(w: "synth.Workload", i: int) -> List[int]:
    """Anchor frames chunk i of workload w reads, by the oracle's reading of its rule."""
    return fo.anchor_frames(w.anchor_rule, i, w.frames_per_chunk, w.latent_frames)


def device() -> torch.device:
    return torch.device("cuda", 0)


def make_cache(w: synth.Workload, stages: Optional[int] = None, layers: Optional[int] = None,
               max_anchor_frames: Optional[int] = None, poison: bool = False) -> ff.RendererCache:
    c = ff.RendererCache(stages=stages or w.stages, layers=layers or w.layers,
                         ring_chunks=w.ring_chunks, frames_per_chunk=w.frames_per_chunk,
                         grid_h=w.grid_h, grid_w=w.grid_w, heads=w.heads, head_dim=w.head_dim,
                         max_anchor_frames=max_anchor_frames or w.max_anchor_frames,
                         dtype=w.torch_dtype, rope_theta=w.rope_theta, device=device())
    if poison:
        c.buffer.fill_(0xFF)   # NaN in bf16 and f32 alike
    return c


def make_oracle(w: synth.Workload, stages: Optional[int] = None,
                layers: Optional[int] = None) -> fo.RendererCacheOracle:
    return fo.RendererCacheOracle(stages=stages or w.stages, layers=layers or w.layers,
                                  W=w.ring_chunks)


def exact(t: torch.Tensor) -> np.ndarray:
    """Stored values as float32 numpy (exact for bf16 and f32)."""
    return t.detach().to("cpu").float().numpy()


def rel_l2(got: np.ndarray, ref: np.ndarray) -> float:
    return float(np.linalg.norm((got - ref).ravel()) / np.linalg.norm(ref.ravel()))


def check_attention(got: np.ndarray, ref: np.ndarray, dtype: str, what: str = "") -> Tuple[float, float]:
    err = np.abs(got.astype(np.float64) - ref)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    mx, rl = float(err.max()), rel_l2(got.astype(np.float64), ref)
    if dtype == "bf16":
        assert mx <= BF16_MAX_ABS and rl <= BF16_REL_L2, f"{what}: max-abs {mx:.3e}, rel-L2 {rl:.3e}"
    else:
        assert mx <= F32_MAX_ABS and rl <= F32_REL_L2, f"{what}: max-abs {mx:.3e}, rel-L2 {rl:.3e}"
    return mx, rl


def bf16_ordered(t: torch.Tensor) -> np.ndarray:
    """bf16 bit patterns mapped to integers that are consecutive for adjacent values."""
    b = t.detach().to("cpu").contiguous().view(torch.int16).numpy().astype(np.int32)
    mag = b & 0x7FFF
    return np.where(b < 0, -mag, mag)


def to_dev(t: torch.Tensor) -> torch.Tensor:
    return t.to(device())


def oracle_rope(w: synth.Workload, x: torch.Tensor, frames: Sequence[int]) -> np.ndarray:
    """Oracle RoPE of stored values, rounded to the storage dtype (float64 array)."""
    r = fo.rope3d(exact(x), frames, w.grid_h, w.grid_w, fo.rope_pair_split(w.head_dim), w.rope_theta)
    return fo.round_to(r, w.dtype)


class PairedRun:
    """Drives the library and the oracle through the same sequence of calls."""

    def __init__(self, w: synth.Workload, stages: Optional[int] = None,
                 layers: Optional[int] = None, rope: bool = True, poison: bool = False,
                 max_anchor_frames: Optional[int] = None):
        self.w = w
        self.stages = stages or w.stages
        self.layers = layers or w.layers
        self.rope = rope
        self.cache = make_cache(w, self.stages, self.layers, max_anchor_frames, poison)
        self.oracle = make_oracle(w, self.stages, self.layers)
        self.anchor_frames: Dict[int, List[int]] = {}
        self.results: List[Tuple[int, int, int, float, float]] = []

    def set_anchors(self, layer: int, frames: Sequence[int]) -> None:
        w = self.w
        if not frames:
            self.cache.anchor_set(layer, [], None, None)
            self.oracle.anchor_set(layer, [], np.zeros((0, w.heads, w.head_dim)),
                                   np.zeros((0, w.heads, w.head_dim)))
            self.anchor_frames[layer] = []
            return
        k, v = synth.anchor_tensors(w, frames, layer)
        kd, vd = to_dev(k), to_dev(v)
        if self.rope:
            self.cache.rope3d(None, kd, frames)
            k_ref = oracle_rope(w, k, frames)
        else:
            k_ref = exact(k)
        self.cache.anchor_set(layer, frames, kd, vd)
        self.oracle.anchor_set(layer, frames, k_ref, exact(v))
        self.anchor_frames[layer] = list(frames)

    def step(self, chunk: int, stage: int, layer: int, check: bool = True,
             rows: Optional[np.ndarray] = None, heads: Optional[Sequence[int]] = None,
             scale: Optional[float] = None) -> Optional[torch.Tensor]:
        """RoPE, attention, publish of one (chunk, stage, layer) on both sides."""
        w = self.w
        frames_a = anchor_frames(w, chunk)
        if self.anchor_frames.get(layer) != frames_a:
            self.set_anchors(layer, frames_a)
        q = synth.chunk_tensor(w, synth.T_Q, chunk, stage, layer)
        k = synth.chunk_tensor(w, synth.T_K, chunk, stage, layer)
        v = synth.chunk_tensor(w, synth.T_V, chunk, stage, layer)
        qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
        frames = fo.chunk_frames(chunk, w.frames_per_chunk)
        if self.rope:
            self.cache.rope3d(qd, kd, frames)
            # the oracle rotates Q only for a checked step (K always: it is published)
            q_ref = oracle_rope(w, q, frames) if check else None
            k_ref = oracle_rope(w, k, frames)
        else:
            q_ref, k_ref = exact(q), exact(k)
        v_ref = exact(v)
        out = self.cache.chunk_attention(stage, layer, chunk, qd, kd, vd, scale=scale)
        self.cache.kv_publish(stage, layer, chunk, kd, vd)
        if check:
            ref = self.oracle.attention(stage, layer, chunk, q_ref, k_ref, v_ref, scale=scale,
                                        heads=heads, rows=rows)
            got = exact(out)
            if rows is not None:
                got = got[rows]
            if heads is not None:
                got = got[:, list(heads)]
            mx, rl = check_attention(got, ref, w.dtype, f"chunk {chunk} stage {stage} layer {layer}")
            self.results.append((chunk, stage, layer, mx, rl))
        self.oracle.publish(stage, layer, chunk, k_ref, v_ref)
        return out
