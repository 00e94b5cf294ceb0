"""Thin Python binding of libff (include/ff.h) over ctypes.

Argument marshalling only: every step runs in the HIP library.  PyTorch is
used for device memory (the cache buffer, tensors) and for the current HIP
stream.  The library must have been built (python -m paper_2609_32540_amd.build);
loading fails loudly otherwise.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import List, Optional, Sequence, Tuple

import torch

_PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG_DIR, "libff.so")

FF_OK = 0
STATUS_NAMES = {0: "FF_OK", 1: "FF_ERR_INVALID_ARG", 2: "FF_ERR_SHAPE", 3: "FF_ERR_ORDER",
                4: "FF_ERR_RANGE", 5: "FF_ERR_UNSUPPORTED", 6: "FF_ERR_HIP", 7: "FF_ERR_BUFFER"}
FF_DT_BF16, FF_DT_F32 = 0, 1
MAX_RING_CHUNKS = 8
MAX_ANCHOR_FRAMES = 8
MAX_ROPE_FRAMES = 16


class FFError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


class CacheDesc(ctypes.Structure):
    _fields_ = [
        ("num_stages", ctypes.c_int32), ("num_layers", ctypes.c_int32),
        ("ring_chunks", ctypes.c_int32), ("frames_per_chunk", ctypes.c_int32),
        ("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32),
        ("num_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("max_anchor_frames", ctypes.c_int32),
        ("rope_pairs_t", ctypes.c_int32), ("rope_pairs_h", ctypes.c_int32),
        ("rope_pairs_w", ctypes.c_int32),
        ("rope_theta", ctypes.c_double),
        ("dtype", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]


# (name, restype, argtypes) of every entry point of include/ff.h
_VP, _I32, _I64, _SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
_PI32, _PI64 = ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64)
SIGNATURES = [
    ("ff_abi_version", _I32, []),
    ("ff_cache_bytes", _SZ, [ctypes.POINTER(CacheDesc)]),
    ("ff_cache_create", _I32, [ctypes.POINTER(CacheDesc), _VP, _SZ, ctypes.POINTER(_VP)]),
    ("ff_cache_destroy", _I32, [_VP]),
    ("ff_rope3d", _I32, [_VP, _VP, _VP, _I32, _PI32, _VP]),
    ("ff_kv_publish", _I32, [_VP, _I32, _I32, _I64, _VP, _VP, _VP]),
    ("ff_anchor_set", _I32, [_VP, _I32, _I32, _PI32, _VP, _VP, _VP]),
    ("ff_chunk_attention", _I32, [_VP, _I32, _I32, _I64, _VP, _VP, _VP, _VP, ctypes.c_float, _VP]),
    ("ff_cache_ring_state", _I32, [_VP, _I32, _I32, _PI64, _PI64]),
    ("ff_cache_anchor_state", _I32, [_VP, _I32, _PI32, _PI32]),
    ("ff_cache_read", _I32, [_VP, _I32, _I32, _I32, _VP, _VP, _VP]),
    ("ff_status_string", ctypes.c_char_p, [_I32]),
    ("ff_last_error", ctypes.c_char_p, []),
]

_lib = None


def lib() -> ctypes.CDLL:
    """Load libff.so (built in-tree); raises if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_32540_amd.build` (the HIP path has no fallback)")
        L = ctypes.CDLL(LIB_PATH)
        for name, res, args in SIGNATURES:
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != FF_OK:
        raise FFError(status, lib().ff_last_error().decode())


def rope_pair_split(head_dim: int) -> Tuple[int, int, int]:
    n_hw = head_dim // 6
    return head_dim // 2 - 2 * n_hw, n_hw, n_hw


def _stream_handle(device: torch.device, stream: Optional[torch.cuda.Stream]) -> int:
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return s.cuda_stream


class RendererCache:
    """A FlashForward renderer cache (anchor segments + per-(stage, layer) history rings) on one GPU."""

    def __init__(self, *, stages: int, layers: int, ring_chunks: int, frames_per_chunk: int,
                 grid_h: int, grid_w: int, heads: int, head_dim: int, max_anchor_frames: int,
                 dtype: torch.dtype = torch.bfloat16, rope_theta: float = 10000.0,
                 rope_pairs: Optional[Tuple[int, int, int]] = None,
                 device: Optional[torch.device] = None):
        if dtype not in (torch.bfloat16, torch.float32):
            raise ValueError("dtype must be torch.bfloat16 or torch.float32")
        rp = rope_pairs if rope_pairs is not None else rope_pair_split(head_dim)
        self.desc = CacheDesc(stages, layers, ring_chunks, frames_per_chunk, grid_h, grid_w, heads,
                              head_dim, max_anchor_frames, rp[0], rp[1], rp[2], rope_theta,
                              FF_DT_BF16 if dtype == torch.bfloat16 else FF_DT_F32, 0)
        self.dtype = dtype
        self.device = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
        self.tokens_per_frame = grid_h * grid_w
        self.chunk_tokens = frames_per_chunk * self.tokens_per_frame
        self.heads, self.head_dim = heads, head_dim
        self.ring_chunks = ring_chunks
        L = lib()
        self.nbytes = L.ff_cache_bytes(ctypes.byref(self.desc))
        if self.nbytes == 0:
            raise FFError(1, L.ff_last_error().decode())
        self.buffer = torch.empty(self.nbytes, dtype=torch.uint8, device=self.device)
        h = ctypes.c_void_p()
        _check(L.ff_cache_create(ctypes.byref(self.desc), self.buffer.data_ptr(), self.nbytes,
                                 ctypes.byref(h)))
        self._h = h

    # ------------------------------------------------------------------
    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().ff_cache_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _tensor(self, t: torch.Tensor, n_tok: int, name: str) -> int:
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a torch.Tensor")
        if t.device != self.device:
            raise ValueError(f"{name} is on {t.device}, the cache is on {self.device}")
        if t.dtype != self.dtype:
            raise ValueError(f"{name} has dtype {t.dtype}, the cache uses {self.dtype}")
        if tuple(t.shape) != (n_tok, self.heads, self.head_dim):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected "
                             f"{(n_tok, self.heads, self.head_dim)}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        return t.data_ptr()

    # ------------------------------------------------------------------
    def rope3d(self, q: Optional[torch.Tensor], k: Optional[torch.Tensor], frame_t: Sequence[int],
               stream: Optional[torch.cuda.Stream] = None) -> None:
        n = len(frame_t)
        n_tok = n * self.tokens_per_frame
        qp = self._tensor(q, n_tok, "q") if q is not None else None
        kp = self._tensor(k, n_tok, "k") if k is not None else None
        ft = (ctypes.c_int32 * max(n, 1))(*frame_t)
        _check(lib().ff_rope3d(self._h, qp, kp, n, ft, _stream_handle(self.device, stream)))

    def kv_publish(self, stage: int, layer: int, chunk: int, k: torch.Tensor, v: torch.Tensor,
                   stream: Optional[torch.cuda.Stream] = None) -> None:
        kp = self._tensor(k, self.chunk_tokens, "k")
        vp = self._tensor(v, self.chunk_tokens, "v")
        _check(lib().ff_kv_publish(self._h, stage, layer, chunk, kp, vp,
                                   _stream_handle(self.device, stream)))

    def anchor_set(self, layer: int, frame_t: Sequence[int], k: Optional[torch.Tensor],
                   v: Optional[torch.Tensor], stream: Optional[torch.cuda.Stream] = None) -> None:
        n = len(frame_t)
        n_tok = n * self.tokens_per_frame
        kp = self._tensor(k, n_tok, "k") if n else None
        vp = self._tensor(v, n_tok, "v") if n else None
        ft = (ctypes.c_int32 * max(n, 1))(*frame_t)
        _check(lib().ff_anchor_set(self._h, layer, n, ft, kp, vp,
                                   _stream_handle(self.device, stream)))

    def chunk_attention(self, stage: int, layer: int, chunk: int, q: torch.Tensor,
                        k: torch.Tensor, v: torch.Tensor, out: Optional[torch.Tensor] = None,
                        scale: Optional[float] = None,
                        stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
        qp = self._tensor(q, self.chunk_tokens, "q")
        kp = self._tensor(k, self.chunk_tokens, "k")
        vp = self._tensor(v, self.chunk_tokens, "v")
        if out is None:
            out = torch.empty_like(q)
        op = self._tensor(out, self.chunk_tokens, "out")
        if scale is None:
            scale = 1.0 / math.sqrt(self.head_dim)
        _check(lib().ff_chunk_attention(self._h, stage, layer, chunk, qp, kp, vp, op,
                                        ctypes.c_float(scale), _stream_handle(self.device, stream)))
        return out

    # ------------------------------------------------------------------
    def ring_state(self, stage: int, layer: int) -> Tuple[List[int], int]:
        slots = (ctypes.c_int64 * self.ring_chunks)()
        count = ctypes.c_int64()
        _check(lib().ff_cache_ring_state(self._h, stage, layer, slots, ctypes.byref(count)))
        return list(slots), count.value

    def anchor_state(self, layer: int) -> List[int]:
        n = ctypes.c_int32()
        fr = (ctypes.c_int32 * MAX_ANCHOR_FRAMES)()
        _check(lib().ff_cache_anchor_state(self._h, layer, ctypes.byref(n), fr))
        return list(fr)[: n.value]

    def read(self, stage: int, layer: int, slot: int = 0,
             stream: Optional[torch.cuda.Stream] = None) -> Tuple[torch.Tensor, torch.Tensor]:
        """Cache contents in logical [tokens][heads][d] layout (stage -1: anchor segment)."""
        if stage == -1:
            n_tok = len(self.anchor_state(layer)) * self.tokens_per_frame
        else:
            n_tok = self.chunk_tokens
        k = torch.empty((n_tok, self.heads, self.head_dim), dtype=self.dtype, device=self.device)
        v = torch.empty_like(k)
        if n_tok:
            _check(lib().ff_cache_read(self._h, stage, layer, slot, k.data_ptr(), v.data_ptr(),
                                       _stream_handle(self.device, stream)))
        return k, v
