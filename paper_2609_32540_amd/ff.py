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
MAX_PACKED_CHUNKS = 128
MAX_BATCH = 4
ABI_VERSION = 4


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


class PackedDesc(ctypes.Structure):
    _fields_ = [
        ("n_chunks", ctypes.c_int32), ("chunk_tokens", ctypes.c_int32),
        ("num_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("window", ctypes.c_int32), ("frame_tokens", ctypes.c_int32),
        ("n_anchor_frames", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("anchors_of_chunk", ctypes.POINTER(ctypes.c_int32)),
    ]


class AttentionItem(ctypes.Structure):
    _fields_ = [
        ("stage", ctypes.c_int32), ("layer", ctypes.c_int32), ("chunk_index", ctypes.c_int64),
        ("q", ctypes.c_void_p), ("k_cur", ctypes.c_void_p), ("v_cur", ctypes.c_void_p),
        ("out", ctypes.c_void_p), ("bank_k", ctypes.c_void_p), ("bank_v", ctypes.c_void_p),
        ("n_frames", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("frame_index", ctypes.POINTER(ctypes.c_int32)),
    ]


# int32_t (*ff_stage_forward_fn)(void* user, int32_t stage, int64_t chunk, void* stream)
STAGE_FORWARD_FN = ctypes.CFUNCTYPE(ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                    ctypes.c_int64, ctypes.c_void_p)

# (name, restype, argtypes) of every entry point of include/ff.h
_VP, _I32, _I64, _SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
_PI32, _PI64 = ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int64)
SIGNATURES = [
    ("ff_abi_version", _I32, []),
    ("ff_cache_bytes", _SZ, [ctypes.POINTER(CacheDesc)]),
    ("ff_cache_create", _I32, [ctypes.POINTER(CacheDesc), _VP, _SZ, ctypes.POINTER(_VP)]),
    ("ff_cache_destroy", _I32, [_VP]),
    ("ff_cache_get_desc", _I32, [_VP, ctypes.POINTER(CacheDesc)]),
    ("ff_rope3d", _I32, [_VP, _VP, _VP, _I32, _PI32, _VP]),
    ("ff_kv_publish", _I32, [_VP, _I32, _I32, _I64, _VP, _VP, _VP]),
    ("ff_anchor_set", _I32, [_VP, _I32, _I32, _PI32, _VP, _VP, _VP]),
    ("ff_chunk_attention", _I32, [_VP, _I32, _I32, _I64, _VP, _VP, _VP, _VP, ctypes.c_float, _VP]),
    ("ff_chunk_attention_workspace_bytes", _SZ, [_VP]),
    ("ff_chunk_attention_ws", _I32, [_VP, _I32, _I32, _I64, _VP, _VP, _VP, _VP, ctypes.c_float,
                                     _VP, _SZ, _VP]),
    ("ff_chunk_attention_bank", _I32, [_VP, _I32, _I32, _I64, _VP, _VP, _VP, _VP, ctypes.c_float,
                                       _VP, _VP, _I32, _PI32, _VP]),
    ("ff_chunk_attention_batch", _I32, [_VP, _I32, ctypes.POINTER(AttentionItem), ctypes.c_float,
                                        _VP]),
    ("ff_cache_ring_state", _I32, [_VP, _I32, _I32, _PI64, _PI64, _PI64]),
    ("ff_cache_anchor_state", _I32, [_VP, _I32, _PI32, _PI32]),
    ("ff_cache_read", _I32, [_VP, _I32, _I32, _I32, _VP, _VP, _VP]),
    ("ff_packed_attention", _I32, [ctypes.POINTER(PackedDesc), _VP, _VP, _VP, _VP, _VP, _VP,
                                   ctypes.c_float, _VP, _VP]),
    ("ff_packed_attention_bwd_workspace", _SZ, [ctypes.POINTER(PackedDesc)]),
    ("ff_packed_attention_bwd", _I32, [ctypes.POINTER(PackedDesc), _VP, _VP, _VP, _VP, _VP, _VP,
                                       _VP, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_float, _VP,
                                       _SZ, _VP]),
    ("ff_packed_attention_bwd_static", _I32, [ctypes.POINTER(PackedDesc), _VP, _VP, _VP, _VP, _VP,
                                              _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP,
                                              ctypes.c_float, _VP]),
    ("ff_anchor_partition", _I32, [_I32, _I32, _PI32, _I32, _PI32]),
    ("ff_anchor_window", _I32, [_I64, _I32, _I32, _I32, _PI32, _PI32]),
    ("ff_anchor_flank", _I32, [_I64, _I32, _I32, _I32, _PI32, _PI32]),
    ("ff_euler_step", _I32, [_VP, _VP, _VP, _I64, ctypes.c_double, _I32, _VP]),
    ("ff_wavefront_run", _I32, [_I64, _I32, ctypes.POINTER(_VP), STAGE_FORWARD_FN, _VP, _PI64,
                                _PI64]),
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


def _stream_handle(device: torch.device, stream: Optional[torch.cuda.Stream]) -> int:
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return s.cuda_stream


def _empty_on(like: torch.Tensor, stream: Optional[torch.cuda.Stream],
              device: Optional[torch.device] = None) -> torch.Tensor:
    """A new tensor of like's shape and dtype (on `device`, default like's), allocated on
    the stream the library writes it on: the caching allocator then keeps its memory from
    being handed out again until that stream's work is done."""
    dev = device if device is not None else like.device
    if stream is None:
        return torch.empty(like.shape, dtype=like.dtype, device=dev)
    with torch.cuda.stream(stream):
        return torch.empty(like.shape, dtype=like.dtype, device=dev)


def _bytes_on(n: int, device: torch.device, stream: Optional[torch.cuda.Stream]) -> torch.Tensor:
    """n device bytes allocated on the stream that uses them (see _empty_on)."""
    if stream is None:
        return torch.empty(n, dtype=torch.uint8, device=device)
    with torch.cuda.stream(stream):
        return torch.empty(n, dtype=torch.uint8, device=device)


class RendererCache:
    """A FlashForward renderer cache (anchor segments + per-(stage, layer) history rings) on one GPU."""

    def __init__(self, *, stages: int, layers: int, ring_chunks: int, frames_per_chunk: int,
                 grid_h: int, grid_w: int, heads: int, head_dim: int, max_anchor_frames: int,
                 dtype: torch.dtype = torch.bfloat16, rope_theta: float = 10000.0,
                 rope_pairs: Optional[Tuple[int, int, int]] = None,
                 device: Optional[torch.device] = None):
        if dtype not in (torch.bfloat16, torch.float32):
            raise ValueError("dtype must be torch.bfloat16 or torch.float32")
        rp = rope_pairs if rope_pairs is not None else (0, 0, 0)   # (0, 0, 0): the library's default
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
        resolved = CacheDesc()
        _check(L.ff_cache_get_desc(h, ctypes.byref(resolved)))
        self.rope_pairs = (resolved.rope_pairs_t, resolved.rope_pairs_h, resolved.rope_pairs_w)

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
            out = _empty_on(q, stream)
        op = self._tensor(out, self.chunk_tokens, "out")
        if scale is None:
            scale = 1.0 / math.sqrt(self.head_dim)
        _check(lib().ff_chunk_attention(self._h, stage, layer, chunk, qp, kp, vp, op,
                                        ctypes.c_float(scale), _stream_handle(self.device, stream)))
        return out

    def workspace_bytes(self) -> int:
        """ff_chunk_attention_workspace_bytes: workspace of one ff_chunk_attention_ws call."""
        return lib().ff_chunk_attention_workspace_bytes(self._h)

    def chunk_attention_ws(self, stage: int, layer: int, chunk: int, q: torch.Tensor,
                           k: torch.Tensor, v: torch.Tensor, workspace: Optional[torch.Tensor],
                           out: Optional[torch.Tensor] = None, scale: Optional[float] = None,
                           stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
        """ff_chunk_attention_ws: the tail-split partials go to `workspace` (a uint8 device
        tensor, or None for an unsplit launch) instead of the cache's per-stage scratch."""
        qp = self._tensor(q, self.chunk_tokens, "q")
        kp = self._tensor(k, self.chunk_tokens, "k")
        vp = self._tensor(v, self.chunk_tokens, "v")
        if out is None:
            out = _empty_on(q, stream)
        op = self._tensor(out, self.chunk_tokens, "out")
        wp, wn = None, 0
        if workspace is not None:
            if workspace.device != self.device or not workspace.is_contiguous():
                raise ValueError("workspace must be a contiguous tensor on the cache's device")
            wp, wn = workspace.data_ptr(), workspace.numel() * workspace.element_size()
        if scale is None:
            scale = 1.0 / math.sqrt(self.head_dim)
        _check(lib().ff_chunk_attention_ws(self._h, stage, layer, chunk, qp, kp, vp, op,
                                           ctypes.c_float(scale), wp, wn,
                                           _stream_handle(self.device, stream)))
        return out

    def chunk_attention_bank(self, stage: int, layer: int, chunk: int, q: torch.Tensor,
                             k: torch.Tensor, v: torch.Tensor, bank_k: torch.Tensor,
                             bank_v: torch.Tensor, frames: Sequence[int],
                             out: Optional[torch.Tensor] = None, scale: Optional[float] = None,
                             stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
        """ff_chunk_attention_bank: anchors = bank frames `frames` (indices into the bank,
        a token-major [n_bank_frames * G][heads][d] array) instead of the anchor segment."""
        qp = self._tensor(q, self.chunk_tokens, "q")
        kp = self._tensor(k, self.chunk_tokens, "k")
        vp = self._tensor(v, self.chunk_tokens, "v")
        if out is None:
            out = _empty_on(q, stream)
        op = self._tensor(out, self.chunk_tokens, "out")
        if bank_k.shape[0] % self.tokens_per_frame:
            raise ValueError("the bank must hold whole frames")
        bk = self._tensor(bank_k, bank_k.shape[0], "bank_k")
        bv = self._tensor(bank_v, bank_k.shape[0], "bank_v")
        n_bank = bank_k.shape[0] // self.tokens_per_frame
        if any(not 0 <= f < n_bank for f in frames):
            raise ValueError(f"bank frame index out of range [0, {n_bank})")
        fr = (ctypes.c_int32 * max(len(frames), 1))(*frames)
        if scale is None:
            scale = 1.0 / math.sqrt(self.head_dim)
        _check(lib().ff_chunk_attention_bank(self._h, stage, layer, chunk, qp, kp, vp, op,
                                             ctypes.c_float(scale), bk, bv, len(frames), fr,
                                             _stream_handle(self.device, stream)))
        return out

    def chunk_attention_batch(self, items: Sequence[dict], scale: Optional[float] = None,
                              stream: Optional[torch.cuda.Stream] = None) -> List[torch.Tensor]:
        """ff_chunk_attention_batch: up to MAX_BATCH attention calls in one launch.  Each
        item is a dict with stage, layer, chunk, q, k, v and optionally out, and bank_k,
        bank_v, frames for the bank path; returns the outputs in item order."""
        if not 1 <= len(items) <= MAX_BATCH:
            raise ValueError(f"1 .. {MAX_BATCH} items per batch, got {len(items)}")
        arr = (AttentionItem * len(items))()
        outs, keep = [], []
        for j, it in enumerate(items):
            a = arr[j]
            a.stage, a.layer, a.chunk_index = it["stage"], it["layer"], it["chunk"]
            a.q = self._tensor(it["q"], self.chunk_tokens, "q")
            a.k_cur = self._tensor(it["k"], self.chunk_tokens, "k")
            a.v_cur = self._tensor(it["v"], self.chunk_tokens, "v")
            out = it.get("out")
            if out is None:
                out = _empty_on(it["q"], stream)
            a.out = self._tensor(out, self.chunk_tokens, "out")
            outs.append(out)
            if it.get("bank_k") is not None:
                bank_k, bank_v, frames = it["bank_k"], it["bank_v"], list(it["frames"])
                if bank_k.shape[0] % self.tokens_per_frame:
                    raise ValueError("the bank must hold whole frames")
                a.bank_k = self._tensor(bank_k, bank_k.shape[0], "bank_k")
                a.bank_v = self._tensor(bank_v, bank_k.shape[0], "bank_v")
                n_bank = bank_k.shape[0] // self.tokens_per_frame
                if any(not 0 <= f < n_bank for f in frames):
                    raise ValueError(f"bank frame index out of range [0, {n_bank})")
                fr = (ctypes.c_int32 * max(len(frames), 1))(*frames)
                keep.append(fr)
                a.n_frames = len(frames)
                a.frame_index = ctypes.cast(fr, ctypes.POINTER(ctypes.c_int32))
        if scale is None:
            scale = 1.0 / math.sqrt(self.head_dim)
        _check(lib().ff_chunk_attention_batch(self._h, len(items), arr, ctypes.c_float(scale),
                                              _stream_handle(self.device, stream)))
        return outs

    # ------------------------------------------------------------------
    def ring_state(self, stage: int, layer: int) -> Tuple[List[int], int]:
        """(slot table, number of chunks published into the ring so far)."""
        slots = (ctypes.c_int64 * self.ring_chunks)()
        count = ctypes.c_int64()
        _check(lib().ff_cache_ring_state(self._h, stage, layer, slots, None, ctypes.byref(count)))
        return list(slots), count.value

    def next_chunk(self, stage: int, layer: int) -> int:
        """The chunk the ring expects next (-1 before its first publish)."""
        nxt = ctypes.c_int64()
        _check(lib().ff_cache_ring_state(self._h, stage, layer, None, ctypes.byref(nxt), None))
        return nxt.value

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
        shape = torch.empty((n_tok, self.heads, self.head_dim), dtype=self.dtype, device="meta")
        k = _empty_on(shape, stream, self.device)
        v = _empty_on(shape, stream, self.device)
        if n_tok:
            _check(lib().ff_cache_read(self._h, stage, layer, slot, k.data_ptr(), v.data_ptr(),
                                       _stream_handle(self.device, stream)))
        return k, v


# ----------------------------------------------------------------------
def _dense(t: torch.Tensor, shape: Tuple[int, ...], dtype: torch.dtype, device: torch.device,
           name: str) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device != device or t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} on {device} (got {t.dtype} on {t.device})")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _packed_desc(q, n_chunks, window, anchor_k, anchor_v, frame_tokens, anchors_of_chunk):
    if q.dim() != 3 or q.shape[0] % n_chunks:
        raise ValueError("q must be [n_chunks * chunk_tokens][heads][d]")
    chunk_tokens = q.shape[0] // n_chunks
    heads, d = q.shape[1], q.shape[2]
    if q.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("dtype must be torch.bfloat16 or torch.float32")
    n_frames = 0
    akp = avp = None
    table = None
    if anchor_k is not None:
        if frame_tokens < 1 or anchor_k.shape[0] % frame_tokens:
            raise ValueError("anchor_k must hold whole frames of frame_tokens tokens")
        n_frames = anchor_k.shape[0] // frame_tokens
        a_shape = (n_frames * frame_tokens, heads, d)
        akp = _dense(anchor_k, a_shape, q.dtype, q.device, "anchor_k")
        avp = _dense(anchor_v, a_shape, q.dtype, q.device, "anchor_v")
        flat = [-1] * (n_chunks * MAX_ANCHOR_FRAMES)
        for i, frames in enumerate(anchors_of_chunk or []):
            if len(frames) > MAX_ANCHOR_FRAMES:
                raise ValueError(f"chunk {i} lists more than {MAX_ANCHOR_FRAMES} anchor frames")
            for j, f in enumerate(frames):
                flat[i * MAX_ANCHOR_FRAMES + j] = int(f)
        table = (ctypes.c_int32 * len(flat))(*flat)
    desc = PackedDesc(n_chunks, chunk_tokens, heads, d, window, frame_tokens, n_frames,
                      FF_DT_BF16 if q.dtype == torch.bfloat16 else FF_DT_F32,
                      ctypes.cast(table, ctypes.POINTER(ctypes.c_int32)) if table is not None else None)
    return desc, table, akp, avp, (n_chunks * chunk_tokens, heads, d), n_frames


def packed_attention(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, *, n_chunks: int,
                     window: int, anchor_k: Optional[torch.Tensor] = None,
                     anchor_v: Optional[torch.Tensor] = None, frame_tokens: int = 0,
                     anchors_of_chunk: Optional[Sequence[Sequence[int]]] = None,
                     out: Optional[torch.Tensor] = None, scale: Optional[float] = None,
                     lse: Optional[torch.Tensor] = None,
                     stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """ff_packed_attention: every chunk of one stage in one launch.

    q, k, v: [n_chunks * chunk_tokens][heads][d]; anchor_k / anchor_v:
    [n_frames * frame_tokens][heads][d]; anchors_of_chunk[i] lists the anchor
    frame indices chunk i sees.  lse (optional, float32 [tokens][heads])
    receives the base-2 log-sum-exp the backward pass needs.
    """
    desc, table, akp, avp, shape, _ = _packed_desc(q, n_chunks, window, anchor_k, anchor_v,
                                                   frame_tokens, anchors_of_chunk)
    dev, dt = q.device, q.dtype
    qp = _dense(q, shape, dt, dev, "q")
    kp = _dense(k, shape, dt, dev, "k")
    vp = _dense(v, shape, dt, dev, "v")
    if out is None:
        out = _empty_on(q, stream)
    op = _dense(out, shape, dt, dev, "out")
    lp = _dense(lse, shape[:2], torch.float32, dev, "lse") if lse is not None else None
    if scale is None:
        scale = 1.0 / math.sqrt(shape[2])
    _check(lib().ff_packed_attention(ctypes.byref(desc), qp, kp, vp, akp, avp, op,
                                     ctypes.c_float(scale), lp, _stream_handle(dev, stream)))
    return out


def packed_attention_bwd(q, k, v, out, dout, lse, *, n_chunks: int, window: int,
                         anchor_k=None, anchor_v=None, frame_tokens: int = 0,
                         anchors_of_chunk=None, scale: Optional[float] = None,
                         stream: Optional[torch.cuda.Stream] = None):
    """ff_packed_attention_bwd: returns (dq, dk, dv, d_anchor_k, d_anchor_v)."""
    desc, table, akp, avp, shape, n_frames = _packed_desc(q, n_chunks, window, anchor_k, anchor_v,
                                                          frame_tokens, anchors_of_chunk)
    dev, dt = q.device, q.dtype
    ptrs = [_dense(t, shape, dt, dev, n) for t, n in ((q, "q"), (k, "k"), (v, "v"), (out, "out"),
                                                      (dout, "dout"))]
    lp = _dense(lse, shape[:2], torch.float32, dev, "lse")
    dq, dk, dv = _empty_on(q, stream), _empty_on(k, stream), _empty_on(v, stream)
    dak = _empty_on(anchor_k, stream) if anchor_k is not None else None
    dav = _empty_on(anchor_v, stream) if anchor_v is not None else None
    ws_bytes = lib().ff_packed_attention_bwd_workspace(ctypes.byref(desc))
    ws = _bytes_on(max(ws_bytes, 16), dev, stream)
    if scale is None:
        scale = 1.0 / math.sqrt(shape[2])
    _check(lib().ff_packed_attention_bwd(
        ctypes.byref(desc), ptrs[0], ptrs[1], ptrs[2], akp, avp, ptrs[3], ptrs[4], lp,
        dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
        dak.data_ptr() if dak is not None else None, dav.data_ptr() if dav is not None else None,
        ctypes.c_float(scale), ws.data_ptr(), ws.numel(), _stream_handle(dev, stream)))
    return dq, dk, dv, dak, dav


def packed_attention_bwd_static(q, k, v, out, dout, lse, dq, dk, dv, d_anchor_k=None,
                                d_anchor_v=None, *, n_chunks: int, window: int, anchor_k=None,
                                anchor_v=None, frame_tokens: int = 0, anchors_of_chunk=None,
                                scale: Optional[float] = None,
                                stream: Optional[torch.cuda.Stream] = None) -> None:
    """ff_packed_attention_bwd_static: the backward into caller-provided gradients,
    its scratch in the library's static device array (this call allocates no
    device memory)."""
    desc, table, akp, avp, shape, n_frames = _packed_desc(q, n_chunks, window, anchor_k, anchor_v,
                                                          frame_tokens, anchors_of_chunk)
    dev, dt = q.device, q.dtype
    ptrs = [_dense(t, shape, dt, dev, n) for t, n in ((q, "q"), (k, "k"), (v, "v"), (out, "out"),
                                                      (dout, "dout"), (dq, "dq"), (dk, "dk"),
                                                      (dv, "dv"))]
    lp = _dense(lse, shape[:2], torch.float32, dev, "lse")
    dak = dav = None
    if anchor_k is not None:
        a_shape = tuple(anchor_k.shape)
        dak = _dense(d_anchor_k, a_shape, dt, dev, "d_anchor_k")
        dav = _dense(d_anchor_v, a_shape, dt, dev, "d_anchor_v")
    if scale is None:
        scale = 1.0 / math.sqrt(shape[2])
    _check(lib().ff_packed_attention_bwd_static(
        ctypes.byref(desc), ptrs[0], ptrs[1], ptrs[2], akp, avp, ptrs[3], ptrs[4], lp,
        ptrs[5], ptrs[6], ptrs[7], dak, dav, ctypes.c_float(scale), _stream_handle(dev, stream)))


def anchor_partition(L: int, delta: int) -> List[int]:
    """ff_anchor_partition: P = {m delta < L} u {L - 1}."""
    n = ctypes.c_int32()
    lib().ff_anchor_partition(L, delta, None, 0, ctypes.byref(n))   # size query
    if n.value <= 0:
        _check(lib().ff_anchor_partition(L, delta, None, 0, ctypes.byref(n)))
    buf = (ctypes.c_int32 * n.value)()
    _check(lib().ff_anchor_partition(L, delta, buf, n.value, ctypes.byref(n)))
    return list(buf)


def anchor_window(i: int, frames_per_chunk: int, delta: int, L: int) -> List[int]:
    """ff_anchor_window: Gamma(i)."""
    out = (ctypes.c_int32 * 3)()
    n = ctypes.c_int32()
    _check(lib().ff_anchor_window(i, frames_per_chunk, delta, L, out, ctypes.byref(n)))
    return list(out)[: n.value]


def anchor_flank(i: int, frames_per_chunk: int, delta: int, L: int) -> List[int]:
    """ff_anchor_flank: {P_0, P_m, P_m+1}, the first anchor and the two flanking chunk i."""
    out = (ctypes.c_int32 * 3)()
    n = ctypes.c_int32()
    _check(lib().ff_anchor_flank(i, frames_per_chunk, delta, L, out, ctypes.byref(n)))
    return list(out)[: n.value]


def anchor_frames(rule: str, i: int, frames_per_chunk: int, L: int) -> List[int]:
    """Anchor frames chunk i reads under a named rule, from the library's index
    sets: "none", "fixed:f0,f1,...", "gamma:<delta>" (ff_anchor_window) or
    "flank:<delta>" (ff_anchor_flank)."""
    if rule == "none":
        return []
    kind, _, arg = rule.partition(":")
    if kind == "fixed":
        return [int(v) for v in arg.split(",")]
    if kind == "gamma":
        return anchor_window(i, frames_per_chunk, int(arg), L)
    if kind == "flank":
        return anchor_flank(i, frames_per_chunk, int(arg), L)
    raise FFError(f"unknown anchor rule {rule!r}")


def euler_step(x: torch.Tensor, v: torch.Tensor, dsigma: float, out: Optional[torch.Tensor] = None,
               stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """ff_euler_step: out = x - dsigma * v (out may be x)."""
    if x.dtype not in (torch.bfloat16, torch.float32) or v.dtype != x.dtype:
        raise ValueError("x and v must both be bf16 or both float32")
    if x.shape != v.shape or not x.is_contiguous() or not v.is_contiguous():
        raise ValueError("x and v must be contiguous tensors of one shape")
    if out is None:
        out = _empty_on(x, stream)
    if out.shape != x.shape or out.dtype != x.dtype or not out.is_contiguous():
        raise ValueError("out must match x")
    _check(lib().ff_euler_step(x.data_ptr(), v.data_ptr(), out.data_ptr(), x.numel(),
                               ctypes.c_double(dsigma),
                               FF_DT_BF16 if x.dtype == torch.bfloat16 else FF_DT_F32,
                               _stream_handle(x.device, stream)))
    return out


def wavefront_run(n_chunks: int, streams: Sequence[torch.cuda.Stream], forward) -> Tuple[int, int]:
    """ff_wavefront_run: rank s = stage s on streams[s]; forward(stage, chunk, stream) enqueues
    one renderer forward on `stream` (a torch stream) and returns nothing.  Returns
    (rounds, forwards).  The caller synchronises the streams."""
    by_handle = {s.cuda_stream: s for s in streams}
    errors = []

    def cb(_user, stage, chunk, handle):
        try:
            forward(int(stage), int(chunk), by_handle[handle or 0])
            return FF_OK
        except Exception as e:  # stop the run, report after it returns
            errors.append(e)
            return 1

    fn = STAGE_FORWARD_FN(cb)
    arr = (ctypes.c_void_p * len(streams))(*[s.cuda_stream for s in streams])
    rounds, forwards = ctypes.c_int64(), ctypes.c_int64()
    st = lib().ff_wavefront_run(n_chunks, len(streams), arr, fn, None, ctypes.byref(rounds),
                                ctypes.byref(forwards))
    if errors:
        raise errors[0]
    _check(st)
    return rounds.value, forwards.value
