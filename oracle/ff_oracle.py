"""Plain float64 CPU oracle of FlashForward's per-stage renderer attention.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module; the product path (the HIP
library and its Python binding) never does, and this module imports nothing
from the product path.

What it computes, following the paper (arxiv 2609.32540):

* Chunk token layout (Sec. 3, notation paragraph): renderer chunk i holds the
  latent frames [B_R i, B_R i + B_R); a frame is a grid_h x grid_w token grid.
* 3D (t, h, w) rotary position embedding of Q and K.  The paper only names the
  Wan2.1 backbone (Sec. 4 setup) and does not define RoPE; the reading used
  here is the one of that backbone: adjacent element pairs (2p, 2p+1), pairs
  split into a t block, then an h block, then a w block of sizes
  (d/2 - 2 floor(d/6), floor(d/6), floor(d/6)), per-axis frequencies
  theta^(-j/n_axis) with theta = 10000, absolute positions.
* The stage-matched renderer history bank B_k (Sec. 3.1, Eq. step-update): an
  ordered list per (stage, layer); a publish appends the chunk's (i, K, V) and
  Tail_W keeps the W most recent entries.
* The clean anchor KV bank A_Gamma(i) (Sec. 3.1): per layer, shared by all
  stages, replaced by an anchor-set call.
* Renderer attention (Sec. 3.1 and the renderer row of the packed mask in
  the packed-SFT algorithm): each query of chunk i at stage k attends to the
  anchor frames, to the history entries of chunks max(0, i-W) .. i-1 at the
  same stage, and to every token of chunk i itself.  Softmax attention with
  scale 1/sqrt(d), in float64, with the visibility given by an explicit mask;
  keys that are not visible are removed before any arithmetic, so their
  contents (even NaN) cannot reach the result.
* The packed form of the same attention (Sec. 3.1, last paragraph, and the
  distillation appendix): all chunks of one stage in one masked attention,
  used by the tests as an independent formulation.
* Planner-side index sets: the anchor partition P (Eq. anchor-infill-
  partition), the block/chunk counts, the window Gamma(i) (Sec. 3 notation),
  the long-horizon anchor set (the first anchor and the two entries of P that
  flank a chunk) and the forward-count model (Eq. forward-count).

Everything is float64 numpy; matrix products use numpy's matmul.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


# --------------------------------------------------------------------------
# Rounding to the storage dtypes
# --------------------------------------------------------------------------

def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value, ties to even.

    bfloat16 keeps 8 significant bits and the float32 exponent range.  Writing
    x = m * 2**e with 0.5 <= |m| < 1 (frexp), the spacing of bfloat16 values
    around x is 2**(e - 8) (never below the subnormal spacing 2**-133), and
    numpy's rint rounds half to even.  Values beyond the largest finite
    bfloat16 become infinities.  The returned float64 values are exactly
    representable in bfloat16.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.array(x, copy=True)
    finite = np.isfinite(x) & (x != 0)
    m, e = np.frexp(x[finite])
    spacing_exp = np.maximum(e - 8, -133)
    q = np.rint(np.ldexp(x[finite], -spacing_exp))
    r = np.ldexp(q, spacing_exp)
    max_bf16 = (2.0 - 2.0 ** -7) * 2.0 ** 127
    # values that round past the largest finite bfloat16 overflow
    r = np.where(np.abs(r) > max_bf16, np.copysign(np.inf, r), r)
    out[finite] = r
    return out


def round_to_f32(x: np.ndarray) -> np.ndarray:
    """Round float64 values to float32 (round to nearest even) and back."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_to_bf16(x)
    if dtype == "f32":
        return round_to_f32(x)
    raise ValueError(dtype)


# --------------------------------------------------------------------------
# (a1) chunk token layout and 3D positions
# --------------------------------------------------------------------------

def chunk_frames(i: int, frames_per_chunk: int) -> List[int]:
    """Latent frames of renderer chunk i (Sec. 3 notation: chunks of B_R latents)."""
    return list(range(frames_per_chunk * i, frames_per_chunk * (i + 1)))


def token_positions(frame_t: Sequence[int], grid_h: int, grid_w: int
                    ) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """(t, y, x) of every token of a run of frames, tokens row-major in (frame, row, col)."""
    G = grid_h * grid_w
    n = np.arange(len(frame_t) * G)
    t = np.asarray(frame_t, dtype=np.int64)[n // G]
    y = (n % G) // grid_w
    x = n % grid_w
    return t, y, x


# --------------------------------------------------------------------------
# (a2) 3D RoPE
# --------------------------------------------------------------------------

def rope_pair_split(head_dim: int) -> Tuple[int, int, int]:
    """Number of rotation pairs given to the t, h and w axes."""
    n_hw = head_dim // 6
    return head_dim // 2 - 2 * n_hw, n_hw, n_hw


def rope_angles(t: np.ndarray, y: np.ndarray, x: np.ndarray,
                split: Tuple[int, int, int], theta: float) -> np.ndarray:
    """Rotation angle of every (token, pair): [n_tokens, n_t + n_h + n_w]."""
    cols = []
    for pos, n_axis in ((t, split[0]), (y, split[1]), (x, split[2])):
        j = np.arange(n_axis, dtype=np.float64)
        omega = theta ** (-j / n_axis)
        cols.append(np.asarray(pos, dtype=np.float64)[:, None] * omega[None, :])
    return np.concatenate(cols, axis=1)


def rope3d(X: np.ndarray, frame_t: Sequence[int], grid_h: int, grid_w: int,
           split: Tuple[int, int, int], theta: float = 10000.0) -> np.ndarray:
    """Rotate X [n_tokens, heads, d] (float64) at the positions of ``frame_t``.

    Pair p holds elements (2p, 2p+1); with angle phi the pair (a, b) becomes
    (a cos phi - b sin phi, a sin phi + b cos phi).
    """
    X = np.asarray(X, dtype=np.float64)
    n_tok, heads, d = X.shape
    assert n_tok == len(frame_t) * grid_h * grid_w
    assert sum(split) == d // 2
    t, y, x = token_positions(frame_t, grid_h, grid_w)
    phi = rope_angles(t, y, x, split, theta)[:, None, :]   # [n_tok, 1, d/2]
    a = X[:, :, 0::2]
    b = X[:, :, 1::2]
    out = np.empty_like(X)
    out[:, :, 0::2] = a * np.cos(phi) - b * np.sin(phi)
    out[:, :, 1::2] = a * np.sin(phi) + b * np.cos(phi)
    return out


# --------------------------------------------------------------------------
# (a5) attention over an explicit visibility mask
# --------------------------------------------------------------------------

def attend(Qh: np.ndarray, Kh: np.ndarray, Vh: np.ndarray, scale: float) -> np.ndarray:
    """softmax(scale * Qh Kh^T) Vh for one head, in float64: Qh [nq, d], Kh, Vh [nk, d]."""
    s = scale * (np.asarray(Qh, np.float64) @ np.asarray(Kh, np.float64).T)   # [nq, nk]
    m = s.max(axis=1, keepdims=True)
    p = np.exp(s - m)
    return (p @ np.asarray(Vh, np.float64)) / p.sum(axis=1, keepdims=True)


def masked_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, visible: np.ndarray,
                     scale: float, heads: Optional[Sequence[int]] = None,
                     rows: Optional[np.ndarray] = None) -> np.ndarray:
    """softmax(scale * Q K^T) V per head over the visible keys only.

    Q [nq, h, d]; K, V [nk, h, d]; visible: bool [nk].  Keys that are not
    visible are dropped before any arithmetic.  Returns float64
    [len(rows), len(heads), d] (all rows / heads when not given).
    """
    visible = np.asarray(visible, dtype=bool)
    if heads is None:
        heads = range(Q.shape[1])
    if rows is None:
        rows = np.arange(Q.shape[0])
    heads = list(heads)
    out = np.empty((len(rows), len(heads), Q.shape[2]), dtype=np.float64)
    for hi, h in enumerate(heads):
        out[:, hi, :] = attend(Q[rows, h, :], K[visible, h, :], V[visible, h, :], scale)
    return out


# --------------------------------------------------------------------------
# (a3, a4) history bank, anchor bank and one renderer step
# --------------------------------------------------------------------------

@dataclass
class HistoryEntry:
    chunk: int
    K: np.ndarray
    V: np.ndarray


class OrderError(RuntimeError):
    pass


@dataclass
class RendererCacheOracle:
    """Anchor bank per layer and one Tail_W history list per (stage, layer)."""
    stages: int
    layers: int
    W: int
    history: Dict[Tuple[int, int], List[HistoryEntry]] = field(default_factory=dict)
    next_chunk: Dict[Tuple[int, int], int] = field(default_factory=dict)
    n_published: Dict[Tuple[int, int], int] = field(default_factory=dict)
    anchors: Dict[int, Tuple[List[int], np.ndarray, np.ndarray]] = field(default_factory=dict)

    def _key(self, stage: int, layer: int) -> Tuple[int, int]:
        if not (0 <= stage < self.stages and 0 <= layer < self.layers):
            raise IndexError((stage, layer))
        return stage, layer

    def anchor_set(self, layer: int, frames: Sequence[int], K: np.ndarray, V: np.ndarray) -> None:
        """Replace layer ``layer``'s anchor segment (already-rotated K, and V)."""
        if not 0 <= layer < self.layers:
            raise IndexError(layer)
        self.anchors[layer] = (list(frames), np.array(K), np.array(V))

    def publish(self, stage: int, layer: int, i: int, K: np.ndarray, V: np.ndarray) -> None:
        """Eq. step-update: B <- Tail_W(B u (i, K, V)); chunks arrive in order."""
        key = self._key(stage, layer)
        expected = self.next_chunk.get(key)
        if expected is not None and i != expected:
            raise OrderError(f"publish chunk {i}, expected {expected}")
        lst = self.history.setdefault(key, [])
        lst.append(HistoryEntry(i, np.array(K), np.array(V)))
        while len(lst) > self.W:
            lst.pop(0)
        self.next_chunk[key] = i + 1
        self.n_published[key] = self.n_published.get(key, 0) + 1

    def ring_state(self, stage: int, layer: int) -> Tuple[List[int], int]:
        """Slot table (slot c mod W holds chunk c, -1 when empty) and the number
        of chunks published into the ring so far."""
        key = self._key(stage, layer)
        table = [-1] * self.W
        for e in self.history.get(key, []):
            table[e.chunk % self.W] = e.chunk
        return table, self.n_published.get(key, 0)

    def expected_chunk(self, stage: int, layer: int) -> int:
        """The chunk the ring expects next (-1 before the first publish)."""
        n = self.next_chunk.get(self._key(stage, layer))
        return -1 if n is None else n

    def history_concat(self, stage: int, layer: int) -> Tuple[np.ndarray, np.ndarray, List[int]]:
        lst = self.history.get(self._key(stage, layer), [])
        if not lst:
            return None, None, []
        return (np.concatenate([e.K for e in lst], 0), np.concatenate([e.V for e in lst], 0),
                [e.chunk for e in lst])

    def read_set(self, stage: int, layer: int, i: int, K_cur: np.ndarray, V_cur: np.ndarray
                 ) -> Tuple[List[np.ndarray], List[np.ndarray], List[bool]]:
        """Key segments [anchors | history entries | current] and their visibility.

        Anchors: every frame of the layer's anchor segment.  History: entries
        whose chunk lies in [max(0, i-W), i-1] (same stage).  Current chunk:
        all of its tokens (bidirectional inside the chunk).
        """
        key = self._key(stage, layer)
        Ks, Vs, vis = [], [], []
        if layer in self.anchors:
            _, Ka, Va = self.anchors[layer]
            Ks.append(Ka); Vs.append(Va); vis.append(True)
        for e in self.history.get(key, []):
            Ks.append(e.K); Vs.append(e.V)
            vis.append(max(0, i - self.W) <= e.chunk <= i - 1)
        Ks.append(np.asarray(K_cur)); Vs.append(np.asarray(V_cur)); vis.append(True)
        return Ks, Vs, vis

    def attention(self, stage: int, layer: int, i: int, Q: np.ndarray, K_cur: np.ndarray,
                  V_cur: np.ndarray, scale: Optional[float] = None,
                  heads: Optional[Sequence[int]] = None,
                  rows: Optional[np.ndarray] = None) -> np.ndarray:
        """Renderer attention of chunk i at (stage, layer); the caller publishes afterwards."""
        key = self._key(stage, layer)
        expected = self.next_chunk.get(key)
        if expected is not None and i != expected:
            raise OrderError(f"attention for chunk {i}, history expects {expected}")
        if scale is None:
            scale = 1.0 / math.sqrt(Q.shape[2])
        Ks, Vs, vis = self.read_set(stage, layer, i, K_cur, V_cur)
        if heads is None:
            heads = range(Q.shape[1])
        if rows is None:
            rows = np.arange(Q.shape[0])
        heads = list(heads)
        out = np.empty((len(rows), len(heads), Q.shape[2]), dtype=np.float64)
        for hi, h in enumerate(heads):
            Kh = np.concatenate([k[:, h, :] for k, v_ in zip(Ks, vis) if v_], 0)
            Vh = np.concatenate([v[:, h, :] for v, v_ in zip(Vs, vis) if v_], 0)
            out[:, hi, :] = attend(Q[rows, h, :], Kh, Vh, scale)
        return out


# --------------------------------------------------------------------------
# Packed block-causal form (all chunks of one stage in one call)
# --------------------------------------------------------------------------

def packed_stage_attention(Qs: Sequence[np.ndarray], Ks: Sequence[np.ndarray],
                           Vs: Sequence[np.ndarray],
                           anchor_frames: Dict[int, Tuple[np.ndarray, np.ndarray]],
                           anchors_of_chunk: Sequence[Sequence[int]], W: int,
                           scale: float) -> List[np.ndarray]:
    """One masked attention over the packed sequence [anchor frames | chunk 0 | chunk 1 | ...].

    The mask gives chunk i's queries its own tokens, the tokens of chunks
    max(0, i-W) .. i-1 and the anchor frames listed for chunk i: the renderer
    row of the packed training mask with the history length H set to W.
    Masked logits are set to -inf before a plain softmax.
    """
    frames = sorted(anchor_frames)
    a_K = [anchor_frames[f][0] for f in frames]
    a_V = [anchor_frames[f][1] for f in frames]
    K_all = np.concatenate(a_K + list(Ks), 0)
    V_all = np.concatenate(a_V + list(Vs), 0)
    G_a = [anchor_frames[f][0].shape[0] for f in frames]
    a_start = np.cumsum([0] + G_a)
    n_anchor = a_start[-1]
    c_len = [q.shape[0] for q in Qs]
    c_start = n_anchor + np.cumsum([0] + c_len)
    outs = []
    for i, Q in enumerate(Qs):
        mask = np.zeros(K_all.shape[0], bool)
        for f in anchors_of_chunk[i]:
            fi = frames.index(f)
            mask[a_start[fi]:a_start[fi + 1]] = True
        for q in range(max(0, i - W), i + 1):
            mask[c_start[q]:c_start[q + 1]] = True
        heads = Q.shape[1]
        o = np.empty_like(np.asarray(Q, dtype=np.float64))
        for h in range(heads):
            s = scale * (np.asarray(Q[:, h, :], np.float64) @ K_all[:, h, :].T)
            s = np.where(mask[None, :], s, -np.inf)
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p = p / p.sum(axis=1, keepdims=True)
            o[:, h, :] = p @ np.where(mask[:, None], V_all[:, h, :], 0.0)
        outs.append(o)
    return outs


def packed_visibility(n_chunks: int, chunk_tokens: int, frame_tokens: int, n_frames: int,
                      anchors_of_chunk: Sequence[Sequence[int]], W: int) -> np.ndarray:
    """Boolean mask [n_chunks*chunk_tokens, n_frames*frame_tokens + n_chunks*chunk_tokens]
    of the packed sequence [anchor frames | chunk 0 | chunk 1 | ...]: the renderer
    rows of the packed training mask (chunk i sees chunks max(0, i-W) .. i and its
    listed anchor frames)."""
    n_anchor = n_frames * frame_tokens
    M = np.zeros((n_chunks * chunk_tokens, n_anchor + n_chunks * chunk_tokens), bool)
    for i in range(n_chunks):
        rows = slice(i * chunk_tokens, (i + 1) * chunk_tokens)
        for f in anchors_of_chunk[i]:
            M[rows, f * frame_tokens:(f + 1) * frame_tokens] = True
        M[rows, n_anchor + max(0, i - W) * chunk_tokens:n_anchor + (i + 1) * chunk_tokens] = True
    return M


def masked_attention_grad(Q: np.ndarray, K: np.ndarray, V: np.ndarray, visible: np.ndarray,
                          dO: np.ndarray, scale: float):
    """Gradients of O = softmax(scale Q K^T, masked) V with respect to Q, K, V, per head,
    in float64, from the definitions: P = softmax, dV = P^T dO, dP = dO V^T,
    dS = P * (dP - rowsum(dP * P)), dQ = scale dS K, dK = scale dS^T Q.
    Q [n][h][d], K, V [m][h][d], visible [n][m] bool, dO [n][h][d]."""
    Q, K, V, dO = (np.asarray(a, np.float64) for a in (Q, K, V, dO))
    dQ, dK, dV = np.zeros_like(Q), np.zeros_like(K), np.zeros_like(V)
    for h in range(Q.shape[1]):
        s = scale * (Q[:, h] @ K[:, h].T)
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        P = np.exp(s)
        P = P / P.sum(axis=1, keepdims=True)
        dV[:, h] = P.T @ dO[:, h]
        dP = dO[:, h] @ V[:, h].T
        dS = P * (dP - (dP * P).sum(axis=1, keepdims=True))
        dQ[:, h] = scale * (dS @ K[:, h])
        dK[:, h] = scale * (dS.T @ Q[:, h])
    return dQ, dK, dV


def log2_sum_exp2(Q: np.ndarray, K: np.ndarray, visible: np.ndarray, scale: float) -> np.ndarray:
    """Per query and head, log2 of sum_j 2^(scale log2(e) q.k_j) over visible keys
    (the forward's base-2 log-sum-exp): [n][h]."""
    Q, K = np.asarray(Q, np.float64), np.asarray(K, np.float64)
    out = np.empty((Q.shape[0], Q.shape[1]))
    for h in range(Q.shape[1]):
        s = (scale * np.log2(np.e)) * (Q[:, h] @ K[:, h].T)
        s = np.where(visible, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        out[:, h] = (m + np.log2(np.exp2(s - m).sum(axis=1, keepdims=True)))[:, 0]
    return out


# --------------------------------------------------------------------------
# Sampler step and the wavefront schedule
# --------------------------------------------------------------------------

def euler_step(x: np.ndarray, v: np.ndarray, dsigma: float, dtype: str) -> np.ndarray:
    """Euler step of the rectified-flow sampler (wavefront algorithm, Step):
    x_{k-1} = x_k - (sigma_k - sigma_{k-1}) v, in float64 (product rounded,
    then the difference), rounded once to the storage dtype ("f64": not rounded)."""
    x64 = np.asarray(x, np.float64)
    prod = np.float64(dsigma) * np.asarray(v, np.float64)
    return x64 - prod if dtype == "f64" else round_to(x64 - prod, dtype)


def wavefront_schedule(n_chunks: int, n_stages: int) -> List[List[Tuple[int, int]]]:
    """Phase B of the wavefront algorithm: round n runs rank r on chunk i = n - r
    (stage k = S - r) when 0 <= i < N_R; N_R + S - 1 rounds.  Returns, per
    round, the active (rank, chunk) pairs."""
    rounds = []
    for n in range(n_chunks + n_stages - 1):
        rounds.append([(r, n - r) for r in range(n_stages) if 0 <= n - r < n_chunks])
    return rounds


# --------------------------------------------------------------------------
# Planner-side index sets and the forward-count model
# --------------------------------------------------------------------------

def anchor_partition(L: int, delta: int) -> List[int]:
    """Eq. anchor-infill-partition: P = {m delta < L} u {L-1}."""
    return sorted({m * delta for m in range((L - 1) // delta + 1)} | {L - 1})


def num_blocks(n: int, block: int) -> int:
    return -(-n // block)


def anchor_window(i: int, B_R: int, delta: int, L: int) -> List[int]:
    """Gamma(i) of Sec. 3 notation; indices past L-1 are replaced by L-1 (boundary side)."""
    u = (B_R * i) // (2 * delta)
    return sorted({min(v, L - 1) for v in (2 * u * delta, (2 * u + 1) * delta, (2 * u + 2) * delta)})


def anchor_flank(i: int, B_R: int, delta: int, L: int) -> List[int]:
    """Long-horizon anchor set of chunk i: the first anchor of P (Eq. anchor-
    infill-partition, spacing delta) and the two entries of P that flank the
    chunk's first latent B_R i, i.e. P_m and P_{m+1} with m = floor(B_R i / delta);
    entries past the end of P are the last entry, the boundary anchor L-1."""
    P = anchor_partition(L, delta)
    m = (B_R * i) // delta

    def at(j: int) -> int:
        return P[min(j, len(P) - 1)]

    return sorted({P[0], at(m), at(m + 1)})


def anchor_frames(rule: str, i: int, B_R: int, L: int) -> List[int]:
    """Anchor frames visible to chunk i under a workload's anchor rule:
    "none"; "fixed:f0,f1,..." (the same frames for every chunk);
    "gamma:<delta>" (Gamma(i) of Sec. 3 notation); "flank:<delta>" (anchor_flank)."""
    if rule == "none":
        return []
    kind, _, arg = rule.partition(":")
    if kind == "fixed":
        return [int(v) for v in arg.split(",")]
    if kind == "gamma":
        return anchor_window(i, B_R, int(arg), L)
    if kind == "flank":
        return anchor_flank(i, B_R, int(arg), L)
    raise ValueError(f"unknown anchor rule {rule!r}")


def forward_counts(L: int, delta: int, B: int, S: int) -> Tuple[int, int, int]:
    """Eq. forward-count: logical forwards of FlashForward, Self-Forcing and HiAR."""
    M = len(anchor_partition(L, delta))
    N_P = num_blocks(M, B)
    N_R = N_C = num_blocks(L, B)
    return N_P * (S + 1) + N_R * S, N_C * S + (N_C - 1), N_C * S + (N_C - 1) * S


def history_lengths(W_ctx: int, B_P: int, B_R: int) -> Tuple[int, int]:
    """(H, H_P) from the context budget (wavefront algorithm constants)."""
    return (W_ctx - B_P - B_R) // B_R, (W_ctx - B_P) // B_P
