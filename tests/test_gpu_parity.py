"""GPU parity of the HIP path (through the C ABI) against the float64 oracle.

Bars: cache contents and ring indices bit-exact; RoPE within 1 bf16 ulp of
the rounded float64 result, differing only where the two float64 evaluations
straddle a rounding tie (float32 tensors: 1e-5); bf16 attention within
max-abs 2e-2 and relative-L2 5e-3 of float64 per call; float32 attention
within 1e-5.
"""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import ff_oracle as fo
from paper_2609_32540_amd import ff

from gpu_util import (PairedRun, bf16_ordered, check_attention, exact, make_cache, make_oracle,
                      oracle_rope, to_dev)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _needs_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ff.lib()


def small(dtype="bf16", head_dim=128, **kw):
    base = dict(dtype=dtype, heads=2, head_dim=head_dim, grid_h=6, grid_w=11, ring_chunks=2,
                stages=2, layers=2, n_chunks=5, anchor_rule="fixed:0,7", max_anchor_frames=3)
    base.update(kw)
    return synth.small_workload("small", **base)


# --------------------------------------------------------------------------
# (a3, a4) publish, anchor set: bit-exact contents and indices
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,head_dim", [("bf16", 128), ("bf16", 64), ("f32", 64), ("f32", 128)])
def test_publish_and_anchor_set_bitexact(dtype, head_dim):
    w = small(dtype, head_dim, heads=3, grid_h=5, grid_w=7, ring_chunks=3)
    cache, orc = make_cache(w, 2, 2), make_oracle(w, 2, 2)
    plan = [(0, 1, c) for c in range(8)] + [(1, 0, c) for c in range(2, 7)]
    plan = [plan[i] for i in np.random.default_rng(0).permutation(len(plan))]
    plan.sort(key=lambda t: (t[0], t[1], t[2]))   # per-ring order kept
    for s, l, c in plan:
        k = synth.chunk_tensor(w, synth.T_K, c, s, l)
        v = synth.chunk_tensor(w, synth.T_V, c, s, l)
        cache.kv_publish(s, l, c, to_dev(k), to_dev(v))
        orc.publish(s, l, c, exact(k), exact(v))
        assert cache.ring_state(s, l) == orc.ring_state(s, l)
    for s in range(2):
        for l in range(2):
            table, _ = orc.ring_state(s, l)
            assert cache.ring_state(s, l)[0] == table
            entries = {e.chunk: e for e in orc.history.get((s, l), [])}
            for slot, c in enumerate(table):
                if c < 0:
                    continue
                kg, vg = cache.read(s, l, slot)
                np.testing.assert_array_equal(exact(kg), entries[c].K)
                np.testing.assert_array_equal(exact(vg), entries[c].V)
    # anchors: set, then replace with a different frame count
    for frames in ([0, 10, 20], [5]):
        k, v = synth.anchor_tensors(w, frames, 1)
        cache.anchor_set(1, frames, to_dev(k), to_dev(v))
        assert cache.anchor_state(1) == frames
        kg, vg = cache.read(-1, 1)
        assert torch.equal(kg.cpu(), k) and torch.equal(vg.cpu(), v)
    assert cache.anchor_state(0) == []


def test_ring_wraparound_long_sequence_bitexact():
    # 87 chunks through a W=4 ring (the long-horizon chunk count)
    w = small("bf16", 64, heads=1, grid_h=2, grid_w=4, ring_chunks=4)
    cache, orc = make_cache(w, 1, 1), make_oracle(w, 1, 1)
    for c in range(87):
        k = synth.chunk_tensor(w, synth.T_K, c, 0, 0)
        v = synth.chunk_tensor(w, synth.T_V, c, 0, 0)
        cache.kv_publish(0, 0, c, to_dev(k), to_dev(v))
        orc.publish(0, 0, c, exact(k), exact(v))
        assert cache.ring_state(0, 0) == orc.ring_state(0, 0)
    Kc, Vc, chunks = orc.history_concat(0, 0)
    assert chunks == [83, 84, 85, 86]
    got_k = np.concatenate([exact(cache.read(0, 0, c % 4)[0]) for c in chunks])
    got_v = np.concatenate([exact(cache.read(0, 0, c % 4)[1]) for c in chunks])
    np.testing.assert_array_equal(got_k, Kc)
    np.testing.assert_array_equal(got_v, Vc)


def test_order_errors_leave_state_unchanged():
    w = small("bf16", 128)
    cache = make_cache(w, 1, 1)
    k = to_dev(synth.chunk_tensor(w, synth.T_K, 0, 0, 0))
    cache.kv_publish(0, 0, 3, k, k)
    before = cache.ring_state(0, 0)
    with pytest.raises(ff.FFError) as e:
        cache.kv_publish(0, 0, 5, k, k)
    assert e.value.status == 3
    with pytest.raises(ff.FFError) as e:
        cache.chunk_attention(0, 0, 3, k, k, k)
    assert e.value.status == 3
    with pytest.raises(ValueError):
        cache.kv_publish(0, 0, 4, k[:-1], k[:-1])
    assert cache.ring_state(0, 0) == before
    cache.kv_publish(0, 0, 4, k, k)
    # two chunks published (the first at chunk 3), chunk 5 expected next
    assert cache.ring_state(0, 0) == ([4, 3], 2)
    assert cache.next_chunk(0, 0) == 5


# --------------------------------------------------------------------------
# (a2) RoPE
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,head_dim,grid,heads", [
    ("bf16", 128, (30, 52), 12), ("bf16", 128, (45, 80), 40), ("bf16", 64, (8, 8), 2),
    ("f32", 64, (8, 8), 2), ("f32", 128, (6, 11), 3)])
def test_rope_parity(dtype, head_dim, grid, heads):
    w = small(dtype, head_dim, heads=heads, grid_h=grid[0], grid_w=grid[1])
    cache = make_cache(w, 1, 1)
    frames = [57, 58, 59]
    q = synth.chunk_tensor(w, synth.T_Q, 19, 0, 0)
    k = synth.chunk_tensor(w, synth.T_K, 19, 0, 0)
    qd, kd = to_dev(q), to_dev(k)
    cache.rope3d(qd, kd, frames)
    for got, x in ((qd, q), (kd, k)):
        ref = oracle_rope(w, x, frames)
        if dtype == "bf16":
            ref_t = torch.from_numpy(ref.astype(np.float32)).to(torch.bfloat16)
            d = np.abs(bf16_ordered(got) - bf16_ordered(ref_t))
            assert d.max() <= 1
            assert (d > 0).mean() < 1e-5
        else:
            assert np.abs(exact(got) - ref).max() <= 1e-5
    # k only, a single frame at t = 0: frame 0, row 0, col 0 is unrotated
    k2 = to_dev(synth.chunk_tensor(w, synth.T_K, 0, 0, 0)[: w.tokens_per_frame].contiguous())
    k2_in = k2.clone()
    cache.rope3d(None, k2, [0])
    assert torch.equal(k2[0], k2_in[0])


# --------------------------------------------------------------------------
# (a5) attention
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,head_dim", [("bf16", 128), ("bf16", 64), ("f32", 64), ("f32", 128)])
def test_attention_direct_inputs(dtype, head_dim):
    # identical stored inputs on both sides (no RoPE): ragged chunk (198 tokens),
    # ragged anchors (2 frames = 132 keys), ring wraparound, two stages, two layers
    w = small(dtype, head_dim)
    run = PairedRun(w, rope=False)
    for c in range(w.n_chunks):
        for s in range(w.stages):
            for l in range(w.layers):
                run.step(c, s, l)


@pytest.mark.parametrize("dtype,head_dim", [("bf16", 128), ("f32", 64)])
def test_attention_end_to_end_with_rope(dtype, head_dim):
    w = small(dtype, head_dim, n_chunks=4)
    run = PairedRun(w, rope=True)
    for c in range(w.n_chunks):
        for s in range(w.stages):
            for l in range(w.layers):
                run.step(c, s, l)


@pytest.mark.parametrize("layers", [1, 2])
def test_tiny_workload_end_to_end(layers):
    # fp32, 2 heads, d 64, 8x8 grid, 3-frame chunks, W=2, 4 stages, anchors at
    # latent frames 0 and 15, 6 chunks, chunk-major order
    w = synth.WORKLOADS["tiny-f32"]
    run = PairedRun(w, layers=layers)
    for c in range(w.n_chunks):
        for s in range(w.stages):
            for l in range(layers):
                run.step(c, s, l)
    assert len(run.results) == w.n_chunks * w.stages * layers


@pytest.mark.parametrize("head_dim", [64, 128])
def test_tiny_shape_bf16(head_dim):
    w = synth.small_workload("tiny-bf16", dtype="bf16", heads=2, head_dim=head_dim, grid_h=8,
                             grid_w=8, ring_chunks=2, stages=4, layers=1, n_chunks=6,
                             anchor_rule="fixed:0,15", max_anchor_frames=2, wid=1)
    run = PairedRun(w)
    for c in range(w.n_chunks):
        for s in range(w.stages):
            run.step(c, s, 0)


def test_attention_degenerate_shapes():
    # W = 1, no anchor segment, one head, a chunk smaller than one key tile (18 tokens)
    w = synth.small_workload("deg", dtype="bf16", heads=1, head_dim=128, grid_h=2, grid_w=3,
                             ring_chunks=1, stages=1, layers=1, n_chunks=4, anchor_rule="none",
                             max_anchor_frames=1)
    run = PairedRun(w)
    for c in range(w.n_chunks):
        run.step(c, 0, 0)


@pytest.mark.parametrize("dtype,head_dim", [("bf16", 128), ("bf16", 64), ("f32", 64)])
def test_attention_one_token_chunks(dtype, head_dim):
    # The most degenerate shape: a 1x1 latent grid and 1-frame chunks, so every
    # chunk, history chunk and anchor frame is one token (each segment one valid
    # key, the second 32-key block of every tile fully masked); anchors at
    # latent frames 0 and 3, a ring of 2, two stages, RoPE included.
    w = synth.small_workload("one-token", dtype=dtype, heads=2, head_dim=head_dim, grid_h=1,
                             grid_w=1, frames_per_chunk=1, ring_chunks=2, stages=2, layers=1,
                             n_chunks=6, anchor_rule="fixed:0,3", max_anchor_frames=2, wid=102)
    run = PairedRun(w)
    for c in range(w.n_chunks):
        for s in range(w.stages):
            run.step(c, s, 0)
    assert len(run.results) == w.n_chunks * w.stages


@pytest.mark.parametrize("head_dim", [64, 128])
@pytest.mark.parametrize("grid", [(6, 11), (12, 22)])
def test_attention_tail_split_into_key_parts(head_dim, grid):
    # Fewer (head, 256-query) units than compute units: the whole launch is
    # the partial last round, run as 2, 3 or 4 key parts (at least 8 key
    # tiles of 64 each) plus the merge.  6x11 grid: 198-token chunks, one
    # ragged query tile; anchors 4 tiles + 4 per chunk, so chunks 2..7 see 16,
    # 20, 24, 28, 32, 32 tiles (2, 2, 3, 3, 4, 4 parts) with part boundaries
    # inside segments.  12x22 grid: 792-token chunks = 4 query tiles (last
    # holds 24 queries), 13 tiles per frame group, up to 104 tiles.
    w = small("bf16", head_dim, heads=2, grid_h=grid[0], grid_w=grid[1], ring_chunks=6,
              stages=1, layers=1, n_chunks=8, anchor_rule="fixed:0,7,20", max_anchor_frames=3)
    run = PairedRun(w, rope=False)
    for c in range(w.n_chunks):
        run.step(c, 0, 0)


@pytest.mark.parametrize("dtype,head_dim,grid", [("bf16", 128, (3, 5)), ("bf16", 128, (6, 11)),
                                                  ("bf16", 64, (6, 11)), ("f32", 64, (3, 5))])
def test_attention_maximum_segments(dtype, head_dim, grid):
    # the largest read set: 8 non-adjacent anchor frames of a 16-frame bank
    # (8 runs), a full ring of W = 8 chunks (wrapped once) and the chunk: 17
    # segments, each shorter than (3x5 grid) or not a multiple of one key tile
    W = ff.MAX_RING_CHUNKS
    w = small(dtype, head_dim, heads=3, grid_h=grid[0], grid_w=grid[1], ring_chunks=W,
              stages=1, layers=1, n_chunks=W + 3, anchor_rule="none",
              max_anchor_frames=ff.MAX_ANCHOR_FRAMES)
    bank_frames = list(range(16))
    bk, bv = synth.anchor_tensors(w, bank_frames, 0)
    bkd, bvd = to_dev(bk), to_dev(bv)
    window = [14, 0, 6, 2, 10, 4, 12, 8]            # listed out of order on purpose
    assert len(window) == ff.MAX_ANCHOR_FRAMES
    G = w.tokens_per_frame
    cache = make_cache(w, 1, 1)
    hist = []
    for c in range(w.n_chunks):
        q, k, v = (synth.chunk_tensor(w, t, c, 0, 0) for t in (synth.T_Q, synth.T_K, synth.T_V))
        out = cache.chunk_attention_bank(0, 0, c, to_dev(q), to_dev(k), to_dev(v), bkd, bvd, window)
        cache.kv_publish(0, 0, c, to_dev(k), to_dev(v))
        keys = [exact(bk[f * G:(f + 1) * G]) for f in window] + [h[0] for h in hist] + [exact(k)]
        vals = [exact(bv[f * G:(f + 1) * G]) for f in window] + [h[1] for h in hist] + [exact(v)]
        K_all, V_all = np.concatenate(keys), np.concatenate(vals)
        ref = fo.masked_attention(exact(q), K_all, V_all, np.ones(len(K_all), bool),
                                  1.0 / math.sqrt(head_dim))
        check_attention(exact(out), ref, dtype, f"chunk {c}")
        hist = (hist + [(exact(k), exact(v))])[-W:]
    table, count = cache.ring_state(0, 0)
    assert count == w.n_chunks and sorted(table) == list(range(w.n_chunks - W, w.n_chunks))


@pytest.mark.parametrize("head_dim,heads,grid", [(128, 3, (6, 11)), (64, 2, (12, 22))])
def test_attention_running_max_rescales(head_dim, heads, grid):
    # Keys of later chunks scaled by 1, 3, 9, 27, ..: each new segment carries
    # logits far above the running max (the rescale path runs again and again,
    # also inside tail-split key parts), then a chunk whose own keys are tiny
    # (no rescale, probabilities underflow to 0 for most keys).
    W = 4
    w = small("bf16", head_dim, heads=heads, grid_h=grid[0], grid_w=grid[1], ring_chunks=W,
              stages=1, layers=1, n_chunks=7, anchor_rule="none", max_anchor_frames=1)
    cache = make_cache(w, 1, 1)
    hist = []
    for c in range(w.n_chunks):
        q, k, v = (synth.chunk_tensor(w, t, c, 0, 0) for t in (synth.T_Q, synth.T_K, synth.T_V))
        factor = 3.0 ** c if c < w.n_chunks - 1 else 1.0 / 64
        k = (k.float() * factor).to(torch.bfloat16)
        out = cache.chunk_attention(0, 0, c, to_dev(q), to_dev(k), to_dev(v))
        cache.kv_publish(0, 0, c, to_dev(k), to_dev(v))
        K_all = np.concatenate([h[0] for h in hist] + [exact(k)])
        V_all = np.concatenate([h[1] for h in hist] + [exact(v)])
        ref = fo.masked_attention(exact(q), K_all, V_all, np.ones(len(K_all), bool),
                                  1.0 / math.sqrt(head_dim))
        check_attention(exact(out), ref, "bf16", f"chunk {c} (key scale {factor:g})")
        hist = (hist + [(exact(k), exact(v))])[-W:]


@pytest.mark.parametrize("head_dim", [128, 64])
def test_attention_reference_far_below_the_max(head_dim):
    # The first chunk's keys are tiny, so the first block a later chunk reads
    # (its oldest history chunk, or itself for chunk 0) gives a reference max
    # near 0 while the largest scores sit far above it: keys scaled by 8 give
    # probabilities up to ~2^35 relative to that reference (strongly peaked
    # rows, no overflow), keys scaled by 24 go past 2^64 (the workgroup's unit
    # runs again with the reference raised per block).
    W = 4
    w = small("bf16", head_dim, heads=2, grid_h=6, grid_w=11, ring_chunks=W,
              stages=1, layers=1, n_chunks=5, anchor_rule="none", max_anchor_frames=1)
    cache = make_cache(w, 1, 1)
    hist = []
    for c, factor in enumerate([0.01, 8.0, 8.0, 24.0, 1.0]):
        q, k, v = (synth.chunk_tensor(w, t, c, 0, 0) for t in (synth.T_Q, synth.T_K, synth.T_V))
        k = (k.float() * factor).to(torch.bfloat16)
        out = cache.chunk_attention(0, 0, c, to_dev(q), to_dev(k), to_dev(v))
        cache.kv_publish(0, 0, c, to_dev(k), to_dev(v))
        K_all = np.concatenate([h[0] for h in hist] + [exact(k)])
        V_all = np.concatenate([h[1] for h in hist] + [exact(v)])
        ref = fo.masked_attention(exact(q), K_all, V_all, np.ones(len(K_all), bool),
                                  1.0 / math.sqrt(head_dim))
        check_attention(exact(out), ref, "bf16", f"chunk {c} (key scale {factor:g})")
        hist = (hist + [(exact(k), exact(v))])[-W:]


@pytest.mark.parametrize("dtype,head_dim", [("bf16", 128), ("bf16", 64), ("f32", 64)])
def test_attention_batch_equals_single_calls(dtype, head_dim):
    # the rounds of a 4-stage wavefront (round n: chunk n - s at stage s), each
    # round's attention as one ff_chunk_attention_batch; stage 3 reads its anchors
    # from a bank.  Bit-identical to the single calls (the batch is never split
    # along keys, and no single call here is), and within the bar of the oracle.
    S = 4
    w = small(dtype, head_dim, heads=3, ring_chunks=2, stages=S, layers=1, n_chunks=5,
              anchor_rule="fixed:0,7", max_anchor_frames=2)
    ca, cb = make_cache(w, S, 1), make_cache(w, S, 1)
    frames = [0, 7]
    ak, av = synth.anchor_tensors(w, frames, 0)
    akd, avd = to_dev(ak), to_dev(av)
    for c in (ca, cb):
        c.anchor_set(0, frames, akd, avd)
    oracle = make_oracle(w, S, 1)
    oracle.anchor_set(0, frames, exact(ak), exact(av))
    scale = 1.0 / math.sqrt(head_dim)
    for n in range(w.n_chunks + S - 1):
        work = [(s, n - s) for s in range(S) if 0 <= n - s < w.n_chunks]
        items, singles, tensors = [], [], []
        for s, i in work:
            q, k, v = (to_dev(synth.chunk_tensor(w, t, i, s, 0))
                       for t in (synth.T_Q, synth.T_K, synth.T_V))
            tensors.append((s, i, q, k, v))
            it = dict(stage=s, layer=0, chunk=i, q=q, k=k, v=v)
            if s == 3:
                it.update(bank_k=akd, bank_v=avd, frames=[1, 0])
                singles.append(cb.chunk_attention_bank(s, 0, i, q, k, v, akd, avd, [1, 0]))
            else:
                singles.append(cb.chunk_attention(s, 0, i, q, k, v))
            items.append(it)
        outs = ca.chunk_attention_batch(items, scale=scale)
        for (s, i, q, k, v), o, o1 in zip(tensors, outs, singles):
            assert torch.equal(o, o1), (n, s, i)
            ref = oracle.attention(s, 0, i, exact(q), exact(k), exact(v), scale=scale)
            check_attention(exact(o), ref, dtype, f"round {n} stage {s} chunk {i}")
            for c in (ca, cb):
                c.kv_publish(s, 0, i, k, v)
            oracle.publish(s, 0, i, exact(k), exact(v))


def test_unfilled_slots_poisoned_with_nan_are_never_read():
    w = small("bf16", 128, ring_chunks=4, anchor_rule="fixed:3", max_anchor_frames=3)
    run = PairedRun(w, poison=True)
    for c in range(3):                       # ring never fills; 2 of 3 anchor frames unset
        for s in range(w.stages):
            for l in range(w.layers):
                run.step(c, s, l)


def test_softmax_scale_argument():
    w = small("bf16", 128, n_chunks=2)
    run = PairedRun(w)
    for c in range(2):
        run.step(c, 0, 0, scale=0.3)


def test_deterministic_and_order_independent():
    # chunk-major order and the anti-diagonal wavefront order of the paper's
    # batched rollout (round n runs chunk n - r at stage r) give the same bits
    w = small("bf16", 128, stages=4, layers=1, n_chunks=5)
    outs = {}
    for order_name in ("chunk-major", "wavefront", "chunk-major-again"):
        cache = make_cache(w, 4, 1)
        k, v = synth.anchor_tensors(w, [0, 7], 0)
        cache.anchor_set(0, [0, 7], to_dev(k), to_dev(v))
        if order_name == "wavefront":
            order = [(n - r, r) for n in range(w.n_chunks + 3) for r in range(4)
                     if 0 <= n - r < w.n_chunks]
        else:
            order = [(c, s) for c in range(w.n_chunks) for s in range(4)]
        res = {}
        for c, s in order:
            q = to_dev(synth.chunk_tensor(w, synth.T_Q, c, s, 0))
            kk = to_dev(synth.chunk_tensor(w, synth.T_K, c, s, 0))
            vv = to_dev(synth.chunk_tensor(w, synth.T_V, c, s, 0))
            res[(c, s)] = cache.chunk_attention(s, 0, c, q, kk, vv).cpu()
            cache.kv_publish(s, 0, c, kk, vv)
        outs[order_name] = res
    for key in outs["chunk-major"]:
        assert torch.equal(outs["chunk-major"][key], outs["wavefront"][key]), key
        assert torch.equal(outs["chunk-major"][key], outs["chunk-major-again"][key]), key


# --------------------------------------------------------------------------
# long horizon: 87 chunks, anchor updates every 8 chunks, ring wraparound
# --------------------------------------------------------------------------

def test_long_horizon_schedule():
    base = synth.WORKLOADS["1.3b-480p-long"]
    # same chunk count, anchor schedule, W, head_dim and input scale; reduced grid and heads
    w = synth.small_workload("long-reduced", dtype="bf16", heads=2, head_dim=128, grid_h=4,
                             grid_w=7, ring_chunks=base.ring_chunks, stages=1, layers=1,
                             n_chunks=base.n_chunks, input_scale=base.input_scale,
                             anchor_rule=base.anchor_rule, max_anchor_frames=3, wid=base.wid)
    run = PairedRun(w)
    for c in range(w.n_chunks):
        run.step(c, 0, 0)
    assert run.cache.anchor_state(0) == [0, 240, 260]
    assert run.cache.ring_state(0, 0) == ([84, 85, 86, 83], 87)


def test_long_horizon_full_grid_sampled_rows():
    # the long-horizon workload at its own shape (30x52 grid, 12 heads, d 128,
    # W = 4, inputs N(0,1)/sqrt(128)) through RoPE, attention and publish for
    # chunks 0 .. 10: the ring wraps from chunk 4 on and the anchor window moves
    # at chunk 8 ({0, 24} -> {0, 24, 48}); sampled rows of chunks 6 .. 10
    w = synth.WORKLOADS["1.3b-480p-long"]
    run = PairedRun(w, stages=1, layers=1)
    nq = w.chunk_tokens
    rows = np.concatenate([np.arange(0, 384), np.arange(nq - 384, nq)])
    heads = [0, w.heads - 1]
    for c in range(11):
        run.step(c, 0, 0, check=c >= 6, rows=rows, heads=heads)
        if c == 7:
            assert run.cache.anchor_state(0) == [0, 24]
    assert run.cache.anchor_state(0) == [0, 24, 48]
    assert run.cache.ring_state(0, 0) == ([8, 9, 10, 7], 11)
    assert len(run.results) == 5


# --------------------------------------------------------------------------
# full-size workloads: one steady-state chunk-stage, sampled rows
# --------------------------------------------------------------------------

@pytest.mark.parametrize("name,rope", [("1.3b-480p", False), ("14b-480p", False), ("14b-720p", True)])
def test_full_size_sampled_rows(name, rope):
    # 14B 720p (the benchmarked chunk-stage) runs the whole step: RoPE of Q and K
    # (and of the anchor K), attention over [anchors | ring | chunk], publish
    w = synth.WORKLOADS[name]
    stage, layer, chunk = 1, 3, w.ring_chunks + 3          # ring full, steady state
    run = PairedRun(w, stages=stage + 1, layers=layer + 1, rope=rope)
    nq = w.chunk_tokens
    rows = np.concatenate([np.arange(0, 512), np.arange(nq - 512, nq)])   # includes the ragged tail tile
    heads = [0, w.heads - 1]
    for c in range(chunk - w.ring_chunks, chunk + 1):
        run.step(c, stage, layer, check=(c == chunk), rows=rows, heads=heads)
    # the ring holds the previous W chunks plus this one; check one full slot bit for bit
    table, count = run.cache.ring_state(stage, layer)
    assert count == w.ring_chunks + 1 and run.cache.next_chunk(stage, layer) == chunk + 1
    assert sorted(table) == list(range(chunk - w.ring_chunks + 1, chunk + 1))
    entries = {e.chunk: e for e in run.oracle.history[(stage, layer)]}
    kg, vg = run.cache.read(stage, layer, chunk % w.ring_chunks)
    np.testing.assert_array_equal(exact(kg), entries[chunk].K)
    np.testing.assert_array_equal(exact(vg), entries[chunk].V)
