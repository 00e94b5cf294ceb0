"""Concurrent calls of one stage with caller workspaces (ff_chunk_attention_ws),
and batch items beside tail-split single calls, against the oracle.

The renderer attention of Sec. 3.1 is the same whatever scratch memory the
launch uses: a workspace only moves the fp32 partial results of the key parts
(the split of a partial last round of workgroups) out of the cache's
per-stage region, so two layers of one stage may run on two streams at once.
"""
from __future__ import annotations

import math

import pytest
import torch

import synth
from gpu_util import anchor_frames, check_attention, exact, make_cache, make_oracle, to_dev
from test_gpu_parity import small

pytestmark = pytest.mark.gpu


def _workload(layers=2, stages=1, head_dim=128):
    # 6x11 grid, 2 heads: 2 units on a 256-CU part, so every launch is the
    # partial last round and runs as 2-4 key parts (16 .. 32 key tiles)
    return small("bf16", head_dim, heads=2, grid_h=6, grid_w=11, ring_chunks=6, stages=stages,
                 layers=layers, n_chunks=8, anchor_rule="fixed:0,7,20", max_anchor_frames=3)


def _set_anchors(w, caches, oracle, layers):
    frames = anchor_frames(w, 0)
    for l in range(layers):
        k, v = synth.anchor_tensors(w, frames, l)
        for c in caches:
            c.anchor_set(l, frames, to_dev(k), to_dev(v))
        oracle.anchor_set(l, frames, exact(k), exact(v))


@pytest.mark.parametrize("head_dim", [128, 64])
def test_two_layers_of_one_stage_on_two_streams(head_dim):
    w = _workload(head_dim=head_dim)
    cache, plain = make_cache(w, 1, 2), make_cache(w, 1, 2)
    oracle = make_oracle(w, 1, 2)
    _set_anchors(w, (cache, plain), oracle, 2)
    n_ws = cache.workspace_bytes()
    assert n_ws > 0
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    workspaces = [torch.empty(n_ws, dtype=torch.uint8, device=cache.device) for _ in streams]
    torch.cuda.synchronize()
    for c in range(w.n_chunks):
        inputs = {l: [to_dev(synth.chunk_tensor(w, t, c, 0, l)) for t in (synth.T_Q, synth.T_K, synth.T_V)]
                  for l in (0, 1)}
        torch.cuda.synchronize()   # inputs in place before the other streams read them
        outs = {}
        for l in (0, 1):           # both layers in flight at once, one stream each
            q, k, v = inputs[l]
            outs[l] = cache.chunk_attention_ws(0, l, c, q, k, v, workspaces[l], stream=streams[l])
            cache.kv_publish(0, l, c, k, v, stream=streams[l])
        torch.cuda.synchronize()
        for l in (0, 1):
            q, k, v = inputs[l]
            ref = oracle.attention(0, l, c, exact(q), exact(k), exact(v))
            check_attention(exact(outs[l]), ref, "bf16", f"chunk {c} layer {l}")
            oracle.publish(0, l, c, exact(k), exact(v))
            # the same call through the cache's own scratch, stream-ordered: bit-identical
            same = plain.chunk_attention(0, l, c, q, k, v)
            plain.kv_publish(0, l, c, k, v)
            torch.cuda.synchronize()
            assert torch.equal(same, outs[l]), f"chunk {c} layer {l}"


def test_workspace_sizes_only_limit_the_split():
    # a workspace too small for the full split, and none at all, stay within the bar
    w = _workload(layers=1)
    caches = [make_cache(w, 1, 1) for _ in range(3)]
    oracle = make_oracle(w, 1, 1)
    _set_anchors(w, caches, oracle, 1)
    n_ws = caches[0].workspace_bytes()
    dev = caches[0].device
    workspaces = [torch.empty(n_ws, dtype=torch.uint8, device=dev),
                  torch.empty(n_ws // 3, dtype=torch.uint8, device=dev), None]
    for c in range(w.n_chunks):
        q, k, v = (to_dev(synth.chunk_tensor(w, t, c, 0, 0)) for t in (synth.T_Q, synth.T_K, synth.T_V))
        ref = oracle.attention(0, 0, c, exact(q), exact(k), exact(v))
        for cache, ws in zip(caches, workspaces):
            out = cache.chunk_attention_ws(0, 0, c, q, k, v, ws)
            cache.kv_publish(0, 0, c, k, v)
            check_attention(exact(out), ref, "bf16", f"chunk {c} workspace {None if ws is None else ws.numel()}")
        oracle.publish(0, 0, c, exact(k), exact(v))


@pytest.mark.parametrize("head_dim", [128, 64])
def test_batch_items_beside_tail_split_single_calls(head_dim):
    # The single calls here are tail-split (2 units on 256 CUs), the batch never
    # is: an item and its single call may differ in low bits, and both stay
    # within the bf16 bar of the oracle (App. Alg. 1: one round's forwards).
    S = 2
    w = _workload(layers=1, stages=S, head_dim=head_dim)
    single, batched = make_cache(w, S, 1), make_cache(w, S, 1)
    oracle = make_oracle(w, S, 1)
    _set_anchors(w, (single, batched), oracle, 1)
    scale = 1.0 / math.sqrt(head_dim)
    for c in range(w.n_chunks):
        items, refs = [], []
        for s in range(S):
            q, k, v = (to_dev(synth.chunk_tensor(w, t, c, s, 0)) for t in (synth.T_Q, synth.T_K, synth.T_V))
            refs.append((oracle.attention(s, 0, c, exact(q), exact(k), exact(v), scale=scale), q, k, v))
            items.append(dict(stage=s, layer=0, chunk=c, q=q, k=k, v=v))
        outs = batched.chunk_attention_batch(items, scale=scale)
        for s, (ref, q, k, v) in enumerate(refs):
            one = single.chunk_attention(s, 0, c, q, k, v, scale=scale)
            check_attention(exact(one), ref, "bf16", f"single chunk {c} stage {s}")
            check_attention(exact(outs[s]), ref, "bf16", f"batch chunk {c} stage {s}")
            for cache in (single, batched):
                cache.kv_publish(s, 0, c, k, v)
            oracle.publish(s, 0, c, exact(k), exact(v))
