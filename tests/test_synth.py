"""The seeded input recipe: determinism, shapes, distributions, anchor schedules."""
import numpy as np
import torch

import synth
from oracle import ff_oracle as fo


def test_recipe_is_deterministic_and_keyed():
    w = synth.small_workload("t", heads=3, head_dim=64, grid_h=20, grid_w=30)
    a = synth.chunk_tensor(w, synth.T_K, 2, 1, 0)
    b = synth.chunk_tensor(w, synth.T_K, 2, 1, 0)
    c = synth.chunk_tensor(w, synth.T_K, 2, 1, 1)
    assert a.shape == (w.chunk_tokens, 3, 64) and a.dtype == torch.bfloat16
    assert torch.equal(a, b) and not torch.equal(a, c)
    x = a.float().numpy()
    assert abs(x.mean()) < 0.01 and abs(x.std() - 1.0) < 0.01


def test_input_scale():
    w = synth.WORKLOADS["1.3b-480p"]
    w2 = synth.small_workload("t", input_scale=w.input_scale, grid_h=30, grid_w=52, heads=1)
    x = synth.chunk_tensor(w2, synth.T_Q, 0, 0, 0).float().numpy()
    assert abs(x.std() - 1 / np.sqrt(128)) < 2e-3


def _frames(w, i):
    return fo.anchor_frames(w.anchor_rule, i, w.frames_per_chunk, w.latent_frames)


def test_workload_shapes():
    w = synth.WORKLOADS["14b-720p"]
    assert w.chunk_tokens == 10800 and w.tokens_per_frame == 3600
    kv = len(_frames(w, 10)) * w.tokens_per_frame + w.ring_chunks * w.chunk_tokens + w.chunk_tokens
    assert kv == 64800
    w = synth.WORKLOADS["1.3b-480p"]
    kv = len(_frames(w, 10)) * w.tokens_per_frame + w.ring_chunks * w.chunk_tokens + w.chunk_tokens
    assert kv == 28080
    for w in synth.WORKLOADS.values():
        assert max(len(_frames(w, i)) for i in range(w.n_chunks)) <= w.max_anchor_frames


def test_window_rule_is_gamma():
    # Gamma(i) by hand for B_R = 3, delta = 10 over 81 latents: u = floor(3i / 20)
    w = synth.WORKLOADS["1.3b-480p"]
    assert w.latent_frames == 81
    assert [_frames(w, i) for i in (0, 6, 7, 13, 14, 26)] == [
        [0, 10, 20], [0, 10, 20], [20, 30, 40], [20, 30, 40], [40, 50, 60], [60, 70, 80]]


def test_long_horizon_anchor_schedule():
    # a 1-frame anchor every 24 latents plus the end latent 260; chunk i reads the
    # first anchor and the two flanking its first latent 3i
    w = synth.WORKLOADS["1.3b-480p-long"]
    assert w.latent_frames == 261
    seq = [_frames(w, i) for i in range(w.n_chunks)]
    assert [i for i in range(w.n_chunks) if i == 0 or seq[i] != seq[i - 1]] == list(range(0, 87, 8))
    assert seq[0] == [0, 24] and seq[8] == [0, 24, 48] and seq[86] == [0, 240, 260]
    assert sorted({f for fr in seq for f in fr}) == list(range(0, 241, 24)) + [260]
    tiny = synth.WORKLOADS["tiny-f32"]
    assert _frames(tiny, 3) == [0, 15]


def test_flanking_anchors_bracket_the_chunk():
    # brute force over small clips: for a chunk whose first latent x lies before
    # the end anchor, the flanking entries are the last anchor at or before x and
    # the first anchor after it
    for L in (2, 9, 25, 48, 49, 100):
        for delta in (1, 4, 7, 24):
            P = fo.anchor_partition(L, delta)
            for B_R in (1, 3):
                for i in range(-(-L // B_R)):
                    x = B_R * i
                    if x >= L - 1:
                        continue
                    lo = max(p for p in P if p <= x)
                    hi = min(p for p in P if p > x)
                    assert fo.anchor_flank(i, B_R, delta, L) == sorted({0, lo, hi}), (L, delta, B_R, i)
    # a chunk that starts on the end anchor (off the grid) keeps the last grid
    # period's pair: the grid anchor before it and the end anchor itself
    assert fo.anchor_flank(8, 1, 7, 9) == [0, 7, 8]
    assert fo.anchor_flank(0, 3, 24, 1) == [0]
