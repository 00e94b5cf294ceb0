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


def test_workload_shapes():
    w = synth.WORKLOADS["14b-720p"]
    assert w.chunk_tokens == 10800 and w.tokens_per_frame == 3600
    kv = len(w.anchor_frames_for_chunk(10)) * w.tokens_per_frame + w.ring_chunks * w.chunk_tokens + w.chunk_tokens
    assert kv == 64800
    w = synth.WORKLOADS["1.3b-480p"]
    kv = len(w.anchor_frames_for_chunk(10)) * w.tokens_per_frame + w.ring_chunks * w.chunk_tokens + w.chunk_tokens
    assert kv == 28080


def test_window_rule_agrees_with_oracle_gamma():
    w = synth.WORKLOADS["1.3b-480p"]
    L = w.latent_frames
    for i in range(w.n_chunks):
        assert w.anchor_frames_for_chunk(i) == fo.anchor_window(i, 3, 10, L)


def test_long_horizon_anchor_schedule():
    w = synth.WORKLOADS["1.3b-480p-long"]
    assert w.latent_frames == 261
    assert w.anchor_update_chunks() == list(range(0, 87, 8))
    assert w.anchor_frames_for_chunk(0) == [0, 24]
    assert w.anchor_frames_for_chunk(8) == [0, 24, 48]
    assert w.anchor_frames_for_chunk(86) == [0, 240, 260]
    tiny = synth.WORKLOADS["tiny-f32"]
    assert tiny.anchor_frames_for_chunk(3) == [0, 15]
