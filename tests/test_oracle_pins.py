"""Pins of the float64 oracle against facts that do not come from the oracle itself.

Each test checks the oracle against a closed form, an invariant, a library
routine, or a value printed in the paper (tests/golden/paper_examples.json),
chosen so that a plausible slip (a dropped term, a swapped axis, a wrong sign,
an off-by-one in the history window) fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import ff_oracle as fo

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_examples.json")))


def rng(seed):
    return np.random.default_rng(seed)


# --------------------------------------------------------------------------
# rounding
# --------------------------------------------------------------------------

def test_bf16_rounding_matches_torch_on_float32_values():
    x = rng(0).standard_normal(200000).astype(np.float32) * np.float32(3.0)
    x = np.concatenate([x, np.float32([1e-39, -3e-40, 65504.0, 3.3e38, -1e-30])])
    ref = torch.from_numpy(x).to(torch.bfloat16).double().numpy()
    got = fo.round_to_bf16(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


def test_bf16_rounding_ties_to_even():
    ulp = 2.0 ** -7                       # bf16 spacing in [1, 2)
    assert fo.round_to_bf16(np.array([1 + ulp / 2]))[0] == 1.0            # tie -> even (1.0)
    assert fo.round_to_bf16(np.array([1 + 3 * ulp / 2]))[0] == 1 + 2 * ulp  # tie -> even
    assert fo.round_to_bf16(np.array([1 + ulp / 2 + 2 ** -30]))[0] == 1 + ulp
    assert fo.round_to_bf16(np.array([-(1 + ulp / 2)]))[0] == -1.0
    assert np.isinf(fo.round_to_bf16(np.array([3.4e38]))[0])


# --------------------------------------------------------------------------
# (a1) token layout
# --------------------------------------------------------------------------

def test_chunk_frames_paper_example():
    ex = GOLDEN["chunk_reads_anchors"][0]
    # the chunk at positions 6-8 is chunk 2 of three-latent chunks
    assert fo.chunk_frames(2, ex["B_R"]) == ex["frames"]


def test_token_positions_row_major():
    t, y, x = fo.token_positions([5, 9], 3, 4)
    assert len(t) == 24
    assert (t[:12] == 5).all() and (t[12:] == 9).all()
    assert list(y[:12]) == [0] * 4 + [1] * 4 + [2] * 4
    assert list(x[:12]) == [0, 1, 2, 3] * 3
    assert (t[13], y[13], x[13]) == (9, 0, 1)


# --------------------------------------------------------------------------
# (a2) RoPE
# --------------------------------------------------------------------------

def unit(d, idx, heads=1):
    v = np.zeros((1, heads, d))
    v[0, :, idx] = 1.0
    return v


def test_rope_split_matches_workload_statement():
    # "head_dim split 22/21/21 across t/h/w" at head_dim 128
    assert fo.rope_pair_split(128) == (22, 21, 21)
    assert fo.rope_pair_split(64) == (12, 10, 10)


@pytest.mark.parametrize("d", [64, 128])
def test_rope_position_zero_is_identity(d):
    split = fo.rope_pair_split(d)
    X = rng(1).standard_normal((4, 3, d))
    out = fo.rope3d(X, [0], 2, 2, split)
    # tokens at y=0,x=0 of frame 0 are not rotated
    np.testing.assert_array_equal(out[0], X[0])


@pytest.mark.parametrize("d", [64, 128])
def test_rope_preserves_pair_norms(d):
    split = fo.rope_pair_split(d)
    X = rng(2).standard_normal((2 * 3 * 5, 4, d))
    out = fo.rope3d(X, [7, 41], 3, 5, split)
    n_in = X[..., 0::2] ** 2 + X[..., 1::2] ** 2
    n_out = out[..., 0::2] ** 2 + out[..., 1::2] ** 2
    np.testing.assert_allclose(n_out, n_in, rtol=1e-13, atol=1e-13)


def test_rope_axis_blocks_and_direction():
    # pair 0 of each axis block has frequency 1: it turns by exactly t, y or x
    # radians, counter-clockwise (a, b) -> (a cos - b sin, a sin + b cos).
    d = 128
    split = fo.rope_pair_split(d)
    c1, s1 = math.cos(1.0), math.sin(1.0)
    grid_h, grid_w = 2, 3
    # token (t=1, y=0, x=0) is token 0 of frame 1
    e = np.zeros((grid_h * grid_w, 1, d)); e[:, 0, 0] = 1.0
    out = fo.rope3d(e, [1], grid_h, grid_w, split)
    assert out[0, 0, 0] == pytest.approx(c1, abs=1e-15)
    assert out[0, 0, 1] == pytest.approx(s1, abs=1e-15)
    # element 44 starts the h block (22 t pairs); token 3 has y=1, x=0
    e = np.zeros((grid_h * grid_w, 1, d)); e[:, 0, 44] = 1.0
    out = fo.rope3d(e, [0], grid_h, grid_w, split)
    assert out[3, 0, 44] == pytest.approx(c1, abs=1e-15)
    assert out[3, 0, 45] == pytest.approx(s1, abs=1e-15)
    assert out[1, 0, 44] == 1.0 and out[1, 0, 45] == 0.0     # y = 0 there
    # element 86 starts the w block; token 1 has y=0, x=1
    e = np.zeros((grid_h * grid_w, 1, d)); e[:, 0, 87] = 1.0   # b component
    out = fo.rope3d(e, [0], grid_h, grid_w, split)
    assert out[1, 0, 86] == pytest.approx(-s1, abs=1e-15)
    assert out[1, 0, 87] == pytest.approx(c1, abs=1e-15)
    assert out[3, 0, 86] == 0.0 and out[3, 0, 87] == 1.0     # x = 0 there


def test_rope_frequency_exponent():
    # with theta = 10000 and 22 t pairs, pair j = 11 has frequency
    # 10000**(-11/22) = 0.01: at t = 100 it turns by one radian.
    d = 128
    split = fo.rope_pair_split(d)
    e = np.zeros((1, 1, d)); e[0, 0, 22] = 1.0
    out = fo.rope3d(e, [100], 1, 1, split)
    assert out[0, 0, 22] == pytest.approx(math.cos(1.0), abs=1e-12)
    assert out[0, 0, 23] == pytest.approx(math.sin(1.0), abs=1e-12)


def test_rope_equals_complex_multiplication():
    d = 64
    split = fo.rope_pair_split(d)
    X = rng(3).standard_normal((2 * 4 * 3, 2, d))
    frames = [3, 11]
    out = fo.rope3d(X, frames, 4, 3, split)
    z = X[..., 0::2] + 1j * X[..., 1::2]
    t, y, x = fo.token_positions(frames, 4, 3)
    n_t, n_h, n_w = split
    freqs = np.concatenate([10000.0 ** (-np.arange(n) / n) for n in (n_t, n_h, n_w)])
    pos = np.concatenate([np.repeat(t[:, None], n_t, 1), np.repeat(y[:, None], n_h, 1),
                          np.repeat(x[:, None], n_w, 1)], axis=1)
    zr = z * np.exp(1j * pos * freqs)[:, None, :]
    np.testing.assert_allclose(out[..., 0::2], zr.real, atol=1e-12)
    np.testing.assert_allclose(out[..., 1::2], zr.imag, atol=1e-12)


def test_rope_relative_position_property():
    # <R(p1) q, R(p2) k> depends only on p1 - p2 (per axis): shift all three axes
    d = 128
    split = fo.rope_pair_split(d)
    r = rng(4)
    q = r.standard_normal((1, 1, d)); k = r.standard_normal((1, 1, d))
    gh, gw = 5, 7

    def rot(v, t, y, x, shift=(0, 0, 0)):
        # place v at token (y, x) of frame t in a grid offset by shift
        G = (gh + shift[1]) * (gw + shift[2])
        X = np.zeros((G, 1, d))
        n = (y + shift[1]) * (gw + shift[2]) + (x + shift[2])
        X[n] = v[0]
        return fo.rope3d(X, [t + shift[0]], gh + shift[1], gw + shift[2], split)[n, 0]

    base = rot(q, 4, 1, 2) @ rot(k, 9, 3, 6)
    shifted = rot(q, 4, 1, 2, (17, 2, 3)) @ rot(k, 9, 3, 6, (17, 2, 3))
    assert shifted == pytest.approx(base, abs=1e-11)
    # a different relative offset changes the product
    other = rot(q, 5, 1, 2) @ rot(k, 9, 3, 6)
    assert abs(other - base) > 1e-3


# --------------------------------------------------------------------------
# (a5) attention
# --------------------------------------------------------------------------

def test_attention_matches_torch_sdpa_float64():
    r = rng(5)
    nq, nk, h, d = 7, 23, 3, 16
    Q = r.standard_normal((nq, h, d)); K = r.standard_normal((nk, h, d)); V = r.standard_normal((nk, h, d))
    vis = r.random(nk) > 0.3
    vis[0] = True
    scale = 1 / math.sqrt(d)
    got = fo.masked_attention(Q, K, V, vis, scale)
    qt = torch.from_numpy(Q).permute(1, 0, 2)
    kt = torch.from_numpy(K).permute(1, 0, 2)
    vt = torch.from_numpy(V).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(
        qt, kt, vt, attn_mask=torch.from_numpy(vis)[None, None, :].expand(h, nq, nk))
    np.testing.assert_allclose(got, ref.permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-13)


def test_attention_identical_keys_gives_mean_of_visible_values():
    r = rng(6)
    nq, nk, h, d = 5, 40, 2, 8
    Q = r.standard_normal((nq, h, d))
    K = np.repeat(r.standard_normal((1, h, d)), nk, axis=0)
    V = r.standard_normal((nk, h, d))
    vis = np.zeros(nk, bool); vis[3:29] = True
    out = fo.masked_attention(Q, K, V, vis, 0.37)
    mean = V[vis].mean(axis=0)
    np.testing.assert_allclose(out, np.broadcast_to(mean, out.shape), rtol=1e-12, atol=1e-13)


def test_attention_constant_values_and_dominant_key():
    r = rng(7)
    nq, nk, h, d = 3, 30, 1, 8
    Q = r.standard_normal((nq, h, d)); K = r.standard_normal((nk, h, d))
    V = np.full((nk, h, d), 2.5)
    out = fo.masked_attention(Q, K, V, np.ones(nk, bool), 1.0)
    np.testing.assert_allclose(out, 2.5, rtol=1e-14)
    # a key parallel to the query with a large norm takes all the weight
    V = r.standard_normal((nk, h, d))
    K[11] = 60.0 * Q[0] / np.linalg.norm(Q[0])
    out = fo.masked_attention(Q[:1], K, V, np.ones(nk, bool), 1.0)
    np.testing.assert_allclose(out[0, 0], V[11, 0], atol=1e-10)


def test_attention_masked_keys_have_no_influence():
    r = rng(8)
    nq, nk, h, d = 4, 50, 2, 8
    Q = r.standard_normal((nq, h, d)); K = r.standard_normal((nk, h, d)); V = r.standard_normal((nk, h, d))
    vis = np.ones(nk, bool); vis[10:30] = False
    a = fo.masked_attention(Q, K, V, vis, 0.5)
    K2, V2 = K.copy(), V.copy()
    K2[10:30] = np.nan; V2[10:30] = 1e30
    b = fo.masked_attention(Q, K2, V2, vis, 0.5)
    np.testing.assert_array_equal(a, b)


def test_attention_key_permutation_invariance():
    r = rng(9)
    nq, nk, h, d = 4, 33, 2, 8
    Q = r.standard_normal((nq, h, d)); K = r.standard_normal((nk, h, d)); V = r.standard_normal((nk, h, d))
    perm = r.permutation(nk)
    a = fo.masked_attention(Q, K, V, np.ones(nk, bool), 0.4)
    b = fo.masked_attention(Q, K[perm], V[perm], np.ones(nk, bool), 0.4)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-14)


# --------------------------------------------------------------------------
# (a3, a4) history bank and anchor bank
# --------------------------------------------------------------------------

@pytest.mark.parametrize("W", [1, 2, 4])
def test_history_is_tail_of_published_sequence(W):
    r = rng(10)
    cache = fo.RendererCacheOracle(stages=2, layers=1, W=W)
    Ks = [r.standard_normal((6, 2, 4)) for _ in range(3 * W + 2)]
    Vs = [r.standard_normal((6, 2, 4)) for _ in range(3 * W + 2)]
    for n in range(1, len(Ks) + 1):
        cache.publish(0, 0, n - 1, Ks[n - 1], Vs[n - 1])
        keep = list(range(max(0, n - W), n))
        Kc, Vc, chunks = cache.history_concat(0, 0)
        assert chunks == keep
        np.testing.assert_array_equal(Kc, np.concatenate([Ks[c] for c in keep], 0))
        np.testing.assert_array_equal(Vc, np.concatenate([Vs[c] for c in keep], 0))
        table, count = cache.ring_state(0, 0)
        assert count == n
        for c in keep:
            assert table[c % W] == c
        assert sum(1 for s in table if s >= 0) == len(keep)
    # the other stage is untouched
    assert cache.ring_state(1, 0) == ([-1] * W, 0)


def test_history_rejects_out_of_order_publish():
    cache = fo.RendererCacheOracle(stages=1, layers=1, W=2)
    z = np.zeros((3, 1, 2))
    cache.publish(0, 0, 5, z, z)
    with pytest.raises(fo.OrderError):
        cache.publish(0, 0, 7, z, z)
    with pytest.raises(fo.OrderError):
        cache.attention(0, 0, 5, z, z, z)


def test_read_set_window_and_anchor_replacement():
    r = rng(11)
    W = 2
    cache = fo.RendererCacheOracle(stages=1, layers=1, W=W)
    a1 = r.standard_normal((4, 1, 2)); a2 = r.standard_normal((8, 1, 2))
    cache.anchor_set(0, [0], a1, a1)
    cache.anchor_set(0, [10, 20], a2, a2)     # replaces, does not append
    for c in range(3):
        cache.publish(0, 0, c, np.full((3, 1, 2), c), np.full((3, 1, 2), c))
    Ks, Vs, vis = cache.read_set(0, 0, 3, np.full((3, 1, 2), 9.0), np.full((3, 1, 2), 9.0))
    assert [k.shape[0] for k in Ks] == [8, 3, 3, 3]
    np.testing.assert_array_equal(Ks[0], a2)
    # history holds chunks 1 and 2; both are in [3-W, 2]
    np.testing.assert_array_equal(Ks[1][:, 0, 0], [1, 1, 1])
    np.testing.assert_array_equal(Ks[2][:, 0, 0], [2, 2, 2])
    assert vis == [True, True, True, True]
    # seen from chunk 4 (history not advanced), chunk 1 falls out of [4-W, 3]
    cache2 = fo.RendererCacheOracle(stages=1, layers=1, W=W)
    for c in range(3):
        cache2.publish(0, 0, c, np.full((3, 1, 2), c), np.full((3, 1, 2), c))
    _, _, vis = cache2.read_set(0, 0, 4, np.zeros((3, 1, 2)), np.zeros((3, 1, 2)))
    assert vis == [False, True, True]


def _stage_sequence(seed, n_chunks, W, nq, h, d, anchors_of_chunk, anchor_data):
    r = rng(seed)
    Qs = [r.standard_normal((nq, h, d)) for _ in range(n_chunks)]
    Ks = [r.standard_normal((nq, h, d)) for _ in range(n_chunks)]
    Vs = [r.standard_normal((nq, h, d)) for _ in range(n_chunks)]
    return Qs, Ks, Vs


@pytest.mark.parametrize("W", [1, 2, 3])
def test_sequential_ring_equals_packed_block_causal_mask(W):
    # The paper states the chunk-by-chunk cache update and one full-clip forward
    # with a chunk-wise causal mask are the same computation.
    r = rng(12 + W)
    n_chunks, nq, h, d, G = 7, 6, 2, 8, 3
    frames = [0, 10, 20, 30]
    anchor_data = {f: (r.standard_normal((G, h, d)), r.standard_normal((G, h, d))) for f in frames}
    anchors_of_chunk = [[0, 10, 20] if i < 4 else [20, 30] for i in range(n_chunks)]
    Qs, Ks, Vs = _stage_sequence(20 + W, n_chunks, W, nq, h, d, anchors_of_chunk, anchor_data)
    scale = 1 / math.sqrt(d)
    packed = fo.packed_stage_attention(Qs, Ks, Vs, anchor_data, anchors_of_chunk, W, scale)
    cache = fo.RendererCacheOracle(stages=1, layers=1, W=W)
    for i in range(n_chunks):
        fr = anchors_of_chunk[i]
        cache.anchor_set(0, fr, np.concatenate([anchor_data[f][0] for f in fr]),
                         np.concatenate([anchor_data[f][1] for f in fr]))
        out = cache.attention(0, 0, i, Qs[i], Ks[i], Vs[i], scale)
        cache.publish(0, 0, i, Ks[i], Vs[i])
        np.testing.assert_allclose(out, packed[i], rtol=1e-11, atol=1e-12)


def test_sequential_ring_differs_from_wrong_window():
    # guard: the packed equivalence is sensitive to the window length
    r = rng(30)
    n_chunks, nq, h, d, G, W = 5, 4, 1, 8, 2, 2
    anchor_data = {0: (r.standard_normal((G, h, d)), r.standard_normal((G, h, d)))}
    anchors_of_chunk = [[0]] * n_chunks
    Qs, Ks, Vs = _stage_sequence(31, n_chunks, W, nq, h, d, anchors_of_chunk, anchor_data)
    packed_w = fo.packed_stage_attention(Qs, Ks, Vs, anchor_data, anchors_of_chunk, W + 1, 0.3)
    cache = fo.RendererCacheOracle(stages=1, layers=1, W=W)
    cache.anchor_set(0, [0], *anchor_data[0])
    diffs = []
    for i in range(n_chunks):
        out = cache.attention(0, 0, i, Qs[i], Ks[i], Vs[i], 0.3)
        cache.publish(0, 0, i, Ks[i], Vs[i])
        diffs.append(np.abs(out - packed_w[i]).max())
    assert max(diffs[:W + 1]) < 1e-12 and min(diffs[W + 1:]) > 1e-6


# --------------------------------------------------------------------------
# planner-side index sets (paper's worked examples)
# --------------------------------------------------------------------------

def test_anchor_partition_examples():
    for ex in GOLDEN["anchor_partition"]:
        assert fo.anchor_partition(ex["L"], ex["delta"]) == ex["P"], ex["cite"]


def test_block_and_chunk_counts():
    for ex in GOLDEN["planner_blocks"]:
        assert fo.num_blocks(ex["M"], ex["B_P"]) == ex["N_P"], ex["cite"]
        sizes = [min(ex["B_P"], ex["M"] - j * ex["B_P"]) for j in range(ex["N_P"])]
        assert sizes == ex["sizes"]
    for ex in GOLDEN["renderer_chunks"]:
        assert fo.num_blocks(ex["L"], ex["B_R"]) == ex["N_R"], ex["cite"]


def test_anchor_windows_examples():
    ex = GOLDEN["chunk_reads_anchors"][0]
    i = ex["frames"][0] // ex["B_R"]
    assert fo.anchor_window(i, ex["B_R"], ex["delta"], ex["L"]) == ex["anchors"]
    ex = GOLDEN["anchor_windows"]
    n = fo.num_blocks(ex["L"], ex["B_R"])
    windows = []
    for i in range(n):
        w = fo.anchor_window(i, ex["B_R"], ex["delta"], ex["L"])
        if w not in windows:
            windows.append(w)
    assert windows == ex["windows"], ex["cite"]
    ex = GOLDEN["chunks_per_window"]
    counts = {}
    for i in range(fo.num_blocks(ex["L"], ex["B_R"])):
        key = tuple(fo.anchor_window(i, ex["B_R"], ex["delta"], ex["L"]))
        counts[key] = counts.get(key, 0) + 1
    assert min(counts.values()) == ex["min"] and max(counts.values()) == ex["max"]


def test_forward_counts_example():
    ex = GOLDEN["forward_counts"]
    assert fo.forward_counts(ex["L"], ex["delta"], ex["B"], ex["S"]) == (
        ex["FlashForward"], ex["SelfForcing"], ex["HiAR"])


def test_history_lengths_and_context_budget():
    ex = GOLDEN["history_lengths"]
    assert fo.history_lengths(ex["W_ctx"], ex["B_P"], ex["B_R"]) == (ex["H"], ex["H_P"])
    c = GOLDEN["context_positions"]
    assert c["anchor"] + ex["H"] * ex["B_R"] + c["current"] == c["total"] == ex["W_ctx"]


def test_video_lengths_map_to_chunks():
    ex = GOLDEN["video_lengths"]
    # 16 FPS, causal VAE with 4x temporal compression: 1 + 4(L-1) frames
    for s, L in zip(ex["seconds"], ex["latents"]):
        assert 1 + 4 * (L - 1) == 16 * s + 1
        assert fo.num_blocks(L, 3) * 3 == L


# --------------------------------------------------------------------------
# Euler step and wavefront schedule

def test_euler_step_follows_rectified_flow_path():
    """On the linear path x_s = (1 - s) x0 + s eps with its exact velocity
    v = eps - x0, one Euler step from sigma_k lands on x at sigma_{k-1}."""
    rng = np.random.default_rng(3)
    x0, eps = rng.standard_normal((2, 4096))
    sig = [1.0, 0.75, 0.5, 0.25, 0.0]
    x = eps.copy()
    for k in range(4):
        x = fo.euler_step(x, eps - x0, sig[k] - sig[k + 1], "f64")
        np.testing.assert_allclose(x, (1 - sig[k + 1]) * x0 + sig[k + 1] * eps, atol=1e-14)
    np.testing.assert_allclose(x, x0, atol=1e-14)


def test_euler_step_rounds_once_to_storage():
    x = np.array([1.0, 1.0, -3.0, 0.0])
    v = np.array([2.0 ** -9, 2.0 ** -8, 0.5, 7.0])
    got = fo.euler_step(x, v, -1.0, "bf16")            # x + v
    # bf16 spacing at 1 is 2^-7: 1 + 2^-9 rounds down, 1 + 2^-8 is the tie and goes to the
    # even neighbour 1; -3 + 0.5 and 0 + 7 are exact
    np.testing.assert_array_equal(got, [1.0, 1.0, -2.5, 7.0])
    assert fo.euler_step(np.array([5.0]), np.array([123.0]), 0.0, "bf16")[0] == 5.0


@pytest.mark.parametrize("N_R,S", [(1, 1), (6, 4), (27, 4), (3, 5)])
def test_wavefront_schedule_rounds_and_coverage(N_R, S):
    rounds = fo.wavefront_schedule(N_R, S)
    assert len(rounds) == N_R + S - 1
    items = [it for r in rounds for it in r]
    assert sorted(items) == sorted((r, i) for r in range(S) for i in range(N_R))  # N_R S forwards
    pos = {it: n for n, r in enumerate(rounds) for it in r}
    for r in range(S):
        for i in range(N_R):
            if r > 0:
                assert pos[(r, i)] == pos[(r - 1, i)] + 1     # the hand-off of x_{i,k}
            if i > 0:
                assert pos[(r, i)] == pos[(r, i - 1)] + 1     # the stage's ring, chunk order
    # the renderer share of the forward-count model is N_R * S
    L, B = 3 * N_R, 3
    total, _, _ = fo.forward_counts(L, 10, B, S)
    M = len(fo.anchor_partition(L, 10))
    assert total - fo.num_blocks(M, B) * (S + 1) == N_R * S


# --------------------------------------------------------------------------
# attention backward (packed training forward)

def _packed_case(seed=0, n=3, Nq=5, G=4, nf=2, h=2, d=8, W=1):
    rng = np.random.default_rng(seed)
    table = [[0], [1, 0], [1]][:n]
    M = fo.packed_visibility(n, Nq, G, nf, table, W)
    Q = rng.standard_normal((n * Nq, h, d))
    K = rng.standard_normal((nf * G + n * Nq, h, d))
    V = rng.standard_normal((nf * G + n * Nq, h, d))
    dO = rng.standard_normal((n * Nq, h, d))
    return Q, K, V, dO, M


def test_packed_visibility_rows():
    M = fo.packed_visibility(3, 2, 1, 2, [[0], [], [0, 1]], 1)
    assert M.shape == (6, 2 + 6)
    np.testing.assert_array_equal(M[0], [1, 0, 1, 1, 0, 0, 0, 0])
    np.testing.assert_array_equal(M[2], [0, 0, 1, 1, 1, 1, 0, 0])
    np.testing.assert_array_equal(M[5], [1, 1, 0, 0, 1, 1, 1, 1])


def test_attention_grad_matches_autograd():
    Q, K, V, dO, M = _packed_case(nf=3)          # anchor frame 2 is listed for no chunk
    scale = 0.35
    dQ, dK, dV = fo.masked_attention_grad(Q, K, V, M, dO, scale)
    tQ, tK, tV = (torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (Q, K, V))
    mask = torch.tensor(M)
    outs = []
    for h in range(Q.shape[1]):
        s = scale * tQ[:, h] @ tK[:, h].T
        s = s.masked_fill(~mask, float("-inf"))
        outs.append(torch.softmax(s, dim=-1) @ tV[:, h])
    out = torch.stack(outs, 1)
    out.backward(torch.tensor(dO))
    np.testing.assert_allclose(dQ, tQ.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(dK, tK.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(dV, tV.grad.numpy(), atol=1e-12)
    # keys no query sees get no gradient
    hidden = ~M.any(axis=0)
    assert hidden.any()
    assert np.all(dK[hidden] == 0) and np.all(dV[hidden] == 0)


def test_attention_grad_finite_differences():
    Q, K, V, dO, M = _packed_case(seed=4, n=2, Nq=3, G=2, nf=2, h=1, d=4)
    scale = 0.5

    def loss(Q, K, V):
        # forward row by row with the oracle's masked attention (one visibility row each)
        O = np.concatenate([fo.masked_attention(Q[r:r + 1], K, V, M[r], scale)
                            for r in range(Q.shape[0])])
        return float((O * dO).sum())
    dQ, dK, dV = fo.masked_attention_grad(Q, K, V, M, dO, scale)
    eps = 1e-6
    for arr, grad in ((Q, dQ), (K, dK), (V, dV)):
        for idx in [(0, 0, 1), (arr.shape[0] - 1, 0, 3), (arr.shape[0] // 2, 0, 0)]:
            a1, a2 = arr.copy(), arr.copy()
            a1[idx] += eps
            a2[idx] -= eps
            args1 = [a1 if arr is x else x for x in (Q, K, V)]
            args2 = [a2 if arr is x else x for x in (Q, K, V)]
            num = (loss(*args1) - loss(*args2)) / (2 * eps)
            assert abs(num - grad[idx]) < 1e-6 * max(1.0, abs(num)), (idx, num, grad[idx])


def test_log2_sum_exp2_recovers_softmax():
    Q, K, V, dO, M = _packed_case(seed=2)
    scale = 0.3
    lse2 = fo.log2_sum_exp2(Q, K, M, scale)
    for h in range(Q.shape[1]):
        s = scale * np.log2(np.e) * (Q[:, h] @ K[:, h].T)
        P = np.where(M, np.exp2(s - lse2[:, h:h + 1]), 0.0)
        np.testing.assert_allclose(P.sum(axis=1), 1.0, atol=1e-12)
