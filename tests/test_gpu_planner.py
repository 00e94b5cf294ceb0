"""Planner side on the GPU: block attention of the planner over
Tail_{H_P}(A) plus its own block (a one-stage ring of H_P blocks with no
anchor segment), publishing each block's clean-endpoint K/V into an
append-only anchor bank, and renderer chunks reading their window Gamma(i)
from that bank.  Each block holds B_P anchor latents of the partition P, at
their own latent positions for RoPE.  Checked against the float64 oracle
(bars as in test_gpu_parity)."""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import ff_oracle as fo
from paper_2609_32540_amd import ff

from gpu_util import check_attention, exact, oracle_rope, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _needs_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ff.lib()


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_planner_blocks_feed_renderer_anchor_windows(dtype, d):
    L, delta, B, H_P = 81, 10, 3, 2
    w = synth.small_workload("planner", dtype=dtype, heads=2, head_dim=d, grid_h=6, grid_w=11,
                             ring_chunks=H_P, stages=1, layers=1, n_chunks=L // B,
                             anchor_rule="none", max_anchor_frames=3)
    P = ff.anchor_partition(L, delta)
    assert P == fo.anchor_partition(L, delta) and len(P) % B == 0
    n_blocks = len(P) // B
    G = w.tokens_per_frame
    scale = 1.0 / math.sqrt(d)
    planner = ff.RendererCache(stages=1, layers=1, ring_chunks=H_P, frames_per_chunk=B,
                               grid_h=w.grid_h, grid_w=w.grid_w, heads=w.heads, head_dim=d,
                               max_anchor_frames=1, dtype=w.torch_dtype, device=torch.device("cuda", 0))
    orc = fo.RendererCacheOracle(stages=1, layers=1, W=H_P)
    bank_k, bank_v = {}, {}          # latent frame -> [G, heads, d] (device), the anchor bank A
    bank_ref = {}                    # latent frame -> (K, V) float64 as stored
    for j in range(n_blocks):
        frames = P[j * B:(j + 1) * B]
        q, k, v = (synth.chunk_tensor(w, t, j, 0, 0, seed=5) for t in (synth.T_Q, synth.T_K, synth.T_V))
        qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
        planner.rope3d(qd, kd, frames)
        out = planner.chunk_attention(0, 0, j, qd, kd, vd, scale=scale)
        planner.kv_publish(0, 0, j, kd, vd)
        q_ref, k_ref = oracle_rope(w, q, frames), oracle_rope(w, k, frames)
        ref = orc.attention(0, 0, j, q_ref, k_ref, exact(v), scale=scale)
        orc.publish(0, 0, j, k_ref, exact(v))
        check_attention(exact(out), ref, dtype, f"planner block {j}")
        # the block's clean-endpoint K/V, read back from its ring slot, joins the bank
        kb, vb = planner.read(0, 0, j % H_P)
        for n, f in enumerate(frames):
            bank_k[f] = kb[n * G:(n + 1) * G].clone()
            bank_v[f] = vb[n * G:(n + 1) * G].clone()
            bank_ref[f] = (k_ref[n * G:(n + 1) * G], exact(v)[n * G:(n + 1) * G])
    torch.cuda.synchronize()
    assert planner.ring_state(0, 0)[1] == n_blocks

    # renderer chunks of one stage read Gamma(i) from the bank
    R2 = ff.RendererCache(stages=1, layers=1, ring_chunks=2, frames_per_chunk=B, grid_h=w.grid_h,
                          grid_w=w.grid_w, heads=w.heads, head_dim=d, max_anchor_frames=3,
                          dtype=w.torch_dtype, device=planner.device)
    rorc2 = fo.RendererCacheOracle(stages=1, layers=1, W=2)
    current = None
    for i in range(9):
        gamma = ff.anchor_window(i, B, delta, L)
        if gamma != current:
            R2.anchor_set(0, gamma, torch.cat([bank_k[f] for f in gamma]).contiguous(),
                          torch.cat([bank_v[f] for f in gamma]).contiguous())
            rorc2.anchor_set(0, gamma, np.concatenate([bank_ref[f][0] for f in gamma]),
                             np.concatenate([bank_ref[f][1] for f in gamma]))
            current = gamma
        frames = fo.chunk_frames(i, B)
        q, k, v = (synth.chunk_tensor(w, t, i, 0, 0, seed=9) for t in (synth.T_Q, synth.T_K, synth.T_V))
        qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
        R2.rope3d(qd, kd, frames)
        out = R2.chunk_attention(0, 0, i, qd, kd, vd, scale=scale)
        R2.kv_publish(0, 0, i, kd, vd)
        q_ref, k_ref = oracle_rope(w, q, frames), oracle_rope(w, k, frames)
        ref = rorc2.attention(0, 0, i, q_ref, k_ref, exact(v), scale=scale)
        rorc2.publish(0, 0, i, k_ref, exact(v))
        check_attention(exact(out), ref, dtype, f"renderer chunk {i}")
