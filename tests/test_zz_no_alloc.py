"""ff_packed_attention_bwd_static (the backward with its scratch in the
library's static device array) against ff_packed_attention_bwd with a caller
workspace: the same kernels on the same inputs, so every gradient must be
bit-identical.  Two calls in a row on one device, the second with a smaller
input, so the second reuses the scratch the first left behind; the first is
also checked against the oracle's gradient (App. Alg. 2, backward of the
packed renderer rows)."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

from oracle import ff_oracle as fo
from paper_2609_32540_amd import ff

from gpu_util import exact, rel_l2

pytestmark = pytest.mark.gpu

GRAD_REL_L2 = 1e-2


def _case(n, Nq, G, frames, W, heads, d, seed):
    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)

    def rnd(shape):
        return torch.randn(shape, generator=g, device=dev).to(torch.bfloat16)
    table = [[j for j in range(frames) if (i + j) % 3 != 2] for i in range(n)]
    q, k, v, dout = (rnd((n * Nq, heads, d)) for _ in range(4))
    ak, av = rnd((frames * G, heads, d)), rnd((frames * G, heads, d))
    kw = dict(n_chunks=n, window=W, anchor_k=ak, anchor_v=av, frame_tokens=G,
              anchors_of_chunk=table, scale=1.0 / math.sqrt(d))
    lse = torch.empty((n * Nq, heads), dtype=torch.float32, device=dev)
    out = ff.packed_attention(q, k, v, lse=lse, **kw)
    return (q, k, v, out, dout, lse), kw, table


def _static_call(args, kw):
    q, k, v = args[:3]
    # gradients start as NaN so that an element the call does not write shows
    grads = [torch.full_like(t, float("nan")) for t in (q, k, v, kw["anchor_k"], kw["anchor_v"])]
    ff.packed_attention_bwd_static(*args, *grads, **kw)
    return grads


def test_static_scratch_backward_matches_workspace_backward():
    cases = [dict(n=5, Nq=200, G=40, frames=3, W=2, heads=3, d=128, seed=11),
             dict(n=3, Nq=72, G=24, frames=2, W=1, heads=2, d=64, seed=12)]   # smaller
    for ci, c in enumerate(cases):
        args, kw, table = _case(**c)
        ref = ff.packed_attention_bwd(*args, **kw)
        got = _static_call(args, kw)
        torch.cuda.synchronize()
        for name, a, b in zip(("dq", "dk", "dv", "d_anchor_k", "d_anchor_v"), got, ref):
            assert torch.equal(a, b), f"call {ci}: {name} differs from the workspace entry point"
        if ci == 0:
            q, k, v, out, dout, lse = args
            n, Nq, G, frames, W = c["n"], c["Nq"], c["G"], c["frames"], c["W"]
            M = fo.packed_visibility(n, Nq, G, frames, table, W)
            K_all = np.concatenate([exact(kw["anchor_k"]), exact(k)])
            V_all = np.concatenate([exact(kw["anchor_v"]), exact(v)])
            rdq, rdk, rdv = fo.masked_attention_grad(exact(q), K_all, V_all, M, exact(dout),
                                                     kw["scale"])
            na = frames * G
            for name, g_, r in (("dq", got[0], rdq), ("dk", got[1], rdk[na:]),
                                ("dv", got[2], rdv[na:]), ("d_anchor_k", got[3], rdk[:na]),
                                ("d_anchor_v", got[4], rdv[:na])):
                assert rel_l2(exact(g_), r) <= GRAD_REL_L2, name
