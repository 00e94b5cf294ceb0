"""Benchmark of the FlashForward renderer-attention hot path on one MI355X.

One step = one chunk-stage forward of the renderer over every layer of the
workload: for each layer, 3D RoPE of the chunk's Q/K, attention of the chunk
over [anchor segment | stage-matched history ring | the chunk itself], and
publish of the chunk's K/V into the ring (plus the anchor-segment update when
the chunk enters a new anchor window).  Steps walk chunk-major through the
stages (chunk i at stages 0..S-1, then chunk i+1), starting with every ring
full, so each step is a steady-state chunk-stage.  Inputs are synthetic
(seeded N(0,1) on the device), one buffer set per layer so the 256 MB
Infinity Cache does not hold the previous layer's data.

Prints one JSON line.  `value` is attention TFLOP/s over the whole timed
region of the headline workload (attention FLOPs of every step / wall time of
the steps, RoPE and publish included).  Events recorded between the launches
of every layer inside the timed region give each kernel's average launch
duration, from which the roofline of the attention kernel is taken; its HBM
traffic comes from the counter summary under profiles/ when that summary was
taken on the current kernel source.  Beside the headline:
  configs        the same steps on the other chunk-stage workloads;
  long_horizon   the 87-chunk clip from empty rings, every chunk at every stage
                 and layer, anchor-set updates inside the timed region, timed
                 per chunk;
  kv_publish_cold / rope3d_cold  the streaming kernels on inputs that no
                 kernel has touched since the previous step;
  packed_clip_attention, wavefront_clip, cpu_baseline.
`--only` runs the named workload's timed region alone (for per-workload
kernel traces).

`--copy-calibration` instead runs only a plain device copy of 1 GiB three
times: the reference dispatch that scales the FETCH_SIZE / WRITE_SIZE counters.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import subprocess
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402
from paper_2609_32540_amd import ff  # noqa: E402

METRIC = "attention TFLOP/s + ms per chunk-stage forward (attn+publish), % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix peak (published)
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E (published)
ATTN_SOURCE = os.path.join(ROOT, "paper_2609_32540_amd", "csrc", "attn_bf16.hip")


def frames_of(w: synth.Workload, i: int):
    """Anchor frames chunk i reads under the workload's rule, from the library."""
    return ff.anchor_frames(w.anchor_rule, i, w.frames_per_chunk, w.latent_frames)


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


class Workspace:
    """Cache, per-layer input buffers and the step schedule of one workload."""

    def __init__(self, w: synth.Workload, seed: int = 0, prefill: bool = True):
        self.w = w
        dev = torch.device("cuda", 0)
        self.dev = dev
        self.cache = ff.RendererCache(stages=w.stages, layers=w.layers, ring_chunks=w.ring_chunks,
                                      frames_per_chunk=w.frames_per_chunk, grid_h=w.grid_h,
                                      grid_w=w.grid_w, heads=w.heads, head_dim=w.head_dim,
                                      max_anchor_frames=w.max_anchor_frames, dtype=w.torch_dtype,
                                      device=dev)
        g = torch.Generator(device=dev)
        g.manual_seed(seed)
        shape = (w.chunk_tokens, w.heads, w.head_dim)

        def randn(s):
            return (torch.randn(s, generator=g, device=dev, dtype=torch.float32)
                    * w.input_scale).to(w.torch_dtype)

        self.q = [randn(shape) for _ in range(w.layers)]
        self.k = [randn(shape) for _ in range(w.layers)]
        self.v = [randn(shape) for _ in range(w.layers)]
        self.out = [torch.empty(shape, dtype=w.torch_dtype, device=dev) for _ in range(w.layers)]
        a_shape = (w.max_anchor_frames * w.tokens_per_frame, w.heads, w.head_dim)
        self.anchor_k = [randn(a_shape) for _ in range(w.layers)]
        self.anchor_v = [randn(a_shape) for _ in range(w.layers)]
        self.anchor_frames = None
        # fill every ring with W chunks (chunks 0 .. W-1) so the steps run at steady state
        first = w.ring_chunks if prefill else 0
        for s in range(w.stages):
            for l in range(w.layers):
                for c in range(first):
                    self.cache.kv_publish(s, l, c, self.k[l], self.v[l])
        self.next = (first, 0)  # (chunk, stage) of the next step
        torch.cuda.synchronize()

    def kv_tokens(self, chunk: int) -> int:
        w = self.w
        n_hist = min(chunk, w.ring_chunks)
        return (len(frames_of(w, chunk)) * w.tokens_per_frame
                + n_hist * w.chunk_tokens + w.chunk_tokens)

    def attn_flops(self, chunk: int) -> float:
        w = self.w
        return 4.0 * w.chunk_tokens * self.kv_tokens(chunk) * w.head_dim * w.heads

    def step(self, events=None) -> float:
        """Enqueue one chunk-stage forward; returns its attention FLOPs (all layers)."""
        w = self.w
        chunk, stage = self.next
        frames_a = frames_of(w, chunk)
        n_a = len(frames_a) * w.tokens_per_frame
        new_window = frames_a != self.anchor_frames
        frames = [chunk * w.frames_per_chunk + f for f in range(w.frames_per_chunk)]
        for l in range(w.layers):
            if new_window:
                ak = self.anchor_k[l][:n_a]
                self.cache.rope3d(None, ak, frames_a)
                self.cache.anchor_set(l, frames_a, ak, self.anchor_v[l][:n_a])
            if events is not None:
                events[l][0].record()
            self.cache.rope3d(self.q[l], self.k[l], frames)
            if events is not None:
                events[l][1].record()
            self.cache.chunk_attention(stage, l, chunk, self.q[l], self.k[l], self.v[l], self.out[l])
            if events is not None:
                events[l][2].record()
            self.cache.kv_publish(stage, l, chunk, self.k[l], self.v[l])
            if events is not None:
                events[l][3].record()
        self.anchor_frames = frames_a
        self.next = (chunk, stage + 1) if stage + 1 < w.stages else (chunk + 1, 0)
        return self.attn_flops(chunk) * w.layers


def measured_traffic(workload: str):
    """HBM bytes per attention launch from the committed counter summary.

    The summary holds a JSON block with the SHA-256 of the kernel source the
    counters were taken on; a summary of another source gives None.
    """
    path = os.path.join(ROOT, "profiles", f"attn_bf16_{workload}_hbm_traffic.md")
    if not os.path.exists(path):
        return None, "no counter summary"
    text = open(path).read()
    try:
        block = text.split("```json", 1)[1].split("```", 1)[0]
        rec = json.loads(block)
    except (IndexError, ValueError):
        return None, "unreadable counter summary"
    sha = hashlib.sha256(open(ATTN_SOURCE, "rb").read()).hexdigest()
    if rec.get("kernel_source_sha256") != sha:
        return None, "kernel changed since the counters were taken"
    return float(rec["hbm_bytes_per_launch"]), os.path.relpath(path, ROOT)


def packed_clip(w: synth.Workload, reps: int = 3, backward: bool = True) -> dict:
    """ff_packed_attention over the workload's whole clip at one stage and layer.

    Q, K, V of all chunks in one token-major array, the anchor frames of
    every window in another; chunk i sees its window Gamma(i) and chunks
    max(0, i - W) .. i.  Seeded N(0,1) inputs drawn on the device.
    """
    dev = torch.device("cuda", 0)
    n, Nq, G = w.n_chunks, w.chunk_tokens, w.tokens_per_frame
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    shape = (n * Nq, w.heads, w.head_dim)
    q, k, v = (torch.randn(shape, generator=g, device=dev).to(w.torch_dtype) for _ in range(3))
    out = torch.empty_like(q)
    frames = sorted({f for c in range(n) for f in frames_of(w, c)})
    a_shape = (max(len(frames), 1) * G, w.heads, w.head_dim)
    ak, av = (torch.randn(a_shape, generator=g, device=dev).to(w.torch_dtype) for _ in range(2))
    table = [[frames.index(f) for f in frames_of(w, c)] for c in range(n)]
    flops = sum(4.0 * Nq * (len(table[c]) * G + (c - max(0, c - w.ring_chunks) + 1) * Nq)
                * w.head_dim * w.heads for c in range(n))

    def launch():
        ff.packed_attention(q, k, v, n_chunks=n, window=w.ring_chunks, anchor_k=ak, anchor_v=av,
                            frame_tokens=G, anchors_of_chunk=table, out=out)

    launch()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    ev[0].record(stream)
    for r in range(reps):
        launch()
        ev[r + 1].record(stream)
    torch.cuda.synchronize()
    ms = [ev[r].elapsed_time(ev[r + 1]) for r in range(reps)]
    avg = float(np.mean(ms))
    tf = flops / (avg * 1e-3) / 1e12
    log(f"packed clip attention: {n} chunks in one launch, {avg:.2f} ms = {tf:.1f} TFLOP/s")
    result = {"chunks": n, "window": w.ring_chunks, "anchor_frames_total": len(frames),
              "ms_per_launch": round(avg, 3), "tflops": round(tf, 2),
              "pct_bf16_peak": round(100 * tf / PEAK_BF16_TFLOPS, 2)}
    if backward:
        # backward of the same launch: forward with its log-sum-exp, then the four
        # backward launches; FLOPs counted as 2.5x the forward (the usual five
        # products), the kernels run seven (S and dP in each of the dQ and the
        # dK/dV pass, then dQ, dK, dV)
        lse = torch.empty((n * Nq, w.heads), dtype=torch.float32, device=dev)
        dout = torch.randn(shape, generator=g, device=dev).to(w.torch_dtype)

        def launch_lse():
            ff.packed_attention(q, k, v, n_chunks=n, window=w.ring_chunks, anchor_k=ak, anchor_v=av,
                                frame_tokens=G, anchors_of_chunk=table, out=out, lse=lse)
        # the training forward: the same launch writing its log-sum-exp
        launch_lse()
        torch.cuda.synchronize()
        evl = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        evl[0].record(stream)
        for r in range(reps):
            launch_lse()
            evl[r + 1].record(stream)
        torch.cuda.synchronize()
        lms = float(np.mean([evl[r].elapsed_time(evl[r + 1]) for r in range(reps)]))
        ltf = flops / (lms * 1e-3) / 1e12
        log(f"packed clip attention with its log-sum-exp: {lms:.2f} ms = {ltf:.1f} TFLOP/s")
        result["with_lse"] = {"ms_per_launch": round(lms, 3), "tflops": round(ltf, 2),
                              "pct_bf16_peak": round(100 * ltf / PEAK_BF16_TFLOPS, 2)}

        def bwd():
            return ff.packed_attention_bwd(q, k, v, out, dout, lse, n_chunks=n, window=w.ring_chunks,
                                           anchor_k=ak, anchor_v=av, frame_tokens=G,
                                           anchors_of_chunk=table)
        grads = bwd()
        torch.cuda.synchronize()
        del grads
        evb = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        evb[0].record(stream)
        for r in range(reps):
            grads = bwd()
            evb[r + 1].record(stream)
            del grads
        torch.cuda.synchronize()
        bms = float(np.mean([evb[r].elapsed_time(evb[r + 1]) for r in range(reps)]))
        btf = 2.5 * flops / (bms * 1e-3) / 1e12
        log(f"packed clip backward: {bms:.2f} ms = {btf:.1f} TFLOP/s (2.5x forward FLOPs), "
            f"{3.5 * flops / (bms * 1e-3) / 1e12:.1f} TFLOP/s of matrix work issued")
        result["backward"] = {"ms_per_call": round(bms, 3), "tflops_2p5x_forward": round(btf, 2),
                              "tflops_issued": round(3.5 * flops / (bms * 1e-3) / 1e12, 2),
                              "pct_bf16_peak_issued": round(100 * 3.5 * flops / (bms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2)}
        del lse, dout
    del q, k, v, out, ak, av
    torch.cuda.empty_cache()
    return result


def wavefront_clip(name: str = "1.3b-480p") -> dict:
    """One-GPU wavefront (one HIP stream per stage) against chunk-major order
    on one stream, over a whole clip of one layer of the workload.

    The forward of (stage, chunk) is a stub around the hot path: Q/K/V from
    the chunk's latent (elementwise), 3D RoPE, attention over [Gamma(i) from
    the anchor bank | the stage's ring | the chunk], publish, and the Euler
    step that hands the latent to the next stage.  Wall time of the whole
    clip, inputs resident in HBM, seeded N(0,1) on the device.
    """
    w = synth.WORKLOADS[name]
    dev = torch.device("cuda", 0)
    S, N_R, G = w.stages, w.n_chunks, w.tokens_per_frame
    sig = [1.0 - j / S for j in range(S, -1, -1)]   # sigma_0 = 0 .. sigma_S = 1
    frames = sorted({f for i in range(N_R) for f in frames_of(w, i)})
    g = torch.Generator(device=dev)
    g.manual_seed(3)
    bank_k = torch.randn((len(frames) * G, w.heads, w.head_dim), generator=g, device=dev).to(w.torch_dtype)
    bank_v = torch.randn_like(bank_k, dtype=torch.float32).to(w.torch_dtype)
    noise = [torch.randn((w.chunk_tokens, w.heads, w.head_dim), generator=g, device=dev)
             .to(w.torch_dtype) for _ in range(N_R)]
    windows = [[frames.index(f) for f in frames_of(w, i)] for i in range(N_R)]

    def run(streams):
        cache = ff.RendererCache(stages=S, layers=1, ring_chunks=w.ring_chunks,
                                 frames_per_chunk=w.frames_per_chunk, grid_h=w.grid_h,
                                 grid_w=w.grid_w, heads=w.heads, head_dim=w.head_dim,
                                 max_anchor_frames=1, dtype=w.torch_dtype, device=dev)
        X = [t.clone() for t in noise]
        torch.cuda.synchronize()

        def forward(s, i, stream):
            with torch.cuda.stream(stream):
                x = X[i]
                q, k, v = x.clone(), (x * 0.5).to(x.dtype), (x + 0.25).to(x.dtype)
                cache.rope3d(q, k, [w.frames_per_chunk * i + f for f in range(w.frames_per_chunk)],
                             stream=stream)
                h = cache.chunk_attention_bank(s, 0, i, q, k, v, bank_k, bank_v, windows[i],
                                               stream=stream)
                cache.kv_publish(s, 0, i, k, v, stream=stream)
                kk = S - s
                ff.euler_step(x, h, sig[kk] - sig[kk - 1], out=x, stream=stream)

        def batched_round(n, stream):
            # the round's forwards on one stream, their attention as one launch
            work = [(s, n - s) for s in range(S) if 0 <= n - s < N_R]
            with torch.cuda.stream(stream):
                items = []
                for s, i in work:
                    x = X[i]
                    q, k, v = x.clone(), (x * 0.5).to(x.dtype), (x + 0.25).to(x.dtype)
                    cache.rope3d(q, k, [w.frames_per_chunk * i + f for f in range(w.frames_per_chunk)],
                                 stream=stream)
                    items.append(dict(stage=s, layer=0, chunk=i, q=q, k=k, v=v, bank_k=bank_k,
                                      bank_v=bank_v, frames=windows[i]))
                outs = cache.chunk_attention_batch(items, stream=stream)
                for (s, i), it, h in zip(work, items, outs):
                    cache.kv_publish(s, 0, i, it["k"], it["v"], stream=stream)
                    kk = S - s
                    ff.euler_step(X[i], h, sig[kk] - sig[kk - 1], out=X[i], stream=stream)

        t0 = time.perf_counter()
        if streams == "batched":
            for n in range(N_R + S - 1):
                batched_round(n, one[0])
            rounds, fwd = N_R + S - 1, N_R * S
        elif len(streams) == 1:
            for i in range(N_R):
                for s in range(S):
                    forward(s, i, streams[0])
            rounds, fwd = N_R + S - 1, N_R * S
        else:
            rounds, fwd = ff.wavefront_run(N_R, streams, forward)
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        del cache
        return el, rounds, fwd, X

    one = [torch.cuda.Stream()]
    many = [torch.cuda.Stream() for _ in range(S)]
    run(one)                                   # warm: code objects and each stream's
    run(many)                                  # pool of the caching allocator
    run("batched")
    t_seq, _, _, X_seq = run(one)
    t_wave, rounds, fwd, X_wave = run(many)
    t_bat, _, _, X_bat = run("batched")
    same = all(torch.equal(a, b) for a, b in zip(X_seq, X_wave))
    same_b = all(torch.equal(a, b) for a, b in zip(X_seq, X_bat))
    log(f"wavefront {name}: {rounds} rounds, {fwd} forwards, {t_wave * 1e3:.1f} ms on {S} streams, "
        f"{t_bat * 1e3:.1f} ms with each round's attention batched on one stream, vs "
        f"{t_seq * 1e3:.1f} ms chunk-major on one stream; identical latents: {same and same_b}")
    return {"workload": name, "layers": 1, "stages": S, "chunks": N_R, "rounds": rounds,
            "forwards": fwd, "ms_wavefront_streams": round(t_wave * 1e3, 2),
            "ms_wavefront_batched_rounds": round(t_bat * 1e3, 2),
            "ms_chunk_major_one_stream": round(t_seq * 1e3, 2),
            "speedup": round(t_seq / t_wave, 3), "speedup_batched": round(t_seq / t_bat, 3),
            "latents_identical": bool(same and same_b)}


def copy_calibration() -> int:
    """Three device-to-device copies of 1 GiB (2**28 float32), nothing else."""
    n = 2 ** 28
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": 4 * n, "copy_calibration_bytes_written": 4 * n,
                      "copies": 3}), flush=True)
    return 0


def cpu_baseline(w: synth.Workload, target_s: float = 12.0) -> dict:
    """The float64 oracle's attention on 1-head x 512-query slices at the full key length."""
    from oracle import ff_oracle as fo
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    chunk = w.ring_chunks + 1
    nkv = (len(frames_of(w, chunk)) * w.tokens_per_frame
           + w.ring_chunks * w.chunk_tokens + w.chunk_tokens)
    rows = 512
    d = w.head_dim
    Q = synth.normal_rows([0, w.wid, 1000, 0, 0, synth.T_Q], rows, d, w.input_scale, w.torch_dtype)
    K = synth.normal_rows([0, w.wid, 1000, 0, 0, synth.T_K], nkv, d, w.input_scale, w.torch_dtype)
    V = synth.normal_rows([0, w.wid, 1000, 0, 0, synth.T_V], nkv, d, w.input_scale, w.torch_dtype)
    Qn, Kn, Vn = (t.float().numpy() for t in (Q, K, V))
    scale = 1.0 / math.sqrt(d)
    fo.attend(Qn[:8], Kn, Vn, scale)   # warm the BLAS threads
    n = 0
    t0 = time.perf_counter()
    while True:
        fo.attend(Qn, Kn, Vn, scale)
        n += 1
        el = time.perf_counter() - t0
        if el >= target_s or n >= 200:
            break
    flops = 4.0 * rows * nkv * d * n
    return {"value": flops / el / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n} x (1 head x {rows} queries x {nkv} keys x d {d}) of the float64 oracle "
                      f"attention, {el:.1f} s; full chunk-stage = {w.heads * w.layers} heads x "
                      f"{w.chunk_tokens} queries",
            "seconds": round(el, 2), "threads_used": int(threads), **host_cpu()}


def measure_steps(w: synth.Workload, steps: int, warmup: int) -> dict:
    """Warm-up, then `steps` timed chunk-stage steps with per-kernel events,
    then each layer's publish once more on cold inputs."""
    t0 = time.time()
    ws = Workspace(w)
    log(f"{w.name}: {ws.cache.nbytes / 2**30:.1f} GiB cache, rings filled ({time.time() - t0:.1f} s)")
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        ws.step()
    torch.cuda.synchronize()
    # timed region: the steps bracketed by events on the launch stream, with
    # events between the kernels of every layer for the per-kernel durations
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    events = [[[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(w.layers)]
              for _ in range(steps)]
    chunks, flops = [], 0.0
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(steps):
        chunks.append(ws.next[0])
        flops += ws.step(events[k])
    stop.record(stream)
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    rope_ms, attn_ms, pub_ms, attn_flops = [], [], [], []
    for k in range(steps):
        for l in range(w.layers):
            ev = events[k][l]
            rope_ms.append(ev[0].elapsed_time(ev[1]))
            attn_ms.append(ev[1].elapsed_time(ev[2]))
            pub_ms.append(ev[2].elapsed_time(ev[3]))
            attn_flops.append(ws.attn_flops(chunks[k]))
    # cold publish: each layer's K/V were last touched a whole step ago (every
    # other layer's kernels have streamed through the caches since)
    chunk, stage = ws.next
    cold = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(w.layers)]
    for l in range(w.layers):
        cold[l][0].record(stream)
        ws.cache.kv_publish(stage, l, chunk, ws.k[l], ws.v[l])
        cold[l][1].record(stream)
    torch.cuda.synchronize()
    pub_cold = float(np.mean([e[0].elapsed_time(e[1]) for e in cold]))
    # per-step durations (first event of the step's first layer to the last
    # event of its last layer) for the spread over the timed steps
    step_ms = [events[k][0][0].elapsed_time(events[k][-1][3]) for k in range(steps)]
    res = dict(ms_total=ms_total, flops=flops, chunks=chunks,
               step_ms_std=float(np.std(step_ms)), attn_ms_std=float(np.std(attn_ms)),
               attn_ms=float(np.mean(attn_ms)), pub_ms=float(np.mean(pub_ms)),
               rope_ms=float(np.mean(rope_ms)), pub_cold_ms=pub_cold,
               attn_flops=float(np.mean(attn_flops)),
               kv_tokens=ws.kv_tokens(chunks[-1]), anchor_frames=len(frames_of(w, chunks[-1])),
               cache_gib=ws.cache.nbytes / 2**30)
    del ws
    torch.cuda.empty_cache()
    return res


def stream_bytes(w: synth.Workload) -> float:
    """Algorithmic bytes of RoPE or publish on one chunk and layer: two
    [chunk_tokens][heads][head_dim] tensors read once and written once."""
    return 4.0 * w.chunk_tokens * w.heads * w.head_dim * (2 if w.dtype == "bf16" else 4)


def summarize(w: synth.Workload, m: dict, steps: int) -> dict:
    """Per-chunk-stage figures of one workload's timed steps."""
    tf = m["attn_flops"] / (m["attn_ms"] * 1e-3) / 1e12
    sb = stream_bytes(w)
    gbs = {k: sb / (m[k] * 1e-3) / 1e9 for k in ("pub_ms", "rope_ms", "pub_cold_ms")}
    target = m["attn_flops"] * w.layers / (0.5 * PEAK_BF16_TFLOPS * 1e12) * 1e3
    value = m["flops"] / (m["ms_total"] * 1e-3) / 1e12
    return {
        "workload": w.name, "heads": w.heads, "head_dim": w.head_dim,
        "grid": f"{w.grid_h}x{w.grid_w}", "chunk_tokens": w.chunk_tokens,
        "kv_tokens": m["kv_tokens"], "ring_chunks": w.ring_chunks, "stages": w.stages,
        "layers": w.layers, "anchor_frames": m["anchor_frames"], "steps": steps,
        "ms_per_step": round(m["ms_total"] / steps, 3),
        "ms_per_step_std": round(m["step_ms_std"], 3),
        "tflops_step": round(value, 2),
        "ms_attn_per_chunk_stage": round(m["attn_ms"] * w.layers, 3),
        "ms_attn_target_at_50pct_peak": round(target, 3),
        "ms_attn_publish_per_chunk_stage": round((m["attn_ms"] + m["pub_ms"]) * w.layers, 3),
        "ms_rope_per_chunk_stage": round(m["rope_ms"] * w.layers, 3),
        "attention": {"ms_per_launch": round(m["attn_ms"], 4), "ms_per_launch_std": round(m["attn_ms_std"], 4),
                      "tflops": round(tf, 2),
                      "pct_bf16_peak": round(100 * tf / PEAK_BF16_TFLOPS, 2)},
        "kv_publish": {"us_per_launch": round(m["pub_ms"] * 1e3, 2), "gbs": round(gbs["pub_ms"], 1),
                       "pct_hbm_peak": round(100 * gbs["pub_ms"] / PEAK_HBM_GBS, 2),
                       "inputs": "K/V just read by the attention launch"},
        "kv_publish_cold": {"us_per_launch": round(m["pub_cold_ms"] * 1e3, 2),
                            "gbs": round(gbs["pub_cold_ms"], 1),
                            "pct_hbm_peak": round(100 * gbs["pub_cold_ms"] / PEAK_HBM_GBS, 2),
                            "inputs": "K/V untouched since the previous step"},
        "rope3d": {"us_per_launch": round(m["rope_ms"] * 1e3, 2), "gbs": round(gbs["rope_ms"], 1),
                   "pct_hbm_peak": round(100 * gbs["rope_ms"] / PEAK_HBM_GBS, 2),
                   "inputs": "Q/K untouched since the previous step"},
    }


def long_horizon(w: synth.Workload) -> dict:
    """The whole clip from empty rings: chunk i at stages 0..S-1 over every
    layer, i = 0 .. n_chunks-1, with every anchor-set update (RoPE of the new
    anchor frames and their copy into each layer's segment) inside the timed
    region.  Events at chunk boundaries give the per-chunk series."""
    ws = Workspace(w, prefill=False)
    stream = torch.cuda.current_stream()
    # warm the code objects on a throw-away cache of the same shape
    warm = Workspace(synth.small_workload("warm", heads=w.heads, head_dim=w.head_dim, grid_h=w.grid_h,
                                          grid_w=w.grid_w, ring_chunks=w.ring_chunks, stages=1,
                                          layers=1, n_chunks=2, anchor_rule="fixed:0"))
    warm.step()
    del warm
    torch.cuda.synchronize()
    n, S = w.n_chunks, w.stages
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    flops_chunk, updates, prev = [], [], None
    ev[0].record(stream)
    for i in range(n):
        fr = frames_of(w, i)
        if fr != prev:
            updates.append(i)
            prev = fr
        f = 0.0
        for _ in range(S):
            f += ws.step()
        flops_chunk.append(f)
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(n)]
    total = float(sum(ms))
    tf = sum(flops_chunk) / (total * 1e-3) / 1e12
    kv = [ws.kv_tokens(i) for i in range(n)]
    log(f"long horizon {w.name}: {n} chunks x {S} stages x {w.layers} layers in {total:.0f} ms "
        f"= {tf:.1f} TFLOP/s, {len(updates)} anchor updates")
    del ws
    torch.cuda.empty_cache()
    return {"workload": w.name, "chunks": n, "stages": S, "layers": w.layers,
            "ms_total": round(total, 2), "tflops": round(tf, 2),
            "pct_bf16_peak": round(100 * tf / PEAK_BF16_TFLOPS, 2),
            "anchor_update_chunks": updates,
            "ms_per_chunk": [round(x, 3) for x in ms],
            "kv_tokens_per_chunk": kv,
            "note": "ms_per_chunk: all stages and layers of the chunk (RoPE, attention, publish, "
                    "and the anchor update at the listed chunks)"}


def host_cpu() -> dict:
    """CPU model and core counts of this host (lscpu), and the CPUs this
    process may run on."""
    info = {}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        kv = dict(line.split(":", 1) for line in out.splitlines() if ":" in line)
        kv = {k.strip(): v.strip() for k, v in kv.items()}
        info["cpu_model"] = kv.get("Model name")
        sockets = int(kv.get("Socket(s)", "0") or 0)
        per = int(kv.get("Core(s) per socket", "0") or 0)
        info["physical_cores"] = sockets * per if sockets and per else None
        info["logical_cpus"] = int(kv.get("CPU(s)", "0") or 0) or None
    except (OSError, ValueError, subprocess.SubprocessError):
        pass
    try:
        info["cpus_allowed"] = len(os.sched_getaffinity(0))
    except OSError:
        pass
    try:
        quota, period = open("/sys/fs/cgroup/cpu.max").read().split()
        if quota != "max":
            info["cgroup_cpu_quota"] = round(int(quota) / int(period), 2)
    except (OSError, ValueError):
        pass
    return info


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="14b-720p", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--configs", default="1.3b-480p,14b-480p",
                    help="other chunk-stage workloads to time beside the headline ('' for none)")
    ap.add_argument("--config-steps", type=int, default=4)
    ap.add_argument("--long-horizon", default="1.3b-480p-long",
                    help="workload of the per-chunk clip series ('' to skip)")
    ap.add_argument("--only", action="store_true",
                    help="time only --workload (a clip series for a long-horizon workload)")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--no-packed", action="store_true",
                    help="skip the packed whole-clip attention measurement")
    ap.add_argument("--no-wavefront", action="store_true",
                    help="skip the one-GPU wavefront measurement")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the stage-per-GPU "
              "split of the paper is not part of this build", file=sys.stderr)
        return 2
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    if args.copy_calibration:
        return copy_calibration()
    w = synth.WORKLOADS[args.workload]
    if w.dtype != "bf16":
        print("the benchmark workloads are the bf16 ones", file=sys.stderr)
        return 2
    ff.lib()
    if args.only and w.anchor_rule.startswith("flank"):
        print(json.dumps({"long_horizon": long_horizon(w)}), flush=True)
        return 0
    log(f"workload {w.name}: {w.heads} heads x {w.head_dim}, {w.chunk_tokens} queries, "
        f"{w.layers} layers, {w.stages} stages")
    m = measure_steps(w, args.steps, args.warmup)
    head = summarize(w, m, args.steps)
    value = m["flops"] / (m["ms_total"] * 1e-3) / 1e12
    attn_tf = head["attention"]["tflops"]
    log(f"timed {args.steps} steps: {head['ms_per_step']:.3f} ms/step, {value:.1f} TFLOP/s; "
        f"attention {m['attn_ms']:.3f} ms/launch = {attn_tf:.1f} TFLOP/s; publish "
        f"{head['kv_publish']['gbs']:.0f} GB/s (cold {head['kv_publish_cold']['gbs']:.0f}); "
        f"rope {head['rope3d']['gbs']:.0f} GB/s")

    traffic, traffic_src = measured_traffic(w.name)
    # compulsory bytes of one launch: Q, K, V, O of the chunk once each, every
    # history and anchor key/value once (the whole read set, all heads)
    elem = 2
    attn_bytes = elem * w.heads * w.head_dim * (2 * w.chunk_tokens + 2 * m["kv_tokens"])
    config = {k: head[k] for k in ("workload", "heads", "head_dim", "grid", "chunk_tokens",
                                   "kv_tokens", "ring_chunks", "stages", "layers",
                                   "anchor_frames")}
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "ms_per_step_std": head["ms_per_step_std"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": config,
        "pct_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "ms_attn_per_chunk_stage": head["ms_attn_per_chunk_stage"],
        "ms_attn_target_at_50pct_peak": head["ms_attn_target_at_50pct_peak"],
        "ms_attn_publish_per_chunk_stage": head["ms_attn_publish_per_chunk_stage"],
        "ms_rope_per_chunk_stage": head["ms_rope_per_chunk_stage"],
        "kernels": {k: head[k] for k in ("attention", "kv_publish", "kv_publish_cold", "rope3d")},
        "roofline": {"bound": "mfma", "achieved": attn_tf, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tf / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic, "traffic_unit": "HBM bytes per launch",
                     "traffic_source": traffic_src,
                     "algorithmic_bytes_per_launch": attn_bytes},
    }
    if not args.only:
        result["configs"] = {}
        for name in [c for c in args.configs.split(",") if c]:
            wc = synth.WORKLOADS[name]
            mc = measure_steps(wc, args.config_steps, 1)
            result["configs"][name] = summarize(wc, mc, args.config_steps)
            sc = result["configs"][name]
            log(f"{name}: attention {sc['ms_attn_per_chunk_stage']:.2f} ms per chunk-stage "
                f"({sc['attention']['pct_bf16_peak']:.1f} % of peak; target "
                f"{sc['ms_attn_target_at_50pct_peak']:.2f} ms at 50 %)")
        if args.long_horizon:
            result["long_horizon"] = long_horizon(synth.WORKLOADS[args.long_horizon])
        if not args.no_packed:
            result["packed_clip_attention"] = packed_clip(w)
        if not args.no_wavefront:
            result["wavefront_clip"] = wavefront_clip()
        if not args.no_cpu_baseline:
            log("timing the CPU oracle")
            result["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
