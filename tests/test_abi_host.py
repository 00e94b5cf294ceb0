"""The C ABI library loads, exports every entry point of include/ff.h, and its
host-side validation behaves as documented.  No GPU: only calls that never
reach a kernel launch are made (the device pointer is never dereferenced by
them)."""
import ctypes
import os
import re

import pytest

from paper_2609_32540_amd import ff

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ff.h")

FAKE_DEV = 0x7f0000000000  # 256-byte aligned; only stored, never dereferenced here


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ff_[a-z0-9_]+)\s*\(", text)))


def desc(**kw):
    base = dict(num_stages=4, num_layers=2, ring_chunks=4, frames_per_chunk=3, grid_h=30,
                grid_w=52, num_heads=12, head_dim=128, max_anchor_frames=3, rope_pairs_t=22,
                rope_pairs_h=21, rope_pairs_w=21, rope_theta=10000.0, dtype=ff.FF_DT_BF16,
                reserved=0)
    base.update(kw)
    return ff.CacheDesc(**base)


def test_library_exports_every_header_symbol():
    L = ff.lib()
    names = header_functions()
    assert len(names) == 27
    for n in names:
        assert hasattr(L, n), n
    assert {n for n, _, _ in ff.SIGNATURES} == set(names)
    assert L.ff_abi_version() == ff.ABI_VERSION == 4


def test_cache_bytes_layout():
    L = ff.lib()
    d = desc()
    # anchors: layers x 2 x (3 frames x 1560 tokens x 12 heads x 128 x 2 B)
    # rings: stages x layers x W x 2 x (4680 x 12 x 128 x 2 B), all 256-aligned
    anchor = 3 * 1560 * 12 * 128 * 2
    slot = 4680 * 12 * 128 * 2
    align = lambda x: (x + 255) // 256 * 256
    # tail-split partials per stage: 4 parts x min(units, 256) units of
    # (256 x 128 + 2 x 256) floats; units = 12 heads x ceil(4680 / 256) = 228
    tail = 4 * 228 * (256 * 128 + 2 * 256) * 4
    assert L.ff_cache_bytes(ctypes.byref(d)) == (2 * 2 * align(anchor) + 4 * 2 * 4 * 2 * align(slot)
                                                 + 4 * align(tail))
    assert L.ff_cache_bytes(ctypes.byref(desc(dtype=ff.FF_DT_F32))) == (
        2 * 2 * align(2 * anchor) + 4 * 2 * 4 * 2 * align(2 * slot))
    # C5-shaped, all 4 stages x 40 layers: ~150 GB fits one MI355X
    d5 = desc(num_layers=40, grid_h=45, grid_w=80, num_heads=40)
    assert 140e9 < L.ff_cache_bytes(ctypes.byref(d5)) < 160e9


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, 5), ("ring_chunks", 0, 5), ("ring_chunks", 9, 5), ("dtype", 7, 5),
    ("rope_pairs_t", 21, 1), ("num_heads", 0, 1), ("max_anchor_frames", 9, 5),
    ("rope_theta", -1.0, 1), ("grid_w", 0, 1),
])
def test_invalid_desc_rejected(field, value, status):
    L = ff.lib()
    d = desc(**{field: value})
    assert L.ff_cache_bytes(ctypes.byref(d)) == 0
    h = ctypes.c_void_p()
    assert L.ff_cache_create(ctypes.byref(d), FAKE_DEV, 1 << 40, ctypes.byref(h)) == status
    assert L.ff_last_error()


def make_handle(**kw):
    L = ff.lib()
    d = desc(**kw)
    n = L.ff_cache_bytes(ctypes.byref(d))
    h = ctypes.c_void_p()
    assert L.ff_cache_create(ctypes.byref(d), FAKE_DEV, n, ctypes.byref(h)) == 0
    return L, h, n


def test_create_checks_buffer():
    L = ff.lib()
    d = desc()
    n = L.ff_cache_bytes(ctypes.byref(d))
    h = ctypes.c_void_p()
    assert L.ff_cache_create(ctypes.byref(d), FAKE_DEV, n - 1, ctypes.byref(h)) == 7
    assert L.ff_cache_create(ctypes.byref(d), FAKE_DEV + 16, n, ctypes.byref(h)) == 7
    assert L.ff_cache_create(ctypes.byref(d), None, n, ctypes.byref(h)) == 1


def test_fresh_cache_state_and_host_validation():
    L, h, _ = make_handle()
    slots = (ctypes.c_int64 * 4)()
    cnt, nxt = ctypes.c_int64(-5), ctypes.c_int64(-5)
    assert L.ff_cache_ring_state(h, 3, 1, slots, ctypes.byref(nxt), ctypes.byref(cnt)) == 0
    assert list(slots) == [-1] * 4 and cnt.value == 0 and nxt.value == -1
    assert L.ff_cache_ring_state(h, 4, 0, slots, None, ctypes.byref(cnt)) == 4   # stage range
    assert L.ff_cache_ring_state(h, 0, 2, slots, None, ctypes.byref(cnt)) == 4   # layer range
    nfr = ctypes.c_int32(-1)
    assert L.ff_cache_anchor_state(h, 0, ctypes.byref(nfr), None) == 0 and nfr.value == 0
    dummy = FAKE_DEV
    # publish / attention argument checks happen before any launch
    assert L.ff_kv_publish(h, 9, 0, 0, dummy, dummy, None) == 4
    assert L.ff_kv_publish(h, 0, 0, -1, dummy, dummy, None) == 4
    assert L.ff_kv_publish(h, 0, 0, 0, None, dummy, None) == 1
    assert L.ff_chunk_attention(h, 0, 0, 0, dummy, dummy, dummy, None, 0.1, None) == 1
    assert L.ff_chunk_attention(h, 0, 0, 0, dummy, dummy, dummy, dummy, 0.0, None) == 1
    assert L.ff_chunk_attention(h, 0, 0, 0, dummy, dummy, dummy, dummy, float("nan"), None) == 1
    assert L.ff_chunk_attention(h, 0, 5, 0, dummy, dummy, dummy, dummy, 0.1, None) == 4
    ft = (ctypes.c_int32 * 4)(0, 10, 20, 30)
    assert L.ff_anchor_set(h, 0, 4, ft, dummy, dummy, None) == 4        # > max_anchor_frames
    assert L.ff_anchor_set(h, 0, 2, ft, None, dummy, None) == 1
    assert L.ff_rope3d(h, dummy, None, 0, ft, None) == 5
    assert L.ff_rope3d(h, dummy, None, 17, ft, None) == 5
    neg = (ctypes.c_int32 * 1)(-3)
    assert L.ff_rope3d(h, dummy, None, 1, neg, None) == 4
    assert L.ff_cache_read(h, 0, 0, 4, dummy, dummy, None) == 4
    # misaligned tensors are rejected before any launch
    assert L.ff_kv_publish(h, 0, 0, 0, dummy + 8, dummy, None) == 1
    assert L.ff_chunk_attention(h, 0, 0, 0, dummy, dummy, dummy + 2, dummy, 0.1, None) == 1
    assert L.ff_rope3d(h, dummy + 4, None, 1, ft, None) == 1
    # anchor_set with 0 frames clears without launching anything
    assert L.ff_anchor_set(h, 1, 0, None, None, None, None) == 0
    # state unchanged by the failed calls
    assert L.ff_cache_ring_state(h, 0, 0, slots, ctypes.byref(nxt), ctypes.byref(cnt)) == 0
    assert list(slots) == [-1] * 4 and cnt.value == 0 and nxt.value == -1
    # the workspace variant validates like ff_chunk_attention; its size is one stage's partials
    assert L.ff_chunk_attention_ws(h, 0, 5, 0, dummy, dummy, dummy, dummy, 0.1, None, 0, None) == 4
    assert L.ff_chunk_attention_ws(h, 0, 0, 0, dummy, dummy, dummy, dummy, 0.1, dummy + 4, 64,
                                   None) == 1
    assert L.ff_chunk_attention_workspace_bytes(h) == 4 * 228 * (256 * 128 + 2 * 256) * 4
    assert L.ff_chunk_attention_workspace_bytes(None) == 0
    assert L.ff_cache_destroy(h) == 0
    assert L.ff_cache_destroy(None) == 0


def test_status_strings():
    L = ff.lib()
    for code, name in ff.STATUS_NAMES.items():
        assert L.ff_status_string(code).decode() == name


# ----------------------------------------------------------------------
# ff_packed_attention: host validation (every case fails before a launch)

def packed_desc(**kw):
    base = dict(n_chunks=6, chunk_tokens=192, num_heads=2, head_dim=64, window=2, frame_tokens=64,
                n_anchor_frames=0, dtype=ff.FF_DT_BF16, anchors_of_chunk=None)
    base.update(kw)
    return ff.PackedDesc(**base)


def packed_call(d, q=FAKE_DEV, k=FAKE_DEV, v=FAKE_DEV, ak=None, av=None, out=FAKE_DEV, scale=0.125):
    L = ff.lib()
    return L.ff_packed_attention(ctypes.byref(d) if d is not None else None, q, k, v, ak, av, out,
                                 ctypes.c_float(scale), None, None)


def table(rows):
    flat = [-1] * (len(rows) * ff.MAX_ANCHOR_FRAMES)
    for i, r in enumerate(rows):
        for j, f in enumerate(r):
            flat[i * ff.MAX_ANCHOR_FRAMES + j] = f
    arr = (ctypes.c_int32 * len(flat))(*flat)
    return arr, ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32))


@pytest.mark.parametrize("kw,status", [
    (dict(n_chunks=0), 5), (dict(n_chunks=129), 5), (dict(chunk_tokens=0), 1),
    (dict(num_heads=0), 1), (dict(window=-1), 1), (dict(head_dim=96), 5), (dict(dtype=3), 5),
    (dict(n_anchor_frames=256), 5), (dict(n_anchor_frames=2), 1),   # no table / pointers
])
def test_packed_desc_rejected(kw, status):
    assert packed_call(packed_desc(**kw)) == status
    assert ff.lib().ff_last_error().decode()


def test_packed_pointer_and_table_validation():
    assert packed_call(None) == 1
    assert packed_call(packed_desc(), q=None) == 1
    assert packed_call(packed_desc(), out=FAKE_DEV + 8) == 1          # misaligned
    assert packed_call(packed_desc(), scale=0.0) == 1
    arr, ptr = table([[0, 1]] * 6)
    ok_anchor = dict(n_anchor_frames=2, anchors_of_chunk=ptr)
    assert packed_call(packed_desc(**ok_anchor), ak=FAKE_DEV, av=FAKE_DEV + 8) == 1
    arr2, ptr2 = table([[0, 1]] * 5 + [[1, 1]])                       # a frame listed twice
    assert packed_call(packed_desc(n_anchor_frames=2, anchors_of_chunk=ptr2), ak=FAKE_DEV,
                       av=FAKE_DEV) == 1
    arr3, ptr3 = table([[0, 2]] * 6)                                  # frame 2 of 2
    assert packed_call(packed_desc(n_anchor_frames=2, anchors_of_chunk=ptr3), ak=FAKE_DEV,
                       av=FAKE_DEV) == 4
    # a chunk window wider than 4 GiB of bytes
    big = packed_desc(n_chunks=8, chunk_tokens=1 << 20, num_heads=40, head_dim=128, window=4)
    assert packed_call(big) == 5


def test_static_backward_rejects_inputs_beyond_its_scratch():
    # rowsum(dO * O) of 64 x 10800 x 40 (token, head) rows is 105 MiB, beyond the
    # 64 MiB static scratch: rejected on the host, before any device call
    L = ff.lib()
    lse = ctypes.cast(FAKE_DEV, ctypes.c_void_p)

    def call(d):
        return L.ff_packed_attention_bwd_static(ctypes.byref(d), FAKE_DEV, FAKE_DEV, FAKE_DEV, None,
                                                None, FAKE_DEV, FAKE_DEV, lse, FAKE_DEV, FAKE_DEV,
                                                FAKE_DEV, None, None, ctypes.c_float(0.125), None)
    big = packed_desc(n_chunks=64, chunk_tokens=10800, num_heads=40, head_dim=128, window=4)
    assert call(big) == 5
    assert "static scratch" in L.ff_last_error().decode()
    assert call(packed_desc(dtype=ff.FF_DT_F32)) == 5                 # bf16 only, as the other entry
    assert call(packed_desc(head_dim=96)) == 5
    # the backward's per-frame tables: at most 64 anchor frames, each seen by at
    # most 8 runs of consecutive chunks
    def call_anchors(d):
        return L.ff_packed_attention_bwd_static(ctypes.byref(d), FAKE_DEV, FAKE_DEV, FAKE_DEV,
                                                FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV, lse, FAKE_DEV,
                                                FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV,
                                                ctypes.c_float(0.125), None)
    arr, ptr = table([[0]] * 6)
    assert call_anchors(packed_desc(n_anchor_frames=65, anchors_of_chunk=ptr)) == 5
    assert "64 anchor frames" in L.ff_last_error().decode()
    arr9, ptr9 = table([[0] if c % 2 == 0 else [] for c in range(18)])   # 9 runs of frame 0
    assert call_anchors(packed_desc(n_chunks=18, n_anchor_frames=1, anchors_of_chunk=ptr9)) == 5
    assert "more than 8 runs" in L.ff_last_error().decode()


# ----------------------------------------------------------------------
# planner-side index sets: the C helpers against the oracle

def test_anchor_partition_matches_oracle():
    from oracle import ff_oracle as fo
    for L in list(range(1, 70)) + [81, 161, 261, 321]:
        for delta in (1, 2, 3, 7, 10, 24):
            assert ff.anchor_partition(L, delta) == fo.anchor_partition(L, delta), (L, delta)
    n = ctypes.c_int32()
    buf = (ctypes.c_int32 * 2)()
    assert ff.lib().ff_anchor_partition(261, 10, buf, 2, ctypes.byref(n)) == 7  # too small
    assert n.value == 27
    assert ff.lib().ff_anchor_partition(0, 10, buf, 2, ctypes.byref(n)) == 1


def test_anchor_window_matches_oracle():
    from oracle import ff_oracle as fo
    for L in (18, 21, 81, 261):
        for B_R in (1, 3, 4):
            for delta in (5, 10):
                for i in range(0, -(-L // B_R) + 3):
                    assert ff.anchor_window(i, B_R, delta, L) == fo.anchor_window(i, B_R, delta, L)
    out = (ctypes.c_int32 * 3)()
    n = ctypes.c_int32()
    assert ff.lib().ff_anchor_window(-1, 3, 10, 261, out, ctypes.byref(n)) == 1


def test_anchor_flank_matches_oracle():
    from oracle import ff_oracle as fo
    for L in (1, 2, 18, 21, 81, 261):
        for B_R in (1, 3, 4):
            for delta in (1, 5, 10, 24):
                for i in range(0, -(-L // B_R) + 3):
                    assert ff.anchor_flank(i, B_R, delta, L) == fo.anchor_flank(i, B_R, delta, L), \
                        (L, B_R, delta, i)
    out = (ctypes.c_int32 * 3)()
    n = ctypes.c_int32()
    assert ff.lib().ff_anchor_flank(-1, 3, 24, 261, out, ctypes.byref(n)) == 1
    assert ff.lib().ff_anchor_flank(0, 3, 0, 261, out, ctypes.byref(n)) == 1
    assert ff.lib().ff_anchor_flank(0, 3, 24, 261, None, ctypes.byref(n)) == 1


def test_workload_anchor_rules_library_equals_oracle():
    # the benchmark takes each chunk's anchor frames from the library, the GPU
    # tests from the oracle: both readings agree on every chunk of every workload
    import synth
    from oracle import ff_oracle as fo
    for w in synth.WORKLOADS.values():
        for i in range(w.n_chunks):
            assert ff.anchor_frames(w.anchor_rule, i, w.frames_per_chunk, w.latent_frames) == \
                fo.anchor_frames(w.anchor_rule, i, w.frames_per_chunk, w.latent_frames), (w.name, i)


def test_euler_and_wavefront_host_validation():
    L = ff.lib()
    assert L.ff_euler_step(FAKE_DEV, FAKE_DEV + 4096, FAKE_DEV, -1, 0.5, 0, None) == 1
    assert L.ff_euler_step(FAKE_DEV, FAKE_DEV + 4096, FAKE_DEV, 8, 0.5, 9, None) == 5
    assert L.ff_euler_step(FAKE_DEV, FAKE_DEV + 4096, FAKE_DEV, 8, float("nan"), 0, None) == 1
    assert L.ff_euler_step(FAKE_DEV, FAKE_DEV + 8, FAKE_DEV + 4096, 8, 0.5, 0, None) == 1  # misaligned v
    assert L.ff_euler_step(FAKE_DEV, FAKE_DEV + 4096, FAKE_DEV + 4096 + 16, 64, 0.5, 0, None) == 1  # out overlaps v
    assert L.ff_euler_step(FAKE_DEV, FAKE_DEV + 4096, FAKE_DEV + 16, 64, 0.5, 0, None) == 1  # out overlaps x
    assert L.ff_euler_step(None, None, None, 0, 0.5, 0, None) == 0                          # empty
    calls = []
    fn = ff.STAGE_FORWARD_FN(lambda u, s, c, st: calls.append((s, c)) or 0)
    arr = (ctypes.c_void_p * 2)(None, None)
    r, f = ctypes.c_int64(), ctypes.c_int64()
    assert L.ff_wavefront_run(0, 2, arr, fn, None, ctypes.byref(r), ctypes.byref(f)) == 1
    assert L.ff_wavefront_run(3, 0, arr, fn, None, ctypes.byref(r), ctypes.byref(f)) == 1
    assert not calls


@pytest.mark.parametrize("head_dim", [64, 128])
def test_rope_split_default_lives_in_the_library(head_dim):
    # all-zero rope pairs select the backbone's split inside the library; it equals
    # the oracle's reading of the paper's (22, 21, 21) split for every head size
    from oracle import ff_oracle as fo
    L, h, _ = make_handle(head_dim=head_dim, rope_pairs_t=0, rope_pairs_h=0, rope_pairs_w=0)
    got = ff.CacheDesc()
    assert L.ff_cache_get_desc(h, ctypes.byref(got)) == 0
    assert (got.rope_pairs_t, got.rope_pairs_h, got.rope_pairs_w) == fo.rope_pair_split(head_dim)
    assert got.head_dim == head_dim and got.num_heads == 12
    assert L.ff_cache_destroy(h) == 0
    # an explicit split is kept as given, and a wrong sum is still rejected
    L, h, _ = make_handle(head_dim=head_dim, rope_pairs_t=head_dim // 2, rope_pairs_h=0,
                          rope_pairs_w=0)
    assert L.ff_cache_get_desc(h, ctypes.byref(got)) == 0
    assert (got.rope_pairs_t, got.rope_pairs_h, got.rope_pairs_w) == (head_dim // 2, 0, 0)
    assert L.ff_cache_destroy(h) == 0
    bad = desc(head_dim=head_dim, rope_pairs_t=1, rope_pairs_h=0, rope_pairs_w=0)
    assert L.ff_cache_bytes(ctypes.byref(bad)) == 0
    assert L.ff_cache_get_desc(None, ctypes.byref(got)) == 1
