// Host side of libff: descriptor validation, the device layout of the cache,
// ring and anchor bookkeeping, the key-segment table of each attention call,
// and the C ABI entry points declared in include/ff.h.
//
// The history ring of (stage, layer) realises the stage-matched renderer
// history bank B_k of Sec. 3.1 (Eq. step-update): chunk c lives in slot
// c mod W, and after publishing chunks c0 .. n-1 the valid slots hold exactly
// Tail_W of that sequence.  The anchor segment of a layer is the clean anchor
// KV window read by every stage.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <atomic>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "ff.h"
#include "ff_internal.h"

namespace {

thread_local std::string g_last_error;

// No exception crosses the C ABI: the message is best effort, and entry points
// that allocate host bookkeeping run their body under no_throw().
ff_status fail(ff_status st, const char* fmt, ...) noexcept {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  try {
    g_last_error = buf;
  } catch (...) {
  }
  return st;
}

ff_status ok() noexcept {
  g_last_error.clear();
  return FF_OK;
}

template <class F>
ff_status no_throw(F&& body) noexcept {
  try {
    return body();
  } catch (...) {
    return fail(FF_ERR_INVALID_ARG, "out of host memory");
  }
}

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Layout {
  size_t elem_bytes;
  size_t tokens_per_frame;
  size_t chunk_tokens;
  size_t anchor_tokens;       // max_anchor_frames * tokens_per_frame
  size_t anchor_tensor_bytes; // one of K / V of one layer's anchor segment
  size_t slot_tensor_bytes;   // one of K / V of one ring slot
  size_t anchor_base;         // offset of layer 0's anchor K
  size_t ring_base;           // offset of (stage 0, layer 0, slot 0) K
  size_t tail_base;           // offset of stage 0's tail-split partials (bf16 only)
  size_t tail_stage_bytes;    // partials of one stage
  int tail_slots;             // partials per stage
  size_t total;
};

// Tail split: at most this many key parts per unit, and partial slots for up
// to kTailUnits units (one round of workgroups on a 256-CU device).
constexpr int kMaxTailSplit = 4;
constexpr int kTailUnits = 256;

// The descriptor as the cache uses it: all-zero rope pairs select the split of
// the Wan2.1 backbone, d/2 - 2 floor(d/6) pairs on t and floor(d/6) on each of
// h and w ((22, 21, 21) at d = 128, (12, 10, 10) at d = 64).
ff_cache_desc resolve_desc(const ff_cache_desc& in) {
  ff_cache_desc d = in;
  if (d.rope_pairs_t == 0 && d.rope_pairs_h == 0 && d.rope_pairs_w == 0 && d.head_dim > 0) {
    const int n_hw = d.head_dim / 6;
    d.rope_pairs_t = d.head_dim / 2 - 2 * n_hw;
    d.rope_pairs_h = n_hw;
    d.rope_pairs_w = n_hw;
  }
  return d;
}

ff_status check_desc(const ff_cache_desc* d) {
  if (!d) return fail(FF_ERR_INVALID_ARG, "desc is NULL");
  if (d->num_stages < 1 || d->num_layers < 1)
    return fail(FF_ERR_INVALID_ARG, "num_stages and num_layers must be >= 1");
  if (d->ring_chunks < 1 || d->ring_chunks > FF_MAX_RING_CHUNKS)
    return fail(FF_ERR_UNSUPPORTED, "ring_chunks must be in [1, %d]", FF_MAX_RING_CHUNKS);
  if (d->frames_per_chunk < 1 || d->frames_per_chunk > FF_MAX_ROPE_FRAMES)
    return fail(FF_ERR_UNSUPPORTED, "frames_per_chunk must be in [1, %d]", FF_MAX_ROPE_FRAMES);
  if (d->grid_h < 1 || d->grid_w < 1) return fail(FF_ERR_INVALID_ARG, "grid must be >= 1x1");
  if (d->num_heads < 1) return fail(FF_ERR_INVALID_ARG, "num_heads must be >= 1");
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(FF_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (d->max_anchor_frames < 0 || d->max_anchor_frames > FF_MAX_ANCHOR_FRAMES)
    return fail(FF_ERR_UNSUPPORTED, "max_anchor_frames must be in [0, %d]", FF_MAX_ANCHOR_FRAMES);
  if (d->rope_pairs_t < 0 || d->rope_pairs_h < 0 || d->rope_pairs_w < 0 ||
      d->rope_pairs_t + d->rope_pairs_h + d->rope_pairs_w != d->head_dim / 2)
    return fail(FF_ERR_INVALID_ARG, "rope pairs must be >= 0 and sum to head_dim / 2");
  if (!(d->rope_theta > 0.0) || !std::isfinite(d->rope_theta))
    return fail(FF_ERR_INVALID_ARG, "rope_theta must be positive");
  if (d->dtype != FF_DT_BF16 && d->dtype != FF_DT_F32)
    return fail(FF_ERR_UNSUPPORTED, "dtype must be FF_DT_BF16 or FF_DT_F32");
  const double tokens = double(d->grid_h) * d->grid_w * d->frames_per_chunk;
  const double anchor_tokens = double(d->grid_h) * d->grid_w * d->max_anchor_frames;
  if (tokens * d->num_heads * d->head_dim > 2.0e9 || anchor_tokens > 2.0e9 ||
      tokens * (d->ring_chunks + 1) + anchor_tokens > 2.0e9)
    return fail(FF_ERR_UNSUPPORTED, "chunk too large (element indices must fit in 32 bits)");
  return FF_OK;
}

Layout make_layout(const ff_cache_desc* d) {
  Layout L;
  L.elem_bytes = d->dtype == FF_DT_BF16 ? 2 : 4;
  L.tokens_per_frame = size_t(d->grid_h) * d->grid_w;
  L.chunk_tokens = L.tokens_per_frame * d->frames_per_chunk;
  L.anchor_tokens = L.tokens_per_frame * d->max_anchor_frames;
  const size_t row = L.elem_bytes * d->head_dim;
  L.anchor_tensor_bytes = align_up(L.anchor_tokens * d->num_heads * row);
  L.slot_tensor_bytes = align_up(L.chunk_tokens * d->num_heads * row);
  L.anchor_base = 0;
  L.ring_base = L.anchor_base + 2 * L.anchor_tensor_bytes * d->num_layers;
  L.tail_base = L.ring_base +
                2 * L.slot_tensor_bytes * size_t(d->ring_chunks) * d->num_layers * d->num_stages;
  L.tail_slots = 0;
  L.tail_stage_bytes = 0;
  if (d->dtype == FF_DT_BF16) {
    const int units = ff::attention_bf16_units(int(L.chunk_tokens), d->num_heads);
    L.tail_slots = kMaxTailSplit * std::min(units, kTailUnits);
    L.tail_stage_bytes = align_up(size_t(L.tail_slots) * ff::attention_bf16_part_bytes(d->head_dim));
  }
  L.total = L.tail_base + L.tail_stage_bytes * d->num_stages;
  return L;
}

}  // namespace

struct ff_cache {
  ff_cache_desc desc;
  Layout layout;
  char* dev;  // caller-owned device buffer
  // ring bookkeeping per (stage, layer): slot -> chunk (-1 empty), next chunk (-1 unset)
  std::vector<int64_t> slot_chunk;
  std::vector<int64_t> next_chunk;
  std::vector<int64_t> n_published;   // publishes into the ring so far
  // anchor bookkeeping per layer
  std::vector<int32_t> anchor_frames;  // [layer][max_anchor_frames]
  std::vector<int32_t> anchor_count;

  size_t ring_index(int s, int l) const { return size_t(s) * desc.num_layers + l; }
  char* anchor_k(int l) const { return dev + layout.anchor_base + 2 * layout.anchor_tensor_bytes * l; }
  char* anchor_v(int l) const { return anchor_k(l) + layout.anchor_tensor_bytes; }
  char* slot_k(int s, int l, int slot) const {
    const size_t i = (ring_index(s, l) * desc.ring_chunks + slot) * 2;
    return dev + layout.ring_base + i * layout.slot_tensor_bytes;
  }
  char* slot_v(int s, int l, int slot) const { return slot_k(s, l, slot) + layout.slot_tensor_bytes; }
  float* tail_part(int s) const {
    return reinterpret_cast<float*>(dev + layout.tail_base + size_t(s) * layout.tail_stage_bytes);
  }
  int row_bytes() const { return int(layout.elem_bytes) * desc.head_dim; }
};

namespace {

ff_status check_stage_layer(const ff_cache* c, int stage, int layer) {
  if (stage < 0 || stage >= c->desc.num_stages)
    return fail(FF_ERR_RANGE, "stage %d out of range [0, %d)", stage, c->desc.num_stages);
  if (layer < 0 || layer >= c->desc.num_layers)
    return fail(FF_ERR_RANGE, "layer %d out of range [0, %d)", layer, c->desc.num_layers);
  return FF_OK;
}

// Kernels move 16-byte vectors: every tensor pointer must be 16-byte aligned.
ff_status check_aligned(const void* p, const char* name) {
  if (reinterpret_cast<uintptr_t>(p) % 16 != 0)
    return fail(FF_ERR_INVALID_ARG, "%s must be 16-byte aligned", name);
  return FF_OK;
}

// Compute units of the current device (queried once per device; a failed
// query falls back to 256, which only affects the tail-split choice).
int device_cus() {
  static std::atomic<int> cus[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
      n = 256;
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Split of the last round of `units` equal workgroups of n_tiles key tiles
// each over `cus` compute units: the units of the partial round run as up
// to kMaxTailSplit key parts (at least 8 tiles each) when that shortens the
// round, estimated as ceil(parts / cus) / split of a whole workgroup.
ff::TailSplit choose_tail_split(int units, int n_tiles, int cus, int slots, float* part) {
  ff::TailSplit t = {units, 1, part};
  const int n_tail = units % cus;
  if (n_tail == 0 || part == nullptr) return t;
  double best = 1.0;
  for (int s = 2; s <= kMaxTailSplit; ++s) {
    if (n_tiles < 8 * s || n_tail * s > slots) break;
    const double cost = double((n_tail * s + cus - 1) / cus) / s;
    if (cost < best - 1e-9) {
      best = cost;
      t.split = s;
    }
  }
  if (t.split > 1) t.n_full = units - n_tail;
  return t;
}

ff_status hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(FF_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" {

int32_t ff_abi_version(void) { return FF_ABI_VERSION; }

size_t ff_cache_bytes(const ff_cache_desc* desc) {
  if (!desc) {
    fail(FF_ERR_INVALID_ARG, "desc is NULL");
    return 0;
  }
  const ff_cache_desc d = resolve_desc(*desc);
  if (check_desc(&d) != FF_OK) return 0;
  g_last_error.clear();
  return make_layout(&d).total;
}

ff_status ff_cache_create(const ff_cache_desc* desc, void* dev_buf, size_t dev_bytes,
                          ff_cache** out) {
  return no_throw([&]() -> ff_status {
    if (!out) return fail(FF_ERR_INVALID_ARG, "out is NULL");
    if (!desc) return fail(FF_ERR_INVALID_ARG, "desc is NULL");
    const ff_cache_desc rd = resolve_desc(*desc);
    ff_status st = check_desc(&rd);
    if (st != FF_OK) return st;
    if (!dev_buf) return fail(FF_ERR_INVALID_ARG, "dev_buf is NULL");
    if (reinterpret_cast<uintptr_t>(dev_buf) % kAlign != 0)
      return fail(FF_ERR_BUFFER, "dev_buf must be %zu-byte aligned", kAlign);
    const Layout L = make_layout(&rd);
    if (dev_bytes < L.total)
      return fail(FF_ERR_BUFFER, "dev_bytes %zu < required %zu", dev_bytes, L.total);
    std::unique_ptr<ff_cache> c(new (std::nothrow) ff_cache);
    if (!c) return fail(FF_ERR_INVALID_ARG, "out of host memory");
    c->desc = rd;
    c->layout = L;
    c->dev = static_cast<char*>(dev_buf);
    const size_t rings = size_t(rd.num_stages) * rd.num_layers;
    c->slot_chunk.assign(rings * rd.ring_chunks, -1);
    c->next_chunk.assign(rings, -1);
    c->n_published.assign(rings, 0);
    c->anchor_frames.assign(size_t(rd.num_layers) * (rd.max_anchor_frames + 1), 0);
    c->anchor_count.assign(rd.num_layers, 0);
    *out = c.release();
    return ok();
  });
}

ff_status ff_cache_destroy(ff_cache* cache) {
  delete cache;
  return ok();
}

ff_status ff_cache_get_desc(const ff_cache* cache, ff_cache_desc* out) {
  if (!cache || !out) return fail(FF_ERR_INVALID_ARG, "cache and out must be non-NULL");
  *out = cache->desc;
  return ok();
}

ff_status ff_rope3d(const ff_cache* cache, void* q, void* k, int32_t n_frames,
                    const int32_t* frame_t, void* stream) {
  if (!cache) return fail(FF_ERR_INVALID_ARG, "cache is NULL");
  if (!q && !k) return ok();
  if (n_frames < 1 || n_frames > FF_MAX_ROPE_FRAMES)
    return fail(FF_ERR_UNSUPPORTED, "n_frames must be in [1, %d]", FF_MAX_ROPE_FRAMES);
  if (!frame_t) return fail(FF_ERR_INVALID_ARG, "frame_t is NULL");
  if (check_aligned(q, "q") != FF_OK || check_aligned(k, "k") != FF_OK) return FF_ERR_INVALID_ARG;
  const ff_cache_desc& d = cache->desc;
  ff::RopeParams p;
  std::memset(&p, 0, sizeof(p));
  for (int f = 0; f < n_frames; ++f) {
    if (frame_t[f] < 0) return fail(FF_ERR_RANGE, "frame_t[%d] = %d < 0", f, frame_t[f]);
    p.frame_t[f] = frame_t[f];
  }
  p.n_t = d.rope_pairs_t;
  p.n_th = d.rope_pairs_t + d.rope_pairs_h;
  const int axis_n[3] = {d.rope_pairs_t, d.rope_pairs_h, d.rope_pairs_w};
  int pair = 0;
  for (int a = 0; a < 3; ++a)
    for (int j = 0; j < axis_n[a]; ++j)
      p.omega[pair++] = std::pow(d.rope_theta, -double(j) / double(axis_n[a]));
  const int n_tok = n_frames * d.grid_h * d.grid_w;
  hipError_t e = ff::launch_rope3d(q, k, n_tok, d.num_heads, d.head_dim, d.dtype, d.grid_w,
                                   d.grid_h * d.grid_w, p, static_cast<hipStream_t>(stream));
  return hip_status(e, "rope3d launch");
}

ff_status ff_kv_publish(ff_cache* cache, int32_t stage, int32_t layer, int64_t chunk_index,
                        const void* k, const void* v, void* stream) {
  if (!cache) return fail(FF_ERR_INVALID_ARG, "cache is NULL");
  if (!k || !v) return fail(FF_ERR_INVALID_ARG, "k and v must be non-NULL");
  if (check_aligned(k, "k") != FF_OK || check_aligned(v, "v") != FF_OK) return FF_ERR_INVALID_ARG;
  ff_status st = check_stage_layer(cache, stage, layer);
  if (st != FF_OK) return st;
  if (chunk_index < 0) return fail(FF_ERR_RANGE, "chunk_index %lld < 0", (long long)chunk_index);
  const size_t r = cache->ring_index(stage, layer);
  const int64_t expected = cache->next_chunk[r];
  if (expected >= 0 && chunk_index != expected)
    return fail(FF_ERR_ORDER, "publish of chunk %lld at (stage %d, layer %d); the ring expects %lld",
                (long long)chunk_index, stage, layer, (long long)expected);
  const int W = cache->desc.ring_chunks;
  const int slot = int(chunk_index % W);
  const ff_cache_desc& d = cache->desc;
  hipError_t e = ff::launch_kv_scatter(
      k, v, cache->slot_k(stage, layer, slot), cache->slot_v(stage, layer, slot),
      int(cache->layout.chunk_tokens), d.num_heads, cache->row_bytes(),
      int64_t(cache->layout.chunk_tokens) * cache->row_bytes(), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_status(e, "kv_publish launch");
  cache->slot_chunk[r * W + slot] = chunk_index;
  cache->next_chunk[r] = chunk_index + 1;
  ++cache->n_published[r];
  return ok();
}

ff_status ff_anchor_set(ff_cache* cache, int32_t layer, int32_t n_frames, const int32_t* frame_t,
                        const void* k, const void* v, void* stream) {
  if (!cache) return fail(FF_ERR_INVALID_ARG, "cache is NULL");
  const ff_cache_desc& d = cache->desc;
  if (layer < 0 || layer >= d.num_layers)
    return fail(FF_ERR_RANGE, "layer %d out of range [0, %d)", layer, d.num_layers);
  if (n_frames < 0 || n_frames > d.max_anchor_frames)
    return fail(FF_ERR_RANGE, "n_frames %d out of range [0, %d]", n_frames, d.max_anchor_frames);
  if (n_frames > 0 && (!k || !v || !frame_t))
    return fail(FF_ERR_INVALID_ARG, "k, v and frame_t must be non-NULL");
  if (n_frames > 0 && (check_aligned(k, "k") != FF_OK || check_aligned(v, "v") != FF_OK))
    return FF_ERR_INVALID_ARG;
  if (n_frames > 0) {
    const int n_tok = n_frames * d.grid_h * d.grid_w;
    hipError_t e = ff::launch_kv_scatter(
        k, v, cache->anchor_k(layer), cache->anchor_v(layer), n_tok, d.num_heads,
        cache->row_bytes(), int64_t(cache->layout.anchor_tokens) * cache->row_bytes(),
        static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_status(e, "anchor_set launch");
  }
  int32_t* fr = &cache->anchor_frames[size_t(layer) * (d.max_anchor_frames + 1)];
  for (int f = 0; f < n_frames; ++f) fr[f] = frame_t[f];
  cache->anchor_count[layer] = n_frames;
  return ok();
}

namespace {

// Shared body of ff_chunk_attention and ff_chunk_attention_bank.  bank_k ==
// nullptr selects the layer's anchor segment.
// Validation and read-set table of one renderer attention call (everything
// but the softmax scale and the launch).
ff_status attention_read_set(ff_cache* cache, int32_t stage, int32_t layer, int64_t chunk_index,
                             const void* q, const void* k_cur, const void* v_cur, void* out,
                             const void* bank_k, const void* bank_v, int32_t n_frames,
                             const int32_t* frame_index, ff::KvSegments* segs_out) {
  if (!cache) return fail(FF_ERR_INVALID_ARG, "cache is NULL");
  if (!q || !k_cur || !v_cur || !out)
    return fail(FF_ERR_INVALID_ARG, "q, k_cur, v_cur and out must be non-NULL");
  if (check_aligned(q, "q") != FF_OK || check_aligned(k_cur, "k_cur") != FF_OK ||
      check_aligned(v_cur, "v_cur") != FF_OK || check_aligned(out, "out") != FF_OK)
    return FF_ERR_INVALID_ARG;
  ff_status st = check_stage_layer(cache, stage, layer);
  if (st != FF_OK) return st;
  if (chunk_index < 0) return fail(FF_ERR_RANGE, "chunk_index %lld < 0", (long long)chunk_index);
  const ff_cache_desc& d = cache->desc;
  const int G = d.grid_h * d.grid_w;
  const int heads = d.num_heads;
  const int D = d.head_dim;
  // bank frames: distinct indices, grouped into runs of consecutive frames
  std::vector<std::pair<int, int>> runs;
  if (bank_k) {
    if (n_frames < 0 || n_frames > FF_MAX_ANCHOR_FRAMES)
      return fail(FF_ERR_RANGE, "n_frames %d outside [0, %d]", n_frames, FF_MAX_ANCHOR_FRAMES);
    if (n_frames > 0 && (!frame_index || !bank_v))
      return fail(FF_ERR_INVALID_ARG, "bank_v and frame_index must be non-NULL");
    if (check_aligned(bank_k, "bank_k") != FF_OK ||
        (n_frames > 0 && check_aligned(bank_v, "bank_v") != FF_OK))
      return FF_ERR_INVALID_ARG;
    std::vector<int> f(frame_index, frame_index + n_frames);
    std::sort(f.begin(), f.end());
    for (int j = 0; j < n_frames; ++j) {
      if (f[j] < 0) return fail(FF_ERR_RANGE, "frame index %d < 0", f[j]);
      if (j > 0 && f[j] == f[j - 1]) return fail(FF_ERR_INVALID_ARG, "frame %d listed twice", f[j]);
      if (!runs.empty() && runs.back().first + runs.back().second == f[j]) ++runs.back().second;
      else runs.push_back({f[j], 1});
    }
    const int64_t row = int64_t(cache->layout.elem_bytes) * heads * D;
    for (auto& rr : runs)
      if (int64_t(rr.second) * G * row > int64_t(UINT32_MAX))
        return fail(FF_ERR_UNSUPPORTED, "a run of %d bank frames spans more than 4 GiB", rr.second);
  }
  const size_t r = cache->ring_index(stage, layer);
  const int64_t expected = cache->next_chunk[r];
  if (expected >= 0 && chunk_index != expected)
    return fail(FF_ERR_ORDER,
                "attention of chunk %lld at (stage %d, layer %d); the ring holds chunks up to %lld",
                (long long)chunk_index, stage, layer, (long long)(expected - 1));
  const int W = d.ring_chunks;
  const int chunk_tokens = int(cache->layout.chunk_tokens);

  ff::KvSegments& segs = *segs_out;
  std::memset(&segs, 0, sizeof(segs));
  auto add = [&](const void* kp, const void* vp, int64_t head_stride, int tok_stride, int len) {
    ff::KvSegment& s = segs.seg[segs.n++];
    s.k = kp;
    s.v = vp;
    s.head_stride = head_stride;
    s.tok_stride = tok_stride;
    s.len = len;
    segs.total += len;
  };
  if (bank_k) {
    // bank runs: token-major
    const int64_t row = int64_t(cache->layout.elem_bytes) * heads * D;
    for (auto& rr : runs)
      add(static_cast<const char*>(bank_k) + int64_t(rr.first) * G * row,
          static_cast<const char*>(bank_v) + int64_t(rr.first) * G * row, D, heads * D,
          rr.second * G);
  } else {
    // the layer's anchor segment: head-major, max_anchor_frames * G token stride per head
    const int n_anchor = cache->anchor_count[layer];
    if (n_anchor > 0)
      add(cache->anchor_k(layer), cache->anchor_v(layer), int64_t(cache->layout.anchor_tokens) * D,
          D, n_anchor * G);
  }
  // history: chunks max(0, i - W) .. i - 1 that the ring holds, in chunk order
  for (int64_t c = chunk_index - W; c < chunk_index; ++c) {
    if (c < 0) continue;
    const int slot = int(c % W);
    if (cache->slot_chunk[r * W + slot] != c) continue;
    add(cache->slot_k(stage, layer, slot), cache->slot_v(stage, layer, slot),
        int64_t(chunk_tokens) * D, D, chunk_tokens);
  }
  // the chunk itself: token-major
  add(k_cur, v_cur, D, heads * D, chunk_tokens);
  return FF_OK;
}

ff_status check_scale(float softmax_scale) {
  if (!(softmax_scale > 0.0f) || !std::isfinite(softmax_scale))
    return fail(FF_ERR_INVALID_ARG, "softmax_scale must be positive and finite");
  return FF_OK;
}

// part / part_slots: where the tail-split partial results go (NULL: no split)
ff_status chunk_attention_impl(ff_cache* cache, int32_t stage, int32_t layer, int64_t chunk_index,
                               const void* q, const void* k_cur, const void* v_cur, void* out,
                               float softmax_scale, const void* bank_k, const void* bank_v,
                               int32_t n_frames, const int32_t* frame_index, float* part,
                               int part_slots, void* stream) {
  ff::KvSegments segs;
  ff_status st = attention_read_set(cache, stage, layer, chunk_index, q, k_cur, v_cur, out,
                                    bank_k, bank_v, n_frames, frame_index, &segs);
  if (st != FF_OK) return st;
  st = check_scale(softmax_scale);
  if (st != FF_OK) return st;
  const ff_cache_desc& d = cache->desc;
  const int heads = d.num_heads, D = d.head_dim;
  const int chunk_tokens = int(cache->layout.chunk_tokens);
  hipError_t e;
  if (d.dtype == FF_DT_BF16) {
    const ff::TailSplit tail =
        choose_tail_split(ff::attention_bf16_units(chunk_tokens, heads),
                          ff::attention_bf16_key_tiles(segs), device_cus(),
                          part_slots, part);
    e = ff::launch_attention_bf16(q, out, chunk_tokens, heads, D, softmax_scale, segs, tail,
                                  static_cast<hipStream_t>(stream));
  }
  else
    e = ff::launch_attention_f32(q, out, chunk_tokens, heads, D, softmax_scale, segs,
                                 static_cast<hipStream_t>(stream));
  return hip_status(e, "chunk_attention launch");
}

}  // namespace

ff_status ff_chunk_attention(ff_cache* cache, int32_t stage, int32_t layer, int64_t chunk_index,
                             const void* q, const void* k_cur, const void* v_cur, void* out,
                             float softmax_scale, void* stream) {
  return no_throw([&]() -> ff_status {
    if (!cache) return fail(FF_ERR_INVALID_ARG, "cache is NULL");
    const int s_ok = stage >= 0 && stage < cache->desc.num_stages;
    return chunk_attention_impl(cache, stage, layer, chunk_index, q, k_cur, v_cur, out,
                                softmax_scale, nullptr, nullptr, 0, nullptr,
                                s_ok ? cache->tail_part(stage) : nullptr,
                                cache->layout.tail_slots, stream);
  });
}

size_t ff_chunk_attention_workspace_bytes(const ff_cache* cache) {
  if (!cache) {
    fail(FF_ERR_INVALID_ARG, "cache is NULL");
    return 0;
  }
  return cache->layout.tail_stage_bytes;
}

ff_status ff_chunk_attention_ws(ff_cache* cache, int32_t stage, int32_t layer, int64_t chunk_index,
                                const void* q, const void* k_cur, const void* v_cur, void* out,
                                float softmax_scale, void* workspace, size_t workspace_bytes,
                                void* stream) {
  return no_throw([&]() -> ff_status {
    if (!cache) return fail(FF_ERR_INVALID_ARG, "cache is NULL");
    if (workspace && check_aligned(workspace, "workspace") != FF_OK) return FF_ERR_INVALID_ARG;
    int slots = 0;
    if (workspace && cache->desc.dtype == FF_DT_BF16)
      slots = int(std::min<size_t>(workspace_bytes / ff::attention_bf16_part_bytes(cache->desc.head_dim),
                                   size_t(cache->layout.tail_slots)));
    return chunk_attention_impl(cache, stage, layer, chunk_index, q, k_cur, v_cur, out,
                                softmax_scale, nullptr, nullptr, 0, nullptr,
                                slots > 0 ? static_cast<float*>(workspace) : nullptr, slots, stream);
  });
}

ff_status ff_chunk_attention_bank(ff_cache* cache, int32_t stage, int32_t layer,
                                  int64_t chunk_index, const void* q, const void* k_cur,
                                  const void* v_cur, void* out, float softmax_scale,
                                  const void* bank_k, const void* bank_v, int32_t n_frames,
                                  const int32_t* frame_index, void* stream) {
  return no_throw([&]() -> ff_status {
    if (!cache) return fail(FF_ERR_INVALID_ARG, "cache is NULL");
    if (!bank_k) return fail(FF_ERR_INVALID_ARG, "bank_k must be non-NULL");
    const int s_ok = stage >= 0 && stage < cache->desc.num_stages;
    return chunk_attention_impl(cache, stage, layer, chunk_index, q, k_cur, v_cur, out,
                                softmax_scale, bank_k, bank_v, n_frames, frame_index,
                                s_ok ? cache->tail_part(stage) : nullptr,
                                cache->layout.tail_slots, stream);
  });
}

ff_status ff_chunk_attention_batch(ff_cache* cache, int32_t n, const ff_attention_item* items,
                                   float softmax_scale, void* stream) {
  return no_throw([&]() -> ff_status {
    if (!cache) return fail(FF_ERR_INVALID_ARG, "cache is NULL");
    if (n < 1 || n > FF_MAX_BATCH)
      return fail(FF_ERR_UNSUPPORTED, "n = %d items; 1 .. %d per batch", n, FF_MAX_BATCH);
    if (!items) return fail(FF_ERR_INVALID_ARG, "items is NULL");
    ff_status st = check_scale(softmax_scale);
    if (st != FF_OK) return st;
    ff::KvBatch b;
    std::memset(&b, 0, sizeof(b));
    for (int j = 0; j < n; ++j) {
      const ff_attention_item& it = items[j];
      st = attention_read_set(cache, it.stage, it.layer, it.chunk_index, it.q, it.k_cur, it.v_cur,
                              it.out, it.bank_k, it.bank_v, it.n_frames, it.frame_index,
                              &b.set[j]);
      if (st != FF_OK) return st;
      b.q[j] = it.q;
      b.out[j] = it.out;
    }
    b.n = n;
    const ff_cache_desc& d = cache->desc;
    const int chunk_tokens = int(cache->layout.chunk_tokens);
    const hipError_t e =
        d.dtype == FF_DT_BF16
            ? ff::launch_attention_bf16_batch(chunk_tokens, d.num_heads, d.head_dim, softmax_scale,
                                              b, static_cast<hipStream_t>(stream))
            : ff::launch_attention_f32_batch(chunk_tokens, d.num_heads, d.head_dim, softmax_scale,
                                             b, static_cast<hipStream_t>(stream));
    return hip_status(e, "chunk_attention_batch launch");
  });
}

ff_status ff_cache_ring_state(const ff_cache* cache, int32_t stage, int32_t layer,
                              int64_t* slot_chunk, int64_t* next_chunk, int64_t* n_published) {
  if (!cache) return fail(FF_ERR_INVALID_ARG, "cache is NULL");
  ff_status st = check_stage_layer(cache, stage, layer);
  if (st != FF_OK) return st;
  const size_t r = cache->ring_index(stage, layer);
  const int W = cache->desc.ring_chunks;
  if (slot_chunk)
    for (int s = 0; s < W; ++s) slot_chunk[s] = cache->slot_chunk[r * W + s];
  if (next_chunk) *next_chunk = cache->next_chunk[r];
  if (n_published) *n_published = cache->n_published[r];
  return ok();
}

ff_status ff_cache_anchor_state(const ff_cache* cache, int32_t layer, int32_t* n_frames,
                                int32_t* frame_t) {
  if (!cache) return fail(FF_ERR_INVALID_ARG, "cache is NULL");
  const ff_cache_desc& d = cache->desc;
  if (layer < 0 || layer >= d.num_layers)
    return fail(FF_ERR_RANGE, "layer %d out of range [0, %d)", layer, d.num_layers);
  const int n = cache->anchor_count[layer];
  if (n_frames) *n_frames = n;
  if (frame_t)
    for (int f = 0; f < n; ++f) frame_t[f] = cache->anchor_frames[size_t(layer) * (d.max_anchor_frames + 1) + f];
  return ok();
}

ff_status ff_cache_read(const ff_cache* cache, int32_t stage, int32_t layer, int32_t slot,
                        void* k_out, void* v_out, void* stream) {
  if (!cache) return fail(FF_ERR_INVALID_ARG, "cache is NULL");
  const ff_cache_desc& d = cache->desc;
  if (layer < 0 || layer >= d.num_layers)
    return fail(FF_ERR_RANGE, "layer %d out of range [0, %d)", layer, d.num_layers);
  if (!k_out && !v_out) return ok();
  if (check_aligned(k_out, "k_out") != FF_OK || check_aligned(v_out, "v_out") != FF_OK)
    return FF_ERR_INVALID_ARG;
  const void *ks, *vs;
  int n_tok;
  int64_t head_stride_bytes;
  if (stage == -1) {
    n_tok = cache->anchor_count[layer] * d.grid_h * d.grid_w;
    ks = cache->anchor_k(layer);
    vs = cache->anchor_v(layer);
    head_stride_bytes = int64_t(cache->layout.anchor_tokens) * cache->row_bytes();
  } else {
    ff_status st = check_stage_layer(cache, stage, layer);
    if (st != FF_OK) return st;
    if (slot < 0 || slot >= d.ring_chunks)
      return fail(FF_ERR_RANGE, "slot %d out of range [0, %d)", slot, d.ring_chunks);
    n_tok = int(cache->layout.chunk_tokens);
    ks = cache->slot_k(stage, layer, slot);
    vs = cache->slot_v(stage, layer, slot);
    head_stride_bytes = int64_t(cache->layout.chunk_tokens) * cache->row_bytes();
  }
  if (n_tok == 0) return ok();
  hipError_t e = ff::launch_kv_gather(k_out ? ks : nullptr, v_out ? vs : nullptr, k_out, v_out,
                                      n_tok, d.num_heads, cache->row_bytes(), head_stride_bytes,
                                      static_cast<hipStream_t>(stream));
  return hip_status(e, "cache_read launch");
}

namespace {

// Validate a packed launch and fill its plan (anchor frames grouped into runs).
ff_status make_packed_plan(const ff_packed_desc* desc, const void* q, const void* k, const void* v,
                           const void* anchor_k, const void* anchor_v, const void* out,
                           float softmax_scale, ff::PackedPlan* plan) {
  if (!desc) return fail(FF_ERR_INVALID_ARG, "desc is NULL");
  const ff_packed_desc& d = *desc;
  if (d.n_chunks < 1 || d.n_chunks > FF_MAX_PACKED_CHUNKS)
    return fail(FF_ERR_UNSUPPORTED, "n_chunks %d outside [1, %d]", d.n_chunks, FF_MAX_PACKED_CHUNKS);
  if (d.chunk_tokens < 1 || d.num_heads < 1 || d.window < 0)
    return fail(FF_ERR_INVALID_ARG, "chunk_tokens and num_heads must be >= 1, window >= 0");
  if (d.head_dim != 64 && d.head_dim != 128)
    return fail(FF_ERR_UNSUPPORTED, "head_dim %d (64 or 128 supported)", d.head_dim);
  if (d.dtype != FF_DT_BF16 && d.dtype != FF_DT_F32)
    return fail(FF_ERR_UNSUPPORTED, "dtype %d", d.dtype);
  if (d.n_anchor_frames < 0 || d.n_anchor_frames > 255)
    return fail(FF_ERR_UNSUPPORTED, "n_anchor_frames %d outside [0, 255]", d.n_anchor_frames);
  if (d.n_anchor_frames > 0 && (d.frame_tokens < 1 || !d.anchors_of_chunk || !anchor_k || !anchor_v))
    return fail(FF_ERR_INVALID_ARG,
                "anchor frames need frame_tokens >= 1, anchors_of_chunk, anchor_k and anchor_v");
  if (!q || !k || !v || !out) return fail(FF_ERR_INVALID_ARG, "q, k, v and out must be non-NULL");
  if (check_aligned(q, "q") != FF_OK || check_aligned(k, "k") != FF_OK ||
      check_aligned(v, "v") != FF_OK || check_aligned(out, "out") != FF_OK)
    return FF_ERR_INVALID_ARG;
  if (d.n_anchor_frames > 0 &&
      (check_aligned(anchor_k, "anchor_k") != FF_OK || check_aligned(anchor_v, "anchor_v") != FF_OK))
    return FF_ERR_INVALID_ARG;
  if (!(softmax_scale > 0.0f) || !std::isfinite(softmax_scale))
    return fail(FF_ERR_INVALID_ARG, "softmax_scale must be positive and finite");
  const int64_t elem = d.dtype == FF_DT_BF16 ? 2 : 4;
  const int64_t row = elem * d.num_heads * d.head_dim;
  // the kernels address a run's rows with 32-bit byte offsets
  const int64_t window_tokens = int64_t(std::min(d.window, d.n_chunks - 1) + 1) * d.chunk_tokens;
  if (window_tokens * row > int64_t(UINT32_MAX))
    return fail(FF_ERR_UNSUPPORTED, "a chunk window of %lld tokens spans more than 4 GiB",
                (long long)window_tokens);

  ff::PackedPlan& plan_ = *plan;
  std::memset(&plan_, 0, sizeof(plan_));
  plan_.k = k;
  plan_.v = v;
  plan_.ak = anchor_k;
  plan_.av = anchor_v;
  plan_.chunk_tokens = d.chunk_tokens;
  plan_.frame_tokens = d.frame_tokens;
  plan_.window = d.window;
  plan_.n_chunks = d.n_chunks;
  for (int c = 0; c < d.n_chunks && d.n_anchor_frames > 0; ++c) {
    bool seen[256] = {false};
    for (int j = 0; j < FF_MAX_ANCHOR_FRAMES; ++j) {
      const int32_t f = d.anchors_of_chunk[c * FF_MAX_ANCHOR_FRAMES + j];
      if (f == -1) continue;
      if (f < 0 || f >= d.n_anchor_frames)
        return fail(FF_ERR_RANGE, "chunk %d lists anchor frame %d of %d", c, f, d.n_anchor_frames);
      if (seen[f]) return fail(FF_ERR_INVALID_ARG, "chunk %d lists anchor frame %d twice", c, f);
      seen[f] = true;
    }
    // runs of consecutive frames, ascending
    int n_runs = 0;
    for (int f = 0; f < d.n_anchor_frames;) {
      if (!seen[f]) { ++f; continue; }
      int e = f;
      while (e < d.n_anchor_frames && seen[e]) ++e;
      if (int64_t(e - f) * d.frame_tokens * row > int64_t(UINT32_MAX))
        return fail(FF_ERR_UNSUPPORTED, "anchor frames %d .. %d span more than 4 GiB", f, e - 1);
      plan_.runs[c][2 * n_runs] = uint8_t(f);
      plan_.runs[c][2 * n_runs + 1] = uint8_t(e - f);
      ++n_runs;
      f = e;
    }
  }
  return FF_OK;
}

}  // namespace

ff_status ff_packed_attention(const ff_packed_desc* desc, const void* q, const void* k,
                              const void* v, const void* anchor_k, const void* anchor_v,
                              void* out, float softmax_scale, float* lse, void* stream) {
  ff::PackedPlan plan;
  ff_status st = make_packed_plan(desc, q, k, v, anchor_k, anchor_v, out, softmax_scale, &plan);
  if (st != FF_OK) return st;
  const ff_packed_desc& d = *desc;
  if (lse) {
    if (d.dtype != FF_DT_BF16) return fail(FF_ERR_UNSUPPORTED, "lse is produced by the bf16 path");
    if (reinterpret_cast<uintptr_t>(lse) % 4 != 0) return fail(FF_ERR_INVALID_ARG, "lse misaligned");
  }
  plan.lse = lse;
  hipError_t e;
  if (d.dtype == FF_DT_BF16)
    e = ff::launch_attention_bf16_packed(q, out, d.num_heads, d.head_dim, softmax_scale, plan,
                                         static_cast<hipStream_t>(stream));
  else
    e = ff::launch_attention_f32_packed(q, out, d.num_heads, d.head_dim, softmax_scale, plan,
                                        static_cast<hipStream_t>(stream));
  return hip_status(e, "packed_attention launch");
}

size_t ff_packed_attention_bwd_workspace(const ff_packed_desc* desc) {
  if (!desc || desc->n_chunks < 1 || desc->chunk_tokens < 1 || desc->num_heads < 1) return 0;
  return size_t(desc->n_chunks) * desc->chunk_tokens * desc->num_heads * sizeof(float);
}

}  // extern "C"

namespace {

// Scratch of ff_packed_attention_bwd_static: rowsum(dO * O) of up to
// kStaticScratchBytes / 4 (token, head) rows.  Every device the library runs
// the entry point on holds one copy until the process ends.  In host code the
// name is only a stand-in: the device address comes from hipGetSymbolAddress.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
__device__ __align__(256) static unsigned char scratch[kStaticScratchBytes];

struct StaticScratch {
  std::once_flag once;
  void* ptr = nullptr;
  hipError_t err = hipSuccess;
};
StaticScratch g_static_scratch[64];

// Device address of `scratch` on the current device, looked up once per device.
ff_status static_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(FF_ERR_UNSUPPORTED, "device %d out of range", dev);
  StaticScratch& s = g_static_scratch[dev];
  std::call_once(s.once, [&s] {
    s.err = hipGetSymbolAddress(&s.ptr, HIP_SYMBOL(scratch));
    if (s.err == hipSuccess && s.ptr == nullptr) s.err = hipErrorInvalidSymbol;
  });
  if (s.err != hipSuccess) return hip_status(s.err, "hipGetSymbolAddress(scratch)");
  *ptr = s.ptr;
  return ok();
}

// Both backward entry points: the workspace is the caller's, or the static
// scratch of the current device when use_static is set.
ff_status packed_bwd_impl(const ff_packed_desc* desc, const void* q, const void* k,
                          const void* v, const void* anchor_k, const void* anchor_v,
                          const void* out, const void* dout, const float* lse, void* dq, void* dk,
                          void* dv, void* d_anchor_k, void* d_anchor_v, float softmax_scale,
                          void* workspace, size_t workspace_bytes, bool use_static, void* stream) {
  {
    ff::PackedPlan plan;
    ff_status st = make_packed_plan(desc, q, k, v, anchor_k, anchor_v, out, softmax_scale, &plan);
    if (st != FF_OK) return st;
    const ff_packed_desc& d = *desc;
    if (d.dtype != FF_DT_BF16) return fail(FF_ERR_UNSUPPORTED, "the backward pass is bf16 only");
    if (d.n_anchor_frames > 64)
      return fail(FF_ERR_UNSUPPORTED, "the backward pass takes at most 64 anchor frames");
    if (!dout || !lse || !dq || !dk || !dv || (!workspace && !use_static))
      return fail(FF_ERR_INVALID_ARG, "dout, lse, dq, dk, dv and workspace must be non-NULL");
    if (d.n_anchor_frames > 0 && (!d_anchor_k || !d_anchor_v))
      return fail(FF_ERR_INVALID_ARG, "d_anchor_k / d_anchor_v must be non-NULL with anchor frames");
    if (check_aligned(dout, "dout") != FF_OK || check_aligned(dq, "dq") != FF_OK ||
        check_aligned(dk, "dk") != FF_OK || check_aligned(dv, "dv") != FF_OK ||
        (!use_static && check_aligned(workspace, "workspace") != FF_OK) ||
        (d.n_anchor_frames > 0 && (check_aligned(d_anchor_k, "d_anchor_k") != FF_OK ||
                                   check_aligned(d_anchor_v, "d_anchor_v") != FF_OK)))
      return FF_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(lse) % 4 != 0) return fail(FF_ERR_INVALID_ARG, "lse misaligned");
    const size_t need = ff_packed_attention_bwd_workspace(desc);
    if (use_static && need > kStaticScratchBytes)
      return fail(FF_ERR_UNSUPPORTED,
                  "%zu bytes of scratch needed (n_chunks * chunk_tokens * num_heads floats); "
                  "the static scratch holds %zu",
                  need, kStaticScratchBytes);
    if (!use_static && workspace_bytes < need)
      return fail(FF_ERR_BUFFER, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
    // chunks that see each anchor frame, as runs of consecutive chunks
    std::array<std::array<uint8_t, 16>, 64> frame_runs;
    for (int f = 0; f < d.n_anchor_frames; ++f) {
      std::fill(frame_runs[f].begin(), frame_runs[f].end(), uint8_t(0));
      int n = 0;
      for (int c = 0; c < d.n_chunks;) {
        bool sees = false;
        for (int j = 0; j < FF_MAX_ANCHOR_FRAMES; ++j)
          sees |= d.anchors_of_chunk[c * FF_MAX_ANCHOR_FRAMES + j] == f;
        if (!sees) { ++c; continue; }
        int e = c + 1;
        for (; e < d.n_chunks; ++e) {
          bool s2 = false;
          for (int j = 0; j < FF_MAX_ANCHOR_FRAMES; ++j)
            s2 |= d.anchors_of_chunk[e * FF_MAX_ANCHOR_FRAMES + j] == f;
          if (!s2) break;
        }
        if (n == 8)
          return fail(FF_ERR_UNSUPPORTED, "anchor frame %d is seen by more than 8 runs of chunks", f);
        if (int64_t(e - c) * d.chunk_tokens * 2 * d.num_heads * d.head_dim > int64_t(UINT32_MAX))
          return fail(FF_ERR_UNSUPPORTED, "a run of chunks spans more than 4 GiB");
        frame_runs[f][2 * n] = uint8_t(c);
        frame_runs[f][2 * n + 1] = uint8_t(e - c);
        ++n;
        c = e;
      }
    }
    if (use_static) {
      st = static_scratch(&workspace);
      if (st != FF_OK) return st;
    }
    hipError_t e = ff::launch_attention_bwd_bf16(
        q, out, dout, lse, static_cast<float*>(workspace), dq, dk, dv, d_anchor_k, d_anchor_v,
        d.num_heads, d.head_dim, softmax_scale, plan,
        reinterpret_cast<const uint8_t(*)[16]>(frame_runs.data()), d.n_anchor_frames,
        static_cast<hipStream_t>(stream));
    return hip_status(e, "packed_attention_bwd launch");
  }
}

}  // namespace

extern "C" {

ff_status ff_packed_attention_bwd(const ff_packed_desc* desc, const void* q, const void* k,
                                  const void* v, const void* anchor_k, const void* anchor_v,
                                  const void* out, const void* dout, const float* lse, void* dq,
                                  void* dk, void* dv, void* d_anchor_k, void* d_anchor_v,
                                  float softmax_scale, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  return no_throw([&]() -> ff_status {
    return packed_bwd_impl(desc, q, k, v, anchor_k, anchor_v, out, dout, lse, dq, dk, dv,
                           d_anchor_k, d_anchor_v, softmax_scale, workspace, workspace_bytes,
                           false, stream);
  });
}

ff_status ff_packed_attention_bwd_static(const ff_packed_desc* desc, const void* q, const void* k,
                                         const void* v, const void* anchor_k,
                                         const void* anchor_v, const void* out, const void* dout,
                                         const float* lse, void* dq, void* dk, void* dv,
                                         void* d_anchor_k, void* d_anchor_v, float softmax_scale,
                                         void* stream) {
  return no_throw([&]() -> ff_status {
    return packed_bwd_impl(desc, q, k, v, anchor_k, anchor_v, out, dout, lse, dq, dk, dv,
                           d_anchor_k, d_anchor_v, softmax_scale, nullptr, 0, true, stream);
  });
}

ff_status ff_anchor_partition(int32_t L, int32_t delta, int32_t* out, int32_t capacity,
                              int32_t* n_out) {
  if (L < 1 || delta < 1) return fail(FF_ERR_INVALID_ARG, "L and delta must be >= 1");
  if (!n_out || (capacity > 0 && !out)) return fail(FF_ERR_INVALID_ARG, "out / n_out is NULL");
  // {m delta : m delta < L} u {L - 1}; L - 1 is new unless delta divides it
  const int32_t n_grid = (L - 1) / delta + 1;
  const int32_t n = n_grid + ((L - 1) % delta != 0 ? 1 : 0);
  *n_out = n;
  if (capacity < n) return fail(FF_ERR_BUFFER, "partition has %d entries, capacity %d", n, capacity);
  for (int32_t m = 0; m < n_grid; ++m) out[m] = m * delta;
  if (n > n_grid) out[n_grid] = L - 1;
  return ok();
}

ff_status ff_anchor_window(int64_t i, int32_t frames_per_chunk, int32_t delta, int32_t L,
                           int32_t* out3, int32_t* n_out) {
  if (i < 0 || frames_per_chunk < 1 || delta < 1 || L < 1)
    return fail(FF_ERR_INVALID_ARG, "need i >= 0, frames_per_chunk >= 1, delta >= 1, L >= 1");
  if (!out3 || !n_out) return fail(FF_ERR_INVALID_ARG, "out3 / n_out is NULL");
  const int64_t u = int64_t(frames_per_chunk) * i / (2 * int64_t(delta));
  int n = 0;
  for (int64_t m = 2 * u; m <= 2 * u + 2; ++m) {
    const int64_t f = std::min<int64_t>(m * delta, L - 1);
    if (n == 0 || out3[n - 1] != f) out3[n++] = int32_t(f);
  }
  *n_out = n;
  return ok();
}

ff_status ff_anchor_flank(int64_t i, int32_t frames_per_chunk, int32_t delta, int32_t L,
                          int32_t* out3, int32_t* n_out) {
  if (i < 0 || frames_per_chunk < 1 || delta < 1 || L < 1)
    return fail(FF_ERR_INVALID_ARG, "need i >= 0, frames_per_chunk >= 1, delta >= 1, L >= 1");
  if (!out3 || !n_out) return fail(FF_ERR_INVALID_ARG, "out3 / n_out is NULL");
  // P_j = j delta on the grid, then L - 1 once past it; indices past |P| - 1 clamp
  const int64_t n_grid = (L - 1) / delta + 1;
  const int64_t last = n_grid - 1 + ((L - 1) % delta != 0 ? 1 : 0);
  auto p = [&](int64_t j) -> int32_t {
    j = std::min(j, last);
    return j < n_grid ? int32_t(j * delta) : L - 1;
  };
  const int64_t m = int64_t(frames_per_chunk) * i / delta;
  int n = 0;
  for (int32_t f : {p(0), p(m), p(m + 1)})   // non-decreasing: p is monotone
    if (n == 0 || out3[n - 1] != f) out3[n++] = f;
  *n_out = n;
  return ok();
}

ff_status ff_euler_step(const void* x, const void* v, void* x_out, int64_t n, double dsigma,
                        int32_t dtype, void* stream) {
  if (n < 0) return fail(FF_ERR_INVALID_ARG, "n %lld < 0", (long long)n);
  if (dtype != FF_DT_BF16 && dtype != FF_DT_F32) return fail(FF_ERR_UNSUPPORTED, "dtype %d", dtype);
  if (!std::isfinite(dsigma)) return fail(FF_ERR_INVALID_ARG, "dsigma must be finite");
  if (n == 0) return ok();
  if (!x || !v || !x_out) return fail(FF_ERR_INVALID_ARG, "x, v and x_out must be non-NULL");
  if (check_aligned(x, "x") != FF_OK || check_aligned(v, "v") != FF_OK ||
      check_aligned(x_out, "x_out") != FF_OK)
    return FF_ERR_INVALID_ARG;
  const int64_t bytes = n * (dtype == FF_DT_BF16 ? 2 : 4);
  auto overlap = [&](const void* a, const void* b) {
    const char* pa = static_cast<const char*>(a);
    const char* pb = static_cast<const char*>(b);
    return pa < pb + bytes && pb < pa + bytes;
  };
  if (overlap(v, x_out) || (x != x_out && overlap(x, x_out)))
    return fail(FF_ERR_INVALID_ARG, "x_out overlaps v, or overlaps x without being x");
  return hip_status(ff::launch_euler(x, v, x_out, n, dsigma, dtype, static_cast<hipStream_t>(stream)),
                    "euler_step launch");
}

ff_status ff_wavefront_run(int64_t n_chunks, int32_t n_stages, void* const* streams,
                           ff_stage_forward_fn forward, void* user, int64_t* n_rounds,
                           int64_t* n_forwards) {
  return no_throw([&]() -> ff_status {
    if (n_chunks < 1 || n_stages < 1 || n_stages > 64)
      return fail(FF_ERR_INVALID_ARG, "need n_chunks >= 1 and 1 <= n_stages <= 64");
    if (!streams || !forward) return fail(FF_ERR_INVALID_ARG, "streams and forward must be non-NULL");
    // done[s]: rank s's latest forward (destroyed on every way out)
    struct Events {
      std::vector<hipEvent_t> e;
      ~Events() {
        for (hipEvent_t x : e)
          if (x) (void)hipEventDestroy(x);
      }
    } ev;
    ev.e.assign(n_stages, nullptr);
    std::vector<hipEvent_t>& done = ev.e;
    ff_status st = FF_OK;
    for (int s = 0; s < n_stages && st == FF_OK; ++s)
      if (hipEventCreateWithFlags(&done[s], hipEventDisableTiming) != hipSuccess)
        st = fail(FF_ERR_HIP, "hipEventCreateWithFlags failed");
    const int64_t rounds = n_chunks + n_stages - 1;
    int64_t forwards = 0;
    for (int64_t n = 0; n < rounds && st == FF_OK; ++n) {
      // ranks in descending order: rank s waits on rank s-1's forward of the same
      // chunk (round n-1) before rank s-1 records its next one in this round
      for (int s = n_stages - 1; s >= 0 && st == FF_OK; --s) {
        const int64_t i = n - s;
        if (i < 0 || i >= n_chunks) continue;
        hipStream_t hs = static_cast<hipStream_t>(streams[s]);
        if (s > 0 && hipStreamWaitEvent(hs, done[s - 1], 0) != hipSuccess) {
          st = fail(FF_ERR_HIP, "hipStreamWaitEvent failed");
          break;
        }
        const int32_t r = forward(user, s, i, streams[s]);
        if (r != FF_OK) {
          st = (r >= 1 && r <= 7) ? ff_status(r) : FF_ERR_INVALID_ARG;
          if (g_last_error.empty())
            fail(st, "forward of stage %d, chunk %lld returned %d", s, (long long)i, r);
          break;
        }
        ++forwards;
        if (hipEventRecord(done[s], hs) != hipSuccess) st = fail(FF_ERR_HIP, "hipEventRecord failed");
      }
    }
    if (st != FF_OK) return st;
    if (n_rounds) *n_rounds = rounds;
    if (n_forwards) *n_forwards = forwards;
    return ok();
  });
}

const char* ff_status_string(ff_status status) {
  switch (status) {
    case FF_OK: return "FF_OK";
    case FF_ERR_INVALID_ARG: return "FF_ERR_INVALID_ARG";
    case FF_ERR_SHAPE: return "FF_ERR_SHAPE";
    case FF_ERR_ORDER: return "FF_ERR_ORDER";
    case FF_ERR_RANGE: return "FF_ERR_RANGE";
    case FF_ERR_UNSUPPORTED: return "FF_ERR_UNSUPPORTED";
    case FF_ERR_HIP: return "FF_ERR_HIP";
    case FF_ERR_BUFFER: return "FF_ERR_BUFFER";
  }
  return "FF_ERR_UNKNOWN";
}

const char* ff_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
