// Host-only stand-ins for the kernel launchers of libff, for an AddressSanitizer
// build of the C ABI's host code (descriptor validation, ring and anchor
// bookkeeping, read-set tables, packed plans, the wavefront driver).  Nothing
// is launched; every stub checks the arguments it is given the way the real
// launcher relies on them and reports a violation as a HIP error, which the
// ABI turns into FF_ERR_HIP.  Test infrastructure only.

#include <hip/hip_runtime.h>

#include "ff_internal.h"

namespace ff {

namespace {
hipError_t check(bool ok) { return ok ? hipSuccess : hipErrorInvalidValue; }

bool segments_ok(const KvSegments& s) {
  if (s.n < 1 || s.n > kMaxSegments) return false;
  int total = 0;
  for (int i = 0; i < s.n; ++i) {
    if (s.seg[i].len <= 0 || !s.seg[i].k || !s.seg[i].v) return false;
    total += s.seg[i].len;
  }
  return total == s.total;
}
}  // namespace

int attention_bf16_units(int nq, int heads) { return heads * ((nq + 255) / 256); }

int attention_bf16_key_tiles(const KvSegments& segs) {
  int n = 0;
  for (int i = 0; i < segs.n; ++i) n += (segs.seg[i].len + 63) / 64;
  return n;
}

size_t attention_bf16_part_bytes(int head_dim) { return size_t(256) * head_dim * 4 + 2 * 256 * 4; }

hipError_t launch_kv_scatter(const void* k_src, const void* v_src, void* k_dst, void* v_dst,
                             int n_tok, int heads, int row_bytes, int64_t dst_head_stride_bytes,
                             hipStream_t) {
  return check(k_src && v_src && k_dst && v_dst && n_tok > 0 && heads > 0 && row_bytes > 0 &&
               dst_head_stride_bytes >= int64_t(n_tok) * row_bytes);
}

hipError_t launch_kv_gather(const void* k_src, const void* v_src, void* k_dst, void* v_dst,
                            int n_tok, int heads, int row_bytes, int64_t src_head_stride_bytes,
                            hipStream_t) {
  return check(k_src && v_src && k_dst && v_dst && n_tok > 0 && heads > 0 && row_bytes > 0 &&
               src_head_stride_bytes >= int64_t(n_tok) * row_bytes);
}

hipError_t launch_rope3d(void* q, void* k, int n_tok, int heads, int head_dim, int, int grid_w,
                         int tokens_per_frame, const RopeParams& p, hipStream_t) {
  return check((q || k) && n_tok > 0 && heads > 0 && (head_dim == 64 || head_dim == 128) &&
               grid_w > 0 && tokens_per_frame >= grid_w && p.n_t <= p.n_th &&
               p.n_th <= head_dim / 2);
}

hipError_t launch_attention_bf16(const void* q, void* out, int nq, int heads, int head_dim,
                                 float, const KvSegments& segs, const TailSplit& tail,
                                 hipStream_t) {
  const int units = attention_bf16_units(nq, heads);
  const bool split_ok = tail.split >= 1 && tail.split <= 4 && tail.n_full <= units &&
                        (tail.split == 1 || (tail.part != nullptr && tail.n_full < units &&
                                             attention_bf16_key_tiles(segs) >= 8 * tail.split));
  return check(q && out && nq > 0 && heads > 0 && (head_dim == 64 || head_dim == 128) &&
               segments_ok(segs) && split_ok);
}

hipError_t launch_attention_f32(const void* q, void* out, int nq, int heads, int head_dim, float,
                                const KvSegments& segs, hipStream_t) {
  return check(q && out && nq > 0 && heads > 0 && (head_dim == 64 || head_dim == 128) &&
               segments_ok(segs));
}

hipError_t launch_attention_bf16_batch(int nq, int heads, int head_dim, float, const KvBatch& b,
                                       hipStream_t) {
  bool ok = nq > 0 && heads > 0 && (head_dim == 64 || head_dim == 128) && b.n >= 1 &&
            b.n <= kMaxBatch;
  for (int j = 0; ok && j < b.n; ++j) ok = b.q[j] && b.out[j] && segments_ok(b.set[j]);
  return check(ok);
}

hipError_t launch_attention_f32_batch(int nq, int heads, int head_dim, float scale,
                                      const KvBatch& b, hipStream_t stream) {
  return launch_attention_bf16_batch(nq, heads, head_dim, scale, b, stream);
}

namespace {
bool plan_ok(const PackedPlan& p, int heads, int head_dim, int elem) {
  if (p.n_chunks < 1 || p.n_chunks > FF_MAX_PACKED_CHUNKS || p.chunk_tokens < 1) return false;
  for (int c = 0; c < p.n_chunks; ++c) {
    const int n = packed_num_segments(p, c);
    if (n < 1 || n > FF_MAX_ANCHOR_FRAMES + 1) return false;
    for (int i = 0; i < n; ++i) {
      const KvSegment s = packed_segment(p, c, i, heads, head_dim, elem);
      if (s.len <= 0 || !s.k || !s.v) return false;
    }
  }
  return true;
}
}  // namespace

hipError_t launch_attention_bf16_packed(const void* q, void* out, int heads, int head_dim, float,
                                        const PackedPlan& plan, hipStream_t) {
  return check(q && out && plan_ok(plan, heads, head_dim, 2));
}

hipError_t launch_attention_f32_packed(const void* q, void* out, int heads, int head_dim, float,
                                       const PackedPlan& plan, hipStream_t) {
  return check(q && out && plan_ok(plan, heads, head_dim, 4));
}

hipError_t launch_attention_bwd_bf16(const void* q, const void* out, const void* dout,
                                     const float* lse, float* delta, void* dq, void* dk, void* dv,
                                     void*, void*, int heads, int head_dim, float,
                                     const PackedPlan& plan, const uint8_t (*frame_runs)[16],
                                     int n_frames, hipStream_t) {
  bool ok = q && out && dout && lse && delta && dq && dk && dv && plan_ok(plan, heads, head_dim, 2);
  for (int f = 0; ok && f < n_frames; ++f)
    for (int r = 0; r < 8 && frame_runs[f][2 * r + 1] != 0; ++r)
      ok = frame_runs[f][2 * r] + frame_runs[f][2 * r + 1] <= plan.n_chunks;
  return check(ok);
}

hipError_t launch_euler(const void* x, const void* v, void* y, int64_t n, double, int, hipStream_t) {
  return check(x && v && y && n > 0);
}

}  // namespace ff
