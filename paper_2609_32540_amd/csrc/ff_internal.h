// Internal interface between the host bookkeeping (ff_cache.cpp) and the HIP
// kernels of libff.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ff.h"

namespace ff {

// Keys of one attention call come as a list of segments: the anchor segment
// (or runs of consecutive frames of a caller's anchor bank), the valid history
// slots in chunk order, and the current chunk.  Token t of a segment, head h,
// element e lives at element offset
//   h * head_stride + t * tok_stride + e
// from k (and v).  Anchor and ring slots are head-major ([heads][tokens][d]);
// the current chunk and a bank are token-major ([tokens][heads][d]).
constexpr int kMaxSegments = FF_MAX_ANCHOR_FRAMES + FF_MAX_RING_CHUNKS + 1;
static_assert(kMaxSegments <= 64, "the segment table lives in one lane per segment");

struct KvSegment {
  const void* k;
  const void* v;
  int64_t head_stride;  // elements
  int32_t tok_stride;   // elements
  int32_t len;          // tokens (> 0)
};

struct KvSegments {
  KvSegment seg[kMaxSegments];
  int32_t n;
  int32_t total;  // sum of len
};

// Read sets of a batched launch (ff_chunk_attention_batch): the queries of
// item j (q[j], out[j], [nq][heads][d] each) read set[j].
constexpr int kMaxBatch = FF_MAX_BATCH;
struct KvBatch {
  KvSegments set[kMaxBatch];
  const void* q[kMaxBatch];
  void* out[kMaxBatch];
  int32_t n;
};

// Read sets of a packed launch (ff_packed_attention): one stage's chunks
// 0 .. n_chunks-1 in one token-major array, and anchor frames in another.
// Chunk c reads its anchor frames, grouped into runs of consecutive frames
// (runs[c] holds (first frame, frame count) pairs; a count of 0 ends the
// list), then chunks max(0, c - window) .. c as one run of the packed array.
struct PackedPlan {
  const void* k;            // [n_chunks * chunk_tokens][heads][d]
  const void* v;
  const void* ak;           // [n_frames * frame_tokens][heads][d]
  const void* av;
  float* lse;               // optional [n_chunks * chunk_tokens][heads]: base-2 log-sum-exp
  int32_t chunk_tokens;
  int32_t frame_tokens;
  int32_t window;
  int32_t n_chunks;
  uint8_t runs[FF_MAX_PACKED_CHUNKS][2 * FF_MAX_ANCHOR_FRAMES];
};

__host__ __device__ inline int packed_num_segments(const PackedPlan& p, int c) {
  int n = 0;
  while (n < FF_MAX_ANCHOR_FRAMES && p.runs[c][2 * n + 1] != 0) ++n;
  return n + 1;
}

// Segment i of chunk c's read set, head stride d and token stride heads * d
// elements (both arrays are token-major).
__host__ __device__ inline KvSegment packed_segment(const PackedPlan& p, int c, int i, int heads,
                                                    int d, int elem_bytes) {
  KvSegment s;
  s.head_stride = d;
  s.tok_stride = heads * d;
  const int64_t row = int64_t(heads) * d * elem_bytes;
  if (i < packed_num_segments(p, c) - 1) {
    const int first = p.runs[c][2 * i], count = p.runs[c][2 * i + 1];
    s.k = static_cast<const char*>(p.ak) + int64_t(first) * p.frame_tokens * row;
    s.v = static_cast<const char*>(p.av) + int64_t(first) * p.frame_tokens * row;
    s.len = count * p.frame_tokens;
  } else {
    const int c0 = c - p.window > 0 ? c - p.window : 0;
    s.k = static_cast<const char*>(p.k) + int64_t(c0) * p.chunk_tokens * row;
    s.v = static_cast<const char*>(p.v) + int64_t(c0) * p.chunk_tokens * row;
    s.len = (c + 1 - c0) * p.chunk_tokens;
  }
  return s;
}

// Rotation parameters of one ff_rope3d call.
struct RopeParams {
  double omega[64];                   // frequency of pair p (head_dim / 2 <= 64)
  int32_t frame_t[FF_MAX_ROPE_FRAMES];
  int32_t n_t;                        // pairs [0, n_t) use t
  int32_t n_th;                       // pairs [n_t, n_th) use the row, the rest the column
};

// Copy token-major [n_tok][heads][d] into head-major storage
// dst + h * dst_head_stride + (dst_tok0 + t) * d, for K and V in one launch.
hipError_t launch_kv_scatter(const void* k_src, const void* v_src, void* k_dst, void* v_dst,
                             int n_tok, int heads, int row_bytes, int64_t dst_head_stride_bytes,
                             hipStream_t stream);

// Inverse copy, head-major storage -> token-major [n_tok][heads][d].
hipError_t launch_kv_gather(const void* k_src, const void* v_src, void* k_dst, void* v_dst,
                            int n_tok, int heads, int row_bytes, int64_t src_head_stride_bytes,
                            hipStream_t stream);

hipError_t launch_rope3d(void* q, void* k, int n_tok, int heads, int head_dim, int dtype,
                         int grid_w, int tokens_per_frame, const RopeParams& p,
                         hipStream_t stream);

// Key split of the last, partial round of workgroups of a launch: units
// (head, 256-query tile) 0 .. n_full-1 run whole; every later unit runs as
// `split` workgroups over consecutive ranges of its key tiles, which write
// unnormalised fp32 partials (attention_bf16_part_bytes each) to `part`, and a
// merge kernel combines them.  split == 1 runs every unit whole (part unused).
struct TailSplit {
  int32_t n_full;
  int32_t split;
  float* part;
};

// Units (head, 256-query tile) of one launch and the bytes of one partial.
int attention_bf16_units(int nq, int heads);
// Key tiles a workgroup of the bf16 kernel walks over the read set segs.
int attention_bf16_key_tiles(const KvSegments& segs);
size_t attention_bf16_part_bytes(int head_dim);

hipError_t launch_attention_bf16(const void* q, void* out, int nq, int heads, int head_dim,
                                 float softmax_scale, const KvSegments& segs,
                                 const TailSplit& tail, hipStream_t stream);

hipError_t launch_attention_f32(const void* q, void* out, int nq, int heads, int head_dim,
                                float softmax_scale, const KvSegments& segs,
                                hipStream_t stream);

// Batched launches: item j of b reads b.set[j]; no tail split.
hipError_t launch_attention_bf16_batch(int nq, int heads, int head_dim, float softmax_scale,
                                       const KvBatch& b, hipStream_t stream);

hipError_t launch_attention_f32_batch(int nq, int heads, int head_dim, float softmax_scale,
                                      const KvBatch& b, hipStream_t stream);

// Packed launches: q and out are [n_chunks * chunk_tokens][heads][d]; the
// queries of chunk c read packed_segment(plan, c, .).
hipError_t launch_attention_bf16_packed(const void* q, void* out, int heads, int head_dim,
                                        float softmax_scale, const PackedPlan& plan,
                                        hipStream_t stream);

hipError_t launch_attention_f32_packed(const void* q, void* out, int heads, int head_dim,
                                       float softmax_scale, const PackedPlan& plan,
                                       hipStream_t stream);

// Backward pass of a packed launch (bf16): delta (workspace, [rows][heads]
// f32) = dO . O, then dQ, dV and dK; frame_runs[f] lists the (first chunk,
// count) runs of chunks that see anchor frame f.
hipError_t launch_attention_bwd_bf16(const void* q, const void* out, const void* dout,
                                     const float* lse, float* delta, void* dq, void* dk, void* dv,
                                     void* dak, void* dav, int heads, int head_dim,
                                     float softmax_scale, const PackedPlan& plan,
                                     const uint8_t (*frame_runs)[16], int n_frames,
                                     hipStream_t stream);

// Euler step x_out = x - dsigma * v over n elements of dtype (x_out may be x).
hipError_t launch_euler(const void* x, const void* v, void* y, int64_t n, double dsigma,
                        int dtype, hipStream_t stream);

}  // namespace ff
