// Internal interface between the host bookkeeping (ff_cache.cpp) and the HIP
// kernels of libff.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ff.h"

namespace ff {

// Keys of one attention call come as a list of segments: the anchor segment,
// the valid history slots in chunk order, and the current chunk.  Token t of a
// segment, head h, element e lives at element offset
//   h * head_stride + t * tok_stride + e
// from k (and v).  Anchor and ring slots are head-major ([heads][tokens][d]);
// the current chunk is token-major ([tokens][heads][d]).
constexpr int kMaxSegments = 2 + FF_MAX_RING_CHUNKS;

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

hipError_t launch_attention_bf16(const void* q, void* out, int nq, int heads, int head_dim,
                                 float softmax_scale, const KvSegments& segs,
                                 hipStream_t stream);

hipError_t launch_attention_f32(const void* q, void* out, int nq, int heads, int head_dim,
                                float softmax_scale, const KvSegments& segs,
                                hipStream_t stream);

}  // namespace ff
