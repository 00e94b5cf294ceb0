// Float32 renderer attention (the fp32 workloads): one thread per query, key
// tiles staged in LDS, online softmax in float32 with expf.  Small sizes
// only; the bf16 kernel is the fast path.
//
// Launch shape: grid (ceil(nq / 128), heads, sets), 128 threads; the read
// set is one KvSegments for the launch, for a packed clip the PackedPlan
// segments of chunk blockIdx.z, for a batch the set of item blockIdx.z.

#include <hip/hip_runtime.h>

#include <math.h>

#include "ff_internal.h"

namespace ff {
namespace {

constexpr int kThreads = 128;
constexpr int kTileK = 32;

template <int D, class Src>
__global__ __launch_bounds__(kThreads) void attn_f32_kernel(const float* __restrict__ q,
                                                            float* __restrict__ out, int nq,
                                                            int heads, float scale, Src src) {
  constexpr bool kPacked = __is_same(Src, PackedPlan);
  constexpr bool kBatch = __is_same(Src, KvBatch);
  const int chunk = blockIdx.z;
  if constexpr (kBatch) {
    q = static_cast<const float*>(src.q[chunk]);
    out = static_cast<float*>(src.out[chunk]);
  } else {
    q += int64_t(chunk) * nq * heads * D;
    out += int64_t(chunk) * nq * heads * D;
  }
  __shared__ float ks[kTileK][D];
  __shared__ float vs[kTileK][D];
  const int head = blockIdx.y;
  const int qi = blockIdx.x * kThreads + threadIdx.x;
  const int qrow = min(qi, nq - 1);

  float qv[D], o[D];
  const float* qp = q + (int64_t(qrow) * heads + head) * D;
#pragma unroll
  for (int e = 0; e < D; ++e) {
    qv[e] = qp[e] * scale;
    o[e] = 0.0f;
  }
  float m = -INFINITY, l = 0.0f;

  int n_segs;
  if constexpr (kPacked) n_segs = packed_num_segments(src, chunk);
  else if constexpr (kBatch) n_segs = src.set[chunk].n;
  else n_segs = src.n;
  for (int sg = 0; sg < n_segs; ++sg) {
    KvSegment seg;
    if constexpr (kPacked) seg = packed_segment(src, chunk, sg, heads, D, 4);
    else if constexpr (kBatch) seg = src.set[chunk].seg[sg];
    else seg = src.seg[sg];
    const float* kb = static_cast<const float*>(seg.k) + head * seg.head_stride;
    const float* vb = static_cast<const float*>(seg.v) + head * seg.head_stride;
    for (int k0 = 0; k0 < seg.len; k0 += kTileK) {
      const int n = min(kTileK, seg.len - k0);
      __syncthreads();
      for (int e = threadIdx.x; e < n * D; e += kThreads) {
        const int r = e / D, c = e % D;
        const int64_t off = int64_t(k0 + r) * seg.tok_stride + c;
        ks[r][c] = kb[off];
        vs[r][c] = vb[off];
      }
      __syncthreads();
      for (int j = 0; j < n; ++j) {
        float s = 0.0f;
#pragma unroll
        for (int e = 0; e < D; ++e) s = fmaf(qv[e], ks[j][e], s);
        if (s > m) {
          const float alpha = expf(m - s);
          l *= alpha;
#pragma unroll
          for (int e = 0; e < D; ++e) o[e] *= alpha;
          m = s;
        }
        const float p = expf(s - m);
        l += p;
#pragma unroll
        for (int e = 0; e < D; ++e) o[e] = fmaf(p, vs[j][e], o[e]);
      }
    }
  }
  if (qi < nq) {
    const float inv = 1.0f / l;
    float* op = out + (int64_t(qi) * heads + head) * D;
#pragma unroll
    for (int e = 0; e < D; ++e) op[e] = o[e] * inv;
  }
}

}  // namespace

hipError_t launch_attention_f32(const void* q, void* out, int nq, int heads, int head_dim,
                                float softmax_scale, const KvSegments& segs, hipStream_t stream) {
  if (nq <= 0) return hipSuccess;
  dim3 grid((nq + kThreads - 1) / kThreads, heads, 1);
  if (head_dim == 64)
    hipLaunchKernelGGL((attn_f32_kernel<64, KvSegments>), grid, dim3(kThreads), 0, stream,
                       static_cast<const float*>(q), static_cast<float*>(out), nq, heads,
                       softmax_scale, segs);
  else
    hipLaunchKernelGGL((attn_f32_kernel<128, KvSegments>), grid, dim3(kThreads), 0, stream,
                       static_cast<const float*>(q), static_cast<float*>(out), nq, heads,
                       softmax_scale, segs);
  return hipGetLastError();
}

hipError_t launch_attention_f32_batch(int nq, int heads, int head_dim, float softmax_scale,
                                      const KvBatch& b, hipStream_t stream) {
  if (nq <= 0 || b.n <= 0) return hipSuccess;
  dim3 grid((nq + kThreads - 1) / kThreads, heads, b.n);
  if (head_dim == 64)
    hipLaunchKernelGGL((attn_f32_kernel<64, KvBatch>), grid, dim3(kThreads), 0, stream, nullptr,
                       nullptr, nq, heads, softmax_scale, b);
  else
    hipLaunchKernelGGL((attn_f32_kernel<128, KvBatch>), grid, dim3(kThreads), 0, stream, nullptr,
                       nullptr, nq, heads, softmax_scale, b);
  return hipGetLastError();
}

hipError_t launch_attention_f32_packed(const void* q, void* out, int heads, int head_dim,
                                       float softmax_scale, const PackedPlan& plan,
                                       hipStream_t stream) {
  const int nq = plan.chunk_tokens;
  if (nq <= 0 || plan.n_chunks <= 0) return hipSuccess;
  dim3 grid((nq + kThreads - 1) / kThreads, heads, plan.n_chunks);
  if (head_dim == 64)
    hipLaunchKernelGGL((attn_f32_kernel<64, PackedPlan>), grid, dim3(kThreads), 0, stream,
                       static_cast<const float*>(q), static_cast<float*>(out), nq, heads,
                       softmax_scale, plan);
  else
    hipLaunchKernelGGL((attn_f32_kernel<128, PackedPlan>), grid, dim3(kThreads), 0, stream,
                       static_cast<const float*>(q), static_cast<float*>(out), nq, heads,
                       softmax_scale, plan);
  return hipGetLastError();
}

}  // namespace ff
