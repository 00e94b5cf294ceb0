// KV publish / anchor set / cache read-out: bit copies between the token-major
// [tokens][heads][d] layout of a chunk and the head-major [heads][tokens][d]
// layout of a ring slot or anchor segment.  These are streaming HBM copies:
// every byte is read once and written once.
//
// Launch shape: grid (token tiles, heads, 2 tensors), 256 threads.  A row of
// one (token, head) is `row_bytes` = d * elem bytes (128 .. 512 B), moved as
// 16-byte vectors; a block moves kTokensPerBlock consecutive tokens of one
// head, so the head-major side is one contiguous run and the token-major side
// is rows of row_bytes at a stride of heads * row_bytes.  Each thread issues
// all of its loads before its stores to keep several 16-byte loads in flight;
// blocks whose tokens are all in range do so without per-lane checks (checked
// loads would each be waited for before the next).

#include <hip/hip_runtime.h>

#include "ff_internal.h"

namespace ff {
namespace {

constexpr int kThreads = 256;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// VPR: 16-byte vectors per row (row_bytes / 16).  ITER: rows per thread.
template <int VPR, int ITER, bool kToHeadMajor>
__global__ __launch_bounds__(kThreads) void kv_copy_kernel(
    const u32x4* __restrict__ k_src, const u32x4* __restrict__ v_src, u32x4* __restrict__ k_dst,
    u32x4* __restrict__ v_dst, int n_tok, int heads, int64_t head_stride_vec) {
  constexpr int kRowsPerPass = kThreads / VPR;
  constexpr int kTokensPerBlock = kRowsPerPass * ITER;
  const u32x4* src = blockIdx.z ? v_src : k_src;
  u32x4* dst = blockIdx.z ? v_dst : k_dst;
  if (src == nullptr || dst == nullptr) return;
  const int head = blockIdx.y;
  const int c = threadIdx.x % VPR;
  const int r = threadIdx.x / VPR;
  const int tok0 = blockIdx.x * kTokensPerBlock + r;

  auto index = [&](int t, bool to_head_major) {
    return to_head_major ? head * head_stride_vec + int64_t(t) * VPR + c     // head-major index
                         : (int64_t(t) * heads + head) * VPR + c;            // token-major index
  };
  u32x4 val[ITER];
  if ((blockIdx.x + 1) * kTokensPerBlock <= n_tok) {
    // a whole block of tokens: no per-lane check, so every load is in flight
    // before the first store
#pragma unroll
    for (int it = 0; it < ITER; ++it)
      val[it] = __builtin_nontemporal_load(src + index(tok0 + it * kRowsPerPass, !kToHeadMajor));
#pragma unroll
    for (int it = 0; it < ITER; ++it)
      __builtin_nontemporal_store(val[it], dst + index(tok0 + it * kRowsPerPass, kToHeadMajor));
    return;
  }
#pragma unroll
  for (int it = 0; it < ITER; ++it) {
    const int t = tok0 + it * kRowsPerPass;
    if (t < n_tok) val[it] = __builtin_nontemporal_load(src + index(t, !kToHeadMajor));
  }
#pragma unroll
  for (int it = 0; it < ITER; ++it) {
    const int t = tok0 + it * kRowsPerPass;
    if (t < n_tok) __builtin_nontemporal_store(val[it], dst + index(t, kToHeadMajor));
  }
}

template <bool kToHeadMajor>
hipError_t launch_copy(const void* k_src, const void* v_src, void* k_dst, void* v_dst, int n_tok,
                       int heads, int row_bytes, int64_t head_stride_bytes, hipStream_t stream) {
  if (n_tok <= 0) return hipSuccess;
  constexpr int ITER = 4;
  const int64_t hs = head_stride_bytes / 16;
  auto go = [&](auto kernel, int vpr) {
    const int tokens_per_block = (kThreads / vpr) * ITER;
    dim3 grid((n_tok + tokens_per_block - 1) / tokens_per_block, heads, 2);
    hipLaunchKernelGGL(kernel, grid, dim3(kThreads), 0, stream,
                       static_cast<const u32x4*>(k_src), static_cast<const u32x4*>(v_src),
                       static_cast<u32x4*>(k_dst), static_cast<u32x4*>(v_dst), n_tok, heads, hs);
    return hipGetLastError();
  };
  switch (row_bytes) {
    case 128: return go(kv_copy_kernel<8, ITER, kToHeadMajor>, 8);
    case 256: return go(kv_copy_kernel<16, ITER, kToHeadMajor>, 16);
    case 512: return go(kv_copy_kernel<32, ITER, kToHeadMajor>, 32);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_kv_scatter(const void* k_src, const void* v_src, void* k_dst, void* v_dst,
                             int n_tok, int heads, int row_bytes, int64_t dst_head_stride_bytes,
                             hipStream_t stream) {
  return launch_copy<true>(k_src, v_src, k_dst, v_dst, n_tok, heads, row_bytes,
                           dst_head_stride_bytes, stream);
}

hipError_t launch_kv_gather(const void* k_src, const void* v_src, void* k_dst, void* v_dst,
                            int n_tok, int heads, int row_bytes, int64_t src_head_stride_bytes,
                            hipStream_t stream) {
  return launch_copy<false>(k_src, v_src, k_dst, v_dst, n_tok, heads, row_bytes,
                            src_head_stride_bytes, stream);
}

}  // namespace ff
