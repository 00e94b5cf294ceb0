// 3D (t, h, w) rotary position embedding of Q and K, in place.
//
// Pair p = (2p, 2p+1) of a head vector is rotated by phi = pos * omega[p],
// with pos the token's latent time t for p < n_t, its grid row for
// n_t <= p < n_th and its grid column otherwise (omega[p] is theta^(-j/n_axis),
// computed on the host in float64).  The angle and its cosine and sine are
// computed once per (token, pair) in float64, kept in LDS and reused by every
// head of Q and K.  The rotation runs in float64 and is rounded once to the
// storage type, to nearest even: for bf16 through a round-to-odd float32
// intermediate, which makes the two-step rounding equal to a direct one.
//
// Launch shape: one block of 256 threads per kTok tokens.  The block's tokens
// form one contiguous run of kTok * heads * d elements in each tensor, swept
// with 16-byte vectors.

#include <hip/hip_runtime.h>

#include "ff_internal.h"
#include "ff_numeric.h"

namespace ff {
namespace {

constexpr int kThreads = 256;
constexpr int kTok = 8;


__device__ inline uint32_t rotate_bf16_pair(uint32_t w, double2 cs) {
  const double a = bf16_lo(w), b = bf16_hi(w);
  const double o0 = a * cs.x - b * cs.y;
  const double o1 = a * cs.y + b * cs.x;
  return pack_bf16_rne(round_to_odd_f32(o0), round_to_odd_f32(o1));
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void rope3d_kernel(T* __restrict__ q, T* __restrict__ k,
                                                          int n_tok, int heads, int grid_w,
                                                          int tokens_per_frame, RopeParams p) {
  constexpr int P = D / 2;
  __shared__ double2 cs_d[kTok][P];
  const int tok0 = blockIdx.x * kTok;

  for (int e = threadIdx.x; e < kTok * P; e += kThreads) {
    const int tt = e / P, pr = e % P;
    const int tok = tok0 + tt;
    if (tok < n_tok) {
      const int f = tok / tokens_per_frame;
      const int in_frame = tok - f * tokens_per_frame;
      const int y = in_frame / grid_w;
      const int x = in_frame - y * grid_w;
      const int pos = pr < p.n_t ? p.frame_t[f] : (pr < p.n_th ? y : x);
      double s, c;
      sincos(double(pos) * p.omega[pr], &s, &c);
      cs_d[tt][pr] = make_double2(c, s);
    }
  }
  __syncthreads();

  constexpr int EPV = 16 / sizeof(T);   // elements per 16-byte vector
  constexpr int VPR = D / EPV;          // vectors per head row
  const int n_rows_tok = min(kTok, n_tok - tok0);
  const int vecs_per_tok = heads * VPR;
  const int total = n_rows_tok * vecs_per_tok;
  for (int tensor = 0; tensor < 2; ++tensor) {
    T* base = tensor ? k : q;
    if (base == nullptr) continue;
    uint4* v = reinterpret_cast<uint4*>(base) + int64_t(tok0) * vecs_per_tok;
    for (int e = threadIdx.x; e < total; e += kThreads) {
      const int tt = e / vecs_per_tok;
      const int c = e % VPR;               // vector within the head row
      uint4 w = v[e];
      if constexpr (sizeof(T) == 2) {
        const int p0 = c * 4;              // 4 pairs per vector
        w.x = rotate_bf16_pair(w.x, cs_d[tt][p0 + 0]);
        w.y = rotate_bf16_pair(w.y, cs_d[tt][p0 + 1]);
        w.z = rotate_bf16_pair(w.z, cs_d[tt][p0 + 2]);
        w.w = rotate_bf16_pair(w.w, cs_d[tt][p0 + 3]);
      } else {
        const int p0 = c * 2;              // 2 pairs per vector
        const double2 c0 = cs_d[tt][p0], c1 = cs_d[tt][p0 + 1];
        const double a0 = __uint_as_float(w.x), b0 = __uint_as_float(w.y);
        const double a1 = __uint_as_float(w.z), b1 = __uint_as_float(w.w);
        w.x = __float_as_uint(float(a0 * c0.x - b0 * c0.y));
        w.y = __float_as_uint(float(a0 * c0.y + b0 * c0.x));
        w.z = __float_as_uint(float(a1 * c1.x - b1 * c1.y));
        w.w = __float_as_uint(float(a1 * c1.y + b1 * c1.x));
      }
      v[e] = w;
    }
  }
}

}  // namespace

hipError_t launch_rope3d(void* q, void* k, int n_tok, int heads, int head_dim, int dtype,
                         int grid_w, int tokens_per_frame, const RopeParams& p,
                         hipStream_t stream) {
  if (n_tok <= 0) return hipSuccess;
  dim3 grid((n_tok + kTok - 1) / kTok);
  if (dtype == FF_DT_BF16) {
    using T = __bf16;
    if (head_dim == 128)
      hipLaunchKernelGGL((rope3d_kernel<T, 128>), grid, dim3(kThreads), 0, stream,
                         static_cast<T*>(q), static_cast<T*>(k), n_tok, heads, grid_w,
                         tokens_per_frame, p);
    else
      hipLaunchKernelGGL((rope3d_kernel<T, 64>), grid, dim3(kThreads), 0, stream,
                         static_cast<T*>(q), static_cast<T*>(k), n_tok, heads, grid_w,
                         tokens_per_frame, p);
  } else {
    using T = float;
    if (head_dim == 128)
      hipLaunchKernelGGL((rope3d_kernel<T, 128>), grid, dim3(kThreads), 0, stream,
                         static_cast<T*>(q), static_cast<T*>(k), n_tok, heads, grid_w,
                         tokens_per_frame, p);
    else
      hipLaunchKernelGGL((rope3d_kernel<T, 64>), grid, dim3(kThreads), 0, stream,
                         static_cast<T*>(q), static_cast<T*>(k), n_tok, heads, grid_w,
                         tokens_per_frame, p);
  }
  return hipGetLastError();
}

}  // namespace ff
