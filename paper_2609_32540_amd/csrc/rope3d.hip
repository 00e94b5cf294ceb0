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
// Launch shape: one block of 256 threads per kTok = 2 tokens (many small blocks
// spread the chunk evenly over the CUs).  The block's tokens form one
// contiguous run of kTok * heads * d elements in each tensor, swept with
// 16-byte vectors, U per tensor and thread in flight: the first ones are
// loaded before the angles are computed and the next ones before the current
// ones are rotated and stored.

#include <hip/hip_runtime.h>

#include "ff_internal.h"
#include "ff_numeric.h"

namespace ff {
namespace {

constexpr int kThreads = 256;
constexpr int kTok = 2;   // tokens per block


__device__ inline uint32_t rotate_bf16_pair(uint32_t w, double2 cs) {
  const double a = bf16_lo(w), b = bf16_hi(w);
  const double o0 = a * cs.x - b * cs.y;
  const double o1 = a * cs.y + b * cs.x;
  return pack_bf16_rne(round_to_odd_f32(o0), round_to_odd_f32(o1));
}

template <typename T>
__device__ inline uint4 rotate_vec(uint4 w, const double2* cs) {
  if constexpr (sizeof(T) == 2) {
    w.x = rotate_bf16_pair(w.x, cs[0]);
    w.y = rotate_bf16_pair(w.y, cs[1]);
    w.z = rotate_bf16_pair(w.z, cs[2]);
    w.w = rotate_bf16_pair(w.w, cs[3]);
  } else {
    const double a0 = __uint_as_float(w.x), b0 = __uint_as_float(w.y);
    const double a1 = __uint_as_float(w.z), b1 = __uint_as_float(w.w);
    w.x = __float_as_uint(float(a0 * cs[0].x - b0 * cs[0].y));
    w.y = __float_as_uint(float(a0 * cs[0].y + b0 * cs[0].x));
    w.z = __float_as_uint(float(a1 * cs[1].x - b1 * cs[1].y));
    w.w = __float_as_uint(float(a1 * cs[1].y + b1 * cs[1].x));
  }
  return w;
}

// Rotation of the block's vectors of Q (when HQ) and K: the steady loop has no
// per-lane branch (every lane holds a vector) and keeps U vectors per tensor in
// flight, the next ones loaded before the current ones are rotated and stored.
template <typename T, int D, bool HQ, int U>
__device__ inline void rotate_block(uint4* __restrict__ vq, uint4* __restrict__ vk, int total,
                                    int vecs_per_tok, const double2 (*cs_d)[D / 2],
                                    uint4 (&bq)[U], uint4 (&bk)[U]) {
  constexpr int EPV = 16 / sizeof(T);
  constexpr int VPR = D / EPV;
  constexpr int PPV = EPV / 2;
  const int full = total / kThreads;          // steps in which every lane has a vector
  const int last = total - 1;
  int j = 0;
  for (; j + U <= full; j += U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = threadIdx.x + (j + u) * kThreads;
      const double2* cs = cs_d[i / vecs_per_tok] + (i % VPR) * PPV;
      const uint4 rq = HQ ? rotate_vec<T>(bq[u], cs) : uint4{};
      const uint4 rk = rotate_vec<T>(bk[u], cs);
      const int n = min(i + U * kThreads, last);   // next vector (clamped: a spare reload at the end)
      if (HQ) bq[u] = vq[n];
      bk[u] = vk[n];
      if (HQ) vq[i] = rq;
      vk[i] = rk;
    }
  }
  // the rest, one vector per lane per step, with a lane check
  for (int i = threadIdx.x + j * kThreads; i < total; i += kThreads) {
    const double2* cs = cs_d[i / vecs_per_tok] + (i % VPR) * PPV;
    if (HQ) vq[i] = rotate_vec<T>(vq[i], cs);
    vk[i] = rotate_vec<T>(vk[i], cs);
  }
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void rope3d_kernel(T* __restrict__ q, T* __restrict__ k,
                                                          int n_tok, int heads, int grid_w,
                                                          int tokens_per_frame, RopeParams p) {
  if (k == nullptr) {   // only Q: rotate it in K's place
    k = q;
    q = nullptr;
  }
  constexpr int P = D / 2;
  constexpr int EPV = 16 / sizeof(T);   // elements per 16-byte vector
  constexpr int VPR = D / EPV;          // vectors per head row
  constexpr int U = 4;                  // vectors per tensor in flight per thread
  __shared__ double2 cs_d[kTok][P];
  const int tok0 = blockIdx.x * kTok;
  const int n_rows_tok = min(kTok, n_tok - tok0);
  const int vecs_per_tok = heads * VPR;
  const int total = n_rows_tok * vecs_per_tok;
  uint4* vq = q ? reinterpret_cast<uint4*>(q) + int64_t(tok0) * vecs_per_tok : nullptr;
  uint4* vk = reinterpret_cast<uint4*>(k) + int64_t(tok0) * vecs_per_tok;

  // the first vectors are loaded before the angles are computed, so that the
  // loads overlap the float64 sincos (clamped indices: a spare load when the
  // block has fewer vectors)
  uint4 bq[U], bk[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int i = min(int(threadIdx.x) + u * kThreads, total - 1);
    if (vq) bq[u] = vq[i];
    bk[u] = vk[i];
  }

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
  if (vq) rotate_block<T, D, true, U>(vq, vk, total, vecs_per_tok, cs_d, bq, bk);
  else rotate_block<T, D, false, U>(vq, vk, total, vecs_per_tok, cs_d, bq, bk);
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
