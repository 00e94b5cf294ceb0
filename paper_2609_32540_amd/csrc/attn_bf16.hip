// bf16 renderer attention on gfx950 matrix cores (flash-attention forward).
//
// One workgroup = 4 waves = 256 queries of one head; each wave owns 64
// queries (two 32-query column blocks) for the whole key loop.  Keys arrive as
// segments (anchor segment, history slots, current chunk); each segment is cut
// into 64-key tiles, and only a segment's last tile is partial (its missing
// keys are masked to -inf), so no tile straddles two segments.
//
// Per tile:
//   S^T = K Q^T     v_mfma_f32_32x32x16_bf16, A = K rows from LDS, B = Q^T held
//                   in registers for the whole loop (loaded once).
//   softmax         S^T's accumulator layout puts one query column in each
//                   lane (32 of its keys per 32-key block, the other 32 in lane
//                   ^ 32), so the running max / sum are in-lane except for one
//                   cross-half exchange of the max; exp2 with log2(e) folded
//                   into the scale.
//   O^T += V^T P^T  A = V^T from LDS, B = P^T = the softmax registers rounded
//                   to bf16 (nearest even) without leaving the lane; the order
//                   of keys inside each 16-key group of the V^T tile is permuted
//                   at staging time to match the accumulator layout.
// K and V tiles are loaded from HBM with 16-byte loads one tile ahead (into
// registers), then staged in LDS: K row-major with a 16-byte row pad, V
// transposed with an XOR swizzle of 16-byte chunks.
// Workgroups are renumbered so that consecutive Q tiles of one head land on
// the same XCD (the hardware deals workgroups to the 8 XCDs round robin) and
// share that XCD's L2 for the head's K/V.

#include <hip/hip_runtime.h>

#include <math.h>

#include "ff_internal.h"

namespace ff {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kQB = 2;                      // 32-query column blocks per wave
constexpr int kWaveQ = 32 * kQB;            // queries per wave
constexpr int kBlockQ = kWaves * kWaveQ;    // queries per workgroup
constexpr int kBK = 64;                     // keys per tile
constexpr int kXcds = 8;

template <int D>
struct Cfg {
  static constexpr int KS = D / 16;                 // 16-wide slices of d in S^T = K Q^T
  static constexpr int DB = D / 32;                 // 32-row blocks of O^T
  static constexpr int CPR = D / 8;                 // 16-byte chunks per K/V row
  static constexpr int KPT = kBK * CPR / kThreads;  // consecutive keys staged per thread
  static constexpr int K_ROW = D * 2 + 16;          // LDS bytes per K row
  static constexpr int V_ROW = kBK * 2;             // LDS bytes per V^T row
  static constexpr int LDS_K = kBK * K_ROW;
  static constexpr int LDS_V = D * V_ROW;
};

__device__ inline uint32_t pack_bf16(float a, float b) {
  f32x2 f = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

// Position of key o (0..63) inside a V^T row: bits 2 and 3 of the offset in its
// 16-key group are swapped, so that the 8 keys one lane feeds to a PV matrix
// op are contiguous.
__device__ inline int vt_pos(int o) { return (o & ~12) | ((o & 4) << 1) | ((o & 8) >> 1); }

// XOR swizzle of the 16-byte chunks of V^T row d.
__device__ inline int vt_swz(int d) { return (d ^ (d >> 3)) & 7; }

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void attn_bf16_kernel(const __bf16* __restrict__ q, __bf16* __restrict__ out, int nq, int heads,
                      float scale_log2, KvSegments segs, int n_qtiles) {
  using C = Cfg<D>;
  __shared__ __attribute__((aligned(16))) char lds_k[C::LDS_K];
  __shared__ __attribute__((aligned(16))) char lds_v[C::LDS_V];

  // XCD-aware renumbering: hardware block b runs on XCD b % 8; give each XCD a
  // contiguous range of logical tiles.
  const int n_wg = gridDim.x;
  const int b = blockIdx.x;
  const int xcd = b % kXcds, idx = b / kXcds;
  const int per = n_wg / kXcds, rem = n_wg % kXcds;
  const int logical = xcd * per + min(xcd, rem) + idx;
  const int head = logical / n_qtiles;
  const int qt = logical % n_qtiles;

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int half = lane >> 5;

  // Q^T operand: lane (l32, half) of column block cb holds query
  // q0 + cb*32 + l32, elements d = 16 s + 8 half .. +7 for slice s.
  const int q_wave0 = qt * kBlockQ + wave * kWaveQ;
  bf16x8 qreg[kQB][C::KS];
#pragma unroll
  for (int cb = 0; cb < kQB; ++cb) {
    const int qi = min(q_wave0 + cb * 32 + l32, nq - 1);
    const __bf16* qp = q + (int64_t(qi) * heads + head) * D + 8 * half;
#pragma unroll
    for (int s = 0; s < C::KS; ++s) qreg[cb][s] = *reinterpret_cast<const bf16x8*>(qp + 16 * s);
  }

  f32x16 o[kQB][C::DB];
#pragma unroll
  for (int cb = 0; cb < kQB; ++cb)
#pragma unroll
    for (int db = 0; db < C::DB; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) o[cb][db][j] = 0.0f;
  float m_run[kQB], l_run[kQB];
#pragma unroll
  for (int cb = 0; cb < kQB; ++cb) {
    m_run[cb] = -INFINITY;
    l_run[cb] = 0.0f;
  }

  // staging map: thread holds keys KPT*g .. KPT*g + KPT-1, d-chunk c
  const int c_ld = tid % C::CPR;
  const int g_ld = tid / C::CPR;
  u32x4 kreg[C::KPT], vreg[C::KPT];

  auto load_tile = [&](int sg, int k0) {
    const KvSegment& seg = segs.seg[sg];
    const __bf16* kb = static_cast<const __bf16*>(seg.k) + head * seg.head_stride + 8 * c_ld;
    const __bf16* vb = static_cast<const __bf16*>(seg.v) + head * seg.head_stride + 8 * c_ld;
#pragma unroll
    for (int i = 0; i < C::KPT; ++i) {
      const int tok = min(k0 + C::KPT * g_ld + i, seg.len - 1);
      const int64_t off = int64_t(tok) * seg.tok_stride;
      kreg[i] = *reinterpret_cast<const u32x4*>(kb + off);
      vreg[i] = *reinterpret_cast<const u32x4*>(vb + off);
    }
  };

  auto stage_tile = [&]() {
#pragma unroll
    for (int i = 0; i < C::KPT; ++i)
      *reinterpret_cast<u32x4*>(lds_k + (C::KPT * g_ld + i) * C::K_ROW + c_ld * 16) = kreg[i];
    // V^T: element e of this thread's chunk is d = 8 c + e; its KPT keys are
    // contiguous in the row at vt_pos(KPT g).
    const int pos = (C::KPT * g_ld) & ~15;
    const int p = pos | vt_pos((C::KPT * g_ld) & 15);
    const int chunk = p >> 3;
    const int within = (p & 7) * 2;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int d = 8 * c_ld + e;
      uint16_t h[C::KPT];
#pragma unroll
      for (int i = 0; i < C::KPT; ++i) {
        const uint32_t w = vreg[i][e >> 1];
        h[i] = (e & 1) ? uint16_t(w >> 16) : uint16_t(w & 0xffff);
      }
      char* dst = lds_v + d * C::V_ROW + ((chunk ^ vt_swz(d)) << 4) + within;
      if constexpr (C::KPT == 4) {
        u32x2 v2;
        v2.x = uint32_t(h[0]) | (uint32_t(h[1]) << 16);
        v2.y = uint32_t(h[2]) | (uint32_t(h[3]) << 16);
        *reinterpret_cast<u32x2*>(dst) = v2;
      } else {
        *reinterpret_cast<uint32_t*>(dst) = uint32_t(h[0]) | (uint32_t(h[1]) << 16);
      }
    }
  };

  int sg = 0, k0 = 0;
  if (segs.n > 0) load_tile(0, 0);
  while (sg < segs.n) {
    const int len = segs.seg[sg].len;
    const int n_valid = min(kBK, len - k0);
    int nsg = sg, nk0 = k0 + kBK;
    if (nk0 >= len) {
      ++nsg;
      nk0 = 0;
    }
    __syncthreads();  // every wave is done with the previous tile
    stage_tile();
    __syncthreads();
    if (nsg < segs.n) load_tile(nsg, nk0);  // next tile, in flight during this one

    // S^T = K Q^T for the two 32-key blocks
    f32x16 s[2][kQB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int cb = 0; cb < kQB; ++cb)
#pragma unroll
        for (int j = 0; j < 16; ++j) s[kb][cb][j] = 0.0f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const char* krow = lds_k + (kb * 32 + l32) * C::K_ROW + half * 16;
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(krow + ks * 32);
#pragma unroll
        for (int cb = 0; cb < kQB; ++cb)
          s[kb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[cb][ks], s[kb][cb], 0, 0, 0);
      }
    }
    if (n_valid < kBK) {
      // key of register j in block kb: kb*32 + 8*(j/4) + 4*half + j%4
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int key = kb * 32 + 8 * (j >> 2) + 4 * half + (j & 3);
          if (key >= n_valid)
#pragma unroll
            for (int cb = 0; cb < kQB; ++cb) s[kb][cb][j] = -INFINITY;
        }
    }

    // online softmax, one query column per lane (partner lane ^ 32 holds the
    // other half of the keys)
    uint32_t pk[2][kQB][8];
#pragma unroll
    for (int cb = 0; cb < kQB; ++cb) {
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[kb][cb][j]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[cb], mx * scale_log2);
      const float alpha = exp2f(m_run[cb] - m_new);
      m_run[cb] = m_new;
      float sum = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 16; j += 2) {
          const float p0 = exp2f(fmaf(s[kb][cb][j], scale_log2, -m_new));
          const float p1 = exp2f(fmaf(s[kb][cb][j + 1], scale_log2, -m_new));
          sum += p0 + p1;
          pk[kb][cb][j >> 1] = pack_bf16(p0, p1);
        }
      l_run[cb] = l_run[cb] * alpha + sum;
#pragma unroll
      for (int db = 0; db < C::DB; ++db)
#pragma unroll
        for (int j = 0; j < 16; ++j) o[cb][db][j] *= alpha;
    }

    // O^T += V^T P^T
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int mh = 0; mh < 2; ++mh) {
        bf16x8 pb[kQB];
#pragma unroll
        for (int cb = 0; cb < kQB; ++cb) {
          u32x4 u = {pk[kb][cb][4 * mh + 0], pk[kb][cb][4 * mh + 1], pk[kb][cb][4 * mh + 2],
                     pk[kb][cb][4 * mh + 3]};
          pb[cb] = __builtin_bit_cast(bf16x8, u);
        }
        const int chunk = 4 * kb + 2 * mh + half;
#pragma unroll
        for (int db = 0; db < C::DB; ++db) {
          const int d = 32 * db + l32;
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(lds_v + d * C::V_ROW +
                                                           ((chunk ^ vt_swz(d)) << 4));
#pragma unroll
          for (int cb = 0; cb < kQB; ++cb)
            o[cb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[cb], o[cb][db], 0, 0, 0);
        }
      }
    sg = nsg;
    k0 = nk0;
  }

  // normalise and store: register j of block db holds d = 32 db + 8 (j/4) + 4 half + j%4
#pragma unroll
  for (int cb = 0; cb < kQB; ++cb) {
    const int qi = q_wave0 + cb * 32 + l32;
    const float l_tot = l_run[cb] + __shfl_xor(l_run[cb], 32);
    const float inv = 1.0f / l_tot;
    if (qi < nq) {
      __bf16* op = out + (int64_t(qi) * heads + head) * D + 4 * half;
#pragma unroll
      for (int db = 0; db < C::DB; ++db)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          u32x2 w;
          w.x = pack_bf16(o[cb][db][4 * a + 0] * inv, o[cb][db][4 * a + 1] * inv);
          w.y = pack_bf16(o[cb][db][4 * a + 2] * inv, o[cb][db][4 * a + 3] * inv);
          *reinterpret_cast<u32x2*>(op + 32 * db + 8 * a) = w;
        }
    }
  }
}

}  // namespace

hipError_t launch_attention_bf16(const void* q, void* out, int nq, int heads, int head_dim,
                                 float softmax_scale, const KvSegments& segs,
                                 hipStream_t stream) {
  if (nq <= 0) return hipSuccess;
  const int n_qtiles = (nq + kBlockQ - 1) / kBlockQ;
  const dim3 grid(n_qtiles * heads);
  const float scale_log2 = float(double(softmax_scale) * 1.4426950408889634);
  if (head_dim == 128)
    hipLaunchKernelGGL(attn_bf16_kernel<128>, grid, dim3(kThreads), 0, stream,
                       static_cast<const __bf16*>(q), static_cast<__bf16*>(out), nq, heads,
                       scale_log2, segs, n_qtiles);
  else
    hipLaunchKernelGGL(attn_bf16_kernel<64>, grid, dim3(kThreads), 0, stream,
                       static_cast<const __bf16*>(q), static_cast<__bf16*>(out), nq, heads,
                       scale_log2, segs, n_qtiles);
  return hipGetLastError();
}

}  // namespace ff
