// bf16 renderer attention on gfx950 matrix cores (flash-attention forward).
//
// Work split: a workgroup = 4 waves = 128 queries of one head; each wave owns
// 32 queries for the whole key loop; two workgroups share a CU, so one's
// softmax overlaps the other's matrix ops.  Keys arrive as segments (anchor
// segment, valid history slots, current chunk); each segment is cut into
// 64-key tiles and only a segment's last tile is partial (its missing keys
// are masked to -inf): no tile straddles two segments and no empty slot is
// touched.
//
// Per tile:
//   S^T = K Q^T     v_mfma_f32_32x32x16_bf16; A = K rows read from LDS, B = the
//                   wave's Q^T, held in registers for the whole loop.
//   softmax         the accumulator layout of S^T puts one query column in each
//                   lane (half of the tile's keys; the other half is in lane ^ 32),
//                   so max and sum are in-lane plus one v_permlane32_swap.  exp2
//                   with log2(e) folded into the scale.  The running max is only
//                   raised (and O rescaled) when a column max exceeds it by more
//                   than 2^8; otherwise the stale max is kept, which leaves the
//                   result exact since the final sum uses the same max.
//   O^T += V^T P^T  A = V^T, read from the row-major V tile with the gfx950
//                   transposing LDS read (ds_read_b64_tr_b16); B = P^T, the
//                   softmax registers rounded to bf16 in place.  The keys of each
//                   8-key operand are chosen to match the accumulator layout.
// K and V tiles are copied from HBM straight into LDS (global_load_lds_dwordx4,
// 16 bytes per lane) one tile ahead, into a double buffer: one barrier per
// tile.  Tile rows are stored without padding, with an XOR swizzle of their
// 16-byte chunks that keeps both the K reads and the transposing V reads free
// of bank conflicts.
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
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))
#define GLOBAL_PTR(p) ((const __attribute__((address_space(1))) void*)(p))

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kWaveQ = 32;                  // queries per wave
constexpr int kBlockQ = kWaves * kWaveQ;    // queries per workgroup
constexpr int kBK = 64;                     // keys per tile
constexpr int kXcds = 8;
constexpr float kRescaleThreshold = 8.0f;   // log2 units

template <int D>
struct Cfg {
  static constexpr int KS = D / 16;          // 16-wide d slices of S^T = K Q^T
  static constexpr int DB = D / 32;          // 32-row blocks of O^T
  static constexpr int ROWB = 2 * D;         // bytes per K/V row in LDS
  static constexpr int CPR = D / 8;          // 16-byte chunks per row
  static constexpr int RPB = 1024 / ROWB;    // rows per 1 KB wave copy
  static constexpr int BLOCKS = kBK / RPB;   // 1 KB copies per tile (per tensor)
  static constexpr int BLOCKS_PER_WAVE = BLOCKS / kWaves;
  static constexpr int TILE = kBK * ROWB;    // bytes of one K (or V) tile
  static constexpr int BUF = 2 * TILE;       // K tile then V tile
};

// XOR swizzle of the 16-byte chunks of tile row r: over any 8 consecutive rows
// it is a permutation of 0..7 (K reads: 32 rows, one chunk), and over any 4
// rows starting at a multiple of 4 its halves are distinct (V transposing
// reads: 4 rows x 2 adjacent chunks).
__device__ inline int swz(int r) { return ((r & 3) << 1) | ((r >> 2) & 1); }

__device__ inline uint32_t pack_bf16(float a, float b) {
  f32x2 f = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

__device__ inline float max_across_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ inline float sum_across_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_bf16_kernel(const __bf16* __restrict__ q, __bf16* __restrict__ out, int nq, int heads,
                      float scale_log2, KvSegments segs, int n_qtiles) {
  using C = Cfg<D>;
  __shared__ __attribute__((aligned(1024))) char lds[2 * C::BUF];

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

  // Q^T operand: lane (l32, half) holds query q0 + l32, d = 16 s + 8 half .. +7
  const int q0 = qt * kBlockQ + wave * kWaveQ;
  bf16x8 qreg[C::KS];
  {
    const int qi = min(q0 + l32, nq - 1);
    const __bf16* qp = q + (int64_t(qi) * heads + head) * D + 8 * half;
#pragma unroll
    for (int s = 0; s < C::KS; ++s) qreg[s] = *reinterpret_cast<const bf16x8*>(qp + 16 * s);
  }

  f32x16 o[C::DB];
#pragma unroll
  for (int db = 0; db < C::DB; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) o[db][j] = 0.0f;
  float m_run = -INFINITY;  // running max of scaled logits (log2 units)
  float l_run = 0.0f;       // this lane's partial sum of probabilities

  // tile copy: 1 KB per wave instruction; lane -> (row, physical chunk)
  const int cp_row = lane / C::CPR;
  const int cp_chunk = lane % C::CPR;
  auto issue_tile = [&](int buf, int sg, int k0) {
    const KvSegment& seg = segs.seg[sg];
    const __bf16* kb = static_cast<const __bf16*>(seg.k) + head * seg.head_stride;
    const __bf16* vb = static_cast<const __bf16*>(seg.v) + head * seg.head_stride;
    char* base = lds + buf * C::BUF;
#pragma unroll
    for (int i = 0; i < C::BLOCKS_PER_WAVE; ++i) {
      const int blk = wave * C::BLOCKS_PER_WAVE + i;
      const int r = blk * C::RPB + cp_row;
      const int tok = min(k0 + r, seg.len - 1);
      const int64_t off = int64_t(tok) * seg.tok_stride + 8 * (cp_chunk ^ swz(r));
      __builtin_amdgcn_global_load_lds(GLOBAL_PTR(kb + off), LDS_PTR(void, base + blk * 1024), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(GLOBAL_PTR(vb + off), LDS_PTR(void, base + C::TILE + blk * 1024),
                                       16, 0, 0);
    }
  };

  // per-lane LDS offsets of the operand reads
  // K (A of S^T): row kb*32 + l32, logical chunk 2 ks + half
  // V (A of O^T, transposing read): lane group g = lane / 16 covers d block
  //   32 db + 16 (g & 1) and key half (g >> 1); lane l' = lane % 16 reads key
  //   row kbase + l' / 4 at d offset 4 (l' % 4).
  const int g = lane >> 4;
  const int lp = lane & 15;
  const int v_half = g >> 1;
  const int v_dsub = 16 * (g & 1) + 4 * (lp & 3);  // d offset within a 32-block
  const int v_rowin = lp >> 2;

  int sg = 0, k0 = 0, buf = 0;
  issue_tile(0, 0, 0);
  while (sg < segs.n) {
    const int len = segs.seg[sg].len;
    const int n_valid = min(kBK, len - k0);
    int nsg = sg, nk0 = k0 + kBK;
    if (nk0 >= len) {
      ++nsg;
      nk0 = 0;
    }
    __builtin_amdgcn_s_waitcnt(0);  // this wave's copies of the current tile have landed
    __syncthreads();                // everyone's have; everyone is done with the other buffer
    if (nsg < segs.n) issue_tile(buf ^ 1, nsg, nk0);
    const char* kt = lds + buf * C::BUF;
    const char* vt = kt + C::TILE;

    // S^T = K Q^T, two 32-key blocks
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int j = 0; j < 16; ++j) s[kb][j] = 0.0f;
      const int r = kb * 32 + l32;
      const char* krow = kt + r * C::ROWB;
      const int sw = swz(r);
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(krow + (((2 * ks + half) ^ sw) << 4));
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[ks], s[kb], 0, 0, 0);
      }
    }
    if (n_valid < kBK) {
      // register j of block kb holds key kb*32 + 8 (j / 4) + 4 half + j % 4
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j)
          if (kb * 32 + 8 * (j >> 2) + 4 * half + (j & 3) >= n_valid) s[kb][j] = -INFINITY;
    }

    // online softmax of this lane's query column
    float mx = s[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[kb][j]);
    mx = max_across_halves(mx) * scale_log2;
    if (__builtin_amdgcn_ballot_w64(mx > m_run + kRescaleThreshold) != 0) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < C::DB; ++db)
#pragma unroll
        for (int j = 0; j < 16; ++j) o[db][j] *= alpha;
    }
    uint32_t pk[2][8];
    float sum = 0.0f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 16; j += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[kb][j], scale_log2, -m_run));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[kb][j + 1], scale_log2, -m_run));
        sum += p0 + p1;
        pk[kb][j >> 1] = pack_bf16(p0, p1);
      }
    l_run += sum;

    // O^T += V^T P^T
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int mh = 0; mh < 2; ++mh) {
        const u32x4 pu = {pk[kb][4 * mh + 0], pk[kb][4 * mh + 1], pk[kb][4 * mh + 2],
                          pk[kb][4 * mh + 3]};
        const bf16x8 pb = __builtin_bit_cast(bf16x8, pu);
        // keys kbase .. +3 and kbase + 8 .. +11 of this 16-key group
        const int r0 = kb * 32 + 16 * mh + 4 * v_half + v_rowin;
        const int r1 = r0 + 8;
#pragma unroll
        for (int db = 0; db < C::DB; ++db) {
          const int c = (32 * db + v_dsub) >> 3;        // logical chunk
          const int byte = ((32 * db + v_dsub) & 7) * 2;  // 0 or 8
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              LDS_PTR(s16x4, vt + r0 * C::ROWB + ((c ^ swz(r0)) << 4) + byte));
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              LDS_PTR(s16x4, vt + r1 * C::ROWB + ((c ^ swz(r1)) << 4) + byte));
          const u32x4 au = {__builtin_bit_cast(u32x2, lo)[0], __builtin_bit_cast(u32x2, lo)[1],
                            __builtin_bit_cast(u32x2, hi)[0], __builtin_bit_cast(u32x2, hi)[1]};
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, au), pb,
                                                          o[db], 0, 0, 0);
        }
      }
    buf ^= 1;
    sg = nsg;
    k0 = nk0;
  }

  // normalise and store: register j of block db holds d = 32 db + 8 (j / 4) + 4 half + j % 4
  const int qi = q0 + l32;
  const float inv = 1.0f / sum_across_halves(l_run);
  if (qi < nq) {
    __bf16* op = out + (int64_t(qi) * heads + head) * D + 4 * half;
#pragma unroll
    for (int db = 0; db < C::DB; ++db)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        u32x2 w;
        w.x = pack_bf16(o[db][4 * a + 0] * inv, o[db][4 * a + 1] * inv);
        w.y = pack_bf16(o[db][4 * a + 2] * inv, o[db][4 * a + 3] * inv);
        *reinterpret_cast<u32x2*>(op + 32 * db + 8 * a) = w;
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
