// bf16 renderer attention on gfx950 matrix cores (flash-attention forward).
//
// Work split: a workgroup = 8 waves = 256 queries of one head, one workgroup
// per CU (two waves per SIMD); each wave owns 32 queries for the whole key
// loop.  Keys arrive as segments (anchor segment, valid history slots, current
// chunk);
// each segment is cut into 64-key tiles and only a segment's last tile is
// partial (its missing keys are masked to -inf): no tile straddles two
// segments and no empty slot is touched.
//
// Products, per 64-key tile:
//   S^T = K Q^T     v_mfma_f32_32x32x16_bf16; A = K rows read from LDS, B = the
//                   wave's Q^T, held in registers for the whole loop.
//   softmax         the accumulator layout of S^T puts one query column in each
//                   lane (half of a 32-key block; the other half is in lane ^ 32),
//                   so max and sum are in-lane plus one v_permlane32_swap.  exp2
//                   with log2(e) folded into the scale.  The running max is only
//                   raised (and O rescaled) when a column max exceeds it by more
//                   than 8 (log2 units, probabilities up to 2^8); otherwise the
//                   stale max stays the reference, which leaves the result exact
//                   since the final sum uses the same max.
//   O^T += V^T P^T  A = V^T, read from the row-major V tile with the gfx950
//                   transposing LDS read (ds_read_b64_tr_b16); B = P^T, the
//                   softmax registers rounded to bf16 in place.  The keys of each
//                   8-key operand are chosen to match the accumulator layout.
// Software pipeline: h1(t) computes block 0 of S^T of tile t+1 on the matrix
// core beside the exponentials of tile t, then O^T += block 0 of tile t;
// h2(t) computes block 1 of S^T(t+1), O^T += block 1 of tile t and the column
// max of tile t+1.  Waves w and
// w + 4 share a SIMD: waves 0-3 run h1(t) h2(t) after barrier t, waves 4-7 run
// h2(t-1) h1(t), half an iteration later, so on every SIMD one wave's
// exponentials run beside the other's matrix work instead of both waves
// wanting the same unit at once.
// K and V tiles are copied from HBM straight into LDS (global_load_lds_dwordx4,
// 16 bytes per lane, issued by waves 0-3) two tiles ahead, into a ring of four
// tile slots: one barrier per tile (plus one at the end).  The last reads of
// tile t (h2(t) of waves 4-7) come before barrier t+2, where tile t+4 is
// copied into its slot.  The loops are unrolled by four so every slot
// reference is static (reads of one slot are never ordered behind the copy
// into another).
// Tile rows are stored without padding, with an XOR swizzle of their 16-byte
// chunks that keeps both the K reads and the transposing V reads free of bank
// conflicts on the 64-bank LDS.
// Workgroups are renumbered so that consecutive Q tiles of one head land on
// the same XCD (the hardware deals workgroups to the 8 XCDs round robin) and
// share that XCD's L2 for the head's K/V (a packed clip deals whole (chunk,
// head) groups round robin instead, since its chunks' read sets differ in
// length).  When the units do not fill the last round of the GPU, the host
// splits that round's units along their keys into up to four parts
// (unnormalised fp32 partials, merged by tail_merge_kernel).

#include <hip/hip_runtime.h>

#include <math.h>

#include "ff_internal.h"

namespace ff {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))
#define GLOBAL_PTR(p) ((const __attribute__((address_space(1))) void*)(p))

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kCB = 1;                      // 32-query column blocks per wave
constexpr int kWaveQ = 32 * kCB;            // queries per wave
constexpr int kBlockQ = kWaves * kWaveQ;    // queries per workgroup
constexpr int kBK = 64;                     // keys per tile
constexpr int kXcds = 8;
constexpr float kRescaleThreshold = 8.0f;   // log2 units
// Waves w and w + 4 share a SIMD and the issue arbiter favours the older one
// (w < 4), which reaches each tile's barrier well ahead of its partner; the
// tile copies are therefore all issued by waves 0-3, off the partner's path.
constexpr int kCopyWaves = kWaves / 2;

template <int D>
struct Cfg {
  static constexpr int KS = D / 16;          // 16-wide d slices of S^T = K Q^T
  static constexpr int DB = D / 32;          // 32-row blocks of O^T
  static constexpr int ROWB = 2 * D;         // bytes per K/V row in LDS
  static constexpr int CPR = D / 8;          // 16-byte chunks per row
  static constexpr int RPB = 1024 / ROWB;    // rows per 1 KB wave copy
  static constexpr int BLOCKS = kBK / RPB;   // 1 KB copies per tile (per tensor)
  static constexpr int BLOCKS_PER_WAVE = BLOCKS / kCopyWaves;   // copies by waves 0 .. kCopyWaves-1
  static constexpr int TILE = kBK * ROWB;    // bytes of one K (or V) tile
  static constexpr int SLOT = 2 * TILE;      // K tile then V tile
  static_assert(BLOCKS % kCopyWaves == 0, "every copying wave copies the same number of 1 KB blocks");
};

// XOR swizzle of the 16-byte chunks of tile row r, for an LDS that serves
// 256 bytes per clock (64 banks): a 16-lane quarter of a 16-byte K read (16
// consecutive rows, one chunk) and a 32-lane half of an 8-byte transposing V
// read (4 rows x 4 adjacent chunks) must each touch 16 (resp. 32) distinct
// 16-byte (8-byte) bank slots.  d = 128 (256-byte rows, 16 chunks): the row's
// low two bits pick the chunk group and the next two the chunk inside it.
// d = 64 (128-byte rows, 8 chunks, two rows per bank line): same idea on the
// row bits above the line parity.
template <int D>
__device__ inline int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

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

// 64-bit value of lane `lane` (wave-uniform index).  The builtin works on
// signed 32-bit words: each half is widened as unsigned, so a low word with
// its top bit set does not sign-extend into the high word.
__device__ inline uint64_t readlane_u64(uint64_t v, int lane) {
  const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v)), lane));
  const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v >> 32)), lane));
  return (uint64_t(hi) << 32) | uint64_t(lo);
}

// Tile cursor over the key segments: tile = (segment, first key).
struct Cursor {
  int sg, k0;
};

// Src is KvSegments (one read set for the whole launch) or PackedPlan (one
// read set per chunk of a packed clip; q and out then hold every chunk).
template <int D, class Src>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_bf16_kernel(const __bf16* __restrict__ q, __bf16* __restrict__ out, int nq, int heads,
                      float scale_log2, Src src, int n_qtiles, TailSplit tail) {
  constexpr bool kPacked = __is_same(Src, PackedPlan);
  constexpr bool kBatch = __is_same(Src, KvBatch);
  constexpr bool kSets = kPacked || kBatch;   // one read set per (chunk or item) of the grid
  using C = Cfg<D>;
  __shared__ __attribute__((aligned(1024))) char lds0[C::SLOT];
  __shared__ __attribute__((aligned(1024))) char lds1[C::SLOT];
  __shared__ __attribute__((aligned(1024))) char lds2[C::SLOT];
  __shared__ __attribute__((aligned(1024))) char lds3[C::SLOT];

  // Workgroups b < tail.n_full run whole units (head, 256-query tile),
  // renumbered XCD-aware: hardware block b runs on XCD b % 8, so each XCD gets
  // a contiguous range of units.  The later ones run key part b % split of
  // unit n_full + (b - n_full) / split (the partial last round, see TailSplit).
  const int b = blockIdx.x;
  int logical, part_id = 0, n_parts = 1;
  const int n_pairs = kSets ? gridDim.x / n_qtiles : 0;       // (set, head) pairs
  const int n_even = n_pairs - n_pairs % kXcds;
  if (kSets) {
    // several read sets (packed chunks, batch items) of different lengths: XCD
    // x takes the (set, head) pairs p = x, x + 8, .. (the q tiles of one pair
    // stay on one XCD and share its L2), so every XCD gets the same mix; the
    // last n_pairs % 8 pairs run in order
    if (b < n_even * n_qtiles) {
      const int xcd = b % kXcds, idx = b / kXcds;
      logical = (xcd + kXcds * (idx / n_qtiles)) * n_qtiles + idx % n_qtiles;
    } else {
      logical = b;
    }
  } else if (b < tail.n_full) {
    const int n_wg = tail.n_full;
    const int xcd = b % kXcds, idx = b / kXcds;
    const int per = n_wg / kXcds, rem = n_wg % kXcds;
    logical = xcd * per + min(xcd, rem) + idx;
  } else {
    const int j = b - tail.n_full;
    logical = tail.n_full + j / tail.split;
    part_id = j % tail.split;
    n_parts = tail.split;
  }
  int chunk = 0, rest = logical;   // chunk: the read set (packed chunk or batch item)
  if constexpr (kSets) {
    chunk = logical / (heads * n_qtiles);
    rest = logical - chunk * (heads * n_qtiles);
  }
  if constexpr (kPacked) {
    q += int64_t(chunk) * nq * heads * D;
    out += int64_t(chunk) * nq * heads * D;
  }
  if constexpr (kBatch) {
    q = static_cast<const __bf16*>(src.q[chunk]);
    out = static_cast<__bf16*>(src.out[chunk]);
  }
  const int head = rest / n_qtiles;
  const int qt = rest % n_qtiles;

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int half = lane >> 5;

  // Q^T operand: lane (l32, half) of column block cb holds query
  // q0 + 32 cb + l32, elements d = 16 s + 8 half .. +7 of slice s.
  const int q0 = qt * kBlockQ + wave * kWaveQ;
  bf16x8 qreg[kCB][C::KS];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
    const int qi = min(q0 + 32 * cb + l32, nq - 1);
    const __bf16* qp = q + (int64_t(qi) * heads + head) * D + 8 * half;
#pragma unroll
    for (int s = 0; s < C::KS; ++s) qreg[cb][s] = *reinterpret_cast<const bf16x8*>(qp + 16 * s);
  }

  f32x16 o[kCB][C::DB];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb)
#pragma unroll
    for (int db = 0; db < C::DB; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) o[cb][db][j] = 0.0f;
  float m_run[kCB], l_run[kCB];
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
    m_run[cb] = -INFINITY;  // running max of scaled logits (log2 units)
    l_run[cb] = 0.0f;       // this lane's partial sum of probabilities
  }

  // Segment table in registers: lane i holds segment i's length, tokens-stride
  // (bytes) and the byte addresses of this head's K and V rows.  Inside the
  // loop a field of segment sg is read with v_readlane: no scalar memory loads
  // there, so the LDS-read counter waits can stay partial.
  int sg_len = 0;
  uint32_t sg_row_bytes = 0;
  uint64_t sg_k = 0, sg_v = 0;
  int n_segs;
  if constexpr (kPacked) n_segs = packed_num_segments(src, chunk);
  else if constexpr (kBatch) n_segs = src.set[chunk].n;
  else n_segs = src.n;
#pragma unroll
  for (int i = 0; i < kMaxSegments; ++i)
    if (lane == i && i < n_segs) {
      KvSegment sgi;
      if constexpr (kPacked) sgi = packed_segment(src, chunk, i, heads, D, 2);
      else if constexpr (kBatch) sgi = src.set[chunk].seg[i];
      else sgi = src.seg[i];
      sg_len = sgi.len;
      sg_row_bytes = 2u * uint32_t(sgi.tok_stride);
      sg_k = reinterpret_cast<uint64_t>(sgi.k) + 2ull * uint64_t(head) * uint64_t(sgi.head_stride);
      sg_v = reinterpret_cast<uint64_t>(sgi.v) + 2ull * uint64_t(head) * uint64_t(sgi.head_stride);
    }
  auto seg_len = [&](int i) { return __builtin_amdgcn_readlane(sg_len, i); };

  // number of tiles
  int n_tiles = 0;
  for (int i = 0; i < n_segs; ++i) n_tiles += (seg_len(i) + kBK - 1) / kBK;
  // this workgroup's share of the tiles: [t_begin, t_begin + n_tiles)
  const int t_begin = part_id * n_tiles / n_parts;
  n_tiles = (part_id + 1) * n_tiles / n_parts - t_begin;
  auto advance = [&](Cursor c) {
    c.k0 += kBK;
    if (c.k0 >= seg_len(c.sg)) {
      ++c.sg;
      c.k0 = 0;
    }
    return c;
  };

  // tile copy: 1 KB per wave instruction; lane -> (row, physical chunk).  A
  // segment's rows are at most 2^31 bytes apart (the host limits a chunk to
  // 2^31 elements), so each lane's source is a 32-bit byte offset from the
  // segment's (uniform) head base; rows past a partial tile's end re-read its
  // last row, whose scores are masked.
  int cp_row[C::BLOCKS_PER_WAVE], cp_choff[C::BLOCKS_PER_WAVE];
#pragma unroll
  for (int i = 0; i < C::BLOCKS_PER_WAVE; ++i) {
    const int r = (wave * C::BLOCKS_PER_WAVE + i) * C::RPB + lane / C::CPR;
    cp_row[i] = r;
    cp_choff[i] = 16 * ((lane % C::CPR) ^ swz<D>(r));
  }
  auto issue_tile = [&](char* base, Cursor c) {
    if (wave >= kCopyWaves) return;
    const int len = seg_len(c.sg);
    const uint32_t row_bytes = uint32_t(__builtin_amdgcn_readlane(int(sg_row_bytes), c.sg));
    const char* kb = reinterpret_cast<const char*>(readlane_u64(sg_k, c.sg));
    const char* vb = reinterpret_cast<const char*>(readlane_u64(sg_v, c.sg));
    const bool partial = c.k0 + kBK > len;
#pragma unroll
    for (int i = 0; i < C::BLOCKS_PER_WAVE; ++i) {
      int tok = c.k0 + cp_row[i];
      if (partial) tok = min(tok, len - 1);
      const uint32_t off = uint32_t(tok) * row_bytes + uint32_t(cp_choff[i]);
      char* dst = base + (wave * C::BLOCKS_PER_WAVE + i) * 1024;
      __builtin_amdgcn_global_load_lds(GLOBAL_PTR(kb + off), LDS_PTR(void, dst), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(GLOBAL_PTR(vb + off), LDS_PTR(void, dst + C::TILE), 16, 0, 0);
    }
  };

  // LDS read addresses.  The swizzle only flips chunk bits that the row offset
  // leaves clear, so each read is (slot + immediate) + (lane base ^ constant):
  //   K (A of S^T), row kb*32 + l32, chunk 2 ks + half: k_lane ^ (ks << 5), +8 KB for kb = 1
  //     (both blocks share the swizzle: it depends on the row's low four bits only);
  //   V (A of O^T, transposing read), lane group g = lane / 16 covers d block
  //     32 db + 16 (g & 1) and key half (g >> 1); lane l' = lane % 16 reads key row
  //     kbase + l' / 4 at d offset 4 (l' % 4): v_lane[lo/hi] ^ (db << 6) for D = 128
  //     (chunk group = db), + (32 kb + 16 mh) rows.
  int k_lane = l32 * C::ROWB + ((half ^ swz<D>(l32)) << 4);
  const int g = lane >> 4;
  const int lp = lane & 15;
  const int v_row = 4 * (g >> 1) + (lp >> 2);               // row of the lo read within a 16-key group
  const int v_dsub = 16 * (g & 1) + 4 * (lp & 3);            // d offset within a 32-d block
  int v_lane[2];
#pragma unroll
  for (int hi = 0; hi < 2; ++hi) {
    const int r = v_row + 8 * hi;
    v_lane[hi] = r * C::ROWB + (((v_dsub >> 3) ^ swz<D>(r)) << 4) + (v_dsub & 7) * 2;
  }
  // chunk bits flipped per d block: D = 128 has 4 chunks per 32-d block, D = 64 as well
  constexpr int kVdbShift = 6;   // (4 chunks per db) << 4 bytes

  // S^T of 32-key block kb of a tile into s[kb][cb], both column blocks
  auto compute_s = [&](const char* kt, int kb, f32x16 (&s)[2][kCB]) {
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb)
#pragma unroll
      for (int j = 0; j < 16; ++j) s[kb][cb][j] = 0.0f;
    const char* kbase = kt + kb * 32 * C::ROWB;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(kbase + (k_lane ^ (ks << 5)));
#pragma unroll
      for (int cb = 0; cb < kCB; ++cb)
        s[kb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[cb][ks], s[kb][cb], 0, 0, 0);
    }
  };

  // mask keys >= n_valid of a partial tile (register j of block kb holds key
  // kb*32 + 8 (j / 4) + 4 half + j % 4)
  auto mask_s = [&](f32x16 (&s)[2][kCB], int n_valid) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 16; ++j)
        if (kb * 32 + 8 * (j >> 2) + 4 * half + (j & 3) >= n_valid)
#pragma unroll
          for (int cb = 0; cb < kCB; ++cb) s[kb][cb][j] = -INFINITY;
  };

  // column max of a tile; raise the running max (and rescale O) when it grows
  // by more than the threshold
  auto update_max = [&](const f32x16 (&s)[2][kCB]) {
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) {
      float mx = s[0][cb][0];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[kb][cb][j]);
      mx = max_across_halves(mx) * scale_log2;
      if (__builtin_amdgcn_ballot_w64(mx > m_run[cb] + kRescaleThreshold) != 0) {
        const float m_new = fmaxf(m_run[cb], mx);
        const float alpha = __builtin_amdgcn_exp2f(m_run[cb] - m_new);
        m_run[cb] = m_new;
        l_run[cb] *= alpha;
#pragma unroll
        for (int db = 0; db < C::DB; ++db)
#pragma unroll
          for (int j = 0; j < 16; ++j) o[cb][db][j] *= alpha;
      }
    }
  };

  // probabilities of 32-key block kb, both column blocks, as packed bf16
  auto probs = [&](const f32x16 (&s)[2][kCB], int kb, uint32_t (&pk)[kCB][8]) {
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) {
      float sum = 0.0f;
#pragma unroll
      for (int j = 0; j < 16; j += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[kb][cb][j], scale_log2, -m_run[cb]));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[kb][cb][j + 1], scale_log2, -m_run[cb]));
        sum += p0 + p1;
        pk[cb][j >> 1] = pack_bf16(p0, p1);
      }
      l_run[cb] += sum;
    }
  };

  // O^T += V^T P^T for 32-key block kb
  auto pv = [&](const char* vt, int kb, const uint32_t (&pk)[kCB][8]) {
#pragma unroll
    for (int mh = 0; mh < 2; ++mh) {
      bf16x8 pb[kCB];
#pragma unroll
      for (int cb = 0; cb < kCB; ++cb) {
        const u32x4 pu = {pk[cb][4 * mh + 0], pk[cb][4 * mh + 1], pk[cb][4 * mh + 2],
                          pk[cb][4 * mh + 3]};
        pb[cb] = __builtin_bit_cast(bf16x8, pu);
      }
      const char* vbase = vt + (kb * 32 + 16 * mh) * C::ROWB;
#pragma unroll
      for (int db = 0; db < C::DB; ++db) {
        // keys kbase .. +3 (lo) and kbase + 8 .. +11 (hi) of this 16-key group
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            LDS_PTR(s16x4, vbase + (v_lane[0] ^ (db << kVdbShift))));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            LDS_PTR(s16x4, vbase + (v_lane[1] ^ (db << kVdbShift))));
        const u32x2 lo2 = __builtin_bit_cast(u32x2, lo), hi2 = __builtin_bit_cast(u32x2, hi);
        const u32x4 au = {lo2[0], lo2[1], hi2[0], hi2[1]};
        const bf16x8 a = __builtin_bit_cast(bf16x8, au);
#pragma unroll
        for (int cb = 0; cb < kCB; ++cb)
          o[cb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[cb], o[cb][db], 0, 0, 0);
      }
    }
  };

  // ---- prologue: tiles 0 and 1 in flight, S^T of tile 0 -----------------------------
  Cursor c_next = {0, 0};                    // the tile whose S^T the iteration computes
  for (int i = 0; i < t_begin; ++i) c_next = advance(c_next);
  Cursor c_dma = advance(c_next);            // the tile the iteration copies
  issue_tile(lds0, c_next);
  if (n_tiles > 1) {
    issue_tile(lds1, c_dma);
    c_dma = advance(c_dma);                  // tile 2
  }
  // S^T of even tiles lives in s_a, of odd tiles in s_b (no copies between them)
  f32x16 s_a[2][kCB], s_b[2][kCB];
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  compute_s(lds0, 0, s_a);
  compute_s(lds0, 1, s_a);
  {
    const int nv = min(kBK, seg_len(c_next.sg) - c_next.k0);
    if (nv < kBK) mask_s(s_a, nv);
  }
  update_max(s_a);
  c_next = advance(c_next);                  // tile 1

  // ---- main loop, in two halves per tile ---------------------------------------
  // h1(t): S^T block 0 of tile t+1, P^T of tile t, O^T += block 0 of tile t.
  // h2(t): S^T block 1 of tile t+1, O^T += block 1 of tile t, column max of t+1.
  // Waves 0-3 run [barrier t, copy of tile t+2, h1(t), h2(t)]; waves 4-7, which
  // share their SIMDs, run half an iteration later, [barrier t, h2(t-1), h1(t)],
  // so each SIMD pairs one wave's exponentials with the other's matrix work.
  // Tile t lives in slot t % 4; the last reads of tile t (waves 4-7, h2(t))
  // precede barrier t+2, where waves 0-3 copy tile t+4 into its slot.
  uint32_t pk0[kCB][8], pk1[kCB][8];
  auto h1 = [&](char* v_slot, char* k_slot, f32x16 (&s_cur)[2][kCB], f32x16 (&s_nxt)[2][kCB])
      __attribute__((always_inline)) {
    asm volatile("" : "+v"(v_lane[0]), "+v"(v_lane[1]));
    compute_s(k_slot, 0, s_nxt);
    probs(s_cur, 0, pk0);
    pv(v_slot + C::TILE, 0, pk0);
    probs(s_cur, 1, pk1);
  };
  auto h2 = [&](int t, char* v_slot, char* k_slot, f32x16 (&s_nxt)[2][kCB])
      __attribute__((always_inline)) {
    asm volatile("" : "+v"(v_lane[0]), "+v"(v_lane[1]));
    compute_s(k_slot, 1, s_nxt);
    pv(v_slot + C::TILE, 1, pk1);
    if (t + 1 < n_tiles) {
      const int nv = min(kBK, seg_len(c_next.sg) - c_next.k0);
      if (nv < kBK) mask_s(s_nxt, nv);
      update_max(s_nxt);
      c_next = advance(c_next);
    }
  };
  // barrier t: every wave's copies of tile t+1 have landed, tile t-2 is free
  auto sync = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };
  if (wave < kCopyWaves) {
    auto step = [&](int t, char* s0, char* s1, char* s2, f32x16 (&sc)[2][kCB],
                    f32x16 (&sn)[2][kCB]) __attribute__((always_inline)) {
      sync();
      if (t + 2 < n_tiles) {
        issue_tile(s2, c_dma);
        c_dma = advance(c_dma);
      }
      h1(s0, s1, sc, sn);
      h2(t, s0, s1, sn);
    };
    for (int t = 0; t < n_tiles;) {
      step(t, lds0, lds1, lds2, s_a, s_b);
      if (++t >= n_tiles) break;
      step(t, lds1, lds2, lds3, s_b, s_a);
      if (++t >= n_tiles) break;
      step(t, lds2, lds3, lds0, s_a, s_b);
      if (++t >= n_tiles) break;
      step(t, lds3, lds0, lds1, s_b, s_a);
      ++t;
    }
    sync();   // matches the extra barrier of the last step of waves 4-7
  } else {
    sync();
    h1(lds0, lds1, s_a, s_b);
    // step t: barrier t, h2(t-1), and h1(t) while t < n_tiles; the step with
    // t = n_tiles only finishes the last tile.  S^T of tile t is in sc.
    auto step = [&](int t, char* sp, char* s0, char* s1, f32x16 (&sc)[2][kCB],
                    f32x16 (&sn)[2][kCB]) __attribute__((always_inline)) {
      sync();
      h2(t - 1, sp, s0, sc);
      if (t < n_tiles) h1(s0, s1, sc, sn);
    };
    for (int t = 1;;) {
      step(t, lds0, lds1, lds2, s_b, s_a);
      if (t++ >= n_tiles) break;
      step(t, lds1, lds2, lds3, s_a, s_b);
      if (t++ >= n_tiles) break;
      step(t, lds2, lds3, lds0, s_b, s_a);
      if (t++ >= n_tiles) break;
      step(t, lds3, lds0, lds1, s_a, s_b);
      if (t++ >= n_tiles) break;
    }
  }

  // normalise and store: register j of block db holds d = 32 db + 8 (j / 4) + 4 half + j % 4
#pragma unroll
  for (int cb = 0; cb < kCB; ++cb) {
    const int qi = q0 + 32 * cb + l32;
    const float l_tot = sum_across_halves(l_run[cb]);
    const float inv = 1.0f / l_tot;
    if constexpr (kPacked) {
      // base-2 log-sum-exp of the scaled logits, for the backward pass
      if (src.lse != nullptr && half == 0 && qi < nq)
        src.lse[(int64_t(chunk) * nq + qi) * heads + head] = m_run[cb] + log2f(l_tot);
    }
    if (n_parts > 1) {
      // unnormalised partial result of this part: O (row = query of the
      // workgroup), the reference max and the sum, merged by the tail kernel
      float* pb = tail.part + size_t((logical - tail.n_full) * n_parts + part_id) *
                                  (kBlockQ * D + 2 * kBlockQ);
      const int row = wave * kWaveQ + 32 * cb + l32;
#pragma unroll
      for (int db = 0; db < C::DB; ++db)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const f32x4 v = {o[cb][db][4 * a + 0], o[cb][db][4 * a + 1], o[cb][db][4 * a + 2],
                           o[cb][db][4 * a + 3]};
          *reinterpret_cast<f32x4*>(pb + row * D + 32 * db + 8 * a + 4 * half) = v;
        }
      if (half == 0) {
        pb[kBlockQ * D + row] = m_run[cb];
        pb[kBlockQ * D + kBlockQ + row] = l_tot;
      }
    } else if (qi < nq) {
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

// Merge of the tail parts: thread = (tail unit, query row, 8 values of d).
template <int D>
__global__ __launch_bounds__(256) void tail_merge_kernel(const float* __restrict__ part,
                                                         __bf16* __restrict__ out, int nq, int heads,
                                                         int n_qtiles, TailSplit tail, int n_units) {
  constexpr int CH = D / 8;
  const int64_t tid = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (tid >= int64_t(n_units) * kBlockQ * CH) return;
  const int u = int(tid / (kBlockQ * CH));
  const int rem = int(tid % (kBlockQ * CH));
  const int row = rem / CH, ch = rem % CH;
  const int unit = tail.n_full + u;
  const int head = unit / n_qtiles, qt = unit % n_qtiles;
  const int qi = qt * kBlockQ + row;
  if (qi >= nq) return;
  const size_t stride = size_t(kBlockQ) * D + 2 * kBlockQ;
  const float* p0 = part + size_t(u) * tail.split * stride;
  float m = -INFINITY;
  for (int s = 0; s < tail.split; ++s) m = fmaxf(m, p0[s * stride + kBlockQ * D + row]);
  float l = 0.0f, acc[8] = {};
  for (int s = 0; s < tail.split; ++s) {
    const float* ps = p0 + s * stride;
    const float w = __builtin_amdgcn_exp2f(ps[kBlockQ * D + row] - m);
    l += w * ps[kBlockQ * D + kBlockQ + row];
    const f32x4 a = *reinterpret_cast<const f32x4*>(ps + row * D + 8 * ch);
    const f32x4 b = *reinterpret_cast<const f32x4*>(ps + row * D + 8 * ch + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[e] += w * a[e];
      acc[4 + e] += w * b[e];
    }
  }
  const float inv = 1.0f / l;
  u32x4 w4;
#pragma unroll
  for (int e = 0; e < 4; ++e) w4[e] = pack_bf16(acc[2 * e] * inv, acc[2 * e + 1] * inv);
  *reinterpret_cast<u32x4*>(out + (int64_t(qi) * heads + head) * D + 8 * ch) = w4;
}

}  // namespace

int attention_bf16_units(int nq, int heads) { return heads * ((nq + kBlockQ - 1) / kBlockQ); }

int attention_bf16_key_tiles(const KvSegments& segs) {
  int n = 0;
  for (int i = 0; i < segs.n; ++i) n += (segs.seg[i].len + kBK - 1) / kBK;
  return n;
}

size_t attention_bf16_part_bytes(int head_dim) {
  return size_t(kBlockQ) * head_dim * 4 + 2 * kBlockQ * 4;
}

hipError_t launch_attention_bf16(const void* q, void* out, int nq, int heads, int head_dim,
                                 float softmax_scale, const KvSegments& segs, const TailSplit& tail,
                                 hipStream_t stream) {
  if (nq <= 0) return hipSuccess;
  const int n_qtiles = (nq + kBlockQ - 1) / kBlockQ;
  const int units = n_qtiles * heads;
  const int n_tail = units - tail.n_full;
  const dim3 grid(tail.n_full + n_tail * tail.split);
  const float scale_log2 = float(double(softmax_scale) * 1.4426950408889634);
  if (head_dim == 128)
    hipLaunchKernelGGL((attn_bf16_kernel<128, KvSegments>), grid, dim3(kThreads), 0, stream,
                       static_cast<const __bf16*>(q), static_cast<__bf16*>(out), nq, heads,
                       scale_log2, segs, n_qtiles, tail);
  else
    hipLaunchKernelGGL((attn_bf16_kernel<64, KvSegments>), grid, dim3(kThreads), 0, stream,
                       static_cast<const __bf16*>(q), static_cast<__bf16*>(out), nq, heads,
                       scale_log2, segs, n_qtiles, tail);
  if (tail.split > 1 && n_tail > 0) {
    const int64_t threads = int64_t(n_tail) * kBlockQ * (head_dim / 8);
    const dim3 g(unsigned((threads + 255) / 256));
    if (head_dim == 128)
      hipLaunchKernelGGL(tail_merge_kernel<128>, g, dim3(256), 0, stream, tail.part,
                         static_cast<__bf16*>(out), nq, heads, n_qtiles, tail, n_tail);
    else
      hipLaunchKernelGGL(tail_merge_kernel<64>, g, dim3(256), 0, stream, tail.part,
                         static_cast<__bf16*>(out), nq, heads, n_qtiles, tail, n_tail);
  }
  return hipGetLastError();
}

hipError_t launch_attention_bf16_batch(int nq, int heads, int head_dim, float softmax_scale,
                                       const KvBatch& b, hipStream_t stream) {
  if (nq <= 0 || b.n <= 0) return hipSuccess;
  const int n_qtiles = (nq + kBlockQ - 1) / kBlockQ;
  const dim3 grid(b.n * n_qtiles * heads);
  const float scale_log2 = float(double(softmax_scale) * 1.4426950408889634);
  const TailSplit whole = {int(grid.x), 1, nullptr};
  if (head_dim == 128)
    hipLaunchKernelGGL((attn_bf16_kernel<128, KvBatch>), grid, dim3(kThreads), 0, stream,
                       nullptr, nullptr, nq, heads, scale_log2, b, n_qtiles, whole);
  else
    hipLaunchKernelGGL((attn_bf16_kernel<64, KvBatch>), grid, dim3(kThreads), 0, stream,
                       nullptr, nullptr, nq, heads, scale_log2, b, n_qtiles, whole);
  return hipGetLastError();
}

hipError_t launch_attention_bf16_packed(const void* q, void* out, int heads, int head_dim,
                                        float softmax_scale, const PackedPlan& plan,
                                        hipStream_t stream) {
  const int nq = plan.chunk_tokens;
  if (nq <= 0 || plan.n_chunks <= 0) return hipSuccess;
  const int n_qtiles = (nq + kBlockQ - 1) / kBlockQ;
  const dim3 grid(plan.n_chunks * n_qtiles * heads);
  const float scale_log2 = float(double(softmax_scale) * 1.4426950408889634);
  const TailSplit whole = {int(grid.x), 1, nullptr};
  if (head_dim == 128)
    hipLaunchKernelGGL((attn_bf16_kernel<128, PackedPlan>), grid, dim3(kThreads), 0, stream,
                       static_cast<const __bf16*>(q), static_cast<__bf16*>(out), nq, heads,
                       scale_log2, plan, n_qtiles, whole);
  else
    hipLaunchKernelGGL((attn_bf16_kernel<64, PackedPlan>), grid, dim3(kThreads), 0, stream,
                       static_cast<const __bf16*>(q), static_cast<__bf16*>(out), nq, heads,
                       scale_log2, plan, n_qtiles, whole);
  return hipGetLastError();
}

}  // namespace ff
