// bf16 renderer attention on gfx950 matrix cores (flash-attention forward).
//
// Work split: a workgroup = 8 waves = 256 queries of one head, one workgroup
// per CU (two waves per SIMD); each wave owns 32 queries for the whole key
// loop.  Keys arrive as segments (anchor segment, valid history slots, current
// chunk); each segment is cut into 64-key tiles and only a segment's last tile
// is partial (its missing keys are masked to -inf): no tile straddles two
// segments and no empty slot is touched.
//
// Products, per 32-key block (two per tile):
//   S^T = K Q^T     v_mfma_f32_32x32x16_bf16; A = K rows read from LDS, B = the
//                   wave's Q^T, held in registers for the whole loop.
//   softmax         the accumulator layout of S^T puts one query column in each
//                   lane (half of a 32-key block; the other half is in lane ^ 32),
//                   so the row sums stay in-lane until the end.  p = exp2(s c -
//                   m) with c = scale * log2 e applied in float32 (one fma; Q is
//                   not rounded again after scaling).  The reference max m is the
//                   first block's column max and is only raised when a block's
//                   probabilities sum past kSumLimit (every kept probability is
//                   then at most kSumLimit, and infinities from scores far above
//                   the reference trip the same test): that rare block is
//                   recomputed from LDS, O and l rescaled and its probabilities
//                   redone.  The result is exact for any reference, since the
//                   final sum uses the same one; no column max is taken per block.
//   O^T += V^T P^T  A = V^T, read from the row-major V tile with the gfx950
//                   transposing LDS read (ds_read_b64_tr_b16); B = P^T, the
//                   softmax registers rounded to bf16 in place.  The keys of each
//                   8-key operand are chosen to match the accumulator layout.
// Software pipeline over blocks b: A(b) computes S^T of block b+1 on the matrix
// core beside the exponentials of block b; B(b) checks block b's sum, adds
// block b into O^T and masks block b+1 if it is partial.  Waves w and w + 4
// share a SIMD: waves 0-3 run A(2t) B(2t) A(2t+1) B(2t+1) after barrier t,
// waves 4-7 run one phase later, B(2t-1) A(2t) B(2t) A(2t+1), so on every SIMD
// one wave's exponentials run beside the other's matrix work.
// K and V tiles are copied from HBM straight into LDS (global_load_lds_dwordx4,
// 16 bytes per lane) by waves 0-3 at the end of their step t, three tiles
// ahead, into a ring of five tile slots (all 160 KB of LDS at d = 128): the
// slot of tile t+3 held tile t-2, whose last read (waves 4-7, B(2t-3)) came
// before barrier t.  Barrier t waits only for the copy of tile t+1, so each
// copy has a whole step to land.  The copies are issued from inline assembly
// and waited for explicitly, so the compiler does not add its own conservative
// waits for them; the loops are unrolled by five so every slot reference is
// static.
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
constexpr float kSumLimit = 16.0f;          // largest block sum of probabilities kept
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

// 16 bytes per lane from global memory (uniform base + per-lane byte offset)
// straight into LDS at dst + 16 * lane.  Written out so that the compiler does
// not track these copies: their completion is waited for explicitly (vmcnt)
// before the barrier that hands a tile to the other waves.
__device__ inline void lds_copy16(uint32_t dst, const char* base, uint32_t off) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
               :: "s"(dst), "v"(off), "s"(base) : "memory");
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
  __shared__ __attribute__((aligned(1024))) char lds4[C::SLOT];

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
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform
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
    m_run[cb] = 0.0f;       // reference max of the scaled logits (log2 units)
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
  auto advance = [&](Cursor c) __attribute__((always_inline)) {
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
  auto issue_tile = [&](char* base, Cursor c) __attribute__((always_inline)) {
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
      const uint32_t dst = uint32_t(size_t(LDS_PTR(char, base))) + (wave * C::BLOCKS_PER_WAVE + i) * 1024;
      lds_copy16(dst, kb, off);
      lds_copy16(dst + C::TILE, vb, off);
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

  // S^T of 32-key block kb of the tile at kt, both column blocks
  auto s_blk = [&](const char* kt, int kb, f32x16 (&s)[kCB]) __attribute__((always_inline)) {
    const char* kbase = kt + kb * 32 * C::ROWB;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(kbase + (k_lane ^ (ks << 5)));
#pragma unroll
      for (int cb = 0; cb < kCB; ++cb)
        s[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[cb][ks], ks == 0 ? f32x16{} : s[cb],
                                                        0, 0, 0);
    }
  };
  // mask keys >= n_valid of a 32-key block (register j holds key 8 (j / 4) + 4 half + j % 4)
  auto mask_blk = [&](f32x16 (&s)[kCB], int n_valid) __attribute__((always_inline)) {
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb)
#pragma unroll
      for (int j = 0; j < 16; ++j)
        s[cb][j] = 8 * (j >> 2) + 4 * half + (j & 3) >= n_valid ? -INFINITY : s[cb][j];
  };
  // reference max from the first block: its column max (O and l are still zero)
  auto first_max = [&](const f32x16 (&s)[kCB]) __attribute__((always_inline)) {
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) {
      float mx = s[cb][0];
#pragma unroll
      for (int j = 1; j < 16; ++j) mx = fmaxf(mx, s[cb][j]);
      m_run[cb] = max_across_halves(mx) * scale_log2;
    }
  };
  // probabilities of a block as packed bf16
  auto p_blk = [&](const f32x16 (&s)[kCB], uint32_t (&pk)[kCB][8], float (&lb)[kCB])
      __attribute__((always_inline)) {
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) {
      float sum = -0.0f;
#pragma unroll
      for (int j = 0; j < 16; j += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[cb][j], scale_log2, -m_run[cb]));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[cb][j + 1], scale_log2, -m_run[cb]));
        sum += p0 + p1;
        pk[cb][j >> 1] = pack_bf16(p0, p1);
      }
      lb[cb] = sum;
    }
  };
  // The reference max is only raised when a block's probabilities (relative to
  // it) sum past kSumLimit: then this block's S^T is recomputed from LDS, the
  // reference raised to its column max (O and l follow) and its probabilities
  // redone.  Below the limit every probability is at most kSumLimit, so nothing
  // overflows; infinities (scores far above the reference) also exceed it.
  auto check_blk = [&](const char* kt, int kb, int nv_blk, uint32_t (&pk)[kCB][8], float (&lb)[kCB])
      __attribute__((always_inline)) {
    bool over = false;
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) over |= lb[cb] > kSumLimit;
    if (__builtin_amdgcn_ballot_w64(over) == 0) return;
    f32x16 sr[kCB];
    s_blk(kt, kb, sr);
    if (nv_blk < 32) mask_blk(sr, nv_blk);
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) {
      float mx = sr[cb][0];
#pragma unroll
      for (int j = 1; j < 16; ++j) mx = fmaxf(mx, sr[cb][j]);
      const float m_new = fmaxf(m_run[cb], max_across_halves(mx) * scale_log2);
      const float alpha = __builtin_amdgcn_exp2f(m_run[cb] - m_new);
      l_run[cb] *= alpha;
#pragma unroll
      for (int db = 0; db < C::DB; ++db)
#pragma unroll
        for (int j = 0; j < 16; ++j) o[cb][db][j] *= alpha;
      m_run[cb] = m_new;
    }
    p_blk(sr, pk, lb);
  };
  // O^T += V^T P^T for 32-key block kb of the tile at vt
  auto pv_blk = [&](const char* vt, int kb, const uint32_t (&pk)[kCB][8]) __attribute__((always_inline)) {
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

  // ---- prologue: tiles 0 and 1 in flight, S^T of block 0 of tile 0 ----------------
  Cursor c_s = {0, 0};                       // the tile of the S^T block being computed
  for (int i = 0; i < t_begin; ++i) c_s = advance(c_s);
  Cursor c_dma = advance(c_s);               // the tile the next copy fetches
  issue_tile(lds0, c_s);
  if (n_tiles > 1) {
    issue_tile(lds1, c_dma);
    c_dma = advance(c_dma);                  // tile 2
  }
  if (n_tiles > 2) {
    issue_tile(lds2, c_dma);
    c_dma = advance(c_dma);                  // tile 3
  }
  // S^T of even blocks (block 0 of a tile) lives in s_a, of odd blocks in s_b
  f32x16 s_a[kCB], s_b[kCB];
  uint32_t pk[kCB][8];
  float lb[kCB];
  int nv_s = min(kBK, seg_len(c_s.sg) - c_s.k0);   // valid keys of tile c_s
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  s_blk(lds0, 0, s_a);
  if (nv_s < 32) mask_blk(s_a, nv_s);
  first_max(s_a);

  // ---- main loop over 32-key blocks -------------------------------------------
  // Block b = 2t + kb is key block kb of tile t.  Phase A(b): S^T of block b+1
  // on the matrix core beside the exponentials of block b.  Phase B(b): O^T +=
  // block b beside the mask and column max of block b+1.  Waves 0-3 run
  // [barrier t, copy of tile t+2, A(2t) B(2t) A(2t+1) B(2t+1)]; waves 4-7, which
  // share their SIMDs, run one phase later, [barrier t, B(2t-1) A(2t) B(2t)
  // A(2t+1)], so each SIMD pairs one wave's exponentials with the other's
  // products.  Tile t lives in slot t % 4; the last read of tile t (waves 4-7,
  // B(2t+1)) precedes barrier t+2, where waves 0-3 copy tile t+4 into its slot.
  // A(2t):   s_b = S^T(tile t, block 1);   P of s_a.
  // A(2t+1): s_a = S^T(tile t+1, block 0); P of s_b (only P for the last tile).
  auto phA0 = [&](char* st) __attribute__((always_inline)) {
    asm volatile("" : "+v"(v_lane[0]), "+v"(v_lane[1]));
    s_blk(st, 1, s_b);
    p_blk(s_a, pk, lb);
  };
  auto phB0 = [&](char* st) __attribute__((always_inline)) {
    asm volatile("" : "+v"(v_lane[0]), "+v"(v_lane[1]));
    check_blk(st, 0, nv_s, pk, lb);
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) l_run[cb] += lb[cb];
    pv_blk(st + C::TILE, 0, pk);
    if (nv_s < kBK) mask_blk(s_b, nv_s - 32);
  };
  auto phA1 = [&](int t, char* sn) __attribute__((always_inline)) {
    asm volatile("" : "+v"(v_lane[0]), "+v"(v_lane[1]));
    s_blk(sn, 0, s_a);   // (after the last tile: stale slot, result unused)
    p_blk(s_b, pk, lb);
  };
  auto phB1 = [&](int t, char* st) __attribute__((always_inline)) {
    asm volatile("" : "+v"(v_lane[0]), "+v"(v_lane[1]));
    check_blk(st, 1, nv_s - 32, pk, lb);
#pragma unroll
    for (int cb = 0; cb < kCB; ++cb) l_run[cb] += lb[cb];
    pv_blk(st + C::TILE, 1, pk);
    if (t + 1 < n_tiles) {
      c_s = advance(c_s);
      nv_s = min(kBK, seg_len(c_s.sg) - c_s.k0);
      if (nv_s < 32) mask_blk(s_a, nv_s);
    }
  };
  // barrier t: tile t+1 has landed (the copy of tile t+2, issued at the end of
  // step t-1, may still be in flight) and every read of tile t-2 is done
  auto sync = [&](int t) __attribute__((always_inline)) {
    if (wave < kCopyWaves && t + 2 < n_tiles)
      __builtin_amdgcn_s_waitcnt(2 * C::BLOCKS_PER_WAVE);   // vmcnt(copies of one tile), lgkmcnt(0)
    else
      __builtin_amdgcn_s_waitcnt(0);
    asm volatile("s_barrier" ::: "memory");
  };
  if (wave < kCopyWaves) {
    // step t: A(2t) B(2t) A(2t+1) B(2t+1), then the copy of tile t+3 into the
    // slot of tile t-2 (last read before barrier t)
    auto step = [&](int t, char* s0, char* s1, char* s3) __attribute__((always_inline)) {
      sync(t);
      phA0(s0);
      phB0(s0);
      phA1(t, s1);
      phB1(t, s0);
      if (t + 3 < n_tiles) {
        issue_tile(s3, c_dma);
        c_dma = advance(c_dma);
      }
    };
    for (int t = 0; t < n_tiles;) {
      step(t, lds0, lds1, lds3);
      if (++t >= n_tiles) break;
      step(t, lds1, lds2, lds4);
      if (++t >= n_tiles) break;
      step(t, lds2, lds3, lds0);
      if (++t >= n_tiles) break;
      step(t, lds3, lds4, lds1);
      if (++t >= n_tiles) break;
      step(t, lds4, lds0, lds2);
      ++t;
    }
    sync(n_tiles);   // matches the extra barrier of the last step of waves 4-7
  } else {
    // step t: barrier t, B(2t-1) (t > 0), then A(2t) B(2t) A(2t+1) while
    // t < n_tiles; the step with t = n_tiles only finishes the last tile.
    auto step = [&](int t, char* sp, char* s0, char* s1) __attribute__((always_inline)) {
      sync(t);
      if (t > 0) phB1(t - 1, sp);
      if (t < n_tiles) {
        phA0(s0);
        phB0(s0);
        phA1(t, s1);
      }
    };
    for (int t = 0;;) {
      step(t, lds4, lds0, lds1);
      if (t++ >= n_tiles) break;
      step(t, lds0, lds1, lds2);
      if (t++ >= n_tiles) break;
      step(t, lds1, lds2, lds3);
      if (t++ >= n_tiles) break;
      step(t, lds2, lds3, lds4);
      if (t++ >= n_tiles) break;
      step(t, lds3, lds4, lds0);
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
