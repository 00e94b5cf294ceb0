// bf16 renderer attention on gfx950 matrix cores (flash-attention forward).
//
// Work split: a workgroup = 8 waves = 256 queries of one head, one workgroup
// per CU (two waves per SIMD); each wave owns 32 queries for the whole key
// loop.  Keys arrive as segments (anchor segment, valid history slots, current
// chunk); each segment is cut into 64-key tiles and only a segment's last tile
// is partial (its missing keys are masked to -inf): no tile straddles two
// segments and no empty slot is touched.
//
// Products, per 32-key block (two per tile), all on v_mfma_f32_16x16x32_bf16
// (16 x 16 outputs, 32-deep sums: the least register traffic per FLOP of the
// bf16 shapes, which matters because the kernel runs power-limited):
//   S^T = K Q^T     four 16 x 16 tiles (key half kh x query half qh), four
//                   32-wide d slices each; A = K rows read from LDS, B = the
//                   wave's Q^T, held in registers for the whole loop.
//   softmax         lane (n, g) = (lane % 16, lane / 16) holds, for query n of
//                   each query half, keys 4g .. 4g+3 of each key half.
//                   p = exp2(s c - m) with c = scale * log2 e applied in
//                   float32 (one fma; Q is not rounded again after scaling).
//   O^T += V^T P^T  16-row d tiles x query halves, one 32-deep sum per block;
//                   A = V^T, read from the row-major V tile with the gfx950
//                   transposing LDS read (ds_read_b64_tr_b16); B = P^T, the
//                   softmax registers rounded to bf16.  The sum runs over the
//                   keys in the order the softmax registers hold them (lane
//                   group g: keys 4g .. 4g+3, then 16+4g .. 16+4g+3).
// Each 32-key step of a wave issues S^T of block b+1 and O^T += P(b-1) V(b-1)
// and places the softmax of block b, which depends on neither, product by
// product between them: a wave's own VALU work overlaps its matrix work far
// better than one wave's VALU work overlaps its SIMD partner's products.  A
// step is two scheduling halves (V reads, S^T products, softmax of query half
// 0 | K reads of the next step, P V products, softmax of query half 1), so the
// next step's K reads cannot be hoisted above the products that still use
// their registers.
// The key loop first runs as a fast pass: the reference max m stays the first
// block's column max and the row sums come from the matrix core (an all-ones A
// operand sums exactly the rounded probabilities the P V products add), so O
// and l share one scale however far m sits below the true max.  A row sum
// above kFastLimit (or not finite) sends the workgroup's unit through the loop
// again as a checked pass that raises m per block (check_blk).  Launches that
// write the log-sum-exp run the fast pass with float32 row sums of the
// unrounded probabilities instead (the log-sum-exp's definition).
// K and V tiles are copied from HBM straight into LDS (global_load_lds_dwordx4,
// 16 bytes per lane) by waves 0-3, three tiles ahead, into a ring of five tile
// slots (all 160 KB of LDS at d = 128): after barrier t (tile t+1 has landed,
// tile t-2 is no longer read) tile t+3 goes into tile t-2's slot.  The copies
// are issued from inline assembly and waited for explicitly, so the compiler
// does not add its own conservative waits for them.  Every LDS read is a
// per-lane base plus immediates except for the slot base, so the tile loop
// stays rolled.
// The tiles are stored without padding in layouts chosen for their reads: a K
// tile chunk-major per 16 keys (one 256-byte line per 16-byte chunk of 16
// keys), a V tile d-blocked (one 256-byte line per 8 keys and 16-wide d tile).
// Each 16-byte K read of a quarter-wave and each transposing V read of a
// half-wave then takes exactly one line, free of bank conflicts on the
// 64-bank LDS, and the d slices and d tiles differ by immediate offsets.
// Workgroups are renumbered so that consecutive Q tiles of one head land on
// the same XCD (the hardware deals workgroups to the 8 XCDs round robin) and
// share that XCD's L2 for the head's K/V (a packed clip deals whole (chunk,
// head) groups round robin instead, since its chunks' read sets differ in
// length).  When the units do not fill the last round of the GPU, the host
// splits that round's units along their keys into up to four parts
// (unnormalised fp32 partials, merged by tail_merge_kernel).

#include <hip/hip_runtime.h>

#include <math.h>

#include <utility>

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
constexpr int kQH = 2;                      // 16-query halves per wave
constexpr int kWaveQ = 16 * kQH;            // queries per wave
constexpr int kBlockQ = kWaves * kWaveQ;    // queries per workgroup
constexpr int kBK = 64;                     // keys per tile
constexpr int kXcds = 8;
constexpr float kSumLimit = 16.0f;          // checked pass: largest block sum of probabilities kept
constexpr float kFastLimit = 0x1p64f;       // fast pass: largest row sum before the checked pass
// passes of the key loop
constexpr int kPassFast = 0;       // fixed reference, row sums of the rounded P on the matrix core
constexpr int kPassFastExact = 1;  // fixed reference, float32 row sums of the unrounded P
constexpr int kPassChecked = 2;    // reference raised per block (check_blk)
constexpr int kVReadsFirst = 0;            // V reads issued ahead of the first S^T product
constexpr int kHalfVALU = 20;               // plain VALU of a query half: 8 fma + 8 add + 4 packs
constexpr int kHalfVALUFast = 16;           // the fast pass: 8 fma + 4 packs and slack
// Waves w and w + 4 share a SIMD and the issue arbiter favours the older one
// (w < 4), which reaches each tile's barrier well ahead of its partner; the
// tile copies are therefore all issued by waves 0-3, off the partner's path.
constexpr int kCopyWaves = kWaves / 2;

template <int D>
struct Cfg {
  static constexpr int KS = D / 32;          // 32-wide d slices of S^T = K Q^T
  static constexpr int DT = D / 16;          // 16-row d tiles of O^T
  static constexpr int ROWB = 2 * D;         // bytes per K/V row in LDS
  static constexpr int CPR = D / 8;          // 16-byte chunks per row
  static constexpr int RPB = 1024 / ROWB;    // rows per 1 KB wave copy
  static constexpr int BLOCKS = kBK / RPB;   // 1 KB copies per tile (per tensor)
  static constexpr int BLOCKS_PER_WAVE = BLOCKS / kCopyWaves;   // copies by waves 0 .. kCopyWaves-1
  static constexpr int TILE = kBK * ROWB;    // bytes of one K (or V) tile
  static constexpr int SLOT = 2 * TILE;      // K tile then V tile
  static constexpr int VGB = D / 64;         // 1 KB blocks per 8-row group of a V tile
  static constexpr int KGB = D / 32;         // 1 KB blocks per 16-row group of a K tile
  static_assert(BLOCKS % kCopyWaves == 0, "every copying wave copies the same number of 1 KB blocks");
};

// N 1 KB copies from global memory straight into LDS: copy i takes 16 bytes
// per lane from base + off[i] + 1024 i into LDS at dst + 1024 i + 16 lane.  The
// instruction's immediate offset moves both addresses, so m0 (the LDS base) is
// written once for all N; callers fold -1024 i into off[i] and lower base by
// 1024 (N - 1) so that every per-lane offset stays non-negative.  Written out so
// that the compiler does not track these copies: their completion is waited
// for explicitly (vmcnt) before the barrier that hands a tile to the other
// waves.
template <int N>
__device__ inline void lds_copy_blocks(uint32_t dst, const char* base, const uint32_t (&off)[N]) {
  static_assert(N == 2 || N == 4, "two or four 1 KB copies per wave and tensor");
  if constexpr (N == 2)
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\t"
                 "global_load_lds_dwordx4 %1, %3\n\t"
                 "global_load_lds_dwordx4 %2, %3 offset:1024"
                 :: "s"(dst), "v"(off[0]), "v"(off[1]), "s"(base) : "memory");
  else
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\t"
                 "global_load_lds_dwordx4 %1, %5\n\t"
                 "global_load_lds_dwordx4 %2, %5 offset:1024\n\t"
                 "global_load_lds_dwordx4 %3, %5 offset:2048\n\t"
                 "global_load_lds_dwordx4 %4, %5 offset:3072"
                 :: "s"(dst), "v"(off[0]), "v"(off[1]), "v"(off[2]), "v"(off[3]), "s"(base) : "memory");
}

__device__ inline uint32_t pack_bf16(float a, float b) {
  f32x2 f = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

// max and sum over the lanes n, n + 16, n + 32, n + 48 (the four lane groups
// holding one query's keys)
__device__ inline float max_across_groups(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ inline float sum_across_groups(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
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

// s_waitcnt immediate: vmcnt = vm; lgkmcnt and expcnt not waited for
constexpr int waitcnt_vm(int vm) { return (vm & 15) | ((vm >> 4) << 14) | (7 << 4) | (15 << 8); }

// Instruction order of one half of a pipeline step, by sched_group_barrier
// classes (0x008 matrix, 0x100 LDS read, 0x002 VALU, 0x400 transcendental):
// NRF of the half's NR LDS reads and a few softmax instructions ahead of the
// first product, then NM products, the first NR - NRF of them each followed by
// one more LDS read, and all of them by their share of the softmax of one query
// half (NV plain VALU instructions: 8 fma, 8 add, 4 packs and some slack; 8
// exponentials).
template <int NM, int NR, int NRF, int NV, int NT, int I>
__device__ __forceinline__ void interleave_one() {
  __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  if constexpr (I < NR - NRF) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  constexpr int v = (NV * (I + 1)) / NM - (NV * I) / NM;
  if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x002, v, 0);
  constexpr int t = (NT * (I + 1)) / NM - (NT * I) / NM;
  if constexpr (t > 0) __builtin_amdgcn_sched_group_barrier(0x400, t, 0);
}

template <int NM, int NR, int NRF, int NV, int NT, int... I>
__device__ __forceinline__ void interleave_seq(std::integer_sequence<int, I...>) {
  (interleave_one<NM, NR, NRF, NV, NT, I>(), ...);
}

template <int NM, int NR, int NRF, int NV>
__device__ __forceinline__ void interleave_half() {
  static_assert(NR - NRF <= NM, "every spread LDS read follows its own product");
  constexpr int kHead = 2, kHeadT = 1;
  if constexpr (NRF > 0) __builtin_amdgcn_sched_group_barrier(0x100, NRF, 0);
  __builtin_amdgcn_sched_group_barrier(0x002, kHead, 0);
  __builtin_amdgcn_sched_group_barrier(0x400, kHeadT, 0);
  interleave_seq<NM, NR, NRF, NV - kHead, 8 - kHeadT>(std::make_integer_sequence<int, NM>{});
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
  __shared__ __attribute__((aligned(1024))) char lds[5 * C::SLOT];
  auto slot = [&](int i) __attribute__((always_inline)) { return lds + i * C::SLOT; };

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
  const int l16 = lane & 15;
  const int grp = lane >> 4;

  // Q^T operand: lane (l16, grp) of query half qh holds query q0 + 16 qh + l16,
  // elements d = 32 s + 8 grp .. +7 of slice s.
  const int q0 = qt * kBlockQ + wave * kWaveQ;
  bf16x8 qreg[kQH][C::KS];
#pragma unroll
  for (int qh = 0; qh < kQH; ++qh) {
    const int qi = min(q0 + 16 * qh + l16, nq - 1);
    const __bf16* qp = q + (int64_t(qi) * heads + head) * D + 8 * grp;
#pragma unroll
    for (int s = 0; s < C::KS; ++s) qreg[qh][s] = *reinterpret_cast<const bf16x8*>(qp + 32 * s);
  }

  // O^T tile (d tile dt, query half qh): lane (l16, grp) holds query
  // q0 + 16 qh + l16 at d = 16 dt + 4 grp + j, j = 0 .. 3
  f32x4 o[C::DT][kQH];
#pragma unroll
  for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
    for (int qh = 0; qh < kQH; ++qh) o[dt][qh] = f32x4{};
  float m_run[kQH], l_run[kQH];
  f32x4 lsum[kQH];          // fast pass: row sums (every row of the tile holds the sum)
#pragma unroll
  for (int qh = 0; qh < kQH; ++qh) {
    m_run[qh] = 0.0f;       // reference max of the scaled logits (log2 units)
    l_run[qh] = 0.0f;       // checked pass: this lane's partial sum of probabilities
    lsum[qh] = f32x4{};
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

  // tile copy: 1 KB per wave instruction, lane l lands at 16 l of the block.
  //   K tile, chunk-major per 16 rows: 16-row group G takes D / 32 blocks, and
  //     in them one 256-byte line per 16-byte chunk c holding that chunk of rows
  //     16 G .. 16 G + 15; block b = (G, m) holds the lines of chunks 4 m .. 4 m + 3,
  //     so lane l carries row 16 G + l % 16, chunk 4 m + l / 16.
  //   V tile, d-blocked: 8-row group G takes D / 64 blocks, and in them one
  //     256-byte line per 16-wide d tile dt holding, for row 8 G + i, chunks
  //     2 dt and 2 dt + 1 at 16 (2 i) and 16 (2 i + 1); block b = (G, H) holds
  //     the lines of d tiles 4 H .. 4 H + 3, so lane l carries row 8 G + (l % 16) / 2,
  //     chunk 8 H + 2 (l / 16) + l % 2.
  // The tile's first row is folded into the (uniform) 64-bit source base, so
  // each lane's source is a small 32-bit offset: its row within the tile times
  // the segment's row stride, plus its chunk; rows past a partial tile's end
  // re-read the segment's last row, whose scores are masked.
  auto issue_tile = [&](char* base, Cursor c) __attribute__((always_inline)) {
    if (wave >= kCopyWaves) return;
    constexpr int N = C::BLOCKS_PER_WAVE;
    constexpr uint32_t kSpan = 1024u * (N - 1);   // largest immediate offset
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const uint32_t row_bytes = uint32_t(__builtin_amdgcn_readlane(int(sg_row_bytes), c.sg));
    // rows past the segment's end (a partial tile) re-read its last row
    const int last = seg_len(c.sg) - 1 - c.k0;
    const uint64_t tile_off = uint64_t(c.k0) * row_bytes - kSpan;
    const char* kb = reinterpret_cast<const char*>(readlane_u64(sg_k, c.sg) + tile_off);
    const char* vb = reinterpret_cast<const char*>(readlane_u64(sg_v, c.sg) + tile_off);
    uint32_t koff[N], voff[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int blk = wave * N + i;
      const int kr = 16 * (blk / C::KGB) + (ln & 15);
      const int kch = 4 * (blk % C::KGB) + (ln >> 4);
      const int vr = 8 * (blk / C::VGB) + ((ln & 15) >> 1);
      const int vch = 8 * (blk % C::VGB) + 2 * (ln >> 4) + (ln & 1);
      koff[i] = uint32_t(min(kr, last)) * row_bytes + (16u * kch + kSpan - 1024u * i);
      voff[i] = uint32_t(min(vr, last)) * row_bytes + (16u * vch + kSpan - 1024u * i);
    }
    const uint32_t dst = uint32_t(size_t(LDS_PTR(char, base))) + wave * N * 1024;
    lds_copy_blocks<N>(dst, kb, koff);
    lds_copy_blocks<N>(dst + C::TILE, vb, voff);
  };

  // LDS read addresses.  The swizzle only flips chunk bits that the row offset
  // leaves clear, so each read is (slot + immediate) + (lane base ^ constant):
  //   K (A of S^T), row 16 kh + l16, chunk 4 ks + grp: k_lane + 1024 ks + 16 ROWB kh
  //     in the chunk-major K tile (a 16-lane quarter reads one whole 256-byte line);
  //   V (A of O^T, transposing read), lane group grp reads key rows 4 grp .. 4 grp+3
  //     (lo) and 16 + 4 grp .. +3 (hi) of the block, lane l16 the row 4 grp + l16 / 4
  //     (+ 16) at d offset 4 (l16 % 4) of the d tile, and receives column l16 of the
  //     four rows: v_lane[lo/hi] + 256 dt for d tile dt in the d-blocked V tile
  //     (a 32-lane half reads one whole 256-byte line: no bank conflicts).
  const int k_lane = 256 * grp + 16 * l16;
  int v_lane[2];
#pragma unroll
  for (int hi = 0; hi < 2; ++hi) {
    const int r = 16 * hi + 4 * grp + (l16 >> 2);
    v_lane[hi] = (r >> 3) * (8 * C::ROWB) + ((2 * (r & 7) + ((l16 >> 1) & 1)) << 4) + 8 * (l16 & 1);
  }

  // K operands of S^T for 32-key block kb of the tile at kt: a[kh][ks] = rows
  // 16 kh + l16, d slice ks
  auto k_read = [&](const char* kt, int kb, bf16x8 (&a)[2][C::KS]) __attribute__((always_inline)) {
    const char* kbase = kt + kb * 32 * C::ROWB;
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks)
        a[kh][ks] = *reinterpret_cast<const bf16x8*>(kbase + kh * 16 * C::ROWB + k_lane + 1024 * ks);
  };
  // S^T of a block: tile (kh, qh) = keys 16 kh .. +15 x queries 16 qh .. +15 of
  // the wave; lane (l16, grp) register j holds key 16 kh + 4 grp + j of query
  // 16 qh + l16
  auto s_mma = [&](const bf16x8 (&a)[2][C::KS], f32x4 (&s)[2][kQH]) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks)
#pragma unroll
      for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int qh = 0; qh < kQH; ++qh)
          s[kh][qh] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[kh][ks], qreg[qh][ks],
                                                              ks == 0 ? f32x4{} : s[kh][qh], 0, 0, 0);
  };
  // V^T operands of O^T for 32-key block kb of the tile at vt, d tile dt
  auto v_read = [&](const char* vt, int kb, bf16x8 (&a)[C::DT]) __attribute__((always_inline)) {
    const char* vbase = vt + kb * 32 * C::ROWB;
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt) {
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, vbase + v_lane[0] + 256 * dt));
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, vbase + v_lane[1] + 256 * dt));
      const u32x2 lo2 = __builtin_bit_cast(u32x2, lo), hi2 = __builtin_bit_cast(u32x2, hi);
      const u32x4 au = {lo2[0], lo2[1], hi2[0], hi2[1]};
      a[dt] = __builtin_bit_cast(bf16x8, au);
    }
  };
  // O^T += V^T P^T for one block; with_sums also adds the block's row sums into
  // lsum (an all-ones A operand: every row of the 16 x 16 result is the column
  // sum of P^T, i.e. the sum of exactly the rounded probabilities O^T adds up)
  auto pv_mma = [&](const bf16x8 (&a)[C::DT], const uint32_t (&pk)[kQH][4], auto with_sums)
      __attribute__((always_inline)) {
    bf16x8 pb[kQH];
#pragma unroll
    for (int qh = 0; qh < kQH; ++qh) {
      const u32x4 pu = {pk[qh][0], pk[qh][1], pk[qh][2], pk[qh][3]};
      pb[qh] = __builtin_bit_cast(bf16x8, pu);
    }
#pragma unroll
    for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
      for (int qh = 0; qh < kQH; ++qh)
        o[dt][qh] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[dt], pb[qh], o[dt][qh], 0, 0, 0);
    if constexpr (decltype(with_sums)::value) {
      const bf16x8 ones = {__bf16(1.0f), __bf16(1.0f), __bf16(1.0f), __bf16(1.0f),
                           __bf16(1.0f), __bf16(1.0f), __bf16(1.0f), __bf16(1.0f)};
#pragma unroll
      for (int qh = 0; qh < kQH; ++qh)
        lsum[qh] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pb[qh], lsum[qh], 0, 0, 0);
    }
  };
  // mask keys >= n_valid of a 32-key block
  auto mask_blk = [&](f32x4 (&s)[2][kQH], int n_valid) __attribute__((always_inline)) {
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int qh = 0; qh < kQH; ++qh)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          s[kh][qh][j] = 4 * grp >= n_valid - 16 * kh - j ? -INFINITY : s[kh][qh][j];
  };
  // column max of a block for query half qh (every lane of the query agrees)
  auto col_max = [&](const f32x4 (&s)[2][kQH], int qh) __attribute__((always_inline)) {
    float mx = fmaxf(fmaxf(s[0][qh][0], s[0][qh][1]), fmaxf(s[0][qh][2], s[0][qh][3]));
    mx = fmaxf(mx, fmaxf(fmaxf(s[1][qh][0], s[1][qh][1]), fmaxf(s[1][qh][2], s[1][qh][3])));
    return max_across_groups(mx);
  };
  // probabilities of query half qh of a block as packed bf16: pk[qh] is the
  // P^T operand of that half, keys 4 grp .. 4 grp+3 then 16 + 4 grp .. +3; with
  // with_sums, lb[qh] is this lane's share of the block's row sum
  auto p_half = [&](const f32x4 (&s)[2][kQH], int qh, uint32_t (&pk)[kQH][4], float (&lb)[kQH],
                    auto with_sums) __attribute__((always_inline)) {
    float sum = 0.0f;
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
      for (int j = 0; j < 4; j += 2) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[kh][qh][j], scale_log2, -m_run[qh]));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[kh][qh][j + 1], scale_log2, -m_run[qh]));
        pk[qh][2 * kh + (j >> 1)] = pack_bf16(p0, p1);
        if constexpr (decltype(with_sums)::value) sum += p0 + p1;
      }
    if constexpr (decltype(with_sums)::value) lb[qh] = sum;
  };
  auto p_blk = [&](const f32x4 (&s)[2][kQH], uint32_t (&pk)[kQH][4], float (&lb)[kQH])
      __attribute__((always_inline)) {
#pragma unroll
    for (int qh = 0; qh < kQH; ++qh) p_half(s, qh, pk, lb, std::true_type{});
  };
  // The reference max is only raised when a block's probabilities (relative to
  // it) sum past kSumLimit: then the reference is raised to the block's column
  // max (O and l follow) and its probabilities are redone from the scores, which
  // are still in registers.  Below the limit every probability is at most
  // kSumLimit, so nothing overflows; infinities (scores far above the
  // reference) also exceed it.  O is rescaled after the products of the previous
  // block (issued in the same step) have been added into it.
  auto check_blk = [&](const f32x4 (&s)[2][kQH], uint32_t (&pk)[kQH][4], float (&lb)[kQH])
      __attribute__((always_inline)) {
    bool over = false;
#pragma unroll
    for (int qh = 0; qh < kQH; ++qh) over |= lb[qh] > kSumLimit;
    if (__builtin_amdgcn_ballot_w64(over) != 0) {
      float alpha[kQH];
#pragma unroll
      for (int qh = 0; qh < kQH; ++qh) {
        const float m_new = fmaxf(m_run[qh], col_max(s, qh) * scale_log2);
        alpha[qh] = __builtin_amdgcn_exp2f(m_run[qh] - m_new);
        l_run[qh] *= alpha[qh];
        m_run[qh] = m_new;
      }
      p_blk(s, pk, lb);
      // O follows the raised reference only in the lanes whose reference moved
      if (alpha[0] != 1.0f || alpha[1] != 1.0f)
#pragma unroll
        for (int qh = 0; qh < kQH; ++qh)
#pragma unroll
          for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
            for (int j = 0; j < 4; ++j) o[dt][qh][j] *= alpha[qh];
    }
#pragma unroll
    for (int qh = 0; qh < kQH; ++qh) l_run[qh] += lb[qh];
  };
  // One step of the block pipeline, in two halves that the scheduler may not
  // mix: (1) the V reads of this step, S^T of block b+1 from the K operands read
  // in the previous step and the softmax of query half 0 of block b; (2) the K
  // reads of the next step (tile kt_next, key block kb_next, into the registers
  // the S^T products have just consumed), O^T += P(b-1) V(b-1) and the softmax
  // of query half 1.  Inside a half every product is followed by its share of
  // the LDS reads and of the softmax work (exponentials, row sums, bf16
  // packing), which depends on no product of the step.  The fast pass sums
  // the probabilities on the matrix core, the other passes with VALU adds (the
  // checked pass's per-block check needs each block's sum; the exact fast pass
  // sums the unrounded probabilities).
  auto step = [&](bf16x8 (&ka)[2][C::KS], const char* vt, int kbv, const char* kt_next, int kb_next,
                  const f32x4 (&s_in)[2][kQH], f32x4 (&s_out)[2][kQH],
                  const uint32_t (&pk_in)[kQH][4], uint32_t (&pk_out)[kQH][4], float (&lb)[kQH],
                  auto pass) __attribute__((always_inline)) {
    constexpr bool kVSums = decltype(pass)::value != kPassFast;   // row sums in VALU
    constexpr int kNV = kVSums ? kHalfVALU : kHalfVALUFast;
    bf16x8 va[C::DT];
    v_read(vt, kbv, va);
    s_mma(ka, s_out);
    p_half(s_in, 0, pk_out, lb, std::bool_constant<kVSums>{});
    interleave_half<4 * C::KS, 2 * C::DT, kVReadsFirst, kNV>();
    __builtin_amdgcn_sched_barrier(0);
    k_read(kt_next, kb_next, ka);
    pv_mma(va, pk_in, std::bool_constant<!kVSums>{});
    p_half(s_in, 1, pk_out, lb, std::bool_constant<kVSums>{});
    interleave_half<2 * C::DT + (kVSums ? 0 : kQH), 2 * C::KS, 0, kNV>();
    // (the softmax results are computed inside this step, not sunk past the
    // branches that follow it)
    asm volatile("" ::"v"(pk_out[0][0]), "v"(pk_out[0][1]), "v"(pk_out[0][2]), "v"(pk_out[0][3]),
                 "v"(pk_out[1][0]), "v"(pk_out[1][1]), "v"(pk_out[1][2]), "v"(pk_out[1][3]));
    if constexpr (kVSums) asm volatile("" ::"v"(lb[0]), "v"(lb[1]));
    __builtin_amdgcn_sched_barrier(0);
  };

  // The key loop runs first as a fast pass: the reference max stays the first
  // block's column max, the row sums come from the matrix core, and nothing is
  // checked per block.  Since O and l then add exactly the same rounded
  // probabilities, how far the reference sits below the true max changes only
  // their common scale, as long as nothing overflows: a sum above kFastLimit
  // (or one that is not finite) at the end of the pass sends the workgroup's
  // unit through the key loop again as a checked pass, whose reference is
  // raised per block (check_blk).  The exact fast pass differs only in its
  // row sums: float32 sums of the unrounded probabilities (VALU adds).
  auto key_loop = [&](auto pass) __attribute__((always_inline)) {
    constexpr int kPass = decltype(pass)::value;
    auto after_step = [&](const f32x4 (&s)[2][kQH], uint32_t (&pk)[kQH][4], float (&lb)[kQH])
        __attribute__((always_inline)) {
      if constexpr (kPass == kPassChecked) {
        check_blk(s, pk, lb);
      } else if constexpr (kPass == kPassFastExact) {
#pragma unroll
        for (int qh = 0; qh < kQH; ++qh) l_run[qh] += lb[qh];
      }
    };

    // ---- prologue: tiles 0 .. 2 in flight, S^T of block 0 ----------------------
    // Tile t lives in slot t % 5.  Block b = 2t + kb is key block kb of tile t.
    Cursor c_t = {0, 0};                       // tile t of the loop below
    for (int i = 0; i < t_begin; ++i) c_t = advance(c_t);
    Cursor c_dma = c_t;                        // the tile the next copy fetches
#pragma unroll
    for (int i = 0; i < 3; ++i)
      if (i < n_tiles) {
        issue_tile(slot(i), c_dma);
        c_dma = advance(c_dma);
      }
    // S^T of even blocks (block 0 of a tile) lives in s_a, of odd blocks in s_b;
    // P of even blocks in pk_a, of odd blocks in pk_b
    f32x4 s_a[2][kQH], s_b[2][kQH];
    uint32_t pk_a[kQH][4], pk_b[kQH][4];
    float lb[kQH];
    bf16x8 ka[2][C::KS];
    int nv = min(kBK, seg_len(c_t.sg) - c_t.k0);   // valid keys of tile t
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    k_read(slot(0), 0, ka);
    s_mma(ka, s_a);
    k_read(slot(0), 1, ka);
    if (nv < 32) mask_blk(s_a, nv);
    // reference max from the first block: its column max (O and l are zero)
#pragma unroll
    for (int qh = 0; qh < kQH; ++qh) m_run[qh] = col_max(s_a, qh) * scale_log2;
    // the first step adds P = 0 times V of tile 0 (finite) into O^T
#pragma unroll
    for (int qh = 0; qh < kQH; ++qh)
#pragma unroll
      for (int i = 0; i < 4; ++i) pk_b[qh][i] = 0;

    // ---- main loop over tiles: a barrier and two pipeline steps per tile -----
    // barrier t: tile t+1 has landed and tile t-2 is no longer read; the waves
    //            copy tile t+3 into its slot.
    // A(t): S^T(2t+1) (tile t);   O^T += P(2t-1) V(2t-1) (tile t-1);  P(2t);
    //       K of tile t+1, block 0.
    // B(t): S^T(2t+2) (tile t+1); O^T += P(2t) V(2t) (tile t);        P(2t+1);
    //       K of tile t+1, block 1.
    // (after the last tile the K reads and S^T products use a stale slot:
    // result unused)
    int i0 = 0;   // slot of tile t
#pragma unroll 1
    for (int t = 0; t < n_tiles; ++t) {
      const int i1 = i0 == 4 ? 0 : i0 + 1;
      const int i4 = i0 == 0 ? 4 : i0 - 1;        // slot of tile t-1
      const int i3 = i0 >= 2 ? i0 - 2 : i0 + 3;   // slot of tile t-2 (and of tile t+3)
      // each copying wave waits for its own copies of tile t+1 (those of tile
      // t+2 may stay in flight); LDS reads need no wait: the last reads of tile
      // t-2 were consumed by products of the previous tile
      if (wave < kCopyWaves) {
        if (t + 2 < n_tiles)
          __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * C::BLOCKS_PER_WAVE));
        else
          __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
      }
      asm volatile("s_barrier" ::: "memory");
      if (t + 3 < n_tiles) {
        issue_tile(slot(i3), c_dma);
        c_dma = advance(c_dma);
      }
      char* st = slot(i0);
      char* sn = slot(i1);
      step(ka, (t == 0 ? st : slot(i4)) + C::TILE, 1, sn, 0, s_a, s_b, pk_b, pk_a, lb, pass);
      if (nv < kBK) mask_blk(s_b, nv - 32);   // keys past a segment's end
      after_step(s_a, pk_a, lb);
      int nv_next = 32;   // valid keys of tile t+1 (no mask after the last tile)
      if (t + 1 < n_tiles) {
        c_t = advance(c_t);
        nv_next = min(kBK, seg_len(c_t.sg) - c_t.k0);
      }
      step(ka, st + C::TILE, 0, sn, 1, s_b, s_a, pk_a, pk_b, lb, pass);
      if (nv_next < 32) mask_blk(s_a, nv_next);
      after_step(s_b, pk_b, lb);
      nv = nv_next;
      i0 = i1;
    }
    {
      // O^T += P(2n-1) V(2n-1): block 1 of the last tile
      bf16x8 va[C::DT];
      v_read(slot(i0 == 0 ? 4 : i0 - 1) + C::TILE, 1, va);
      pv_mma(va, pk_b, std::bool_constant<kPass == kPassFast>{});
    }
  };

  // A launch that also writes the log-sum-exp (the packed forward of the
  // training path) runs the exact fast pass: its row sums are float32 sums of
  // the unrounded probabilities, as the backward's log-sum-exp is defined.
  bool exact_sums = false;
  if constexpr (kPacked) exact_sums = src.lse != nullptr;
  float l_tot[kQH];   // the row sum of the lane's query
  bool checked_pass = true;
  {
    if (kPacked && exact_sums) {
      if constexpr (kPacked) {
        key_loop(std::integral_constant<int, kPassFastExact>{});
#pragma unroll
        for (int qh = 0; qh < kQH; ++qh) l_tot[qh] = sum_across_groups(l_run[qh]);
      }
    } else {
      key_loop(std::integral_constant<int, kPassFast>{});
#pragma unroll
      for (int qh = 0; qh < kQH; ++qh) l_tot[qh] = lsum[qh][0];
    }
    bool overflow = false;
#pragma unroll
    for (int qh = 0; qh < kQH; ++qh)
      overflow |= !(l_tot[qh] <= kFastLimit);   // (a NaN sum counts as an overflow)
    // One flag per wave through LDS (the tiles are no longer read after the
    // first barrier; the last one keeps the flags from being overwritten by
    // the checked pass's copies before every wave has read them).
    const bool mine = __builtin_amdgcn_ballot_w64(overflow) != 0;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    int* flags = reinterpret_cast<int*>(lds);
    if (lane == 0) flags[wave] = mine ? 1 : 0;
    __syncthreads();
    bool any = false;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) any |= flags[w] != 0;
    __syncthreads();
    checked_pass = any;
    if (any) {
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt)
#pragma unroll
        for (int qh = 0; qh < kQH; ++qh) o[dt][qh] = f32x4{};
#pragma unroll
      for (int qh = 0; qh < kQH; ++qh) l_run[qh] = 0.0f;
    }
  }
  if (checked_pass) {
    key_loop(std::integral_constant<int, kPassChecked>{});
#pragma unroll
    for (int qh = 0; qh < kQH; ++qh) l_tot[qh] = sum_across_groups(l_run[qh]);
  }

  // normalise and store: lane (l16, grp) of tile (dt, qh) holds query
  // q0 + 16 qh + l16 at d = 16 dt + 4 grp + j
#pragma unroll
  for (int qh = 0; qh < kQH; ++qh) {
    const int qi = q0 + 16 * qh + l16;
    const float inv = 1.0f / l_tot[qh];
    if constexpr (kPacked) {
      // base-2 log-sum-exp of the scaled logits, for the backward pass
      if (src.lse != nullptr && grp == 0 && qi < nq)
        src.lse[(int64_t(chunk) * nq + qi) * heads + head] = m_run[qh] + log2f(l_tot[qh]);
    }
    if (n_parts > 1) {
      // unnormalised partial result of this part: O (row = query of the
      // workgroup), the reference max and the sum, merged by the tail kernel
      float* pb = tail.part + size_t((logical - tail.n_full) * n_parts + part_id) *
                                  (kBlockQ * D + 2 * kBlockQ);
      const int row = wave * kWaveQ + 16 * qh + l16;
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt)
        *reinterpret_cast<f32x4*>(pb + row * D + 16 * dt + 4 * grp) = o[dt][qh];
      if (grp == 0) {
        pb[kBlockQ * D + row] = m_run[qh];
        pb[kBlockQ * D + kBlockQ + row] = l_tot[qh];
      }
    } else if (qi < nq) {
      __bf16* op = out + (int64_t(qi) * heads + head) * D + 4 * grp;
#pragma unroll
      for (int dt = 0; dt < C::DT; ++dt) {
        u32x2 w;
        w.x = pack_bf16(o[dt][qh][0] * inv, o[dt][qh][1] * inv);
        w.y = pack_bf16(o[dt][qh][2] * inv, o[dt][qh][3] * inv);
        *reinterpret_cast<u32x2*>(op + 16 * dt) = w;
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
