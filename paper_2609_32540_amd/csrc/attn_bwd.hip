// Backward pass of the packed block-causal attention (bf16 in and out, float32
// accumulation), the gradient of the packed training forward through its KV
// edges.  With c = scale * log2(e) and the forward's base-2 log-sum-exp L_i:
//   P_ij  = 2^(c q_i.k_j - L_i)                 (visible pairs only)
//   D_i   = dO_i . O_i
//   dV_j  = sum_i P_ij dO_i
//   dS_ij = P_ij (dO_i . v_j - D_i)
//   dQ_i  = scale sum_j dS_ij k_j
//   dK_j  = scale sum_i dS_ij q_i
// Three launches: D; dQ (query-stationary: a workgroup holds 256 queries of
// one chunk and head and streams the 64-key tiles of their read set, like the
// forward); dK and dV together (key-stationary: a workgroup holds 256 keys of
// one chunk or anchor frame and head and streams the query tiles of every
// chunk that sees them, 32 rows per tile at d = 128, 64 at d = 64).  Every
// output element is written by exactly one workgroup: no atomics.
//
// Products on v_mfma_f32_32x32x16_bf16 with the forward's operand layouts: the
// stationary side (Q^T and dO^T, or K^T and V^T) sits in registers as the B
// operand (the second one, where registers run out, in a swizzled LDS copy),
// tiles of the streamed side are copied HBM -> LDS (global_load_lds) ahead of
// use into a ring of two to four slots and read as the A operand (16-byte
// rows) or, transposed, with ds_read_b64_tr_b16; P and dS go from the
// accumulators to the B operand of the next product as bf16 (nearest even).
// With three or more slots the two waves of each SIMD work half a tile apart,
// as in the forward kernel (see Ring).

#include <hip/hip_runtime.h>

#include <math.h>

#include <cstring>

#include "ff_internal.h"

namespace ff {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))
#define GLOBAL_PTR(p) ((const __attribute__((address_space(1))) void*)(p))

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kBlockN = 32 * kWaves;   // stationary columns (queries or keys) per workgroup
constexpr int kBT = 64;                // streamed rows per tile (32 in the d = 128 dK/dV pass)
constexpr int kXcds = 8;
constexpr int kMaxRuns = 2 * FF_MAX_ANCHOR_FRAMES + 1;   // segments of one streamed set

template <int D, int BT = kBT>
struct Cfg {
  static constexpr int KS = D / 16;
  static constexpr int DB = D / 32;
  static constexpr int ROWB = 2 * D;
  static constexpr int CPR = D / 8;
  static constexpr int RPB = 1024 / ROWB;
  static constexpr int BLOCKS = BT / RPB;               // 1 KB copies per tile and tensor
  static constexpr int TILE = BT * ROWB;
  static constexpr int VEC = BT * 4;                    // one float per streamed row
  static_assert(BLOCKS % kWaves == 0, "every wave copies the same number of 1 KB blocks");
};

// Ring schedules.  NS = 2: all eight waves copy tile t+1 after barrier t and
// then work on tile t in lock step.  NS >= 3: waves 0-3 copy tile t + NS - 2
// after barrier t (before their blocks with three slots, after them with
// four) and run both 32-row blocks of tile t; their SIMD partners,
// waves 4-7, run block 1 of tile t-1 and then block 0 of tile t, half a tile
// later, so one wave's exponentials meet the other's matrix work.  Tile u
// sits in slot u % NS; its last reads (block 1 by waves 4-7) precede barrier
// u+2, and its slot is refilled at barrier u + 2 at the earliest.
template <int NS>
struct Ring {
  static_assert(NS >= 2 && NS <= 4, "two to four slots");
  static constexpr bool kOffset = NS >= 3;
  static constexpr int kCopyWaves = kOffset ? kWaves / 2 : kWaves;
  static constexpr int kAhead = kOffset ? NS - 2 : 1;   // tiles copied ahead of the first reader
};

// the forward's LDS swizzle (conflict-free 16-byte row reads and transposing reads)
template <int D>
__device__ inline int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

__device__ inline uint32_t pack_bf16(float a, float b) {
  f32x2 f = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

__device__ inline uint64_t readlane_u64(uint64_t v, int lane) {
  const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v)), lane));
  const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(v >> 32)), lane));
  return (uint64_t(hi) << 32) | uint64_t(lo);
}

// Streams the tiles of up to kMaxRuns runs of rows through an LDS ring of
// two to four slots.  Run i (held by lane i, read with v_readlane): `len` rows of two
// token-major tensors (row r at a + r * row_bytes and b + r * row_bytes, this
// head's columns) and, with kVec, two float vectors (element r at
// va + r * vec_bytes and vb + r * vec_bytes).
template <int D, bool kVec, int kCopyWaves, int BT = kBT>
struct Stream {
  using C = Cfg<D, BT>;
  static constexpr int BPW = C::BLOCKS / kCopyWaves;   // 1 KB blocks per copying wave and tensor
  int len = 0;
  uint64_t a = 0, b = 0, va = 0, vb = 0;
  uint32_t row_bytes, vec_bytes;
  int n_runs, n_tiles;
  int sg = 0, k0 = 0;    // tile being copied next
  int cp_row[BPW], cp_choff[BPW];
  int wave, lane;

  __device__ void init_copy_lanes() {
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      const int r = (wave * BPW + i) * C::RPB + lane / C::CPR;
      cp_row[i] = r;
      cp_choff[i] = 16 * ((lane % C::CPR) ^ swz<D>(r));
    }
  }

  __device__ int run_len(int i) const { return __builtin_amdgcn_readlane(len, i); }
  __device__ void advance(int& s, int& k) const {
    k += BT;
    if (k >= run_len(s)) {
      ++s;
      k = 0;
    }
  }
  // copy the next tile into `slot` (rows past a partial tile's end repeat its
  // last row); called by waves 0 .. kCopyWaves-1
  __device__ void issue(char* slot) {
    const int n = run_len(sg);
    const char* ga = reinterpret_cast<const char*>(readlane_u64(a, sg));
    const char* gb = reinterpret_cast<const char*>(readlane_u64(b, sg));
    const bool partial = k0 + BT > n;
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      int tok = k0 + cp_row[i];
      if (partial) tok = min(tok, n - 1);
      const uint32_t off = uint32_t(tok) * row_bytes + uint32_t(cp_choff[i]);
      char* dst = slot + (wave * BPW + i) * 1024;
      __builtin_amdgcn_global_load_lds(GLOBAL_PTR(ga + off), LDS_PTR(void, dst), 16, 0, 0);
      __builtin_amdgcn_global_load_lds(GLOBAL_PTR(gb + off), LDS_PTR(void, dst + C::TILE), 16, 0, 0);
    }
    if constexpr (kVec) {
      if (wave == 0 && lane < BT) {   // one float per row: lanes 0 .. BT-1
        const char* pa = reinterpret_cast<const char*>(readlane_u64(va, sg));
        const char* pb = reinterpret_cast<const char*>(readlane_u64(vb, sg));
        const uint32_t off = uint32_t(min(k0 + lane, n - 1)) * vec_bytes;
        __builtin_amdgcn_global_load_lds(GLOBAL_PTR(pa + off), LDS_PTR(void, slot + 2 * C::TILE), 4, 0, 0);
        __builtin_amdgcn_global_load_lds(GLOBAL_PTR(pb + off), LDS_PTR(void, slot + 2 * C::TILE + C::VEC), 4, 0, 0);
      }
    }
    advance(sg, k0);
  }
};

// Drives the tile loop of one workgroup over n > 0 tiles of kBlocks 32-row
// blocks with the Ring<NS> schedule.  issue(slot) copies the stream's next
// tile into slot (copy waves only); next_nv() returns the valid rows of the
// next tile this wave works on and advances its cursor; block(slot, kb, nv)
// works on block kb of the tile in slot.  With one block per tile, waves 4-7
// work on tile t-1 while waves 0-3 work on tile t.  Slots are distinct __shared__ arrays, referenced
// statically (the loops are unrolled by NS), so the compiler never orders a
// read of one slot behind a copy into another.
template <int NS, int kBlocks, int kPerTile, class Issue, class NextNv, class Block>
__device__ __attribute__((always_inline)) inline void run_ring(int n, int wave, char* s0, char* s1,
                                                               char* s2, char* s3, Issue& issue,
                                                               NextNv& next_nv, Block& block) {
  using R = Ring<NS>;
  auto sync = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };
  // Barrier of a copying wave before step t when tiles are copied two ahead:
  // tile t must have landed, but tile t + 1 (issued after it, at least
  // kPerTile memory instructions) may stay in flight if it was issued at all
  // (t + 1 < n).  A bare s_barrier, since the workgroup fence of
  // __syncthreads would wait for every copy.
  static_assert(R::kAhead <= 2, "at most one tile in flight past the one read next");
  constexpr int kKeep = (R::kAhead - 1) * kPerTile;
  static_assert(kKeep < 16, "vmcnt field");
  auto copy_sync = [&](int t) __attribute__((always_inline)) {
    if constexpr (kKeep == 0) {
      sync();
    } else {
      // vmcnt = kKeep or 0, lgkmcnt = 0, expcnt not waited for
      if (t + 1 < n)
        __builtin_amdgcn_s_waitcnt(kKeep | (7 << 4));
      else
        __builtin_amdgcn_s_waitcnt(7 << 4);
      asm volatile("s_barrier" ::: "memory");
    }
  };
  if constexpr (!R::kOffset) {
    issue(s0);
    auto step = [&](int t, char* cur, char* nxt) __attribute__((always_inline)) {
      sync();
      if (t + 1 < n) issue(nxt);
      const int nv = next_nv();
      block(cur, 0, nv);
      if constexpr (kBlocks == 2) block(cur, 1, nv);
    };
    for (int t = 0; t < n;) {
      step(t, s0, s1);
      if (++t >= n) break;
      step(t, s1, s0);
      ++t;
    }
  } else if (wave < R::kCopyWaves) {
    issue(s0);
    if (R::kAhead > 1 && n > 1) issue(s1);
    // With two tiles ahead the copies go out after the step's blocks (what the
    // blocks reload from scratch then waits only for older copies); with one,
    // before them (the copy needs the whole step to land).
    auto step = [&](int t, char* cur, char* ahead) __attribute__((always_inline)) {
      copy_sync(t);
      if constexpr (R::kAhead < 2)
        if (t + R::kAhead < n) issue(ahead);
      const int nv = next_nv();
      block(cur, 0, nv);
      if constexpr (kBlocks == 2) block(cur, 1, nv);
      if constexpr (R::kAhead >= 2)
        if (t + R::kAhead < n) issue(ahead);
    };
    for (int t = 0; t < n;) {
      if constexpr (NS == 3) {
        step(t, s0, s1);
        if (++t >= n) break;
        step(t, s1, s2);
        if (++t >= n) break;
        step(t, s2, s0);
        ++t;
      } else {
        step(t, s0, s2);
        if (++t >= n) break;
        step(t, s1, s3);
        if (++t >= n) break;
        step(t, s2, s0);
        if (++t >= n) break;
        step(t, s3, s1);
        ++t;
      }
    }
    sync();   // matches the extra barrier of waves 4-7
  } else if constexpr (kBlocks == 1) {
    sync();
    // step t: barrier t, tile t-1
    auto step = [&](int t, char* prev) __attribute__((always_inline)) {
      sync();
      block(prev, 0, next_nv());
    };
    for (int t = 1;;) {
      if constexpr (NS == 3) {
        step(t, s0);
        if (t++ >= n) break;
        step(t, s1);
        if (t++ >= n) break;
        step(t, s2);
        if (t++ >= n) break;
      } else {
        step(t, s0);
        if (t++ >= n) break;
        step(t, s1);
        if (t++ >= n) break;
        step(t, s2);
        if (t++ >= n) break;
        step(t, s3);
        if (t++ >= n) break;
      }
    }
  } else {
    sync();
    int nv_prev = next_nv();
    block(s0, 0, nv_prev);
    // step t: barrier t, block 1 of tile t-1, block 0 of tile t while t < n
    auto step = [&](int t, char* prev, char* cur) __attribute__((always_inline)) {
      sync();
      block(prev, 1, nv_prev);
      if (t < n) {
        nv_prev = next_nv();
        block(cur, 0, nv_prev);
      }
    };
    for (int t = 1;;) {
      if constexpr (NS == 3) {
        step(t, s0, s1);
        if (t++ >= n) break;
        step(t, s1, s2);
        if (t++ >= n) break;
        step(t, s2, s0);
        if (t++ >= n) break;
      } else {
        step(t, s0, s1);
        if (t++ >= n) break;
        step(t, s1, s2);
        if (t++ >= n) break;
        step(t, s2, s3);
        if (t++ >= n) break;
        step(t, s3, s0);
        if (t++ >= n) break;
      }
    }
  }
}

// acc[kb] = A(rows kb*32 .. +31 of the tile) x B^T, B the stationary operand
// (lane (l32, half) holds column l32, elements 16 ks + 8 half .. +7)
// (kInit: added to the accumulator's initial value; kPattern: with its own
// read-ahead schedule)
template <int D, bool kInit = false, bool kPattern = true>
__device__ inline void rows_times_b(const char* tile, int kb, int a_lane, const bf16x8 (&breg)[D / 16],
                                    f32x16& acc) {
  if constexpr (!kInit)
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = 0.0f;
  const char* base = tile + kb * 32 * Cfg<D>::ROWB;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const bf16x8 a = *reinterpret_cast<const bf16x8*>(base + (a_lane ^ (ks << 5)));
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, breg[ks], acc, 0, 0, 0);
  }
  if constexpr (kPattern) {
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      if (ks + 2 < D / 16) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
  }
}

// out[db] += (rows kb*32 .. +31 of the tile)^T x P, P packed bf16 from the
// accumulator layout (register j of the block = row 8 (j/4) + 4 half + j%4)
template <int D>
__device__ inline void rows_t_times_p(const char* tile, int kb, const int (&t_lane)[2],
                                      const uint32_t (&pk)[8], f32x16 (&out)[D / 32]) {
#pragma unroll
  for (int mh = 0; mh < 2; ++mh) {
    const u32x4 pu = {pk[4 * mh + 0], pk[4 * mh + 1], pk[4 * mh + 2], pk[4 * mh + 3]};
    const bf16x8 pb = __builtin_bit_cast(bf16x8, pu);
    const char* base = tile + (kb * 32 + 16 * mh) * Cfg<D>::ROWB;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, base + (t_lane[0] ^ (db << 6))));
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(LDS_PTR(s16x4, base + (t_lane[1] ^ (db << 6))));
      const u32x2 lo2 = __builtin_bit_cast(u32x2, lo), hi2 = __builtin_bit_cast(u32x2, hi);
      const u32x4 au = {lo2[0], lo2[1], hi2[0], hi2[1]};
      out[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, au), pb, out[db], 0, 0, 0);
    }
  }
}

// lane address bases of the two LDS read patterns (as in the forward)
template <int D>
struct Lanes {
  int a_lane;
  int t_lane[2];
  __device__ Lanes(int lane) {
    const int l32 = lane & 31, half = lane >> 5;
    a_lane = l32 * Cfg<D>::ROWB + ((half ^ swz<D>(l32)) << 4);
    const int g = lane >> 4, lp = lane & 15;
    const int v_row = 4 * (g >> 1) + (lp >> 2);
    const int v_dsub = 16 * (g & 1) + 4 * (lp & 3);
#pragma unroll
    for (int hi = 0; hi < 2; ++hi) {
      const int r = v_row + 8 * hi;
      t_lane[hi] = r * Cfg<D>::ROWB + (((v_dsub >> 3) ^ swz<D>(r)) << 4) + (v_dsub & 7) * 2;
    }
  }
};

// load the stationary B operand of one wave: 32 columns (rows of a token-major
// tensor, clamped to n - 1), lane (l32, half) gets elements 16 ks + 8 half .. +7
template <int D>
__device__ inline void load_b(const __bf16* base, int64_t row_elems, int col0, int n, int lane,
                              bf16x8 (&breg)[D / 16]) {
  const int r = min(col0 + (lane & 31), n - 1);
  const __bf16* p = base + int64_t(r) * row_elems + 8 * (lane >> 5);
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) breg[ks] = *reinterpret_cast<const bf16x8*>(p + 16 * ks);
}

// Stationary operand kept in LDS instead of registers (register budget): the
// 32 rows of wave w at stat + (32 w + r) * ROWB, 16-byte chunks swizzled as in
// the tiles, so reading it back as a B operand is conflict-free.
template <int D>
__device__ inline void stash_b(char* stat, const __bf16* base, int64_t row_elems, int col0, int n,
                               int wave, int lane) {
  // lane l writes chunks l % CPR (and l % CPR + ..) of rows: 64 lanes cover 64 * 16 B per pass
  constexpr int CPR = Cfg<D>::CPR;
#pragma unroll
  for (int pass = 0; pass < 32 * CPR / 64; ++pass) {
    const int idx = pass * 64 + lane;
    const int r = idx / CPR, ch = idx % CPR;
    const int src = min(col0 + r, n - 1);
    const u32x4 v = *reinterpret_cast<const u32x4*>(base + int64_t(src) * row_elems + 8 * ch);
    *reinterpret_cast<u32x4*>(stat + (32 * wave + r) * Cfg<D>::ROWB + ((ch ^ swz<D>(r)) << 4)) = v;
  }
}

// acc = A(rows kb*32 .. +31 of the tile) x B^T with B read from the stash
// (kPattern: with its own read-ahead schedule)
template <int D, bool kPattern = true>
__device__ inline void rows_times_stash(const char* tile, int kb, int a_lane, const char* stat_w,
                                        f32x16& acc) {
#pragma unroll
  for (int j = 0; j < 16; ++j) acc[j] = 0.0f;
  const char* base = tile + kb * 32 * Cfg<D>::ROWB;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const bf16x8 a = *reinterpret_cast<const bf16x8*>(base + (a_lane ^ (ks << 5)));
    const bf16x8 b = *reinterpret_cast<const bf16x8*>(stat_w + (a_lane ^ (ks << 5)));
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
  }
  if constexpr (kPattern) {
    // operands read two products ahead at most (register budget)
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      if (ks + 2 < D / 16) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
  }
}

// store scale * acc^T: acc rows = d (32 db + 8 (j/4) + 4 half + j%4), columns = lanes
template <int D>
__device__ inline void store_t(__bf16* base, int64_t row_elems, int col, int n, int lane,
                               const f32x16 (&acc)[D / 32], float scale) {
  if (col >= n) return;
  __bf16* p = base + int64_t(col) * row_elems + 4 * (lane >> 5);
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      u32x2 w;
      w.x = pack_bf16(acc[db][4 * a + 0] * scale, acc[db][4 * a + 1] * scale);
      w.y = pack_bf16(acc[db][4 * a + 2] * scale, acc[db][4 * a + 3] * scale);
      *reinterpret_cast<u32x2*>(p + 32 * db + 8 * a) = w;
    }
}

__device__ inline int xcd_logical(int b, int n_wg) {
  const int xcd = b % kXcds, idx = b / kXcds;
  const int per = n_wg / kXcds, rem = n_wg % kXcds;
  return xcd * per + min(xcd, rem) + idx;
}

// Groups of `group` consecutive logical units that share a read set (the q
// tiles of one (chunk, head)) but cost differently from group to group: XCD x
// takes the groups x, x + 8, .. so every XCD gets the same mix; the last
// n_groups % 8 groups run in order.
__device__ inline int xcd_interleaved(int b, int n_wg, int group) {
  const int n_groups = n_wg / group;
  const int n_even = n_groups - n_groups % kXcds;
  if (b >= n_even * group) return b;
  const int xcd = b % kXcds, idx = b / kXcds;
  return (xcd + kXcds * (idx / group)) * group + idx % group;
}

// ---- D_i = dO_i . O_i ---------------------------------------------------------------
// L = d / 8 consecutive lanes per row (16 bytes of O and of dO each, so a wave
// reads contiguous memory), partial sums combined across the L lanes.
template <int L>
__global__ __launch_bounds__(256) void bwd_delta_kernel(const __bf16* __restrict__ o,
                                                        const __bf16* __restrict__ dout,
                                                        float* __restrict__ delta, int64_t rows) {
  const int64_t t = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int64_t r = t / L;
  float acc = 0.0f;
  if (r < rows) {
    const u32x4 a = reinterpret_cast<const u32x4*>(o)[t];
    const u32x4 b = reinterpret_cast<const u32x4*>(dout)[t];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      acc = fmaf(__uint_as_float(a[j] << 16), __uint_as_float(b[j] << 16), acc);
      acc = fmaf(__uint_as_float(a[j] & 0xffff0000u), __uint_as_float(b[j] & 0xffff0000u), acc);
    }
  }
#pragma unroll
  for (int off = L / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, L);
  if (r < rows && (t % L) == 0) delta[r] = acc;
}

// ---- dQ: query-stationary ---------------------------------------------------------------
// Slot = K tile then V tile (the queries' log-sum-exp and D sit in lanes).
template <int D, int NS>
__device__ __attribute__((always_inline)) inline void dq_body(
    const __bf16* __restrict__ q, const __bf16* __restrict__ dout, const float* __restrict__ lse,
    const float* __restrict__ delta, __bf16* __restrict__ dq, int heads, float c_log2, float scale,
    const PackedPlan& plan, int n_qtiles, char* s0, char* s1, char* s2, char* s3, char* stash) {
  using C = Cfg<D>;
  using R = Ring<NS>;
  const int nq = plan.chunk_tokens;
  const int logical = xcd_interleaved(blockIdx.x, gridDim.x, n_qtiles);
  const int chunk = logical / (heads * n_qtiles);
  const int rest = logical - chunk * heads * n_qtiles;
  const int head = rest / n_qtiles, qt = rest % n_qtiles;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, l32 = lane & 31, half = lane >> 5;
  const int64_t tok0 = int64_t(chunk) * nq;
  const int64_t row_elems = int64_t(heads) * D;
  const int q0 = qt * kBlockN + wave * 32;

  bf16x8 qreg[C::KS];
  load_b<D>(q + tok0 * row_elems + head * D, row_elems, q0, nq, lane, qreg);
  stash_b<D>(stash, dout + tok0 * row_elems + head * D, row_elems, q0, nq, wave, lane);
  const char* stash_w = stash + 32 * wave * C::ROWB;
  const int qi = min(q0 + l32, nq - 1);
  const float L = lse[(tok0 + qi) * heads + head];
  const float Dq = delta[(tok0 + qi) * heads + head];
  f32x16 acc[C::DB];
#pragma unroll
  for (int db = 0; db < C::DB; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[db][j] = 0.0f;

  Stream<D, false, R::kCopyWaves> st;
  st.wave = wave;
  st.lane = lane;
  st.row_bytes = uint32_t(2 * row_elems);
  st.n_runs = packed_num_segments(plan, chunk);
#pragma unroll
  for (int i = 0; i < kMaxRuns; ++i)
    if (lane == i && i < st.n_runs) {
      const KvSegment sg = packed_segment(plan, chunk, i, heads, D, 2);
      st.len = sg.len;
      st.a = reinterpret_cast<uint64_t>(sg.k) + 2ull * uint64_t(head) * D;
      st.b = reinterpret_cast<uint64_t>(sg.v) + 2ull * uint64_t(head) * D;
    }
  st.n_tiles = 0;
  for (int i = 0; i < st.n_runs; ++i) st.n_tiles += (st.run_len(i) + kBT - 1) / kBT;
  st.init_copy_lanes();
  Lanes<D> ln(lane);
  int csg = 0, ck0 = 0;   // next tile this wave works on

  auto issue = [&](char* slot) __attribute__((always_inline)) { st.issue(slot); };
  auto next_nv = [&]() __attribute__((always_inline)) {
    const int nv = min(kBT, st.run_len(csg) - ck0);
    st.advance(csg, ck0);
    return nv;
  };
  auto block = [&](const char* cur, int kb, int nv) __attribute__((always_inline)) {
    // keep the per-read address arithmetic inside the loop (no hoisted copies)
    asm volatile("" : "+v"(ln.a_lane), "+v"(ln.t_lane[0]), "+v"(ln.t_lane[1]));
    f32x16 sv, dp;
    rows_times_b<D>(cur, kb, ln.a_lane, qreg, sv);                      // S^T = K Q^T
    __builtin_amdgcn_sched_barrier(0);
    rows_times_stash<D>(cur + C::TILE, kb, ln.a_lane, stash_w, dp);     // dP^T = V dO^T
    __builtin_amdgcn_sched_barrier(0);
    uint32_t pk[8];
#pragma unroll
    for (int j = 0; j < 16; j += 2) {
      float v2[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int key = kb * 32 + 8 * ((j + e) >> 2) + 4 * half + ((j + e) & 3);
        const float p = key < nv ? __builtin_amdgcn_exp2f(fmaf(sv[j + e], c_log2, -L)) : 0.0f;
        v2[e] = p * (dp[j + e] - Dq);
      }
      pk[j >> 1] = pack_bf16(v2[0], v2[1]);
    }
    rows_t_times_p<D>(cur, kb, ln.t_lane, pk, acc);                     // dQ^T += K^T dS^T
    __builtin_amdgcn_sched_barrier(0);   // one 32-key block at a time (register budget)
  };
  if (st.n_tiles > 0)
    run_ring<NS, 2, 2 * decltype(st)::BPW>(st.n_tiles, wave, s0, s1, s2, s3, issue, next_nv, block);
  store_t<D>(dq + tok0 * row_elems + head * D, row_elems, q0 + l32, nq, lane, acc, scale);
}

template <int D, int NS>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void bwd_dq_kernel(const __bf16* __restrict__ q, const __bf16* __restrict__ dout,
                   const float* __restrict__ lse, const float* __restrict__ delta,
                   __bf16* __restrict__ dq, int heads, float c_log2, float scale, PackedPlan plan,
                   int n_qtiles) {
  constexpr int kSlot = 2 * Cfg<D>::TILE;
  __shared__ __attribute__((aligned(1024))) char stash[kBlockN * Cfg<D>::ROWB];
  __shared__ __attribute__((aligned(1024))) char l0[kSlot];
  __shared__ __attribute__((aligned(1024))) char l1[kSlot];
  if constexpr (NS == 2) {
    dq_body<D, NS>(q, dout, lse, delta, dq, heads, c_log2, scale, plan, n_qtiles, l0, l1, l1, l1, stash);
  } else if constexpr (NS == 3) {
    __shared__ __attribute__((aligned(1024))) char l2[kSlot];
    dq_body<D, NS>(q, dout, lse, delta, dq, heads, c_log2, scale, plan, n_qtiles, l0, l1, l2, l2, stash);
  } else {
    __shared__ __attribute__((aligned(1024))) char l2[kSlot];
    __shared__ __attribute__((aligned(1024))) char l3[kSlot];
    dq_body<D, NS>(q, dout, lse, delta, dq, heads, c_log2, scale, plan, n_qtiles, l0, l1, l2, l3, stash);
  }
}

// ---- dK or dV: key-stationary -----------------------------------------------------------
// Key units: unit u < n_chunks * kpc is keys [256 k, 256 k + 256) of chunk
// u / kpc; the rest are anchor frames, kpf units each.  Each unit streams the
// query runs that see it (chunks max(0, .) .. c + window of the packed clip,
// or the chunk runs listed for the anchor frame).
struct KeyUnits {
  int32_t kpc, kpf, n_frames;
  uint8_t frame_runs[FF_MAX_ANCHOR_FRAMES * 8][16];   // per anchor frame: (first chunk, count) pairs
};

// dK and dV of one key unit.  Slot = Q tile, dO tile, their log-sum-exp and D.
template <int D, int NS, int BT>
__device__ __attribute__((always_inline)) inline void dkv_body(
    const __bf16* __restrict__ q, const __bf16* __restrict__ dout, const float* __restrict__ lse,
    const float* __restrict__ delta, __bf16* __restrict__ dk_chunks, __bf16* __restrict__ dk_anchor,
    __bf16* __restrict__ dv_chunks, __bf16* __restrict__ dv_anchor, int heads, float c_log2,
    float scale, const PackedPlan& plan, const KeyUnits& ku, char* s0, char* s1, char* s2, char* s3,
    char* stash) {
  using C = Cfg<D, BT>;
  using R = Ring<NS>;
  constexpr int kBlocks = BT / 32;
  const int nq = plan.chunk_tokens, G = plan.frame_tokens;
  const int n_units = plan.n_chunks * ku.kpc + ku.n_frames * ku.kpf;
  const int logical = xcd_logical(blockIdx.x, gridDim.x);
  const int head = logical / n_units;
  const int unit = logical - head * n_units;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, l32 = lane & 31, half = lane >> 5;
  const int64_t row_elems = int64_t(heads) * D;
  const bool is_chunk = unit < plan.n_chunks * ku.kpc;
  int owner, k_first, n_keys;
  const __bf16 *kbase, *vbase;
  __bf16 *obase_k, *obase_v;
  if (is_chunk) {
    owner = unit / ku.kpc;
    k_first = (unit % ku.kpc) * kBlockN;
    n_keys = nq;
    kbase = static_cast<const __bf16*>(plan.k) + int64_t(owner) * nq * row_elems;
    vbase = static_cast<const __bf16*>(plan.v) + int64_t(owner) * nq * row_elems;
    obase_k = dk_chunks + int64_t(owner) * nq * row_elems;
    obase_v = dv_chunks + int64_t(owner) * nq * row_elems;
  } else {
    const int a = unit - plan.n_chunks * ku.kpc;
    owner = a / ku.kpf;
    k_first = (a % ku.kpf) * kBlockN;
    n_keys = G;
    kbase = static_cast<const __bf16*>(plan.ak) + int64_t(owner) * G * row_elems;
    vbase = static_cast<const __bf16*>(plan.av) + int64_t(owner) * G * row_elems;
    obase_k = dk_anchor + int64_t(owner) * G * row_elems;
    obase_v = dv_anchor + int64_t(owner) * G * row_elems;
  }
  const int k0 = k_first + wave * 32;
  bf16x8 kreg[C::KS];
  load_b<D>(kbase + head * D, row_elems, k0, n_keys, lane, kreg);
  stash_b<D>(stash, vbase + head * D, row_elems, k0, n_keys, wave, lane);
  const char* stash_w = stash + 32 * wave * C::ROWB;
  f32x16 acc[C::DB], acc_v[C::DB];   // dK^T, dV^T
#pragma unroll
  for (int db = 0; db < C::DB; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      acc[db][j] = 0.0f;
      acc_v[db][j] = 0.0f;
    }

  // query runs of this unit
  Stream<D, true, R::kCopyWaves, BT> st;
  st.wave = wave;
  st.lane = lane;
  st.row_bytes = uint32_t(2 * row_elems);
  st.vec_bytes = uint32_t(4 * heads);
  auto set_run = [&](int i, int c0, int c1) {   // chunks c0 .. c1 - 1
    if (lane == i) {
      const int64_t t0 = int64_t(c0) * nq;
      st.len = (c1 - c0) * nq;
      st.a = reinterpret_cast<uint64_t>(q + t0 * row_elems + head * D);
      st.b = reinterpret_cast<uint64_t>(dout + t0 * row_elems + head * D);
      st.va = reinterpret_cast<uint64_t>(lse + t0 * heads + head);
      st.vb = reinterpret_cast<uint64_t>(delta + t0 * heads + head);
    }
  };
  if (is_chunk) {
    set_run(0, owner, min(owner + plan.window + 1, plan.n_chunks));
    st.n_runs = 1;
  } else {
    int n = 0;
    while (n < 8 && ku.frame_runs[owner][2 * n + 1] != 0) {
      const int c0 = ku.frame_runs[owner][2 * n];
      set_run(n, c0, c0 + ku.frame_runs[owner][2 * n + 1]);
      ++n;
    }
    st.n_runs = n;
  }
  st.n_tiles = 0;
  for (int i = 0; i < st.n_runs; ++i) st.n_tiles += (st.run_len(i) + BT - 1) / BT;
  st.init_copy_lanes();
  Lanes<D> ln(lane);
  int csg = 0, ck0 = 0;   // next tile this wave works on

  auto issue = [&](char* slot) __attribute__((always_inline)) { st.issue(slot); };
  auto next_nv = [&]() __attribute__((always_inline)) {
    const int nv = min(BT, st.run_len(csg) - ck0);
    st.advance(csg, ck0);
    return nv;
  };
  // One 32-query block in four scheduling regions: (1) S - L / c (L / c as the
  // accumulator's initial value); (2) dP, with P = 2^(c (S - L / c)) computed
  // under its products; (3) dV^T += dO^T P, with dS = P (dP - D) computed and
  // packed under its products; (4) dK^T += Q^T dS.
  const float neg_inv_c = -1.0f / c_log2;
  auto block = [&](const char* cur, int kb, int nv) __attribute__((always_inline)) {
    // keep the per-read address arithmetic inside the loop (no hoisted copies)
    asm volatile("" : "+v"(ln.a_lane), "+v"(ln.t_lane[0]), "+v"(ln.t_lane[1]));
    const float* lse_t = reinterpret_cast<const float*>(cur + 2 * C::TILE);
    const float* del_t = reinterpret_cast<const float*>(cur + 2 * C::TILE + C::VEC);
    const int row0 = kb * 32 + 4 * half;   // register 4 g + e: row row0 + 8 g + e
    f32x16 sv;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 Lr = *reinterpret_cast<const f32x4*>(lse_t + row0 + 8 * g);
#pragma unroll
      for (int e = 0; e < 4; ++e) sv[4 * g + e] = Lr[e] * neg_inv_c;
    }
    rows_times_b<D, true, false>(cur, kb, ln.a_lane, kreg, sv);   // S - L / c (rows = queries)
    __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);   // L and the first two operands
    __builtin_amdgcn_sched_group_barrier(0x002, 16, 0);
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      if (ks + 2 < C::KS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    f32x16 dp;
    rows_times_stash<D, false>(cur + C::TILE, kb, ln.a_lane, stash_w, dp);   // dP = dO V^T
    float p[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) p[j] = __builtin_amdgcn_exp2f(sv[j] * c_log2);
    // the first two products' operands; then per product two reads, two
    // multiplies and two exponentials
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (ks + 2 < C::KS) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x400, 2, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (nv < BT) {   // rows past a partial tile's end
#pragma unroll
      for (int j = 0; j < 16; ++j)
        if (row0 + 8 * (j >> 2) + (j & 3) >= nv) p[j] = 0.0f;
    }
    uint32_t pk[8], pv[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) pv[i] = pack_bf16(p[2 * i], p[2 * i + 1]);
    rows_t_times_p<D>(cur + C::TILE, kb, ln.t_lane, pv, acc_v);   // dV^T += dO^T P
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 Dr = *reinterpret_cast<const f32x4*>(del_t + row0 + 8 * g);
      float ds[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) ds[e] = p[4 * g + e] * (dp[4 * g + e] - Dr[e]);
      pk[2 * g] = pack_bf16(ds[0], ds[1]);
      pk[2 * g + 1] = pack_bf16(ds[2], ds[3]);
    }
    // D and the first two products' operands, the packs they need; then per
    // product two reads and five VALU (the other packs, dS)
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
#pragma unroll
    for (int i = 0; i < 2 * C::DB; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (i + 2 < 2 * C::DB) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    rows_t_times_p<D>(cur, kb, ln.t_lane, pk, acc);              // dK^T += Q^T dS
    __builtin_amdgcn_sched_barrier(0);   // one 32-query block at a time (register budget)
  };
  if (st.n_tiles > 0)
    run_ring<NS, kBlocks, 2 * decltype(st)::BPW>(st.n_tiles, wave, s0, s1, s2, s3, issue, next_nv,
                                                 block);
  store_t<D>(obase_k + head * D, row_elems, k0 + l32, n_keys, lane, acc, scale);
  store_t<D>(obase_v + head * D, row_elems, k0 + l32, n_keys, lane, acc_v, 1.0f);
}

template <int D, int NS, int BT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void bwd_dkv_kernel(const __bf16* __restrict__ q, const __bf16* __restrict__ dout,
                    const float* __restrict__ lse, const float* __restrict__ delta,
                    __bf16* __restrict__ dk_chunks, __bf16* __restrict__ dk_anchor,
                    __bf16* __restrict__ dv_chunks, __bf16* __restrict__ dv_anchor, int heads,
                    float c_log2, float scale, PackedPlan plan, KeyUnits ku) {
  constexpr int kSlot = 2 * Cfg<D, BT>::TILE + 2 * Cfg<D, BT>::VEC;
  __shared__ __attribute__((aligned(1024))) char stash[kBlockN * Cfg<D>::ROWB];
  __shared__ __attribute__((aligned(1024))) char l0[kSlot];
  __shared__ __attribute__((aligned(1024))) char l1[kSlot];
  if constexpr (NS == 2) {
    dkv_body<D, NS, BT>(q, dout, lse, delta, dk_chunks, dk_anchor, dv_chunks, dv_anchor, heads,
                           c_log2, scale, plan, ku, l0, l1, l1, l1, stash);
  } else if constexpr (NS == 3) {
    __shared__ __attribute__((aligned(1024))) char l2[kSlot];
    dkv_body<D, NS, BT>(q, dout, lse, delta, dk_chunks, dk_anchor, dv_chunks, dv_anchor, heads,
                           c_log2, scale, plan, ku, l0, l1, l2, l2, stash);
  } else {
    __shared__ __attribute__((aligned(1024))) char l2[kSlot];
    __shared__ __attribute__((aligned(1024))) char l3[kSlot];
    dkv_body<D, NS, BT>(q, dout, lse, delta, dk_chunks, dk_anchor, dv_chunks, dv_anchor, heads,
                           c_log2, scale, plan, ku, l0, l1, l2, l3, stash);
  }
}

}  // namespace

hipError_t launch_attention_bwd_bf16(const void* q, const void* out, const void* dout,
                                     const float* lse, float* delta, void* dq, void* dk, void* dv,
                                     void* dak, void* dav, int heads, int head_dim,
                                     float softmax_scale, const PackedPlan& plan,
                                     const uint8_t (*frame_runs)[16], int n_frames,
                                     hipStream_t stream) {
  const int nq = plan.chunk_tokens;
  const int64_t rows = int64_t(plan.n_chunks) * nq * heads;
  if (rows == 0) return hipSuccess;
  {
    const int64_t threads = rows * (head_dim / 8);   // the last block may run past the rows
    const dim3 g(unsigned((threads + 255) / 256));
    if (head_dim == 128)
      hipLaunchKernelGGL(bwd_delta_kernel<16>, g, dim3(256), 0, stream,
                         static_cast<const __bf16*>(out), static_cast<const __bf16*>(dout), delta, rows);
    else
      hipLaunchKernelGGL(bwd_delta_kernel<8>, g, dim3(256), 0, stream,
                         static_cast<const __bf16*>(out), static_cast<const __bf16*>(dout), delta, rows);
  }
  const float c_log2 = float(double(softmax_scale) * 1.4426950408889634);
  const int n_qtiles = (nq + kBlockN - 1) / kBlockN;
  KeyUnits ku;
  std::memset(&ku, 0, sizeof(ku));
  ku.kpc = n_qtiles;
  ku.kpf = (plan.frame_tokens + kBlockN - 1) / kBlockN;
  ku.n_frames = n_frames;
  for (int f = 0; f < n_frames; ++f) std::memcpy(ku.frame_runs[f], frame_runs[f], 16);
  const int n_units = plan.n_chunks * ku.kpc + n_frames * ku.kpf;
  const dim3 g_q(unsigned(plan.n_chunks * heads * n_qtiles)), g_k(unsigned(n_units * heads));
  const __bf16* qp = static_cast<const __bf16*>(q);
  const __bf16* dp = static_cast<const __bf16*>(dout);
  __bf16 *dkp = static_cast<__bf16*>(dk), *dvp = static_cast<__bf16*>(dv);
  __bf16 *dakp = static_cast<__bf16*>(dak), *davp = static_cast<__bf16*>(dav);
  // Rings (LDS: 160 KB per workgroup): d = 128 dQ fits three 32 KB slots beside its 64 KB
  // dO stash; the d = 128 dK/dV pass (V stash plus the streamed vectors) four slots of
  // 32-row tiles, which also keeps the per-block registers within two waves per SIMD
  // beside both accumulators; d = 64 takes four 64-row slots in both passes.
  if (head_dim == 128) {
    hipLaunchKernelGGL((bwd_dq_kernel<128, 3>), g_q, dim3(kThreads), 0, stream, qp, dp, lse, delta,
                       static_cast<__bf16*>(dq), heads, c_log2, softmax_scale, plan, n_qtiles);
    hipLaunchKernelGGL((bwd_dkv_kernel<128, 4, 32>), g_k, dim3(kThreads), 0, stream, qp, dp, lse,
                       delta, dkp, dakp, dvp, davp, heads, c_log2, softmax_scale, plan, ku);
  } else {
    hipLaunchKernelGGL((bwd_dq_kernel<64, 4>), g_q, dim3(kThreads), 0, stream, qp, dp, lse, delta,
                       static_cast<__bf16*>(dq), heads, c_log2, softmax_scale, plan, n_qtiles);
    hipLaunchKernelGGL((bwd_dkv_kernel<64, 4, 64>), g_k, dim3(kThreads), 0, stream, qp, dp, lse,
                       delta, dkp, dakp, dvp, davp, heads, c_log2, softmax_scale, plan, ku);
  }
  return hipGetLastError();
}

}  // namespace ff
