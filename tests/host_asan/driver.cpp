// Drives every C ABI entry point of libff through its host-side paths (with
// launch_stubs.cpp in place of the kernels), for an AddressSanitizer /
// UndefinedBehaviorSanitizer build.  Device pointers are host addresses that
// the host code only stores and compares.  Exit status 0 = every expectation
// held.  Test infrastructure only.

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "ff.h"

static int g_failures = 0;
#define EXPECT(cond)                                                             \
  do {                                                                           \
    if (!(cond)) {                                                               \
      std::fprintf(stderr, "%s:%d: expectation failed: %s (last error: %s)\n", \
                   __FILE__, __LINE__, #cond, ff_last_error());                  \
      ++g_failures;                                                              \
    }                                                                            \
  } while (0)

static ff_cache_desc desc(int stages, int layers, int W, int grid_h, int grid_w, int heads, int d,
                          int max_anchor, int dtype) {
  ff_cache_desc c = {};
  c.num_stages = stages;
  c.num_layers = layers;
  c.ring_chunks = W;
  c.frames_per_chunk = 3;
  c.grid_h = grid_h;
  c.grid_w = grid_w;
  c.num_heads = heads;
  c.head_dim = d;
  c.max_anchor_frames = max_anchor;
  c.rope_pairs_t = d / 2 - 2 * (d / 6);
  c.rope_pairs_h = d / 6;
  c.rope_pairs_w = d / 6;
  c.rope_theta = 10000.0;
  c.dtype = dtype;
  return c;
}

// 256-byte aligned stand-in for device memory (only its address is used)
struct FakeDevice {
  std::vector<unsigned char> bytes;
  explicit FakeDevice(size_t n) : bytes(n + 256) {}
  void* ptr() {
    const uintptr_t p = reinterpret_cast<uintptr_t>(bytes.data());
    return reinterpret_cast<void*>((p + 255) / 256 * 256);
  }
};

static void ring_sequences() {
  for (int dtype : {FF_DT_BF16, FF_DT_F32})
    for (int W : {1, 3, 8}) {
      ff_cache_desc d = desc(2, 2, W, 6, 11, 3, 128, 8, dtype);
      const size_t n = ff_cache_bytes(&d);
      EXPECT(n > 0);
      FakeDevice dev(n);
      ff_cache* h = nullptr;
      EXPECT(ff_cache_create(&d, dev.ptr(), n, &h) == FF_OK && h);
      ff_cache_desc used = {};
      EXPECT(ff_cache_get_desc(h, &used) == FF_OK && used.ring_chunks == W);
      FakeDevice chunk(2 * 198 * 3 * 128 * 4 + 1024);
      char* t = static_cast<char*>(chunk.ptr());
      std::vector<int32_t> ft(8);
      for (int f = 0; f < 8; ++f) ft[f] = 10 * f;
      EXPECT(ff_anchor_set(h, 1, 8, ft.data(), t, t, nullptr) == FF_OK);
      EXPECT(ff_anchor_set(h, 1, 9, ft.data(), t, t, nullptr) == FF_ERR_RANGE);
      int32_t nf = -1;
      std::vector<int32_t> got(8, -1);
      EXPECT(ff_cache_anchor_state(h, 1, &nf, got.data()) == FF_OK && nf == 8 && got[7] == 70);
      for (int64_t c = 5; c < 5 + 3 * W + 2; ++c)
        for (int s = 0; s < 2; ++s)
          for (int l = 0; l < 2; ++l) {
            EXPECT(ff_chunk_attention(h, s, l, c, t, t, t, t, 0.125f, nullptr) == FF_OK);
            // a caller workspace: the stage's full size, a smaller one, none
            const size_t ws = ff_chunk_attention_workspace_bytes(h);
            EXPECT(ff_chunk_attention_ws(h, s, l, c, t, t, t, t, 0.125f, dev.ptr(), ws, nullptr) ==
                   FF_OK);
            EXPECT(ff_chunk_attention_ws(h, s, l, c, t, t, t, t, 0.125f, dev.ptr(), ws / 3,
                                         nullptr) == FF_OK);
            EXPECT(ff_chunk_attention_ws(h, s, l, c, t, t, t, t, 0.125f, nullptr, 0, nullptr) ==
                   FF_OK);
            // the bank path: out-of-order frames, runs of consecutive frames, a duplicate
            const int32_t frames[5] = {7, 2, 3, 0, 1};
            EXPECT(ff_chunk_attention_bank(h, s, l, c, t, t, t, t, 0.125f, t, t, 5, frames,
                                           nullptr) == FF_OK);
            const int32_t dup[3] = {4, 1, 4};
            EXPECT(ff_chunk_attention_bank(h, s, l, c, t, t, t, t, 0.125f, t, t, 3, dup,
                                           nullptr) == FF_ERR_INVALID_ARG);
            if (c > 5)   // the first publish of a ring may start at any chunk
              EXPECT(ff_kv_publish(h, s, l, c + 1, t, t, nullptr) == FF_ERR_ORDER);
            // the same call as one item of a batch, beside a bank item and a duplicate
            ff_attention_item items[FF_MAX_BATCH + 1] = {};
            for (int j = 0; j <= FF_MAX_BATCH; ++j) {
              items[j].stage = s;
              items[j].layer = l;
              items[j].chunk_index = c;
              items[j].q = items[j].k_cur = items[j].v_cur = t;
              items[j].out = t;
            }
            items[1].bank_k = items[1].bank_v = t;
            items[1].n_frames = 5;
            items[1].frame_index = frames;
            EXPECT(ff_chunk_attention_batch(h, 2, items, 0.125f, nullptr) == FF_OK);
            EXPECT(ff_chunk_attention_batch(h, FF_MAX_BATCH, items, 0.125f, nullptr) == FF_OK);
            EXPECT(ff_chunk_attention_batch(h, FF_MAX_BATCH + 1, items, 0.125f, nullptr) ==
                   FF_ERR_UNSUPPORTED);
            EXPECT(ff_chunk_attention_batch(h, 0, items, 0.125f, nullptr) == FF_ERR_UNSUPPORTED);
            items[2].chunk_index = c + 1;   // out of order: the whole batch is refused
            if (c > 5)                      // (an empty ring accepts any chunk)
              EXPECT(ff_chunk_attention_batch(h, 3, items, 0.125f, nullptr) == FF_ERR_ORDER);
            EXPECT(ff_kv_publish(h, s, l, c, t, t, nullptr) == FF_OK);
            std::vector<int64_t> slots(W, -2);
            int64_t next = -1, count = -1;   // first publish was chunk 5
            EXPECT(ff_cache_ring_state(h, s, l, slots.data(), &next, &count) == FF_OK &&
                   next == c + 1 && count == c - 4);
            for (int slot = 0; slot < W; ++slot) {   // Tail_W of chunks 5 .. c
              int64_t want = -1;
              for (int64_t x = c; x >= 5 && x > c - W; --x)
                if (x % W == slot) want = x;
              EXPECT(slots[slot] == want);
            }
            EXPECT(ff_cache_read(h, s, l, int(c % W), t, t, nullptr) == FF_OK);
          }
      EXPECT(ff_chunk_attention(h, 0, 0, 3, t, t, t, t, 0.125f, nullptr) == FF_ERR_ORDER);
      EXPECT(ff_cache_read(h, -1, 1, 0, t, t, nullptr) == FF_OK);
      EXPECT(ff_cache_read(h, 0, 0, W, t, t, nullptr) == FF_ERR_RANGE);
      const int32_t fr[3] = {9, 10, 11};
      EXPECT(ff_rope3d(h, t, t, 3, fr, nullptr) == FF_OK);
      EXPECT(ff_cache_destroy(h) == FF_OK);
    }
}

static void invalid_descriptors() {
  ff_cache_desc d = desc(2, 2, 4, 6, 11, 3, 96, 3, FF_DT_BF16);
  EXPECT(ff_cache_bytes(&d) == 0);
  ff_cache* h = reinterpret_cast<ff_cache*>(1);
  FakeDevice dev(4096);
  EXPECT(ff_cache_create(&d, dev.ptr(), 4096, &h) == FF_ERR_UNSUPPORTED);
  d = desc(2, 2, 4, 6, 11, 3, 128, 3, FF_DT_BF16);
  EXPECT(ff_cache_create(&d, dev.ptr(), 16, &h) == FF_ERR_BUFFER);
  EXPECT(ff_cache_create(&d, static_cast<char*>(dev.ptr()) + 16, 1ull << 40, &h) == FF_ERR_BUFFER);
  EXPECT(ff_cache_create(nullptr, dev.ptr(), 1ull << 40, &h) == FF_ERR_INVALID_ARG);
  EXPECT(ff_cache_destroy(nullptr) == FF_OK);
}

static void packed_paths() {
  FakeDevice buf(1 << 20);
  char* t = static_cast<char*>(buf.ptr());
  for (int window : {0, 2, 9})
    for (int n_frames : {0, 5, 64}) {
      const int n_chunks = 12;
      std::vector<int32_t> table(n_chunks * FF_MAX_ANCHOR_FRAMES, -1);
      for (int c = 0; c < n_chunks && n_frames > 0; ++c)
        for (int j = 0; j < 3; ++j) table[c * FF_MAX_ANCHOR_FRAMES + j] = (c * 2 + 5 * j) % n_frames;
      ff_packed_desc pd = {n_chunks, 198, 2, 128, window, 66, n_frames, FF_DT_BF16,
                           n_frames > 0 ? table.data() : nullptr};
      // a frame listed twice in one chunk is rejected when it happens
      bool dup = false;
      for (int c = 0; c < n_chunks && n_frames > 0; ++c)
        for (int a = 0; a < 3; ++a)
          for (int b = a + 1; b < 3; ++b)
            dup |= table[c * FF_MAX_ANCHOR_FRAMES + a] == table[c * FF_MAX_ANCHOR_FRAMES + b];
      const ff_status want = dup ? FF_ERR_INVALID_ARG : FF_OK;
      float* lse = reinterpret_cast<float*>(t);
      EXPECT(ff_packed_attention(&pd, t, t, t, n_frames ? t : nullptr, n_frames ? t : nullptr, t,
                                 0.1f, lse, nullptr) == want);
      const size_t ws = ff_packed_attention_bwd_workspace(&pd);
      EXPECT(ws == size_t(n_chunks) * 198 * 2 * 4);
      const ff_status b = ff_packed_attention_bwd(&pd, t, t, t, n_frames ? t : nullptr,
                                                  n_frames ? t : nullptr, t, t, lse, t, t, t,
                                                  n_frames ? t : nullptr, n_frames ? t : nullptr,
                                                  0.1f, t, ws, nullptr);
      EXPECT(b == want || (want == FF_OK && b == FF_ERR_UNSUPPORTED));
      EXPECT(ff_packed_attention_bwd(&pd, t, t, t, n_frames ? t : nullptr, n_frames ? t : nullptr,
                                     t, t, lse, t, t, t, n_frames ? t : nullptr,
                                     n_frames ? t : nullptr, 0.1f, t, ws - 4, nullptr) != FF_OK);
    }
  // one frame seen by more than 8 runs of chunks: unsupported by the backward
  std::vector<int32_t> table(40 * FF_MAX_ANCHOR_FRAMES, -1);
  for (int c = 0; c < 40; c += 2) table[c * FF_MAX_ANCHOR_FRAMES] = 0;
  ff_packed_desc pd = {40, 64, 1, 64, 0, 64, 1, FF_DT_BF16, table.data()};
  EXPECT(ff_packed_attention(&pd, t, t, t, t, t, t, 0.1f, nullptr, nullptr) == FF_OK);
  EXPECT(ff_packed_attention_bwd(&pd, t, t, t, t, t, t, t, reinterpret_cast<float*>(t), t, t, t,
                                 t, t, 0.1f, t, 1 << 20, nullptr) == FF_ERR_UNSUPPORTED);
  EXPECT(ff_packed_attention_bwd_static(&pd, t, t, t, t, t, t, t, reinterpret_cast<float*>(t), t,
                                        t, t, t, t, 0.1f, nullptr) == FF_ERR_UNSUPPORTED);
  // beyond the 64 MiB static scratch: rejected before the device is touched
  ff_packed_desc big = {64, 10800, 40, 128, 4, 3600, 0, FF_DT_BF16, nullptr};
  EXPECT(ff_packed_attention_bwd_static(&big, t, t, t, nullptr, nullptr, t, t,
                                        reinterpret_cast<float*>(t), t, t, t, nullptr, nullptr,
                                        0.1f, nullptr) == FF_ERR_UNSUPPORTED);
}

static int32_t forward_calls = 0;
static int32_t forward_ok(void*, int32_t, int64_t, void*) {
  ++forward_calls;
  return FF_OK;
}

static void planner_euler_wavefront() {
  std::vector<int32_t> out(64);
  int32_t n = 0;
  EXPECT(ff_anchor_partition(81, 10, out.data(), 64, &n) == FF_OK && n == 9 && out[8] == 80);
  EXPECT(ff_anchor_partition(261, 10, out.data(), 2, &n) == FF_ERR_BUFFER && n == 27);
  int32_t w3[3];
  EXPECT(ff_anchor_window(2, 3, 10, 81, w3, &n) == FF_OK && n == 3 && w3[0] == 0 && w3[2] == 20);
  EXPECT(ff_anchor_flank(86, 3, 24, 261, w3, &n) == FF_OK && n == 3 && w3[1] == 240 && w3[2] == 260);
  EXPECT(ff_anchor_flank(0, 3, 24, 261, w3, &n) == FF_OK && n == 2 && w3[1] == 24);
  FakeDevice buf(1 << 16);
  char* t = static_cast<char*>(buf.ptr());
  EXPECT(ff_euler_step(t, t + 8192, t, 64, 0.25, FF_DT_BF16, nullptr) == FF_OK);
  EXPECT(ff_euler_step(t, t + 8192, t + 16, 64, 0.25, FF_DT_BF16, nullptr) == FF_ERR_INVALID_ARG);
  EXPECT(ff_euler_step(t, t + 8192, t, 64, NAN, FF_DT_BF16, nullptr) == FF_ERR_INVALID_ARG);
  void* streams[4] = {nullptr, nullptr, nullptr, nullptr};
  int64_t rounds = -1, fwd = -1;
  // without a GPU the event calls fail: the driver reports FF_ERR_HIP and frees what it made
  const ff_status st = ff_wavefront_run(5, 4, streams, forward_ok, nullptr, &rounds, &fwd);
  EXPECT(st == FF_OK || st == FF_ERR_HIP);
  if (st == FF_OK) EXPECT(rounds == 8 && fwd == 20 && forward_calls == 20);
  EXPECT(ff_wavefront_run(0, 4, streams, forward_ok, nullptr, &rounds, &fwd) == FF_ERR_INVALID_ARG);
  for (int s = 0; s <= 7; ++s) EXPECT(ff_status_string(ff_status(s)) != nullptr);
}

int main() {
  EXPECT(ff_abi_version() == FF_ABI_VERSION);
  invalid_descriptors();
  ring_sequences();
  packed_paths();
  planner_euler_wavefront();
  if (g_failures) std::fprintf(stderr, "%d expectation(s) failed\n", g_failures);
  else std::printf("host ABI checks passed\n");
  return g_failures ? 1 : 0;
}
