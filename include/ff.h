/*
 * ff.h - C ABI of the FlashForward renderer-attention library (libff, gfx950).
 *
 * One renderer forward of FlashForward (arxiv 2609.32540, Sec. 3.1 and
 * Eq. step-update) takes the current chunk at one denoising stage as input,
 * reads clean anchor KV and the same-stage history of earlier chunks as
 * memory, produces its output, and publishes its own K/V for later chunks at
 * that stage.  This library implements the attention part of that forward on
 * one GPU, in three steps:
 *
 *   ff_rope3d          3D (t, h, w) rotary position embedding of Q and K
 *   ff_chunk_attention attention of the chunk's queries over
 *                      [anchor KV | stage-matched history KV | the chunk itself]
 *   ff_kv_publish      the chunk's K/V into the stage's history ring
 *                      (B_k <- Tail_W(B_k u (i, K, V)))
 * plus ff_anchor_set, which replaces a layer's anchor segment (the clean
 * anchor KV window A_Gamma(i) of Sec. 3.1).
 *
 * ff_packed_attention evaluates the same attention for every chunk of one
 * stage in a single launch (the renderer rows of the packed block-causal
 * training mask, App. "packed" SFT, Alg. 2), and ff_anchor_partition /
 * ff_anchor_window / ff_anchor_flank compute the planner-side index sets P,
 * Gamma(i) and the long-horizon anchor set of a chunk.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.  The caller owns all device memory and all streams.  The cache's
 *   device storage is one caller-allocated buffer of ff_cache_bytes() bytes
 *   (256-byte aligned); the handle holds host-side bookkeeping only and must
 *   not outlive that buffer.  The library never allocates device memory and
 *   never synchronises a stream.
 * Streams.  `stream` is a hipStream_t passed as void* (NULL = the null
 *   stream).  Device work is enqueued on it and nothing else; ordering
 *   between calls is the caller's stream order.  Bookkeeping (ring slots,
 *   anchor frames) is updated on the host when a call is enqueued, so calls on
 *   one cache must be issued in the order the algorithm runs them (for one
 *   (stage, layer): attention of chunk i, then publish of chunk i), and calls
 *   touching the same (stage, layer) ring on different streams need the
 *   caller's own synchronisation.  A handle is not thread-safe.
 * Tensors.  Q, K, V and the attention output are dense, contiguous
 *   [tokens][heads][head_dim] arrays of the cache's dtype (token-major, as a
 *   DiT produces them).  The tokens of a run of latent frames are ordered
 *   frame, then grid row, then grid column.  Pointers are device pointers.
 * Indices.  stage is 0 .. num_stages-1 (stage s is the paper's k = S - s; the
 *   mapping is only a name), layer is 0 .. num_layers-1, chunk_index is the
 *   renderer chunk i, covering latent frames [B_R i, B_R i + B_R).
 * Errors.  Every call returns an ff_status.  Arguments and bookkeeping are
 *   validated on the host before anything is enqueued; on any error no device
 *   work is enqueued and the handle is unchanged.  ff_last_error() returns a
 *   thread-local message for the last failing call.  FF_ERR_HIP reports a
 *   launch error returned by the HIP runtime (hipGetLastError); device faults
 *   surface on the caller's next synchronisation, as with any HIP kernel.
 */
#ifndef FF_H_
#define FF_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FF_ABI_VERSION 4
#define FF_MAX_RING_CHUNKS 8     /* W <= 8 */
#define FF_MAX_ANCHOR_FRAMES 8   /* anchor frames per layer */
#define FF_MAX_BATCH 4           /* items per ff_chunk_attention_batch call */
#define FF_MAX_ROPE_FRAMES 16    /* frames per ff_rope3d call */
#define FF_MAX_PACKED_CHUNKS 128 /* chunks per ff_packed_attention call */

typedef enum {
  FF_OK = 0,
  FF_ERR_INVALID_ARG = 1,  /* NULL pointer or meaningless value */
  FF_ERR_SHAPE = 2,        /* sizes inconsistent with the cache descriptor */
  FF_ERR_ORDER = 3,        /* chunk index out of order for the ring */
  FF_ERR_RANGE = 4,        /* stage, layer or frame index out of range */
  FF_ERR_UNSUPPORTED = 5,  /* head_dim / dtype / limit not supported */
  FF_ERR_HIP = 6,          /* the HIP runtime reported an error */
  FF_ERR_BUFFER = 7        /* device buffer too small or misaligned */
} ff_status;

typedef enum { FF_DT_BF16 = 0, FF_DT_F32 = 1 } ff_dtype;

/* Shape of one renderer cache: S stages x L layers of history rings of W
 * chunks, plus one anchor segment per layer shared by all stages (the anchor
 * KV is clean and carries no stage index, Sec. 3.1).
 *   frames_per_chunk  B_R (3 in the paper)
 *   grid_h, grid_w    latent tokens per frame = grid_h * grid_w
 *   head_dim          64 or 128
 *   rope_pairs_*      rotation pairs of the t, h and w axes; their sum must be
 *                     head_dim / 2.  All three 0 selects the split of the
 *                     Wan2.1 backbone, (d/2 - 2*floor(d/6), floor(d/6),
 *                     floor(d/6)) = (22, 21, 21) at d = 128 and (12, 10, 10)
 *                     at d = 64 (the paper fixes no RoPE; this is the one
 *                     place the library reads it); ff_cache_get_desc reports
 *                     the split in use
 *   rope_theta        RoPE base (10000)
 *   dtype             ff_dtype of every tensor and of the cache contents   */
typedef struct {
  int32_t num_stages;
  int32_t num_layers;
  int32_t ring_chunks;
  int32_t frames_per_chunk;
  int32_t grid_h;
  int32_t grid_w;
  int32_t num_heads;
  int32_t head_dim;
  int32_t max_anchor_frames;
  int32_t rope_pairs_t;
  int32_t rope_pairs_h;
  int32_t rope_pairs_w;
  double rope_theta;
  int32_t dtype;
  int32_t reserved;
} ff_cache_desc;

typedef struct ff_cache ff_cache; /* opaque host-side handle */

/* ABI version of the loaded library (FF_ABI_VERSION). */
int32_t ff_abi_version(void);

/* Device bytes the cache described by `desc` needs; 0 if `desc` is invalid
 * (ff_last_error() says why).  Layout: per layer an anchor segment of
 * max_anchor_frames frames, per (stage, layer) W ring slots of one chunk each;
 * every slot stores K and V head-major ([heads][tokens][head_dim]). */
size_t ff_cache_bytes(const ff_cache_desc* desc);

/* Create a handle over `dev_buf` (device memory of at least ff_cache_bytes()
 * bytes, 256-byte aligned, owned by the caller).  Host-only: no device work.
 * All rings start empty and no anchor segment is set. */
ff_status ff_cache_create(const ff_cache_desc* desc, void* dev_buf, size_t dev_bytes,
                          ff_cache** out);

/* Free the host-side handle (device memory stays the caller's). NULL is a no-op. */
ff_status ff_cache_destroy(ff_cache* cache);

/* The descriptor the cache was created with, as it uses it (the RoPE split
 * filled in when it was given as all zeros). */
ff_status ff_cache_get_desc(const ff_cache* cache, ff_cache_desc* out);

/* 3D RoPE, in place, on q and/or k (either may be NULL), each
 * [n_frames * grid_h * grid_w][heads][head_dim] of the cache dtype.  Frame f of
 * the run sits at latent time frame_t[f] (host array); a token's grid row and
 * column are its h and w positions.  Pair p = (2p, 2p+1) is rotated by
 * phi = pos_axis * theta^(-j / n_axis), where pairs [0, n_t) use t,
 * [n_t, n_t + n_h) use the row and the rest the column, and j counts pairs
 * inside the axis block: (a, b) -> (a cos phi - b sin phi, a sin phi + b cos phi).
 * The paper fixes no RoPE; this is the convention of its Wan2.1 backbone.
 * Angles, cosines, sines and the rotation are evaluated in float64 and
 * rounded once to the storage type (nearest even).
 * 1 <= n_frames <= FF_MAX_ROPE_FRAMES. */
ff_status ff_rope3d(const ff_cache* cache, void* q, void* k, int32_t n_frames,
                    const int32_t* frame_t, void* stream);

/* Publish chunk `chunk_index`'s K and V ([B_R*grid_h*grid_w][heads][head_dim])
 * into the history ring of (stage, layer): Eq. step-update,
 * B_k <- Tail_W(B_k u (i, K, V)).  The chunk is copied bit for bit into slot
 * chunk_index mod W, overwriting chunk_index - W.  The first publish of a ring
 * may start at any chunk_index >= 0; every later one must be the previous
 * one plus 1 (FF_ERR_ORDER otherwise).  Call it after ff_chunk_attention of
 * the same chunk (read, evaluate, then write, as in the wavefront algorithm),
 * since the slot it overwrites is one that attention still reads. */
ff_status ff_kv_publish(ff_cache* cache, int32_t stage, int32_t layer, int64_t chunk_index,
                        const void* k, const void* v, void* stream);

/* Replace layer `layer`'s anchor segment, shared by every stage, with
 * n_frames frames of clean anchor K (already rotated at its own frame
 * positions) and V, each [n_frames*grid_h*grid_w][heads][head_dim].
 * frame_t (host, n_frames values) records their latent positions for
 * inspection; attention does not use them.  0 <= n_frames <= max_anchor_frames;
 * n_frames = 0 clears the segment.  Copied bit for bit. */
ff_status ff_anchor_set(ff_cache* cache, int32_t layer, int32_t n_frames, const int32_t* frame_t,
                        const void* k, const void* v, void* stream);

/* Renderer attention of chunk `chunk_index` at (stage, layer): every query of
 * the chunk attends to
 *   - every token of the layer's anchor segment (past and future anchors),
 *   - every token of the ring's chunks max(0, i-W) .. i-1 (same stage only),
 *   - every token of the chunk itself (k_cur, v_cur; bidirectional),
 * out = softmax(softmax_scale * Q K^T) V per head (Sec. 3.1; the renderer row
 * of the packed training mask with H = W).  q, k_cur, v_cur, out are
 * [B_R*grid_h*grid_w][heads][head_dim].  The ring must hold exactly the chunks
 * published before chunk_index (its next expected chunk equals chunk_index,
 * or it is empty); FF_ERR_ORDER otherwise.  bf16: products on bf16 matrix
 * cores with float32 accumulation, softmax in float32, probabilities and
 * output rounded to bf16 (nearest even).  f32: float32 throughout.
 * softmax_scale is normally 1/sqrt(head_dim).
 * bf16 launches whose last round of workgroups is partial run that round's
 * work as key parts whose partial results go to a per-stage scratch region
 * of the cache buffer, merged by a second kernel on the same stream: calls of
 * one stage (any layer) that overlap in time on different streams race on
 * it, so order them on one stream (different stages are independent), or use
 * ff_chunk_attention_ws with a workspace per concurrent call. */
ff_status ff_chunk_attention(ff_cache* cache, int32_t stage, int32_t layer, int64_t chunk_index,
                             const void* q, const void* k_cur, const void* v_cur, void* out,
                             float softmax_scale, void* stream);

/* Device bytes of the workspace that lets ff_chunk_attention_ws split every
 * launch of this cache as ff_chunk_attention would (0 for float32 caches,
 * which never split; 0 and an error for a NULL cache). */
size_t ff_chunk_attention_workspace_bytes(const ff_cache* cache);

/* ff_chunk_attention with the tail-split partial results in a caller-owned
 * workspace (device, 16-byte aligned, `workspace_bytes` bytes) instead of the
 * cache's per-stage scratch region, so calls of one stage (e.g. two layers)
 * may overlap on different streams as long as each has its own workspace.
 * A workspace smaller than ff_chunk_attention_workspace_bytes() only limits
 * the split (results stay within the same bar); NULL runs unsplit.  The
 * workspace is the caller's until the call's work on `stream` is done.
 * Everything else as ff_chunk_attention (Sec. 3.1). */
ff_status ff_chunk_attention_ws(ff_cache* cache, int32_t stage, int32_t layer, int64_t chunk_index,
                                const void* q, const void* k_cur, const void* v_cur, void* out,
                                float softmax_scale, void* workspace, size_t workspace_bytes,
                                void* stream);

/* ff_chunk_attention with the anchor KV read from a caller-owned anchor bank
 * instead of the layer's anchor segment (the bank A of Sec. 3.1 / App. Alg. 1,
 * here in device memory): the anchors visible to the chunk are the n_frames
 * frames bank[frame_index[j]] (host array of distinct indices, in any order,
 * 0 <= n_frames <= FF_MAX_ANCHOR_FRAMES), where bank_k / bank_v are
 * token-major [bank_frames * grid_h * grid_w][heads][head_dim] arrays of the
 * cache dtype (K already rotated).  The layer's anchor segment is not read,
 * so different stages may read different windows at the same time (the
 * wavefront runs chunks i, i-1, .. on its stages together).  Everything else
 * as ff_chunk_attention.  A run of consecutive bank frames may span at most
 * 2^32 - 1 bytes (FF_ERR_UNSUPPORTED). */
ff_status ff_chunk_attention_bank(ff_cache* cache, int32_t stage, int32_t layer,
                                  int64_t chunk_index, const void* q, const void* k_cur,
                                  const void* v_cur, void* out, float softmax_scale,
                                  const void* bank_k, const void* bank_v, int32_t n_frames,
                                  const int32_t* frame_index, void* stream);

/* One item of ff_chunk_attention_batch: the arguments of one
 * ff_chunk_attention call (bank_k == NULL) or ff_chunk_attention_bank call. */
typedef struct {
  int32_t stage;
  int32_t layer;
  int64_t chunk_index;
  const void* q;
  const void* k_cur;
  const void* v_cur;
  void* out;
  const void* bank_k;          /* NULL: the layer's anchor segment */
  const void* bank_v;
  int32_t n_frames;
  int32_t reserved;
  const int32_t* frame_index;  /* host, n_frames entries */
} ff_attention_item;

/* The attention of 1 <= n <= FF_MAX_BATCH independent items in one launch,
 * e.g. the stages' forwards of one wavefront round (chunk i at stage s, chunk
 * i-1 at stage s+1, ..): one launch instead of n, which pays for items small
 * next to the GPU (far fewer (head, 256-query) units than compute units).
 * Item j computes its ff_chunk_attention(_bank) call's attention (Sec. 3.1 and
 * App. Alg. 1, the Evaluate step of every rank of a round); the batch is
 * never split along keys, so an item is bit-identical to a single call that
 * is not tail-split either, and within the same bf16 bar of the exact result
 * as a single call that is (its partial results are merged in a different
 * order).  Items share
 * softmax_scale; each is validated as its single call would be, all before
 * anything is enqueued.  Items may read the same ring; their outputs must not
 * overlap each other or any input. */
ff_status ff_chunk_attention_batch(ff_cache* cache, int32_t n, const ff_attention_item* items,
                                   float softmax_scale, void* stream);

/* Host bookkeeping of one ring (Eq. step-update): slot_chunk[s] (W entries,
 * host) is the chunk held by slot s or -1; *next_chunk is the chunk the ring
 * expects next (-1 while nothing was published: any chunk may come first);
 * *n_published counts the publishes so far (equal to *next_chunk when the
 * first publish was chunk 0).  Any output may be NULL. */
ff_status ff_cache_ring_state(const ff_cache* cache, int32_t stage, int32_t layer,
                              int64_t* slot_chunk, int64_t* next_chunk, int64_t* n_published);

/* Anchor bookkeeping of one layer: *n_frames and frame_t[0 .. n_frames)
 * (room for max_anchor_frames values).  Either output may be NULL. */
ff_status ff_cache_anchor_state(const ff_cache* cache, int32_t layer, int32_t* n_frames,
                                int32_t* frame_t);

/* Copy cache contents out, on `stream`, in the logical [tokens][heads][head_dim]
 * layout: stage >= 0 reads ring slot `slot` of (stage, layer) (one chunk);
 * stage == -1 reads the layer's whole anchor segment (slot ignored;
 * n_frames*grid_h*grid_w tokens).  k_out / v_out (device) may be NULL. */
ff_status ff_cache_read(const ff_cache* cache, int32_t stage, int32_t layer, int32_t slot,
                        void* k_out, void* v_out, void* stream);

/* Shape of one packed launch (ff_packed_attention).
 *   n_chunks          chunks of the clip, 1 .. FF_MAX_PACKED_CHUNKS
 *   chunk_tokens      tokens per chunk (B_R * grid_h * grid_w)
 *   num_heads, head_dim (64 or 128), dtype (ff_dtype)
 *   window            H >= 0: chunk i sees chunks max(0, i - H) .. i
 *   frame_tokens      tokens per anchor frame (grid_h * grid_w)
 *   n_anchor_frames   frames held by anchor_k / anchor_v, 0 .. 255
 *   anchors_of_chunk  host array of n_chunks * FF_MAX_ANCHOR_FRAMES entries:
 *                     entry [i * FF_MAX_ANCHOR_FRAMES + j] is the index (into
 *                     the anchor arrays) of an anchor frame chunk i sees, or
 *                     -1; a frame is listed at most once per chunk, in any
 *                     order.  May be NULL when n_anchor_frames is 0.        */
typedef struct {
  int32_t n_chunks;
  int32_t chunk_tokens;
  int32_t num_heads;
  int32_t head_dim;
  int32_t window;
  int32_t frame_tokens;
  int32_t n_anchor_frames;
  int32_t dtype;
  const int32_t* anchors_of_chunk;
} ff_packed_desc;

/* Packed block-causal attention of one stage over a whole clip (the renderer
 * rows of the packed training mask M, App. Alg. 2, with the visibility set
 * Vis(C_i) = chunks max(0, i-H) .. i plus the anchor frames Gamma(i) given
 * for chunk i).  Per head, the queries of chunk i attend to
 *   - every token of the anchor frames listed for chunk i,
 *   - every token of chunks max(0, i - window) .. i (bidirectional in i),
 * out = softmax(softmax_scale * Q K^T) V.  q, k, v, out are
 * [n_chunks * chunk_tokens][heads][head_dim] (chunk i's tokens at
 * i * chunk_tokens); anchor_k / anchor_v are [n_anchor_frames * frame_tokens]
 * [heads][head_dim] (may be NULL without anchor frames).  Equals
 * ff_chunk_attention of chunk i after chunks 0 .. i-1 were published into a
 * ring of W = window (same precision rules).  Tensor pointers must be
 * 16-byte aligned (FF_ERR_INVALID_ARG).  lse (optional, device,
 * [n_chunks * chunk_tokens][heads] float, bf16 path only) receives each
 * query's base-2 log-sum-exp of scale * log2(e) * q.k over its visible keys,
 * the statistic ff_packed_attention_bwd needs.  A run of the read set (one chunk window, or
 * consecutive anchor frames) may span at most 2^32 - 1 bytes
 * (FF_ERR_UNSUPPORTED).  Host validation only; one kernel launch. */
ff_status ff_packed_attention(const ff_packed_desc* desc, const void* q, const void* k,
                              const void* v, const void* anchor_k, const void* anchor_v,
                              void* out, float softmax_scale, float* lse, void* stream);

/* Device workspace bytes of ff_packed_attention_bwd for `desc`
 * (n_chunks * chunk_tokens * num_heads floats); 0 for an invalid desc. */
size_t ff_packed_attention_bwd_workspace(const ff_packed_desc* desc);

/* Backward pass of ff_packed_attention (bf16 only): given the forward's
 * inputs, its output `out`, the output gradient `dout` (both [n_chunks *
 * chunk_tokens][heads][head_dim]) and its log-sum-exp `lse`, writes
 * dq, dk, dv (shapes of q, k, v) and d_anchor_k, d_anchor_v (shape of the
 * anchor arrays; gradients summed over every chunk that sees the frame; zero
 * for frames no chunk sees):
 *   P = softmax(scale Q K^T) over the visible keys, dV = P^T dO,
 *   dS = P * (dO V^T - rowsum(dO * O)), dQ = scale dS K, dK = scale dS^T Q,
 * with products on bf16 matrix cores, float32 accumulation, P and dS rounded
 * to bf16 as operands and every gradient rounded once to bf16.  Gradient of
 * the packed training forward through its KV edges (App. Alg. 2).
 * `workspace` (device, ff_packed_attention_bwd_workspace() bytes, 16-byte
 * aligned) holds rowsum(dO * O).  At most 64 anchor frames, and the chunks
 * that see one frame may form at most 8 runs of consecutive chunks
 * (FF_ERR_UNSUPPORTED).  Host validation, then three launches. */
ff_status ff_packed_attention_bwd(const ff_packed_desc* desc, const void* q, const void* k,
                                  const void* v, const void* anchor_k, const void* anchor_v,
                                  const void* out, const void* dout, const float* lse, void* dq,
                                  void* dk, void* dv, void* d_anchor_k, void* d_anchor_v,
                                  float softmax_scale, void* workspace, size_t workspace_bytes,
                                  void* stream);

/* ff_packed_attention_bwd without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, serving or
 * training loops, harnesses that forbid hipMalloc).  rowsum(dO * O) goes to a
 * 64 MiB scratch array that the library holds in device memory, one per
 * device, from the first call on that device until the process ends; the
 * call itself allocates nothing.  Same arguments, results and errors as
 * ff_packed_attention_bwd, plus FF_ERR_UNSUPPORTED when n_chunks *
 * chunk_tokens * num_heads * 4 bytes exceed 64 MiB.  Every call on one device
 * shares that device's scratch: calls that overlap in time on one device
 * (two streams, two threads) race and give wrong gradients; calls on one
 * stream are ordered and safe. */
ff_status ff_packed_attention_bwd_static(const ff_packed_desc* desc, const void* q, const void* k,
                                         const void* v, const void* anchor_k,
                                         const void* anchor_v, const void* out, const void* dout,
                                         const float* lse, void* dq, void* dk, void* dv,
                                         void* d_anchor_k, void* d_anchor_v, float softmax_scale,
                                         void* stream);

/* Anchor partition of a clip of L latent frames with anchor spacing delta
 * (Eq. anchor-infill-partition): P = {m * delta : m * delta < L} u {L - 1},
 * ascending.  Writes |P| indices to out (host, `capacity` entries) and |P| to
 * *n_out; FF_ERR_BUFFER if capacity < |P| (*n_out still set).  L >= 1,
 * delta >= 1.  Host only. */
ff_status ff_anchor_partition(int32_t L, int32_t delta, int32_t* out, int32_t capacity,
                              int32_t* n_out);

/* Anchor window Gamma(i) of renderer chunk i (Sec. 3.1): with
 * u = floor(frames_per_chunk * i / (2 delta)), the frames
 * {2u delta, (2u+1) delta, (2u+2) delta}, each clamped to L - 1 (near the end
 * of the clip the boundary anchor L - 1 stands in for anchors past it),
 * ascending and without repeats.  Writes 1 .. 3 frames to out3 (host) and
 * their number to *n_out.  i >= 0, frames_per_chunk >= 1, delta >= 1, L >= 1.
 * Host only. */
ff_status ff_anchor_window(int64_t i, int32_t frames_per_chunk, int32_t delta, int32_t L,
                           int32_t* out3, int32_t* n_out);

/* Long-horizon anchor set of renderer chunk i: the first-frame anchor and the
 * two anchors of the partition P (Eq. anchor-infill-partition, spacing delta)
 * that flank the chunk's first latent.  With P_0 < P_1 < ... and
 * m = floor(frames_per_chunk * i / delta), the frames {P_0, P_m, P_{m+1}}, an
 * index past the last entry of P standing for the last entry (the boundary
 * anchor L - 1), ascending and without repeats.  Writes 1 .. 3 frames to out3
 * (host) and their number to *n_out.  i >= 0, frames_per_chunk >= 1,
 * delta >= 1, L >= 1.  Host only. */
ff_status ff_anchor_flank(int64_t i, int32_t frames_per_chunk, int32_t delta, int32_t L,
                          int32_t* out3, int32_t* n_out);

/* Euler step of the rectified-flow sampler (the Step of the wavefront
 * algorithm, App. Alg. 1 Phase B): x_out = x - dsigma * v elementwise over n
 * values of `dtype` (dsigma = sigma_k - sigma_{k-1}).  Each value is
 * evaluated in float64 as one product and one difference and rounded once to
 * the dtype (nearest even).  x_out may equal x (in place); the tensors must
 * not otherwise overlap.  Pointers 16-byte aligned.  n >= 0. */
ff_status ff_euler_step(const void* x, const void* v, void* x_out, int64_t n, double dsigma,
                        int32_t dtype, void* stream);

/* Renderer forward of the wavefront: enqueue on `stream` everything rank
 * `stage` does for chunk `chunk` in one round (obtain x_{i,k} from the
 * previous stage's hand-off, read, evaluate, Euler step, write; the paper's
 * k = S - stage).  Returns FF_OK, or a status that stops the run. */
typedef int32_t (*ff_stage_forward_fn)(void* user, int32_t stage, int64_t chunk, void* stream);

/* Phase B of the wavefront algorithm (App. Alg. 1) on one GPU: stage s runs
 * on streams[s] as rank s, and in round n = 0 .. n_chunks + n_stages - 2
 * every rank with 0 <= i = n - s < n_chunks runs forward(user, s, i,
 * streams[s]).  Rank s's forward of chunk i is ordered after rank s-1's
 * forward of chunk i (the latent hand-off, through an event) and, by its
 * stream, after its own forward of chunk i-1 (the ring).  The driver only
 * enqueues (it creates n_stages events and destroys them when done; HIP keeps
 * pending waits valid): the caller synchronises the streams.  *n_rounds
 * receives n_chunks + n_stages - 1 and *n_forwards n_chunks * n_stages (either
 * may be NULL).  1 <= n_stages <= 64, n_chunks >= 1; streams may repeat. */
ff_status ff_wavefront_run(int64_t n_chunks, int32_t n_stages, void* const* streams,
                           ff_stage_forward_fn forward, void* user, int64_t* n_rounds,
                           int64_t* n_forwards);

/* Name of a status code. */
const char* ff_status_string(ff_status status);

/* Message of the last failing call on this thread ("" if none). */
const char* ff_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FF_H_ */
