/*
 * epic_link.h -- C ABI of libepic_link, the link step of LegoLink
 * position-independent caching (EPIC, arXiv 2410.15332) on AMD MI355X (gfx950).
 *
 * The link step (Sec. 2.2 "link", Sec. 4.2): per-chunk KV caches were computed
 * independently, each with positions starting at 0 (the compile step).  A request
 * names chunks (in order) and a suffix of new (mutable) tokens.  The linked
 * sequence is the chunks concatenated, then the suffix.  Only the selected set S
 * is computed: the first k tokens of every chunk except the first, plus every
 * suffix token (LegoLink-k, Sec. 4.2).  Each S row attends causally over the
 * whole linked KV, in which S rows carry their newly computed K/V at their own
 * linked positions (Eq. 1).  k < 0 selects every token (Fully Recompute, Sec. 2.3).
 *
 * Conventions used everywhere below
 *  - bf16 values are passed as uint16_t bit patterns.
 *  - Paged KV cache of one layer: fixed blocks of `block_size` (16) token slots.
 *      K cache: [num_blocks][Hkv][block_size][head_dim]   (a key's vector is contiguous)
 *      V cache: [num_blocks][Hkv][head_dim][block_size]   (a block's keys are contiguous per dim)
 *    Slot id = block * block_size + offset.
 *  - Shared chunk blocks are read only.  Every block that receives a recomputed
 *    row is a request-private block taken from the caller's free list; a private
 *    block that also holds cached rows is first copied from the shared block
 *    (copy-on-write).  The "updated linked KV" is the linked block table of the
 *    plan plus the contents of the private blocks.
 *  - Device pointers are caller-owned device memory (e.g. torch tensors).  Device
 *    entry points enqueue work on `stream` (a hipStream_t; NULL = default stream)
 *    and return without synchronising.  Argument errors are detected on the host
 *    before anything is enqueued; nothing is launched when a call fails.
 *  - No entry point allocates device memory; scratch space is the caller's
 *    `workspace` of at least the size the matching *_workspace_bytes call returns
 *    (epic_link_attention_noalloc instead uses a fixed device array of the library).
 *  - Return value: EPIC_OK or an error code; epic_last_error() gives detail
 *    (thread-local, valid until the next call on the same thread).
 */
#ifndef EPIC_LINK_H
#define EPIC_LINK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EPIC_OK = 0,
  EPIC_ERR_INVALID_ARG = 1,     /* malformed sizes, ids out of range, NULL where data is needed */
  EPIC_ERR_UNSUPPORTED = 2,     /* a shape the library does not implement */
  EPIC_ERR_NO_PRIVATE_BLOCKS = 3,/* free list shorter than the plan needs */
  EPIC_ERR_WORKSPACE = 4,       /* workspace smaller than required */
  EPIC_ERR_HIP = 5              /* a HIP runtime call failed (launch error) */
} epic_status;

/* Static description of a status code; never freed. */
const char* epic_status_string(int status);
/* Detail of the last failure on this thread ("" if none). */
const char* epic_last_error(void);
/* Library version string, e.g. "epic_link 0.1 gfx950". */
const char* epic_version(void);

/* Attention shape.  Supported: head_dim in {64, 128}; block_size == 16;
 * num_q_heads a multiple of num_kv_heads with G = num_q_heads / num_kv_heads a
 * power of two <= 128.  Query head h reads KV head floor(h / G).
 * softmax_scale == 0 means 1 / sqrt(head_dim).
 * kv_split_blocks: key blocks per split-KV work item (0 = library default);
 * rows whose keys span several work items are merged with a log-sum-exp combine.
 * tile_rows: query rows (S row x head) per attention workgroup, 16, 128 or 256
 * (0 = library default: 16 when every request has at most 16 / G S rows, as in
 * decode; else 256 when the rows of a tile need nearly the same keys, else 128).
 * 16-row tiles need G <= 16.
 * rope_theta: the rotary base theta (inverse frequency theta^(-2i/D), pairs (i, i + D/2))
 * that cached K was rotated with; a plan with re-rotated blocks needs it > 0. */
typedef struct {
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t block_size;
  float softmax_scale;
  int32_t kv_split_blocks;
  int32_t tile_rows;
  float rope_theta;    /* rotary base of the cached K; used only by plans that re-rotate (else may be 0) */
} epic_attn_cfg;

/* One request, host memory, caller-owned.
 * chunk_blocks[chunk_block_off[j] .. chunk_block_off[j+1]) are the physical
 * blocks of chunk j in token order: token t of the chunk is in block t / bs at
 * offset t % bs; a chunk needs exactly ceil(chunk_len[j] / bs) blocks.
 * Chunk ids may repeat inside a request and across requests (shared caches).
 * Cached K is stored rotated at the chunk's own positions 0..L-1 (the compile
 * step).  By default the link reuses it as stored (the paper reuses cached KV
 * unchanged).  rerotate = 1 instead rotates the cached K rows of every chunk j > 0
 * by its linked offset off_j (RoPE composes, so R(off_j) R(t) = R(off_j + t)): all
 * blocks of those chunks become private copies, written by the link write with K
 * rotated in fp32 from float64 angles and rounded to bf16, V copied unchanged.
 * Chunk 0 (offset 0) stays shared.  Ignored for k < 0 (every token recomputed). */
typedef struct {
  int32_t num_chunks;
  const int32_t* chunk_len;        /* [num_chunks], each >= 1 */
  const int32_t* chunk_block_off;  /* [num_chunks + 1], CSR offsets, [0] == 0 */
  const int32_t* chunk_blocks;     /* physical block ids */
  int32_t suffix_len;              /* mutable tokens after the chunks, >= 0 */
  int32_t k;                       /* LegoLink-k; k < 0 = recompute every token */
  int32_t rerotate;                /* 1: cached K of chunk j > 0 is re-rotated to its linked positions */
} epic_link_request;

/* Sizes of a plan for a batch of requests. */
typedef struct {
  int32_t batch;
  int32_t n_s;              /* rows of S over the batch */
  int32_t n_linked_blocks;  /* entries of the linked block tables */
  int32_t n_private;        /* private blocks taken from the free list */
  int32_t n_tiles;          /* attention query tiles (per KV head) */
  int32_t n_work;           /* attention work items (per KV head) */
  int32_t n_partials;       /* split-KV partial results (per KV head) */
  int32_t tile_rows;        /* query rows (S row x head) per tile: 16, 128 or 256 */
  int32_t max_pos;          /* 1 + largest linked position in the batch */
  int32_t n_rerotated;      /* private blocks whose copied rows are re-rotated */
  int64_t total_ints;       /* int32 entries of the plan buffer */
} epic_plan_sizes;

/* Plan arrays (all int32).  epic_plan_layout() points them into one contiguous
 * buffer of sizes.total_ints int32 so that the plan can be uploaded with a
 * single copy; the same layout call on the device copy gives the device plan.
 *   s_pos[n_s]            linked position of each S row (ascending per request)
 *   s_req[n_s]            request of each S row
 *   s_slot[n_s]           slot id receiving the row's K/V
 *   s_off[batch + 1]      S rows of request r: [s_off[r], s_off[r+1])
 *   linked_blocks[n_lb]   linked block table (physical ids, position order)
 *   block_pos0[n_lb]      linked position of slot 0 of each linked block
 *   block_len[n_lb]       valid slots of each linked block (1..block_size)
 *   blk_off[batch + 1]    linked blocks of request r
 *   priv_block[n_private] private block ids (taken from free_blocks in order)
 *   priv_src[n_private]   shared block copied into it first, or -1
 *   priv_rows[n_private * block_size]  S row stored in each slot, or -1
 *   priv_rot[n_private]   linked offset by which the rows copied from priv_src are
 *                         re-rotated (K only), or 0
 *   tiles[n_tiles * 4]    (first S row, S rows, first partial or -1, splits)
 *   work[n_work * 8]      (tile, first linked block, end linked block, partial or -1,
 *                         leading 4-block KV tiles that need no mask, 0, 0, 0)
 */
typedef struct {
  int32_t* s_pos;
  int32_t* s_req;
  int32_t* s_slot;
  int32_t* s_off;
  int32_t* linked_blocks;
  int32_t* block_pos0;
  int32_t* block_len;
  int32_t* blk_off;
  int32_t* priv_block;
  int32_t* priv_src;
  int32_t* priv_rows;
  int32_t* tiles;
  int32_t* work;
  int32_t* priv_rot;
} epic_plan;

/* Host only, integer, synchronous.  Validates the requests and computes the
 * plan sizes for a batch.  n_free is the number of free blocks the caller can
 * offer; EPIC_ERR_NO_PRIVATE_BLOCKS if the plan needs more. */
epic_status epic_plan_sizes_get(const epic_link_request* reqs, int32_t batch,
                                const epic_attn_cfg* cfg, int32_t n_free,
                                epic_plan_sizes* out);

/* Points the arrays of `plan` into `base` (host or device memory of
 * sizes->total_ints int32).  Pure pointer arithmetic; never dereferences base. */
epic_status epic_plan_layout(const epic_plan_sizes* sizes, int32_t* base, epic_plan* plan);

/* Host only, integer, synchronous: builds the plan (selection of S per
 * LegoLink-k, linked block tables, private blocks with copy sources and slot
 * map, attention tiles and split-KV work items) into host arrays laid out by
 * epic_plan_layout.  free_blocks[0..n_free) must be distinct and must not be
 * chunk blocks; private blocks are taken in order.  Block ids must be
 * < num_blocks (the pool size, used for validation only). */
epic_status epic_plan_link(const epic_link_request* reqs, int32_t batch,
                           const epic_attn_cfg* cfg, const int32_t* free_blocks,
                           int32_t n_free, int32_t num_blocks,
                           const epic_plan_sizes* sizes, epic_plan* plan);

/* Decode over the linked cache (the step after the link: each request appends
 * new tokens after its last linked position and only those are computed).
 * prev / prev_sizes: the host arrays of the previous plan of these requests (the
 * link plan, or the previous decode plan).  new_tokens[b] >= 0 tokens are
 * appended to request b: S = those, at positions n_b .. n_b + t_b - 1 where n_b is
 * the request's linked length in prev.  They fill the request's last block if the
 * previous plan wrote it (a private block) and it has free slots -- that block is
 * its own copy source, so its earlier tokens stay -- and then new blocks taken in
 * order from free_blocks (distinct, not linked by prev).  The new plan links
 * everything prev linked plus the new blocks; it lists as private only the blocks
 * that receive a new token, so epic_link_attention with it (q_s / k_s / v_s of the
 * new tokens) writes nothing else.  Host only, integer, synchronous. */
epic_status epic_plan_decode_sizes(const epic_plan_sizes* prev_sizes, const epic_plan* prev,
                                   const int32_t* new_tokens, const epic_attn_cfg* cfg, int32_t n_free,
                                   epic_plan_sizes* out);
epic_status epic_plan_decode(const epic_plan_sizes* prev_sizes, const epic_plan* prev, const int32_t* new_tokens,
                             const epic_attn_cfg* cfg, const int32_t* free_blocks, int32_t n_free,
                             int32_t num_blocks, const epic_plan_sizes* sizes, epic_plan* plan);

/* Compile step (Sec. 2.2): every chunk is prefilled alone, positions from 0, and
 * its K/V per layer become the chunk's cache.  LegoLink-0 (Sec. 5.4) prepends
 * n_dummy dummy tokens to every chunk for this prefill and drops their K/V, so
 * the cache holds the chunk's L tokens only (token t at block t / bs, offset
 * t % bs), rotated at their compile positions n_dummy + t.
 * chunk_blocks[chunk_block_off[j] .. chunk_block_off[j+1]): the ceil(L_j / bs)
 * blocks that receive chunk j's cache (all distinct).  n_dummy >= 0. */
typedef struct {
  int32_t num_chunks;
  const int32_t* chunk_len;        /* [num_chunks], each >= 1 */
  const int32_t* chunk_block_off;  /* [num_chunks + 1], CSR offsets, [0] == 0 */
  const int32_t* chunk_blocks;     /* physical block ids receiving the caches */
  int32_t n_dummy;                 /* dummy tokens prepended to every chunk (0 = plain compile) */
} epic_compile_batch;

/* Host only, integer, synchronous.  The compile plan has one request per chunk,
 * in order: S = its n_dummy + L_j tokens at positions 0 .. n_dummy + L_j - 1, the
 * dummies first, so the caller's S rows (hidden states) of chunk j are n_dummy
 * dummy rows then the chunk's L_j token rows.  With n_dummy == 0 the linked
 * blocks are the chunk blocks and free_blocks is not used.  With n_dummy > 0
 * the attention reads the n_dummy + L_j tokens from ceil((n_dummy + L_j) / bs)
 * staging blocks per chunk taken in order from free_blocks (distinct, not chunk
 * blocks; EPIC_ERR_NO_PRIVATE_BLOCKS if too few), and the chunk blocks are
 * private blocks outside the linked table that receive rows n_dummy .. (the
 * staging blocks hold the dummy-inclusive K/V afterwards and may be reused).
 * epic_link_model (or epic_link_attention per layer) with this plan is the
 * compile step; s_slot gives the linked (staging) slot of every row. */
epic_status epic_plan_compile_sizes(const epic_compile_batch* batch, const epic_attn_cfg* cfg, int32_t n_free,
                                    epic_plan_sizes* out);
epic_status epic_plan_compile(const epic_compile_batch* batch, const epic_attn_cfg* cfg,
                              const int32_t* free_blocks, int32_t n_free, int32_t num_blocks,
                              const epic_plan_sizes* sizes, epic_plan* plan);

/* Workspace bytes epic_link_attention needs for this plan (split-KV partials). */
size_t epic_link_workspace_bytes(const epic_attn_cfg* cfg, const epic_plan_sizes* sizes);

/* One attention layer of the link step (Sec. 4.2, Eq. 1), on the device:
 *   1. build every private block: copy its source block (if any; K rotated by
 *      priv_rot when that is non-zero, see epic_link_request.rerotate), then
 *      store k_s / v_s of the S rows into their slots (bit-exact copies);
 *   2. for each S row r at linked position p and query head h: softmax over the
 *      linked keys at positions <= p of scale * <q, k>, times V; write out[r, h]
 *      (bf16) and lse[r, h] = natural log of the softmax denominator (fp32).
 * q_s [n_s][Hq][D], k_s / v_s [n_s][Hkv][D] (bf16, ascending S order, already
 * rotated); k_cache / v_cache: the layer's paged caches (layouts above);
 * out [n_s][Hq][D] bf16; lse [n_s][Hq] fp32 or NULL.  plan_dev: plan arrays in
 * device memory.  Empty S: EPIC_OK, nothing launched. */
epic_status epic_link_attention(const epic_attn_cfg* cfg, const epic_plan_sizes* sizes,
                                const epic_plan* plan_dev,
                                const uint16_t* q_s, const uint16_t* k_s, const uint16_t* v_s,
                                uint16_t* k_cache, uint16_t* v_cache,
                                uint16_t* out, float* lse,
                                void* workspace, size_t workspace_bytes, void* stream);

/* epic_link_attention for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * steps, kernels and results, with the split-KV partials kept in a fixed array of
 * EPIC_NOALLOC_SCRATCH_BYTES of device memory that the library holds, one copy per
 * GPU, from the time its code is loaded on that GPU until the process ends.  The
 * caller still passes inputs, caches and outputs (as for epic_link_attention); no
 * device memory is allocated or freed by the call.  A plan whose partials need more
 * than EPIC_NOALLOC_SCRATCH_BYTES (epic_link_workspace_bytes) is rejected with
 * EPIC_ERR_WORKSPACE before anything is enqueued (a larger kv_split_blocks gives fewer
 * partials).  Every call on one GPU shares that GPU's array: calls whose work overlaps
 * in time on one GPU (other streams, other threads) race and give wrong results;
 * calls in one stream are ordered and safe.  Nothing in the array needs to start at
 * any value: each call writes every partial it reads. */
#define EPIC_NOALLOC_SCRATCH_BYTES (96u << 20)
epic_status epic_link_attention_noalloc(const epic_attn_cfg* cfg, const epic_plan_sizes* sizes,
                                        const epic_plan* plan_dev,
                                        const uint16_t* q_s, const uint16_t* k_s, const uint16_t* v_s,
                                        uint16_t* k_cache, uint16_t* v_cache,
                                        uint16_t* out, float* lse, void* stream);

/* Profiling hook for callers that time the step's kernels.  events: NULL (off)
 * or 4 hipEvent_t created by the caller; each entry may be NULL.  Until the
 * next call on the same thread, every device entry point records, on its
 * stream, events[0] before the link write, events[1] before the attention
 * kernel, events[2] after it and events[3] after the split-KV combine (per
 * layer for the model entry points; each record overwrites the previous one).
 * Never fails. */
epic_status epic_set_profile_events(void* const* events);

/* ---------------------------------------------------------------- model level */

/* Llama-style decoder (Sec. 5.1 models): pre-norm RMSNorm, rotary embedding
 * (pairs (i, i + D/2), inverse frequency theta^(-2i/D), angles in float64),
 * GQA attention, SwiGLU MLP, final RMSNorm.  hidden % 128 == 0,
 * ffn % 128 == 0 and (Hq + 2 Hkv) D % 128 == 0 are required. */
typedef struct {
  epic_attn_cfg attn;
  int32_t hidden;
  int32_t ffn;
  int32_t n_layers;
  float rope_theta;
  float rms_eps;
} epic_model_cfg;

/* Device pointers to one layer's bf16 weights, [out][in] row-major (y = x W^T):
 *   attn_norm [hidden], wqkv [(Hq + 2 Hkv) D][hidden] (rows: q | k | v),
 *   wo [hidden][Hq D], mlp_norm [hidden], w_gate_up [2 ffn][hidden] (rows: gate | up),
 *   w_down [hidden][ffn]. */
typedef struct {
  const uint16_t* attn_norm;
  const uint16_t* wqkv;
  const uint16_t* wo;
  const uint16_t* mlp_norm;
  const uint16_t* w_gate_up;
  const uint16_t* w_down;
} epic_layer_weights;

/* Workspace bytes for epic_link_layer / epic_link_model with this plan. */
size_t epic_model_workspace_bytes(const epic_model_cfg* cfg, const epic_plan_sizes* sizes);

/* One decoder layer for the S rows (Sec. 4.2 per-layer recipe): hidden_s
 * [n_s][hidden] fp32 residual stream, updated in place; the layer's K/V caches
 * receive the rotated K and the V of every S row (private blocks, as in
 * epic_link_attention). */
epic_status epic_link_layer(const epic_model_cfg* cfg, const epic_layer_weights* w,
                            const epic_plan_sizes* sizes, const epic_plan* plan_dev,
                            float* hidden_s, uint16_t* k_cache, uint16_t* v_cache,
                            void* workspace, size_t workspace_bytes, void* stream);

/* All layers, then the final RMSNorm: out_hidden [n_s][hidden] fp32.
 * layers: host array [n_layers] of device weight pointers; k_caches / v_caches:
 * host arrays [n_layers] of device cache pointers.  hidden_s holds the layer-0
 * rows (embeddings of the S tokens) on entry and is overwritten.
 * The compile step (Sec. 2.2) is this call on a request with no chunks whose
 * suffix is the chunk's tokens: positions 0..L-1, every token computed. */
epic_status epic_link_model(const epic_model_cfg* cfg, const epic_layer_weights* layers,
                            const uint16_t* final_norm,
                            const epic_plan_sizes* sizes, const epic_plan* plan_dev,
                            float* hidden_s, uint16_t* const* k_caches, uint16_t* const* v_caches,
                            float* out_hidden, void* workspace, size_t workspace_bytes,
                            void* stream);

/* ---------------------------------------------------------------- projections */

/* The projection GEMM that epic_link_layer / epic_link_model run for the S rows
 * (Sec. 4.2: Q = E W_Q, K = E W_K, V = E W_V of the selected rows, then the output
 * projection W_O; the model's SwiGLU MLP), on its own:
 *   C[i][j] = sum_t a[i][t] w[j][t]     a: bf16 [m][k]; w: bf16 [n][k] ([out][in]);
 *                                       fp32 accumulation
 * epilogue EPIC_GEMM_STORE:    c[i][j] = C[i][j]                       c: fp32 [m][n]
 *          EPIC_GEMM_RESIDUAL: c[i][j] += C[i][j]                      c: fp32 [m][n], in place
 *          EPIC_GEMM_SWIGLU:   act[i][j] = bf16(silu(C[i][j]) C[i][j + n/2]), j < n/2
 *                              (rows [0, n/2) of w: gate; [n/2, n): up)   act: bf16 [m][n/2]
 * Shapes: m >= 0, k % 64 == 0, n % 128 == 0, and with m rounded up to a multiple
 * of 256 every operand and output below 2^31 bytes; else EPIC_ERR_UNSUPPORTED.
 * Device pointers, 16-byte aligned.  workspace: at least epic_gemm_workspace_bytes()
 * bytes of device memory, 256-byte aligned, owned by the caller; it holds the
 * partial sums of output tiles cut along k and their arrival counters (cleared by
 * this call), so calls in flight at the same time need separate workspaces.
 * A tile cut along k is summed in a fixed order (the part that holds the tile's last
 * k stage, then the others in k order), so results do not depend on timing.  The
 * environment variable EPIC_GEMM_FINISH_POLLS (read at each launch, default 4096)
 * bounds how long that last part's workgroup polls for the others before falling
 * back to the last-to-arrive protocol; 0 forces the fallback (a test hook; the sums
 * are the same either way).
 * Enqueued on `stream` (NULL: the default stream); returns after the enqueue. */
typedef enum { EPIC_GEMM_STORE = 0, EPIC_GEMM_RESIDUAL = 1, EPIC_GEMM_SWIGLU = 2 } epic_gemm_epilogue;
size_t epic_gemm_workspace_bytes(void);
epic_status epic_gemm(int32_t epilogue, const uint16_t* a, const uint16_t* w, int32_t m, int32_t n, int32_t k,
                      float* c, uint16_t* act, void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* EPIC_LINK_H */
