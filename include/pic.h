/*
 * pic.h - C ABI of the position-independent KV-cache hit path on MI355X (gfx950).
 *
 * The path serves a request from document KV caches compiled offline, each on its own,
 * from position 0 (SemPIC, Sec. 2 and Sec. 5 "Cache-hit serving"):
 *   1. plan:    give every cached token its logical position in the request's canonical
 *               order (prefix, D_1, ..., D_m, then the query) - the link operator of Sec. 2,
 *               realised as the token-level slot -> position map of App. C.1;
 *   2. compose: gather each document's per-layer K/V into the request's cache, turning
 *               every key from its compile position a to its logical position b,
 *               k_b = R(b) R(a)^-1 k_a (Sec. 2, Eq. 3); values are copied unchanged;
 *   3. prefill: append the suffix tokens' K/V after the composed context and run causal
 *               attention of the suffix queries over it, with the frontier mask of App. C.1;
 *   4. decode:  one-token attention steps over the completed cache (App. C.1, last sentence).
 *
 * Conventions shared by every call
 *   - Pointers are DEVICE pointers unless marked [host].  The library never allocates or
 *     frees memory and never synchronises: the caller owns every buffer, and every call
 *     that takes a stream only enqueues work on it (stream is a hipStream_t; NULL is the
 *     null stream).  Results are visible once that stream has reached the call.
 *   - Element type of q/k/v/caches/outputs is model->dtype (PIC_F32: float, PIC_BF16:
 *     bfloat16 bit patterns).  Arithmetic is fp32; stores round to nearest even.
 *   - model->n_layers is the number of layers the buffers passed to the call hold (a
 *     per-layer call passes 1 and pointers offset to that layer).
 *   - Layouts (row-major, D = head_dim, L = model->n_layers):
 *       pool   [L][Hkv][pool_tokens][D]    documents' compiled K or V, concatenated
 *       cache  [L][batch][Hkv][cache_cap][D]  slot index = logical position
 *       suffix q / out       [L][batch][n_suffix][Hq][D]
 *       suffix k / v         [L][batch][n_suffix][Hkv][D]
 *       decode q / out       [L][batch][Hq][D];  decode k_new / v_new [L][batch][Hkv][D]
 *   - Device pointers must be 16-byte aligned.  Query head h reads kv head h / (Hq/Hkv).
 *   - Every argument check runs on the host before anything is enqueued.  A failing call
 *     returns a negative pic_status, enqueues nothing, and leaves a description for
 *     pic_last_error() (thread-local).  A launch failure returns PIC_ERR_HIP.  Faults during
 *     asynchronous execution surface at the caller's next synchronisation.
 *   - Device-side tables (gather blocks, context lengths) are read as given; kernels clamp
 *     every index they derive from them to the buffer sizes passed on the host, so a bad
 *     table gives wrong values, never an out-of-bounds access.
 *   - Attention on bf16 caches runs on the matrix-core kernels (prefill 3, 3a-3c and decode 4,
 *     head_dim 128 or 64).  Attention on float32 caches runs on a row-wise kernel (one
 *     workgroup per query row, float32 arithmetic) that needs no workspace and never splits.
 */
#ifndef PIC_H
#define PIC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PIC_OK = 0,
  PIC_ERR_INVALID_ARG = -1,  /* null pointer, negative size, inconsistent shape */
  PIC_ERR_UNSUPPORTED = -2,  /* valid but not built: head_dim, dtype, head ratio */
  PIC_ERR_WORKSPACE = -3,    /* workspace missing or smaller than the query call says */
  PIC_ERR_CAPACITY = -4,     /* output array or cache too small for the request */
  PIC_ERR_MISALIGNED = -5,   /* a device pointer is not 16-byte aligned */
  PIC_ERR_RANGE = -6,        /* a position shift or index beyond the table or pool */
  PIC_ERR_HIP = -7           /* the HIP runtime refused a launch */
} pic_status;

typedef enum { PIC_F32 = 0, PIC_BF16 = 1 } pic_dtype;

/* Which two elements of a head form rotary pair i. */
typedef enum {
  PIC_ROPE_HALF = 0,        /* elements i and i + D/2 (rotate-half; Llama, Qwen) */
  PIC_ROPE_INTERLEAVED = 1  /* elements 2i and 2i + 1 */
} pic_rope_pairing;

/* Attention shape and rotary transform of the decoder whose caches are served.  head_dim
   must be 64 or 128; n_q_heads must be a multiple of n_kv_heads.  At position p, rotary
   pair i of a head turns by p * theta_i, with theta_i = rope_theta^(-2i/D) (the tables
   pic_rope_table_init builds) or the frequencies given to pic_rope_table_init_freq (e.g.
   Llama-3.1 frequency scaling).
     rope_pairing  PIC_ROPE_HALF (0, the default) or PIC_ROPE_INTERLEAVED
     rope_tables   0 or 1: one transform for every layer; n_layers: layer l has its own
                   frequencies (a layer-specific R_l, Sec. 2) and the delta-angle table
                   holds one block per layer */
typedef struct {
  int32_t n_layers;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  pic_dtype dtype;
  double rope_theta;
  int32_t rope_pairing;
  int32_t rope_tables;
} pic_model;

/* Most tokens one gather block carries. */
#define PIC_BLOCK_TOKENS 64

/* One gather block of the composition map: n_tokens (1..PIC_BLOCK_TOKENS) consecutive pool
   tokens starting at src_token go to consecutive cache slots of `request` starting at
   dst_slot, their keys turned by `delta` = logical position - compile position (one value
   per document, since both run contiguously inside it; Sec. 2, Eq. 3). */
typedef struct {
  int32_t request;
  int32_t src_token;
  int32_t dst_slot;
  int32_t n_tokens;
  int32_t delta;
} pic_block;

/* ---- 1. plan (host only; Sec. 2 canonical order and link operator; App. C.1 token map) ----
   Lays each request's pool entries (documents, and a stored prefix if any) back to back from
   logical position 0 in the order given, and splits them into gather blocks.
     batch                      number of requests (>= 1)
     n_entries [host, batch]    entries each request composes (>= 0)
     entries   [host, sum n]    pool entry ids, request by request, in logical order; an entry
                                may appear more than once (a shared block-boundary header placed
                                before every document, Sec. 5), each placement getting its own
                                slots and shift
     n_pool_entries             size of the three per-entry arrays below
     entry_offset [host]        first pool token of each entry
     entry_len    [host]        tokens in each entry (>= 1)
     entry_compile_pos [host]   position the entry's first token was compiled at
     pool_tokens                tokens in the pool; every entry must lie inside it
     blocks [host out]          room for block_cap blocks
     n_blocks [host out]        blocks written; on PIC_ERR_CAPACITY, blocks needed
     ctx_len [host out, batch]  composed context length of each request
   Fails with PIC_ERR_RANGE for an entry id or token range outside the pool or a context
   longer than INT32_MAX, and PIC_ERR_CAPACITY when block_cap is too small. */
pic_status pic_plan_layout(int32_t batch, const int32_t* n_entries, const int32_t* entries,
                           int32_t n_pool_entries, const int32_t* entry_offset,
                           const int32_t* entry_len, const int32_t* entry_compile_pos,
                           int64_t pool_tokens, pic_block* blocks, int32_t block_cap,
                           int32_t* n_blocks, int32_t* ctx_len);

/* ---- 1b. plan with inline spans (Sec. 2 canonical order P, D_1, S_1, ..., D_m, S_m, Q;
   App. C.1 token map) ----
   Like pic_plan_layout, but a request's items mix pool entries (id >= 0) with inline spans,
   written -n for n >= 1 inline tokens: tokens computed at request time (an inline prefix P,
   the spans S_i, the query Q) whose K/V the caller supplies already rotated at their
   positions and whose queries pic_frontier_prefill_attn computes.  Items are laid back to
   back from position 0.
     n_items [host, batch], items [host, sum n_items]   per request, in logical order
     total_len [host out, batch]        positions the request occupies (cached + inline)
     inline_pos [host out, batch x inline_cap]  each request's inline positions, increasing;
                                        entries past n_inline[b] are set to -1
     n_inline [host out, batch]         inline tokens of each request
   The other arguments and failures are those of pic_plan_layout; in addition
   PIC_ERR_CAPACITY when a request has more than inline_cap inline tokens. */
pic_status pic_plan_frontier(int32_t batch, const int32_t* n_items, const int32_t* items,
                             int32_t n_pool_entries, const int32_t* entry_offset,
                             const int32_t* entry_len, const int32_t* entry_compile_pos,
                             int64_t pool_tokens, pic_block* blocks, int32_t block_cap,
                             int32_t* n_blocks, int32_t* total_len, int32_t* inline_pos,
                             int32_t inline_cap, int32_t* n_inline);

/* ---- 2a. delta-angle table (Sec. 2, Eq. 3: R(b) R(a)^-1 = R(b - a)) ----
   Table of (cos, sin) of delta * theta_i for delta = 0..max_abs_delta and i = 0..D/2-1,
   float32 pairs laid out [n_tables][max_abs_delta + 1][D/2][2] (n_tables = rope_tables if
   it exceeds 1, else 1); angles and cos/sin are evaluated in float64 and rounded once.
   Negative shifts use the same row with sin negated.
   pic_rope_table_bytes returns the size (0 for an unsupported model or a negative or too
   large max_abs_delta, at most 1 << 20).  pic_rope_table_init fills every block from
   rope_theta; pic_rope_table_init_freq from inv_freq [host, n_tables x D/2], finite and
   >= 0 (block l from row l).  Both enqueue on `stream`. */
size_t pic_rope_table_bytes(const pic_model* model, int32_t max_abs_delta);
pic_status pic_rope_table_init(const pic_model* model, int32_t max_abs_delta, void* table,
                               size_t table_bytes, void* stream);
pic_status pic_rope_table_init_freq(const pic_model* model, const double* inv_freq,
                                    int32_t max_abs_delta, void* table, size_t table_bytes,
                                    void* stream);

/* Host helper: the frequency-scaled rotary frequencies of the Llama-3.1 family for
   pic_rope_table_init_freq.  Starting from theta_i = theta^(-2i/D): a frequency whose
   wavelength 2 pi / theta_i is below original_max_position / high_freq_factor is kept, one
   above original_max_position / low_freq_factor is divided by factor, and in between the
   two are blended linearly in original_max_position / wavelength.  Writes D/2 values to
   inv_freq [host]; fails with PIC_ERR_INVALID_ARG for a head_dim other than 64 or 128 or
   non-positive / inconsistent factors (high_freq_factor must exceed low_freq_factor). */
pic_status pic_rope_llama3_freq(int32_t head_dim, double theta, double factor,
                                double low_freq_factor, double high_freq_factor,
                                double original_max_position, double* inv_freq);

/* ---- 2b. standalone key re-rotation (Sec. 2, Eq. 3) ----
   k_out[t][h] = R(delta[t]) k_in[t][h] for t < n_tokens, h < n_heads; rows of head_dim.
   k_in/k_out [n_tokens][n_heads][D] (may be the same buffer), delta [n_tokens] device int32
   with |delta| <= max_abs_delta (a larger entry is clamped to the table), table from
   pic_rope_table_init(_freq) for this model and max_abs_delta.  model->n_layers is ignored
   (fold layers into n_tokens); the first table block is used, so with per-layer tables
   pass a pointer to layer l's block (l * (max_abs_delta + 1) * D/2 float pairs in).
   n_tokens * n_heads above 2^48 rows fails with PIC_ERR_RANGE. */
pic_status pic_rerotate_keys(const pic_model* model, const void* k_in, void* k_out,
                             int64_t n_tokens, int32_t n_heads, const int32_t* delta,
                             const void* table, int32_t max_abs_delta, void* stream);

/* ---- 2c. composition: fused re-rotate + gather (Sec. 2 link operator and Eq. 3; App. C.1) ----
   For every layer, gather block and kv head: cache_k rows = R(delta) * pool_k rows and
   cache_v rows = pool_v rows (bit-exact copy).  blocks [n_blocks] is a device copy of
   pic_plan_layout's output; a block whose request, source range, destination range or delta
   falls outside batch, pool_tokens, cache_cap or max_abs_delta is skipped.  Slots no block
   covers are left untouched. */
pic_status pic_compose(const pic_model* model, const void* pool_k, const void* pool_v,
                       int64_t pool_tokens, const pic_block* blocks, int32_t n_blocks,
                       const void* table, int32_t max_abs_delta, void* cache_k, void* cache_v,
                       int32_t batch, int32_t cache_cap, void* stream);

/* ---- 2d. composition with shared sources (Sec. 2 link operator; App. C.1) ----
   A document placed in several requests of a batch is one pool entry, and pic_plan_layout cuts
   every placement of it into the same source runs.  pic_plan_shared (host only) orders a block
   list so that blocks reading the same run (equal src_token and n_tokens) are neighbours, and
   pic_compose_shared reads each such run once per kv head and layer and writes it to all of
   its blocks: pool reads fall from one per composed row to one per distinct run.  The cache it
   writes is bit-identical to pic_compose's for the same blocks.
     blocks [host, n_blocks]            gather blocks (pic_plan_layout / pic_plan_frontier)
     sorted [host out, n_blocks]        the same blocks, grouped by source run (stable)
     group_start [host out, n_blocks+1] group g = sorted[group_start[g] .. group_start[g+1]);
                                        group_start[n_groups] = n_blocks; a run placed more
                                        than 8 times spans several groups of at most 8 blocks
     n_groups [host out]                number of groups
   PIC_ERR_INVALID_ARG for NULL arrays or a negative count. */
pic_status pic_plan_shared(const pic_block* blocks, int32_t n_blocks, pic_block* sorted,
                           int32_t* group_start, int32_t* n_groups);
/* As pic_compose, with blocks [device, n_blocks] = pic_plan_shared's sorted list and
   group_start [device, n_groups + 1] its group starts.  A block whose source differs from its
   group's first block is skipped, as is a block out of range (see pic_compose); group starts
   are clamped to [0, n_blocks].  PIC_ERR_INVALID_ARG also when n_groups > n_blocks. */
pic_status pic_compose_shared(const pic_model* model, const void* pool_k, const void* pool_v,
                              int64_t pool_tokens, const pic_block* blocks, int32_t n_blocks,
                              const int32_t* group_start, int32_t n_groups, const void* table,
                              int32_t max_abs_delta, void* cache_k, void* cache_v, int32_t batch,
                              int32_t cache_cap, void* stream);

/* ---- 3. suffix prefill (App. C.1: inline KVs interleaved, frontier causal mask) ----
   Appends k_suf/v_suf of request b at cache slots [ctx_len[b], ctx_len[b] + n_suffix), then
   for suffix token i (logical position ctx_len[b] + i) and query head h computes
     out = sum_{j <= ctx_len[b] + i} softmax_j(scale * q . k_j) v_j
   over kv head h / (Hq/Hkv).  Suffix q/k must already carry their own rotation.
     ctx_len [device, batch]  composed lengths; entries are clamped to [0, max_ctx]
     max_ctx [host]           bound on ctx_len; max_ctx + n_suffix <= cache_cap
     scale                    softmax scale; 0 means 1/sqrt(head_dim)
     workspace                pic_prefill_workspace_bytes(...) bytes (may be 0 bytes)
   The prefill kernels (this call and 3a-3c) address one cache stream [cache_cap][D], one
   request's suffix rows [n_suffix][Hkv][D] and one pool head [pool_tokens][D] with 32-bit byte
   offsets: each of cache_cap, n_suffix * Hkv and pool_tokens must be below 2^24
   (PIC_ERR_UNSUPPORTED otherwise). */
size_t pic_prefill_workspace_bytes(const pic_model* model, int32_t batch, int32_t n_suffix,
                                   int32_t max_ctx);
pic_status pic_suffix_prefill_attn(const pic_model* model, const void* q, const void* k_suf,
                                   const void* v_suf, void* cache_k, void* cache_v,
                                   int32_t batch, int32_t cache_cap, const int32_t* ctx_len,
                                   int32_t max_ctx, int32_t n_suffix, float scale, void* out,
                                   void* workspace, size_t ws_bytes, void* stream);

/* ---- 3a. suffix prefill with fused RoPE (Sec. 5: the Reader turns request-time tokens to
   their positions; Eq. 3's R(p) from the delta-angle table) ----
   As pic_suffix_prefill_attn, but q and k_suf are given unrotated: the kernel turns query and
   key rows of suffix token i of request b by R(ctx_len[b] + i) (the model's pairing and, with
   per-layer tables, layer l's frequencies) as it loads them, in the float32 arithmetic and bf16
   rounding of pic_rerotate_keys, and stores the turned keys into the cache.  The result is
   bit-identical to turning q and k_suf with pic_rerotate_keys first and then calling
   pic_suffix_prefill_attn.  bf16 only.
     table, max_abs_delta   a pic_rope_table_init table with max_abs_delta >= max_ctx + n_suffix - 1
   (other arguments and the workspace as for pic_suffix_prefill_attn) */
pic_status pic_suffix_prefill_attn_rope(const pic_model* model, const void* q, const void* k_suf,
                                        const void* v_suf, void* cache_k, void* cache_v,
                                        int32_t batch, int32_t cache_cap, const int32_t* ctx_len,
                                        int32_t max_ctx, int32_t n_suffix, const void* table,
                                        int32_t max_abs_delta, float scale, void* out,
                                        void* workspace, size_t ws_bytes, void* stream);

/* ---- 3c. zero-copy (paged) suffix prefill (App. C.1 token map; Sec. 2, Eq. 3) ----
   pic_build_slot_map expands gather blocks into the token-level map from cache slots to the
   pool: slot_src[b][p] / slot_delta[b][p] = pool token and position shift of slot p of
   request b ([batch][map_cap] device int32; slots no block covers get 0 / 0; blocks outside
   batch or map_cap are skipped).  With tile_map (device int32, may be NULL) it also writes,
   for every 64-slot tile T = slots [64 T, 64 T + 64) of request b,
   tile_map[(b * ceil(map_cap / 64) + T) * 2 + {0, 1}] = (src, shift) when those slots are pool
   tokens src .. src + 63 under one shift, else (-1, 0).  One map serves every layer.
   pic_paged_prefill_attn computes what pic_compose followed by pic_suffix_prefill_attn
   computes, without writing the composed cache: attention reads the documents' K/V straight
   from the pool through the slot map.
   * tile_map NULL: every key is turned by its shift on load, with the float32 arithmetic and
     bf16 rounding of pic_compose, so outputs are bit-identical to compose + prefill.
   * tile_map from pic_build_slot_map (same blocks, batch and map_cap): a context tile that is
     one pool run under one shift is loaded in one piece, unturned, and the queries are turned
     by -shift for its scores instead (<R(-d) q, k> = <q, R(d) k>: RoPE's relative property
     applied to Eq. 3), in float32 with one bf16 rounding of the turned query.  Every other
     context tile (document boundaries off the 64-slot grid, short documents, a partial last
     tile) is first composed into the cache from the slot map (pic_compose's arithmetic, a
     launch of its own on the same stream) and read from there.  Outputs then match compose +
     prefill to within bf16 rounding, not bit for bit: the turned query's rounding moves a
     score by about 2^-9 |q (*) k| scale, which stays inside the attention tolerance for
     unit-scale q and k but reaches ~3 % of the output at scores near 90 nats (use tile_map
     NULL where such scores occur).  Entries outside the pool, the table or the context are
     treated as (-1, 0).
   The suffix K/V are stored (slots [ctx_len[b], ctx_len[b] + n_suffix)), and with a tile map
   the non-run context tiles; a later pic_compose (or pic_compose_shared) fills the document
   slots for decoding.  bf16 only.
   pic_compose_tiles composes, for every layer of `model` in one launch, the context tiles a
   tile map does not mark as whole runs: the step each pic_paged_prefill_attn call with a tile
   map otherwise takes for its own layer (same cache contents).  After it, the per-layer calls
   may pass slot_src = slot_delta = NULL with the tile map: they then skip that step, reading
   whole runs from the pool and every other tile from the cache (bf16 only; results identical
   to passing the slot map).
     pool_k, pool_v, pool_tokens, table, max_abs_delta   as for pic_compose
     slot_src, slot_delta, map_cap   the map; map_cap >= max_ctx (entries are clamped to the
                                     pool and to max_abs_delta)
     q, k_suf, v_suf, cache_k, cache_v, batch, cache_cap, ctx_len, max_ctx, n_suffix, scale,
     out, workspace   as for pic_suffix_prefill_attn (same workspace size)
     pic_compose_tiles: the same pool, map, table, ctx_len, max_ctx (<= cache_cap) and caches,
     all layers of the model */
pic_status pic_build_slot_map(const pic_block* blocks, int32_t n_blocks, int32_t batch,
                              int32_t map_cap, int32_t* slot_src, int32_t* slot_delta,
                              int32_t* tile_map, void* stream);
pic_status pic_compose_tiles(const pic_model* model, const void* pool_k, const void* pool_v,
                             int64_t pool_tokens, const int32_t* slot_src, const int32_t* slot_delta,
                             int32_t map_cap, const int32_t* tile_map, const void* table,
                             int32_t max_abs_delta, const int32_t* ctx_len, int32_t max_ctx,
                             void* cache_k, void* cache_v, int32_t batch, int32_t cache_cap,
                             void* stream);
pic_status pic_paged_prefill_attn(const pic_model* model, const void* pool_k, const void* pool_v,
                                  int64_t pool_tokens, const int32_t* slot_src,
                                  const int32_t* slot_delta, int32_t map_cap,
                                  const int32_t* tile_map, const void* table,
                                  int32_t max_abs_delta, const void* q, const void* k_suf,
                                  const void* v_suf, void* cache_k, void* cache_v, int32_t batch,
                                  int32_t cache_cap, const int32_t* ctx_len, int32_t max_ctx,
                                  int32_t n_suffix, float scale, void* out, void* workspace,
                                  size_t ws_bytes, void* stream);

/* ---- 3b. frontier prefill (App. C.1: inline KVs interleaved with the prepared states at
   their logical slots; a query never sees a logically later position) ----
   Stores k_inl/v_inl of inline token i of request b at cache slot pos[b][i], then for that
   token and query head h computes
     out = sum_{j <= pos[b][i]} softmax_j(scale * q . k_j) v_j
   over kv head h / (Hq/Hkv).  Every slot up to a request's largest position must hold its
   K/V once the call's own tokens are stored (pic_compose for the documents).
     q / out        [L][batch][n_inline][Hq][D];  k_inl / v_inl [L][batch][n_inline][Hkv][D]
     pos            [device, batch x n_inline] positions (pic_plan_frontier's inline_pos);
                    entries are clamped to [0, max_len - 1]
     n_valid        [device, batch] inline tokens used per request; rows i >= n_valid[b]
                    are neither stored nor computed (their out rows are left untouched)
     max_len [host] bound on every request's length; max_len <= cache_cap
     scale          softmax scale; 0 means 1/sqrt(head_dim)
     workspace      pic_frontier_workspace_bytes(...) bytes (may be 0 bytes)
   Results assume each request's positions increase with i (as the planner gives them). */
size_t pic_frontier_workspace_bytes(const pic_model* model, int32_t batch, int32_t n_inline,
                                    int32_t max_len);
pic_status pic_frontier_prefill_attn(const pic_model* model, const void* q, const void* k_inl,
                                     const void* v_inl, void* cache_k, void* cache_v,
                                     int32_t batch, int32_t cache_cap, const int32_t* pos,
                                     const int32_t* n_valid, int32_t n_inline, int32_t max_len,
                                     float scale, void* out, void* workspace, size_t ws_bytes,
                                     void* stream);

/* ---- 4. decode (App. C.1: ordinary autoregressive decoding over the completed cache) ----
   For request b the new token sits at slot p = base_len[b] + step: k_new/v_new are written
   there, then its query attends over slots [0, p].  Split-K over the context: n_splits
   chunks per (request, kv head) (0 picks a value), merged by log-sum-exp; a kv head with
   more than 16 query heads is served in groups of 16.  The row-wise path (float32 caches)
   ignores n_splits.
     base_len [device, batch]  valid slots before the first decode step; clamped to
                               [0, max_base_len]; max_base_len + step + 1 <= cache_cap
     workspace                 pic_decode_workspace_bytes(...) bytes for the same batch,
                               max_base_len + step + 1 and n_splits; 0 bytes (NULL allowed)
                               when the split count is 1 */
size_t pic_decode_workspace_bytes(const pic_model* model, int32_t batch, int32_t max_len,
                                  int32_t n_splits);
pic_status pic_decode_attn(const pic_model* model, const void* q, const void* k_new,
                           const void* v_new, void* cache_k, void* cache_v, int32_t batch,
                           int32_t cache_cap, const int32_t* base_len, int32_t step,
                           int32_t max_base_len, float scale, int32_t n_splits, void* out,
                           void* workspace, size_t ws_bytes, void* stream);

/* ---- 4a. decode with fused RoPE ----
   As pic_decode_attn, but q and k_new are given unrotated: the kernel turns them to the new
   token's position p = base_len[b] + step (the model's pairing; per-layer tables: layer l's
   frequencies) in the float32 arithmetic and bf16 rounding of pic_rerotate_keys, and stores
   the turned key into the cache; bit-identical to turning them first and calling
   pic_decode_attn.  bf16 only.
     table, max_abs_delta   a pic_rope_table_init table with max_abs_delta >= max_base_len + step
   (other arguments and the workspace as for pic_decode_attn) */
pic_status pic_decode_attn_rope(const pic_model* model, const void* q, const void* k_new,
                                const void* v_new, void* cache_k, void* cache_v, int32_t batch,
                                int32_t cache_cap, const int32_t* base_len, int32_t step,
                                int32_t max_base_len, const void* table, int32_t max_abs_delta,
                                float scale, int32_t n_splits, void* out, void* workspace,
                                size_t ws_bytes, void* stream);

/* ---- 4b. decode without a workspace, for callers that cannot allocate ----
   For code that must not allocate device memory (HIP graph capture, tight serving loops,
   harnesses that forbid hipMalloc): pic_decode_attn with its split partials kept in a scratch
   array the library holds on each GPU (PIC_DECODE_SCRATCH_BYTES, alive until the process ends)
   instead of a caller workspace.  Allocates and frees nothing; the first call on a device looks
   the array up (hipGetSymbolAddress) with that device current.
   Same arguments, checks and results as pic_decode_attn (bit-identical outputs for the same
   n_splits).  PIC_ERR_WORKSPACE when the split partials,
   pic_decode_workspace_bytes(model, batch, max_base_len + step + 1, n_splits), exceed
   PIC_DECODE_SCRATCH_BYTES.  Every call on one GPU shares that GPU's array: calls that overlap
   on one GPU (other streams, other threads) race and must be ordered by the caller.  Nothing in
   the array needs clearing: each split launch writes every partial it combines. */
#define PIC_DECODE_SCRATCH_BYTES ((size_t)8 << 20)
pic_status pic_decode_attn_noalloc(const pic_model* model, const void* q, const void* k_new,
                                   const void* v_new, void* cache_k, void* cache_v, int32_t batch,
                                   int32_t cache_cap, const int32_t* base_len, int32_t step,
                                   int32_t max_base_len, float scale, int32_t n_splits, void* out,
                                   void* stream);

/* ---- diagnostics ---- */
const char* pic_status_string(pic_status status);
/* Thread-local description of the last failure on this thread ("" if none). */
const char* pic_last_error(void);
/* Split count pic_decode_attn picks for n_splits = 0 (host only). */
int32_t pic_decode_auto_splits(const pic_model* model, int32_t batch, int32_t max_len);

#ifdef __cplusplus
}
#endif

#endif /* PIC_H */
