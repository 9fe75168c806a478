// Internal declarations of libpic: device helpers and the kernel launchers the C ABI calls.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pic.h"
#include "pic_bounds.h"

namespace pic {

typedef uint16_t bf16_t;  // bfloat16 bit pattern

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __builtin_bit_cast(float, b << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats -> packed bfloat16 (lo in bits 0..15), round to nearest even: one
// v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

// ---- launchers (each returns hipSuccess or the launch error) ----

hipError_t launch_rope_table(const double* inv_freq_host, int half, int32_t max_abs_delta,
                             float2* table, hipStream_t stream);

hipError_t launch_rerotate(pic_dtype dt, int head_dim, bool interleaved, const void* k_in,
                           void* k_out, int64_t n_rows, int32_t n_heads, const int32_t* delta,
                           const float2* table, int32_t max_abs_delta, hipStream_t stream);

// table_stride: float2 entries between consecutive layers' tables (0: one shared table).
hipError_t launch_compose(pic_dtype dt, int head_dim, bool interleaved, int n_layers,
                          int n_kv_heads, const void* pool_k, const void* pool_v,
                          int64_t pool_tokens, const pic_block* blocks, int32_t n_blocks,
                          const float2* table, int64_t table_stride, int32_t max_abs_delta,
                          void* cache_k, void* cache_v, int32_t batch, int32_t cache_cap,
                          hipStream_t stream);
// Composition with shared sources: blocks sorted into groups that read one pool run each
// (group g = blocks [group_start[g], group_start[g + 1])); each run is read once per group.
hipError_t launch_compose_shared(pic_dtype dt, int head_dim, bool interleaved, int n_layers,
                                 int n_kv_heads, const void* pool_k, const void* pool_v,
                                 int64_t pool_tokens, const pic_block* blocks, int32_t n_blocks,
                                 const int32_t* group_start, int32_t n_groups, const float2* table,
                                 int64_t table_stride, int32_t max_abs_delta, void* cache_k,
                                 void* cache_v, int32_t batch, int32_t cache_cap, hipStream_t stream);

// Logical position (= cache slot) of row i of request b among n per-request rows (suffix
// tokens, inline tokens, a decode token): either base[b] clamped to [0, max_base], plus
// offset + i; or, with a table, table[b * n + i] clamped to [0, max_pos] for i < n_valid[b]
// and -1 (row unused) otherwise.
struct RowPos {
  const int32_t* base = nullptr;
  int32_t max_base = 0, offset = 0;
  const int32_t* table = nullptr;
  const int32_t* n_valid = nullptr;
  int32_t n = 0, max_pos = 0;

  PIC_HD int64_t operator()(int b, int i) const {
    if (table) {
      if (i >= n_valid[b]) return -1;
      return clamp_len(table[(int64_t)b * n + i], max_pos);
    }
    return (int64_t)clamp_len(base[b], max_base) + offset + i;
  }
};

// Writes the K/V rows [L][B][n_new][Hkv][D] of per-request tokens into the cache slots `pos`
// gives them (rows with no position or a slot past cache_cap are skipped).
hipError_t launch_append(pic_dtype dt, int head_dim, int n_layers, int n_kv_heads,
                         const void* k_new, const void* v_new, void* cache_k, void* cache_v,
                         int32_t batch, int32_t cache_cap, const RowPos& pos, int32_t n_new,
                         hipStream_t stream);

struct AttnShape {
  int n_layers, n_q_heads, n_kv_heads, head_dim, batch, cache_cap;
  float scale_log2;  // softmax scale * log2(e)
};

// Tiling the host planner (pic_plan.cpp) shares with the bf16 attention kernels (each kernel
// file checks its own constants against these).
constexpr int kPrefillRowsPerWG = 256;     // query rows per prefill workgroup
constexpr int kPrefillKeys = 64;           // keys per prefill tile
constexpr int kPrefillMaxSplits = 32;      // most key-range splits the planner picks
constexpr int kDecodeWaves = 4;            // waves per decode workgroup
constexpr int kDecodeMinWaveKeys = 64;     // fewest keys a decode wave is given

// Key-range split of a prefill launch: m-tiles of query rows, splits per (m-tile, request,
// kv head) and key tiles per split.
struct SplitPlan {
  int m_tiles, n_splits, tiles_per_split;
};
SplitPlan plan_prefill_splits(const AttnShape& s, int32_t n_suffix, int32_t max_ctx);

// Row-wise attention (float32 caches; bf16 caches at head_dim 64), one query row per
// workgroup.  Rows [L][B][n_q][Hq]: query token i of request b sits at position pos(b, i) and
// sees slots [0, that position]; rows without a position are left untouched.  Options (bf16):
// q_table turns each query to its position first (fused RoPE); pool_k non-NULL reads context
// slots below clamp(ctx_len[b], max_ctx) from the pool through the slot map, keys turned by
// the slot's shift with k_table (zero-copy composition).
template <typename T>
struct RowArgs {
  AttnShape s;
  const T* q = nullptr;
  const T* cache_k = nullptr;
  const T* cache_v = nullptr;
  RowPos pos;
  int32_t n_q = 0;
  T* out = nullptr;
  const float2* q_table = nullptr;   // [L or 1][max_abs_delta + 1][D/2], block l at l * table_stride
  const float2* k_table = nullptr;
  int64_t table_stride = 0;
  int32_t max_abs_delta = 0;
  bool interleaved = false;
  const T* pool_k = nullptr;         // [L][Hkv][pool_tokens][D]
  const T* pool_v = nullptr;
  int64_t pool_tokens = 0;
  const int32_t* smap = nullptr;     // [B][map_cap]
  const int32_t* dmap = nullptr;
  int32_t map_cap = 0;
  const int32_t* ctx_len = nullptr;
  int32_t max_ctx = 0;
  hipStream_t stream = nullptr;
};
hipError_t launch_attn_rows(const RowArgs<float>& a);
hipError_t launch_attn_rows(const RowArgs<bf16_t>& a);

// launch_append for bf16 rows whose keys are turned to their slot's position on the way
// (fused RoPE of request-time keys; the re-rotation kernel's arithmetic); values copied.
hipError_t launch_append_rope(int head_dim, bool interleaved, int n_layers, int n_kv_heads,
                              const bf16_t* k_new, const bf16_t* v_new, bf16_t* cache_k,
                              bf16_t* cache_v, int32_t batch, int32_t cache_cap, const RowPos& pos,
                              int32_t n_new, const float2* table, int64_t table_stride,
                              int32_t max_abs_delta, hipStream_t stream);

size_t prefill_bf16_workspace(const AttnShape& s, int32_t n_suffix, int32_t max_ctx);
// Also writes k_suf / v_suf into cache slots [ctx_len[b], ctx_len[b] + n_suffix).
hipError_t launch_prefill_bf16(const AttnShape& s, const bf16_t* q, const bf16_t* k_suf,
                               const bf16_t* v_suf, bf16_t* cache_k, bf16_t* cache_v,
                               const int32_t* ctx_len, int32_t max_ctx,
                               int32_t n_suffix, bf16_t* out, void* workspace, size_t ws_bytes,
                               hipStream_t stream);
// General layout: n_q query tokens per request at the positions of `pos` (a table); every
// slot up to the largest position must already hold its K/V.  Workspace as for a suffix
// prefill of n_q tokens after max_len - n_q context tokens.
hipError_t launch_prefill_bf16_table(const AttnShape& s, const bf16_t* q, const bf16_t* cache_k,
                                     const bf16_t* cache_v, const RowPos& pos, int32_t n_q,
                                     int32_t max_len, bf16_t* out, void* workspace,
                                     size_t ws_bytes, hipStream_t stream);

// Suffix prefill with q / k_suf given unrotated: both are turned to positions ctx_len[b] + i
// with the delta-angle table (layer l's block at table + l * table_stride) as they are loaded;
// the cache receives the turned keys.  Positions must be <= max_abs_delta.
hipError_t launch_prefill_bf16_rope(const AttnShape& s, bool interleaved, const bf16_t* q,
                                    const bf16_t* k_suf, const bf16_t* v_suf, bf16_t* cache_k,
                                    bf16_t* cache_v, const int32_t* ctx_len, int32_t max_ctx,
                                    int32_t n_suffix, const float2* table, int64_t table_stride,
                                    int32_t max_abs_delta, bf16_t* out, void* workspace,
                                    size_t ws_bytes, hipStream_t stream);

// Token-level slot map: slot_src / slot_delta [batch][map_cap] = pool token and position shift
// of every slot the gather blocks cover (0 / 0 elsewhere).  With tile_map (may be NULL):
// [batch][slot_map_tiles(map_cap)][2] = (src, shift) for every 64-slot tile that is pool tokens
// src .. src + 63 under one shift, (-1, 0) for any other tile.
int32_t slot_map_tiles(int32_t map_cap);
// The context tiles of a paged prefill that are not whole pool runs (tile map), composed into
// the cache from the slot map (bf16, head_dim 128 or 64; compose arithmetic).
hipError_t launch_compose_tiles(bool interleaved, int head_dim, int n_layers, int n_kv_heads, const bf16_t* pool_k,
                                const bf16_t* pool_v, int64_t pool_tokens, const int32_t* smap,
                                const int32_t* dmap, int32_t map_cap, const int32_t* tmap,
                                int32_t map_tiles, const int32_t* ctx_len, int32_t max_ctx,
                                const float2* table, int64_t table_stride, int32_t max_abs_delta,
                                bf16_t* cache_k, bf16_t* cache_v, int32_t batch, int32_t cache_cap,
                                hipStream_t stream);
hipError_t launch_slot_map(const pic_block* blocks, int32_t n_blocks, int32_t batch, int32_t map_cap,
                           int32_t* slot_src, int32_t* slot_delta, int32_t* tile_map,
                           hipStream_t stream);
// Zero-copy composition: the documents' K/V are read from the pool through the slot map (keys
// turned on load by their shift); only the suffix rows are stored into the cache.  With a tile
// map, whole-run tiles are loaded in one piece and the queries are turned by -shift for them
// instead.  Workspace as for launch_prefill_bf16.
hipError_t launch_prefill_bf16_paged(const AttnShape& s, bool interleaved, const bf16_t* q,
                                     const bf16_t* k_suf, const bf16_t* v_suf, bf16_t* cache_k,
                                     bf16_t* cache_v, const int32_t* ctx_len, int32_t max_ctx,
                                     int32_t n_suffix, const bf16_t* pool_k, const bf16_t* pool_v,
                                     int64_t pool_tokens, const int32_t* slot_src,
                                     const int32_t* slot_delta, int32_t map_cap,
                                     const int32_t* tile_map, const float2* table,
                                     int64_t table_stride, int32_t max_abs_delta, bf16_t* out,
                                     void* workspace, size_t ws_bytes, hipStream_t stream);

int32_t decode_bf16_auto_splits(const AttnShape& s, int32_t max_len);
// Workgroups per (request, kv head, split) of the decode: one per group of up to 16 query heads.
inline int32_t decode_head_groups(const AttnShape& s) { return (s.n_q_heads / s.n_kv_heads + 15) / 16; }
// The decode scratch array (split-K partials of the allocation-free entry point): its size,
// and the current device's copy of it (looked up on the first call on that device).
size_t decode_scratch_bytes();
hipError_t decode_scratch_ptr(void** out);
size_t decode_bf16_workspace(const AttnShape& s, int32_t max_len, int32_t n_splits);
// Also writes k_new / v_new into slot base_len[b] + step of the cache.  With rope_table, q and
// k_new are given unrotated and turned to that position (table block of layer l at
// rope_table + l * table_stride; positions <= max_abs_delta).
hipError_t launch_decode_bf16(const AttnShape& s, const bf16_t* q, const bf16_t* k_new,
                              const bf16_t* v_new, bf16_t* cache_k, bf16_t* cache_v,
                              const int32_t* base_len, int32_t max_base, int32_t step,
                              int32_t n_splits, bf16_t* out, void* workspace, size_t ws_bytes,
                              const float2* rope_table, int64_t table_stride, int32_t max_abs_delta,
                              bool interleaved, hipStream_t stream);

}  // namespace pic
