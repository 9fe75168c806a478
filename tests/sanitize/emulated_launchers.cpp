// CPU emulation of libpic's kernel launches, for the sanitizer build of the host library.
//
// Each launcher below walks the grid its kernel launches and derives, with the same index
// clamping (pic_bounds.h) and the same launch planning (pic_plan.cpp), every row the kernel
// reads or writes, then touches the first and the last element of that row in host memory.
// The test driver hands the C ABI host buffers of exactly the sizes the call's documented
// contract gives them, so AddressSanitizer reports any row a kernel would address outside its
// buffer, whatever the device-side tables hold.  No arithmetic of the method happens here.
#include <cstdint>
#include <cstdlib>
#include <cstring>

#include "pic_internal.h"

namespace pic {
namespace emu {

long launches = 0;   // kernel launches the emulation has run (test driver reads it)

namespace {

template <typename T>
void rd(const T* p, int64_t row, int64_t n) {   // read row `row` of n elements
  volatile T a = p[row * n];
  volatile T b = p[row * n + n - 1];
  (void)a;
  (void)b;
}
template <typename T>
void wr(T* p, int64_t row, int64_t n) {         // write row `row` of n elements
  std::memset(&p[row * n], 0, sizeof(T));
  std::memset(&p[row * n + n - 1], 0, sizeof(T));
}
int64_t elem_size(pic_dtype dt) { return dt == PIC_F32 ? 4 : 2; }
const uint8_t* bytes(const void* p) { return static_cast<const uint8_t*>(p); }
uint8_t* bytes(void* p) { return static_cast<uint8_t*>(p); }
int32_t iabs(int32_t x) { return x < 0 ? -x : x; }

// rows of `row_bytes` bytes
void rd_row(const void* base, int64_t row, int64_t row_bytes) { rd(bytes(base), row, row_bytes); }
void wr_row(void* base, int64_t row, int64_t row_bytes) { wr(bytes(base), row, row_bytes); }

}  // namespace
}  // namespace emu

using emu::iabs;
using emu::rd_row;
using emu::wr_row;

hipError_t launch_rope_table(const double*, int half, int32_t max_abs_delta, float2* table, hipStream_t) {
  ++emu::launches;
  for (int64_t d = 0; d <= max_abs_delta; ++d) wr_row(table, d, (int64_t)half * 8);
  return hipSuccess;
}

hipError_t launch_rerotate(pic_dtype dt, int head_dim, bool, const void* k_in, void* k_out, int64_t n_rows,
                           int32_t n_heads, const int32_t* delta, const float2* table, int32_t max_abs_delta,
                           hipStream_t) {
  if (n_rows == 0) return hipSuccess;
  ++emu::launches;
  const int64_t rb = head_dim * emu::elem_size(dt), half = head_dim / 2;
  for (int64_t row = 0; row < n_rows; ++row) {
    const int32_t d = clamp_delta(delta[row / n_heads], max_abs_delta);
    rd_row(table, iabs(d), half * 8);
    rd_row(k_in, row, rb);
    wr_row(k_out, row, rb);
  }
  return hipSuccess;
}

namespace {
void compose_block(int64_t rb, int64_t half, int l, int h, int Hkv, const void* pool_k, const void* pool_v,
                   int64_t pool_tokens, const pic_block& src, const pic_block& dst, const float2* table,
                   int64_t table_stride, void* cache_k, void* cache_v, int32_t batch, int32_t cache_cap) {
  rd_row(table + l * table_stride, iabs(dst.delta), half * 8);
  for (int t = 0; t < dst.n_tokens; ++t) {
    const int64_t s = ((int64_t)l * Hkv + h) * pool_tokens + src.src_token + t;
    const int64_t d = (((int64_t)l * batch + dst.request) * Hkv + h) * cache_cap + dst.dst_slot + t;
    rd_row(pool_k, s, rb);
    rd_row(pool_v, s, rb);
    wr_row(cache_k, d, rb);
    wr_row(cache_v, d, rb);
  }
}
}  // namespace

hipError_t launch_compose(pic_dtype dt, int head_dim, bool, int n_layers, int n_kv_heads, const void* pool_k,
                          const void* pool_v, int64_t pool_tokens, const pic_block* blocks, int32_t n_blocks,
                          const float2* table, int64_t table_stride, int32_t max_abs_delta, void* cache_k,
                          void* cache_v, int32_t batch, int32_t cache_cap, hipStream_t) {
  ++emu::launches;
  const int64_t rb = head_dim * emu::elem_size(dt);
  for (int32_t i = 0; i < n_blocks; ++i) {
    const pic_block blk = blocks[i];
    if (!block_ok(blk, batch, pool_tokens, cache_cap, max_abs_delta)) continue;
    for (int l = 0; l < n_layers; ++l)
      for (int h = 0; h < n_kv_heads; ++h)
        compose_block(rb, head_dim / 2, l, h, n_kv_heads, pool_k, pool_v, pool_tokens, blk, blk, table,
                      table_stride, cache_k, cache_v, batch, cache_cap);
  }
  return hipSuccess;
}

hipError_t launch_compose_shared(pic_dtype dt, int head_dim, bool, int n_layers, int n_kv_heads,
                                 const void* pool_k, const void* pool_v, int64_t pool_tokens,
                                 const pic_block* blocks, int32_t n_blocks, const int32_t* group_start,
                                 int32_t n_groups, const float2* table, int64_t table_stride,
                                 int32_t max_abs_delta, void* cache_k, void* cache_v, int32_t batch,
                                 int32_t cache_cap, hipStream_t) {
  ++emu::launches;
  const int64_t rb = head_dim * emu::elem_size(dt), half = head_dim / 2;
  for (int32_t gi = 0; gi < n_groups; ++gi) {
    int32_t g0, g1;
    group_range(group_start[gi], group_start[gi + 1], n_blocks, g0, g1);
    if (g0 >= g1) continue;
    const pic_block src = blocks[g0];
    if (!block_source_ok(src, pool_tokens)) continue;
    for (int l = 0; l < n_layers; ++l)
      for (int h = 0; h < n_kv_heads; ++h) {
        for (int t = 0; t < src.n_tokens; ++t) {   // the run, read once
          const int64_t s = ((int64_t)l * n_kv_heads + h) * pool_tokens + src.src_token + t;
          rd_row(pool_k, s, rb);
          rd_row(pool_v, s, rb);
        }
        for (int32_t i = g0; i < g1; ++i) {
          const pic_block blk = blocks[i];
          // every block's cos/sin row is read (with the shift clamped), valid or not
          rd_row(table + l * table_stride, iabs(clamp_delta(blk.delta, max_abs_delta)), half * 8);
          if (!shared_block_ok(blk, src, batch, cache_cap, max_abs_delta)) continue;
          for (int t = 0; t < blk.n_tokens; ++t) {
            const int64_t d = (((int64_t)l * batch + blk.request) * n_kv_heads + h) * cache_cap + blk.dst_slot + t;
            wr_row(cache_k, d, rb);
            wr_row(cache_v, d, rb);
          }
        }
      }
  }
  return hipSuccess;
}

hipError_t launch_append(pic_dtype dt, int head_dim, int n_layers, int n_kv_heads, const void* k_new,
                         const void* v_new, void* cache_k, void* cache_v, int32_t batch, int32_t cache_cap,
                         const RowPos& pos, int32_t n_new, hipStream_t) {
  const int64_t n_rows = (int64_t)n_layers * batch * n_new * n_kv_heads;
  if (n_rows == 0) return hipSuccess;
  ++emu::launches;
  const int64_t rb = head_dim * emu::elem_size(dt);
  for (int64_t row = 0; row < n_rows; ++row) {
    const int h = (int)(row % n_kv_heads);
    const int64_t r1 = row / n_kv_heads;
    const int i = (int)(r1 % n_new);
    const int64_t lb = r1 / n_new;
    const int b = (int)(lb % batch);
    const int64_t slot = pos(b, i);
    if (slot < 0 || slot >= cache_cap) continue;
    rd_row(k_new, row, rb);
    rd_row(v_new, row, rb);
    wr_row(cache_k, (lb * n_kv_heads + h) * cache_cap + slot, rb);
    wr_row(cache_v, (lb * n_kv_heads + h) * cache_cap + slot, rb);
  }
  return hipSuccess;
}

namespace {
template <typename T>
hipError_t rows_walk(const RowArgs<T>& a) {
  const AttnShape& s = a.s;
  const int HD = s.head_dim, Hq = s.n_q_heads, Hkv = s.n_kv_heads, n_q = a.n_q;
  const int64_t rows = (int64_t)s.batch * n_q * Hq;
  if (rows == 0 || s.n_layers == 0) return hipSuccess;
  ++emu::launches;
  for (int l = 0; l < s.n_layers; ++l)
    for (int64_t row = 0; row < rows; ++row) {
      const int h = (int)(row % Hq), i = (int)((row / Hq) % n_q), b = (int)(row / ((int64_t)Hq * n_q));
      const int g = h / (Hq / Hkv);
      const int64_t qpos = a.pos(b, i);
      if (qpos < 0) continue;
      int64_t n_vis = qpos + 1;
      if (n_vis > s.cache_cap) n_vis = s.cache_cap;
      const int64_t qrow = (int64_t)l * s.batch * n_q * Hq + row;
      emu::rd(a.q, qrow, HD);
      if (a.q_table) rd_row(a.q_table + l * a.table_stride, std::min<int64_t>(qpos, a.max_abs_delta), (int64_t)HD / 2 * 8);
      const int64_t kv0 = (((int64_t)l * s.batch + b) * Hkv + g) * s.cache_cap;
      const int32_t ctx = a.pool_k ? clamp_len(a.ctx_len[b], a.max_ctx) : 0;
      for (int64_t j = 0; j < n_vis; ++j) {
        if (a.pool_k && j < ctx) {
          const int32_t src = clamp_pool_token(a.smap[(int64_t)b * a.map_cap + j], a.pool_tokens);
          const int32_t dl = clamp_delta(a.dmap[(int64_t)b * a.map_cap + j], a.max_abs_delta);
          rd_row(a.k_table + l * a.table_stride, iabs(dl), (int64_t)HD / 2 * 8);
          emu::rd(a.pool_k, ((int64_t)l * Hkv + g) * a.pool_tokens + src, HD);
          emu::rd(a.pool_v, ((int64_t)l * Hkv + g) * a.pool_tokens + src, HD);
        } else {
          emu::rd(a.cache_k, kv0 + j, HD);
          emu::rd(a.cache_v, kv0 + j, HD);
        }
      }
      emu::wr(a.out, qrow, HD);
    }
  return hipSuccess;
}
}  // namespace

hipError_t launch_attn_rows(const RowArgs<float>& a) { return rows_walk(a); }
hipError_t launch_attn_rows(const RowArgs<bf16_t>& a) { return rows_walk(a); }

hipError_t launch_append_rope(int head_dim, bool, int n_layers, int n_kv_heads, const bf16_t* k_new,
                              const bf16_t* v_new, bf16_t* cache_k, bf16_t* cache_v, int32_t batch,
                              int32_t cache_cap, const RowPos& pos, int32_t n_new, const float2* table,
                              int64_t table_stride, int32_t max_abs_delta, hipStream_t stream) {
  const int64_t n_rows = (int64_t)n_layers * batch * n_new * n_kv_heads;
  if (n_rows == 0) return hipSuccess;
  for (int64_t row = 0; row < n_rows; ++row) {   // the table row of each placed key
    const int64_t r1 = row / n_kv_heads;
    const int i = (int)(r1 % n_new);
    const int64_t lb = r1 / n_new;
    const int b = (int)(lb % batch), l = (int)(lb / batch);
    const int64_t slot = pos(b, i);
    if (slot < 0 || slot >= cache_cap) continue;
    rd_row(table + l * table_stride, std::min<int64_t>(slot, max_abs_delta), (int64_t)head_dim / 2 * 8);
  }
  return launch_append(PIC_BF16, head_dim, n_layers, n_kv_heads, k_new, v_new, cache_k, cache_v, batch, cache_cap,
                       pos, n_new, stream);
}

// ---- bf16 prefill: one walk serves every mode of prefill_bf16_kernel ----
namespace {

constexpr int kModeSuffix = 0, kModeTable = 1, kModePaged = 2, kModeRope = 3, kModeRuns = 4;

struct PrefillEmu {
  const bf16_t *q = nullptr, *k_suf = nullptr, *v_suf = nullptr;
  bf16_t *cache_k = nullptr, *cache_v = nullptr, *out = nullptr;
  const int32_t* ctx_len = nullptr;
  RowPos pos;                              // table mode
  int32_t max_ctx = 0;
  const bf16_t *pool_k = nullptr, *pool_v = nullptr;
  int64_t pool_tokens = 0;
  const int32_t *smap = nullptr, *dmap = nullptr, *tmap = nullptr;
  int32_t map_cap = 0, map_tiles = 0;
  const float2* table = nullptr;
  int64_t table_stride = 0;
  int32_t max_abs_delta = 0;
};

hipError_t prefill_walk(const AttnShape& s, const PrefillEmu& a, int mode, int32_t n_q, int32_t max_ctx,
                        void* workspace, size_t ws_bytes) {
  const int n_rep = s.n_q_heads / s.n_kv_heads;
  const int64_t M = (int64_t)n_q * n_rep;
  if (M == 0 || s.batch == 0 || s.n_layers == 0) return hipSuccess;
  const SplitPlan p = plan_prefill_splits(s, n_q, max_ctx);
  if (M >= (int64_t(1) << 27)) return hipErrorInvalidValue;
  if (p.n_splits > 1 && (workspace == nullptr || ws_bytes < prefill_bf16_workspace(s, n_q, max_ctx)))
    return hipErrorInvalidValue;
  if (p.n_splits > kPrefillMaxSplits) return hipErrorInvalidValue;
  ++emu::launches;
  const bool table = mode == kModeTable, paged = mode == kModePaged, runs = mode == kModeRuns;
  const bool rope = mode == kModeRope, pool = paged || runs;
  const int64_t rows_total = (int64_t)s.n_layers * s.batch * n_q * s.n_q_heads;
  bf16_t* ws_o = static_cast<bf16_t*>(workspace);
  float2* ws_ml = ws_o ? reinterpret_cast<float2*>(ws_o + (size_t)p.n_splits * rows_total * s.head_dim) : nullptr;
  const int64_t rb = (int64_t)s.head_dim * 2, half = s.head_dim / 2;   // bf16 row bytes (128 or 64 dims)
  const int n_wg = p.m_tiles * p.n_splits * s.batch * s.n_kv_heads;
  for (int l = 0; l < s.n_layers; ++l)
    for (int logical = 0; logical < n_wg; ++logical) {
      const int mt = p.m_tiles - 1 - logical % p.m_tiles;
      const int split = (logical / p.m_tiles) % p.n_splits;
      const int bg = logical / (p.m_tiles * p.n_splits);
      const int b = bg / s.n_kv_heads, g = bg % s.n_kv_heads;
      const int row0 = mt * kPrefillRowsPerWG;
      int ctx, pos_max_wg;
      int qpos[kPrefillRowsPerWG];
      bool ok[kPrefillRowsPerWG];
      int tok[kPrefillRowsPerWG], hq[kPrefillRowsPerWG];
      for (int j = 0; j < kPrefillRowsPerWG; ++j) {
        const int r = row0 + j;
        ok[j] = r < M;
        tok[j] = ok[j] ? r / n_rep : n_q - 1;
        hq[j] = g * n_rep + (ok[j] ? r % n_rep : 0);
      }
      if (!table) {
        ctx = clamp_len(a.ctx_len[b], a.max_ctx);
        pos_max_wg = ctx + (int)((std::min<int64_t>(row0 + kPrefillRowsPerWG, M) - 1) / n_rep);
        for (int j = 0; j < kPrefillRowsPerWG; ++j) qpos[j] = ctx + tok[j];
      } else {
        const int nv = clamp_len(a.pos.n_valid[b], n_q);
        int hi = -1;
        for (int j = 0; j < kPrefillRowsPerWG; ++j) {
          ok[j] = ok[j] && tok[j] < nv;
          qpos[j] = ok[j] ? clamp_len(a.pos.table[(int64_t)b * n_q + tok[j]], a.pos.max_pos) : -1;
          if (qpos[j] > hi) hi = qpos[j];
        }
        pos_max_wg = hi;
        ctx = pos_max_wg + 1;
      }
      const int n_keys = table ? pos_max_wg + 1 : ctx + n_q;
      const int t0 = split * p.tiles_per_split;
      const int n_tiles = std::min((pos_max_wg + kPrefillKeys) / kPrefillKeys - t0, p.tiles_per_split);
      const int64_t bh_kv = (((int64_t)l * s.batch + b) * s.n_kv_heads + g) * s.cache_cap;
      const int64_t suf0 = ((int64_t)l * s.batch + b) * n_q * s.n_kv_heads + g;   // in rows
      const float2* ltab = a.table ? a.table + l * a.table_stride : nullptr;
      if (!table && mt == 0 && split == 0)   // cache assembly: the suffix rows into their slots
        for (int i = 0; i < n_q; ++i) {
          rd_row(a.k_suf, suf0 + (int64_t)i * s.n_kv_heads, rb);
          rd_row(a.v_suf, suf0 + (int64_t)i * s.n_kv_heads, rb);
          if (rope) rd_row(ltab, std::min(ctx + i, a.max_abs_delta), half * 8);
          wr_row(a.cache_k, bh_kv + ctx + i, rb);
          wr_row(a.cache_v, bh_kv + ctx + i, rb);
        }
      auto orow = [&](int j) { return (((int64_t)l * s.batch + b) * n_q + tok[j]) * s.n_q_heads + hq[j]; };
      if (n_tiles <= 0) {
        if (p.n_splits > 1)
          for (int j = 0; j < kPrefillRowsPerWG; ++j)
            if (ok[j]) wr_row(ws_ml, split * rows_total + orow(j), 8);
        continue;
      }
      for (int j = 0; j < kPrefillRowsPerWG; ++j) {
        if (ok[j]) rd_row(a.q, orow(j), rb);
        if (rope) rd_row(ltab, std::min(qpos[j], a.max_abs_delta), half * 8);
      }
      const int32_t* smap = paged ? a.smap + (int64_t)b * a.map_cap : nullptr;
      const int32_t* dmap = paged ? a.dmap + (int64_t)b * a.map_cap : nullptr;
      for (int t = t0; t < t0 + n_tiles; ++t) {
        // a whole pool run (paged and runs modes, with a tile map): one piece from the pool
        int32_t run = -1;
        if (pool && a.tmap != nullptr && t < a.map_tiles && (t + 1) * kPrefillKeys <= ctx) {
          // the kernel reads the tile map 64 tiles at a time: entries t .. t + 63 below map_tiles
          for (int jj = t; jj < std::min(t + 64, a.map_tiles); ++jj) rd_row(a.tmap, (int64_t)b * a.map_tiles + jj, 8);
          const int32_t src = a.tmap[((int64_t)b * a.map_tiles + t) * 2];
          const int32_t d = a.tmap[((int64_t)b * a.map_tiles + t) * 2 + 1];
          if (tile_run_ok(src, d, t * kPrefillKeys, ctx, a.pool_tokens, a.max_abs_delta)) {
            run = src;
            rd_row(ltab, iabs(d), half * 8);   // the operand turn's cos/sin row
          }
        }
        const int64_t ph = ((int64_t)l * s.n_kv_heads + g) * a.pool_tokens;
        for (int r = 0; r < kPrefillKeys; ++r) {
          if (run >= 0) {
            rd_row(a.pool_k, ph + run + r, rb);
            rd_row(a.pool_v, ph + run + r, rb);
            continue;
          }
          if (!paged && (t + 1) * kPrefillKeys <= ctx) {
            rd_row(a.cache_k, bh_kv + (int64_t)t * kPrefillKeys + r, rb);
            rd_row(a.cache_v, bh_kv + (int64_t)t * kPrefillKeys + r, rb);
            continue;
          }
          const int kk = std::min(t * kPrefillKeys + r, n_keys - 1);
          if (paged && ctx > 0) {   // the slot map row is read (clamped) for every row of the tile
            const int slot = std::min(t * kPrefillKeys + r, ctx - 1);
            const int32_t st = smap[slot];
            const int32_t dl = dmap[slot];
            if (kk < ctx) {
              rd_row(a.pool_k, ph + clamp_pool_token(st, a.pool_tokens), rb);
              rd_row(a.pool_v, ph + clamp_pool_token(st, a.pool_tokens), rb);
              rd_row(ltab, iabs(clamp_delta(dl, a.max_abs_delta)), half * 8);
              continue;
            }
          } else if (kk < ctx) {
            rd_row(a.cache_k, bh_kv + kk, rb);
            rd_row(a.cache_v, bh_kv + kk, rb);
            continue;
          }
          if (kk >= ctx) {   // a suffix row, straight from k_suf / v_suf
            rd_row(a.k_suf, suf0 + (int64_t)(kk - ctx) * s.n_kv_heads, rb);
            rd_row(a.v_suf, suf0 + (int64_t)(kk - ctx) * s.n_kv_heads, rb);
            if (rope) rd_row(ltab, std::min(kk, a.max_abs_delta), half * 8);
          }
        }
      }
      for (int j = 0; j < kPrefillRowsPerWG; ++j) {
        if (!ok[j]) continue;
        if (p.n_splits == 1) {
          wr_row(a.out, orow(j), rb);
        } else {
          wr_row(ws_o, split * rows_total + orow(j), rb);
          wr_row(ws_ml, split * rows_total + orow(j), 8);
        }
      }
    }
  if (p.n_splits == 1) return hipSuccess;
  ++emu::launches;   // the split combine
  for (int64_t row = 0; row < rows_total; ++row) {
    if (table) {
      const int64_t ti = row / s.n_q_heads;
      const int i = (int)(ti % n_q);
      const int b = (int)((ti / n_q) % s.batch);
      if (i >= a.pos.n_valid[b]) continue;
    }
    for (int sp = 0; sp < p.n_splits; ++sp) {
      rd_row(ws_ml, sp * rows_total + row, 8);
      rd_row(ws_o, sp * rows_total + row, rb);
    }
    wr_row(a.out, row, rb);
  }
  return hipSuccess;
}

}  // namespace

hipError_t launch_prefill_bf16(const AttnShape& s, const bf16_t* q, const bf16_t* k_suf, const bf16_t* v_suf,
                               bf16_t* cache_k, bf16_t* cache_v, const int32_t* ctx_len, int32_t max_ctx,
                               int32_t n_suffix, bf16_t* out, void* workspace, size_t ws_bytes, hipStream_t) {
  PrefillEmu a;
  a.q = q; a.k_suf = k_suf; a.v_suf = v_suf; a.cache_k = cache_k; a.cache_v = cache_v;
  a.ctx_len = ctx_len; a.out = out; a.max_ctx = max_ctx;
  return prefill_walk(s, a, kModeSuffix, n_suffix, max_ctx, workspace, ws_bytes);
}

hipError_t launch_prefill_bf16_rope(const AttnShape& s, bool, const bf16_t* q, const bf16_t* k_suf,
                                    const bf16_t* v_suf, bf16_t* cache_k, bf16_t* cache_v, const int32_t* ctx_len,
                                    int32_t max_ctx, int32_t n_suffix, const float2* table, int64_t table_stride,
                                    int32_t max_abs_delta, bf16_t* out, void* workspace, size_t ws_bytes,
                                    hipStream_t) {
  PrefillEmu a;
  a.q = q; a.k_suf = k_suf; a.v_suf = v_suf; a.cache_k = cache_k; a.cache_v = cache_v;
  a.ctx_len = ctx_len; a.out = out; a.max_ctx = max_ctx;
  a.table = table; a.table_stride = table_stride; a.max_abs_delta = max_abs_delta;
  return prefill_walk(s, a, kModeRope, n_suffix, max_ctx, workspace, ws_bytes);
}

hipError_t launch_prefill_bf16_table(const AttnShape& s, const bf16_t* q, const bf16_t* cache_k,
                                     const bf16_t* cache_v, const RowPos& pos, int32_t n_q, int32_t max_len,
                                     bf16_t* out, void* workspace, size_t ws_bytes, hipStream_t) {
  PrefillEmu a;
  a.q = q; a.cache_k = const_cast<bf16_t*>(cache_k); a.cache_v = const_cast<bf16_t*>(cache_v);
  a.pos = pos; a.out = out;
  const int32_t max_ctx = max_len > n_q ? max_len - n_q : 0;
  return prefill_walk(s, a, kModeTable, n_q, max_ctx, workspace, ws_bytes);
}

hipError_t launch_compose_tiles(bool, int head_dim, int n_layers, int n_kv_heads, const bf16_t* pool_k, const bf16_t* pool_v,
                                int64_t pool_tokens, const int32_t* smap, const int32_t* dmap, int32_t map_cap,
                                const int32_t* tmap, int32_t map_tiles, const int32_t* ctx_len, int32_t max_ctx,
                                const float2* table, int64_t table_stride, int32_t max_abs_delta, bf16_t* cache_k,
                                bf16_t* cache_v, int32_t batch, int32_t cache_cap, hipStream_t) {
  ++emu::launches;
  const int64_t rb = (int64_t)head_dim * 2;   // bf16 row bytes
  for (int l = 0; l < n_layers; ++l)
    for (int h = 0; h < n_kv_heads; ++h)
      for (int64_t x = 0; x < (int64_t)batch * map_tiles; ++x) {
        const int b = (int)(x / map_tiles), tile = (int)(x - (int64_t)b * map_tiles);
        const int ctx = clamp_len(ctx_len[b], max_ctx);
        const int s0 = tile * PIC_BLOCK_TOKENS;
        if (s0 >= ctx) continue;
        const int32_t src = tmap[((int64_t)b * map_tiles + tile) * 2];
        const int32_t dl = tmap[((int64_t)b * map_tiles + tile) * 2 + 1];
        if (tile_run_ok(src, dl, s0, ctx, pool_tokens, max_abs_delta)) continue;
        for (int slot = s0; slot < std::min(s0 + PIC_BLOCK_TOKENS, ctx); ++slot) {
          const int32_t st = clamp_pool_token(smap[(int64_t)b * map_cap + slot], pool_tokens);
          const int32_t d = clamp_delta(dmap[(int64_t)b * map_cap + slot], max_abs_delta);
          rd_row(table + l * table_stride, iabs(d), (int64_t)head_dim / 2 * 8);
          rd_row(pool_k, ((int64_t)l * n_kv_heads + h) * pool_tokens + st, rb);
          rd_row(pool_v, ((int64_t)l * n_kv_heads + h) * pool_tokens + st, rb);
          wr_row(cache_k, (((int64_t)l * batch + b) * n_kv_heads + h) * cache_cap + slot, rb);
          wr_row(cache_v, (((int64_t)l * batch + b) * n_kv_heads + h) * cache_cap + slot, rb);
        }
      }
  return hipSuccess;
}

hipError_t launch_slot_map(const pic_block* blocks, int32_t n_blocks, int32_t batch, int32_t map_cap,
                           int32_t* smap, int32_t* dmap, int32_t* tmap, hipStream_t) {
  const int64_t n_map = (int64_t)batch * map_cap;
  if (n_map == 0) return hipSuccess;
  ++emu::launches;
  for (int64_t i = 0; i < n_map; ++i) smap[i] = dmap[i] = 0;
  for (int32_t i = 0; i < n_blocks; ++i) {
    const pic_block blk = blocks[i];
    if (!map_block_ok(blk, batch, map_cap)) continue;
    for (int t = 0; t < blk.n_tokens; ++t) {
      smap[(int64_t)blk.request * map_cap + blk.dst_slot + t] = blk.src_token + t;
      dmap[(int64_t)blk.request * map_cap + blk.dst_slot + t] = blk.delta;
    }
  }
  if (tmap == nullptr) return hipSuccess;
  const int32_t mt = slot_map_tiles(map_cap);
  for (int64_t i = 0; i < (int64_t)batch * mt; ++i) {
    const int64_t b = i / mt;
    const int32_t k0 = (int32_t)(i - b * mt) * PIC_BLOCK_TOKENS;
    if (k0 + PIC_BLOCK_TOKENS <= map_cap) {
      emu::rd(smap + b * map_cap + k0, 0, PIC_BLOCK_TOKENS);
      emu::rd(dmap + b * map_cap + k0, 0, PIC_BLOCK_TOKENS);
    }
    tmap[2 * i] = -1;
    tmap[2 * i + 1] = 0;
  }
  return hipSuccess;
}

hipError_t launch_prefill_bf16_paged(const AttnShape& s, bool interleaved, const bf16_t* q, const bf16_t* k_suf,
                                     const bf16_t* v_suf, bf16_t* cache_k, bf16_t* cache_v, const int32_t* ctx_len,
                                     int32_t max_ctx, int32_t n_suffix, const bf16_t* pool_k, const bf16_t* pool_v,
                                     int64_t pool_tokens, const int32_t* slot_src, const int32_t* slot_delta,
                                     int32_t map_cap, const int32_t* tile_map, const float2* table,
                                     int64_t table_stride, int32_t max_abs_delta, bf16_t* out, void* workspace,
                                     size_t ws_bytes, hipStream_t stream) {
  PrefillEmu a;
  a.q = q; a.k_suf = k_suf; a.v_suf = v_suf; a.cache_k = cache_k; a.cache_v = cache_v;
  a.ctx_len = ctx_len; a.out = out; a.max_ctx = max_ctx;
  a.pool_k = pool_k; a.pool_v = pool_v; a.pool_tokens = pool_tokens;
  a.smap = slot_src; a.dmap = slot_delta; a.tmap = tile_map; a.map_cap = map_cap;
  a.map_tiles = slot_map_tiles(map_cap);
  a.table = table; a.table_stride = table_stride; a.max_abs_delta = max_abs_delta;
  if (tile_map == nullptr) return prefill_walk(s, a, kModePaged, n_suffix, max_ctx, workspace, ws_bytes);
  if (slot_src != nullptr) {   // no slot map: the tiles were composed beforehand
    const hipError_t e = launch_compose_tiles(interleaved, s.head_dim, s.n_layers, s.n_kv_heads, pool_k, pool_v, pool_tokens,
                                              slot_src, slot_delta, map_cap, tile_map, a.map_tiles, ctx_len,
                                              max_ctx, table, table_stride, max_abs_delta, cache_k, cache_v,
                                              s.batch, s.cache_cap, stream);
    if (e != hipSuccess) return e;
  }
  return prefill_walk(s, a, kModeRuns, n_suffix, max_ctx, workspace, ws_bytes);
}

hipError_t launch_decode_bf16(const AttnShape& s, const bf16_t* q, const bf16_t* k_new, const bf16_t* v_new,
                              bf16_t* cache_k, bf16_t* cache_v, const int32_t* base_len, int32_t max_base,
                              int32_t step, int32_t n_splits, bf16_t* out, void* workspace, size_t,
                              const float2* rope_table, int64_t table_stride, int32_t max_abs_delta, bool,
                              hipStream_t) {
  if (s.batch == 0 || s.n_layers == 0) return hipSuccess;
  ++emu::launches;
  constexpr int kTile = 32;
  const int64_t rb = (int64_t)s.head_dim * 2;   // bf16 row bytes (head_dim 128 or 64)
  const int32_t max_len = max_base + step + 1;
  const int64_t rows_all = (int64_t)s.n_layers * s.batch * s.n_q_heads * n_splits;
  float* ws_o = static_cast<float*>(workspace);
  float* ws_ml = ws_o ? ws_o + rows_all * s.head_dim : nullptr;
  int32_t chunk = (max_len + n_splits - 1) / n_splits;
  chunk = (chunk + kDecodeWaves * kTile - 1) / (kDecodeWaves * kTile) * (kDecodeWaves * kTile);
  const int n_rep = s.n_q_heads / s.n_kv_heads;
  const int groups = decode_head_groups(s);
  for (int l = 0; l < s.n_layers; ++l)
    for (int x = 0; x < groups * n_splits * s.batch * s.n_kv_heads; ++x) {
      const int hgrp = x % groups, split = (x / groups) % n_splits, bg = x / (groups * n_splits);
      const int rep0 = 16 * hgrp, n_here = std::min(16, n_rep - rep0);
      const int b = bg / s.n_kv_heads, g = bg % s.n_kv_heads;
      const int p = clamp_len(base_len[b], max_base) + step;
      const int n_vis = std::min(p + 1, s.cache_cap);
      const int wc0 = std::min(split * chunk, n_vis), wc1 = std::min(wc0 + chunk, n_vis);
      const int64_t bh_kv = ((int64_t)l * s.batch + b) * s.n_kv_heads + g;
      if (hgrp == 0 && p < s.cache_cap && p >= wc0 && p < wc1) {
        rd_row(k_new, bh_kv, rb);
        rd_row(v_new, bh_kv, rb);
        wr_row(cache_k, bh_kv * s.cache_cap + p, rb);
        wr_row(cache_v, bh_kv * s.cache_cap + p, rb);
      }
      if (rope_table) rd_row(rope_table + l * table_stride, std::min(p, max_abs_delta), (int64_t)s.head_dim / 2 * 8);
      for (int n = 0; n < n_here; ++n) rd_row(q, ((int64_t)l * s.batch + b) * s.n_q_heads + g * n_rep + rep0 + n, rb);
      const int sub = chunk / kDecodeWaves;
      for (int w = 0; w < kDecodeWaves; ++w) {
        const int c0 = std::min(wc0 + w * sub, wc1), c1 = std::min(c0 + sub, wc1);
        for (int k0 = c0; k0 < c1; k0 += kTile)
          for (int r = 0; r < kTile; ++r) {
            const int row = std::min(k0 + r, c1 - 1);
            if (row == p) {
              rd_row(k_new, bh_kv, rb);
              rd_row(v_new, bh_kv, rb);
            } else {
              rd_row(cache_k, bh_kv * s.cache_cap + row, rb);
              rd_row(cache_v, bh_kv * s.cache_cap + row, rb);
            }
          }
      }
      for (int n = 0; n < n_here; ++n) {
        const int64_t row = ((int64_t)l * s.batch + b) * s.n_q_heads + g * n_rep + rep0 + n;
        if (n_splits == 1) {
          wr_row(out, row, rb);
        } else {
          const int64_t slot = row * n_splits + split;
          emu::wr(ws_o, slot, s.head_dim);
          emu::wr(ws_ml, slot, 2);
        }
      }
    }
  if (n_splits == 1) return hipSuccess;
  ++emu::launches;   // the split combine
  for (int64_t row = 0; row < (int64_t)s.n_layers * s.batch * s.n_q_heads; ++row) {
    for (int sp = 0; sp < n_splits; ++sp) {
      emu::rd(ws_ml, row * n_splits + sp, 2);
      emu::rd(ws_o, row * n_splits + sp, s.head_dim);
    }
    wr_row(out, row, rb);
  }
  return hipSuccess;
}

// The allocation-free decode's per-GPU array: host memory of the same size here.
size_t decode_scratch_bytes() { return PIC_DECODE_SCRATCH_BYTES; }
hipError_t decode_scratch_ptr(void** out) {
  static void* buf = std::malloc(PIC_DECODE_SCRATCH_BYTES);
  *out = buf;
  return buf ? hipSuccess : hipErrorOutOfMemory;
}

}  // namespace pic

// The one HIP runtime function the host library calls.
extern "C" const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "emulated launch error"; }
