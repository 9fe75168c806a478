// C ABI of libpic: argument validation, the layout planner and dispatch to the HIP kernels.
// Every check runs before anything is enqueued; a failing call launches nothing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "pic.h"
#include "pic_internal.h"

#define PIC_API extern "C" __attribute__((visibility("default")))

namespace {

thread_local std::string g_last_error;

pic_status fail(pic_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

pic_status ok() {
  g_last_error.clear();
  return PIC_OK;
}

pic_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(PIC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define PIC_CHECK(expr)              \
  do {                               \
    pic_status _s = (expr);          \
    if (_s != PIC_OK) return _s;     \
  } while (0)

pic_status check_ptr(const void* p, const char* name) {
  if (p == nullptr) return fail(PIC_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned16(p)) return fail(PIC_ERR_MISALIGNED, "%s is not 16-byte aligned", name);
  return PIC_OK;
}

pic_status check_model(const pic_model* m) {
  if (m == nullptr) return fail(PIC_ERR_INVALID_ARG, "model is NULL");
  if (m->n_layers < 0) return fail(PIC_ERR_INVALID_ARG, "n_layers < 0");
  if (m->n_q_heads <= 0 || m->n_kv_heads <= 0)
    return fail(PIC_ERR_INVALID_ARG, "head counts must be positive");
  if (m->n_q_heads % m->n_kv_heads != 0)
    return fail(PIC_ERR_INVALID_ARG, "n_q_heads (%d) is not a multiple of n_kv_heads (%d)",
                m->n_q_heads, m->n_kv_heads);
  if (m->head_dim != 64 && m->head_dim != 128)
    return fail(PIC_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", m->head_dim);
  if (m->dtype != PIC_F32 && m->dtype != PIC_BF16)
    return fail(PIC_ERR_UNSUPPORTED, "dtype %d", (int)m->dtype);
  if (m->rope_pairing != PIC_ROPE_HALF && m->rope_pairing != PIC_ROPE_INTERLEAVED)
    return fail(PIC_ERR_INVALID_ARG, "rope_pairing %d", m->rope_pairing);
  if (m->rope_tables < 0 || (m->rope_tables > 1 && m->rope_tables != m->n_layers))
    return fail(PIC_ERR_INVALID_ARG, "rope_tables %d (0, 1 or n_layers = %d)", m->rope_tables,
                m->n_layers);
  return PIC_OK;
}

int32_t n_tables(const pic_model* m) { return m->rope_tables > 1 ? m->rope_tables : 1; }

constexpr int32_t kMaxAbsDelta = 1 << 20;
// Rows one re-rotation call may cover: their element offsets stay far inside int64.
constexpr int64_t kMaxRerotateRows = int64_t(1) << 48;
// The bf16 attention kernels address a cache stream (one layer, request and kv head), one
// request's suffix rows and a pool head (one layer and kv head) with 32-bit byte offsets from
// a buffer base: each must stay under 2^32 bytes (rows of 256 bytes).
constexpr int64_t kMaxRows32 = (int64_t(1) << 32) / 256 - 1;
static pic_status check_rows32(int64_t cache_cap, int64_t suffix_rows, int64_t pool_tokens) {
  if (cache_cap > kMaxRows32 || suffix_rows > kMaxRows32 || pool_tokens > kMaxRows32)
    return fail(PIC_ERR_UNSUPPORTED,
                "a cache stream, a request's suffix rows or a pool head exceeds %lld rows",
                (long long)kMaxRows32);
  return ok();
}

size_t elem_bytes(const pic_model* m) { return m->dtype == PIC_F32 ? 4 : 2; }

float scale_log2_of(const pic_model* m, float scale) {
  const double s = scale == 0.f ? 1.0 / std::sqrt((double)m->head_dim) : (double)scale;
  return (float)(s * 1.4426950408889634);  // log2(e)
}

pic::AttnShape shape_of(const pic_model* m, int32_t batch, int32_t cache_cap, float scale) {
  pic::AttnShape s;
  s.n_layers = m->n_layers;
  s.n_q_heads = m->n_q_heads;
  s.n_kv_heads = m->n_kv_heads;
  s.head_dim = m->head_dim;
  s.batch = batch;
  s.cache_cap = cache_cap;
  s.scale_log2 = scale_log2_of(m, scale);
  return s;
}

pic_status check_attn_model(const pic_model* m) { return check_model(m); }

// bf16 caches run on the matrix-core kernels (prefill in every mode and decode, head_dim 128 or
// 64); float32 caches on the row-wise kernel.
bool mfma_prefill(const pic_model* m) { return m->dtype == PIC_BF16; }
bool mfma_decode(const pic_model* m) { return m->dtype == PIC_BF16; }

// Row-wise attention of n_q query rows per request at the positions `pos` gives them.
// Options for bf16 rows: q_table (fused RoPE of the query), and a paged key source.
struct RowOpts {
  const void* q_table = nullptr;
  int64_t table_stride = 0;
  int32_t max_abs_delta = 0;
  const void* pool_k = nullptr;
  const void* pool_v = nullptr;
  int64_t pool_tokens = 0;
  const int32_t* smap = nullptr;
  const int32_t* dmap = nullptr;
  int32_t map_cap = 0;
  const int32_t* ctx_len = nullptr;
  int32_t max_ctx = 0;
  const void* k_table = nullptr;
};
template <typename T>
hipError_t launch_rows_as(const pic_model* m, const pic::AttnShape& s, const void* q, const void* ck,
                          const void* cv, const pic::RowPos& pos, int32_t n_q, void* out, const RowOpts& o,
                          hipStream_t st) {
  pic::RowArgs<T> a;
  a.s = s;
  a.q = static_cast<const T*>(q);
  a.cache_k = static_cast<const T*>(ck);
  a.cache_v = static_cast<const T*>(cv);
  a.pos = pos;
  a.n_q = n_q;
  a.out = static_cast<T*>(out);
  a.q_table = static_cast<const float2*>(o.q_table);
  a.k_table = static_cast<const float2*>(o.k_table);
  a.table_stride = o.table_stride;
  a.max_abs_delta = o.max_abs_delta;
  a.interleaved = m->rope_pairing == PIC_ROPE_INTERLEAVED;
  a.pool_k = static_cast<const T*>(o.pool_k);
  a.pool_v = static_cast<const T*>(o.pool_v);
  a.pool_tokens = o.pool_tokens;
  a.smap = o.smap;
  a.dmap = o.dmap;
  a.map_cap = o.map_cap;
  a.ctx_len = o.ctx_len;
  a.max_ctx = o.max_ctx;
  a.stream = st;
  return pic::launch_attn_rows(a);
}
pic_status launch_rows(const pic_model* m, const pic::AttnShape& s, const void* q, const void* ck, const void* cv,
                       const pic::RowPos& pos, int32_t n_q, void* out, hipStream_t st, const char* what,
                       const RowOpts& o = RowOpts()) {
  return hip_status(m->dtype == PIC_F32 ? launch_rows_as<float>(m, s, q, ck, cv, pos, n_q, out, o, st)
                                        : launch_rows_as<pic::bf16_t>(m, s, q, ck, cv, pos, n_q, out, o, st),
                    what);
}

}  // namespace

PIC_API const char* pic_status_string(pic_status s) {
  switch (s) {
    case PIC_OK: return "PIC_OK";
    case PIC_ERR_INVALID_ARG: return "PIC_ERR_INVALID_ARG";
    case PIC_ERR_UNSUPPORTED: return "PIC_ERR_UNSUPPORTED";
    case PIC_ERR_WORKSPACE: return "PIC_ERR_WORKSPACE";
    case PIC_ERR_CAPACITY: return "PIC_ERR_CAPACITY";
    case PIC_ERR_MISALIGNED: return "PIC_ERR_MISALIGNED";
    case PIC_ERR_RANGE: return "PIC_ERR_RANGE";
    case PIC_ERR_HIP: return "PIC_ERR_HIP";
  }
  return "PIC_ERR_UNKNOWN";
}

PIC_API const char* pic_last_error(void) { return g_last_error.c_str(); }

// ---------------------------------------------------------------------------------------------
// 1. plan
// ---------------------------------------------------------------------------------------------

namespace {

// Shared by both planners: items are pool entry ids (>= 0) or, when inline spans are allowed,
// -n for n inline tokens.  Items are laid back to back from position 0.
pic_status plan_items(int32_t batch, const int32_t* n_items, const int32_t* items, bool allow_inline,
                      int32_t n_pool_entries, const int32_t* entry_offset, const int32_t* entry_len,
                      const int32_t* entry_compile_pos, int64_t pool_tokens, pic_block* blocks,
                      int32_t block_cap, int32_t* n_blocks, int32_t* total_len, int32_t* inline_pos,
                      int32_t inline_cap, int32_t* n_inline) {
  if (batch <= 0) return fail(PIC_ERR_INVALID_ARG, "batch must be >= 1");
  if (!n_items || !entry_offset || !entry_len || !entry_compile_pos || !n_blocks || !total_len)
    return fail(PIC_ERR_INVALID_ARG, "a required host array is NULL");
  if (allow_inline && !n_inline) return fail(PIC_ERR_INVALID_ARG, "n_inline is NULL");
  if (n_pool_entries < 0 || block_cap < 0 || pool_tokens < 0 || inline_cap < 0)
    return fail(PIC_ERR_INVALID_ARG, "negative size");
  int64_t total_items = 0;
  for (int32_t b = 0; b < batch; ++b) {
    if (n_items[b] < 0) return fail(PIC_ERR_INVALID_ARG, "item count of request %d < 0", b);
    total_items += n_items[b];
  }
  if (total_items > 0 && !items) return fail(PIC_ERR_INVALID_ARG, "the item list is NULL");
  for (int32_t e = 0; e < n_pool_entries; ++e) {
    if (entry_len[e] <= 0) return fail(PIC_ERR_INVALID_ARG, "entry_len[%d] must be >= 1", e);
    if (entry_offset[e] < 0 || (int64_t)entry_offset[e] + entry_len[e] > pool_tokens)
      return fail(PIC_ERR_RANGE, "pool entry %d [%d, %lld) lies outside the %lld-token pool", e,
                  entry_offset[e], (long long)entry_offset[e] + entry_len[e],
                  (long long)pool_tokens);
    if (entry_compile_pos[e] < 0 || (int64_t)entry_compile_pos[e] + entry_len[e] > INT32_MAX)
      return fail(PIC_ERR_RANGE, "entry_compile_pos[%d] out of range", e);
  }
  // count blocks and inline tokens and check ranges first, so a failing call writes nothing
  int64_t need = 0;
  const int32_t* it = items;
  for (int32_t b = 0; b < batch; ++b) {
    int64_t pos = 0, inl = 0;
    for (int32_t k = 0; k < n_items[b]; ++k) {
      const int32_t e = it[k];
      if (e < 0 && allow_inline) {
        if (e == INT32_MIN) return fail(PIC_ERR_RANGE, "request %d item %d: span too long", b, k);
        pos += -(int64_t)e;
        inl += -(int64_t)e;
      } else {
        if (e < 0 || e >= n_pool_entries)
          return fail(PIC_ERR_RANGE, "request %d item %d: pool entry id %d out of [0, %d)", b, k,
                      e, n_pool_entries);
        need += (entry_len[e] + PIC_BLOCK_TOKENS - 1) / PIC_BLOCK_TOKENS;
        pos += entry_len[e];
      }
      if (pos > INT32_MAX) return fail(PIC_ERR_RANGE, "request %d exceeds INT32_MAX positions", b);
    }
    if (allow_inline && inl > inline_cap)
      return fail(PIC_ERR_CAPACITY, "request %d has %lld inline tokens, room for %d", b,
                  (long long)inl, inline_cap);
    it += n_items[b];
  }
  if (need > INT32_MAX) return fail(PIC_ERR_CAPACITY, "too many blocks");
  *n_blocks = (int32_t)need;
  if (need > block_cap)
    return fail(PIC_ERR_CAPACITY, "%lld blocks needed, room for %d", (long long)need, block_cap);
  if (need > 0 && !blocks) return fail(PIC_ERR_INVALID_ARG, "blocks is NULL");
  if (allow_inline && inline_cap > 0 && !inline_pos)
    return fail(PIC_ERR_INVALID_ARG, "inline_pos is NULL");

  int32_t nb = 0;
  it = items;
  for (int32_t b = 0; b < batch; ++b) {
    int32_t pos = 0;   // logical position = cache slot
    int32_t inl = 0;
    for (int32_t k = 0; k < n_items[b]; ++k) {
      const int32_t e = it[k];
      if (e < 0) {   // inline span (Sec. 2: P and the S_i are computed at request time)
        for (int32_t t = 0; t < -e; ++t) inline_pos[(int64_t)b * inline_cap + inl++] = pos + t;
        pos += -e;
        continue;
      }
      const int32_t len = entry_len[e];
      const int32_t delta = pos - entry_compile_pos[e];  // b_i - a_i, Eq. 3
      for (int32_t t = 0; t < len; t += PIC_BLOCK_TOKENS) {
        pic_block& blk = blocks[nb++];
        blk.request = b;
        blk.src_token = entry_offset[e] + t;
        blk.dst_slot = pos + t;
        blk.n_tokens = len - t < PIC_BLOCK_TOKENS ? len - t : PIC_BLOCK_TOKENS;
        blk.delta = delta;
      }
      pos += len;
    }
    total_len[b] = pos;
    if (allow_inline) {
      n_inline[b] = inl;
      for (int32_t i = inl; i < inline_cap; ++i) inline_pos[(int64_t)b * inline_cap + i] = -1;
    }
    it += n_items[b];
  }
  return ok();
}

}  // namespace

PIC_API pic_status pic_plan_layout(int32_t batch, const int32_t* n_entries, const int32_t* entries,
                                   int32_t n_pool_entries, const int32_t* entry_offset,
                                   const int32_t* entry_len, const int32_t* entry_compile_pos,
                                   int64_t pool_tokens, pic_block* blocks, int32_t block_cap,
                                   int32_t* n_blocks, int32_t* ctx_len) {
  return plan_items(batch, n_entries, entries, false, n_pool_entries, entry_offset, entry_len,
                    entry_compile_pos, pool_tokens, blocks, block_cap, n_blocks, ctx_len, nullptr,
                    0, nullptr);
}

PIC_API pic_status pic_plan_frontier(int32_t batch, const int32_t* n_items, const int32_t* items,
                                     int32_t n_pool_entries, const int32_t* entry_offset,
                                     const int32_t* entry_len, const int32_t* entry_compile_pos,
                                     int64_t pool_tokens, pic_block* blocks, int32_t block_cap,
                                     int32_t* n_blocks, int32_t* total_len, int32_t* inline_pos,
                                     int32_t inline_cap, int32_t* n_inline) {
  return plan_items(batch, n_items, items, true, n_pool_entries, entry_offset, entry_len,
                    entry_compile_pos, pool_tokens, blocks, block_cap, n_blocks, total_len,
                    inline_pos, inline_cap, n_inline);
}

// ---------------------------------------------------------------------------------------------
// 2. re-rotation and composition
// ---------------------------------------------------------------------------------------------

PIC_API size_t pic_rope_table_bytes(const pic_model* model, int32_t max_abs_delta) {
  if (check_model(model) != PIC_OK) return 0;
  if (max_abs_delta < 0 || max_abs_delta > kMaxAbsDelta) return 0;
  return (size_t)n_tables(model) * (max_abs_delta + 1) * (model->head_dim / 2) * sizeof(float) * 2;
}

namespace {

// Fills every table block from inv_freq (row l for block l, or row 0 for all when `shared`).
pic_status fill_tables(const pic_model* model, const double* inv_freq, bool shared,
                       int32_t max_abs_delta, void* table, size_t table_bytes, void* stream) {
  if (max_abs_delta < 0 || max_abs_delta > kMaxAbsDelta)
    return fail(PIC_ERR_RANGE, "max_abs_delta %d outside [0, %d]", max_abs_delta, kMaxAbsDelta);
  PIC_CHECK(check_ptr(table, "table"));
  const size_t need = pic_rope_table_bytes(model, max_abs_delta);
  if (table_bytes < need)
    return fail(PIC_ERR_CAPACITY, "table needs %zu bytes, got %zu", need, table_bytes);
  const int half = model->head_dim / 2;
  const int64_t block = (int64_t)(max_abs_delta + 1) * half;
  for (int32_t t = 0; t < n_tables(model); ++t)
    PIC_CHECK(hip_status(pic::launch_rope_table(inv_freq + (shared ? 0 : (int64_t)t * half), half,
                                                max_abs_delta,
                                                static_cast<float2*>(table) + t * block,
                                                (hipStream_t)stream),
                         "rope table launch"));
  return ok();
}

}  // namespace

PIC_API pic_status pic_rope_table_init(const pic_model* model, int32_t max_abs_delta, void* table,
                                       size_t table_bytes, void* stream) {
  PIC_CHECK(check_model(model));
  if (!(model->rope_theta > 1.0) || !std::isfinite(model->rope_theta))
    return fail(PIC_ERR_INVALID_ARG, "rope_theta must be finite and > 1");
  const int half = model->head_dim / 2;
  double inv_freq[64];
  for (int i = 0; i < half; ++i)
    inv_freq[i] = std::pow(model->rope_theta, -2.0 * i / model->head_dim);
  return fill_tables(model, inv_freq, true, max_abs_delta, table, table_bytes, stream);
}

PIC_API pic_status pic_rope_table_init_freq(const pic_model* model, const double* inv_freq,
                                            int32_t max_abs_delta, void* table,
                                            size_t table_bytes, void* stream) {
  PIC_CHECK(check_model(model));
  if (!inv_freq) return fail(PIC_ERR_INVALID_ARG, "inv_freq is NULL");
  const int64_t n = (int64_t)n_tables(model) * (model->head_dim / 2);
  for (int64_t i = 0; i < n; ++i)
    if (!(inv_freq[i] >= 0.0) || !std::isfinite(inv_freq[i]))
      return fail(PIC_ERR_INVALID_ARG, "inv_freq[%lld] must be finite and >= 0", (long long)i);
  return fill_tables(model, inv_freq, false, max_abs_delta, table, table_bytes, stream);
}

PIC_API pic_status pic_rope_llama3_freq(int32_t head_dim, double theta, double factor,
                                        double low_freq_factor, double high_freq_factor,
                                        double original_max_position, double* inv_freq) {
  if (head_dim != 64 && head_dim != 128)
    return fail(PIC_ERR_INVALID_ARG, "head_dim %d (supported: 64, 128)", head_dim);
  if (!inv_freq) return fail(PIC_ERR_INVALID_ARG, "inv_freq is NULL");
  if (!(theta > 1.0) || !(factor > 0.0) || !(low_freq_factor > 0.0) ||
      !(high_freq_factor > low_freq_factor) || !(original_max_position > 0.0) ||
      !std::isfinite(theta) || !std::isfinite(factor) || !std::isfinite(high_freq_factor) ||
      !std::isfinite(original_max_position))
    return fail(PIC_ERR_INVALID_ARG, "inconsistent frequency-scaling parameters");
  const double pi = 3.14159265358979323846;
  const double long_wave = original_max_position / low_freq_factor;   // divided by factor above
  const double short_wave = original_max_position / high_freq_factor; // kept below
  for (int i = 0; i < head_dim / 2; ++i) {
    const double f = std::pow(theta, -2.0 * i / head_dim);
    const double wavelength = 2.0 * pi / f;
    double g;
    if (wavelength < short_wave) {
      g = f;
    } else if (wavelength > long_wave) {
      g = f / factor;
    } else {
      const double t = (original_max_position / wavelength - low_freq_factor) /
                       (high_freq_factor - low_freq_factor);
      g = t * f + (1.0 - t) * f / factor;
    }
    inv_freq[i] = g;
  }
  return ok();
}

PIC_API pic_status pic_rerotate_keys(const pic_model* model, const void* k_in, void* k_out,
                                     int64_t n_tokens, int32_t n_heads, const int32_t* delta,
                                     const void* table, int32_t max_abs_delta, void* stream) {
  PIC_CHECK(check_model(model));
  if (n_tokens < 0 || n_heads <= 0) return fail(PIC_ERR_INVALID_ARG, "n_tokens < 0 or n_heads < 1");
  if (n_tokens > kMaxRerotateRows / n_heads)
    return fail(PIC_ERR_RANGE, "n_tokens * n_heads exceeds %lld rows", (long long)kMaxRerotateRows);
  if (max_abs_delta < 0 || max_abs_delta > kMaxAbsDelta)
    return fail(PIC_ERR_RANGE, "max_abs_delta %d outside [0, %d]", max_abs_delta, kMaxAbsDelta);
  if (n_tokens == 0) return ok();
  PIC_CHECK(check_ptr(k_in, "k_in"));
  PIC_CHECK(check_ptr(k_out, "k_out"));
  PIC_CHECK(check_ptr(table, "table"));
  if (!delta) return fail(PIC_ERR_INVALID_ARG, "delta is NULL");
  return hip_status(pic::launch_rerotate(model->dtype, model->head_dim,
                                         model->rope_pairing == PIC_ROPE_INTERLEAVED, k_in, k_out,
                                         n_tokens * n_heads, n_heads, delta,
                                         static_cast<const float2*>(table), max_abs_delta,
                                         (hipStream_t)stream),
                    "rerotate launch");
}

PIC_API pic_status pic_compose(const pic_model* model, const void* pool_k, const void* pool_v,
                               int64_t pool_tokens, const pic_block* blocks, int32_t n_blocks,
                               const void* table, int32_t max_abs_delta, void* cache_k,
                               void* cache_v, int32_t batch, int32_t cache_cap, void* stream) {
  PIC_CHECK(check_model(model));
  if (pool_tokens < 0 || n_blocks < 0 || batch < 0 || cache_cap < 0)
    return fail(PIC_ERR_INVALID_ARG, "negative size");
  if (max_abs_delta < 0 || max_abs_delta > kMaxAbsDelta)
    return fail(PIC_ERR_RANGE, "max_abs_delta %d outside [0, %d]", max_abs_delta, kMaxAbsDelta);
  if (model->n_kv_heads > 65535 || model->n_layers > 65535)
    return fail(PIC_ERR_UNSUPPORTED, "more than 65535 kv heads or layers in one call");
  if (n_blocks == 0 || model->n_layers == 0) return ok();
  PIC_CHECK(check_ptr(pool_k, "pool_k"));
  PIC_CHECK(check_ptr(pool_v, "pool_v"));
  PIC_CHECK(check_ptr(cache_k, "cache_k"));
  PIC_CHECK(check_ptr(cache_v, "cache_v"));
  PIC_CHECK(check_ptr(table, "table"));
  if (!blocks) return fail(PIC_ERR_INVALID_ARG, "blocks is NULL");
  const int64_t stride = n_tables(model) > 1 ? (int64_t)(max_abs_delta + 1) * (model->head_dim / 2) : 0;
  return hip_status(pic::launch_compose(model->dtype, model->head_dim,
                                        model->rope_pairing == PIC_ROPE_INTERLEAVED,
                                        model->n_layers, model->n_kv_heads, pool_k, pool_v,
                                        pool_tokens, blocks, n_blocks,
                                        static_cast<const float2*>(table), stride, max_abs_delta,
                                        cache_k, cache_v, batch, cache_cap, (hipStream_t)stream),
                    "compose launch");
}

PIC_API pic_status pic_plan_shared(const pic_block* blocks, int32_t n_blocks, pic_block* sorted,
                                   int32_t* group_start, int32_t* n_groups) {
  if (n_blocks < 0) return fail(PIC_ERR_INVALID_ARG, "negative size");
  if (!n_groups || !group_start) return fail(PIC_ERR_INVALID_ARG, "a required host array is NULL");
  if (n_blocks > 0 && (!blocks || !sorted)) return fail(PIC_ERR_INVALID_ARG, "blocks or sorted is NULL");
  // stable order by source run: blocks that read the same pool tokens become neighbours
  std::vector<int32_t> order(n_blocks);
  for (int32_t i = 0; i < n_blocks; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](int32_t x, int32_t y) {
    const pic_block &a = blocks[x], &b = blocks[y];
    return a.src_token != b.src_token ? a.src_token < b.src_token : a.n_tokens < b.n_tokens;
  });
  // a group holds at most kMaxGroup blocks: its workgroup stores them one after another, so a
  // run placed very often (a shared block-boundary header precedes every document of every
  // request) becomes several groups instead of one long serial tail
  constexpr int32_t kMaxGroup = 8;
  int32_t ng = 0, in_group = 0;
  for (int32_t i = 0; i < n_blocks; ++i) {
    const pic_block& b = blocks[order[i]];
    if (i == 0 || b.src_token != sorted[i - 1].src_token || b.n_tokens != sorted[i - 1].n_tokens ||
        in_group == kMaxGroup) {
      group_start[ng++] = i;
      in_group = 0;
    }
    ++in_group;
    sorted[i] = b;
  }
  group_start[ng] = n_blocks;
  *n_groups = ng;
  return ok();
}

PIC_API pic_status pic_compose_shared(const pic_model* model, const void* pool_k, const void* pool_v,
                                      int64_t pool_tokens, const pic_block* blocks, int32_t n_blocks,
                                      const int32_t* group_start, int32_t n_groups,
                                      const void* table, int32_t max_abs_delta, void* cache_k,
                                      void* cache_v, int32_t batch, int32_t cache_cap, void* stream) {
  PIC_CHECK(check_model(model));
  if (pool_tokens < 0 || n_blocks < 0 || n_groups < 0 || batch < 0 || cache_cap < 0)
    return fail(PIC_ERR_INVALID_ARG, "negative size");
  if (n_groups > n_blocks) return fail(PIC_ERR_INVALID_ARG, "more groups (%d) than blocks (%d)", n_groups, n_blocks);
  if (max_abs_delta < 0 || max_abs_delta > kMaxAbsDelta)
    return fail(PIC_ERR_RANGE, "max_abs_delta %d outside [0, %d]", max_abs_delta, kMaxAbsDelta);
  if (model->n_kv_heads > 65535 || model->n_layers > 65535)
    return fail(PIC_ERR_UNSUPPORTED, "more than 65535 kv heads or layers in one call");
  if (n_groups == 0 || model->n_layers == 0) return ok();
  PIC_CHECK(check_ptr(pool_k, "pool_k"));
  PIC_CHECK(check_ptr(pool_v, "pool_v"));
  PIC_CHECK(check_ptr(cache_k, "cache_k"));
  PIC_CHECK(check_ptr(cache_v, "cache_v"));
  PIC_CHECK(check_ptr(table, "table"));
  if (!blocks) return fail(PIC_ERR_INVALID_ARG, "blocks is NULL");
  if (!group_start) return fail(PIC_ERR_INVALID_ARG, "group_start is NULL");
  const int64_t stride = n_tables(model) > 1 ? (int64_t)(max_abs_delta + 1) * (model->head_dim / 2) : 0;
  return hip_status(pic::launch_compose_shared(model->dtype, model->head_dim,
                                               model->rope_pairing == PIC_ROPE_INTERLEAVED,
                                               model->n_layers, model->n_kv_heads, pool_k, pool_v,
                                               pool_tokens, blocks, n_blocks, group_start, n_groups,
                                               static_cast<const float2*>(table), stride,
                                               max_abs_delta, cache_k, cache_v, batch, cache_cap,
                                               (hipStream_t)stream),
                    "compose launch");
}

// ---------------------------------------------------------------------------------------------
// 3. suffix prefill
// ---------------------------------------------------------------------------------------------

PIC_API size_t pic_prefill_workspace_bytes(const pic_model* model, int32_t batch, int32_t n_suffix,
                                           int32_t max_ctx) {
  if (check_attn_model(model) != PIC_OK || batch < 0 || n_suffix < 0 || max_ctx < 0) return 0;
  if (!mfma_prefill(model)) return 0;
  return pic::prefill_bf16_workspace(shape_of(model, batch, max_ctx + n_suffix, 0.f), n_suffix,
                                     max_ctx);
}

PIC_API pic_status pic_suffix_prefill_attn(const pic_model* model, const void* q, const void* k_suf,
                                           const void* v_suf, void* cache_k, void* cache_v,
                                           int32_t batch, int32_t cache_cap, const int32_t* ctx_len,
                                           int32_t max_ctx, int32_t n_suffix, float scale,
                                           void* out, void* workspace, size_t ws_bytes,
                                           void* stream) {
  PIC_CHECK(check_attn_model(model));
  if (batch < 0 || cache_cap < 0 || max_ctx < 0 || n_suffix < 0)
    return fail(PIC_ERR_INVALID_ARG, "negative size");
  if (!(scale >= 0.f) || !std::isfinite(scale))
    return fail(PIC_ERR_INVALID_ARG, "scale must be finite and >= 0");
  if ((int64_t)max_ctx + n_suffix > cache_cap)
    return fail(PIC_ERR_CAPACITY, "max_ctx + n_suffix = %lld exceeds cache_cap %d",
                (long long)max_ctx + n_suffix, cache_cap);
  if ((int64_t)batch * model->n_q_heads * n_suffix > INT32_MAX ||
      (int64_t)n_suffix * (model->n_q_heads / model->n_kv_heads) >= (int64_t(1) << 27))
    return fail(PIC_ERR_UNSUPPORTED, "too many query rows");
  if (model->n_layers > 65535) return fail(PIC_ERR_UNSUPPORTED, "more than 65535 layers");
  PIC_CHECK(check_rows32(cache_cap, (int64_t)n_suffix * model->n_kv_heads, 0));
  if (batch == 0 || n_suffix == 0 || model->n_layers == 0) return ok();
  PIC_CHECK(check_ptr(q, "q"));
  PIC_CHECK(check_ptr(k_suf, "k_suf"));
  PIC_CHECK(check_ptr(v_suf, "v_suf"));
  PIC_CHECK(check_ptr(cache_k, "cache_k"));
  PIC_CHECK(check_ptr(cache_v, "cache_v"));
  PIC_CHECK(check_ptr(out, "out"));
  if (!ctx_len) return fail(PIC_ERR_INVALID_ARG, "ctx_len is NULL");
  const size_t need = pic_prefill_workspace_bytes(model, batch, n_suffix, max_ctx);
  if (need > 0 && (workspace == nullptr || ws_bytes < need))
    return fail(PIC_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  const hipStream_t st = (hipStream_t)stream;
  const pic::AttnShape s = shape_of(model, batch, cache_cap, scale);
  // a4: suffix K/V into slots [ctx, ctx + n_suffix) (App. C.1: inline KVs interleaved); the
  // bf16 matrix-core kernel does this itself
  if (!mfma_prefill(model)) {
    pic::RowPos pos;
    pos.base = ctx_len;
    pos.max_base = max_ctx;
    PIC_CHECK(hip_status(pic::launch_append(model->dtype, model->head_dim, model->n_layers,
                                            model->n_kv_heads, k_suf, v_suf, cache_k, cache_v,
                                            batch, cache_cap, pos, n_suffix, st),
                         "suffix append launch"));
    return launch_rows(model, s, q, cache_k, cache_v, pos, n_suffix, out, st, "prefill attention launch");
  }
  return hip_status(pic::launch_prefill_bf16(s, static_cast<const pic::bf16_t*>(q),
                                             static_cast<const pic::bf16_t*>(k_suf),
                                             static_cast<const pic::bf16_t*>(v_suf),
                                             static_cast<pic::bf16_t*>(cache_k),
                                             static_cast<pic::bf16_t*>(cache_v), ctx_len,
                                             max_ctx, n_suffix, static_cast<pic::bf16_t*>(out),
                                             workspace, ws_bytes, st),
                    "prefill attention launch");
}

PIC_API pic_status pic_suffix_prefill_attn_rope(const pic_model* model, const void* q,
                                                const void* k_suf, const void* v_suf,
                                                void* cache_k, void* cache_v, int32_t batch,
                                                int32_t cache_cap, const int32_t* ctx_len,
                                                int32_t max_ctx, int32_t n_suffix,
                                                const void* table, int32_t max_abs_delta,
                                                float scale, void* out, void* workspace,
                                                size_t ws_bytes, void* stream) {
  PIC_CHECK(check_attn_model(model));
  if (model->dtype != PIC_BF16)
    return fail(PIC_ERR_UNSUPPORTED, "the fused-RoPE prefill is built for bf16 caches");
  if (batch < 0 || cache_cap < 0 || max_ctx < 0 || n_suffix < 0)
    return fail(PIC_ERR_INVALID_ARG, "negative size");
  if (!(scale >= 0.f) || !std::isfinite(scale))
    return fail(PIC_ERR_INVALID_ARG, "scale must be finite and >= 0");
  if (max_abs_delta < 0 || max_abs_delta > kMaxAbsDelta)
    return fail(PIC_ERR_RANGE, "max_abs_delta %d outside [0, %d]", max_abs_delta, kMaxAbsDelta);
  if ((int64_t)max_ctx + n_suffix > cache_cap)
    return fail(PIC_ERR_CAPACITY, "max_ctx + n_suffix = %lld exceeds cache_cap %d",
                (long long)max_ctx + n_suffix, cache_cap);
  if ((int64_t)max_ctx + n_suffix - 1 > max_abs_delta)
    return fail(PIC_ERR_RANGE, "positions up to %lld need a table with max_abs_delta >= that, got %d",
                (long long)max_ctx + n_suffix - 1, max_abs_delta);
  if ((int64_t)batch * model->n_q_heads * n_suffix > INT32_MAX ||
      (int64_t)n_suffix * (model->n_q_heads / model->n_kv_heads) >= (int64_t(1) << 27))
    return fail(PIC_ERR_UNSUPPORTED, "too many query rows");
  if (model->n_layers > 65535) return fail(PIC_ERR_UNSUPPORTED, "more than 65535 layers");
  PIC_CHECK(check_rows32(cache_cap, (int64_t)n_suffix * model->n_kv_heads, 0));
  if (batch == 0 || n_suffix == 0 || model->n_layers == 0) return ok();
  PIC_CHECK(check_ptr(q, "q"));
  PIC_CHECK(check_ptr(k_suf, "k_suf"));
  PIC_CHECK(check_ptr(v_suf, "v_suf"));
  PIC_CHECK(check_ptr(cache_k, "cache_k"));
  PIC_CHECK(check_ptr(cache_v, "cache_v"));
  PIC_CHECK(check_ptr(table, "table"));
  PIC_CHECK(check_ptr(out, "out"));
  if (!ctx_len) return fail(PIC_ERR_INVALID_ARG, "ctx_len is NULL");
  const size_t need = pic_prefill_workspace_bytes(model, batch, n_suffix, max_ctx);
  if (need > 0 && (workspace == nullptr || ws_bytes < need))
    return fail(PIC_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  const pic::AttnShape s = shape_of(model, batch, cache_cap, scale);
  const int64_t stride = n_tables(model) > 1 ? (int64_t)(max_abs_delta + 1) * (model->head_dim / 2) : 0;
  return hip_status(pic::launch_prefill_bf16_rope(
                        s, model->rope_pairing == PIC_ROPE_INTERLEAVED,
                        static_cast<const pic::bf16_t*>(q), static_cast<const pic::bf16_t*>(k_suf),
                        static_cast<const pic::bf16_t*>(v_suf), static_cast<pic::bf16_t*>(cache_k),
                        static_cast<pic::bf16_t*>(cache_v), ctx_len, max_ctx, n_suffix,
                        static_cast<const float2*>(table), stride, max_abs_delta,
                        static_cast<pic::bf16_t*>(out), workspace, ws_bytes, (hipStream_t)stream),
                    "fused-RoPE prefill launch");
}

PIC_API pic_status pic_build_slot_map(const pic_block* blocks, int32_t n_blocks, int32_t batch,
                                      int32_t map_cap, int32_t* slot_src, int32_t* slot_delta,
                                      int32_t* tile_map, void* stream) {
  if (n_blocks < 0 || batch < 0 || map_cap < 0) return fail(PIC_ERR_INVALID_ARG, "negative size");
  if ((int64_t)batch * map_cap == 0) return ok();
  if (n_blocks > 0 && !blocks) return fail(PIC_ERR_INVALID_ARG, "blocks is NULL");
  if (!slot_src || !slot_delta) return fail(PIC_ERR_INVALID_ARG, "slot map is NULL");
  if (tile_map) PIC_CHECK(check_ptr(tile_map, "tile_map"));
  return hip_status(pic::launch_slot_map(blocks, n_blocks, batch, map_cap, slot_src, slot_delta,
                                         tile_map, (hipStream_t)stream),
                    "slot map launch");
}

PIC_API pic_status pic_compose_tiles(const pic_model* model, const void* pool_k, const void* pool_v,
                                     int64_t pool_tokens, const int32_t* slot_src,
                                     const int32_t* slot_delta, int32_t map_cap,
                                     const int32_t* tile_map, const void* table,
                                     int32_t max_abs_delta, const int32_t* ctx_len, int32_t max_ctx,
                                     void* cache_k, void* cache_v, int32_t batch, int32_t cache_cap,
                                     void* stream) {
  PIC_CHECK(check_attn_model(model));
  if (!mfma_prefill(model)) return fail(PIC_ERR_UNSUPPORTED, "tile composition is built for bf16 caches");
  if (batch < 0 || cache_cap < 0 || max_ctx < 0 || pool_tokens < 0 || map_cap < 0)
    return fail(PIC_ERR_INVALID_ARG, "negative size");
  if (max_abs_delta < 0 || max_abs_delta > kMaxAbsDelta)
    return fail(PIC_ERR_RANGE, "max_abs_delta %d outside [0, %d]", max_abs_delta, kMaxAbsDelta);
  if (max_ctx > cache_cap)
    return fail(PIC_ERR_CAPACITY, "max_ctx %d exceeds cache_cap %d", max_ctx, cache_cap);
  if (map_cap < max_ctx)
    return fail(PIC_ERR_CAPACITY, "map_cap %d is below max_ctx %d", map_cap, max_ctx);
  if (max_ctx > 0 && pool_tokens == 0) return fail(PIC_ERR_RANGE, "empty pool");
  if (model->n_layers > 65535) return fail(PIC_ERR_UNSUPPORTED, "more than 65535 layers");
  PIC_CHECK(check_rows32(cache_cap, 0, pool_tokens));
  if (batch == 0 || max_ctx == 0 || model->n_layers == 0) return ok();
  PIC_CHECK(check_ptr(pool_k, "pool_k"));
  PIC_CHECK(check_ptr(pool_v, "pool_v"));
  PIC_CHECK(check_ptr(table, "table"));
  PIC_CHECK(check_ptr(cache_k, "cache_k"));
  PIC_CHECK(check_ptr(cache_v, "cache_v"));
  if (!slot_src || !slot_delta) return fail(PIC_ERR_INVALID_ARG, "slot map is NULL");
  PIC_CHECK(check_ptr(tile_map, "tile_map"));
  if (!ctx_len) return fail(PIC_ERR_INVALID_ARG, "ctx_len is NULL");
  const int64_t stride = n_tables(model) > 1 ? (int64_t)(max_abs_delta + 1) * (model->head_dim / 2) : 0;
  return hip_status(pic::launch_compose_tiles(model->rope_pairing == PIC_ROPE_INTERLEAVED, model->head_dim, model->n_layers,
                                              model->n_kv_heads, static_cast<const pic::bf16_t*>(pool_k),
                                              static_cast<const pic::bf16_t*>(pool_v), pool_tokens, slot_src,
                                              slot_delta, map_cap > 0 ? map_cap : 1, tile_map,
                                              pic::slot_map_tiles(map_cap > 0 ? map_cap : 1), ctx_len,
                                              max_ctx, static_cast<const float2*>(table), stride,
                                              max_abs_delta, static_cast<pic::bf16_t*>(cache_k),
                                              static_cast<pic::bf16_t*>(cache_v), batch, cache_cap,
                                              (hipStream_t)stream),
                    "tile compose launch");
}

PIC_API pic_status pic_paged_prefill_attn(const pic_model* model, const void* pool_k,
                                          const void* pool_v, int64_t pool_tokens,
                                          const int32_t* slot_src, const int32_t* slot_delta,
                                          int32_t map_cap, const int32_t* tile_map,
                                          const void* table, int32_t max_abs_delta,
                                          const void* q, const void* k_suf, const void* v_suf,
                                          void* cache_k, void* cache_v, int32_t batch,
                                          int32_t cache_cap, const int32_t* ctx_len,
                                          int32_t max_ctx, int32_t n_suffix, float scale,
                                          void* out, void* workspace, size_t ws_bytes,
                                          void* stream) {
  PIC_CHECK(check_attn_model(model));
  if (model->dtype != PIC_BF16)
    return fail(PIC_ERR_UNSUPPORTED, "the paged prefill is built for bf16 caches");
  if (batch < 0 || cache_cap < 0 || max_ctx < 0 || n_suffix < 0 || pool_tokens < 0 || map_cap < 0)
    return fail(PIC_ERR_INVALID_ARG, "negative size");
  if (!(scale >= 0.f) || !std::isfinite(scale))
    return fail(PIC_ERR_INVALID_ARG, "scale must be finite and >= 0");
  if (max_abs_delta < 0 || max_abs_delta > kMaxAbsDelta)
    return fail(PIC_ERR_RANGE, "max_abs_delta %d outside [0, %d]", max_abs_delta, kMaxAbsDelta);
  if ((int64_t)max_ctx + n_suffix > cache_cap)
    return fail(PIC_ERR_CAPACITY, "max_ctx + n_suffix = %lld exceeds cache_cap %d",
                (long long)max_ctx + n_suffix, cache_cap);
  if (map_cap < max_ctx)
    return fail(PIC_ERR_CAPACITY, "map_cap %d is below max_ctx %d", map_cap, max_ctx);
  if (max_ctx > 0 && pool_tokens == 0) return fail(PIC_ERR_RANGE, "empty pool");
  if ((int64_t)batch * model->n_q_heads * n_suffix > INT32_MAX ||
      (int64_t)n_suffix * (model->n_q_heads / model->n_kv_heads) >= (int64_t(1) << 27))
    return fail(PIC_ERR_UNSUPPORTED, "too many query rows");
  if (model->n_layers > 65535) return fail(PIC_ERR_UNSUPPORTED, "more than 65535 layers");
  PIC_CHECK(check_rows32(cache_cap, (int64_t)n_suffix * model->n_kv_heads, pool_tokens));
  if (batch == 0 || n_suffix == 0 || model->n_layers == 0) return ok();
  PIC_CHECK(check_ptr(pool_k, "pool_k"));
  PIC_CHECK(check_ptr(pool_v, "pool_v"));
  PIC_CHECK(check_ptr(table, "table"));
  PIC_CHECK(check_ptr(q, "q"));
  PIC_CHECK(check_ptr(k_suf, "k_suf"));
  PIC_CHECK(check_ptr(v_suf, "v_suf"));
  PIC_CHECK(check_ptr(cache_k, "cache_k"));
  PIC_CHECK(check_ptr(cache_v, "cache_v"));
  PIC_CHECK(check_ptr(out, "out"));
  if (tile_map) PIC_CHECK(check_ptr(tile_map, "tile_map"));
  if (!slot_src != !slot_delta) return fail(PIC_ERR_INVALID_ARG, "one of the slot maps is NULL");
  // no slot map: the non-run tiles were composed beforehand (pic_compose_tiles), and the
  // call reads whole runs from the pool and every other tile from the cache
  if (!slot_src && !tile_map) return fail(PIC_ERR_INVALID_ARG, "slot map is NULL (allowed only with a tile map)");
  if (!ctx_len) return fail(PIC_ERR_INVALID_ARG, "ctx_len is NULL");
  const size_t need = pic_prefill_workspace_bytes(model, batch, n_suffix, max_ctx);
  if (need > 0 && (workspace == nullptr || ws_bytes < need))
    return fail(PIC_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  const pic::AttnShape s = shape_of(model, batch, cache_cap, scale);
  const int64_t stride = n_tables(model) > 1 ? (int64_t)(max_abs_delta + 1) * (model->head_dim / 2) : 0;
  return hip_status(pic::launch_prefill_bf16_paged(
                        s, model->rope_pairing == PIC_ROPE_INTERLEAVED,
                        static_cast<const pic::bf16_t*>(q), static_cast<const pic::bf16_t*>(k_suf),
                        static_cast<const pic::bf16_t*>(v_suf), static_cast<pic::bf16_t*>(cache_k),
                        static_cast<pic::bf16_t*>(cache_v), ctx_len, max_ctx, n_suffix,
                        static_cast<const pic::bf16_t*>(pool_k),
                        static_cast<const pic::bf16_t*>(pool_v), pool_tokens, slot_src, slot_delta,
                        map_cap > 0 ? map_cap : 1, tile_map, static_cast<const float2*>(table), stride,
                        max_abs_delta, static_cast<pic::bf16_t*>(out), workspace, ws_bytes,
                        (hipStream_t)stream),
                    "paged prefill launch");
}

PIC_API size_t pic_frontier_workspace_bytes(const pic_model* model, int32_t batch,
                                            int32_t n_inline, int32_t max_len) {
  if (check_attn_model(model) != PIC_OK || batch < 0 || n_inline < 0 || max_len < 0) return 0;
  if (!mfma_prefill(model)) return 0;
  const int32_t max_ctx = max_len > n_inline ? max_len - n_inline : 0;
  return pic::prefill_bf16_workspace(shape_of(model, batch, max_len, 0.f), n_inline, max_ctx);
}

PIC_API pic_status pic_frontier_prefill_attn(const pic_model* model, const void* q,
                                             const void* k_inl, const void* v_inl, void* cache_k,
                                             void* cache_v, int32_t batch, int32_t cache_cap,
                                             const int32_t* pos, const int32_t* n_valid,
                                             int32_t n_inline, int32_t max_len, float scale,
                                             void* out, void* workspace, size_t ws_bytes,
                                             void* stream) {
  PIC_CHECK(check_attn_model(model));
  if (batch < 0 || cache_cap < 0 || n_inline < 0 || max_len < 0)
    return fail(PIC_ERR_INVALID_ARG, "negative size");
  if (!(scale >= 0.f) || !std::isfinite(scale))
    return fail(PIC_ERR_INVALID_ARG, "scale must be finite and >= 0");
  if (max_len > cache_cap)
    return fail(PIC_ERR_CAPACITY, "max_len %d exceeds cache_cap %d", max_len, cache_cap);
  if ((int64_t)batch * model->n_q_heads * n_inline > INT32_MAX ||
      (int64_t)n_inline * (model->n_q_heads / model->n_kv_heads) >= (int64_t(1) << 27))
    return fail(PIC_ERR_UNSUPPORTED, "too many query rows");
  if (model->n_layers > 65535) return fail(PIC_ERR_UNSUPPORTED, "more than 65535 layers");
  PIC_CHECK(check_rows32(cache_cap, 0, 0));
  if (batch == 0 || n_inline == 0 || model->n_layers == 0 || max_len == 0) return ok();
  PIC_CHECK(check_ptr(q, "q"));
  PIC_CHECK(check_ptr(k_inl, "k_inl"));
  PIC_CHECK(check_ptr(v_inl, "v_inl"));
  PIC_CHECK(check_ptr(cache_k, "cache_k"));
  PIC_CHECK(check_ptr(cache_v, "cache_v"));
  PIC_CHECK(check_ptr(out, "out"));
  if (!pos) return fail(PIC_ERR_INVALID_ARG, "pos is NULL");
  if (!n_valid) return fail(PIC_ERR_INVALID_ARG, "n_valid is NULL");
  const size_t need = pic_frontier_workspace_bytes(model, batch, n_inline, max_len);
  if (need > 0 && (workspace == nullptr || ws_bytes < need))
    return fail(PIC_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  const hipStream_t st = (hipStream_t)stream;
  const pic::AttnShape s = shape_of(model, batch, cache_cap, scale);
  pic::RowPos rp;
  rp.table = pos;
  rp.n_valid = n_valid;
  rp.n = n_inline;
  rp.max_pos = max_len - 1;
  // inline K/V at their logical slots, interleaved with the composed documents (App. C.1)
  PIC_CHECK(hip_status(pic::launch_append(model->dtype, model->head_dim, model->n_layers,
                                          model->n_kv_heads, k_inl, v_inl, cache_k, cache_v,
                                          batch, cache_cap, rp, n_inline, st),
                       "inline append launch"));
  if (!mfma_prefill(model))
    return launch_rows(model, s, q, cache_k, cache_v, rp, n_inline, out, st, "frontier attention launch");
  return hip_status(pic::launch_prefill_bf16_table(s, static_cast<const pic::bf16_t*>(q),
                                                   static_cast<const pic::bf16_t*>(cache_k),
                                                   static_cast<const pic::bf16_t*>(cache_v), rp,
                                                   n_inline, max_len,
                                                   static_cast<pic::bf16_t*>(out), workspace,
                                                   ws_bytes, st),
                    "frontier attention launch");
}

// ---------------------------------------------------------------------------------------------
// 4. decode
// ---------------------------------------------------------------------------------------------

PIC_API int32_t pic_decode_auto_splits(const pic_model* model, int32_t batch, int32_t max_len) {
  if (check_attn_model(model) != PIC_OK || batch <= 0 || max_len <= 0) return 1;
  if (!mfma_decode(model)) return 1;
  return pic::decode_bf16_auto_splits(shape_of(model, batch, max_len, 0.f), max_len);
}

PIC_API size_t pic_decode_workspace_bytes(const pic_model* model, int32_t batch, int32_t max_len,
                                          int32_t n_splits) {
  if (check_attn_model(model) != PIC_OK || batch < 0 || max_len < 0 || n_splits < 0) return 0;
  if (!mfma_decode(model)) return 0;
  if (n_splits == 0) n_splits = pic_decode_auto_splits(model, batch, max_len);
  return pic::decode_bf16_workspace(shape_of(model, batch, max_len, 0.f), max_len, n_splits);
}

namespace {

// use_scratch: the split partials go to the library's per-device scratch array instead of a
// caller workspace (workspace / ws_bytes are then ignored).
pic_status decode_impl(const pic_model* model, const void* q, const void* k_new, const void* v_new,
                       void* cache_k, void* cache_v, int32_t batch, int32_t cache_cap,
                       const int32_t* base_len, int32_t step, int32_t max_base_len,
                       const void* table, int32_t max_abs_delta, float scale, int32_t n_splits,
                       void* out, void* workspace, size_t ws_bytes, void* stream,
                       bool use_scratch = false) {
  PIC_CHECK(check_attn_model(model));
  if (batch < 0 || cache_cap < 0 || step < 0 || max_base_len < 0 || n_splits < 0)
    return fail(PIC_ERR_INVALID_ARG, "negative size");
  if (!(scale >= 0.f) || !std::isfinite(scale))
    return fail(PIC_ERR_INVALID_ARG, "scale must be finite and >= 0");
  const int64_t max_len = (int64_t)max_base_len + step + 1;
  if (max_len > cache_cap)
    return fail(PIC_ERR_CAPACITY, "max_base_len + step + 1 = %lld exceeds cache_cap %d",
                (long long)max_len, cache_cap);
  if (model->n_layers > 65535) return fail(PIC_ERR_UNSUPPORTED, "more than 65535 layers");
  if ((int64_t)batch * model->n_q_heads > INT32_MAX)
    return fail(PIC_ERR_UNSUPPORTED, "too many query rows");
  if (batch == 0 || model->n_layers == 0) return ok();
  PIC_CHECK(check_ptr(q, "q"));
  PIC_CHECK(check_ptr(k_new, "k_new"));
  PIC_CHECK(check_ptr(v_new, "v_new"));
  PIC_CHECK(check_ptr(cache_k, "cache_k"));
  PIC_CHECK(check_ptr(cache_v, "cache_v"));
  PIC_CHECK(check_ptr(out, "out"));
  if (!base_len) return fail(PIC_ERR_INVALID_ARG, "base_len is NULL");
  if (table) {   // fused RoPE: every position the call turns must be in the table
    if (model->dtype != PIC_BF16)
      return fail(PIC_ERR_UNSUPPORTED, "the fused-RoPE decode is built for bf16 caches");
    PIC_CHECK(check_ptr(table, "table"));
    if (max_abs_delta < 0 || max_abs_delta > kMaxAbsDelta || max_len - 1 > max_abs_delta)
      return fail(PIC_ERR_RANGE, "position %lld needs a table with max_abs_delta >= that, got %d",
                  (long long)(max_len - 1), max_abs_delta);
  }
  const hipStream_t st = (hipStream_t)stream;
  const pic::AttnShape s = shape_of(model, batch, cache_cap, scale);
  if (!mfma_decode(model)) {   // float32: row-wise kernel, no splits
    pic::RowPos pos;
    pos.base = base_len;
    pos.max_base = max_base_len;
    pos.offset = step;
    const int64_t stride = n_tables(model) > 1 ? (int64_t)(max_abs_delta + 1) * (model->head_dim / 2) : 0;
    if (table)
      PIC_CHECK(hip_status(pic::launch_append_rope(model->head_dim, model->rope_pairing == PIC_ROPE_INTERLEAVED,
                                                   model->n_layers, model->n_kv_heads,
                                                   static_cast<const pic::bf16_t*>(k_new),
                                                   static_cast<const pic::bf16_t*>(v_new),
                                                   static_cast<pic::bf16_t*>(cache_k),
                                                   static_cast<pic::bf16_t*>(cache_v), batch, cache_cap, pos, 1,
                                                   static_cast<const float2*>(table), stride, max_abs_delta, st),
                           "decode append launch"));
    else
      PIC_CHECK(hip_status(pic::launch_append(model->dtype, model->head_dim, model->n_layers,
                                              model->n_kv_heads, k_new, v_new, cache_k, cache_v,
                                              batch, cache_cap, pos, 1, st),
                           "decode append launch"));
    RowOpts o;
    o.q_table = table;
    o.table_stride = stride;
    o.max_abs_delta = max_abs_delta;
    return launch_rows(model, s, q, cache_k, cache_v, pos, 1, out, st, "decode attention launch", o);
  }
  if (n_splits == 0) n_splits = pic::decode_bf16_auto_splits(s, (int32_t)max_len);
  if ((int64_t)n_splits * batch * model->n_kv_heads * ((model->n_q_heads / model->n_kv_heads + 15) / 16) > INT32_MAX)
    return fail(PIC_ERR_UNSUPPORTED, "too many splits");
  if (n_splits > max_len) n_splits = (int32_t)max_len;
  const size_t need = pic::decode_bf16_workspace(s, (int32_t)max_len, n_splits);
  if (use_scratch) {
    workspace = nullptr;
    ws_bytes = 0;
    if (need > pic::decode_scratch_bytes())
      return fail(PIC_ERR_WORKSPACE,
                  "%d splits need %zu bytes of partials; the allocation-free decode holds %zu "
                  "(pass fewer splits, or use pic_decode_attn with a workspace)",
                  n_splits, need, pic::decode_scratch_bytes());
    if (need > 0) {
      PIC_CHECK(hip_status(pic::decode_scratch_ptr(&workspace), "decode scratch lookup"));
      ws_bytes = pic::decode_scratch_bytes();
    }
  }
  if (need > 0 && (workspace == nullptr || ws_bytes < need))
    return fail(PIC_ERR_WORKSPACE, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  if (need > 0) PIC_CHECK(check_ptr(workspace, "workspace"));
  return hip_status(pic::launch_decode_bf16(s, static_cast<const pic::bf16_t*>(q),
                                            static_cast<const pic::bf16_t*>(k_new),
                                            static_cast<const pic::bf16_t*>(v_new),
                                            static_cast<pic::bf16_t*>(cache_k),
                                            static_cast<pic::bf16_t*>(cache_v), base_len,
                                            max_base_len, step, n_splits,
                                            static_cast<pic::bf16_t*>(out), workspace, ws_bytes,
                                            static_cast<const float2*>(table),
                                            n_tables(model) > 1 ? (int64_t)(max_abs_delta + 1) * (model->head_dim / 2) : 0,
                                            max_abs_delta, model->rope_pairing == PIC_ROPE_INTERLEAVED, st),
                    "decode attention launch");
}

}  // namespace

PIC_API pic_status pic_decode_attn(const pic_model* model, const void* q, const void* k_new,
                                   const void* v_new, void* cache_k, void* cache_v, int32_t batch,
                                   int32_t cache_cap, const int32_t* base_len, int32_t step,
                                   int32_t max_base_len, float scale, int32_t n_splits, void* out,
                                   void* workspace, size_t ws_bytes, void* stream) {
  return decode_impl(model, q, k_new, v_new, cache_k, cache_v, batch, cache_cap, base_len, step,
                     max_base_len, nullptr, 0, scale, n_splits, out, workspace, ws_bytes, stream);
}

PIC_API pic_status pic_decode_attn_rope(const pic_model* model, const void* q, const void* k_new,
                                        const void* v_new, void* cache_k, void* cache_v,
                                        int32_t batch, int32_t cache_cap, const int32_t* base_len,
                                        int32_t step, int32_t max_base_len, const void* table,
                                        int32_t max_abs_delta, float scale, int32_t n_splits,
                                        void* out, void* workspace, size_t ws_bytes, void* stream) {
  if (!table) return fail(PIC_ERR_INVALID_ARG, "table is NULL");
  return decode_impl(model, q, k_new, v_new, cache_k, cache_v, batch, cache_cap, base_len, step,
                     max_base_len, table, max_abs_delta, scale, n_splits, out, workspace, ws_bytes,
                     stream);
}

PIC_API pic_status pic_decode_attn_noalloc(const pic_model* model, const void* q, const void* k_new,
                                           const void* v_new, void* cache_k, void* cache_v,
                                           int32_t batch, int32_t cache_cap, const int32_t* base_len,
                                           int32_t step, int32_t max_base_len, float scale,
                                           int32_t n_splits, void* out, void* stream) {
  return decode_impl(model, q, k_new, v_new, cache_k, cache_v, batch, cache_cap, base_len, step,
                     max_base_len, nullptr, 0, scale, n_splits, out, nullptr, 0, stream, true);
}
