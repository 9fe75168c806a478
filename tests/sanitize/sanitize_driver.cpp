// Sanitizer driver for libpic's host code: the C ABI (argument checks, the layout planners,
// the shared-source planner, launch planning) built with AddressSanitizer and
// UndefinedBehaviorSanitizer against the CPU emulation of the kernel launches
// (emulated_launchers.cpp).
//
// Every buffer is a separate host allocation of exactly the size the call's contract gives it
// (rows x head_dim elements of the documented layout), so a row any kernel would address
// outside its buffer is an AddressSanitizer report.  Device-side tables (gather blocks, group
// starts, slot and tile maps, context and base lengths, position tables) are filled with
// valid plans and with random garbage; the kernels promise to clamp every index they derive
// from them.  Calls that fail their checks must launch nothing.
//
// usage: sanitize_driver [seed] [rounds]      prints "sanitizer driver: OK" and exits 0
//        sanitize_driver --plant              a cache one row short: must end in an ASan report
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "pic.h"

namespace pic {
namespace emu {
extern long launches;
}
}  // namespace pic

namespace {

std::mt19937_64 rng;

int64_t rnd(int64_t lo, int64_t hi) { return std::uniform_int_distribution<int64_t>(lo, hi)(rng); }

// A heap buffer of exactly n bytes, 16-byte aligned as the ABI requires of device pointers.
struct Buf {
  void* p = nullptr;
  size_t n = 0;
  explicit Buf(size_t bytes) : n(bytes) {   // exactly `bytes` (no rounding that could hide an overrun)
    if (posix_memalign(&p, 16, bytes == 0 ? 1 : bytes) != 0) std::abort();
    std::memset(p, 0, bytes == 0 ? 1 : bytes);
  }
  ~Buf() { std::free(p); }
  Buf(const Buf&) = delete;
  Buf& operator=(const Buf&) = delete;
  template <typename T>
  T* as() { return static_cast<T*>(p); }
};

int failures = 0;
#define EXPECT(cond)                                                                   \
  do {                                                                                 \
    if (!(cond)) {                                                                     \
      std::fprintf(stderr, "FAILED %s:%d: %s (%s)\n", __FILE__, __LINE__, #cond,       \
                   pic_last_error());                                                  \
      ++failures;                                                                      \
    }                                                                                  \
  } while (0)

// garbage int32 table values: mostly plausible, some wildly out of range
int32_t garbage(int32_t scale) {
  switch (rnd(0, 5)) {
    case 0: return (int32_t)rnd(INT32_MIN, INT32_MAX);
    case 1: return -(int32_t)rnd(1, 1 << 20);
    case 2: return (int32_t)rnd(0, 2 * (int64_t)scale + 8);
    default: return (int32_t)rnd(0, scale > 0 ? scale - 1 : 0);
  }
}

pic_model model(int L, int hq, int hkv, int D, pic_dtype dt, int pairing = 0, int tables = 1) {
  pic_model m;
  m.n_layers = L;
  m.n_q_heads = hq;
  m.n_kv_heads = hkv;
  m.head_dim = D;
  m.dtype = dt;
  m.rope_theta = 1e4;
  m.rope_pairing = pairing;
  m.rope_tables = tables;
  return m;
}

size_t eb(const pic_model& m) { return m.dtype == PIC_F32 ? 4 : 2; }

// ---- planners ----
void fuzz_planners() {
  for (int it = 0; it < 300; ++it) {
    const int32_t n_pool = (int32_t)rnd(0, 12), batch = (int32_t)rnd(0, 5);
    std::vector<int32_t> off(n_pool), len(n_pool), cpos(n_pool);
    int64_t pool_tokens = 0;
    for (int e = 0; e < n_pool; ++e) {
      len[e] = (int32_t)rnd(it % 7 == 0 ? 0 : 1, 300);
      off[e] = (int32_t)pool_tokens;
      pool_tokens += len[e];
      cpos[e] = (int32_t)rnd(0, 40);
    }
    if (it % 11 == 0 && n_pool) off[rnd(0, n_pool - 1)] += 5;   // an entry past the pool
    std::vector<int32_t> n_items(batch), items;
    for (int b = 0; b < batch; ++b) {
      n_items[b] = (int32_t)rnd(0, 6);
      for (int k = 0; k < n_items[b]; ++k)
        items.push_back(it % 5 == 0 ? (int32_t)rnd(-40, n_pool + 1) : (n_pool ? (int32_t)rnd(0, n_pool - 1) : 0));
    }
    std::vector<int32_t> ctx(batch > 0 ? batch : 1), total(batch > 0 ? batch : 1), n_inl(batch > 0 ? batch : 1);
    int32_t n_blocks = 0;
    const int32_t cap = (int32_t)rnd(0, 60);
    std::vector<pic_block> blocks(cap > 0 ? cap : 1);
    const int32_t inline_cap = (int32_t)rnd(0, 80);
    std::vector<int32_t> inl((size_t)(batch > 0 ? batch : 1) * (inline_cap > 0 ? inline_cap : 1));
    const pic_status s1 = pic_plan_layout(batch, n_items.data(), items.empty() ? nullptr : items.data(), n_pool,
                                          off.data(), len.data(), cpos.data(), pool_tokens,
                                          cap ? blocks.data() : nullptr, cap, &n_blocks, ctx.data());
    if (s1 == PIC_OK) {
      // blocks tile each request's context exactly, in slot order, inside the pool
      for (int32_t i = 0; i < n_blocks; ++i) {
        const pic_block& b = blocks[i];
        EXPECT(b.request >= 0 && b.request < batch && b.n_tokens >= 1 && b.n_tokens <= PIC_BLOCK_TOKENS);
        EXPECT(b.src_token >= 0 && (int64_t)b.src_token + b.n_tokens <= pool_tokens);
        EXPECT(b.dst_slot >= 0 && b.dst_slot + b.n_tokens <= ctx[b.request]);
      }
      std::vector<int64_t> covered(batch, 0);
      for (int32_t i = 0; i < n_blocks; ++i) covered[blocks[i].request] += blocks[i].n_tokens;
      for (int b = 0; b < batch; ++b) EXPECT(covered[b] == ctx[b]);
      // grouping by source run
      std::vector<pic_block> sorted(n_blocks > 0 ? n_blocks : 1);
      std::vector<int32_t> starts(n_blocks + 1);
      int32_t n_groups = 0;
      EXPECT(pic_plan_shared(blocks.data(), n_blocks, sorted.data(), starts.data(), &n_groups) == PIC_OK);
      EXPECT(n_groups <= n_blocks && starts[n_groups] == n_blocks);
      for (int g = 0; g < n_groups; ++g) {
        EXPECT(starts[g] < starts[g + 1] && starts[g + 1] - starts[g] <= 8);
        for (int i = starts[g]; i < starts[g + 1]; ++i)
          EXPECT(sorted[i].src_token == sorted[starts[g]].src_token && sorted[i].n_tokens == sorted[starts[g]].n_tokens);
      }
    }
    const pic_status s2 = pic_plan_frontier(batch, n_items.data(), items.empty() ? nullptr : items.data(), n_pool,
                                            off.data(), len.data(), cpos.data(), pool_tokens,
                                            cap ? blocks.data() : nullptr, cap, &n_blocks, total.data(),
                                            inline_cap ? inl.data() : nullptr, inline_cap, n_inl.data());
    if (s2 == PIC_OK)
      for (int b = 0; b < batch; ++b) {
        EXPECT(n_inl[b] >= 0 && n_inl[b] <= inline_cap);
        for (int i = 0; i < n_inl[b]; ++i) EXPECT(inl[(size_t)b * inline_cap + i] >= 0 && inl[(size_t)b * inline_cap + i] < total[b]);
      }
  }
}

// ---- composition and re-rotation over garbage tables ----
void fuzz_compose() {
  for (int it = 0; it < 60; ++it) {
    const pic_dtype dt = rnd(0, 1) ? PIC_BF16 : PIC_F32;
    const int D = rnd(0, 1) ? 128 : 64, L = (int)rnd(1, 2), Hkv = (int)rnd(1, 3);
    const int tables = rnd(0, 3) == 0 ? L : 1;
    pic_model m = model(L, Hkv * 2, Hkv, D, dt, (int)rnd(0, 1), tables);
    const int64_t pool_tokens = rnd(1, 400);
    const int32_t batch = (int32_t)rnd(1, 3), cap = (int32_t)rnd(1, 300), mad = (int32_t)rnd(0, 500);
    const size_t row = (size_t)D * eb(m);
    Buf pk(L * Hkv * pool_tokens * row), pv(L * Hkv * pool_tokens * row);
    Buf ck((size_t)L * batch * Hkv * cap * row), cv((size_t)L * batch * Hkv * cap * row);
    Buf table(pic_rope_table_bytes(&m, mad));
    EXPECT(table.n > 0);
    EXPECT(pic_rope_table_init(&m, mad, table.p, table.n, nullptr) == PIC_OK);
    const int32_t nb = (int32_t)rnd(0, 40);
    Buf blk(nb * sizeof(pic_block));
    for (int i = 0; i < nb; ++i) {
      pic_block& b = blk.as<pic_block>()[i];
      b.request = garbage(batch);
      b.src_token = garbage((int32_t)pool_tokens);
      b.dst_slot = garbage(cap);
      b.n_tokens = rnd(0, 3) ? (int32_t)rnd(1, 64) : garbage(64);
      b.delta = rnd(0, 3) ? (int32_t)rnd(-mad, mad) : garbage(mad);
    }
    EXPECT(pic_compose(&m, pk.p, pv.p, pool_tokens, blk.as<pic_block>(), nb, table.p, mad, ck.p, cv.p, batch, cap,
                       nullptr) == PIC_OK);
    const int32_t ng = nb ? (int32_t)rnd(0, nb) : 0;
    Buf gs((ng + 1) * sizeof(int32_t));
    for (int g = 0; g <= ng; ++g) gs.as<int32_t>()[g] = garbage(nb + 1);
    EXPECT(pic_compose_shared(&m, pk.p, pv.p, pool_tokens, blk.as<pic_block>(), nb, gs.as<int32_t>(), ng, table.p,
                              mad, ck.p, cv.p, batch, cap, nullptr) == PIC_OK);
    // standalone re-rotation of [n][H][D] rows, shifts anywhere
    const int64_t n = rnd(0, 50);
    const int32_t H = (int32_t)rnd(1, 4);
    Buf k(n * H * row), dl(n * sizeof(int32_t));
    for (int64_t i = 0; i < n; ++i) dl.as<int32_t>()[i] = garbage(mad);
    EXPECT(pic_rerotate_keys(&m, k.p, k.p, n, H, dl.as<int32_t>(), table.p, mad, nullptr) == PIC_OK);
  }
}

// ---- composition of valid plans (every block moved), per block and with shared sources ----
void valid_compose() {
  for (int it = 0; it < 40; ++it) {
    const pic_dtype dt = rnd(0, 1) ? PIC_BF16 : PIC_F32;
    const int D = rnd(0, 1) ? 128 : 64, Hkv = (int)rnd(1, 2);
    pic_model m = model(1, Hkv, Hkv, D, dt);
    const int32_t n_pool = (int32_t)rnd(1, 6), batch = (int32_t)rnd(1, 4);
    std::vector<int32_t> off(n_pool), len(n_pool), cpos(n_pool, 0);
    int64_t pool_tokens = 0;
    for (int e = 0; e < n_pool; ++e) {
      len[e] = (int32_t)rnd(1, 200);
      off[e] = (int32_t)pool_tokens;
      pool_tokens += len[e];
    }
    std::vector<int32_t> n_items(batch), items;
    for (int b = 0; b < batch; ++b) {
      n_items[b] = (int32_t)rnd(0, 5);
      for (int k = 0; k < n_items[b]; ++k) items.push_back((int32_t)rnd(0, n_pool - 1));
    }
    std::vector<int32_t> ctx(batch);
    int32_t nb = 0;
    pic_plan_layout(batch, n_items.data(), items.empty() ? nullptr : items.data(), n_pool, off.data(), len.data(),
                    cpos.data(), pool_tokens, nullptr, 0, &nb, ctx.data());
    Buf blk((nb ? nb : 1) * sizeof(pic_block)), sorted((nb ? nb : 1) * sizeof(pic_block));
    EXPECT(pic_plan_layout(batch, n_items.data(), items.empty() ? nullptr : items.data(), n_pool, off.data(),
                           len.data(), cpos.data(), pool_tokens, blk.as<pic_block>(), nb, &nb, ctx.data()) == PIC_OK);
    int32_t cap = 1;
    for (int b = 0; b < batch; ++b) cap = ctx[b] > cap ? ctx[b] : cap;   // the tightest cache
    const int32_t mad = cap;
    const size_t row = (size_t)D * eb(m);
    Buf pk(Hkv * pool_tokens * row), pv(Hkv * pool_tokens * row);
    Buf ck((size_t)batch * Hkv * cap * row), cv((size_t)batch * Hkv * cap * row);
    Buf table(pic_rope_table_bytes(&m, mad));
    EXPECT(pic_compose(&m, pk.p, pv.p, pool_tokens, blk.as<pic_block>(), nb, table.p, mad, ck.p, cv.p, batch, cap,
                       nullptr) == PIC_OK);
    std::vector<int32_t> starts(nb + 1);
    int32_t ng = 0;
    EXPECT(pic_plan_shared(blk.as<pic_block>(), nb, sorted.as<pic_block>(), starts.data(), &ng) == PIC_OK);
    Buf gs((ng + 1) * sizeof(int32_t));
    std::memcpy(gs.p, starts.data(), (ng + 1) * sizeof(int32_t));
    EXPECT(pic_compose_shared(&m, pk.p, pv.p, pool_tokens, sorted.as<pic_block>(), nb, gs.as<int32_t>(), ng, table.p,
                              mad, ck.p, cv.p, batch, cap, nullptr) == PIC_OK);
  }
}

// A planted mistake: a cache allocated one row short of what its contract gives it, and a
// block that writes the last slot.  AddressSanitizer must stop the run here.
void planted_short_cache() {
  pic_model m = model(1, 1, 1, 128, PIC_BF16);
  const int32_t cap = 64, mad = 64;
  const size_t row = 256;
  Buf pk(64 * row), pv(64 * row), ck((cap - 1) * row), cv(cap * row), table(pic_rope_table_bytes(&m, mad));
  Buf blk(sizeof(pic_block));
  *blk.as<pic_block>() = pic_block{0, 0, 0, 64, 0};
  pic_compose(&m, pk.p, pv.p, 64, blk.as<pic_block>(), 1, table.p, mad, ck.p, cv.p, 1, cap, nullptr);
}

// ---- attention over garbage lengths, positions and maps ----
void fuzz_attention() {
  for (int it = 0; it < 40; ++it) {
    const bool bf16 = rnd(0, 3) != 0;
    const int D = rnd(0, 2) ? 128 : 64;
    const int Hkv = (int)rnd(1, 2), rep = bf16 ? (rnd(0, 4) ? (int)rnd(1, 7) : (int)rnd(17, 40)) : (int)rnd(1, 3);
    pic_model m = model((int)rnd(1, 2), Hkv * rep, Hkv, D, bf16 ? PIC_BF16 : PIC_F32);
    const int L = m.n_layers;
    const int32_t batch = (int32_t)rnd(1, 3), n_suf = (int32_t)rnd(1, 70), max_ctx = (int32_t)rnd(0, bf16 ? 3000 : 300);
    const int32_t cap = max_ctx + n_suf + (int32_t)rnd(0, 5);
    const size_t row = (size_t)D * eb(m);
    const int Hq = m.n_q_heads;
    Buf q((size_t)L * batch * n_suf * Hq * row), out((size_t)L * batch * n_suf * Hq * row);
    Buf ks((size_t)L * batch * n_suf * Hkv * row), vs((size_t)L * batch * n_suf * Hkv * row);
    Buf ck((size_t)L * batch * Hkv * cap * row), cv((size_t)L * batch * Hkv * cap * row);
    Buf ctx(batch * sizeof(int32_t));
    for (int b = 0; b < batch; ++b) ctx.as<int32_t>()[b] = garbage(max_ctx + 1);
    Buf ws(pic_prefill_workspace_bytes(&m, batch, n_suf, max_ctx));
    const long before = pic::emu::launches;
    EXPECT(pic_suffix_prefill_attn(&m, q.p, ks.p, vs.p, ck.p, cv.p, batch, cap, ctx.as<int32_t>(), max_ctx, n_suf,
                                   0.f, out.p, ws.n ? ws.p : nullptr, ws.n, nullptr) == PIC_OK);
    EXPECT(pic::emu::launches > before);
    // a workspace one byte short fails and launches nothing
    if (ws.n) {
      const long b2 = pic::emu::launches;
      EXPECT(pic_suffix_prefill_attn(&m, q.p, ks.p, vs.p, ck.p, cv.p, batch, cap, ctx.as<int32_t>(), max_ctx,
                                     n_suf, 0.f, out.p, ws.p, ws.n - 1, nullptr) == PIC_ERR_WORKSPACE);
      EXPECT(pic::emu::launches == b2);
    }
    // decode over garbage base lengths, every split count
    const int32_t step = (int32_t)rnd(0, 3);
    const int32_t dmax = cap - step - 1;
    if (dmax >= 0) {
      Buf dq((size_t)L * batch * Hq * row), dout((size_t)L * batch * Hq * row);
      Buf kn((size_t)L * batch * Hkv * row), vn((size_t)L * batch * Hkv * row);
      Buf base(batch * sizeof(int32_t));
      for (int b = 0; b < batch; ++b) base.as<int32_t>()[b] = garbage(dmax + 1);
      const int32_t splits = bf16 ? (int32_t)rnd(0, 9) : 0;
      Buf dws(pic_decode_workspace_bytes(&m, batch, dmax + step + 1, splits));
      if (bf16)
        EXPECT(pic_decode_attn(&m, dq.p, kn.p, vn.p, ck.p, cv.p, batch, cap, base.as<int32_t>(), step, dmax, 0.f,
                               splits, dout.p, dws.n ? dws.p : nullptr, dws.n, nullptr) == PIC_OK);
      if (bf16)   // the allocation-free entry point: partials in the scratch array
        EXPECT(pic_decode_attn_noalloc(&m, dq.p, kn.p, vn.p, ck.p, cv.p, batch, cap, base.as<int32_t>(), step, dmax,
                                       0.f, splits, dout.p, nullptr) == PIC_OK);
      if (!bf16)
        EXPECT(pic_decode_attn(&m, dq.p, kn.p, vn.p, ck.p, cv.p, batch, cap, base.as<int32_t>(), step, dmax, 0.f,
                               0, dout.p, nullptr, 0, nullptr) == PIC_OK);
    }
    // frontier: positions from the table, garbage entries clamped into [0, max_len)
    const int32_t max_len = cap - (int32_t)rnd(0, 3);
    Buf pos((size_t)batch * n_suf * sizeof(int32_t)), nv(batch * sizeof(int32_t));
    for (int i = 0; i < batch * n_suf; ++i) pos.as<int32_t>()[i] = garbage(max_len);
    for (int b = 0; b < batch; ++b) nv.as<int32_t>()[b] = garbage(n_suf + 1);
    Buf fws(pic_frontier_workspace_bytes(&m, batch, n_suf, max_len));
    EXPECT(pic_frontier_prefill_attn(&m, q.p, ks.p, vs.p, ck.p, cv.p, batch, cap, pos.as<int32_t>(), nv.as<int32_t>(),
                                     n_suf, max_len, 0.f, out.p, fws.n ? fws.p : nullptr, fws.n, nullptr) == PIC_OK);
    if (!bf16) continue;
    // zero-copy prefill: garbage slot and tile maps over a small pool
    const int64_t pool_tokens = rnd(1, 3000);
    const int32_t mad = (int32_t)rnd(0, 4000), map_cap = max_ctx + (int32_t)rnd(0, 70);
    Buf pk((size_t)L * Hkv * pool_tokens * row), pv((size_t)L * Hkv * pool_tokens * row);
    Buf table(pic_rope_table_bytes(&m, mad));
    Buf sm((size_t)batch * map_cap * sizeof(int32_t)), dm((size_t)batch * map_cap * sizeof(int32_t));
    const int32_t map_tiles = (map_cap + 63) / 64;
    Buf tm((size_t)batch * map_tiles * 2 * sizeof(int32_t));
    for (int64_t i = 0; i < (int64_t)batch * map_cap; ++i) {
      sm.as<int32_t>()[i] = garbage((int32_t)pool_tokens);
      dm.as<int32_t>()[i] = garbage(mad);
    }
    for (int64_t i = 0; i < (int64_t)batch * map_tiles; ++i) {
      tm.as<int32_t>()[2 * i] = garbage((int32_t)pool_tokens);
      tm.as<int32_t>()[2 * i + 1] = garbage(mad);
    }
    for (int with_map = 0; with_map < 2; ++with_map)
      EXPECT(pic_paged_prefill_attn(&m, pk.p, pv.p, pool_tokens, sm.as<int32_t>(), dm.as<int32_t>(), map_cap,
                                    with_map ? tm.as<int32_t>() : nullptr, table.p, mad, q.p, ks.p, vs.p, ck.p, cv.p,
                                    batch, cap, ctx.as<int32_t>(), max_ctx, n_suf, 0.f, out.p,
                                    ws.n ? ws.p : nullptr, ws.n, nullptr) == PIC_OK);
    // the non-run tiles of every layer composed ahead, then the per-layer form without the slot map
    EXPECT(pic_compose_tiles(&m, pk.p, pv.p, pool_tokens, sm.as<int32_t>(), dm.as<int32_t>(), map_cap,
                             tm.as<int32_t>(), table.p, mad, ctx.as<int32_t>(), max_ctx, ck.p, cv.p, batch, cap,
                             nullptr) == PIC_OK);
    EXPECT(pic_paged_prefill_attn(&m, pk.p, pv.p, pool_tokens, nullptr, nullptr, map_cap, tm.as<int32_t>(), table.p,
                                  mad, q.p, ks.p, vs.p, ck.p, cv.p, batch, cap, ctx.as<int32_t>(), max_ctx, n_suf,
                                  0.f, out.p, ws.n ? ws.p : nullptr, ws.n, nullptr) == PIC_OK);
    // the slot map from garbage blocks
    const int32_t nb = (int32_t)rnd(0, 30);
    Buf blk(nb * sizeof(pic_block));
    for (int i = 0; i < nb; ++i) {
      pic_block& b = blk.as<pic_block>()[i];
      b.request = garbage(batch);
      b.src_token = garbage((int32_t)pool_tokens);
      b.dst_slot = garbage(map_cap);
      b.n_tokens = garbage(65);
      b.delta = garbage(mad);
    }
    EXPECT(pic_build_slot_map(blk.as<pic_block>(), nb, batch, map_cap, sm.as<int32_t>(), dm.as<int32_t>(),
                              tm.as<int32_t>(), nullptr) == PIC_OK);
    // fused-RoPE prefill (table covering every position)
    const int32_t mad2 = max_ctx + n_suf;
    Buf table2(pic_rope_table_bytes(&m, mad2));
    EXPECT(pic_suffix_prefill_attn_rope(&m, q.p, ks.p, vs.p, ck.p, cv.p, batch, cap, ctx.as<int32_t>(), max_ctx,
                                        n_suf, table2.p, mad2, 0.f, out.p, ws.n ? ws.p : nullptr, ws.n,
                                        nullptr) == PIC_OK);
  }
}

// ---- argument checks: failures launch nothing ----
void argument_checks() {
  pic_model m = model(1, 32, 8, 128, PIC_BF16);
  Buf a(1 << 20);
  void* P = a.p;
  int32_t* I = a.as<int32_t>();
  const long before = pic::emu::launches;
  EXPECT(pic_suffix_prefill_attn(&m, P, P, P, P, P, 2, 600, I, 580, 64, 0.f, P, P, 1 << 20, nullptr) == PIC_ERR_CAPACITY);
  EXPECT(pic_suffix_prefill_attn(&m, P, P, P, P, P, 2, 600, nullptr, 500, 64, 0.f, P, P, 1 << 20, nullptr) ==
         PIC_ERR_INVALID_ARG);
  EXPECT(pic_decode_attn(&m, P, P, P, P, P, 2, 600, I, 100, 500, 0.f, 0, P, P, 1 << 20, nullptr) == PIC_ERR_CAPACITY);
  EXPECT(pic_decode_attn_noalloc(&m, P, P, P, P, P, 64, 700, I, 1, 600, 0.f, 64, P, nullptr) == PIC_ERR_WORKSPACE);
  EXPECT(pic_compose(&m, P, P, 100, nullptr, 4, P, 10, P, P, 2, 100, nullptr) == PIC_ERR_INVALID_ARG);
  EXPECT(pic_rerotate_keys(&m, static_cast<char*>(P) + 8, P, 4, 1, I, P, 10, nullptr) == PIC_ERR_MISALIGNED);
  pic_model bad = model(1, 30, 8, 128, PIC_BF16);
  EXPECT(pic_compose(&bad, P, P, 100, reinterpret_cast<pic_block*>(P), 4, P, 10, P, P, 2, 100, nullptr) ==
         PIC_ERR_INVALID_ARG);
  // tile composition: the tile map is required, and map_cap must cover max_ctx
  EXPECT(pic_compose_tiles(&m, P, P, 100, I, I, 64, nullptr, P, 10, I, 64, P, P, 2, 100, nullptr) ==
         PIC_ERR_INVALID_ARG);
  EXPECT(pic_compose_tiles(&m, P, P, 100, I, I, 32, I, P, 10, I, 64, P, P, 2, 100, nullptr) == PIC_ERR_CAPACITY);
  // the paged prefill without a slot map needs a tile map
  EXPECT(pic_paged_prefill_attn(&m, P, P, 100, nullptr, nullptr, 64, nullptr, P, 10, P, P, P, P, P, 2, 200, I, 64,
                                16, 0.f, P, P, 1 << 20, nullptr) == PIC_ERR_INVALID_ARG);
  EXPECT(pic_paged_prefill_attn(&m, P, P, 100, I, nullptr, 64, I, P, 10, P, P, P, P, P, 2, 200, I, 64, 16, 0.f, P,
                                P, 1 << 20, nullptr) == PIC_ERR_INVALID_ARG);
  EXPECT(pic::emu::launches == before);
}

}  // namespace

int main(int argc, char** argv) {
  if (argc > 1 && std::strcmp(argv[1], "--plant") == 0) {
    planted_short_cache();
    std::printf("planted mistake not caught\n");
    return 0;
  }
  const uint64_t seed = argc > 1 ? std::strtoull(argv[1], nullptr, 10) : 1;
  const int rounds = argc > 2 ? std::atoi(argv[2]) : 1;
  rng.seed(seed);
  for (int r = 0; r < rounds; ++r) {
    fuzz_planners();
    fuzz_compose();
    valid_compose();
    fuzz_attention();
  }
  argument_checks();
  if (failures) {
    std::printf("sanitizer driver: %d failures\n", failures);
    return 1;
  }
  std::printf("sanitizer driver: OK (%ld emulated launches)\n", pic::emu::launches);
  return 0;
}
