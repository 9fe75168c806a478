// RoPE relocation of cached keys and composition of document caches (Sec. 2, Eq. 3; App. C.1).
//
// A key compiled at position a moves to position b by R(b) R(a)^-1 = R(b - a): each pair
// turns by delta * theta_i.  Both positions run contiguously through a document, so one delta
// serves a whole gather block and its cos/sin row is loaded once per workgroup from a table
// built in float64 (one table, or one per layer for a layer-specific transform).  Values are
// copied unchanged.
//
// Memory traffic is the whole cost (6 flops per 2 elements), so every access is a 16-byte
// vector and a row of D elements is split across lanes such that the two members of every
// rotated pair sit in the same lane: for the rotate-half pairing (x_i, x_{i+D/2}) a lane owns
// element chunk [c, c + VEC) of both halves; for the interleaved pairing (x_2i, x_2i+1) it
// owns the 2 VEC consecutive elements of pairs [c, c + VEC).  bf16 output rows are stored
// non-temporally (written once; the caches stay with the pool rows, which several requests read).
#include "pic_bounds.h"
#include "pic_internal.h"

namespace pic {
namespace {

struct InvFreq {
  double v[64];
};

__global__ void rope_table_kernel(InvFreq invf, int half, int32_t max_abs_delta, float2* table) {
  const int64_t n = (int64_t)(max_abs_delta + 1) * half;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t d = idx / half;
    const int i = (int)(idx - d * half);
    const double ang = (double)d * invf.v[i];
    table[idx] = make_float2((float)cos(ang), (float)sin(ang));
  }
}

template <typename T>
struct Vec16;  // 16 bytes of T as float lanes

template <>
struct Vec16<float> {
  static constexpr int N = 4;
  __device__ static void load(const float* p, float (&x)[4]) {
    const float4 v = *reinterpret_cast<const float4*>(p);
    x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
  }
  __device__ static void store(float* p, const float (&x)[4]) {
    *reinterpret_cast<float4*>(p) = make_float4(x[0], x[1], x[2], x[3]);
  }
  __device__ static void load_nt(const float* p, float (&x)[4]) {
    typedef uint32_t u32x4_nt __attribute__((ext_vector_type(4)));
    const u32x4_nt v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(p));
    x[0] = __uint_as_float(v.x); x[1] = __uint_as_float(v.y); x[2] = __uint_as_float(v.z); x[3] = __uint_as_float(v.w);
  }
  __device__ static uint4 load_raw(const float* p) { return *reinterpret_cast<const uint4*>(p); }
  __device__ static void widen(uint4 v, float (&x)[4]) {
    x[0] = __uint_as_float(v.x); x[1] = __uint_as_float(v.y); x[2] = __uint_as_float(v.z); x[3] = __uint_as_float(v.w);
  }
  __device__ static void store_raw(float* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }
};

template <>
struct Vec16<bf16_t> {
  static constexpr int N = 8;
  __device__ static void load(const bf16_t* p, float (&x)[8]) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  // Non-temporal: an output row is written once and not read again by the launch; streaming
  // it past the caches keeps them for the pool rows that other requests' blocks read again
  // (the loads stay ordinary).
  __device__ static void store(bf16_t* p, const float (&x)[8]) {
    typedef uint32_t u32x4_nt __attribute__((ext_vector_type(4)));
    const u32x4_nt v = {pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                        pack_bf16x2(x[6], x[7])};
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4_nt*>(p));
  }
  // Non-temporal: a row read once by a streaming launch (the in-place re-rotation)
  __device__ static void load_nt(const bf16_t* p, float (&x)[8]) {
    typedef uint32_t u32x4_nt __attribute__((ext_vector_type(4)));
    const u32x4_nt v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_nt*>(p));
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  __device__ static uint4 load_raw(const bf16_t* p) { return *reinterpret_cast<const uint4*>(p); }
  __device__ static void widen(uint4 v, float (&x)[8]) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  __device__ static void store_raw(bf16_t* p, uint4 w) {
    typedef uint32_t u32x4_nt __attribute__((ext_vector_type(4)));
    const u32x4_nt v = {w.x, w.y, w.z, w.w};
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4_nt*>(p));
  }
};

// cos/sin of the lane's VEC frequencies for shift delta (|delta| already within the table).
template <int VEC, int HALF>
__device__ __forceinline__ void load_cs(const float2* table, int32_t delta, int c0, float (&cs)[VEC],
                                        float (&sn)[VEC]) {
  const int32_t ad = delta < 0 ? -delta : delta;
  const float2* row = table + (int64_t)ad * HALF + c0;
#pragma unroll
  for (int i = 0; i < VEC; ++i) {
    const float2 t = row[i];
    cs[i] = t.x;
    sn[i] = delta < 0 ? -t.y : t.y;
  }
}

__device__ __forceinline__ void turn(float& a, float& b, float c, float s) {
  const float x = a, y = b;
  a = fmaf(x, c, -(y * s));
  b = fmaf(x, s, y * c);
}

// Pair i of the lane's VEC pairs turned by (cs[i], sn[i]).  IL = false: pair i is
// (x1[i], x2[i]) (rotate-half chunks); IL = true: x1, x2 are consecutive elements and pair i
// is elements (2i, 2i + 1) of their concatenation.
template <int VEC, bool IL>
__device__ __forceinline__ void rotate(float (&x1)[VEC], float (&x2)[VEC], const float (&cs)[VEC],
                                       const float (&sn)[VEC]) {
#pragma unroll
  for (int i = 0; i < VEC; ++i) {
    if constexpr (IL) {
      float* x = i < VEC / 2 ? x1 : x2;
      const int e = 2 * (i % (VEC / 2));
      turn(x[e], x[e + 1], cs[i], sn[i]);
    } else {
      turn(x1[i], x2[i], cs[i], sn[i]);
    }
  }
}

// Element offsets of the lane's two 16-byte vectors for pair chunk c0 (see rotate()).
template <int VEC, int HALF, bool IL>
__device__ __forceinline__ int off1(int c0) { return IL ? 2 * c0 : c0; }
template <int VEC, int HALF, bool IL>
__device__ __forceinline__ int off2(int c0) { return IL ? 2 * c0 + VEC : HALF + c0; }

// grid (n_blocks, Hkv, L), 256 threads.  One workgroup moves one gather block of one kv head.
// Layer l reads its cos/sin from table + l * table_stride (0: one table for all layers).
template <typename T, int HD, bool IL>
__global__ void __launch_bounds__(256) compose_kernel(
    const T* __restrict__ pool_k, const T* __restrict__ pool_v, int64_t pool_tokens,
    const pic_block* __restrict__ blocks, const float2* __restrict__ table, int64_t table_stride,
    int32_t max_abs_delta, T* __restrict__ cache_k, T* __restrict__ cache_v, int32_t batch,
    int32_t cache_cap) {
  using V = Vec16<T>;
  constexpr int VEC = V::N;
  constexpr int HALF = HD / 2;
  constexpr int LPR = HALF / VEC;          // lanes per row
  constexpr int RPP = 256 / LPR;           // rows per pass
  constexpr int PASSES = (PIC_BLOCK_TOKENS + RPP - 1) / RPP;

  const pic_block blk = blocks[blockIdx.x];
  if (!block_ok(blk, batch, pool_tokens, cache_cap, max_abs_delta)) return;

  const int h = blockIdx.y, l = blockIdx.z, Hkv = gridDim.y;
  const int j = threadIdx.x % LPR, r0 = threadIdx.x / LPR;
  const int c0 = j * VEC;

  float cs[VEC], sn[VEC];
  load_cs<VEC, HALF>(table + l * table_stride, blk.delta, c0, cs, sn);
  const int o1 = off1<VEC, HALF, IL>(c0), o2 = off2<VEC, HALF, IL>(c0);

  const int64_t src_row0 = ((int64_t)l * Hkv + h) * pool_tokens + blk.src_token;
  const int64_t dst_row0 = (((int64_t)l * batch + blk.request) * Hkv + h) * cache_cap + blk.dst_slot;

  float k1[PASSES][VEC], k2[PASSES][VEC], v1[PASSES][VEC], v2[PASSES][VEC];
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int t = r0 + p * RPP;
    if (t < blk.n_tokens) {
      const int64_t s = (src_row0 + t) * HD;
      V::load(pool_k + s + o1, k1[p]);
      V::load(pool_k + s + o2, k2[p]);
      V::load(pool_v + s + o1, v1[p]);
      V::load(pool_v + s + o2, v2[p]);
    }
  }
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int t = r0 + p * RPP;
    if (t < blk.n_tokens) {
      rotate<VEC, IL>(k1[p], k2[p], cs, sn);
      const int64_t d = (dst_row0 + t) * HD;
      V::store(cache_k + d + o1, k1[p]);
      V::store(cache_k + d + o2, k2[p]);
      V::store(cache_v + d + o1, v1[p]);
      V::store(cache_v + d + o2, v2[p]);
    }
  }
}

// grid (n_groups, Hkv, L), 256 threads.  Composition with shared sources: blocks is sorted so
// that the blocks of group g, [group_start[g], group_start[g + 1]), all read the same pool run
// (the first block's src_token and n_tokens: one document chunk placed in several requests).
// One workgroup reads that run of one kv head once and writes it to every block of its group,
// each with its own shift, in exactly the arithmetic of compose_kernel.  A block that does not
// share its group's source, or whose request, destination or delta is out of range, is skipped.
template <typename T, int HD, bool IL>
__global__ void __launch_bounds__(256) compose_shared_kernel(
    const T* __restrict__ pool_k, const T* __restrict__ pool_v, int64_t pool_tokens,
    const pic_block* __restrict__ blocks, const int32_t* __restrict__ group_start, int32_t n_blocks,
    const float2* __restrict__ table, int64_t table_stride, int32_t max_abs_delta,
    T* __restrict__ cache_k, T* __restrict__ cache_v, int32_t batch, int32_t cache_cap) {
  using V = Vec16<T>;
  constexpr int VEC = V::N;
  constexpr int HALF = HD / 2;
  constexpr int LPR = HALF / VEC;          // lanes per row
  constexpr int RPP = 256 / LPR;           // rows per pass
  constexpr int PASSES = (PIC_BLOCK_TOKENS + RPP - 1) / RPP;

  int32_t g0, g1;
  group_range(group_start[blockIdx.x], group_start[blockIdx.x + 1], n_blocks, g0, g1);
  if (g0 >= g1) return;
  const pic_block src = blocks[g0];
  if (!block_source_ok(src, pool_tokens)) return;

  const int h = blockIdx.y, l = blockIdx.z, Hkv = gridDim.y;
  const int j = threadIdx.x % LPR, r0 = threadIdx.x / LPR;
  const int c0 = j * VEC;
  const int o1 = off1<VEC, HALF, IL>(c0), o2 = off2<VEC, HALF, IL>(c0);
  const float2* ltable = table + l * table_stride;
  const int64_t src_row0 = ((int64_t)l * Hkv + h) * pool_tokens + src.src_token;

  // the run's rows, held as loaded (16 bytes per vector; keys widened per destination)
  uint4 k1[PASSES], k2[PASSES], v1[PASSES], v2[PASSES];
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int t = r0 + p * RPP;
    if (t < src.n_tokens) {
      const int64_t s = (src_row0 + t) * HD;
      k1[p] = V::load_raw(pool_k + s + o1);
      k2[p] = V::load_raw(pool_k + s + o2);
      v1[p] = V::load_raw(pool_v + s + o1);
      v2[p] = V::load_raw(pool_v + s + o2);
    }
  }
  // The next block's descriptor and cos/sin row are read while this block is stored, so a
  // destination costs no memory round trip of its own.
  auto cs_of = [&](const pic_block& b, float (&cs)[VEC], float (&sn)[VEC]) {
    // (an out-of-range block is skipped below; clamp for the read)
    load_cs<VEC, HALF>(ltable, clamp_delta(b.delta, max_abs_delta), c0, cs, sn);
  };
  pic_block nxt = src;
  float ncs[VEC], nsn[VEC];
  cs_of(nxt, ncs, nsn);
  for (int i = g0; i < g1; ++i) {
    const pic_block blk = nxt;
    float cs[VEC], sn[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      cs[e] = ncs[e];
      sn[e] = nsn[e];
    }
    if (i + 1 < g1) {
      nxt = blocks[i + 1];
      cs_of(nxt, ncs, nsn);
    }
    if (!shared_block_ok(blk, src, batch, cache_cap, max_abs_delta)) continue;
    const int64_t dst_row0 = (((int64_t)l * batch + blk.request) * Hkv + h) * cache_cap + blk.dst_slot;
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int t = r0 + p * RPP;
      if (t < blk.n_tokens) {
        float x1[VEC], x2[VEC];
        V::widen(k1[p], x1);
        V::widen(k2[p], x2);
        rotate<VEC, IL>(x1, x2, cs, sn);
        const int64_t d = (dst_row0 + t) * HD;
        V::store(cache_k + d + o1, x1);
        V::store(cache_k + d + o2, x2);
        V::store_raw(cache_v + d + o1, v1[p]);
        V::store_raw(cache_v + d + o2, v2[p]);
      }
    }
  }
}

// compose_shared_kernel for interleaved pairs on bf16 rows of 128 elements: a pair (x_2i,
// x_2i+1) sits inside one 16-byte chunk, so 16 lanes cover a row chunk by chunk and every load
// and store instruction of a wave moves 4 whole rows (1 KB contiguous).  (The generic layout,
// whose lanes hold pairs of neighbouring chunks, leaves every store instruction writing half of
// each 32-byte sector.)  Same arithmetic as compose_kernel: bit-identical results.
__global__ void __launch_bounds__(256) compose_shared_il_rows_kernel(
    const bf16_t* __restrict__ pool_k, const bf16_t* __restrict__ pool_v, int64_t pool_tokens,
    const pic_block* __restrict__ blocks, const int32_t* __restrict__ group_start, int32_t n_blocks,
    const float2* __restrict__ table, int64_t table_stride, int32_t max_abs_delta,
    bf16_t* __restrict__ cache_k, bf16_t* __restrict__ cache_v, int32_t batch, int32_t cache_cap) {
  using V = Vec16<bf16_t>;
  constexpr int HD = 128, HALF = 64;
  constexpr int RPP = 16;                                   // rows per pass
  constexpr int PASSES = PIC_BLOCK_TOKENS / RPP;

  int32_t g0, g1;
  group_range(group_start[blockIdx.x], group_start[blockIdx.x + 1], n_blocks, g0, g1);
  if (g0 >= g1) return;
  const pic_block src = blocks[g0];
  if (!block_source_ok(src, pool_tokens)) return;

  const int h = blockIdx.y, l = blockIdx.z, Hkv = gridDim.y;
  const int j = threadIdx.x & 15, r0 = threadIdx.x >> 4;   // chunk j = pairs 4 j .. 4 j + 3
  const float2* ltable = table + l * table_stride;
  const int64_t src_row0 = ((int64_t)l * Hkv + h) * pool_tokens + src.src_token;

  uint4 k[PASSES], v[PASSES];
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int t = r0 + p * RPP;
    if (t < src.n_tokens) {
      const int64_t sr = (src_row0 + t) * HD + 8 * j;
      k[p] = V::load_raw(pool_k + sr);
      v[p] = V::load_raw(pool_v + sr);
    }
  }
  auto cs_of = [&](const pic_block& b, float (&cs)[4], float (&sn)[4]) {
    const int32_t d = clamp_delta(b.delta, max_abs_delta);
    const int32_t ad = d < 0 ? -d : d;
    const float2* row = ltable + (int64_t)ad * HALF + 4 * j;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float2 t = row[i];
      cs[i] = t.x;
      sn[i] = d < 0 ? -t.y : t.y;
    }
  };
  pic_block nxt = src;
  float ncs[4], nsn[4];
  cs_of(nxt, ncs, nsn);
  for (int i = g0; i < g1; ++i) {
    const pic_block blk = nxt;
    float cs[4], sn[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      cs[e] = ncs[e];
      sn[e] = nsn[e];
    }
    if (i + 1 < g1) {
      nxt = blocks[i + 1];
      cs_of(nxt, ncs, nsn);
    }
    if (!shared_block_ok(blk, src, batch, cache_cap, max_abs_delta)) continue;
    const int64_t dst_row0 = (((int64_t)l * batch + blk.request) * Hkv + h) * cache_cap + blk.dst_slot;
#pragma unroll
    for (int p = 0; p < PASSES; ++p) {
      const int t = r0 + p * RPP;
      if (t < blk.n_tokens) {
        float x[8];
        V::widen(k[p], x);
#pragma unroll
        for (int q = 0; q < 4; ++q) turn(x[2 * q], x[2 * q + 1], cs[q], sn[q]);
        const int64_t dr = (dst_row0 + t) * HD + 8 * j;
        V::store(cache_k + dr, x);
        V::store_raw(cache_v + dr, v[p]);
      }
    }
  }
}

// grid (batch * map_tiles, Hkv, L), 256 threads.  Zero-copy prefill with a tile map: the
// prefill reads a context tile straight from the pool when it is one pool run under one shift
// (tile map entry (src, delta) with src >= 0, the run inside the pool, |delta| within the
// table and the tile inside the context: the test the prefill applies); every other context
// tile is composed here into the cache from the slot map, row by row, with compose_kernel's
// arithmetic, so the prefill can read it from there.  Whole-run tiles are left alone.
template <typename T, int HD, bool IL>
__global__ void __launch_bounds__(256) compose_tiles_kernel(
    const T* __restrict__ pool_k, const T* __restrict__ pool_v, int64_t pool_tokens,
    const int32_t* __restrict__ smap, const int32_t* __restrict__ dmap, int32_t map_cap,
    const int32_t* __restrict__ tmap, int32_t map_tiles, const int32_t* __restrict__ ctx_len,
    int32_t max_ctx, const float2* __restrict__ table, int64_t table_stride,
    int32_t max_abs_delta, T* __restrict__ cache_k, T* __restrict__ cache_v, int32_t batch,
    int32_t cache_cap) {
  using V = Vec16<T>;
  constexpr int VEC = V::N;
  constexpr int HALF = HD / 2;
  constexpr int LPR = HALF / VEC;
  constexpr int RPP = 256 / LPR;
  constexpr int PASSES = (PIC_BLOCK_TOKENS + RPP - 1) / RPP;

  const int b = blockIdx.x / map_tiles, tile = blockIdx.x - b * map_tiles;
  const int ctx = clamp_len(ctx_len[b], max_ctx);
  const int s0 = tile * PIC_BLOCK_TOKENS;
  if (s0 >= ctx) return;
  const int32_t src = tmap[((int64_t)b * map_tiles + tile) * 2];
  const int32_t dl = tmap[((int64_t)b * map_tiles + tile) * 2 + 1];
  if (tile_run_ok(src, dl, s0, ctx, pool_tokens, max_abs_delta))
    return;   // a whole run: the prefill reads it from the pool

  const int h = blockIdx.y, l = blockIdx.z, Hkv = gridDim.y;
  const int j = threadIdx.x % LPR, r0 = threadIdx.x / LPR;
  const int c0 = j * VEC;
  const int o1 = off1<VEC, HALF, IL>(c0), o2 = off2<VEC, HALF, IL>(c0);
  const float2* ltable = table + l * table_stride;
  const int64_t pool0 = ((int64_t)l * Hkv + h) * pool_tokens;
  const int64_t dst0 = (((int64_t)l * batch + b) * Hkv + h) * cache_cap;
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    const int slot = s0 + r0 + p * RPP;
    if (slot >= ctx) continue;
    const int32_t st = clamp_pool_token(smap[(int64_t)b * map_cap + slot], pool_tokens);
    const int32_t d = clamp_delta(dmap[(int64_t)b * map_cap + slot], max_abs_delta);
    float cs[VEC], sn[VEC], x1[VEC], x2[VEC];
    load_cs<VEC, HALF>(ltable, d, c0, cs, sn);
    const int64_t sr = (pool0 + st) * HD, dr = (dst0 + slot) * HD;
    V::load(pool_k + sr + o1, x1);
    V::load(pool_k + sr + o2, x2);
    const uint4 w1 = V::load_raw(pool_v + sr + o1), w2 = V::load_raw(pool_v + sr + o2);
    rotate<VEC, IL>(x1, x2, cs, sn);
    V::store(cache_k + dr + o1, x1);
    V::store(cache_k + dr + o2, x2);
    V::store_raw(cache_v + dr + o1, w1);
    V::store_raw(cache_v + dr + o2, w2);
  }
}

// rows [n_tokens][n_heads][HD]; one (row, pair chunk) item per thread, LPR items per row, so a
// wave's two 16-byte loads cover 64 / LPR whole rows.  The grid covers every item in one pass
// for up to 2^31 items (a streaming launch runs fastest with one item per thread), with a
// grid-stride loop beyond; rows are read and written non-temporally.  kWide: 64-bit item
// indices (2^32 items or more), else 32-bit index arithmetic.
template <typename T, int HD, bool IL, bool kWide>
__global__ void __launch_bounds__(256) rerotate_kernel(const T* k_in, T* k_out, int64_t n_rows,
                                                       int32_t n_heads, const int32_t* __restrict__ delta,
                                                       const float2* __restrict__ table,
                                                       int32_t max_abs_delta) {
  using V = Vec16<T>;
  constexpr int VEC = V::N;
  constexpr int HALF = HD / 2;
  constexpr int LPR = HALF / VEC;
  const int64_t n_items = n_rows * LPR;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n_items;
       idx += (int64_t)gridDim.x * blockDim.x) {
    int64_t row, token;
    if constexpr (kWide) {
      row = idx / LPR;
      token = row / n_heads;
    } else {
      const uint32_t r32 = (uint32_t)idx / LPR;
      row = r32;
      token = r32 / (uint32_t)n_heads;
    }
    const int c0 = (int)(idx - row * LPR) * VEC;
    const int32_t d = clamp_delta(delta[token], max_abs_delta);
    float cs[VEC], sn[VEC], x1[VEC], x2[VEC];
    const int o1 = off1<VEC, HALF, IL>(c0), o2 = off2<VEC, HALF, IL>(c0);
    V::load_nt(k_in + row * HD + o1, x1);
    V::load_nt(k_in + row * HD + o2, x2);
    load_cs<VEC, HALF>(table, d, c0, cs, sn);
    rotate<VEC, IL>(x1, x2, cs, sn);
    V::store(k_out + row * HD + o1, x1);
    V::store(k_out + row * HD + o2, x2);
  }
}

// New rows [L][B][n_new][Hkv][HD] -> cache slots base[b] + offset + i.  16 bytes per thread.
template <typename T, int HD>
__global__ void __launch_bounds__(256) append_kernel(const T* __restrict__ k_new, const T* __restrict__ v_new,
                                                     T* __restrict__ cache_k, T* __restrict__ cache_v,
                                                     int n_kv_heads, int32_t batch, int32_t cache_cap,
                                                     RowPos pos, int32_t n_new, int64_t n_rows) {
  constexpr int CPR = HD * sizeof(T) / 16;  // 16-byte chunks per row
  const int64_t n_items = n_rows * CPR;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n_items;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = idx / CPR;
    const int c = (int)(idx - row * CPR);
    // row = ((l * B + b) * n_new + i) * Hkv + h
    const int h = (int)(row % n_kv_heads);
    const int64_t r1 = row / n_kv_heads;
    const int i = (int)(r1 % n_new);
    const int64_t lb = r1 / n_new;  // l * B + b
    const int b = (int)(lb % batch);
    const int64_t slot = pos(b, i);
    if (slot < 0 || slot >= cache_cap) continue;
    const int64_t dst = ((lb * n_kv_heads + h) * cache_cap + slot) * HD;
    const uint4* sk = reinterpret_cast<const uint4*>(k_new + row * HD) + c;
    const uint4* sv = reinterpret_cast<const uint4*>(v_new + row * HD) + c;
    reinterpret_cast<uint4*>(cache_k + dst)[c] = *sk;
    reinterpret_cast<uint4*>(cache_v + dst)[c] = *sv;
  }
}

// append_kernel for bf16 rows whose keys are turned to their slot's position on the way, with
// rerotate_kernel's arithmetic (table block of layer l at table + l * table_stride); one
// (row, chunk pair) per thread, values copied as they are.
template <int HD, bool IL>
__global__ void __launch_bounds__(256) append_rope_kernel(const bf16_t* __restrict__ k_new,
                                                          const bf16_t* __restrict__ v_new,
                                                          bf16_t* __restrict__ cache_k, bf16_t* __restrict__ cache_v,
                                                          int n_kv_heads, int32_t batch, int32_t cache_cap,
                                                          RowPos pos, int32_t n_new, int64_t n_rows,
                                                          const float2* __restrict__ table, int64_t table_stride,
                                                          int32_t max_abs_delta) {
  using V = Vec16<bf16_t>;
  constexpr int VEC = V::N;
  constexpr int HALF = HD / 2;
  constexpr int LPR = HALF / VEC;
  const int64_t n_items = n_rows * LPR;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n_items;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = idx / LPR;
    const int c0 = (int)(idx - row * LPR) * VEC;
    // row = ((l * B + b) * n_new + i) * Hkv + h
    const int h = (int)(row % n_kv_heads);
    const int64_t r1 = row / n_kv_heads;
    const int i = (int)(r1 % n_new);
    const int64_t lb = r1 / n_new;  // l * B + b
    const int b = (int)(lb % batch);
    const int l = (int)(lb / batch);
    const int64_t slot = pos(b, i);
    if (slot < 0 || slot >= cache_cap) continue;
    float cs[VEC], sn[VEC], x1[VEC], x2[VEC];
    load_cs<VEC, HALF>(table + l * table_stride, (int32_t)(slot < max_abs_delta ? slot : max_abs_delta), c0, cs, sn);
    const int o1 = off1<VEC, HALF, IL>(c0), o2 = off2<VEC, HALF, IL>(c0);
    V::load(k_new + row * HD + o1, x1);
    V::load(k_new + row * HD + o2, x2);
    rotate<VEC, IL>(x1, x2, cs, sn);
    const int64_t dst = ((lb * n_kv_heads + h) * cache_cap + slot) * HD;
    V::store(cache_k + dst + o1, x1);
    V::store(cache_k + dst + o2, x2);
    V::store_raw(cache_v + dst + o1, V::load_raw(v_new + row * HD + o1));
    V::store_raw(cache_v + dst + o2, V::load_raw(v_new + row * HD + o2));
  }
}

int grid_for(int64_t items, int threads) {
  int64_t g = (items + threads - 1) / threads;
  if (g < 1) g = 1;
  if (g > 65536) g = 65536;
  return (int)g;
}

}  // namespace

hipError_t launch_rope_table(const double* inv_freq_host, int half, int32_t max_abs_delta,
                             float2* table, hipStream_t stream) {
  InvFreq f;
  for (int i = 0; i < 64; ++i) f.v[i] = i < half ? inv_freq_host[i] : 0.0;
  const int64_t n = (int64_t)(max_abs_delta + 1) * half;
  hipLaunchKernelGGL(rope_table_kernel, dim3(grid_for(n, 256)), dim3(256), 0, stream, f, half,
                     max_abs_delta, table);
  return hipGetLastError();
}

#define PIC_DISPATCH_TD(dt, hd, KERNEL_CALL)                                      \
  do {                                                                            \
    if ((dt) == PIC_F32 && (hd) == 64) { using T = float; constexpr int HD = 64; KERNEL_CALL; } \
    else if ((dt) == PIC_F32) { using T = float; constexpr int HD = 128; KERNEL_CALL; }         \
    else if ((hd) == 64) { using T = bf16_t; constexpr int HD = 64; KERNEL_CALL; }               \
    else { using T = bf16_t; constexpr int HD = 128; KERNEL_CALL; }                              \
  } while (0)

hipError_t launch_rerotate(pic_dtype dt, int head_dim, bool interleaved, const void* k_in,
                           void* k_out, int64_t n_rows, int32_t n_heads, const int32_t* delta,
                           const float2* table, int32_t max_abs_delta, hipStream_t stream) {
  if (n_rows == 0) return hipSuccess;
  PIC_DISPATCH_TD(dt, head_dim, {
    constexpr int LPR = HD / 2 / (16 / (int)sizeof(T));
    const int64_t items = n_rows * LPR;
    const int64_t blocks = (items + 255) / 256;
    const dim3 grid((unsigned)(blocks < (1 << 23) ? blocks : (1 << 23)));   // one pass up to 2^31 items
    const bool wide = items >= (int64_t(1) << 32);
    if (interleaved && wide)
      hipLaunchKernelGGL((rerotate_kernel<T, HD, true, true>), grid, dim3(256), 0, stream, (const T*)k_in,
                         (T*)k_out, n_rows, n_heads, delta, table, max_abs_delta);
    else if (interleaved)
      hipLaunchKernelGGL((rerotate_kernel<T, HD, true, false>), grid, dim3(256), 0, stream, (const T*)k_in,
                         (T*)k_out, n_rows, n_heads, delta, table, max_abs_delta);
    else if (wide)
      hipLaunchKernelGGL((rerotate_kernel<T, HD, false, true>), grid, dim3(256), 0, stream, (const T*)k_in,
                         (T*)k_out, n_rows, n_heads, delta, table, max_abs_delta);
    else
      hipLaunchKernelGGL((rerotate_kernel<T, HD, false, false>), grid, dim3(256), 0, stream, (const T*)k_in,
                         (T*)k_out, n_rows, n_heads, delta, table, max_abs_delta);
  });
  return hipGetLastError();
}

hipError_t launch_compose(pic_dtype dt, int head_dim, bool interleaved, int n_layers,
                          int n_kv_heads, const void* pool_k, const void* pool_v,
                          int64_t pool_tokens, const pic_block* blocks, int32_t n_blocks,
                          const float2* table, int64_t table_stride, int32_t max_abs_delta,
                          void* cache_k, void* cache_v, int32_t batch, int32_t cache_cap,
                          hipStream_t stream) {
  if (n_blocks == 0 || n_layers == 0) return hipSuccess;
  const dim3 grid(n_blocks, n_kv_heads, n_layers);
  PIC_DISPATCH_TD(dt, head_dim, {
    if (interleaved)
      hipLaunchKernelGGL((compose_kernel<T, HD, true>), grid, dim3(256), 0, stream,
                         (const T*)pool_k, (const T*)pool_v, pool_tokens, blocks, table,
                         table_stride, max_abs_delta, (T*)cache_k, (T*)cache_v, batch, cache_cap);
    else
      hipLaunchKernelGGL((compose_kernel<T, HD, false>), grid, dim3(256), 0, stream,
                         (const T*)pool_k, (const T*)pool_v, pool_tokens, blocks, table,
                         table_stride, max_abs_delta, (T*)cache_k, (T*)cache_v, batch, cache_cap);
  });
  return hipGetLastError();
}

hipError_t launch_compose_shared(pic_dtype dt, int head_dim, bool interleaved, int n_layers,
                                 int n_kv_heads, const void* pool_k, const void* pool_v,
                                 int64_t pool_tokens, const pic_block* blocks, int32_t n_blocks,
                                 const int32_t* group_start, int32_t n_groups, const float2* table,
                                 int64_t table_stride, int32_t max_abs_delta, void* cache_k,
                                 void* cache_v, int32_t batch, int32_t cache_cap, hipStream_t stream) {
  if (n_groups == 0 || n_layers == 0) return hipSuccess;
  const dim3 grid(n_groups, n_kv_heads, n_layers);
  if (interleaved && dt == PIC_BF16 && head_dim == 128) {   // whole-row moves
    hipLaunchKernelGGL(compose_shared_il_rows_kernel, grid, dim3(256), 0, stream, (const bf16_t*)pool_k,
                       (const bf16_t*)pool_v, pool_tokens, blocks, group_start, n_blocks, table, table_stride,
                       max_abs_delta, (bf16_t*)cache_k, (bf16_t*)cache_v, batch, cache_cap);
    return hipGetLastError();
  }
  PIC_DISPATCH_TD(dt, head_dim, {
    if (interleaved)
      hipLaunchKernelGGL((compose_shared_kernel<T, HD, true>), grid, dim3(256), 0, stream,
                         (const T*)pool_k, (const T*)pool_v, pool_tokens, blocks, group_start,
                         n_blocks, table, table_stride, max_abs_delta, (T*)cache_k, (T*)cache_v,
                         batch, cache_cap);
    else
      hipLaunchKernelGGL((compose_shared_kernel<T, HD, false>), grid, dim3(256), 0, stream,
                         (const T*)pool_k, (const T*)pool_v, pool_tokens, blocks, group_start,
                         n_blocks, table, table_stride, max_abs_delta, (T*)cache_k, (T*)cache_v,
                         batch, cache_cap);
  });
  return hipGetLastError();
}

hipError_t launch_compose_tiles(bool interleaved, int head_dim, int n_layers, int n_kv_heads, const bf16_t* pool_k,
                                const bf16_t* pool_v, int64_t pool_tokens, const int32_t* smap,
                                const int32_t* dmap, int32_t map_cap, const int32_t* tmap,
                                int32_t map_tiles, const int32_t* ctx_len, int32_t max_ctx,
                                const float2* table, int64_t table_stride, int32_t max_abs_delta,
                                bf16_t* cache_k, bf16_t* cache_v, int32_t batch, int32_t cache_cap,
                                hipStream_t stream) {
  if ((int64_t)batch * map_tiles == 0 || n_layers == 0) return hipSuccess;
  const dim3 grid((unsigned)((int64_t)batch * map_tiles), n_kv_heads, n_layers);
#define PIC_COMPOSE_TILES(HD, IL)                                                                          \
  hipLaunchKernelGGL((compose_tiles_kernel<bf16_t, HD, IL>), grid, dim3(256), 0, stream, pool_k, pool_v,    \
                     pool_tokens, smap, dmap, map_cap, tmap, map_tiles, ctx_len, max_ctx, table,            \
                     table_stride, max_abs_delta, cache_k, cache_v, batch, cache_cap)
  if (head_dim == 64 && interleaved) PIC_COMPOSE_TILES(64, true);
  else if (head_dim == 64) PIC_COMPOSE_TILES(64, false);
  else if (head_dim == 128 && interleaved) PIC_COMPOSE_TILES(128, true);
  else if (head_dim == 128) PIC_COMPOSE_TILES(128, false);
  else return hipErrorInvalidValue;
#undef PIC_COMPOSE_TILES
  return hipGetLastError();
}

hipError_t launch_append(pic_dtype dt, int head_dim, int n_layers, int n_kv_heads,
                         const void* k_new, const void* v_new, void* cache_k, void* cache_v,
                         int32_t batch, int32_t cache_cap, const RowPos& pos, int32_t n_new,
                         hipStream_t stream) {
  const int64_t n_rows = (int64_t)n_layers * batch * n_new * n_kv_heads;
  if (n_rows == 0) return hipSuccess;
  PIC_DISPATCH_TD(dt, head_dim, {
    constexpr int CPR = HD * (int)sizeof(T) / 16;
    hipLaunchKernelGGL((append_kernel<T, HD>), dim3(grid_for(n_rows * CPR, 256)), dim3(256), 0,
                       stream, (const T*)k_new, (const T*)v_new, (T*)cache_k, (T*)cache_v,
                       n_kv_heads, batch, cache_cap, pos, n_new, n_rows);
  });
  return hipGetLastError();
}

hipError_t launch_append_rope(int head_dim, bool interleaved, int n_layers, int n_kv_heads,
                              const bf16_t* k_new, const bf16_t* v_new, bf16_t* cache_k,
                              bf16_t* cache_v, int32_t batch, int32_t cache_cap, const RowPos& pos,
                              int32_t n_new, const float2* table, int64_t table_stride,
                              int32_t max_abs_delta, hipStream_t stream) {
  const int64_t n_rows = (int64_t)n_layers * batch * n_new * n_kv_heads;
  if (n_rows == 0) return hipSuccess;
  const dim3 grid(grid_for(n_rows * (head_dim / 16), 256));
#define PIC_APPEND_ROPE(HDV, ILV)                                                                    \
  hipLaunchKernelGGL((append_rope_kernel<HDV, ILV>), grid, dim3(256), 0, stream, k_new, v_new, cache_k, \
                     cache_v, n_kv_heads, batch, cache_cap, pos, n_new, n_rows, table, table_stride,  \
                     max_abs_delta)
  if (head_dim == 64 && interleaved) PIC_APPEND_ROPE(64, true);
  else if (head_dim == 64) PIC_APPEND_ROPE(64, false);
  else if (interleaved) PIC_APPEND_ROPE(128, true);
  else PIC_APPEND_ROPE(128, false);
#undef PIC_APPEND_ROPE
  return hipGetLastError();
}

}  // namespace pic
