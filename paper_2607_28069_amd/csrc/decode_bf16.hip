// Single-token decode attention over the completed cache (App. C.1: the linked cache then serves
// ordinary autoregressive decoding), bf16 storage.
//
// Per (layer, request b, kv head g) the n_rep query heads of g (one token) attend over slots
// [0, p] with p = base_len[b] + step, the new token's slot.  A step reads every cached K/V row
// once, so it is bound by HBM bandwidth; arithmetic goes to MFMA only so that it costs no VALU
// time:
//  * a workgroup of 4 waves covers one context range of one (request, kv head); each wave
//    streams its own quarter in 32-key tiles, with the next tile's loads in flight while the
//    current one is used and no barrier inside the loop;
//  * S^T = K Q^T on v_mfma_f32_16x16x32_bf16 with up to 16 query heads along N (unused columns
//    zero); a kv head with more query heads is served by one workgroup per group of 16 heads,
//    each streaming the context range: K goes straight from global memory into the A-operand layout (16 bytes per
//    lane, 64 contiguous bytes per row per instruction);
//  * O^T = V^T P^T with the same instruction: V moves global -> LDS with global_load_lds_dwordx4
//    (row-major, chunk-swizzled) and its A operand comes from two transposing reads
//    (ds_read_b64_tr_b16); the swizzle keeps those reads free of bank conflicts;
//  * every row is read once per step: the V moves (whole rows per instruction) are non-temporal,
//    while the K loads, which take a row in four 64-byte pieces, stay cached;
//  * the new token's K/V are read straight from k_new/v_new by the wave whose range holds slot p,
//    and written into the cache by that workgroup (no separate append launch);
//  * the 4 waves merge by log-sum-exp in LDS; a context split over several workgroups (only when
//    (request, kv head) pairs alone do not fill the GPU) leaves fp32 partials for a combine pass;
//  * rope variant: q and k_new arrive unrotated and are turned to position p (the delta-angle
//    table's row p) in registers -- the query once, the new key in the tile that holds it and
//    where it is stored -- with the float32 arithmetic of the re-rotation kernel.
#include <mutex>
#include <type_traits>

#include "pic_bounds.h"
#include "pic_internal.h"

namespace pic {
namespace {

// Split-K partials of the allocation-free decode entry point: one array per GPU, held until the
// process ends.  Host code never names it as an address: each device's copy is looked up once
// with hipGetSymbolAddress and that pointer is what the kernels receive.
constexpr size_t kScratchBytes = PIC_DECODE_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kWaves = 4;
constexpr int kTile = 32;                          // keys per wave tile
constexpr int kMinWaveKeys = 64;
// Sizes that follow the head dim HD (128 or 64): a row is HD/8 16-byte chunks; a lane's
// operands hold HD/32 steps of 32 head dims; the output is HD/16 blocks of 16 head dims.
template <int HD>
struct Dims {
  static_assert(HD == 128 || HD == 64, "head_dim 128 or 64");
  static constexpr int kRowBytes = HD * 2;                  // 256 or 128
  static constexpr int kVTileBytes = kTile * kRowBytes;     // per wave per buffer
  static constexpr int kChunks = HD / 8;                    // 16-byte chunks per row
  static constexpr int kSteps = HD / 32;                    // k steps of Q^T / K operands
  static constexpr int kBlocks = HD / 16;                   // 16-dim output blocks
  static constexpr int kRowsPerMove = 64 / kChunks;         // rows one 1 KB V move fills
};
static_assert(kWaves == kDecodeWaves && kMinWaveKeys == kDecodeMinWaveKeys, "host split planner tiling");
constexpr int kNonTemporal = 2;                    // cache-policy bits of a streaming load

#define LDS_AS __attribute__((address_space(3)))
#define GLOBAL_AS __attribute__((address_space(1)))

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// 16-byte chunk c of V row `key` sits at slot c ^ v_swz(key) of its row in LDS (256-byte rows:
// 16 slots; 128-byte rows: 8 slots, so the XOR keeps to the low three bits).
template <int HD>
__device__ __forceinline__ int v_swz(int key) {
  if constexpr (HD == 128) return ((key & 3) << 1) | (((key >> 2) & 1) << 3);
  else return (key & 3) << 1;
}

struct DecodeArgs {
  const bf16_t* q;        // [L][B][Hq][D]
  const bf16_t* k_new;    // [L][B][Hkv][D]
  const bf16_t* v_new;
  bf16_t* cache_k;        // [L][B][Hkv][cap][D]
  bf16_t* cache_v;
  const int32_t* base_len;
  bf16_t* out;            // [L][B][Hq][D]
  float* ws_o;            // [L][B][Hq][S][D]   (n_splits > 1)
  float* ws_ml;           // [L][B][Hq][S][2]
  int32_t batch, cache_cap, n_q_heads, n_kv_heads, max_base, step, n_splits, chunk;
  int32_t head_groups;    // groups of up to 16 query heads per kv head (ceil(n_rep / 16))
  float scale_log2;
  const float2* table;    // rope variant: [L or 1][max_abs_delta + 1][D/2] cos/sin rows
  int64_t table_stride;
  int32_t max_abs_delta;
};

// (x, y) turned by (c, s) in the float32 form of the re-rotation kernel.
__device__ __forceinline__ void rot_pair(float& x, float& y, float c, float s) {
  const float u = x, v = y;
  x = fmaf(u, c, -(v * s));
  y = fmaf(u, s, v * c);
}
__device__ __forceinline__ void unpack8(u32x4 w, float (&x)[8]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = __uint_as_float(w[e] << 16);
    x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ u32x4 pack8(const float (&x)[8]) {
  return u32x4{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
               pack_bf16x2(x[6], x[7])};
}
// The head dims 32 ks + 8 g4 .. + 8 (ks < HD/32) a lane holds of one row (the A / B operand
// layout below), turned by row `trow` of the table: rotate-half pairs are chunks ks and
// ks + HD/64 (frequencies 32 ks + 8 g4 + j), interleaved pairs sit inside a chunk (16 ks + 4 g4 + m).
template <int HD, bool kInterleaved>
__device__ __forceinline__ void rot_operand(u32x4 (&c)[Dims<HD>::kSteps], const float2* trow, int g4) {
  constexpr int KS = Dims<HD>::kSteps;
  if constexpr (!kInterleaved) {
#pragma unroll
    for (int ks = 0; ks < KS / 2; ++ks) {
      float x[8], y[8];
      unpack8(c[ks], x);
      unpack8(c[ks + KS / 2], y);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float2 cs = trow[32 * ks + 8 * g4 + j];
        rot_pair(x[j], y[j], cs.x, cs.y);
      }
      c[ks] = pack8(x);
      c[ks + KS / 2] = pack8(y);
    }
  } else {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      float x[8];
      unpack8(c[ks], x);
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const float2 cs = trow[16 * ks + 4 * g4 + m];
        rot_pair(x[2 * m], x[2 * m + 1], cs.x, cs.y);
      }
      c[ks] = pack8(x);
    }
  }
}

// grid (S * B * Hkv, L), 256 threads
template <int HD, bool kRope, bool kInterleaved>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
decode_bf16_kernel(DecodeArgs a) {
  constexpr int kHD = HD, kRowBytes = Dims<HD>::kRowBytes, kVTileBytes = Dims<HD>::kVTileBytes;
  constexpr int KC = Dims<HD>::kChunks, KS = Dims<HD>::kSteps, DB = Dims<HD>::kBlocks;
  constexpr int RPM = Dims<HD>::kRowsPerMove;
  __shared__ __attribute__((aligned(16))) uint8_t v_lds0[kWaves * kVTileBytes];
  __shared__ __attribute__((aligned(16))) uint8_t v_lds1[kWaves * kVTileBytes];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hgrp = blockIdx.x % a.head_groups;           // query heads 16 hgrp .. of kv head g
  const int split = (blockIdx.x / a.head_groups) % a.n_splits;
  const int bg = blockIdx.x / (a.head_groups * a.n_splits);
  const int b = bg / a.n_kv_heads, g = bg % a.n_kv_heads;
  const int l = blockIdx.y;
  const int n_rep = a.n_q_heads / a.n_kv_heads;
  const int rep0 = 16 * hgrp;                             // first query head of this group
  const int n_here = min(16, n_rep - rep0);               // query heads of this group

  const int32_t base = clamp_len(a.base_len[b], a.max_base);
  const int p = base + a.step;                       // the new token's slot
  int n_vis = p + 1;
  if (n_vis > a.cache_cap) n_vis = a.cache_cap;
  const int wc0 = min(split * a.chunk, n_vis);
  const int wc1 = min(wc0 + a.chunk, n_vis);
  const int sub = a.chunk / kWaves;                  // multiple of kTile
  const int c0 = min(wc0 + wave * sub, wc1);
  const int c1 = min(c0 + sub, wc1);

  const int64_t bh_kv = (((int64_t)l * a.batch + b) * a.n_kv_heads + g);
  const bf16_t* Kg = a.cache_k + bh_kv * a.cache_cap * kHD;
  const bf16_t* Vg = a.cache_v + bh_kv * a.cache_cap * kHD;
  const bf16_t* Kn = a.k_new + bh_kv * kHD;
  const bf16_t* Vn = a.v_new + bh_kv * kHD;

  // The workgroup holding slot p writes the new token into the cache.  Nobody reads that row
  // from the cache during this launch: the wave whose range holds it reads k_new / v_new.
  const float2* trow = kRope ? a.table + (int64_t)l * a.table_stride + (int64_t)min(p, a.max_abs_delta) * (kHD / 2)
                             : nullptr;   // rope variant: cos/sin of position p
  if (hgrp == 0 && p < a.cache_cap && p >= wc0 && p < wc1 && wave == 0 && lane < 2 * KC) {
    const int c = lane & (KC - 1);   // lanes [0, KC): K chunks, [KC, 2 KC): V chunks
    u32x4* dst = reinterpret_cast<u32x4*>((lane < KC ? a.cache_k : a.cache_v) + (bh_kv * a.cache_cap + p) * kHD);
    if (kRope && lane < KC) {   // the new key turned to p: lane c < KC/2 takes a chunk pair
      if (c < KC / 2) {
        // rotate-half: chunks c, c + KC/2 (frequencies 8 c ..); interleaved: 2 c, 2 c + 1 (8 c ..)
        const int ca = kInterleaved ? 2 * c : c, cb = kInterleaved ? 2 * c + 1 : c + KC / 2;
        float x[8], y[8];
        unpack8(reinterpret_cast<const u32x4*>(Kn)[ca], x);
        unpack8(reinterpret_cast<const u32x4*>(Kn)[cb], y);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float2 cs = trow[8 * c + i];
          if constexpr (kInterleaved) {
            float* z = i < 4 ? x : y;
            rot_pair(z[2 * (i & 3)], z[2 * (i & 3) + 1], cs.x, cs.y);
          } else {
            rot_pair(x[i], y[i], cs.x, cs.y);
          }
        }
        dst[ca] = pack8(x);
        dst[cb] = pack8(y);
      }
    } else {
      dst[c] = reinterpret_cast<const u32x4*>(lane < KC ? Kn : Vn)[c];
    }
  }

  const int n = lane & 15, g4 = lane >> 4;
  // Q^T operand: lane (n, g4) holds q[head g*n_rep + n][32 ks + 8 g4 .. +8)
  bf16x8_t qop[KS];
  {
    const bool ok = n < n_here;
    const int64_t qrow = ((int64_t)l * a.batch + b) * a.n_q_heads + g * n_rep + rep0 + (ok ? n : 0);
    const u32x4* qp = reinterpret_cast<const u32x4*>(a.q + qrow * kHD);
    u32x4 qv[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qv[ks] = ok ? qp[4 * ks + g4] : u32x4{0, 0, 0, 0};
    if constexpr (kRope) rot_operand<HD, kInterleaved>(qv, trow, g4);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qop[ks] = as_bf16x8(qv[ks]);
  }

  // K of one tile, straight into the A-operand layout: [mb][ks] = row k0 + 16 mb + n, head
  // dims 32 ks + 8 g4 .. +8.  Rows past the range are clamped (their scores are masked).
  auto load_k = [&](int k0, u32x4 (&kr)[2][KS]) {
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      const int row = min(k0 + 16 * mb + n, c1 - 1);
      const bf16_t* src = row == p ? Kn : Kg + (int64_t)row * kHD;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        kr[mb][ks] = *reinterpret_cast<const u32x4*>(src + 32 * ks + 8 * g4);
    }
  };
  // V of one tile into this wave's LDS buffer: instruction i fills rows RPM i .. RPM i + RPM - 1
  // (RPM = 64 / KC rows of KC chunks), lane -> row RPM i + lane / KC, chunk slot lane % KC
  // (holding chunk slot ^ v_swz(row)).
  const int ld_r = lane / KC, ld_slot = lane & (KC - 1);
  auto load_v = [&](int k0, uint8_t* buf) {
#pragma unroll
    for (int i = 0; i < kTile / RPM; ++i) {
      const int rl = RPM * i + ld_r;
      const int row = min(k0 + rl, c1 - 1);
      const int c = ld_slot ^ v_swz<HD>(rl);
      const bf16_t* src = (row == p ? Vn : Vg + (int64_t)row * kHD) + 8 * c;
      __builtin_amdgcn_global_load_lds((const GLOBAL_AS void*)src,
                                       (LDS_AS void*)(buf + wave * kVTileBytes + RPM * i * kRowBytes), 16, 0,
                                       kNonTemporal);
    }
  };

  // Transposing-read offsets: 16-lane group G = g4, lane j = 4 rr + qq points at row
  // 16 half + 4 G + rr, head dims 16 db + 4 qq .. +3; lane i then receives head dim 16 db + i.
  // Kept in registers: computed inline, the compiler makes these reads wait for the V loads in
  // flight into the other buffer.
  const int rr = (lane & 15) >> 2, qq = lane & 3;
  int v_rd_off[DB][2];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int row = 16 * half + 4 * g4 + rr;
      v_rd_off[db][half] = row * kRowBytes + (((2 * db + (qq >> 1)) ^ v_swz<HD>(row)) << 4) + 8 * (qq & 1);
    }
  auto v_rd = [&](int db, int half) { return v_rd_off[db][half]; };

  f32x4_t oacc[DB];
#pragma unroll
  for (int i = 0; i < DB; ++i) oacc[i] = f32x4_t{};
  float m_run = -INFINITY, l_part = 0.f;
  const bf16x2_t ones = __builtin_bit_cast(bf16x2_t, 0x3F803F80u);

  // One tile at k0; P = tile parity selects the (static) LDS buffers, so the compiler sees
  // that the loads in flight into one buffer do not alias reads from the other.
  auto tile = [&](int k0, auto parity, u32x4 (&kcur)[2][KS], u32x4 (&knext)[2][KS]) {
    constexpr int P = decltype(parity)::value;
    const uint8_t* vcur = P ? v_lds1 : v_lds0;
    uint8_t* vnext = P ? v_lds0 : v_lds1;
    if (k0 + kTile < c1) {
      load_k(k0 + kTile, knext);
      load_v(k0 + kTile, vnext);
    }
    if constexpr (kRope) {   // the new token's key, read unrotated from k_new, turned to p
      if (p >= k0 && p < k0 + kTile) {
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
          if (min(k0 + 16 * mb + n, c1 - 1) == p) rot_operand<HD, kInterleaved>(kcur[mb], trow, g4);
      }
    }
    f32x4_t sacc[2] = {f32x4_t{}, f32x4_t{}};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int mb = 0; mb < 2; ++mb)
        sacc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kcur[mb][ks]), qop[ks], sacc[mb], 0, 0, 0);
    float mx = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (k0 + 16 * mb + 4 * g4 + e >= c1) sacc[mb][e] = -INFINITY;
        mx = fmaxf(mx, sacc[mb][e]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_tile = mx * a.scale_log2;
    if (__any(m_tile > m_run + 8.f)) {   // lazy reference max, as in the prefill kernel
      const float m_new = fmaxf(m_run, m_tile);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_part *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
    }
    uint32_t pw[4];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      pw[j] = pack_bf16x2(__builtin_amdgcn_exp2f(fmaf(sacc[0][2 * j], a.scale_log2, -m_run)),
                          __builtin_amdgcn_exp2f(fmaf(sacc[0][2 * j + 1], a.scale_log2, -m_run)));
      pw[2 + j] = pack_bf16x2(__builtin_amdgcn_exp2f(fmaf(sacc[1][2 * j], a.scale_log2, -m_run)),
                              __builtin_amdgcn_exp2f(fmaf(sacc[1][2 * j + 1], a.scale_log2, -m_run)));
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
      l_part = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pw[j]), ones, l_part, false);
    // P^T operand: k index 8 g4 + j <-> key 16 (j / 4) + 4 g4 + j % 4 (accumulator order)
    const bf16x8_t pop = as_bf16x8(u32x4{pw[0], pw[1], pw[2], pw[3]});
    const uint8_t* vw = vcur + wave * kVTileBytes;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS i16x4*)(vw + v_rd(db, 0)));
      const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS i16x4*)(vw + v_rd(db, 1)));
      const bf16x8_t vv = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      oacc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vv, pop, oacc[db], 0, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): the next tile is resident
  };

  u32x4 k_a[2][KS], k_b[2][KS];
  if (c0 < c1) {
    load_k(c0, k_a);
    load_v(c0, v_lds0);
    __builtin_amdgcn_s_waitcnt(0x0F70);
    for (int k0 = c0; k0 < c1; k0 += 2 * kTile) {
      tile(k0, std::integral_constant<int, 0>{}, k_a, k_b);
      if (k0 + kTile < c1) tile(k0 + kTile, std::integral_constant<int, 1>{}, k_b, k_a);
    }
  }

  // ---- merge the 4 waves (log-sum-exp) through LDS, reusing the V buffers
  float l_tot = l_part + __shfl_xor(l_part, 16, 64);
  l_tot += __shfl_xor(l_tot, 32, 64);
  __syncthreads();
  float* o_lds = reinterpret_cast<float*>(v_lds0);    // [4][16][HD] fp32: all of v_lds0
  float* ml_lds = reinterpret_cast<float*>(v_lds1);   // [4][16][2]
  if (n < n_here) {
#pragma unroll
    for (int db = 0; db < DB; ++db)
      *reinterpret_cast<float4*>(o_lds + (wave * 16 + n) * kHD + 16 * db + 4 * g4) =
          make_float4(oacc[db][0], oacc[db][1], oacc[db][2], oacc[db][3]);
    if (g4 == 0) {
      ml_lds[(wave * 16 + n) * 2] = m_run;
      ml_lds[(wave * 16 + n) * 2 + 1] = l_tot;
    }
  }
  __syncthreads();
  // thread -> (query n = tid / KC, head dims 8 (tid % KC) .. +8)
  const int mn = tid / KC, md = 8 * (tid & (KC - 1));
  if (mn < n_here) {
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, ml_lds[(w * 16 + mn) * 2]);
    float den = 0.f, o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float mw = ml_lds[(w * 16 + mn) * 2];
      if (mw == -INFINITY) continue;   // an empty wave range
      const float wt = __builtin_amdgcn_exp2f(mw - M);
      den += wt * ml_lds[(w * 16 + mn) * 2 + 1];
      const float4 x0 = *reinterpret_cast<const float4*>(o_lds + (w * 16 + mn) * kHD + md);
      const float4 x1 = *reinterpret_cast<const float4*>(o_lds + (w * 16 + mn) * kHD + md + 4);
      o[0] += wt * x0.x; o[1] += wt * x0.y; o[2] += wt * x0.z; o[3] += wt * x0.w;
      o[4] += wt * x1.x; o[5] += wt * x1.y; o[6] += wt * x1.z; o[7] += wt * x1.w;
    }
    const int64_t row = ((int64_t)l * a.batch + b) * a.n_q_heads + g * n_rep + rep0 + mn;
    if (a.n_splits == 1) {
      const float inv = 1.f / den;
      uint4 v;
      v.x = pack_bf16x2(o[0] * inv, o[1] * inv);
      v.y = pack_bf16x2(o[2] * inv, o[3] * inv);
      v.z = pack_bf16x2(o[4] * inv, o[5] * inv);
      v.w = pack_bf16x2(o[6] * inv, o[7] * inv);
      *reinterpret_cast<uint4*>(a.out + row * kHD + md) = v;
    } else {
      const int64_t slot = row * a.n_splits + split;
      float* wo = a.ws_o + slot * kHD + md;
      *reinterpret_cast<float4*>(wo) = make_float4(o[0], o[1], o[2], o[3]);
      *reinterpret_cast<float4*>(wo + 4) = make_float4(o[4], o[5], o[6], o[7]);
      if (md == 0) *reinterpret_cast<float2*>(a.ws_ml + 2 * slot) = make_float2(M, den);
    }
  }
}

// grid (B * Hq, L), HD / 2 threads (two head dims each): merge the splits of one query head by
// log-sum-exp.  The loads of kCombineBatch splits are issued together before any is used (one
// pass for the maximum, one for the weighted sums); a split that saw no key (maximum -inf) adds
// nothing.
constexpr int kCombineBatch = 8;
template <int HD>
__global__ void __launch_bounds__(64) decode_combine_kernel(const float* __restrict__ ws_o,
                                                            const float* __restrict__ ws_ml,
                                                            int32_t n_splits, int64_t rows_per_layer,
                                                            bf16_t* __restrict__ out) {
  const int64_t row = (int64_t)blockIdx.y * rows_per_layer + blockIdx.x;
  const float* ml = ws_ml + row * n_splits * 2;
  float M = -INFINITY;
  for (int s0 = 0; s0 < n_splits; s0 += kCombineBatch) {
    float mv[kCombineBatch];
#pragma unroll
    for (int u = 0; u < kCombineBatch; ++u) mv[u] = s0 + u < n_splits ? ml[2 * (s0 + u)] : -INFINITY;
#pragma unroll
    for (int u = 0; u < kCombineBatch; ++u) M = fmaxf(M, mv[u]);
  }
  float den = 0.f, o0 = 0.f, o1 = 0.f;
  const int d = 2 * threadIdx.x;
  for (int s0 = 0; s0 < n_splits; s0 += kCombineBatch) {
    float2 mlv[kCombineBatch], ov[kCombineBatch];
#pragma unroll
    for (int u = 0; u < kCombineBatch; ++u) {
      const int s = s0 + u;
      mlv[u] = s < n_splits ? *reinterpret_cast<const float2*>(ml + 2 * s) : make_float2(-INFINITY, 0.f);
      ov[u] = s < n_splits ? *reinterpret_cast<const float2*>(ws_o + (row * n_splits + s) * HD + d)
                           : make_float2(0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < kCombineBatch; ++u) {
      if (mlv[u].x == -INFINITY) continue;
      const float w = __builtin_amdgcn_exp2f(mlv[u].x - M);
      den += w * mlv[u].y;
      o0 += w * ov[u].x;
      o1 += w * ov[u].y;
    }
  }
  const float inv = 1.f / den;
  reinterpret_cast<uint32_t*>(out + row * HD)[threadIdx.x] = pack_bf16x2(o0 * inv, o1 * inv);
}

template <int HD>
hipError_t launch_decode_hd(const DecodeArgs& a, dim3 grid, bool rope, bool interleaved, int32_t n_splits,
                            const AttnShape& s, hipStream_t stream) {
  if (!rope)
    hipLaunchKernelGGL((decode_bf16_kernel<HD, false, false>), grid, dim3(256), 0, stream, a);
  else if (interleaved)
    hipLaunchKernelGGL((decode_bf16_kernel<HD, true, true>), grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL((decode_bf16_kernel<HD, true, false>), grid, dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || n_splits == 1) return e;
  hipLaunchKernelGGL(decode_combine_kernel<HD>, dim3(s.batch * s.n_q_heads, s.n_layers), dim3(HD / 2), 0,
                     stream, a.ws_o, a.ws_ml, n_splits, (int64_t)s.batch * s.n_q_heads, a.out);
  return hipGetLastError();
}

}  // namespace

size_t decode_scratch_bytes() { return kScratchBytes; }

hipError_t decode_scratch_ptr(void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* ptr[kMaxDevices] = {};
  *out = nullptr;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (ptr[dev] == nullptr) {   // first call on this device (it is the current one)
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    ptr[dev] = p;
  }
  *out = ptr[dev];
  return hipSuccess;
}

hipError_t launch_decode_bf16(const AttnShape& s, const bf16_t* q, const bf16_t* k_new,
                              const bf16_t* v_new, bf16_t* cache_k, bf16_t* cache_v,
                              const int32_t* base_len, int32_t max_base, int32_t step,
                              int32_t n_splits, bf16_t* out, void* workspace, size_t,
                              const float2* rope_table, int64_t table_stride, int32_t max_abs_delta,
                              bool interleaved, hipStream_t stream) {
  if (s.batch == 0 || s.n_layers == 0) return hipSuccess;
  const int32_t max_len = max_base + step + 1;
  DecodeArgs a;
  a.q = q;
  a.k_new = k_new;
  a.v_new = v_new;
  a.cache_k = cache_k;
  a.cache_v = cache_v;
  a.base_len = base_len;
  a.out = out;
  const size_t rows = (size_t)s.n_layers * s.batch * s.n_q_heads * n_splits;
  a.ws_o = static_cast<float*>(workspace);
  a.ws_ml = a.ws_o ? a.ws_o + rows * s.head_dim : nullptr;
  a.batch = s.batch;
  a.cache_cap = s.cache_cap;
  a.n_q_heads = s.n_q_heads;
  a.n_kv_heads = s.n_kv_heads;
  a.max_base = max_base;
  a.step = step;
  a.n_splits = n_splits;
  const int32_t chunk = (max_len + n_splits - 1) / n_splits;
  a.chunk = (chunk + kWaves * kTile - 1) / (kWaves * kTile) * (kWaves * kTile);
  a.scale_log2 = s.scale_log2;
  a.table = rope_table;
  a.table_stride = table_stride;
  a.max_abs_delta = max_abs_delta;
  a.head_groups = decode_head_groups(s);
  const dim3 grid(a.head_groups * n_splits * s.batch * s.n_kv_heads, s.n_layers);
  if (s.head_dim == 64) return launch_decode_hd<64>(a, grid, rope_table != nullptr, interleaved, n_splits, s, stream);
  return launch_decode_hd<128>(a, grid, rope_table != nullptr, interleaved, n_splits, s, stream);
}

}  // namespace pic
