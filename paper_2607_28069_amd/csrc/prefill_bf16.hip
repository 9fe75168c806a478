// Suffix prefill attention on bf16 MFMA (App. C.1: inline tokens attend over the linked cache
// under the frontier causal mask; Sec. 5 "Cache-hit serving").
//
// Problem per (layer, request b, kv head g): M = n_suffix * n_rep query rows (the n_rep query
// heads of kv head g are packed into the row dimension, row r = token r / n_rep, head
// g * n_rep + r % n_rep) against n_keys = ctx + n_suffix keys.  Query token i sits at
// position ctx + i and sees keys [0, ctx + i]; only the last key tiles need a mask.
//
// Kernel shape (gfx950, wave64):
//  * 4 waves per workgroup, 32 query rows per wave (128 rows per workgroup), key tiles of 64.
//  * Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: A = K rows
//    from LDS, B = Q^T held in registers for the whole key loop.  In the accumulator layout
//    each lane then owns ONE query column and 32 of the tile's keys, so the row max needs a
//    single cross-lane exchange (lane l <-> l ^ 32) and the row sum none until the end.
//  * O^T = V^T P^T with the same instruction: the probabilities, rounded to bf16, are already
//    in the B-operand layout (keys along k) once the tile's keys are numbered in the order
//    the accumulator holds them; V is written transposed into LDS in that key order, so each
//    A operand is one 16-byte LDS read.
//  * K and V tiles are double-buffered in LDS: the next tile's global loads are in flight
//    while the current tile is multiplied; one barrier per tile.
//  * Workgroups sharing a (request, kv head) key stream are mapped onto the same XCD (blocks
//    are dealt round-robin over the 8 XCDs), so that stream is fetched into one L2.
#include "pic_internal.h"

namespace pic {
namespace {

constexpr int kWaves = 4;
constexpr int kRowsPerWave = 32;
constexpr int kRowsPerWG = kWaves * kRowsPerWave;
constexpr int kKeys = 64;                 // keys per tile
constexpr int kHD = 128;
constexpr int kKStride = kHD / 2 + 4;     // dwords per K row in LDS (bank spread, 16-B aligned)
constexpr int kVStride = kKeys / 2 + 4;   // dwords per transposed V row (one head dim) in LDS
constexpr int kKBuf = kKeys * kKStride;   // dwords
constexpr int kVBuf = kHD * kVStride;     // dwords
constexpr int kNumXcd = 8;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// Position of key `key` (0..63) of a tile inside a transposed-V row: swap bits 2 and 3, the
// order in which the S^T accumulator hands probabilities to the B operand.
__device__ __forceinline__ int key_perm(int key) {
  return (key & ~12) | ((key & 4) << 1) | ((key & 8) >> 1);
}

// Dword column swizzle of transposed-V rows: rows 8 apart start in different bank groups.
__device__ __forceinline__ int v_swz(int d) { return ((d >> 3) & 3) * 8; }

struct PrefillArgs {
  const bf16_t* q;
  const bf16_t* cache_k;
  const bf16_t* cache_v;
  const int32_t* ctx_len;
  bf16_t* out;
  int32_t max_ctx, n_suffix, batch, cache_cap, n_q_heads, n_kv_heads;
  int32_t m_tiles;   // ceil(n_suffix * n_rep / kRowsPerWG)
  int32_t n_wg;      // m_tiles * batch * n_kv_heads
  float scale_log2;
};

__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
prefill_bf16_kernel(PrefillArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t k_lds[2 * kKBuf];
  __shared__ __attribute__((aligned(16))) uint32_t v_lds[2 * kVBuf];

  // XCD-aware block order: hardware block w runs on XCD w % 8; give each XCD a contiguous
  // range of logical blocks so the m-tiles of one (request, kv head) share an L2.
  const int per_xcd = (a.n_wg + kNumXcd - 1) / kNumXcd;
  const int w = blockIdx.x;
  const int logical = (w % kNumXcd) * per_xcd + w / kNumXcd;
  if (logical >= a.n_wg) return;
  const int mt = logical % a.m_tiles;
  const int bg = logical / a.m_tiles;
  const int b = bg / a.n_kv_heads, g = bg % a.n_kv_heads;
  const int l = blockIdx.y;

  const int n_rep = a.n_q_heads / a.n_kv_heads;
  const int M = a.n_suffix * n_rep;
  int32_t ctx = a.ctx_len[b];
  ctx = ctx < 0 ? 0 : (ctx > a.max_ctx ? a.max_ctx : ctx);
  const int n_keys = ctx + a.n_suffix;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, hh = lane >> 5;   // query column, lane half

  // ---- rows of this wave and workgroup
  const int row0_wg = mt * kRowsPerWG;
  const int last_row_wg = min(row0_wg + kRowsPerWG, M) - 1;
  const int pos_max_wg = ctx + last_row_wg / n_rep;   // furthest key any row here sees
  const int n_tiles = (pos_max_wg + kKeys) / kKeys;

  const int r = row0_wg + wave * kRowsPerWave + n;    // this lane's query row
  const bool row_ok = r < M;
  const int tok = row_ok ? r / n_rep : a.n_suffix - 1;
  const int hq = g * n_rep + (row_ok ? r % n_rep : 0);
  const int qpos = ctx + tok;

  const int64_t bh_kv = (((int64_t)l * a.batch + b) * a.n_kv_heads + g) * a.cache_cap;
  const bf16_t* Kg = a.cache_k + bh_kv * kHD;
  const bf16_t* Vg = a.cache_v + bh_kv * kHD;
  const int64_t qrow = (((int64_t)l * a.batch + b) * a.n_suffix + tok) * a.n_q_heads + hq;

  // ---- Q^T operand: lane (n, hh) holds q[row n][16 ks + 8 hh .. +8) for ks = 0..7
  bf16x8_t qop[8];
  {
    const u32x4* qp = reinterpret_cast<const u32x4*>(a.q + qrow * kHD);
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      u32x4 v = row_ok ? qp[2 * ks + hh] : u32x4{0, 0, 0, 0};
      qop[ks] = as_bf16x8(v);
    }
  }

  // ---- tile staging: thread -> (16-byte chunk dc, key group) for K and V
  const int dc = tid & 15;          // 8 head dims [8 dc, 8 dc + 8)
  const int kq = tid >> 4;          // K: keys kq + 16 u;  V: keys 4 kq + u   (u = 0..3)
  u32x4 kreg[4], vreg[4];

  // Rows past the last key are clamped to it: their scores are masked, so they enter the
  // PV product with probability 0 (finite values, no branch around the loads).
  auto load_tile = [&](int t) {
    const int k0 = t * kKeys;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int kk = min(k0 + kq + 16 * u, n_keys - 1);
      kreg[u] = *reinterpret_cast<const u32x4*>(Kg + (int64_t)kk * kHD + 8 * dc);
      const int kv = min(k0 + 4 * kq + u, n_keys - 1);
      vreg[u] = *reinterpret_cast<const u32x4*>(Vg + (int64_t)kv * kHD + 8 * dc);
    }
  };

  auto store_tile = [&](int buf) {
    uint32_t* kb = k_lds + buf * kKBuf;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      *reinterpret_cast<u32x4*>(kb + (kq + 16 * u) * kKStride + 4 * dc) = kreg[u];
    // V transposed: row = head dim, 4 consecutive keys 4kq..4kq+3 packed into 8 bytes.
    uint32_t* vb = v_lds + buf * kVBuf;
    const int col = key_perm(4 * kq) >> 1;   // dword column of key 4kq (even)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int word = e >> 1;
      uint32_t lo, hi;
      if (e & 1) {
        lo = (vreg[0][word] >> 16) | (vreg[1][word] & 0xFFFF0000u);
        hi = (vreg[2][word] >> 16) | (vreg[3][word] & 0xFFFF0000u);
      } else {
        lo = (vreg[0][word] & 0xFFFFu) | (vreg[1][word] << 16);
        hi = (vreg[2][word] & 0xFFFFu) | (vreg[3][word] << 16);
      }
      const int d = 8 * dc + e;
      *reinterpret_cast<uint2*>(vb + d * kVStride + (col ^ v_swz(d))) = make_uint2(lo, hi);
    }
  };

  f32x16_t oacc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) oacc[i] = f32x16_t{};
  float m_run = -INFINITY, l_part = 0.f;

  load_tile(0);
  store_tile(0);
  __syncthreads();

  for (int t = 0; t < n_tiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < n_tiles) load_tile(t + 1);

    // ---- S^T = K Q^T for keys [64 t, 64 t + 64): two 32-key blocks
    const uint32_t* kb = k_lds + buf * kKBuf;
    // two independent accumulation chains, interleaved
    f32x16_t sacc[2] = {f32x16_t{}, f32x16_t{}};
    const uint32_t* krow = kb + n * kKStride + 4 * hh;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2) {
        const u32x4 kv = *reinterpret_cast<const u32x4*>(krow + 32 * kb2 * kKStride + 8 * ks);
        sacc[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kv), qop[ks], sacc[kb2], 0, 0, 0);
      }

    // ---- online softmax over this lane's query column.  Scores stay unscaled until the
    // exponent: p = exp2(s * scale * log2(e) - m), one FMA and one v_exp_f32 per score.
    const int k0 = t * kKeys;
    if (k0 + kKeys - 1 > ctx) {   // tile reaches into the suffix (or past the last key)
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = k0 + 32 * kb2 + 8 * (e >> 2) + 4 * hh + (e & 3);
          if (key > qpos) sacc[kb2][e] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, sacc[kb2][e]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_tile = mx * a.scale_log2;
    // The reference max only moves when a score exceeds it by more than 2^8 (then the
    // accumulators are rescaled, for the whole wave at once); otherwise p <= 256, which
    // float32 sums and bf16 probabilities hold without loss of relative precision.
    if (__any(m_tile > m_run + 8.f)) {
      const float m_new = fmaxf(m_run, m_tile);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_part *= alpha;
#pragma unroll
      for (int db = 0; db < 4; ++db) oacc[db] *= alpha;
    }

    // ---- P^T (bf16) slice by slice, each followed by its four O^T += V^T P^T products
    // (four independent accumulators), so the exponentials of the next slice can overlap the
    // matrix products of the current one.
    const uint32_t* vb = v_lds + buf * kVBuf;
    float psum = 0.f;
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
      const int kb2 = s4 >> 1, u = s4 & 1;
      uint32_t pw[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[kb2][8 * u + 2 * j], a.scale_log2, -m_run));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[kb2][8 * u + 2 * j + 1], a.scale_log2, -m_run));
        psum += p0 + p1;
        pw[j] = pack_bf16x2(p0, p1);
      }
      const bf16x8_t pop = as_bf16x8(u32x4{pw[0], pw[1], pw[2], pw[3]});
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const int d = 32 * db + n;
        const u32x4 vv = *reinterpret_cast<const u32x4*>(vb + d * kVStride + ((8 * s4 + 4 * hh) ^ v_swz(d)));
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv), pop, oacc[db], 0, 0, 0);
      }
    }
    l_part += psum;

    if (t + 1 < n_tiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  // ---- normalise and store: lane holds head dims 32 db + 8 q + 4 hh + (0..3) of its row
  const float l_tot = l_part + __shfl_xor(l_part, 32, 64);
  const float inv = 1.f / l_tot;
  if (row_ok) {
    bf16_t* orow = a.out + qrow * kHD;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int d = 32 * db + 8 * qd + 4 * hh;
        uint2 v;
        v.x = pack_bf16x2(oacc[db][4 * qd] * inv, oacc[db][4 * qd + 1] * inv);
        v.y = pack_bf16x2(oacc[db][4 * qd + 2] * inv, oacc[db][4 * qd + 3] * inv);
        *reinterpret_cast<uint2*>(orow + d) = v;
      }
  }
}

}  // namespace

size_t prefill_bf16_workspace(const AttnShape&, int32_t, int32_t) { return 0; }

hipError_t launch_prefill_bf16(const AttnShape& s, const bf16_t* q, const bf16_t* cache_k,
                               const bf16_t* cache_v, const int32_t* ctx_len, int32_t max_ctx,
                               int32_t n_suffix, bf16_t* out, void*, size_t, hipStream_t stream) {
  const int n_rep = s.n_q_heads / s.n_kv_heads;
  const int64_t M = (int64_t)n_suffix * n_rep;
  if (M == 0 || s.batch == 0 || s.n_layers == 0) return hipSuccess;
  PrefillArgs a;
  a.q = q;
  a.cache_k = cache_k;
  a.cache_v = cache_v;
  a.ctx_len = ctx_len;
  a.out = out;
  a.max_ctx = max_ctx;
  a.n_suffix = n_suffix;
  a.batch = s.batch;
  a.cache_cap = s.cache_cap;
  a.n_q_heads = s.n_q_heads;
  a.n_kv_heads = s.n_kv_heads;
  a.m_tiles = (int32_t)((M + kRowsPerWG - 1) / kRowsPerWG);
  a.n_wg = a.m_tiles * s.batch * s.n_kv_heads;
  a.scale_log2 = s.scale_log2;
  const int per_xcd = (a.n_wg + kNumXcd - 1) / kNumXcd;
  const dim3 grid(per_xcd * kNumXcd, s.n_layers);
  hipLaunchKernelGGL(prefill_bf16_kernel, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace pic
