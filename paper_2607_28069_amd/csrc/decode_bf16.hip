// Single-token decode attention over the completed cache (App. C.1: the linked cache then serves
// ordinary autoregressive decoding), bf16 storage, split over the context.
//
// Per (layer, request b, kv head g) the n_rep query heads of g (one token) attend over slots
// [0, p] with p = base_len[b] + step.  The step reads every cached K/V row once, so it is bound
// by HBM bandwidth; arithmetic goes to MFMA only so that it costs no VALU time:
//  * one wave per workgroup, one context chunk per workgroup; the chunk is streamed in 32-key
//    tiles with 16-byte loads that cover 4 whole rows per instruction, the next tile's loads
//    in flight while the current one is used;
//  * S^T = K Q^T and O^T = V^T P^T on v_mfma_f32_16x16x32_bf16 with the query heads along
//    N (n_rep <= 16; unused columns are zero), K and transposed V staged in the wave's LDS;
//  * each chunk leaves (m, l, unnormalised O) in fp32 workspace and a second kernel merges the
//    chunks by log-sum-exp and writes bf16.
#include "pic_internal.h"

namespace pic {
namespace {

constexpr int kHD = 128;
constexpr int kTile = 32;                    // keys per tile
constexpr int kKStride = kHD / 2 + 4;        // dwords per K row in LDS
constexpr int kVStride = kTile / 2 + 4;      // dwords per transposed-V row in LDS
constexpr int kMaxRep = 16;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// Order of a tile's keys along the k axis of the P^T operand.  The S^T accumulator gives lane
// group g4 = lane / 16 keys {4 g4 + e} and {16 + 4 g4 + e}; the B operand wants lane group g4
// to hold k = 8 g4 .. 8 g4 + 7.  kappa(key) is the k index a key takes.
__device__ __forceinline__ int kappa(int key) {
  return (((key >> 2) & 3) << 3) | (((key >> 4) & 1) << 2) | (key & 3);
}

struct DecodeArgs {
  const bf16_t* q;        // [L][B][Hq][D]
  const bf16_t* cache_k;  // [L][B][Hkv][cap][D]
  const bf16_t* cache_v;
  const int32_t* base_len;
  float* ws_o;            // [L][B][Hq][S][D]
  float* ws_ml;           // [L][B][Hq][S][2]
  int32_t batch, cache_cap, n_q_heads, n_kv_heads, max_base, step, n_splits, chunk;
  float scale_log2;
};

// grid (S * B * Hkv, L), 64 threads
__global__ void __launch_bounds__(64) decode_bf16_kernel(DecodeArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t k_lds[kTile * kKStride];
  __shared__ __attribute__((aligned(16))) uint32_t v_lds[kHD * kVStride];

  const int lane = threadIdx.x;
  const int split = blockIdx.x % a.n_splits;
  const int bg = blockIdx.x / a.n_splits;
  const int b = bg / a.n_kv_heads, g = bg % a.n_kv_heads;
  const int l = blockIdx.y;
  const int n_rep = a.n_q_heads / a.n_kv_heads;

  int32_t base = a.base_len[b];
  base = base < 0 ? 0 : (base > a.max_base ? a.max_base : base);
  int n_vis = base + a.step + 1;
  if (n_vis > a.cache_cap) n_vis = a.cache_cap;
  const int c0 = split * a.chunk;
  const int c1 = min(c0 + a.chunk, n_vis);

  const int n = lane & 15, g4 = lane >> 4;
  const int64_t bh_kv = (((int64_t)l * a.batch + b) * a.n_kv_heads + g) * a.cache_cap;
  const bf16_t* Kg = a.cache_k + bh_kv * kHD;
  const bf16_t* Vg = a.cache_v + bh_kv * kHD;

  // Q^T operand: lane (n, g4) holds q[head g*n_rep + n][32 ks + 8 g4 .. +8)
  bf16x8_t qop[4];
  {
    const bool ok = n < n_rep;
    const int64_t qrow = ((int64_t)l * a.batch + b) * a.n_q_heads + g * n_rep + (ok ? n : 0);
    const u32x4* qp = reinterpret_cast<const u32x4*>(a.q + qrow * kHD);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) qop[ks] = as_bf16x8(ok ? qp[4 * ks + g4] : u32x4{0, 0, 0, 0});
  }

  const int dc = lane & 15;   // 16-byte chunk of a row: head dims [8 dc, 8 dc + 8)
  const int kr = lane >> 4;   // K: keys kr + 4 u (u = 0..7); V: keys 4 (kr + 4 i) + u
  u32x4 kreg[8], vreg[8];
  auto load_tile = [&](int k0) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int kk = k0 + kr + 4 * u;
      kreg[u] = kk < c1 ? *reinterpret_cast<const u32x4*>(Kg + (int64_t)kk * kHD + 8 * dc)
                        : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int kv = k0 + 4 * (kr + 4 * i) + u;
        vreg[4 * i + u] = kv < c1 ? *reinterpret_cast<const u32x4*>(Vg + (int64_t)kv * kHD + 8 * dc)
                                  : u32x4{0, 0, 0, 0};
      }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int u = 0; u < 8; ++u)
      *reinterpret_cast<u32x4*>(k_lds + (kr + 4 * u) * kKStride + 4 * dc) = kreg[u];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int col = kappa(4 * (kr + 4 * i)) >> 1;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int word = e >> 1;
        uint32_t lo, hi;
        if (e & 1) {
          lo = (vreg[4 * i + 0][word] >> 16) | (vreg[4 * i + 1][word] & 0xFFFF0000u);
          hi = (vreg[4 * i + 2][word] >> 16) | (vreg[4 * i + 3][word] & 0xFFFF0000u);
        } else {
          lo = (vreg[4 * i + 0][word] & 0xFFFFu) | (vreg[4 * i + 1][word] << 16);
          hi = (vreg[4 * i + 2][word] & 0xFFFFu) | (vreg[4 * i + 3][word] << 16);
        }
        *reinterpret_cast<uint2*>(v_lds + (8 * dc + e) * kVStride + col) = make_uint2(lo, hi);
      }
    }
  };

  f32x4_t oacc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) oacc[i] = f32x4_t{};
  float m_run = -INFINITY, l_part = 0.f;

  if (c0 < c1) load_tile(c0);
  for (int k0 = c0; k0 < c1; k0 += kTile) {
    __syncthreads();            // previous tile's LDS reads are done
    store_tile();
    __syncthreads();
    if (k0 + kTile < c1) load_tile(k0 + kTile);

    // S^T: keys [k0 + 16 mb, +16) x 16 query columns
    f32x4_t sacc[2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
      sacc[mb] = f32x4_t{};
      const uint32_t* krow = k_lds + (16 * mb + n) * kKStride + 4 * g4;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const u32x4 kv = *reinterpret_cast<const u32x4*>(krow + 16 * ks);
        sacc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kv), qop[ks], sacc[mb], 0, 0, 0);
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = k0 + 16 * mb + 4 * g4 + e;
        if (key >= c1) sacc[mb][e] = -INFINITY;
        mx = fmaxf(mx, sacc[mb][e]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx * a.scale_log2);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    float p[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      p[e] = __builtin_amdgcn_exp2f(fmaf(sacc[0][e], a.scale_log2, -m_new));
      p[4 + e] = __builtin_amdgcn_exp2f(fmaf(sacc[1][e], a.scale_log2, -m_new));
    }
    float psum = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) psum += p[j];
    l_part = l_part * alpha + psum;
    const bf16x8_t pop = as_bf16x8(u32x4{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                                         pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])});
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      oacc[db] *= alpha;
      const u32x4 vv = *reinterpret_cast<const u32x4*>(v_lds + (16 * db + n) * kVStride + 4 * g4);
      oacc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vv), pop, oacc[db], 0, 0, 0);
    }
  }

  float l_tot = l_part + __shfl_xor(l_part, 16, 64);
  l_tot += __shfl_xor(l_tot, 32, 64);
  if (n < n_rep) {
    const int hq = g * n_rep + n;
    const int64_t slot = (((int64_t)l * a.batch + b) * a.n_q_heads + hq) * a.n_splits + split;
    float* wo = a.ws_o + slot * kHD;
#pragma unroll
    for (int db = 0; db < 8; ++db)
      *reinterpret_cast<float4*>(wo + 16 * db + 4 * g4) =
          make_float4(oacc[db][0], oacc[db][1], oacc[db][2], oacc[db][3]);
    if (g4 == 0) *reinterpret_cast<float2*>(a.ws_ml + 2 * slot) = make_float2(m_run, l_tot);
  }
}

// grid (B * Hq, L), 64 threads: merge the chunks of one query head by log-sum-exp.
__global__ void __launch_bounds__(64) decode_combine_kernel(const float* __restrict__ ws_o,
                                                            const float* __restrict__ ws_ml,
                                                            int32_t n_splits, int64_t rows_per_layer,
                                                            bf16_t* __restrict__ out) {
  const int64_t row = (int64_t)blockIdx.y * rows_per_layer + blockIdx.x;
  const float* ml = ws_ml + row * n_splits * 2;
  float M = -INFINITY;
  for (int s = 0; s < n_splits; ++s) M = fmaxf(M, ml[2 * s]);
  float den = 0.f, o0 = 0.f, o1 = 0.f;
  const int d = 2 * threadIdx.x;
  for (int s = 0; s < n_splits; ++s) {
    const float ms = ml[2 * s];
    if (ms == -INFINITY) continue;
    const float w = __builtin_amdgcn_exp2f(ms - M);
    den += w * ml[2 * s + 1];
    const float2 o = *reinterpret_cast<const float2*>(ws_o + (row * n_splits + s) * kHD + d);
    o0 += w * o.x;
    o1 += w * o.y;
  }
  const float inv = 1.f / den;
  reinterpret_cast<uint32_t*>(out + row * kHD)[threadIdx.x] = pack_bf16x2(o0 * inv, o1 * inv);
}

}  // namespace

int32_t decode_bf16_auto_splits(const AttnShape& s, int32_t max_len) {
  const int64_t pairs = (int64_t)s.batch * s.n_kv_heads;
  const int64_t target_waves = 2048;   // about one resident round of waves
  int64_t splits = (target_waves + pairs - 1) / pairs;
  const int64_t max_splits = (max_len + 255) / 256;   // keep chunks >= 256 keys
  if (splits > max_splits) splits = max_splits;
  if (splits < 1) splits = 1;
  return (int32_t)splits;
}

size_t decode_bf16_workspace(const AttnShape& s, int32_t, int32_t n_splits) {
  const size_t rows = (size_t)s.n_layers * s.batch * s.n_q_heads * n_splits;
  return rows * (kHD + 2) * sizeof(float);
}

hipError_t launch_decode_bf16(const AttnShape& s, const bf16_t* q, const bf16_t* cache_k,
                              const bf16_t* cache_v, const int32_t* base_len, int32_t max_base,
                              int32_t step, int32_t n_splits, bf16_t* out, void* workspace,
                              size_t, hipStream_t stream) {
  if (s.batch == 0 || s.n_layers == 0) return hipSuccess;
  const int32_t max_len = max_base + step + 1;
  DecodeArgs a;
  a.q = q;
  a.cache_k = cache_k;
  a.cache_v = cache_v;
  a.base_len = base_len;
  const size_t rows = (size_t)s.n_layers * s.batch * s.n_q_heads * n_splits;
  a.ws_o = static_cast<float*>(workspace);
  a.ws_ml = a.ws_o + rows * kHD;
  a.batch = s.batch;
  a.cache_cap = s.cache_cap;
  a.n_q_heads = s.n_q_heads;
  a.n_kv_heads = s.n_kv_heads;
  a.max_base = max_base;
  a.step = step;
  a.n_splits = n_splits;
  int32_t chunk = (max_len + n_splits - 1) / n_splits;
  a.chunk = (chunk + kTile - 1) / kTile * kTile;
  a.scale_log2 = s.scale_log2;
  hipLaunchKernelGGL(decode_bf16_kernel, dim3(n_splits * s.batch * s.n_kv_heads, s.n_layers),
                     dim3(64), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_combine_kernel, dim3(s.batch * s.n_q_heads, s.n_layers), dim3(64), 0,
                     stream, a.ws_o, a.ws_ml, n_splits, (int64_t)s.batch * s.n_q_heads, out);
  return hipGetLastError();
}

}  // namespace pic
