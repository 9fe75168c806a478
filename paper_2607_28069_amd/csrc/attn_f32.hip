// float32 attention of query rows over the composed cache with the frontier mask of App. C.1:
// the query at logical position p sees slots [0, p] (slot index = logical position).  The
// position of each query token comes from a RowPos (contiguous after a base, or a table).
//
// This path serves float32 caches (small models and exact checks); it is plain VALU code,
// one workgroup per query row: keys are scored 256 at a time into LDS, then the weighted
// value sum runs with lanes over head dimensions so V rows are read coalesced.
#include "pic_internal.h"

namespace pic {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

template <bool IS_MAX>
__device__ float block_reduce(float x, float* red) {
  x = IS_MAX ? wave_max(x) : wave_sum(x);
  const int w = threadIdx.x / 64;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = x;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < kThreads / 64; ++i) r = IS_MAX ? fmaxf(r, red[i]) : r + red[i];
  return r;
}

// grid (B * n_q * Hq, L)
template <int HD>
__global__ void __launch_bounds__(kThreads) attn_rows_f32_kernel(
    AttnShape s, const float* __restrict__ q, const float* __restrict__ cache_k,
    const float* __restrict__ cache_v, RowPos pos, int32_t n_q, float* __restrict__ out) {
  constexpr int G = kThreads / HD;  // key groups in the value pass
  __shared__ float q_s[HD];
  __shared__ float p_s[kThreads];
  __shared__ float red[kThreads / 64];
  __shared__ float o_s[G][HD];

  const int Hq = s.n_q_heads, Hkv = s.n_kv_heads;
  const int l = blockIdx.y;
  const int64_t row = blockIdx.x;  // ((b * n_q + i) * Hq + h)
  const int h = (int)(row % Hq);
  const int i = (int)((row / Hq) % n_q);
  const int b = (int)(row / ((int64_t)Hq * n_q));
  const int g = h / (Hq / Hkv);

  const int64_t qpos = pos(b, i);
  if (qpos < 0) return;   // (uniform) an unused row
  int64_t n_vis = qpos + 1;
  if (n_vis > s.cache_cap) n_vis = s.cache_cap;

  const int64_t qrow = ((int64_t)l * s.batch * n_q * Hq + row) * HD;
  for (int d = threadIdx.x; d < HD; d += kThreads) q_s[d] = q[qrow + d];
  const int64_t kv0 = (((int64_t)l * s.batch + b) * Hkv + g) * s.cache_cap * HD;
  const float* K = cache_k + kv0;
  const float* V = cache_v + kv0;
  __syncthreads();

  const int dd = threadIdx.x % HD, grp = threadIdx.x / HD;
  float m = -INFINITY, lsum = 0.f, acc = 0.f;
  for (int64_t c0 = 0; c0 < n_vis; c0 += kThreads) {
    const int64_t j = c0 + threadIdx.x;
    float sc = -INFINITY;
    if (j < n_vis) {
      const float* kr = K + j * HD;
      float dot = 0.f;
#pragma unroll 8
      for (int d = 0; d < HD; d += 4) {
        const float4 kv = *reinterpret_cast<const float4*>(kr + d);
        dot = fmaf(q_s[d], kv.x, dot);
        dot = fmaf(q_s[d + 1], kv.y, dot);
        dot = fmaf(q_s[d + 2], kv.z, dot);
        dot = fmaf(q_s[d + 3], kv.w, dot);
      }
      sc = dot * s.scale_log2;
    }
    const float m_new = fmaxf(m, block_reduce<true>(sc, red));
    const float alpha = exp2f(m - m_new);
    const float p = j < n_vis ? exp2f(sc - m_new) : 0.f;
    p_s[threadIdx.x] = p;
    lsum = lsum * alpha + block_reduce<false>(p, red);
    m = m_new;
    __syncthreads();
    const int64_t n_here = (n_vis - c0) < kThreads ? (n_vis - c0) : kThreads;
    float a = 0.f;
    for (int jj = grp; jj < n_here; jj += G) a = fmaf(p_s[jj], V[(c0 + jj) * HD + dd], a);
    acc = acc * alpha + a;
    __syncthreads();
  }
  o_s[grp][dd] = acc;
  __syncthreads();
  if (threadIdx.x < HD) {
    float o = 0.f;
#pragma unroll
    for (int k = 0; k < G; ++k) o += o_s[k][threadIdx.x];
    out[qrow + threadIdx.x] = o / lsum;
  }
}

}  // namespace

hipError_t launch_attn_rows_f32(const AttnShape& s, const float* q, const float* cache_k,
                                const float* cache_v, const RowPos& pos, int32_t n_q, float* out,
                                hipStream_t stream) {
  const int64_t rows = (int64_t)s.batch * n_q * s.n_q_heads;
  if (rows == 0 || s.n_layers == 0) return hipSuccess;
  const dim3 grid((unsigned)rows, s.n_layers);
  if (s.head_dim == 64)
    hipLaunchKernelGGL(attn_rows_f32_kernel<64>, grid, dim3(kThreads), 0, stream, s, q, cache_k,
                       cache_v, pos, n_q, out);
  else
    hipLaunchKernelGGL(attn_rows_f32_kernel<128>, grid, dim3(kThreads), 0, stream, s, q, cache_k,
                       cache_v, pos, n_q, out);
  return hipGetLastError();
}

}  // namespace pic
