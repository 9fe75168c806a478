// Row-wise attention of query rows over a cache with the frontier mask of App. C.1: the query
// at logical position p sees slots [0, p] (slot index = logical position).  The position of
// each query token comes from a RowPos (contiguous after a base, or a table).
//
// This path serves the shapes the bf16 matrix-core kernels are not built for: float32 caches
// (small models and exact checks) and bf16 caches at head_dim 64.  It is plain VALU code with
// float32 arithmetic, one workgroup per query row: keys are scored 256 at a time into LDS, then
// the weighted value sum runs with lanes over head dimensions so V rows are read coalesced.
// Options, both for bf16 rows:
//  * fused RoPE of the query: the query row is turned to its position with the delta-angle
//    table (the re-rotation kernel's float32 arithmetic, one bf16 rounding), as if turned by
//    pic_rerotate_keys first;
//  * paged keys (zero-copy composition): a context slot's K/V come from the pool through the
//    token-level slot map, the key turned by the slot's shift with the compose kernel's
//    float32 arithmetic and bf16 rounding (Sec. 2, Eq. 3), so the result equals composing
//    first; slots at or past the request's context length come from the cache.
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

__device__ __forceinline__ float ld(const float* p) { return *p; }
__device__ __forceinline__ float ld(const bf16_t* p) { return __uint_as_float((uint32_t)*p << 16); }
__device__ __forceinline__ void st(float* p, float x) { *p = x; }
__device__ __forceinline__ void st(bf16_t* p, float x) {
  *p = (bf16_t)(pack_bf16x2(x, 0.f) & 0xFFFFu);
}
__device__ __forceinline__ float round_bf16(float x) { return __uint_as_float(pack_bf16x2(x, 0.f) << 16); }

// (x, y) turned by the angle with cosine c and sine s, in the float32 form of the re-rotation
// and compose kernels
__device__ __forceinline__ void turn(float& x, float& y, float c, float s) {
  const float u = x, v = y;
  x = fmaf(u, c, -(v * s));
  y = fmaf(u, s, v * c);
}

template <typename T, int HD, bool kPaged>
__global__ void __launch_bounds__(kThreads) attn_rows_kernel(RowArgs<T> a) {
  constexpr int G = kThreads / HD;  // key groups in the value pass
  constexpr int HALF = HD / 2;
  __shared__ float q_s[HD];
  __shared__ float p_s[kThreads];
  __shared__ float red[kThreads / 64];
  __shared__ float o_s[G][HD];

  const AttnShape& s = a.s;
  const int Hq = s.n_q_heads, Hkv = s.n_kv_heads, n_q = a.n_q;
  const int l = blockIdx.y;
  const int64_t row = blockIdx.x;  // ((b * n_q + i) * Hq + h)
  const int h = (int)(row % Hq);
  const int i = (int)((row / Hq) % n_q);
  const int b = (int)(row / ((int64_t)Hq * n_q));
  const int g = h / (Hq / Hkv);

  const int64_t qpos = a.pos(b, i);
  if (qpos < 0) return;   // (uniform) an unused row
  int64_t n_vis = qpos + 1;
  if (n_vis > s.cache_cap) n_vis = s.cache_cap;

  const int64_t qrow = ((int64_t)l * s.batch * n_q * Hq + row) * HD;
  for (int d = threadIdx.x; d < HD; d += kThreads) q_s[d] = ld(a.q + qrow + d);
  if (a.q_table != nullptr) {   // fused RoPE: the query turned to its position, rounded to bf16
    __syncthreads();
    const float2* trow = a.q_table + (int64_t)l * a.table_stride + (int64_t)min(qpos, (int64_t)a.max_abs_delta) * HALF;
    float x = 0.f, y = 0.f;
    int ix = 0, iy = 0;
    if (threadIdx.x < HALF) {   // pair f = threadIdx.x
      const int f = threadIdx.x;
      ix = a.interleaved ? 2 * f : f;
      iy = a.interleaved ? 2 * f + 1 : f + HALF;
      x = q_s[ix];
      y = q_s[iy];
      turn(x, y, trow[f].x, trow[f].y);
    }
    __syncthreads();
    if (threadIdx.x < HALF) {
      q_s[ix] = round_bf16(x);
      q_s[iy] = round_bf16(y);
    }
  }
  const int64_t kv0 = (((int64_t)l * s.batch + b) * Hkv + g) * s.cache_cap * HD;
  const T* K = a.cache_k + kv0;
  const T* V = a.cache_v + kv0;
  // paged: context slots below ctx come from the pool through the slot map
  int32_t ctx = 0;
  const T* PK = nullptr;
  const T* PV = nullptr;
  const float2* ktab = nullptr;
  if constexpr (kPaged) {
    ctx = clamp_len(a.ctx_len[b], a.max_ctx);
    PK = a.pool_k + ((int64_t)l * Hkv + g) * a.pool_tokens * HD;
    PV = a.pool_v + ((int64_t)l * Hkv + g) * a.pool_tokens * HD;
    ktab = a.k_table + (int64_t)l * a.table_stride;
  }
  __syncthreads();

  const int dd = threadIdx.x % HD, grp = threadIdx.x / HD;
  float m = -INFINITY, lsum = 0.f, acc = 0.f;
  for (int64_t c0 = 0; c0 < n_vis; c0 += kThreads) {
    const int64_t j = c0 + threadIdx.x;
    float sc = -INFINITY;
    if (j < n_vis) {
      float dot = 0.f;
      if (kPaged && j < ctx) {   // a document slot: its pool row, turned by the slot's shift
        const int32_t src = clamp_pool_token(a.smap[(int64_t)b * a.map_cap + j], a.pool_tokens);
        const int32_t dl = clamp_delta(a.dmap[(int64_t)b * a.map_cap + j], a.max_abs_delta);
        const float2* trow = ktab + (int64_t)(dl < 0 ? -dl : dl) * HALF;
        const T* kr = PK + (int64_t)src * HD;
        // element d in order (the summation order of a cached key): its pair turned, rounded
        for (int d = 0; d < HD; ++d) {
          const int f = a.interleaved ? d >> 1 : (d < HALF ? d : d - HALF);
          const bool first = a.interleaved ? (d & 1) == 0 : d < HALF;
          const int ix = a.interleaved ? 2 * f : f, iy = a.interleaved ? 2 * f + 1 : f + HALF;
          float x = ld(kr + ix), y = ld(kr + iy);
          const float2 cs = trow[f];
          turn(x, y, cs.x, dl < 0 ? -cs.y : cs.y);
          dot = fmaf(q_s[d], round_bf16(first ? x : y), dot);
        }
      } else {
        const T* kr = K + j * HD;
        for (int d = 0; d < HD; ++d) dot = fmaf(q_s[d], ld(kr + d), dot);
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
    float acc_t = 0.f;
    for (int jj = grp; jj < n_here; jj += G) {
      const int64_t k = c0 + jj;
      const T* vr;
      if (kPaged && k < ctx)
        vr = PV + (int64_t)clamp_pool_token(a.smap[(int64_t)b * a.map_cap + k], a.pool_tokens) * HD;
      else
        vr = V + k * HD;
      acc_t = fmaf(p_s[jj], ld(vr + dd), acc_t);
    }
    acc = acc * alpha + acc_t;
    __syncthreads();
  }
  o_s[grp][dd] = acc;
  __syncthreads();
  if (threadIdx.x < HD) {
    float o = 0.f;
#pragma unroll
    for (int k = 0; k < G; ++k) o += o_s[k][threadIdx.x];
    st(a.out + qrow + threadIdx.x, o / lsum);
  }
}

template <typename T, int HD>
hipError_t launch_rows(const RowArgs<T>& a) {
  const int64_t rows = (int64_t)a.s.batch * a.n_q * a.s.n_q_heads;
  if (rows == 0 || a.s.n_layers == 0) return hipSuccess;
  const dim3 grid((unsigned)rows, a.s.n_layers);
  if (a.pool_k != nullptr)
    hipLaunchKernelGGL((attn_rows_kernel<T, HD, true>), grid, dim3(kThreads), 0, a.stream, a);
  else
    hipLaunchKernelGGL((attn_rows_kernel<T, HD, false>), grid, dim3(kThreads), 0, a.stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_rows(const RowArgs<float>& a) {
  return a.s.head_dim == 64 ? launch_rows<float, 64>(a) : launch_rows<float, 128>(a);
}

hipError_t launch_attn_rows(const RowArgs<bf16_t>& a) {
  return a.s.head_dim == 64 ? launch_rows<bf16_t, 64>(a) : launch_rows<bf16_t, 128>(a);
}

}  // namespace pic
