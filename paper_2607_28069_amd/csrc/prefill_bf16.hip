// Suffix prefill attention on bf16 MFMA (App. C.1: inline tokens attend over the linked cache
// under the frontier causal mask; Sec. 5 "Cache-hit serving").
//
// Problem per (layer, request b, kv head g): M = n_q * n_rep query rows (the n_rep query
// heads of kv head g are packed into the row dimension, row r = token r / n_rep, head
// g * n_rep + r % n_rep).  A query token at position p sees keys [0, p].  Suffix mode: token
// i sits at ctx + i after the composed context (n_keys = ctx + n_q).  Table mode (general
// frontier layout, inline tokens interleaved with documents): token i sits at a position
// from a table, and a workgroup's key range ends at its furthest row's position.  Only tiles
// past a workgroup's nearest row position need a mask.
//
// Kernel shape (gfx950, wave64):
//  * 8 waves per workgroup, 32 query rows per wave (256 rows per workgroup), key tiles of 64:
//    every K/V tile brought into LDS serves 256 query rows.
//  * Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: A = K rows
//    from LDS, B = Q^T held in registers for the whole key loop.  In the accumulator layout
//    each lane then owns ONE query column and 32 of the tile's keys, so the row max needs a
//    single cross-lane exchange (lane l <-> l ^ 32) and the row sum none until the end.
//  * O^T = V^T P^T with the same instruction: the probabilities, rounded to bf16, are already
//    in the B-operand layout (keys along k) once the tile's keys are numbered in the order
//    the accumulator holds them.  V stays row-major in LDS; its A operand (8 keys at one head
//    dim per lane) comes from two transposing reads (ds_read_b64_tr_b16), which also apply
//    that key order.
//  * Tiles move global -> LDS with buffer_load_dwordx4 ... lds (no register staging).  The
//    16-byte chunks of a row are XOR-swizzled so that every LDS read is free of bank conflicts.
//  * Software pipeline, one barrier per tile: K runs one tile ahead of V.  While the matrix
//    core computes the scores of tile t+1, the vector unit turns the scores of tile t into
//    probabilities, which then feed the PV products of tile t.  The tile body is ordered by
//    hand (scheduling barriers): each LDS operand is read one product ahead of its use, and
//    the PV products of a tile's last slice are issued after the tile barrier, covering the
//    latency of the next tile's first reads.
//  * Head dim D = 128 in every mode, or 64 in the suffix and table modes.  At 64 a row is 8
//    chunks, one load instruction moves 8 rows, the score chains take 4 k steps and the output
//    2 blocks of 32 dims; the tile body keeps its order, with one score product per two pairs
//    of probabilities (the exponentials per flop double, so the vector unit limits it sooner).
//  * Workgroups sharing a (request, kv head) key stream are mapped onto the same XCD (blocks
//    are dealt round-robin over the 8 XCDs), so that stream is fetched into one L2.
//  * The suffix's own keys/values are read straight from k_suf / v_suf; the workgroups of a
//    (request, kv head) also store them into cache slots [ctx, ctx + n_suffix), each a share
//    of the rows (no separate append launch, and no workgroup reads those slots from the cache).
//  * Paged mode (zero-copy composition): the documents' rows come straight from the pool
//    through the token-level slot map (pool token and position shift of every context slot);
//    the composed cache is not written.  A key tile that is one pool run under one shift (the
//    tile map says so) is loaded like a cache tile and the wave turns its queries by -shift
//    for that tile's scores instead of turning 64 keys (RoPE's relative property; the turned
//    operand is rebuilt from an unturned copy in LDS whenever the shift changes).  Any other
//    tile is loaded row by row and each wave turns the key rows it loaded by their shift
//    (Eq. 3) in LDS, with the same float32 arithmetic and rounding as the compose kernel,
//    before the tile is used.
#include <climits>
#include <type_traits>

#include "pic_bounds.h"
#include "pic_internal.h"

namespace pic {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kRowsPerWave = 32;
constexpr int kRowsPerWG = kWaves * kRowsPerWave;
constexpr int kKeys = 64;                      // keys per tile
constexpr int kNumXcd = 8;
// Sizes that follow the head dim D (128; or 64 in the suffix and table modes).  A row is D / 8
// 16-byte chunks, and one 1 KB load instruction of a wave moves 64 / (D / 8) rows of a tile.
template <int HD>
struct Dims {
  static constexpr int kRowBytes = HD * 2;                   // 256 at D = 128
  static constexpr int kTileBytes = kKeys * kRowBytes;       // 16 KB at D = 128
  static constexpr int kChunks = HD / 8;                     // 16-byte chunks per row
  static constexpr int kRowsPerLoad = 64 / kChunks;          // rows per 1 KB load instruction
  static constexpr int kLoadSteps = kKeys / (kRowsPerLoad * kWaves);   // per wave and tile
  static constexpr int kKSteps = HD / 16;                    // k steps of a score product
  static constexpr int kDBlocks = HD / 32;                   // 32-dim blocks of the output
};
static_assert(kRowsPerWG == kPrefillRowsPerWG && kKeys == kPrefillKeys, "host split planner tiling");

#define LDS_AS __attribute__((address_space(3)))
#define GLOBAL_AS __attribute__((address_space(1)))

// Global -> LDS moves go through buffer instructions (buffer_load_dwordx4 ... lds): a wave-
// uniform base in a buffer resource, a uniform byte offset (soffset) and a per-lane byte
// offset.  (The global-address form of the same move counts as an access to both memory and
// LDS, and the compiler then waits for every outstanding load before any LDS read result or
// any global load result is used; the buffer form keeps those waits to the operands needed.)
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t make_rsrc(const void* base) {
  // raw buffer (stride 0), no range limit: every offset the kernel forms is in bounds
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, -1, 0x00020000);
}
// 16 bytes per lane from base + soff + voff into LDS at lds + 16 * lane
__device__ __forceinline__ void dma16(rsrc_t r, uint32_t voff, uint32_t soff, void* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (LDS_AS void*)lds, 16, voff, soff, 0, 0);
}
// the same move in the indexed form (index 0), for the second of two moves under
// complementary lane masks, so the compiler cannot fold the two into one
__device__ __forceinline__ void dma16_other(rsrc_t r, uint32_t voff, void* lds) {
  __builtin_amdgcn_struct_ptr_buffer_load_lds(r, (LDS_AS void*)lds, 16, 0, voff, 0, 0, 0);
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// Key order inside a tile as the S^T accumulator hands probabilities to the B operand of the
// PV product: k index kappa <-> key with bits 2 and 3 swapped (an involution).
__device__ __forceinline__ int key_perm(int key) {
  return (key & ~12) | ((key & 4) << 1) | ((key & 8) >> 1);
}

// Byte offset of 16-byte chunk c of tile row `key`.  K is read 16 bytes per lane across 32
// rows, V 8 bytes per lane across 4 rows by the transposing read; each has its own XOR
// swizzle of the chunk index that keeps those reads free of bank conflicts (for 32 or 64
// four-byte banks at D = 128).  At D = 64 a row is 128 bytes, half of the 64 banks' span, so
// rows of the same parity share banks: K's swizzle takes key bits 1..3 (the 16 lanes of a
// read phase, rows n .. n + 15 at one chunk, land on 16 distinct (parity, chunk) pairs), V's
// moves rows 2 and 3 of each group of four to the other four-chunk half (the 4 rows x 4
// chunks of a 32-lane phase cover all 64 banks once).
template <int HD>
__device__ __forceinline__ int k_swz(int key) {
  if constexpr (HD == 128) return key & 15;
  else return (key >> 1) & 7;
}
template <int HD>
__device__ __forceinline__ int v_swz(int key) {
  if constexpr (HD == 128) return ((key & 3) * 5) & 15;
  else return (key & 2) << 1;
}
template <int HD>
__device__ __forceinline__ int k_off(int key, int c) { return key * Dims<HD>::kRowBytes + ((c ^ k_swz<HD>(key)) << 4); }
template <int HD>
__device__ __forceinline__ int v_off(int key, int c) { return key * Dims<HD>::kRowBytes + ((c ^ v_swz<HD>(key)) << 4); }

// Two ways to place the query tokens (n_suffix per request):
//  * suffix: token i of request b at position ctx_len[b] + i, after the composed context;
//    its K/V come from k_suf / v_suf and are stored into the cache by this kernel;
//  * table (general frontier layout): token i at q_pos[b * n_suffix + i] for i < n_valid[b];
//    every visible slot, the tokens' own included, is already in the cache.
struct PrefillArgs {
  // paged mode: the pool, the slot map and the delta-angle table
  const bf16_t* pool_k;     // [L][Hkv][pool_tokens][D]
  const bf16_t* pool_v;
  int64_t pool_tokens;
  const int32_t* smap;      // [B][map_cap] pool token of each context slot
  const int32_t* dmap;      // [B][map_cap] position shift of each context slot
  int32_t map_cap;
  const int32_t* tmap;      // [B][map_tiles][2] (pool token of a tile's first key, shift) of
                            // tiles that are one pool run with one shift, else (-1, 0); or NULL
  int32_t map_tiles;
  const float2* table;      // [L or 1][max_abs_delta + 1][D/2]
  int64_t table_stride;
  int32_t max_abs_delta;
  const bf16_t* q;
  const bf16_t* k_suf;      // [L][B][n_suffix][Hkv][D]
  const bf16_t* v_suf;
  bf16_t* cache_k;
  bf16_t* cache_v;
  const int32_t* ctx_len;
  const int32_t* q_pos;     // table mode: [B][n_suffix]
  const int32_t* n_valid;   // table mode: [B]
  int32_t max_pos;          // table mode: positions are clamped to [0, max_pos]
  bf16_t* out;
  int32_t max_ctx, n_suffix, batch, cache_cap, n_q_heads, n_kv_heads;
  int32_t n_rep;            // n_q_heads / n_kv_heads
  uint64_t rep_magic;       // ceil(2^32 / n_rep): x / n_rep = (x * rep_magic) >> 32 for x < 2^27
  int32_t m_tiles;          // ceil(n_suffix * n_rep / kRowsPerWG)
  int32_t n_splits;         // key-range splits per (m-tile, request, kv head)
  int32_t tiles_per_split;  // key tiles per split
  int32_t n_wg;             // m_tiles * n_splits * batch * n_kv_heads
  int64_t rows_total;       // L * batch * n_suffix * Hq (query rows of one split's partials)
  bf16_t* ws_o;             // [n_splits][rows_total][D] each split's normalised output
  float2* ws_ml;            // [n_splits][rows_total] (reference max, row sum)
  float scale_log2;
};

// Rope mode = suffix mode with the suffix queries and keys given unrotated: the kernel turns
// them to their positions (RoPE at ctx + i, from the delta-angle table) as they are loaded.
// Runs mode = paged mode with a tile map whose non-run context tiles have been composed into
// the cache beforehand: whole-run tiles come from the pool (queries turned), all others from
// the cache, so the loop carries no per-key rotation.
constexpr int kModeSuffix = 0, kModeTable = 1, kModePaged = 2, kModeRope = 3, kModeRuns = 4;

// (x, y) turned by the angle with cosine c and sine s, in the float32 arithmetic the compose
// and re-rotation kernels use, so fused and separate rotations round identically.
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
// Pairs of two 16-byte chunks x1, x2 turned by frequencies f0 .. f0 + 7 of table row `row`
// (cos, sin pairs): rotate-half pairs (x1[i], x2[i]); interleaved pairs (2i, 2i + 1) of x1 then x2.
template <bool kInterleaved>
__device__ __forceinline__ void rot_chunks(float (&x1)[8], float (&x2)[8], const float2* row, int f0) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float2 cs = row[f0 + i];
    if constexpr (kInterleaved) {
      float* x = i < 4 ? x1 : x2;
      rot_pair(x[2 * (i & 3)], x[2 * (i & 3) + 1], cs.x, cs.y);
    } else {
      rot_pair(x1[i], x2[i], cs.x, cs.y);
    }
  }
}

template <int HD, int kMode, bool kInterleaved>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
prefill_bf16_kernel(PrefillArgs a) {
  constexpr bool kTable = kMode == kModeTable, kPaged = kMode == kModePaged, kRope = kMode == kModeRope;
  constexpr bool kRuns = kMode == kModeRuns, kPool = kPaged || kRuns;   // kPool: whole-run tiles from the pool
  static_assert(HD == 128 || HD == 64, "head dim");
  constexpr int kHD = HD;
  constexpr int kRowBytes = Dims<HD>::kRowBytes, kTileBytes = Dims<HD>::kTileBytes;
  constexpr int kChunks = Dims<HD>::kChunks, kRowsPerLoad = Dims<HD>::kRowsPerLoad;
  constexpr int kLoadSteps = Dims<HD>::kLoadSteps, kKS = Dims<HD>::kKSteps, kDB = Dims<HD>::kDBlocks;
  constexpr int kHalfChunks = kChunks / 2;   // rotate-half partner of chunk c: c + C / 2
  constexpr int kQBytes = kKS * 1024;        // one wave's Q^T operand (paged mode keeps a copy)
  // Four distinct buffers (not one array indexed by parity) so the compiler can see that
  // loads in flight into one buffer do not alias reads from another.  (The larger alignment
  // places them first, at the bottom of LDS, ahead of the paged mode's bigger areas.)
  __shared__ __attribute__((aligned(4096))) uint8_t k_lds0[kTileBytes];
  __shared__ __attribute__((aligned(4096))) uint8_t k_lds1[kTileBytes];
  __shared__ __attribute__((aligned(4096))) uint8_t v_lds0[kTileBytes];
  __shared__ __attribute__((aligned(4096))) uint8_t v_lds1[kTileBytes];
  // paged and rope modes: each wave's cos/sin of the key rows it turns (4 KB per wave)
  __shared__ __attribute__((aligned(16))) uint8_t cs_lds[(kPool || kRope) ? kWaves * 4096 : 16];
  // paged mode: each wave's unturned Q^T operand (8 KB per wave), the source of every turn
  __shared__ __attribute__((aligned(16))) uint8_t q_lds[kPool ? kWaves * kQBytes : 16];

  // XCD-aware block order: hardware block w runs on XCD w % 8; give each XCD a contiguous
  // range of logical blocks so the m-tiles of one (request, kv head) share an L2.
  const int per_xcd = (a.n_wg + kNumXcd - 1) / kNumXcd;
  const int w = blockIdx.x;
  const int logical = (w % kNumXcd) * per_xcd + w / kNumXcd;
  if (logical >= a.n_wg) return;
  // m-tiles of one (request, kv head) are dispatched one after another (so they stream its
  // keys concurrently, sharing the XCD's L2), the last one first: later query rows see more
  // keys, so the longest workgroups start earliest and short ones fill the end of the launch
  const int mt = a.m_tiles - 1 - logical % a.m_tiles;
  const int split = (logical / a.m_tiles) % a.n_splits;
  const int bg = logical / (a.m_tiles * a.n_splits);
  const int b = bg / a.n_kv_heads, g = bg % a.n_kv_heads;
  const int l = blockIdx.y;

  // (divisions by n_rep as multiply-highs: uniform operands then stay in scalar registers,
  // and with them every tile count, mask decision and load path derived from them)
  const int n_rep = a.n_rep;
  auto div_rep = [&](int x) { return (int)(((uint64_t)(uint32_t)x * a.rep_magic) >> 32); };
  const int M = a.n_suffix * n_rep;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: LDS bases in SGPRs
  const int n = lane & 31, hh = lane >> 5;   // query column, lane half

  const int row0_wg = mt * kRowsPerWG;
  const int r = row0_wg + wave * kRowsPerWave + n;    // this lane's query row
  bool row_ok = r < M;
  const int tok = row_ok ? div_rep(r) : a.n_suffix - 1;
  const int hq = g * n_rep + (row_ok ? r - div_rep(r) * n_rep : 0);
  // ctx: keys below it come from the cache (suffix mode: the composed context);
  // pos_min_wg / pos_max_wg: nearest / furthest position of this workgroup's query rows
  int ctx, qpos, pos_min_wg, pos_max_wg;
  if constexpr (!kTable) {
    ctx = clamp_len(a.ctx_len[b], a.max_ctx);
    pos_min_wg = ctx + div_rep(row0_wg);
    pos_max_wg = ctx + div_rep(min(row0_wg + kRowsPerWG, M) - 1);
    qpos = ctx + tok;
  } else {
    __shared__ int red_lo[kWaves], red_hi[kWaves];
    int nv = a.n_valid[b];
    nv = nv < 0 ? 0 : (nv > a.n_suffix ? a.n_suffix : nv);
    row_ok = row_ok && tok < nv;
    int p = row_ok ? a.q_pos[(int64_t)b * a.n_suffix + tok] : -1;
    if (row_ok) p = p < 0 ? 0 : (p > a.max_pos ? a.max_pos : p);
    int lo = row_ok ? p : INT_MAX, hi = p;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      lo = min(lo, __shfl_xor(lo, o, 64));
      hi = max(hi, __shfl_xor(hi, o, 64));
    }
    if (lane == 0) {
      red_lo[wave] = lo;
      red_hi[wave] = hi;
    }
    __syncthreads();
    pos_min_wg = red_lo[0];
    pos_max_wg = red_hi[0];
#pragma unroll
    for (int i = 1; i < kWaves; ++i) {
      pos_min_wg = min(pos_min_wg, red_lo[i]);
      pos_max_wg = max(pos_max_wg, red_hi[i]);
    }
    qpos = row_ok ? p : pos_max_wg;
    ctx = pos_max_wg + 1;   // every visible key is in the cache
  }
  const int n_keys = kTable ? pos_max_wg + 1 : ctx + a.n_suffix;
  // table mode: the wave's furthest query position.  A tile that starts past it holds no key
  // any of the wave's rows sees, so the wave skips the products and exponentials of every
  // tile from there on (it still moves its share of each tile and meets each barrier).  Rows
  // of different inline spans share a workgroup, so on the general frontier layout waves
  // whose spans end early skip whole tiles.
  int wave_max = INT_MAX;
  if constexpr (kTable) {
    int wm = row_ok ? qpos : -1;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) wm = max(wm, __shfl_xor(wm, o, 64));
    wave_max = __builtin_amdgcn_readfirstlane(wm);
  }
  constexpr int kChunkShift = HD == 128 ? 4 : 3;   // log2(C)
  const int ld_row = kRowsPerLoad * wave + (lane >> kChunkShift), ld_slot = lane & (kChunks - 1);   // load row within a step
  // this workgroup's key tiles: [t0, t0 + n_tiles) of the (pos_max_wg + 1) visible keys
  const int t0 = split * a.tiles_per_split;
  const int n_tiles = min((pos_max_wg + kKeys) / kKeys - t0, a.tiles_per_split);

  const int64_t bh_kv = (((int64_t)l * a.batch + b) * a.n_kv_heads + g) * a.cache_cap;
  const bf16_t* Kg = a.cache_k + bh_kv * kHD;
  const bf16_t* Vg = a.cache_v + bh_kv * kHD;
  // suffix token i of this (request, kv head): row i with a stride of Hkv rows
  const int64_t suf0 = (((int64_t)l * a.batch + b) * a.n_suffix * a.n_kv_heads + g) * kHD;
  const int64_t suf_stride = (int64_t)a.n_kv_heads * kHD;
  const bf16_t* Ks = kTable ? nullptr : a.k_suf + suf0;
  const bf16_t* Vs = kTable ? nullptr : a.v_suf + suf0;
  // Cache assembly: the suffix rows go into slots [ctx, ctx + n_suffix), shared out over the
  // (request, kv head)'s workgroups (every m-tile and split stores a contiguous share of the
  // rows), so no workgroup carries the whole store ahead of its key loop.
  const int asm_parts = a.m_tiles * a.n_splits, asm_part = split * a.m_tiles + mt;
  const int asm_per = (a.n_suffix + asm_parts - 1) / asm_parts;
  const int asm_i0 = min(asm_part * asm_per, a.n_suffix), asm_i1 = min(asm_i0 + asm_per, a.n_suffix);
  if (kRope) {   // with the suffix keys turned to ctx + i
    // item c: row i = c / (3 C / 2), C = D / 8 chunks; part < C / 2: K chunk pair part
    // (rotate-half: chunks part, part + C / 2; interleaved: 2 part, 2 part + 1; both:
    // frequencies 8 part .. 8 part + 7), part >= C / 2: V chunk part - C / 2.  Three items per
    // thread per pass, all loads issued before any math.
    constexpr int kItems = 3 * kHalfChunks;   // per row
    const float2* trow0 = a.table + (int64_t)l * a.table_stride;
    const int total = asm_i1 * kItems;
    for (int c0 = asm_i0 * kItems + tid; c0 < total; c0 += 3 * kThreads) {
      u32x4 w1[3], w2[3];
      float4 cs[3][4];
#pragma unroll
      for (int u = 0; u < 3; ++u) {
        const int c = c0 + u * kThreads;
        if (c >= total) continue;
        const int i = c / kItems, part = c - kItems * i;
        if (part < kHalfChunks) {
          const int o1 = kInterleaved ? 16 * part : 8 * part, o2 = kInterleaved ? 16 * part + 8 : kHD / 2 + 8 * part;
          w1[u] = *reinterpret_cast<const u32x4*>(Ks + i * suf_stride + o1);
          w2[u] = *reinterpret_cast<const u32x4*>(Ks + i * suf_stride + o2);
          const float4* row = reinterpret_cast<const float4*>(trow0 + (int64_t)min(ctx + i, a.max_abs_delta) * (kHD / 2));
#pragma unroll
          for (int j = 0; j < 4; ++j) cs[u][j] = row[4 * part + j];
        } else {
          w1[u] = *reinterpret_cast<const u32x4*>(Vs + i * suf_stride + 8 * (part - kHalfChunks));
        }
      }
#pragma unroll
      for (int u = 0; u < 3; ++u) {
        const int c = c0 + u * kThreads;
        if (c >= total) continue;
        const int i = c / kItems, part = c - kItems * i;
        if (part < kHalfChunks) {
          const int o1 = kInterleaved ? 16 * part : 8 * part, o2 = kInterleaved ? 16 * part + 8 : kHD / 2 + 8 * part;
          float x1[8], x2[8];
          unpack8(w1[u], x1);
          unpack8(w2[u], x2);
          const float2* cs2 = reinterpret_cast<const float2*>(cs[u]);   // frequencies 8 part + 0..7
#pragma unroll
          for (int f = 0; f < 8; ++f) {
            if constexpr (kInterleaved) {
              float* z = f < 4 ? x1 : x2;
              rot_pair(z[2 * (f & 3)], z[2 * (f & 3) + 1], cs2[f].x, cs2[f].y);
            } else {
              rot_pair(x1[f], x2[f], cs2[f].x, cs2[f].y);
            }
          }
          bf16_t* dst = a.cache_k + (bh_kv + ctx + i) * kHD;
          *reinterpret_cast<u32x4*>(dst + o1) = pack8(x1);
          *reinterpret_cast<u32x4*>(dst + o2) = pack8(x2);
        } else {
          *reinterpret_cast<u32x4*>(a.cache_v + (bh_kv + ctx + i) * kHD + 8 * (part - kHalfChunks)) = w1[u];
        }
      }
    }
  } else if (!kTable) {
    // item c: row i = c / (2 C), 16-byte chunk c % C of K (c % 2C < C) or V, C = D / 8 chunks
    // per row; eight items per thread per pass, the loads issued before the stores
    constexpr int kU = 8, kItemShift = HD == 128 ? 5 : 4;   // log2(2 C)
    const int total = asm_i1 * 2 * kChunks;
    for (int c0 = asm_i0 * 2 * kChunks + tid; c0 < total; c0 += kU * kThreads) {
      u32x4 w[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int c = c0 + u * kThreads, i = c >> kItemShift, part = c & (2 * kChunks - 1);
        if (c < total)
          w[u] = *reinterpret_cast<const u32x4*>((part < kChunks ? Ks : Vs) + i * suf_stride + 8 * (part & (kChunks - 1)));
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int c = c0 + u * kThreads, i = c >> kItemShift, part = c & (2 * kChunks - 1);
        if (c < total)
          *reinterpret_cast<u32x4*>((part < kChunks ? a.cache_k : a.cache_v) + (bh_kv + ctx + i) * kHD + 8 * (part & (kChunks - 1))) = w[u];
      }
    }
  }
  const int64_t qrow = (((int64_t)l * a.batch + b) * a.n_suffix + tok) * a.n_q_heads + hq;

  const int64_t orow = (((int64_t)l * a.batch + b) * a.n_suffix + tok) * a.n_q_heads + hq;
  if (n_tiles <= 0) {   // (uniform) a split past this workgroup's last visible key
    if (a.n_splits > 1 && row_ok && hh == 0) a.ws_ml[split * a.rows_total + orow] = make_float2(-INFINITY, 0.f);
    return;
  }

  // ---- Q^T operand: lane (n, hh) holds q[row n][16 ks + 8 hh .. +8) for ks = 0 .. D / 16 - 1
  bf16x8_t qop[kKS];
  {
    const u32x4* qp = reinterpret_cast<const u32x4*>(a.q + qrow * kHD);
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks) qop[ks] = as_bf16x8(row_ok ? qp[2 * ks + hh] : u32x4{0, 0, 0, 0});
  }
  // rope mode: queries turned to their positions (called once the first tiles' loads are in
  // flight, so the table reads overlap them)
  auto rope_q = [&]() {
    const float2* trow = a.table + (int64_t)l * a.table_stride + (int64_t)min(qpos, a.max_abs_delta) * (kHD / 2);
    if constexpr (!kInterleaved) {
      // pairs (d, d + D / 2): operand steps ks and ks + D / 32, frequencies 16 ks + 8 hh .. + 7
#pragma unroll
      for (int ks = 0; ks < kKS / 2; ++ks) {
        float x1[8], x2[8];
        unpack8(__builtin_bit_cast(u32x4, qop[ks]), x1);
        unpack8(__builtin_bit_cast(u32x4, qop[ks + kKS / 2]), x2);
        rot_chunks<false>(x1, x2, trow, 16 * ks + 8 * hh);
        qop[ks] = as_bf16x8(pack8(x1));
        qop[ks + kKS / 2] = as_bf16x8(pack8(x2));
      }
    } else {
      // pairs (2i, 2i + 1) inside each chunk: dims 16 ks + 8 hh + 2m, frequency 8 ks + 4 hh + m
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) {
        float x[8];
        unpack8(__builtin_bit_cast(u32x4, qop[ks]), x);
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const float2 cs = trow[8 * ks + 4 * hh + m];
          rot_pair(x[2 * m], x[2 * m + 1], cs.x, cs.y);
        }
        qop[ks] = as_bf16x8(pack8(x));
      }
    }
  };
  if constexpr (kPool) {   // keep the unturned operand (lane-private slots)
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks)
      *reinterpret_cast<u32x4*>(q_lds + wave * kQBytes + (ks * 64 + lane) * 16) = __builtin_bit_cast(u32x4, qop[ks]);
  }

  // ---- global -> LDS tile loads.  Instruction i of wave w writes 1 KB of LDS = tile rows
  // 4 (kWaves i + w) .. +3, lane `lane` landing at byte 16 * lane: row 4 kWaves i + 4 w +
  // lane / 16, chunk slot lane % 16, filled from the global chunk the swizzle puts in that
  // slot.  The swizzles use key bits 0..3 (K) and 0..1 (V), which do not change with i, so
  // each lane's source offset within one step is a constant.  Rows past the last key (only in the last
  // tile) are clamped to it: their scores are masked, so they enter PV with probability 0.
  const int k_goff = ld_row * kHD + 8 * (ld_slot ^ k_swz<HD>(ld_row));   // elements
  const int v_goff = ld_row * kHD + 8 * (ld_slot ^ v_swz<HD>(ld_row));
  const int v_gc = ld_slot ^ v_swz<HD>(ld_row), k_gc = ld_slot ^ k_swz<HD>(ld_row);
  // paged mode: pool rows of this (layer, kv head), and the slot map of this request
  const bf16_t* PKg = kPool ? a.pool_k + ((int64_t)l * a.n_kv_heads + g) * a.pool_tokens * kHD : nullptr;
  const bf16_t* PVg = kPool ? a.pool_v + ((int64_t)l * a.n_kv_heads + g) * a.pool_tokens * kHD : nullptr;
  const int32_t* smap = kPaged ? a.smap + (int64_t)b * a.map_cap : nullptr;
  // buffer resources (byte offsets from these bases fit in 32 bits: a cache stream holds
  // cache_cap rows, the suffix n_suffix * Hkv rows, a pool head pool_tokens rows and a
  // table (max_abs_delta + 1) rows of 512 bytes, each under 2^32 bytes by the host checks)
  const rsrc_t r_k = make_rsrc(Kg), r_v = make_rsrc(Vg);
  const rsrc_t r_ks = make_rsrc(kTable ? Kg : Ks), r_vs = make_rsrc(kTable ? Vg : Vs);
  const rsrc_t r_pk = make_rsrc(kPool ? PKg : Kg), r_pv = make_rsrc(kPool ? PVg : Vg);
  const rsrc_t r_tab = make_rsrc((kPool || kRope) ? a.table + (int64_t)l * a.table_stride : (const float2*)Kg);
  const int32_t* dmap = kPaged ? a.dmap + (int64_t)b * a.map_cap : nullptr;
  // pool token of load row i (0, 1) of global tile t for this lane (0 past the context)
  // (map entries are loaded raw and checked after the tile's loads have landed: a use right
  // after the load would make the wave wait for every load in flight, the tile's included)
  auto raw_src = [&](int t, int i) -> int32_t {   // ctx > 0
    return smap[min(t * kKeys + kRowsPerLoad * kWaves * i + ld_row, ctx - 1)];
  };
  auto fin_src = [&](int t, int i, int32_t v) -> int32_t {
    if (t * kKeys + kRowsPerLoad * kWaves * i + ld_row >= ctx) v = 0;
    return clamp_pool_token(v, a.pool_tokens);
  };
  auto map_src = [&](int t, int i) { return ctx > 0 ? fin_src(t, i, raw_src(t, i)) : 0; };
  // rotation item of this lane: one of the wave's own load rows, 16-byte chunks c and c + C / 2.
  // D = 128: row 32 i + 4 w + rr (i = lane / 32, rr = (lane / 8) % 4), c = lane % 8.  D = 64: row
  // 8 w + (lane / 4) % 8, c = lane % 4; lanes 32 .. 63 repeat the items of lanes 0 .. 31 (rot_on
  // false: they stage the same cos/sin and leave the rows to their twins).
  const int rot_row = HD == 128 ? 32 * (lane >> 5) + 4 * wave + ((lane >> 3) & 3) : 8 * wave + ((lane >> 2) & 7);
  const int rot_c = lane & (kHalfChunks - 1);
  const bool rot_on = HD == 128 || lane < 32;
  // shift of this lane's rotation row of global tile t (0 past the context)
  auto raw_delta = [&](int t) -> int32_t { return dmap[min(t * kKeys + rot_row, ctx - 1)]; };   // ctx > 0
  auto fin_delta = [&](int t, int32_t d) -> int32_t {
    if (t * kKeys + rot_row >= ctx) d = 0;
    return clamp_delta(d, a.max_abs_delta);
  };
  auto map_delta = [&](int t) { return ctx > 0 ? fin_delta(t, raw_delta(t)) : 0; };
  // cos/sin of the lane's 8 pair frequencies at |delta| into this wave's cos/sin area:
  // instruction j moves float pairs (f_j, f_j + 1) to byte j * 1 KB + 16 * lane
  // (a lane reloads only when its |shift| changes: a document keeps one shift for all its tiles)
  int32_t cs_held = -1;   // |shift| whose per-lane cos/sin this lane's area holds (-1: none)
  auto load_cs = [&](int32_t delta) {
    const int32_t ad = delta < 0 ? -delta : delta;
    if (ad == cs_held) return;
    cs_held = ad;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // rotate-half: pairs 8c .. 8c + 7 (chunks c and c + C / 2); interleaved: pairs 4c .. 4c + 3
      // (chunk c) and D / 4 + 4c .. D / 4 + 4c + 3 (chunk c + C / 2)
      const int f = kInterleaved ? (j < 2 ? 4 * rot_c + 2 * j : kHD / 4 + 4 * rot_c + 2 * (j - 2)) : 8 * rot_c + 2 * j;
      dma16(r_tab, (uint32_t)(ad * (kHD / 2) + f) * 8u, 0, cs_lds + wave * 4096 + j * 1024);
    }
  };
  // Paged mode, whole-run tiles: when the 64 keys of context tile T are pool tokens
  // src .. src + 63 with one shift delta (the tile map says so, and the run lies inside the
  // pool, the table and the context), the tile is loaded like a cache tile (one base address)
  // and, instead of turning its 64 keys by delta, the wave turns its queries by -delta for
  // that tile's scores: <R(-delta) q, k> = <q, R(delta) k> (Eq. 3 and RoPE's relative
  // property).  Other tiles take the per-key path.  Returns src (uniform), or -1.
  // The tile map entries are read 64 tiles at a time (lane j: tile win + j) and taken out
  // with readlane, so a tile costs no memory instruction for them.
  int32_t win = INT_MIN / 2, w_src = -1, w_del = 0;
  auto tile_run = [&](int T, int32_t& delta) -> int32_t {   // T uniform
    delta = 0;
    if (a.tmap == nullptr || T >= a.map_tiles || (T + 1) * kKeys > ctx) return -1;
    if (T < win || T >= win + 64) {   // refill the window
      win = T;
      const int Tj = T + lane;
      if (Tj < a.map_tiles) {
        const int2 e = *reinterpret_cast<const int2*>(a.tmap + ((int64_t)b * a.map_tiles + Tj) * 2);
        w_src = e.x;
        w_del = e.y;
      } else {
        w_src = -1;
        w_del = 0;
      }
    }
    const int32_t src = __builtin_amdgcn_readlane(w_src, T - win);
    const int32_t d = __builtin_amdgcn_readlane(w_del, T - win);
    if (!tile_run_ok(src, d, T * kKeys, ctx, a.pool_tokens, a.max_abs_delta)) return -1;
    delta = d;
    return src;
  };
  // Turn the Q^T operand (from its unturned copy) by -shift, in float32, rounded to bf16.
  // The cos/sin row of |shift| must have been staged in this wave's cos/sin area
  // (stage_row, landed); shift 0 restores the unturned operand.
  int32_t q_shift = 0;   // shift the operand is turned by (uniform)
  auto stage_row = [&](int32_t shift) {
    const int32_t ad = shift < 0 ? -shift : shift;
    if (lane < kHD / 4)   // 32 lanes x 16 bytes = the row's 64 (cos, sin) pairs
      dma16(r_tab, 16u * lane, (uint32_t)ad * (kHD / 2) * 8u, cs_lds + wave * 4096);
    cs_held = -1;
  };
  auto turn_q = [&](int32_t shift) {
    if (shift == q_shift) return;
    q_shift = shift;
    const uint8_t* qs = q_lds + wave * kQBytes + lane * 16;
    if (shift == 0) {
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) qop[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(qs + ks * 1024));
      return;
    }
    const float sg = shift < 0 ? -1.f : 1.f;   // sin(shift theta) = sg * sin(|shift| theta)
    const float4* row = reinterpret_cast<const float4*>(cs_lds + wave * 4096);
    cs_held = -1;
    auto unpack = [](u32x4 w, float (&x)[8]) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[2 * e] = __uint_as_float(w[e] << 16);
        x[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
      }
    };
    auto pack = [](const float (&x)[8]) {
      return as_bf16x8(u32x4{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                             pack_bf16x2(x[6], x[7])});
    };
    // (x, y) -> (x cos + y sin, y cos - x sin): the pair turned by -shift
    auto turn = [](float& x, float& y, float c, float sn) {
      const float u = x, v = y;
      x = fmaf(u, c, v * sn);
      y = fmaf(v, c, -(u * sn));
    };
    if constexpr (!kInterleaved) {
      // pairs (d, d + D / 2): operand steps ks and ks + D / 32, frequencies 16 ks + 8 hh + j
#pragma unroll
      for (int ks = 0; ks < kKS / 2; ++ks) {
        float x[8], y[8];
        unpack(*reinterpret_cast<const u32x4*>(qs + ks * 1024), x);
        unpack(*reinterpret_cast<const u32x4*>(qs + (ks + kKS / 2) * 1024), y);
#pragma unroll
        for (int j4 = 0; j4 < 4; ++j4) {
          const float4 cs = row[8 * ks + 4 * hh + j4];
          turn(x[2 * j4], y[2 * j4], cs.x, sg * cs.y);
          turn(x[2 * j4 + 1], y[2 * j4 + 1], cs.z, sg * cs.w);
        }
        qop[ks] = pack(x);
        qop[ks + kKS / 2] = pack(y);
      }
    } else {
      // pairs (2i, 2i + 1) inside each chunk: frequencies 8 ks + 4 hh + m
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) {
        float x[8];
        unpack(*reinterpret_cast<const u32x4*>(qs + ks * 1024), x);
#pragma unroll
        for (int m2 = 0; m2 < 2; ++m2) {
          const float4 cs = row[4 * ks + 2 * hh + m2];
          turn(x[4 * m2], x[4 * m2 + 1], cs.x, sg * cs.y);
          turn(x[4 * m2 + 2], x[4 * m2 + 3], cs.z, sg * cs.w);
        }
        qop[ks] = pack(x);
      }
    }
  };
  int32_t src_v[kLoadSteps], src_k[kLoadSteps], src_f[kLoadSteps];   // rows of tiles t+1, t+2, t+3
  int32_t d_k = 0, d_f = 0;                                            // rotation shift, tiles t+2, t+3

  auto load_tile = [&](uint8_t* dst_tile, int t, bool is_v, int32_t run = -1) {
    const uint32_t goff = 2u * (is_v ? v_goff : k_goff);   // bytes
    const uint32_t coff = 16u * (is_v ? v_gc : k_gc);
    const rsrc_t rc = is_v ? r_v : r_k, rs = is_v ? r_vs : r_ks;
    if (kPool && run >= 0) {   // a whole-run tile: pool rows run .. run + 63
#pragma unroll
      for (int i = 0; i < kLoadSteps; ++i)
        dma16(is_v ? r_pv : r_pk, goff, (uint32_t)(run + kRowsPerLoad * kWaves * i) * kRowBytes,
              dst_tile + (kRowsPerLoad * kWaves * i + kRowsPerLoad * wave) * kRowBytes);
    } else if constexpr (kPaged) {
      const int32_t* rows = is_v ? src_v : src_k;
#pragma unroll
      for (int i = 0; i < kLoadSteps; ++i) {
        const int kk = min(t * kKeys + kRowsPerLoad * kWaves * i + ld_row, n_keys - 1);
        uint8_t* dst = dst_tile + (kRowsPerLoad * kWaves * i + kRowsPerLoad * wave) * kRowBytes;
        // (two separate moves: one move with a per-lane choice of base would need a loop
        // over the distinct bases)
        if (kk < ctx) dma16(is_v ? r_pv : r_pk, (uint32_t)rows[i] * kRowBytes + coff, 0, dst);
        if (kk >= ctx) dma16_other(rs, (uint32_t)((kk - ctx) * suf_stride) * 2u + coff, dst);
      }
    } else if ((t + 1) * kKeys <= ctx) {
#pragma unroll
      for (int i = 0; i < kLoadSteps; ++i)
        dma16(rc, goff, (uint32_t)(t * kKeys + kRowsPerLoad * kWaves * i) * kRowBytes,
              dst_tile + (kRowsPerLoad * kWaves * i + kRowsPerLoad * wave) * kRowBytes);
    } else {
      // a tile reaching the suffix: its keys come from k_suf / v_suf
#pragma unroll
      for (int i = 0; i < kLoadSteps; ++i) {
        const int kk = min(t * kKeys + kRowsPerLoad * kWaves * i + ld_row, n_keys - 1);
        uint8_t* dst = dst_tile + (kRowsPerLoad * kWaves * i + kRowsPerLoad * wave) * kRowBytes;
        if (kk < ctx) dma16(rc, (uint32_t)kk * kRowBytes + coff, 0, dst);
        if (kk >= ctx) dma16_other(rs, (uint32_t)((kk - ctx) * suf_stride) * 2u + coff, dst);
      }
    }
  };
  // Paged mode: turn this lane's item of the wave's own rows of K tile t (in `kt`, landed)
  // by its shift, as the compose kernel does: fp32 x cos - y sin, x sin + y cos, rounded to
  // bf16.  Context rows only: suffix rows and clamped rows stay as loaded.
  auto rotate_own = [&](uint8_t* kt, int t, int32_t delta) {
    if (t * kKeys + rot_row >= ctx || !rot_on) return;
    uint8_t* p1 = kt + rot_row * kRowBytes + ((rot_c ^ k_swz<HD>(rot_row)) << 4);
    uint8_t* p2 = kt + rot_row * kRowBytes + (((rot_c + kHalfChunks) ^ k_swz<HD>(rot_row)) << 4);
    const u32x4 w1 = *reinterpret_cast<const u32x4*>(p1);
    const u32x4 w2 = *reinterpret_cast<const u32x4*>(p2);
    float cs[8], sn[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float4 v = *reinterpret_cast<const float4*>(cs_lds + wave * 4096 + j * 1024 + 16 * lane);
      cs[2 * j] = v.x;
      sn[2 * j] = delta < 0 ? -v.y : v.y;
      cs[2 * j + 1] = v.z;
      sn[2 * j + 1] = delta < 0 ? -v.w : v.w;
    }
    float x1[8], x2[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x1[2 * e] = __uint_as_float(w1[e] << 16);
      x1[2 * e + 1] = __uint_as_float(w1[e] & 0xFFFF0000u);
      x2[2 * e] = __uint_as_float(w2[e] << 16);
      x2[2 * e + 1] = __uint_as_float(w2[e] & 0xFFFF0000u);
    }
    auto turn = [](float& u, float& v, float c, float s) {
      const float x = u, y = v;
      u = fmaf(x, c, -(y * s));
      v = fmaf(x, s, y * c);
    };
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      if constexpr (kInterleaved) {   // pairs (2e, 2e + 1) of each chunk; chunk c + C / 2 uses cs[4..7]
        float* x = k < 4 ? x1 : x2;
        turn(x[2 * (k & 3)], x[2 * (k & 3) + 1], cs[k], sn[k]);
      } else {
        turn(x1[k], x2[k], cs[k], sn[k]);
      }
    }
    *reinterpret_cast<u32x4*>(p1) = u32x4{pack_bf16x2(x1[0], x1[1]), pack_bf16x2(x1[2], x1[3]),
                                         pack_bf16x2(x1[4], x1[5]), pack_bf16x2(x1[6], x1[7])};
    *reinterpret_cast<u32x4*>(p2) = u32x4{pack_bf16x2(x2[0], x2[1]), pack_bf16x2(x2[2], x2[3]),
                                         pack_bf16x2(x2[4], x2[5]), pack_bf16x2(x2[6], x2[7])};
  };
  auto wait_loads = [&]() { __builtin_amdgcn_s_waitcnt(0x0F70); };   // vmcnt(0)
  // Rope mode: turn the suffix rows (keys ctx .. n_keys - 1) of K tile t, landed in `kt`, to
  // their positions; this lane's item is chunks rot_c and rot_c + C / 2 of row rot_row.
  auto rope_cs = [&](int t) {   // this lane's cos/sin for its suffix row of K tile t -> cos/sin area
    const int k = t * kKeys + rot_row;
    if (k < ctx || k >= n_keys) return;
    const uint32_t row = (uint32_t)min(k, a.max_abs_delta) * (kHD / 2);
#pragma unroll
    for (int j = 0; j < 4; ++j) {   // the frequency pairs the paged key turn uses (see load_cs)
      const int f = kInterleaved ? (j < 2 ? 4 * rot_c + 2 * j : kHD / 4 + 4 * rot_c + 2 * (j - 2)) : 8 * rot_c + 2 * j;
      dma16(r_tab, (row + f) * 8u, 0, cs_lds + wave * 4096 + j * 1024);
    }
  };
  auto rope_own = [&](uint8_t* kt, int t) {   // after rope_cs(t) has landed
    const int k = t * kKeys + rot_row;
    if (k < ctx || k >= n_keys || !rot_on) return;
    uint8_t* p1 = kt + rot_row * kRowBytes + ((rot_c ^ k_swz<HD>(rot_row)) << 4);
    uint8_t* p2 = kt + rot_row * kRowBytes + (((rot_c + kHalfChunks) ^ k_swz<HD>(rot_row)) << 4);
    float x1[8], x2[8];
    unpack8(*reinterpret_cast<const u32x4*>(p1), x1);
    unpack8(*reinterpret_cast<const u32x4*>(p2), x2);
    float cs[8], sn[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float4 v = *reinterpret_cast<const float4*>(cs_lds + wave * 4096 + j * 1024 + 16 * lane);
      cs[2 * j] = v.x;
      sn[2 * j] = v.y;
      cs[2 * j + 1] = v.z;
      sn[2 * j + 1] = v.w;
    }
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      if constexpr (kInterleaved) {   // chunk c: pairs of frequencies 4 c ..; chunk c + C / 2: D / 4 + 4 c ..
        float* x = f < 4 ? x1 : x2;
        rot_pair(x[2 * (f & 3)], x[2 * (f & 3) + 1], cs[f], sn[f]);
      } else {                         // pairs (d, d + D / 2): frequencies 8 c ..
        rot_pair(x1[f], x2[f], cs[f], sn[f]);
      }
    }
    *reinterpret_cast<u32x4*>(p1) = pack8(x1);
    *reinterpret_cast<u32x4*>(p2) = pack8(x2);
  };

  // ---- per-lane LDS read offsets, fixed for the whole loop (buffer, 32-row block and
  // 16-row slice steps are immediate offsets)
  int k_rd[kKS];   // S^T A operand: row n, chunk 2 ks + hh
#pragma unroll
  for (int ks = 0; ks < kKS; ++ks) k_rd[ks] = k_off<HD>(n, 2 * ks + hh);
  // Transposing reads of V^T: 16-lane group G = lane / 16, lane j = lane % 16 = 4 rr + qq
  // points at row key_perm(16 s4 + 8 hh + 4 half + rr) = 16 s4 + 8 half + 4 hh + rr, head dims
  // 32 db + 16 (G & 1) + 4 qq .. +3; lane i of the group then receives head dim
  // 32 db + (lane & 31) of those 4 rows.
  const int tr_rr = (lane & 15) >> 2, tr_qq = lane & 3, tr_g1 = (lane >> 4) & 1;
  int v_rd[kDB][2];
#pragma unroll
  for (int db = 0; db < kDB; ++db)
#pragma unroll
    for (int half = 0; half < 2; ++half)
      v_rd[db][half] = v_off<HD>(8 * half + 4 * hh + tr_rr, 4 * db + 2 * tr_g1 + (tr_qq >> 1)) + 8 * (tr_qq & 1);

  // ---- S^T = K Q^T for one tile: two independent 32-key accumulation chains
  auto scores = [&](const uint8_t* kt, f32x16_t (&s)[2]) {
    s[0] = f32x16_t{};
    s[1] = f32x16_t{};
#pragma unroll
    for (int ks = 0; ks < kKS; ++ks)
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2) {
        const u32x4 kv = *reinterpret_cast<const u32x4*>(kt + k_rd[ks] + 32 * kb2 * kRowBytes);
        s[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kv), qop[ks], s[kb2], 0, 0, 0);
      }
  };

  f32x16_t oacc[kDB];
#pragma unroll
  for (int i = 0; i < kDB; ++i) oacc[i] = f32x16_t{};
  float m_run = -INFINITY, l_part = 0.f;
  // The PV products of a tile's last slice are issued after the tile barrier, at the start of
  // the next tile, while that tile's first LDS reads are in flight.  Pending: probabilities
  // pend_p and V^T operands pend_v (zero before the first tile: the products then add 0).
  bf16x8_t pend_p = as_bf16x8(u32x4{0, 0, 0, 0});
  bf16x8_t pend_v[kDB];
#pragma unroll
  for (int db = 0; db < kDB; ++db) pend_v[db] = as_bf16x8(u32x4{0, 0, 0, 0});
  // (not in paged mode, whose loop holds more state: there the slice is issued in its tile)
  constexpr bool kDefer = !kPaged;
  auto flush_pending = [&]() {
    if constexpr (!kDefer) return;
#pragma unroll
    for (int db = 0; db < kDB; ++db)
      oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pend_v[db], pend_p, oacc[db], 0, 0, 0);
  };

  // Both lane halves hold keys of the same query column: (x[l], x[l ^ 32]) as a pair, for
  // all lanes, from one v_permlane32_swap.
  auto pair_max = [](float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  };
  auto pair_sum = [](float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
  };

  // Scores of tile t are complete: apply the frontier mask where the tile reaches past a
  // query's position, and move the reference max if a score exceeds it by more than 2^8
  // (rescaling what has been accumulated, for the whole wave at once).  Otherwise p <= 256,
  // which float32 sums and bf16 probabilities hold without loss of relative precision.
  auto finish_scores = [&](int t, f32x16_t (&s)[2]) {   // t: global tile index
    const int k0 = t * kKeys;
    if (k0 + kKeys - 1 > pos_min_wg) {
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = k0 + 32 * kb2 + 8 * (e >> 2) + 4 * hh + (e & 3);
          if (key > qpos) s[kb2][e] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kb2][e]);
    const float m_tile = pair_max(mx) * a.scale_log2;
    if (__any(m_tile > m_run + 8.f)) {
      flush_pending();   // the pending products belong to the old reference max
      pend_p = as_bf16x8(u32x4{0, 0, 0, 0});
      const float m_new = fmaxf(m_run, m_tile);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_part *= alpha;
#pragma unroll
      for (int db = 0; db < kDB; ++db) oacc[db] *= alpha;
    }
  };

  // ---- prologue: K0, V0, K1 resident (paged: turned); scores of tile 0
  // paged mode: whole-run descriptors of tiles t+1 (V, and the scores computed during tile t)
  // and t+2 (K) as the tile loop enters tile t, with their shifts
  int32_t run_v = -1, run_k = -1, del_v = 0, del_k = 0;
  if constexpr (kPaged) {
    int32_t del0 = 0, del1 = 0;
    const int32_t run0 = tile_run(t0, del0), run1 = n_tiles > 1 ? tile_run(t0 + 1, del1) : -1;
    if (run0 >= 0 && del0 != 0) {   // the operand for the scores of tile 0
      stage_row(del0);
      wait_loads();
      turn_q(del0);
    }
#pragma unroll
    for (int i = 0; i < kLoadSteps; ++i) {
      src_k[i] = map_src(t0, i);
      src_v[i] = map_src(t0, i);
    }
    d_k = map_delta(t0);
    wait_loads();
    load_tile(k_lds0, t0, false, run0);
    load_tile(v_lds0, t0, true, run0);
    if (run0 < 0) load_cs(d_k);
#pragma unroll
    for (int i = 0; i < kLoadSteps; ++i) src_k[i] = map_src(t0 + 1, i);
    d_f = map_delta(t0 + 1);
    wait_loads();
    if (run0 < 0) rotate_own(k_lds0, t0, d_k);
    if (n_tiles > 1) {
      load_tile(k_lds1, t0 + 1, false, run1);
      if (run1 < 0) load_cs(d_f);
      // V(t0 + 1) is loaded by tile 0 and K(t0 + 2) by tile 0: their rows
#pragma unroll
      for (int i = 0; i < kLoadSteps; ++i) {
        src_v[i] = src_k[i];
        src_k[i] = map_src(t0 + 2, i);
      }
      d_k = map_delta(t0 + 2);
      wait_loads();
      if (run1 < 0) rotate_own(k_lds1, t0 + 1, d_f);
    }
    run_v = run1;
    del_v = del1;
    run_k = n_tiles > 2 ? tile_run(t0 + 2, del_k) : -1;
    // the row the first tile turns the operand with, for the scores of tile 1 (the cos/sin
    // area is free: tile 1 is a whole run, so nothing rotates with it)
    if (run_v >= 0 && del_v != 0 && del_v != q_shift) {
      stage_row(del_v);
      wait_loads();
    }
  } else if constexpr (kRuns) {
    int32_t del0 = 0, del1 = 0;
    const int32_t run0 = tile_run(t0, del0), run1 = n_tiles > 1 ? tile_run(t0 + 1, del1) : -1;
    if (run0 >= 0 && del0 != 0) {   // the operand for the scores of tile 0
      stage_row(del0);
      wait_loads();
      turn_q(del0);
    }
    load_tile(k_lds0, t0, false, run0);
    load_tile(v_lds0, t0, true, run0);
    if (n_tiles > 1) load_tile(k_lds1, t0 + 1, false, run1);
    run_v = run1;
    del_v = del1;
    run_k = n_tiles > 2 ? tile_run(t0 + 2, del_k) : -1;
    // the row the first tile turns the operand with, for the scores of tile 1
    if (run_v >= 0 && del_v != 0 && del_v != q_shift) stage_row(del_v);
    wait_loads();
  } else {
    load_tile(k_lds0, t0, false);
    load_tile(v_lds0, t0, true);
    if (n_tiles > 1) load_tile(k_lds1, t0 + 1, false);
    if constexpr (kRope) {
      if ((t0 + 1) * kKeys > ctx) rope_cs(t0);
      rope_q();
    }
    wait_loads();
    if constexpr (kRope) {
      if ((t0 + 1) * kKeys > ctx) rope_own(k_lds0, t0);
      if (n_tiles > 1 && (t0 + 2) * kKeys > ctx) {
        rope_cs(t0 + 1);
        wait_loads();
        rope_own(k_lds1, t0 + 1);
      }
    }
  }
  __syncthreads();
  f32x16_t s_a[2], s_b[2];   // scores of the current / next tile, swapped every tile
  scores(k_lds0, s_a);
  finish_scores(t0, s_a);
  __syncthreads();   // every wave is done with K buffer 0 before tile 2 lands there

  // One tile.  Resident on entry: K(t+1) in K slot (t+1)&1, V(t) in V slot t&1 (P = t & 1,
  // a compile-time constant so every buffer below is a distinct, known array); the scores of
  // tile t are finished.  The body between the loads and the next-tile bookkeeping has no
  // branches, so the scheduler can interleave the matrix products of the next tile's scores
  // and of this tile's PV with the exponentials of this tile.
  auto tile = [&](int t, auto parity, f32x16_t (&scur)[2], f32x16_t (&snext)[2]) {   // t: local
    constexpr int P = decltype(parity)::value;
    uint8_t* const k_next = P ? k_lds0 : k_lds1;   // holds K(t+1)
    uint8_t* const k_free = P ? k_lds1 : k_lds0;   // receives K(t+2)
    const uint8_t* const v_cur = P ? v_lds1 : v_lds0;   // holds V(t)
    uint8_t* const v_free = P ? v_lds0 : v_lds1;   // receives V(t+1)
    // paged: the operand for the scores of tile t + 1, computed below (its cos/sin row, if
    // any, was staged during the previous tile; read before this tile's cos/sin loads)
    int32_t run_f = -1, del_f = 0;   // paged: tile t + 3 (K issued by the next tile)
    if constexpr (kPool) {
      turn_q(run_v >= 0 ? del_v : 0);
      if (t + 3 < n_tiles) run_f = tile_run(t0 + t + 3, del_f);
    }
    // this tile's loads (K(t+2), V(t+1)): issued after the first slice outside paged mode,
    // so the waves' first LDS reads and products of the tile go ahead of them
    auto issue_loads = [&]() {
      if (t + 2 < n_tiles) load_tile(k_free, t0 + t + 2, false, run_k);
      if (t + 1 < n_tiles) load_tile(v_free, t0 + t + 1, true, run_v);
    };
    if constexpr (kPaged) issue_loads();
    if constexpr (kRope) {
      if (t + 2 < n_tiles && (t0 + t + 3) * kKeys > ctx) rope_cs(t0 + t + 2);
    }
    int32_t rdl_f = 0;   // raw shift of this lane's rotation row of tile t + 3
    if constexpr (kPool) {
      if (kPaged && t + 2 < n_tiles && run_k < 0) load_cs(d_k);
      // the row the next tile turns the operand with (tile t + 2 is a whole run, so nothing
      // uses the cos/sin area during this tile)
      if (run_k >= 0 && del_k != 0 && del_k != q_shift) stage_row(del_k);
    }
    if constexpr (kPaged) {
      // tile t + 3 not a whole run: the rows and shifts of its keys, loaded now and checked
      // once the tile's loads have landed
      if (run_f < 0 && ctx > 0) {
#pragma unroll
        for (int i = 0; i < kLoadSteps; ++i) src_f[i] = raw_src(t0 + t + 3, i);
        rdl_f = raw_delta(t0 + t + 3);
      }
    }

    // (scores of a tile past the last one are computed on stale LDS and dropped)
    // Hand-ordered body: the K operands of the next tile's score products are read one pair
    // of products ahead and the V^T operands of slice s4 + 1 while slice s4's PV products
    // issue, so no matrix product waits on an LDS read issued just before it.  Scheduling
    // barriers keep this order.
    float psum = 0.f;
    const bf16x2_t ones = __builtin_bit_cast(bf16x2_t, 0x3F803F80u);
    auto kread = [&](int ks, int kb2) {
      return *reinterpret_cast<const u32x4*>(k_next + k_rd[ks] + 32 * kb2 * kRowBytes);
    };
    auto vread = [&](int s4, int db, int half) {
      return __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS i16x4*)(v_cur + v_rd[db][half] + 16 * s4 * kRowBytes));
    };
    u32x4 kq[kKS][2];
    i16x4 vq[4][kDB][2];
    kq[0][0] = kread(0, 0);
    kq[0][1] = kread(0, 1);
    kq[1][0] = kread(1, 0);
    kq[1][1] = kread(1, 1);
#pragma unroll
    for (int db = 0; db < kDB; ++db) {
      vq[0][db][0] = vread(0, db, 0);
      vq[0][db][1] = vread(0, db, 1);
    }
    __builtin_amdgcn_sched_barrier(0);
    flush_pending();   // the previous tile's last slice
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
      const int kb2 = s4 >> 1, u = s4 & 1;
      uint32_t pw[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(scur[kb2][8 * u + 2 * j], a.scale_log2, -m_run));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(scur[kb2][8 * u + 2 * j + 1], a.scale_log2, -m_run));
        pw[j] = pack_bf16x2(p0, p1);
        psum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pw[j]), ones, psum, false);
        __builtin_amdgcn_sched_barrier(0);
        // score product pj of this slice (D = 128: one per pair of probabilities, pj = j;
        // D = 64: one per two pairs): k step ks = (D / 64) s4 + (pj >> 1), block kb = pj & 1
        constexpr int kJPer = 8 / kKS;   // probability pairs per score product
        if (j % kJPer == 0) {
          const int pj = j / kJPer, ks = (kKS / 4) * s4 + (pj >> 1), kb = pj & 1;
          if (kb == 0) snext[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kq[ks][0]), qop[ks], ks == 0 ? f32x16_t{} : snext[0], 0, 0, 0);
          else snext[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kq[ks][1]), qop[ks], ks == 0 ? f32x16_t{} : snext[1], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
          if (ks + 2 < kKS) kq[ks + 2][kb] = kread(ks + 2, kb);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      const bf16x8_t pop = as_bf16x8(u32x4{pw[0], pw[1], pw[2], pw[3]});
      if (s4 == 3 && kDefer) pend_p = pop;
#pragma unroll
      for (int db = 0; db < kDB; ++db) {
        if (s4 + 1 < 4) {
          vq[s4 + 1][db][0] = vread(s4 + 1, db, 0);
          vq[s4 + 1][db][1] = vread(s4 + 1, db, 1);
        }
        __builtin_amdgcn_sched_barrier(0);
        const bf16x8_t vv = __builtin_bit_cast(
            bf16x8_t, __builtin_shufflevector(vq[s4][db][0], vq[s4][db][1], 0, 1, 2, 3, 4, 5, 6, 7));
        if (s4 < 3 || !kDefer) oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vv, pop, oacc[db], 0, 0, 0);
        else pend_v[db] = vv;
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (!kPaged) {
        if (s4 == 0) issue_loads();
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    l_part += psum;

    if (t + 1 < n_tiles) finish_scores(t0 + t + 1, snext);
    wait_loads();
    if constexpr (kRope) {
      if (t + 2 < n_tiles && (t0 + t + 3) * kKeys > ctx) rope_own(k_free, t0 + t + 2);
    }
    if constexpr (kPaged) {
      if (t + 2 < n_tiles && run_k < 0) rotate_own(k_free, t0 + t + 2, d_k);
      const bool rows_f = run_f < 0 && ctx > 0;
#pragma unroll
      for (int i = 0; i < kLoadSteps; ++i) {
        src_v[i] = src_k[i];
        src_k[i] = rows_f ? fin_src(t0 + t + 3, i, src_f[i]) : 0;
      }
      d_k = rows_f ? fin_delta(t0 + t + 3, rdl_f) : 0;
    }
    if constexpr (kPool) {
      run_v = run_k;
      del_v = del_k;
      run_k = run_f;
      del_k = del_f;
    }
    __syncthreads();
  };

  // local tiles [0, t_live) hold keys some row of this wave sees (all of them outside table mode)
  const int t_live = !kTable ? n_tiles
                             : (wave_max < t0 * kKeys ? 0 : min(n_tiles, wave_max / kKeys - t0 + 1));
  for (int t = 0; t < t_live; t += 2) {
    tile(t, std::integral_constant<int, 0>{}, s_a, s_b);
    if (t + 1 < t_live) tile(t + 1, std::integral_constant<int, 1>{}, s_b, s_a);
  }
  if constexpr (kTable) {   // the rest: this wave's share of the loads and the barriers only
    auto idle = [&](int t, auto parity) {
      constexpr int P = decltype(parity)::value;
      flush_pending();   // the last computed tile's last slice (then nothing is pending)
      pend_p = as_bf16x8(u32x4{0, 0, 0, 0});
      if (t + 2 < n_tiles) load_tile(P ? k_lds1 : k_lds0, t0 + t + 2, false);
      if (t + 1 < n_tiles) load_tile(P ? v_lds0 : v_lds1, t0 + t + 1, true);
      wait_loads();
      __syncthreads();
    };
    for (int t = t_live; t < n_tiles; ++t) {
      if (t & 1) idle(t, std::integral_constant<int, 1>{});
      else idle(t, std::integral_constant<int, 0>{});
    }
  }

  // ---- lane holds head dims 32 db + 8 qd + 4 hh + (0..3) of its row
  flush_pending();   // the last tile's last slice
  const float l_tot = pair_sum(l_part);
  if (!row_ok) return;
  // normalised and rounded to bf16: the output, or one split's share of it (with its reference
  // max and row sum, the weights the combine needs)
  const float inv = 1.f / l_tot;
  bf16_t* op = a.n_splits == 1 ? a.out + orow * kHD : a.ws_o + (split * a.rows_total + orow) * kHD;
#pragma unroll
  for (int db = 0; db < kDB; ++db)
#pragma unroll
    for (int qd = 0; qd < 4; ++qd) {
      const int d = 32 * db + 8 * qd + 4 * hh;
      uint2 v;
      v.x = pack_bf16x2(oacc[db][4 * qd] * inv, oacc[db][4 * qd + 1] * inv);
      v.y = pack_bf16x2(oacc[db][4 * qd + 2] * inv, oacc[db][4 * qd + 3] * inv);
      *reinterpret_cast<uint2*>(op + d) = v;
    }
  if (a.n_splits > 1 && hh == 0) a.ws_ml[split * a.rows_total + orow] = make_float2(m_run, l_tot);
}

// Merge the key-range splits of each query row by log-sum-exp.  Split s left its output
// normalised by its own row sum l_s (bf16) with its reference max m_s: the row is
// sum_s w_s O_s / sum_s w_s with w_s = 2^(m_s - M) l_s, M any common reference.  grid (rows_total / 16),
// 2 D threads: D / 8 lanes per row, 8 head dims per lane; every split's loads are issued without a branch
// between them (a split that saw no key of the row, reference max -inf, is dropped by a
// select: its sums are not finite).  With n_valid (table mode), rows of tokens past
// n_valid[b] are left untouched.
// kBatch: splits whose loads are issued together (4, 8 or 16, the smallest that covers n_splits:
// a larger batch holds more registers and lowers the occupancy that few splits need)
constexpr int kCombineRowsPerWG = 16;
template <int HD, int kCombineBatch>
__global__ void __launch_bounds__(256) prefill_combine_kernel(const bf16_t* __restrict__ ws_o,
                                                              const float2* __restrict__ ws_ml,
                                                              int32_t n_splits, int64_t rows_total,
                                                              const int32_t* __restrict__ n_valid,
                                                              int32_t n_q, int32_t n_q_heads,
                                                              int32_t batch,
                                                              bf16_t* __restrict__ out) {
  constexpr int kLanes = HD / 8;   // lanes per row
  const int64_t row = (int64_t)blockIdx.x * kCombineRowsPerWG + threadIdx.x / kLanes;
  if (row >= rows_total) return;
  if (n_valid) {   // row = ((l * B + b) * n_q + i) * Hq + h
    const int64_t ti = row / n_q_heads;
    const int i = (int)(ti % n_q);
    const int b = (int)((ti / n_q) % batch);
    if (i >= n_valid[b]) return;
  }
  const int d = 8 * (threadIdx.x & (kLanes - 1));
  // one pass with a running reference max, kCombineBatch splits at a time: all their loads
  // are issued before the first is used (a split past n_splits reads as one that saw no key)
  float M = -INFINITY, den = 0.f, o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < n_splits; s0 += kCombineBatch) {
    float2 mls[kCombineBatch];
    uint4 xs[kCombineBatch];
#pragma unroll
    for (int u = 0; u < kCombineBatch; ++u) {
      const int64_t s = s0 + u;
      mls[u] = s < n_splits ? ws_ml[s * rows_total + row] : make_float2(-INFINITY, 0.f);
      xs[u] = s < n_splits ? *reinterpret_cast<const uint4*>(ws_o + (s * rows_total + row) * HD + d)
                           : uint4{0u, 0u, 0u, 0u};
    }
#pragma unroll
  for (int u = 0; u < kCombineBatch; ++u) {
    const float2 ml = mls[u];
    const uint4 x = xs[u];
    const bool seen = ml.x != -INFINITY;
    const float m_new = seen ? fmaxf(M, ml.x) : M;
    const float keep = seen ? __builtin_amdgcn_exp2f(M - m_new) : 1.f;   // 0 while M is -inf
    const float w = seen ? __builtin_amdgcn_exp2f(ml.x - m_new) * ml.y : 0.f;
    M = m_new;
    den = den * keep + w;
    const uint32_t xw[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[2 * e] = o[2 * e] * keep + (seen ? w * __uint_as_float(xw[e] << 16) : 0.f);
      o[2 * e + 1] = o[2 * e + 1] * keep + (seen ? w * __uint_as_float(xw[e] & 0xFFFF0000u) : 0.f);
    }
  }
  }
  const float inv = 1.f / den;
  uint4 v;
  v.x = pack_bf16x2(o[0] * inv, o[1] * inv);
  v.y = pack_bf16x2(o[2] * inv, o[3] * inv);
  v.z = pack_bf16x2(o[4] * inv, o[5] * inv);
  v.w = pack_bf16x2(o[6] * inv, o[7] * inv);
  *reinterpret_cast<uint4*>(out + row * HD + d) = v;
}

}  // namespace

namespace {

// Token-level slot map (App. C.1) of the paged mode: every context slot of every request
// gets the pool token and the position shift of the gather block covering it.
__global__ void __launch_bounds__(256) map_clear_kernel(int32_t* smap, int32_t* dmap, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    smap[i] = 0;
    dmap[i] = 0;
  }
}

// grid (n_blocks), 64 threads: one gather block per workgroup, invalid blocks skipped.
__global__ void __launch_bounds__(64) map_expand_kernel(const pic_block* __restrict__ blocks,
                                                        int32_t batch, int32_t map_cap,
                                                        int32_t* smap, int32_t* dmap) {
  const pic_block blk = blocks[blockIdx.x];
  if (!map_block_ok(blk, batch, map_cap)) return;
  const int t = threadIdx.x;
  if (t < blk.n_tokens) {
    const int64_t i = (int64_t)blk.request * map_cap + blk.dst_slot + t;
    smap[i] = blk.src_token + t;
    dmap[i] = blk.delta;
  }
}

// One wave per (request, 64-slot tile), four per 256-thread workgroup, grid-stride: a tile
// whose 64 slots map to pool tokens src .. src + 63 with one shift is recorded as (src, shift),
// any other tile as (-1, 0).  Lane j reads slot k0 + j, so a tile's map entries load at once.
__global__ void __launch_bounds__(256) map_tiles_kernel(const int32_t* __restrict__ smap,
                                                        const int32_t* __restrict__ dmap,
                                                        int64_t n_tiles, int32_t map_cap,
                                                        int32_t map_tiles, int32_t* tmap) {
  static_assert(kKeys == 64, "one lane per key of a tile");
  const int lane = threadIdx.x & 63;
  for (int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); i < n_tiles; i += (int64_t)gridDim.x * 4) {
    const int64_t b = i / map_tiles;
    const int32_t k0 = (int32_t)(i - b * map_tiles) * kKeys;
    int32_t src = -1, d = 0;
    if (k0 + kKeys <= map_cap) {   // (uniform over the wave)
      const int32_t sj = smap[b * map_cap + k0 + lane], dj = dmap[b * map_cap + k0 + lane];
      const int32_t s0 = __shfl(sj, 0, 64), d0 = __shfl(dj, 0, 64);
      const bool ok = s0 >= 0 && (int64_t)sj == (int64_t)s0 + lane && dj == d0;
      if (__all(ok)) {
        src = s0;
        d = d0;
      }
    }
    if (lane == 0) {
      tmap[2 * i] = src;
      tmap[2 * i + 1] = d;
    }
  }
}

template <int HD>
hipError_t launch_hd(const AttnShape& s, const PrefillArgs& a, const SplitPlan& p, int mode, bool interleaved,
                     int32_t n_q, hipStream_t stream) {
  const int per_xcd = (a.n_wg + kNumXcd - 1) / kNumXcd;
  const dim3 grid(per_xcd * kNumXcd, s.n_layers);
  if (mode == kModeTable)
    hipLaunchKernelGGL((prefill_bf16_kernel<HD, kModeTable, false>), grid, dim3(kThreads), 0, stream, a);
  else if (mode == kModeRope && interleaved)
    hipLaunchKernelGGL((prefill_bf16_kernel<HD, kModeRope, true>), grid, dim3(kThreads), 0, stream, a);
  else if (mode == kModeRope)
    hipLaunchKernelGGL((prefill_bf16_kernel<HD, kModeRope, false>), grid, dim3(kThreads), 0, stream, a);
  else if (mode == kModePaged && interleaved)
    hipLaunchKernelGGL((prefill_bf16_kernel<HD, kModePaged, true>), grid, dim3(kThreads), 0, stream, a);
  else if (mode == kModeRuns && interleaved)
    hipLaunchKernelGGL((prefill_bf16_kernel<HD, kModeRuns, true>), grid, dim3(kThreads), 0, stream, a);
  else if (mode == kModeRuns)
    hipLaunchKernelGGL((prefill_bf16_kernel<HD, kModeRuns, false>), grid, dim3(kThreads), 0, stream, a);
  else if (mode == kModePaged)
    hipLaunchKernelGGL((prefill_bf16_kernel<HD, kModePaged, false>), grid, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL((prefill_bf16_kernel<HD, kModeSuffix, false>), grid, dim3(kThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.n_splits == 1) return e;
  const dim3 cgrid((unsigned)((a.rows_total + kCombineRowsPerWG - 1) / kCombineRowsPerWG));
  const dim3 cblock(kCombineRowsPerWG * HD / 8);
  const int32_t* nv = mode == kModeTable ? a.n_valid : nullptr;
  if (p.n_splits <= 4)
    hipLaunchKernelGGL((prefill_combine_kernel<HD, 4>), cgrid, cblock, 0, stream, a.ws_o, a.ws_ml, p.n_splits,
                       a.rows_total, nv, n_q, s.n_q_heads, s.batch, a.out);
  else if (p.n_splits <= 8)
    hipLaunchKernelGGL((prefill_combine_kernel<HD, 8>), cgrid, cblock, 0, stream, a.ws_o, a.ws_ml, p.n_splits,
                       a.rows_total, nv, n_q, s.n_q_heads, s.batch, a.out);
  else
    hipLaunchKernelGGL((prefill_combine_kernel<HD, 16>), cgrid, cblock, 0, stream, a.ws_o, a.ws_ml, p.n_splits,
                       a.rows_total, nv, n_q, s.n_q_heads, s.batch, a.out);
  return hipGetLastError();
}

hipError_t launch(const AttnShape& s, PrefillArgs a, int mode, bool interleaved, int32_t n_q,
                  int32_t max_ctx, void* workspace, size_t ws_bytes, hipStream_t stream) {
  const int n_rep = s.n_q_heads / s.n_kv_heads;
  const int64_t M = (int64_t)n_q * n_rep;
  if (M == 0 || s.batch == 0 || s.n_layers == 0) return hipSuccess;
  const SplitPlan p = plan_prefill_splits(s, n_q, max_ctx);
  a.n_suffix = n_q;
  a.n_rep = n_rep;
  a.rep_magic = ((uint64_t(1) << 32) + n_rep - 1) / n_rep;
  if (M >= (int64_t(1) << 27)) return hipErrorInvalidValue;   // beyond the exact range of the division
  a.batch = s.batch;
  a.cache_cap = s.cache_cap;
  a.n_q_heads = s.n_q_heads;
  a.n_kv_heads = s.n_kv_heads;
  a.m_tiles = p.m_tiles;
  a.n_splits = p.n_splits;
  a.tiles_per_split = p.tiles_per_split;
  a.n_wg = p.m_tiles * p.n_splits * s.batch * s.n_kv_heads;
  a.rows_total = (int64_t)s.n_layers * s.batch * n_q * s.n_q_heads;
  a.ws_o = static_cast<bf16_t*>(workspace);
  a.ws_ml = a.ws_o ? reinterpret_cast<float2*>(a.ws_o + (size_t)p.n_splits * a.rows_total * s.head_dim) : nullptr;
  a.scale_log2 = s.scale_log2;
  if (p.n_splits > 1 && (workspace == nullptr || ws_bytes < prefill_bf16_workspace(s, n_q, max_ctx)))
    return hipErrorInvalidValue;
  if (s.head_dim == 64) return launch_hd<64>(s, a, p, mode, interleaved, n_q, stream);
  if (s.head_dim == 128) return launch_hd<128>(s, a, p, mode, interleaved, n_q, stream);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_prefill_bf16(const AttnShape& s, const bf16_t* q, const bf16_t* k_suf,
                               const bf16_t* v_suf, bf16_t* cache_k, bf16_t* cache_v,
                               const int32_t* ctx_len, int32_t max_ctx,
                               int32_t n_suffix, bf16_t* out, void* workspace, size_t ws_bytes,
                               hipStream_t stream) {
  PrefillArgs a = {};
  a.q = q;
  a.k_suf = k_suf;
  a.v_suf = v_suf;
  a.cache_k = cache_k;
  a.cache_v = cache_v;
  a.ctx_len = ctx_len;
  a.out = out;
  a.max_ctx = max_ctx;
  return launch(s, a, kModeSuffix, false, n_suffix, max_ctx, workspace, ws_bytes, stream);
}

hipError_t launch_prefill_bf16_rope(const AttnShape& s, bool interleaved, const bf16_t* q,
                                    const bf16_t* k_suf, const bf16_t* v_suf, bf16_t* cache_k,
                                    bf16_t* cache_v, const int32_t* ctx_len, int32_t max_ctx,
                                    int32_t n_suffix, const float2* table, int64_t table_stride,
                                    int32_t max_abs_delta, bf16_t* out, void* workspace,
                                    size_t ws_bytes, hipStream_t stream) {
  PrefillArgs a = {};
  a.q = q;
  a.k_suf = k_suf;
  a.v_suf = v_suf;
  a.cache_k = cache_k;
  a.cache_v = cache_v;
  a.ctx_len = ctx_len;
  a.out = out;
  a.max_ctx = max_ctx;
  a.table = table;
  a.table_stride = table_stride;
  a.max_abs_delta = max_abs_delta;
  return launch(s, a, kModeRope, interleaved, n_suffix, max_ctx, workspace, ws_bytes, stream);
}

hipError_t launch_prefill_bf16_table(const AttnShape& s, const bf16_t* q, const bf16_t* cache_k,
                                     const bf16_t* cache_v, const RowPos& pos, int32_t n_q,
                                     int32_t max_len, bf16_t* out, void* workspace,
                                     size_t ws_bytes, hipStream_t stream) {
  PrefillArgs a = {};
  a.q = q;
  a.cache_k = const_cast<bf16_t*>(cache_k);
  a.cache_v = const_cast<bf16_t*>(cache_v);
  a.q_pos = pos.table;
  a.n_valid = pos.n_valid;
  a.max_pos = pos.max_pos;
  a.out = out;
  const int32_t max_ctx = max_len > n_q ? max_len - n_q : 0;
  return launch(s, a, kModeTable, false, n_q, max_ctx, workspace, ws_bytes, stream);
}

hipError_t launch_slot_map(const pic_block* blocks, int32_t n_blocks, int32_t batch, int32_t map_cap,
                           int32_t* smap, int32_t* dmap, int32_t* tmap, hipStream_t stream) {
  const int64_t n_map = (int64_t)batch * map_cap;
  if (n_map == 0) return hipSuccess;
  int64_t g = (n_map + 255) / 256;
  g = g < 1 ? 1 : (g > 65536 ? 65536 : g);
  hipLaunchKernelGGL(map_clear_kernel, dim3((unsigned)g), dim3(256), 0, stream, smap, dmap, n_map);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (n_blocks > 0) {
    hipLaunchKernelGGL(map_expand_kernel, dim3(n_blocks), dim3(64), 0, stream, blocks, batch, map_cap,
                       smap, dmap);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (tmap == nullptr) return hipSuccess;
  const int32_t mt = slot_map_tiles(map_cap);
  const int64_t n_tiles = (int64_t)batch * mt;
  int64_t gt = (n_tiles + 3) / 4;   // four tiles (waves) per workgroup
  gt = gt < 1 ? 1 : (gt > 65536 ? 65536 : gt);
  hipLaunchKernelGGL(map_tiles_kernel, dim3((unsigned)gt), dim3(256), 0, stream, smap, dmap, n_tiles,
                     map_cap, mt, tmap);
  return hipGetLastError();
}

hipError_t launch_prefill_bf16_paged(const AttnShape& s, bool interleaved, const bf16_t* q,
                                     const bf16_t* k_suf, const bf16_t* v_suf, bf16_t* cache_k,
                                     bf16_t* cache_v, const int32_t* ctx_len, int32_t max_ctx,
                                     int32_t n_suffix, const bf16_t* pool_k, const bf16_t* pool_v,
                                     int64_t pool_tokens, const int32_t* smap, const int32_t* dmap,
                                     int32_t map_cap, const int32_t* tmap, const float2* table,
                                     int64_t table_stride,
                                     int32_t max_abs_delta, bf16_t* out, void* workspace,
                                     size_t ws_bytes, hipStream_t stream) {
  PrefillArgs a = {};
  a.pool_k = pool_k;
  a.pool_v = pool_v;
  a.pool_tokens = pool_tokens;
  a.smap = smap;
  a.dmap = dmap;
  a.map_cap = map_cap;
  a.tmap = tmap;
  a.map_tiles = slot_map_tiles(map_cap);
  a.table = table;
  a.table_stride = table_stride;
  a.max_abs_delta = max_abs_delta;
  a.q = q;
  a.k_suf = k_suf;
  a.v_suf = v_suf;
  a.cache_k = cache_k;
  a.cache_v = cache_v;
  a.ctx_len = ctx_len;
  a.out = out;
  a.max_ctx = max_ctx;
  if (tmap == nullptr)   // every tile read through the slot map, keys turned in LDS
    return launch(s, a, kModePaged, interleaved, n_suffix, max_ctx, workspace, ws_bytes, stream);
  // with a tile map: the tiles that are not whole runs are composed into the cache first (here,
  // or beforehand by the caller when no slot map is given), then the prefill reads whole runs
  // from the pool and everything else from the cache
  if (smap != nullptr) {
    const hipError_t e = launch_compose_tiles(interleaved, s.head_dim, s.n_layers, s.n_kv_heads, pool_k, pool_v,
                                              pool_tokens, smap, dmap, map_cap, tmap, a.map_tiles,
                                              ctx_len, max_ctx, table, table_stride, max_abs_delta,
                                              cache_k, cache_v, s.batch, s.cache_cap, stream);
    if (e != hipSuccess) return e;
  }
  return launch(s, a, kModeRuns, interleaved, n_suffix, max_ctx, workspace, ws_bytes, stream);
}

}  // namespace pic
