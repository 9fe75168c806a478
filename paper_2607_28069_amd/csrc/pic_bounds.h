// Index clamping of libpic's kernels: every index a kernel derives from a device-side table
// (gather blocks, group starts, slot and tile maps, context and base lengths, position shifts)
// goes through one of these checks before it addresses memory, so a wrong table gives wrong
// values, never an access outside the buffers whose sizes the host passed.
//
// The functions are __host__ __device__: the kernels call them, and the CPU emulation of the
// launches that the sanitizer tests build (AddressSanitizer, UndefinedBehaviorSanitizer) calls
// the same code on host buffers of the exact sizes.
#pragma once

#include <stdint.h>

#include "pic.h"

#if defined(__HIPCC__) || defined(__HIP__)
#include <hip/hip_runtime.h>
#define PIC_HD __host__ __device__ __forceinline__
#else
#define PIC_HD inline
#endif

namespace pic {

PIC_HD int32_t clamp_i32(int32_t v, int32_t lo, int32_t hi) { return v < lo ? lo : (v > hi ? hi : v); }

// A position shift, clamped to the table's rows (|delta| <= max_abs_delta).
PIC_HD int32_t clamp_delta(int32_t d, int32_t max_abs_delta) { return clamp_i32(d, -max_abs_delta, max_abs_delta); }

// A per-request length read from the device (context or base length), clamped to [0, max_len].
PIC_HD int32_t clamp_len(int32_t n, int32_t max_len) { return clamp_i32(n, 0, max_len); }

// A pool token read from a slot map, clamped into the pool (pool_tokens >= 1).
PIC_HD int32_t clamp_pool_token(int32_t t, int64_t pool_tokens) {
  return t < 0 ? 0 : (t >= pool_tokens ? (int32_t)(pool_tokens - 1) : t);
}

// The pool run a gather block reads lies inside the pool.
PIC_HD bool block_source_ok(const pic_block& b, int64_t pool_tokens) {
  return b.n_tokens > 0 && b.n_tokens <= PIC_BLOCK_TOKENS && b.src_token >= 0 &&
         (int64_t)b.src_token + b.n_tokens <= pool_tokens;
}

// The cache slots a gather block writes lie inside the caches, and its shift inside the table.
PIC_HD bool block_dest_ok(const pic_block& b, int32_t batch, int32_t cache_cap, int32_t max_abs_delta) {
  return b.request >= 0 && b.request < batch && b.n_tokens > 0 && b.n_tokens <= PIC_BLOCK_TOKENS &&
         b.dst_slot >= 0 && (int64_t)b.dst_slot + b.n_tokens <= cache_cap && b.delta <= max_abs_delta &&
         b.delta >= -max_abs_delta;
}

// A gather block composition may move (compose_kernel).
PIC_HD bool block_ok(const pic_block& b, int32_t batch, int64_t pool_tokens, int32_t cache_cap,
                     int32_t max_abs_delta) {
  return block_source_ok(b, pool_tokens) && block_dest_ok(b, batch, cache_cap, max_abs_delta);
}

// A block of a shared-source group: it must read its group's run (the first block's) and write
// inside the caches.
PIC_HD bool shared_block_ok(const pic_block& b, const pic_block& run, int32_t batch, int32_t cache_cap,
                            int32_t max_abs_delta) {
  return b.src_token == run.src_token && b.n_tokens == run.n_tokens &&
         block_dest_ok(b, batch, cache_cap, max_abs_delta);
}

// Blocks [g0, g1) of a group, from two group starts clamped to [0, n_blocks].
PIC_HD void group_range(int32_t start, int32_t end, int32_t n_blocks, int32_t& g0, int32_t& g1) {
  g0 = start < 0 ? 0 : start;
  g1 = end > n_blocks ? n_blocks : end;
}

// A gather block the slot map may expand: its request and slots inside the map.
PIC_HD bool map_block_ok(const pic_block& b, int32_t batch, int32_t map_cap) {
  return b.request >= 0 && b.request < batch && b.n_tokens > 0 && b.n_tokens <= PIC_BLOCK_TOKENS &&
         b.dst_slot >= 0 && (int64_t)b.dst_slot + b.n_tokens <= map_cap;
}

// A tile-map entry (src, delta) for context tile [s0, s0 + 64) of a request with ctx context
// tokens is read from the pool in one piece only when the whole run lies in the pool, its shift
// in the table, and the tile in the context.
PIC_HD bool tile_run_ok(int32_t src, int32_t delta, int32_t s0, int32_t ctx, int64_t pool_tokens,
                        int32_t max_abs_delta) {
  return src >= 0 && (int64_t)src + PIC_BLOCK_TOKENS <= pool_tokens && delta >= -max_abs_delta &&
         delta <= max_abs_delta && s0 + PIC_BLOCK_TOKENS <= ctx;
}

}  // namespace pic
