// Host-side launch planning of libpic's attention kernels: how many workgroups split a key
// range, and the workspace their partial results need.  Plain C++ (no device code), so the
// sanitizer build of the host library compiles this file as it is.
#include "pic_internal.h"

namespace pic {

// Key-range splits of the prefill.  A launch whose (m-tile, request, kv head) units already
// occupy half the 256 compute units is not split: under load the chip runs at its power limit,
// where busy units speed up as others idle, so the last round's idle units cost little and the
// partials and the combine cost more (measured: 224 units of the 32K Qwen workload 898 us
// unsplit against 921 us in 8 key ranges; the frontier workload's 1152 units 900 against
// 934 us in 2).  Smaller launches are split so that they cover the compute units in whole
// rounds, each split keeping at least 8 key tiles.  Cost in units of one workgroup-tile
// (~2 us): rounds * tiles per split, plus, for split runs, one tile (the combine launch; the
// splits' own prologues run in parallel) and the partials each split writes and the combine
// reads back (bf16 output and fp32 (max, sum): 264 bytes per query row, twice, at ~4 TB/s).  Ties (within 3%) go to
// fewer splits.
SplitPlan plan_prefill_splits(const AttnShape& s, int32_t n_suffix, int32_t max_ctx) {
  SplitPlan p;
  const int64_t M = (int64_t)n_suffix * (s.n_q_heads / s.n_kv_heads);
  p.m_tiles = (int)((M + kPrefillRowsPerWG - 1) / kPrefillRowsPerWG);
  const int64_t base = (int64_t)p.m_tiles * s.batch * s.n_kv_heads * s.n_layers;
  const double rows = (double)s.n_layers * s.batch * n_suffix * s.n_q_heads;
  const int tiles = (int)(((int64_t)max_ctx + n_suffix + kPrefillKeys - 1) / kPrefillKeys);
  int best = 1;
  double best_cost = 1e30;
  for (int sp = 1; sp <= (base >= 128 ? 1 : kPrefillMaxSplits); ++sp) {
    const int tps = (tiles + sp - 1) / sp;
    if (sp > 1 && tps < 8) break;
    const int64_t rounds = (base * sp + 255) / 256;
    const double partials = sp > 1 ? 1.0 + sp * rows * 2.0 * (s.head_dim * 2 + 8) / 4e12 / 2e-6 : 0.0;
    const double cost = (double)rounds * tps + partials;
    if (cost < best_cost * 0.97) {
      best_cost = cost;
      best = sp;
    }
  }
  p.n_splits = best;
  p.tiles_per_split = (tiles + best - 1) / best;
  return p;
}

size_t prefill_bf16_workspace(const AttnShape& s, int32_t n_suffix, int32_t max_ctx) {
  const SplitPlan p = plan_prefill_splits(s, n_suffix, max_ctx);
  if (p.n_splits == 1) return 0;
  // per split and query row: the split's normalised output (bf16) and its (max, sum) pair
  const size_t rows = (size_t)s.n_layers * s.batch * n_suffix * s.n_q_heads;
  return (size_t)p.n_splits * rows * (s.head_dim * 2 + 2 * sizeof(float));
}

int32_t slot_map_tiles(int32_t map_cap) { return (int32_t)(((int64_t)map_cap + kPrefillKeys - 1) / kPrefillKeys); }

// Decode workgroups per (request, kv head, group of 16 query heads): enough 4-wave workgroups
// for one per compute unit
// (256 per launch; measured faster than two per unit on split launches), each wave keeping at
// least kDecodeMinWaveKeys keys.
int32_t decode_bf16_auto_splits(const AttnShape& s, int32_t max_len) {
  const int64_t pairs = (int64_t)s.batch * s.n_kv_heads * s.n_layers * decode_head_groups(s);
  int64_t splits = (256 + pairs - 1) / pairs;
  const int64_t per_split = (int64_t)kDecodeWaves * kDecodeMinWaveKeys;
  const int64_t max_splits = (max_len + per_split - 1) / per_split;
  if (splits > max_splits) splits = max_splits;
  if (splits < 1) splits = 1;
  return (int32_t)splits;
}

size_t decode_bf16_workspace(const AttnShape& s, int32_t, int32_t n_splits) {
  if (n_splits <= 1) return 0;
  const size_t rows = (size_t)s.n_layers * s.batch * s.n_q_heads * n_splits;
  return rows * (s.head_dim + 2) * sizeof(float);
}

}  // namespace pic
