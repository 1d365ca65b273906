// Host-side planner: the compact workqueue of Sec. 3.4 computed on the CPU from host
// lengths, with the same split policies, bounds and task order as the device planner.
// A serving loop uses it to size buffers and to price routes (the cost model of
// Sec. 3.5) without a device round trip.
#include <algorithm>
#include <cstdint>
#include <vector>

#include "../../include/pkv.h"
#include "pkv_internal.h"

namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// nsplit_i for every row under the policy (Sec. 3.5 readings; see pkv_plan_params)
void split_counts(const std::vector<int64_t>& tiles, const pkv_plan_params& p, std::vector<int32_t>* ns) {
  const int64_t B = (int64_t)tiles.size();
  ns->assign(tiles.size(), 0);
  if (p.policy == PKV_SPLIT_BATCH) {
    int64_t active = 0;
    for (int64_t t : tiles) active += t > 0;
    int64_t S = ceil_div(p.target_tasks, std::max<int64_t>(1, active) * p.num_kv_heads);
    S = std::min<int64_t>(std::max<int64_t>(S, p.split_min), p.split_max);
    for (int64_t i = 0; i < B; ++i) (*ns)[i] = (int32_t)std::min(tiles[i], S);
    return;
  }
  // tile quota: the smallest Q >= 1 whose task count fits target_tasks (the count only
  // falls as Q grows), else the largest tile count (one split per row)
  const int64_t per_head = p.target_tasks / p.num_kv_heads;
  int64_t max_tiles = 0;
  for (int64_t t : tiles) max_tiles = std::max(max_tiles, t);
  auto count = [&](int64_t q) {
    int64_t c = 0;
    for (int64_t t : tiles) c += t > 0 ? std::min<int64_t>(p.split_max, ceil_div(t, q)) : 0;
    return c;
  };
  int64_t lo = 1, hi = std::max<int64_t>(1, max_tiles);
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (count(mid) <= per_head) hi = mid; else lo = mid + 1;
  }
  for (int64_t i = 0; i < B; ++i)
    (*ns)[i] = tiles[i] > 0 ? (int32_t)std::min<int64_t>(p.split_max, ceil_div(tiles[i], lo)) : 0;
}

}  // namespace

extern "C" {

int pkv_plan_host(const int32_t* seq_lens, int32_t B, int32_t max_pages_per_row, const pkv_plan_params* params,
                  pkv_task* tasks, int32_t max_tasks, int32_t* split_offsets, int32_t* num_tasks) {
  if (!seq_lens || !params || !num_tasks || B < 1 || max_pages_per_row < 1) return PKV_ERR_INVALID_ARG;
  const pkv_plan_params p = *params;
  if (p.page_size != pkv::kPageSize) return PKV_ERR_UNSUPPORTED;
  if (p.tile_tokens <= 0 || p.tile_tokens % p.page_size != 0) return PKV_ERR_UNSUPPORTED;
  if (p.num_kv_heads < 1 || p.split_min < 1 || p.split_min > p.split_max || p.split_max > pkv::kMaxSplits ||
      p.target_tasks < 1)
    return PKV_ERR_INVALID_ARG;
  if (p.policy != PKV_SPLIT_BATCH && p.policy != PKV_SPLIT_QUOTA) return PKV_ERR_INVALID_ARG;
  if (pkv_max_tasks(B, p.num_kv_heads, p.split_max) < 0) return PKV_ERR_INVALID_ARG;
  const int64_t cap = (int64_t)max_pages_per_row * p.page_size;
  std::vector<int64_t> tiles(B);
  for (int32_t i = 0; i < B; ++i) {
    if (seq_lens[i] < 0 || seq_lens[i] > cap) return PKV_ERR_INVALID_ARG;
    tiles[i] = ceil_div(seq_lens[i], p.tile_tokens);
  }
  std::vector<int32_t> ns;
  split_counts(tiles, p, &ns);
  int64_t total = 0;
  for (int32_t v : ns) total += v;
  const int64_t n = total * p.num_kv_heads;
  *num_tasks = (int32_t)n;
  if (split_offsets) {
    int32_t run = 0;
    for (int32_t i = 0; i < B; ++i) {
      split_offsets[i] = run;
      run += ns[i];
    }
    split_offsets[B] = run;
  }
  if (!tasks) return PKV_OK;
  if (max_tasks < n) return PKV_ERR_WORKSPACE;
  int64_t k = 0;
  for (int32_t i = 0; i < B; ++i) {
    for (int32_t s = 0; s < ns[i]; ++s) {
      // balanced tile bounds of split s (Sec. 3.4 reading R6)
      const int64_t b0 = (int64_t)s * tiles[i] / ns[i];
      const int64_t b1 = (int64_t)(s + 1) * tiles[i] / ns[i];
      const int32_t t0 = (int32_t)(b0 * p.tile_tokens);
      const int32_t t1 = (int32_t)std::min<int64_t>(b1 * p.tile_tokens, seq_lens[i]);
      for (int32_t g = 0; g < p.num_kv_heads; ++g) tasks[k++] = pkv_task{i, g, s, t0, t1};
    }
  }
  return PKV_OK;
}

}  // extern "C"
