// C ABI of libpkv.so: argument validation, workspace layout and kernel launches.
// Every check here runs on the host before anything is enqueued, so a rejected call
// leaves the stream untouched.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cmath>
#include <utility>
#include <vector>
#include <cstdint>
#include <cstring>

#include "pkv_internal.h"

using namespace pkv;

namespace {

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int from_hip(hipError_t e) { return e == hipSuccess ? PKV_OK : PKV_ERR_HIP; }

int check_heads(int32_t Hq, int32_t Hkv, int32_t d, int* G) {
  if (Hq < 1 || Hkv < 1 || Hq % Hkv != 0) return PKV_ERR_INVALID_ARG;
  if (d != kHeadDim) return PKV_ERR_UNSUPPORTED;
  const int g = Hq / Hkv;
  if (g != 1 && g != 2 && g != 4 && g != 8) return PKV_ERR_UNSUPPORTED;
  *G = g;
  return PKV_OK;
}

// Inputs and output of a decode call (the workspace is checked by check_ws).
int check_pool(const uint16_t* q, const uint16_t* k, const uint16_t* v, int32_t num_pages,
               const int32_t* bt, int32_t maxp, const int32_t* seq_lens, int32_t B, uint16_t* out) {
  if (!q || !k || !v || !bt || !seq_lens || !out) return PKV_ERR_INVALID_ARG;
  if (B < 1 || num_pages < 1 || maxp < 1) return PKV_ERR_INVALID_ARG;
  if ((int64_t)maxp * kPageSize > INT32_MAX) return PKV_ERR_INVALID_ARG;
  // 16-byte vector loads of Q/K/V, 4-byte output stores
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 4)) return PKV_ERR_INVALID_ARG;
  return PKV_OK;
}

// A caller's workspace: 16-byte rows.
int check_ws(const void* ws) { return ws && aligned(ws, 16) ? PKV_OK : PKV_ERR_INVALID_ARG; }

// Where a call's device error word, completion counters and partial-state slots live.
struct Scratch {
  unsigned* err;
  int32_t* counters;
  float* partials;
};

// The layout of a caller's workspace (pkv_workspace_size).
Scratch ws_layout(void* ws, int32_t B, int32_t Hkv) {
  char* w = static_cast<char*>(ws);
  return Scratch{reinterpret_cast<unsigned*>(w), reinterpret_cast<int32_t*>(w + kWsHeaderBytes),
                 reinterpret_cast<float*>(w + partials_offset(B, Hkv))};
}

DecodeArgs make_args(const uint16_t* q, const uint16_t* k, const uint16_t* v, int32_t num_pages,
                     const int32_t* bt, int32_t maxp, const int32_t* seq_lens, int32_t B, int32_t Hq,
                     int32_t Hkv, float sm_scale, uint16_t* out, const Scratch& sc) {
  DecodeArgs a;
  std::memset(&a, 0, sizeof(a));
  a.q = q;
  a.k = k;
  a.v = v;
  a.block_table = bt;
  a.seq_lens = seq_lens;
  a.out = out;
  a.err = sc.err;
  a.counters = sc.counters;
  a.partials = sc.partials;
  a.num_pages = num_pages;
  a.max_pages_per_row = maxp;
  a.B = B;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.scale_log2 = (float)((double)sm_scale * 1.4426950408889634);  // log2(e)
  return a;
}

// Planner arguments; the error word and counters come from `sc`.
int make_plan_args(const int32_t* seq_lens, const int32_t* block_table, int32_t B, int32_t max_pages_per_row,
                   int32_t num_pages, const pkv_plan_params* params, pkv_task* tasks, int32_t max_tasks,
                   int32_t* split_offsets, int32_t* num_tasks, const Scratch& sc, PlanArgs* out) {
  if (!seq_lens || !params || !tasks || !split_offsets || !num_tasks) return PKV_ERR_INVALID_ARG;
  if (B < 1 || B > kMaxPlanBatch || max_pages_per_row < 1) return PKV_ERR_INVALID_ARG;
  if (block_table && num_pages < 1) return PKV_ERR_INVALID_ARG;
  if (!aligned(tasks, 4)) return PKV_ERR_INVALID_ARG;
  const pkv_plan_params p = *params;
  if (p.page_size != kPageSize) return PKV_ERR_UNSUPPORTED;
  if (p.tile_tokens <= 0 || p.tile_tokens % p.page_size != 0) return PKV_ERR_UNSUPPORTED;
  if (p.num_kv_heads < 1 || p.split_min < 1 || p.split_min > p.split_max || p.split_max > kMaxSplits ||
      p.target_tasks < 1)
    return PKV_ERR_INVALID_ARG;
  if (p.policy != PKV_SPLIT_BATCH && p.policy != PKV_SPLIT_QUOTA) return PKV_ERR_INVALID_ARG;
  if ((int64_t)max_pages_per_row * p.page_size > INT32_MAX) return PKV_ERR_INVALID_ARG;
  const int32_t bound = pkv_max_tasks(B, p.num_kv_heads, p.split_max);
  if (bound < 0) return PKV_ERR_INVALID_ARG;
  if (max_tasks < bound) return PKV_ERR_WORKSPACE;
  PlanArgs& a = *out;
  std::memset(&a, 0, sizeof(a));
  a.seq_lens = seq_lens;
  a.block_table = block_table;
  a.B = B;
  a.max_pages_per_row = max_pages_per_row;
  a.num_pages = num_pages;
  a.page_size = p.page_size;
  a.tile_tokens = p.tile_tokens;
  a.Hkv = p.num_kv_heads;
  a.split_min = p.split_min;
  a.split_max = p.split_max;
  a.target_tasks = p.target_tasks;
  a.policy = p.policy;
  a.tasks = tasks;
  a.max_tasks = max_tasks;
  a.split_offsets = split_offsets;
  a.num_tasks = num_tasks;
  a.err = sc.err;
  a.counters = sc.counters;
  return PKV_OK;
}

}  // namespace

extern "C" {

int32_t pkv_max_tasks(int32_t B, int32_t Hkv, int32_t split_max) {
  if (B < 1 || Hkv < 1 || split_max < 1) return -1;
  const int64_t n = (int64_t)B * Hkv * split_max;
  return n > INT32_MAX ? -1 : (int32_t)n;
}

size_t pkv_workspace_size(int32_t B, int32_t Hq, int32_t Hkv, int32_t d, int32_t max_tasks) {
  int G = 0;
  if (B < 1 || max_tasks < 0 || check_heads(Hq, Hkv, d, &G) != PKV_OK) return 0;
  return partials_offset(B, Hkv) + (size_t)max_tasks * slot_floats(G) * sizeof(float);
}

int pkv_workspace_init(void* ws, size_t ws_bytes, int32_t B, int32_t Hkv, hipStream_t stream) {
  if (!ws || B < 1 || Hkv < 1 || !aligned(ws, 16)) return PKV_ERR_INVALID_ARG;
  const size_t n = partials_offset(B, Hkv);
  if (ws_bytes < n) return PKV_ERR_WORKSPACE;
  if ((int64_t)B * Hkv > INT32_MAX) return PKV_ERR_INVALID_ARG;
  return from_hip(launch_ws_init(ws, n, (uint32_t)(B * Hkv), stream));
}

int pkv_plan(const int32_t* seq_lens, const int32_t* block_table, int32_t B, int32_t max_pages_per_row,
             int32_t num_pages, const pkv_plan_params* params, pkv_task* tasks, int32_t max_tasks,
             int32_t* split_offsets, int32_t* num_tasks, void* ws, size_t ws_bytes, hipStream_t stream) {
  int st = check_ws(ws);
  if (st != PKV_OK) return st;
  PlanArgs a;
  st = make_plan_args(seq_lens, block_table, B, max_pages_per_row, num_pages, params, tasks, max_tasks,
                      split_offsets, num_tasks, ws_layout(ws, B, 1), &a);
  if (st != PKV_OK) return st;
  if (ws_bytes < partials_offset(B, params->num_kv_heads)) return PKV_ERR_WORKSPACE;  // header + counters
  return from_hip(launch_plan(a, stream));
}

int pkv_decode_timed(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t num_pages,
                     const int32_t* block_table, int32_t max_pages_per_row, const int32_t* seq_lens, int32_t B,
                     int32_t Hq, int32_t Hkv, int32_t d, const pkv_task* tasks, const int32_t* split_offsets,
                     const int32_t* num_tasks, int32_t max_tasks, float sm_scale, int32_t flags, uint16_t* out,
                     void* ws, size_t ws_bytes, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
  int st = check_pool(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, out);
  if (st != PKV_OK || (st = check_ws(ws)) != PKV_OK) return st;
  if (!tasks || !split_offsets || !num_tasks || !aligned(tasks, 4)) return PKV_ERR_INVALID_ARG;
  int G = 0;
  if ((st = check_heads(Hq, Hkv, d, &G)) != PKV_OK) return st;
  if (flags != 0 && flags != PKV_FUSED_MERGE) return PKV_ERR_INVALID_ARG;
  if (!std::isfinite(sm_scale)) return PKV_ERR_INVALID_ARG;
  if (max_tasks < 1) return PKV_ERR_INVALID_ARG;
  if (ws_bytes < pkv_workspace_size(B, Hq, Hkv, d, max_tasks)) return PKV_ERR_WORKSPACE;
  if ((int64_t)max_tasks * (int64_t)slot_floats(G) * 4 > INT32_MAX) return PKV_ERR_INVALID_ARG;  // 32-bit slot offsets
  DecodeArgs a = make_args(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, Hq,
                           Hkv, sm_scale, out, ws_layout(ws, B, Hkv));
  a.tasks = tasks;
  a.split_offsets = split_offsets;
  a.num_tasks = num_tasks;
  a.max_tasks = max_tasks;
  // grid: max_tasks, capped at the workgroups the device holds at once (each workgroup
  // loops over tasks with the grid as stride)
  return from_hip(launch_decode(a, G, flags == PKV_FUSED_MERGE ? 1 : 0, max_tasks, stream, start, stop));
}

int pkv_decode(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t num_pages,
               const int32_t* block_table, int32_t max_pages_per_row, const int32_t* seq_lens, int32_t B,
               int32_t Hq, int32_t Hkv, int32_t d, const pkv_task* tasks, const int32_t* split_offsets,
               const int32_t* num_tasks, int32_t max_tasks, float sm_scale, int32_t flags, uint16_t* out,
               void* ws, size_t ws_bytes, hipStream_t stream) {
  return pkv_decode_timed(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, Hq, Hkv,
                          d, tasks, split_offsets, num_tasks, max_tasks, sm_scale, flags, out, ws, ws_bytes, stream,
                          nullptr, nullptr);
}

int pkv_decode_rect(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t num_pages,
                    const int32_t* block_table, int32_t max_pages_per_row, const int32_t* seq_lens, int32_t B,
                    int32_t Hq, int32_t Hkv, int32_t d, const int32_t* row_ids, int32_t n_rows, int32_t S,
                    int32_t tile_tokens, float sm_scale, uint16_t* out, void* ws, size_t ws_bytes,
                    hipStream_t stream) {
  int st = check_pool(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, out);
  if (st != PKV_OK || (st = check_ws(ws)) != PKV_OK) return st;
  int G = 0;
  if ((st = check_heads(Hq, Hkv, d, &G)) != PKV_OK) return st;
  if (S < 1 || S > kMaxSplits || !std::isfinite(sm_scale)) return PKV_ERR_INVALID_ARG;
  if (tile_tokens <= 0 || tile_tokens % kPageSize != 0) return PKV_ERR_UNSUPPORTED;
  if (row_ids) {
    if (n_rows < 1 || n_rows > kMaxRectRows) return PKV_ERR_INVALID_ARG;
    for (int j = 0; j < n_rows; ++j)
      if (row_ids[j] < 0 || row_ids[j] >= B) return PKV_ERR_INVALID_ARG;
  }
  const int32_t rows = row_ids ? n_rows : B;
  const int32_t slots = pkv_max_tasks(rows, Hkv, S);
  if (slots < 0) return PKV_ERR_INVALID_ARG;
  if (ws_bytes < pkv_workspace_size(B, Hq, Hkv, d, slots)) return PKV_ERR_WORKSPACE;
  if ((int64_t)slots * (int64_t)slot_floats(G) * 4 > INT32_MAX) return PKV_ERR_INVALID_ARG;  // 32-bit slot offsets
  DecodeArgs a = make_args(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, Hq,
                           Hkv, sm_scale, out, ws_layout(ws, B, Hkv));
  a.S = S;
  a.tile_tokens = tile_tokens;
  a.max_tasks = slots;
  a.n_rows = row_ids ? n_rows : 0;
  for (int j = 0; j < a.n_rows; ++j) a.row_ids[j] = row_ids[j];
  return from_hip(launch_decode(a, G, 2, slots, stream));
}

int pkv_decode_buckets(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t num_pages,
                       const int32_t* block_table, int32_t max_pages_per_row, const int32_t* seq_lens,
                       const int32_t* host_seq_lens, int32_t B, int32_t Hq, int32_t Hkv, int32_t d,
                       int32_t bucket_tokens, const pkv_plan_params* params, float sm_scale, uint16_t* out,
                       void* ws, size_t ws_bytes, hipStream_t stream, int32_t* launches) {
  int st = check_pool(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, out);
  if (st != PKV_OK || (st = check_ws(ws)) != PKV_OK) return st;
  int G = 0;
  if ((st = check_heads(Hq, Hkv, d, &G)) != PKV_OK) return st;
  if (!host_seq_lens || !params || bucket_tokens < 0 || !std::isfinite(sm_scale)) return PKV_ERR_INVALID_ARG;
  const pkv_plan_params p = *params;
  if (p.page_size != kPageSize || p.tile_tokens <= 0 || p.tile_tokens % kPageSize != 0) return PKV_ERR_UNSUPPORTED;
  if (p.num_kv_heads != Hkv || p.split_min < 1 || p.split_min > p.split_max || p.target_tasks < 1)
    return PKV_ERR_INVALID_ARG;
  // group rows by route length (exact length, or ceil(length / bucket_tokens)); empty
  // rows form their own group so that their output is written as zeros
  std::vector<std::pair<int64_t, int32_t>> keyed(B);
  for (int32_t i = 0; i < B; ++i) {
    const int32_t n = host_seq_lens[i];
    if (n < 0) return PKV_ERR_INVALID_ARG;
    const int64_t key = n == 0 ? -1 : (bucket_tokens == 0 ? n : (n + bucket_tokens - 1) / bucket_tokens);
    keyed[i] = {key, i};
  }
  std::stable_sort(keyed.begin(), keyed.end(),
                   [](const std::pair<int64_t, int32_t>& x, const std::pair<int64_t, int32_t>& y) {
                     return x.first < y.first;
                   });
  struct Bucket {
    int32_t first, count, S;
  };
  std::vector<Bucket> buckets;
  int64_t need = 0;
  for (int32_t b = 0; b < B;) {
    int32_t e = b;
    while (e < B && keyed[e].first == keyed[b].first && e - b < kMaxRectRows) ++e;
    const int32_t nb = e - b;
    int64_t S = (p.target_tasks + (int64_t)nb * Hkv - 1) / ((int64_t)nb * Hkv);
    S = std::min<int64_t>(std::max<int64_t>(S, p.split_min), p.split_max);
    buckets.push_back({b, nb, (int32_t)S});
    need = std::max<int64_t>(need, (int64_t)nb * Hkv * S);
    b = e;
  }
  if (need > INT32_MAX || ws_bytes < pkv_workspace_size(B, Hq, Hkv, d, (int32_t)need)) return PKV_ERR_WORKSPACE;
  if (need * (int64_t)slot_floats(G) * 4 > INT32_MAX) return PKV_ERR_INVALID_ARG;
  int32_t count = 0;
  for (const Bucket& bk : buckets) {  // one rectangular split launch + one merge launch per bucket
    int32_t ids[kMaxRectRows];
    for (int32_t j = 0; j < bk.count; ++j) ids[j] = keyed[bk.first + j].second;
    st = pkv_decode_rect(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, Hq, Hkv, d,
                         ids, bk.count, bk.S, p.tile_tokens, sm_scale, out, ws, ws_bytes, stream);
    if (st != PKV_OK) return st;
    count += 2;
  }
  if (launches) *launches = count;
  return PKV_OK;
}

int pkv_check_device_status(void* ws, hipStream_t stream, uint32_t* error_bits) {
  if (!ws) return PKV_ERR_INVALID_ARG;
  if (hipStreamSynchronize(stream) != hipSuccess) return PKV_ERR_HIP;
  uint32_t hdr[3] = {0, 0, 0};
  if (hipMemcpy(hdr, ws, sizeof(hdr), hipMemcpyDeviceToHost) != hipSuccess) return PKV_ERR_HIP;
  const uint32_t bits = hdr[0];
  if (launch_zero(ws, sizeof(uint32_t), stream) != hipSuccess) return PKV_ERR_HIP;
  // A flagged call may have skipped tasks before they were counted (a task list or
  // split_offsets that is not a plan of this batch), leaving completion counters short
  // of their split count. Every call has finished here, so the counters recorded by
  // pkv_workspace_init are restored to zero for the next fused call.
  if (bits && hdr[1] > 0 && (hdr[1] ^ kWsCheckKey) == hdr[2] &&
      launch_zero(static_cast<char*>(ws) + kWsHeaderBytes, (size_t)hdr[1] * 4, stream) != hipSuccess)
    return PKV_ERR_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return PKV_ERR_HIP;
  if (error_bits) *error_bits = bits;
  return bits ? PKV_ERR_DEVICE : PKV_OK;
}

const char* pkv_status_string(int status) {
  switch (status) {
    case PKV_OK: return "ok";
    case PKV_ERR_INVALID_ARG: return "invalid argument";
    case PKV_ERR_UNSUPPORTED: return "unsupported shape or parameter";
    case PKV_ERR_WORKSPACE: return "workspace or task capacity too small";
    case PKV_ERR_HIP: return "HIP runtime error";
    case PKV_ERR_DEVICE: return "device-side error flagged";
    default: return "unknown status";
  }
}

int pkv_stream_copy(const void* src, void* dst, size_t bytes, hipStream_t stream) {
  if (!src || !dst || bytes % 16 != 0 || !aligned(src, 16) || !aligned(dst, 16)) return PKV_ERR_INVALID_ARG;
  return from_hip(launch_copy(src, dst, bytes, stream));
}

int pkv_stream_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream) {
  return pkv_stream_read_timed(src, bytes, sink, stream, nullptr, nullptr);
}

int pkv_stream_read_timed(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream, hipEvent_t start,
                          hipEvent_t stop) {
  if (!src || !sink || bytes % 16 != 0 || !aligned(src, 16) || !aligned(sink, 4)) return PKV_ERR_INVALID_ARG;
  return from_hip(launch_read(src, bytes, sink, stream, start, stop));
}

int pkv_stream_read_nt_timed(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream, hipEvent_t start,
                             hipEvent_t stop) {
  if (!src || !sink || bytes % 16 != 0 || !aligned(src, 16) || !aligned(sink, 4)) return PKV_ERR_INVALID_ARG;
  return from_hip(launch_read(src, bytes, sink, stream, start, stop, true));
}

int pkv_stream_read_pages(const uint16_t* k_cache, const uint16_t* v_cache, int32_t num_pages,
                          const int32_t* block_table, int32_t max_pages_per_row, int32_t B, int32_t Hkv, int32_t d,
                          const pkv_task* tasks, const int32_t* num_tasks, int32_t max_tasks,
                          int32_t heads_per_workgroup, uint32_t* sink, hipStream_t stream, hipEvent_t start,
                          hipEvent_t stop) {
  if (!k_cache || !v_cache || !block_table || !tasks || !num_tasks || !sink) return PKV_ERR_INVALID_ARG;
  if (num_pages < 1 || max_pages_per_row < 1 || B < 1 || Hkv < 1 || Hkv > 256 || max_tasks < 1)
    return PKV_ERR_INVALID_ARG;
  if ((int64_t)max_pages_per_row * kPageSize > INT32_MAX) return PKV_ERR_INVALID_ARG;
  if (d != kHeadDim) return PKV_ERR_UNSUPPORTED;
  if (heads_per_workgroup != 1 && heads_per_workgroup != 2) return PKV_ERR_INVALID_ARG;
  if (Hkv % heads_per_workgroup != 0) return PKV_ERR_INVALID_ARG;
  if (!aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(tasks, 4) || !aligned(num_tasks, 4) ||
      !aligned(sink, 4))
    return PKV_ERR_INVALID_ARG;
  const PageReadArgs a{k_cache, v_cache, block_table, tasks, num_tasks, sink, num_pages, max_pages_per_row, B, Hkv,
                       max_tasks};
  return from_hip(launch_page_read(a, heads_per_workgroup, stream, start, stop));
}

}  // extern "C"

namespace {

// pkv_plan_decode and pkv_plan_decode_noalloc: every check, then the one-launch kernel
// with its error word, counters and slots at `*sc`, or (sc == nullptr) in the library's
// scratch of the current device with the error word `err`. `slot_bytes` is the room for
// partial-state slots.
int plan_decode(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t num_pages,
                const int32_t* block_table, int32_t max_pages_per_row, const int32_t* seq_lens, int32_t B, int32_t Hq,
                int32_t Hkv, int32_t d, const pkv_plan_params* params, pkv_task* tasks, int32_t max_tasks,
                int32_t* split_offsets, int32_t* num_tasks, float sm_scale, uint16_t* out, const Scratch* sc,
                unsigned* err, size_t slot_bytes, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
  int st = check_pool(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, out);
  if (st != PKV_OK) return st;
  int G = 0;
  if ((st = check_heads(Hq, Hkv, d, &G)) != PKV_OK) return st;
  if (!std::isfinite(sm_scale)) return PKV_ERR_INVALID_ARG;
  if (B > kMaxFusedPlanBatch) return PKV_ERR_UNSUPPORTED;
  if (params && params->num_kv_heads != Hkv) return PKV_ERR_INVALID_ARG;
  PlanArgs pa;
  if ((st = make_plan_args(seq_lens, nullptr, B, max_pages_per_row, num_pages, params, tasks, max_tasks,
                           split_offsets, num_tasks, Scratch{nullptr, nullptr, nullptr}, &pa)) != PKV_OK)
    return st;
  const int64_t state_bytes = (int64_t)max_tasks * (int64_t)slot_floats(G) * 4;
  if (state_bytes > (int64_t)slot_bytes) return PKV_ERR_WORKSPACE;
  if (state_bytes > INT32_MAX) return PKV_ERR_INVALID_ARG;  // 32-bit slot offsets
  Scratch at{};
  if (sc) {
    at = *sc;
  } else {  // every check has passed: only now is the device touched
    char* base = nullptr;
    if (static_scratch(stream, &base) != hipSuccess) return PKV_ERR_HIP;
    at = Scratch{err, reinterpret_cast<int32_t*>(base), reinterpret_cast<float*>(base + kScratchCounterBytes)};
  }
  pa.err = at.err;
  pa.counters = at.counters;
  DecodeArgs a = make_args(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, Hq,
                           Hkv, sm_scale, out, at);
  a.tasks = tasks;
  a.split_offsets = split_offsets;
  a.num_tasks = num_tasks;
  a.max_tasks = max_tasks;
  a.plan = pa;
  return from_hip(launch_decode(a, G, 3, max_tasks, stream, start, stop));
}

}  // namespace

extern "C" {

int pkv_plan_decode_timed(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t num_pages,
                          const int32_t* block_table, int32_t max_pages_per_row, const int32_t* seq_lens,
                          int32_t B, int32_t Hq, int32_t Hkv, int32_t d, const pkv_plan_params* params,
                          pkv_task* tasks, int32_t max_tasks, int32_t* split_offsets, int32_t* num_tasks,
                          float sm_scale, uint16_t* out, void* ws, size_t ws_bytes, hipStream_t stream,
                          hipEvent_t start, hipEvent_t stop) {
  int st = check_ws(ws);
  if (st != PKV_OK) return st;
  if (B < 1 || Hkv < 1) return PKV_ERR_INVALID_ARG;
  const size_t slots_at = partials_offset(B, Hkv);
  if (ws_bytes < slots_at) return PKV_ERR_WORKSPACE;
  const Scratch sc = ws_layout(ws, B, Hkv);
  return plan_decode(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, Hq, Hkv, d, params,
                     tasks, max_tasks, split_offsets, num_tasks, sm_scale, out, &sc, nullptr, ws_bytes - slots_at,
                     stream, start, stop);
}

int pkv_plan_decode_noalloc(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                            int32_t num_pages, const int32_t* block_table, int32_t max_pages_per_row,
                            const int32_t* seq_lens, int32_t B, int32_t Hq, int32_t Hkv, int32_t d,
                            const pkv_plan_params* params, pkv_task* tasks, int32_t max_tasks,
                            int32_t* split_offsets, int32_t* num_tasks, float sm_scale, uint16_t* out,
                            uint32_t* error_bits, hipStream_t stream) {
  if (!error_bits || !aligned(error_bits, 4)) return PKV_ERR_INVALID_ARG;
  if (B < 1 || Hkv < 1) return PKV_ERR_INVALID_ARG;
  if ((int64_t)B * Hkv > kScratchCounters) return PKV_ERR_WORKSPACE;
  return plan_decode(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, Hq, Hkv, d, params,
                     tasks, max_tasks, split_offsets, num_tasks, sm_scale, out, nullptr, error_bits,
                     kScratchBytes - kScratchCounterBytes, stream, nullptr, nullptr);
}

int pkv_plan_decode(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache, int32_t num_pages,
                    const int32_t* block_table, int32_t max_pages_per_row, const int32_t* seq_lens, int32_t B,
                    int32_t Hq, int32_t Hkv, int32_t d, const pkv_plan_params* params, pkv_task* tasks,
                    int32_t max_tasks, int32_t* split_offsets, int32_t* num_tasks, float sm_scale, uint16_t* out,
                    void* ws, size_t ws_bytes, hipStream_t stream) {
  return pkv_plan_decode_timed(q, k_cache, v_cache, num_pages, block_table, max_pages_per_row, seq_lens, B, Hq,
                               Hkv, d, params, tasks, max_tasks, split_offsets, num_tasks, sm_scale, out, ws,
                               ws_bytes, stream, nullptr, nullptr);
}

}  // extern "C"
