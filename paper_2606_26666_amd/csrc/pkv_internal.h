// Internal interface between the C ABI (pkv_capi.cpp) and the kernels (pkv_kernels.hip).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/pkv.h"

namespace pkv {

constexpr int kHeadDim = 128;
constexpr int kPageSize = 16;
constexpr int kMaxPlanBatch = 4096;
constexpr int kMaxFusedPlanBatch = 1024;
constexpr int kMaxSplits = 65536;  // split_max and the rectangular S: keeps split bounds in 32 bits
constexpr int kMaxRectRows = 64;  // rows a rectangular launch can name (kernel arguments)
constexpr size_t kWsHeaderBytes = 256;
// workspace header words: 0 device error bits, 1 completion-counter count (written by
// pkv_workspace_init), 2 that count xor kWsCheckKey
constexpr int kWsCountWord = 1;
constexpr int kWsCheckWord = 2;
constexpr uint32_t kWsCheckKey = 0x5A17C0DEu;
// library-held scratch of pkv_plan_decode_noalloc, per device: counters for up to
// kScratchCounters (row, KV head) pairs, then partial-state slots
constexpr size_t kScratchBytes = size_t(16) << 20;
constexpr int kScratchCounters = 16384;
constexpr size_t kScratchCounterBytes = size_t(kScratchCounters) * 4;
constexpr int kMaxDevices = 64;

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
// fp32 acc[G][d], m[G], l[G], padded to 16 bytes
inline size_t slot_floats(int G) { return size_t(G * kHeadDim + ((2 * G + 3) / 4) * 4); }
inline size_t counters_bytes(int B, int Hkv) { return align256(size_t(B) * size_t(Hkv) * 4); }
inline size_t partials_offset(int B, int Hkv) { return kWsHeaderBytes + counters_bytes(B, Hkv); }

struct PlanArgs {
  const int32_t* seq_lens;
  const int32_t* block_table;
  int32_t B, max_pages_per_row, num_pages;
  int32_t page_size, tile_tokens, Hkv, split_min, split_max, target_tasks, policy;
  pkv_task* tasks;
  int32_t max_tasks;
  int32_t* split_offsets;
  int32_t* num_tasks;
  unsigned* err;
  int32_t* counters;
};

struct DecodeArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const pkv_task* tasks;
  const int32_t* split_offsets;
  const int32_t* num_tasks;
  uint16_t* out;
  unsigned* err;
  int32_t* counters;
  float* partials;
  int32_t num_pages;
  int32_t max_pages_per_row;
  int32_t B, Hq, Hkv;
  int32_t max_tasks;
  int32_t S;            // rectangular route only
  int32_t tile_tokens;  // rectangular route only
  int32_t n_rows;       // rectangular route: rows named in row_ids (0: rows 0..B-1)
  float scale_log2;     // sm_scale * log2(e)
  PlanArgs plan;        // planning inside the decode launch (pkv_plan_decode)
  int32_t row_ids[kMaxRectRows];  // last: only the rectangular route reads it
};


hipError_t launch_plan(const PlanArgs& a, hipStream_t s);
// mode: 0 split + merge kernels, 1 fused merge, 2 rectangular split + merge,
//       3 plan + split + fused merge in one launch
// start/stop (may be null): stamped when the call's first kernel starts and its last ends
hipError_t launch_decode(const DecodeArgs& a, int G, int mode, int grid, hipStream_t s,
                         hipEvent_t start = nullptr, hipEvent_t stop = nullptr);
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);
hipError_t launch_ws_init(void* ws, size_t bytes, uint32_t counters, hipStream_t s);
// device address of the current device's library-held scratch; the first call on a
// device zeroes its counters on stream s
hipError_t static_scratch(hipStream_t s, char** base);
hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t s);
// Arguments of the read-only probe of the decode's page pattern (pkv_stream_read_pages).
struct PageReadArgs {
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* block_table;
  const pkv_task* tasks;
  const int32_t* num_tasks;
  unsigned* sink;
  int32_t num_pages, max_pages_per_row, B, Hkv, max_tasks;
};
hipError_t launch_page_read(const PageReadArgs& a, int heads_per_workgroup, hipStream_t s, hipEvent_t start,
                            hipEvent_t stop);
hipError_t launch_read(const void* src, size_t bytes, unsigned* sink, hipStream_t s, hipEvent_t start = nullptr,
                       hipEvent_t stop = nullptr, bool non_temporal = false);

}  // namespace pkv
