/*
 * pkv: paged grouped-query decode attention for MI355X (gfx950).
 *
 * C ABI of libpkv.so. One decode step is
 *
 *     pkv_plan   : seq_lens -> compact task list + split_offsets       (one kernel)
 *     pkv_decode : tasks, Q, paged K/V -> out                          (one fused kernel,
 *                                                                       or split + merge)
 *
 * The operation is single-token decode attention, Eq. (1) of the paper, with grouped
 * query heads (Sec. 3.1): query head h reads KV head h / G, G = Hq / Hkv. K and V are
 * read in place through a block table (Sec. 3.2). The sequence is cut into splits whose
 * online-softmax partial states are merged exactly (Sec. 3.3), and the workqueue holds
 * only non-empty (row, KV head, split) tasks (Sec. 3.4).
 *
 * Conventions shared by every call:
 *  - Device pointers are HIP device memory owned by the caller. The library never
 *    allocates or frees memory and never synchronizes, except pkv_check_device_status.
 *    (pkv_plan_decode_noalloc keeps its counters and partial states in a fixed scratch
 *    area of each device's memory that the loaded library holds.)
 *  - All work is enqueued on `stream` and is asynchronous. A nonzero return means
 *    nothing was enqueued.
 *  - Tensors are row-major and contiguous; fp16 buffers hold IEEE binary16 bit patterns
 *    (uint16_t) and the arithmetic is fp32.
 *  - Host-side validation returns a status synchronously. Faults found on the device
 *    (a page id outside the pool, a length beyond the block table) set bits in the
 *    workspace's error word, read back by pkv_check_device_status, and the affected
 *    rows' outputs are written as zeros.
 *  - Concurrent calls on different streams need separate workspaces and separate
 *    output buffers (task list, split_offsets, num_tasks, out).
 */
#ifndef PKV_H
#define PKV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define PKV_OK 0
#define PKV_ERR_INVALID_ARG 1 /* null pointer, non-positive size, Hq % Hkv != 0, bad bounds */
#define PKV_ERR_UNSUPPORTED 2 /* d != 128, page_size != 16, G not in {1,2,4,8}, tile not a page multiple */
#define PKV_ERR_WORKSPACE 3   /* workspace, max_tasks or a split count too small */
#define PKV_ERR_HIP 4         /* a HIP runtime call or kernel launch failed */
#define PKV_ERR_DEVICE 5      /* pkv_check_device_status found device error bits */

/* Device error bits (pkv_check_device_status). */
#define PKV_DEVERR_SEQ_LEN 1u /* seq_len < 0 or > max_pages_per_row * page_size: row dropped */
#define PKV_DEVERR_PAGE_ID 2u /* block_table entry outside [0, num_pages): row's output zeroed */
#define PKV_DEVERR_TASK 4u    /* a task outside the batch or its row's block table: skipped;
                                 outputs are unspecified unless the task list came from
                                 pkv_plan for the same seq_lens */

/* pkv_decode flags. */
#define PKV_FUSED_MERGE 1 /* merge in the split kernel by the last-arriving split (Sec. 3.4) */

/* One workqueue task (Sec. 3.4): KV head `kvh` of batch row `row`, split `split`,
 * tokens [t_begin, t_end) of that row. 20 bytes, tightly packed. */
typedef struct {
  int32_t row, kvh, split, t_begin, t_end;
} pkv_task;

/* Split policies (pkv_plan_params.policy). tiles_i = ceil(seq_len_i / tile_tokens).
 *   PKV_SPLIT_BATCH  one split count for the step, from the active batch size
 *                    (Sec. 3.5): S = clamp(ceil(target_tasks / max(1, B_active * Hkv)),
 *                    split_min, split_max), B_active = rows with seq_len > 0;
 *                    nsplit_i = min(S, tiles_i)
 *   PKV_SPLIT_QUOTA  per-row split counts from the step's total work, so that every
 *                    task covers about the same number of tiles (the per-row split
 *                    count the paper names as future work, Sec. 5):
 *                    nsplit_i(Q) = min(split_max, ceil(tiles_i / Q)) with Q the
 *                    smallest tile quota >= 1 for which Hkv * sum_i nsplit_i(Q) <=
 *                    target_tasks (max tiles_i if none: one split per row);
 *                    split_min is not used */
#define PKV_SPLIT_BATCH 0
#define PKV_SPLIT_QUOTA 1

/* Planner parameters (host struct).
 *   page_size    tokens per KV page; must be 16
 *   tile_tokens  split granularity in tokens (the paper's 32-token tile, Sec. 3.2);
 *                a positive multiple of page_size
 *   num_kv_heads Hkv
 *   split_min, split_max  split-count bounds, 1 <= split_min <= split_max <= 65536
 *   target_tasks desired task count, >= 1 (see the policies above)
 *   policy       PKV_SPLIT_BATCH or PKV_SPLIT_QUOTA
 * Split s of row i owns tiles [floor(s*tiles_i/nsplit_i), floor((s+1)*tiles_i/nsplit_i)). */
typedef struct {
  int32_t page_size;
  int32_t tile_tokens;
  int32_t num_kv_heads;
  int32_t split_min;
  int32_t split_max;
  int32_t target_tasks;
  int32_t policy;
} pkv_plan_params;

/* Upper bound on the task count of any plan: B * Hkv * split_max. Returns -1 on a
 * non-positive argument or int32 overflow. */
int32_t pkv_max_tasks(int32_t B, int32_t Hkv, int32_t split_max);

/* Bytes of workspace for batches of up to B rows and up to max_tasks partial-state
 * slots: a 256-byte header (error word), B*Hkv completion counters, and max_tasks
 * slots of fp32 {acc[G][d], m[G], l[G]} padded to 16 bytes (2080 bytes at G=4,
 * d=128). Returns 0 on a bad argument. The rectangular route needs
 * max_tasks >= B * Hkv * S. One workspace serves calls with one B: pkv_plan and
 * pkv_decode of a step must pass the same B. */
size_t pkv_workspace_size(int32_t B, int32_t Hq, int32_t Hkv, int32_t d, int32_t max_tasks);

/* Zero the workspace header and completion counters and record the counter count
 * (B * Hkv) in the header (enqueued on `stream`). Call once after allocating a
 * workspace; afterwards every call leaves the counters at zero, and
 * pkv_check_device_status clears the error word and, when it finds error bits, re-zeroes
 * the counters that a flagged call may have left short (see pkv_plan_decode). */
int pkv_workspace_init(void* ws, size_t ws_bytes, int32_t B, int32_t Hkv, hipStream_t stream);

/* Build the compact workqueue of Sec. 3.4 on the device (one kernel).
 *   seq_lens      device int32 [B]: N*_i, the row-local lengths (Sec. 3.3)
 *   block_table   device int32 [B, max_pages_per_row] or NULL; when given, the entries
 *                 each row uses are checked against [0, num_pages) and a row with a bad
 *                 entry gets PKV_DEVERR_PAGE_ID (pkv_decode checks them in any case)
 *   params        host pointer, see pkv_plan_params
 *   tasks         device pkv_task [max_tasks]; entries [0, *num_tasks) are written in
 *                 (row, split, kvh) order, kvh fastest; task k's partial state lives in
 *                 slot k = (split_offsets[row] + split) * Hkv + kvh
 *   split_offsets device int32 [B+1]: split_offsets[i+1] - split_offsets[i] = nsplit_i
 *   num_tasks     device int32 [1]
 *   ws            workspace of at least pkv_workspace_size(B, ., Hkv, ., 0) bytes; the
 *                 plan zeroes the completion counters
 * max_tasks must be >= pkv_max_tasks(B, Hkv, split_max). B <= 4096. Rows whose
 * seq_len is out of range are planned as empty and flagged (PKV_DEVERR_SEQ_LEN). */
int pkv_plan(const int32_t* seq_lens, const int32_t* block_table, int32_t B,
             int32_t max_pages_per_row, int32_t num_pages, const pkv_plan_params* params,
             pkv_task* tasks, int32_t max_tasks, int32_t* split_offsets, int32_t* num_tasks,
             void* ws, size_t ws_bytes, hipStream_t stream);

/* The same plan computed on the host (Sec. 3.4-3.5), for buffer sizing and route
 * costing without a device round trip. Identical task list, split_offsets and count to
 * pkv_plan on the same lengths and parameters.
 *   seq_lens      host int32 [B]; every length must lie in [0, max_pages_per_row * 16]
 *                 (else PKV_ERR_INVALID_ARG: the host reports it at once)
 *   tasks         host pkv_task [max_tasks], or NULL to compute only the counts
 *   split_offsets host int32 [B+1], or NULL
 *   num_tasks     host int32 [1] (always written on success)
 * PKV_ERR_WORKSPACE when tasks is given and max_tasks < the task count (num_tasks and
 * split_offsets are still written). */
int pkv_plan_host(const int32_t* seq_lens, int32_t B, int32_t max_pages_per_row,
                  const pkv_plan_params* params, pkv_task* tasks, int32_t max_tasks,
                  int32_t* split_offsets, int32_t* num_tasks);

/* Decode attention over the task list (Sec. 3.3-3.4).
 *   q          device fp16 [B, Hq, d]
 *   k_cache, v_cache  device fp16 [num_pages, page_size=16, Hkv, d] (token-major pages)
 *   block_table device int32 [B, max_pages_per_row]: logical page -> physical page
 *   seq_lens   device int32 [B]
 *   tasks, split_offsets, num_tasks  as written by pkv_plan for the same seq_lens
 *   max_tasks  capacity used by that plan (bounds the launch)
 *   sm_scale   softmax scale (1/sqrt(d) of Eq. 1 unless Q is pre-scaled)
 *   flags      0: split kernel + merge kernel; PKV_FUSED_MERGE: one kernel in which the
 *              last split of each (row, KV head) to finish merges, in split order
 *   out        device fp16 [B, Hq, d]; rows with seq_len 0 are written as zeros
 *   ws         workspace of at least pkv_workspace_size(B, Hq, Hkv, d, max_tasks) bytes
 * Both flag values give bit-identical outputs. Supported: d = 128, G in {1,2,4,8}. */
int pkv_decode(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
               int32_t num_pages, const int32_t* block_table, int32_t max_pages_per_row,
               const int32_t* seq_lens, int32_t B, int32_t Hq, int32_t Hkv, int32_t d,
               const pkv_task* tasks, const int32_t* split_offsets, const int32_t* num_tasks,
               int32_t max_tasks, float sm_scale, int32_t flags, uint16_t* out, void* ws,
               size_t ws_bytes, hipStream_t stream);

/* pkv_plan followed by pkv_decode with PKV_FUSED_MERGE, in one kernel launch: every
 * workgroup runs the planner's arithmetic on seq_lens and takes its task from the
 * result, and the first workgroup also writes tasks, split_offsets and num_tasks exactly
 * as pkv_plan writes them. Arguments as for pkv_plan and pkv_decode; the block table is
 * checked by the decode (not by the planner), B <= 1024, params->num_kv_heads == Hkv.
 * The completion counters must be zero at launch: pkv_workspace_init zeroes them,
 * and every completed pkv_plan, pkv_plan_decode or pkv_decode call leaves them zero,
 * except a pkv_decode whose task list or split_offsets is not a plan of its seq_lens
 * (PKV_DEVERR_TASK): such a call may leave counters short of their split count, and
 * pkv_check_device_status re-zeroes them when it reports the error (for a workspace
 * set up by pkv_workspace_init; pkv_plan also zeroes them).
 * The previous contents of `tasks` (for B <= 64) are read as a scheduling hint: each
 * workgroup starts loading the task listed at its own index while the planner runs and
 * keeps those loads only if the new plan gives it the same pages. Any contents are
 * allowed (out-of-range records are ignored) and never change a result.
 * With G = 4, Hkv even and params->target_tasks at least twice the workgroups the
 * device holds at once (512 on MI355X), each workgroup runs two tasks together: KV heads
 * g and g + 1 of one split, whose slices of each token are adjacent (its hint is then
 * the record at twice its index). This changes only which workgroup computes what.
 * Outputs are bit-identical to the two-call sequence. */
int pkv_plan_decode(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                    int32_t num_pages, const int32_t* block_table, int32_t max_pages_per_row,
                    const int32_t* seq_lens, int32_t B, int32_t Hq, int32_t Hkv, int32_t d,
                    const pkv_plan_params* params, pkv_task* tasks, int32_t max_tasks,
                    int32_t* split_offsets, int32_t* num_tasks, float sm_scale, uint16_t* out,
                    void* ws, size_t ws_bytes, hipStream_t stream);

/* pkv_plan_decode for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same launch, with
 * the completion counters and partial-state slots in a scratch area the library holds in
 * each device's memory (16 MiB per device that runs this call, held until the process
 * ends) instead of a caller's workspace. The call allocates nothing and performs no
 * memset; its first call on a device looks up the scratch's address and zeroes its
 * counters with a small kernel on `stream`.
 *   error_bits  device uint32 [1], OR-ed with the device error bits of pkv_plan_decode
 *               (PKV_DEVERR_*); the caller zeroes it and reads it when it wishes
 *   other arguments as for pkv_plan_decode
 * Limits: B * Hkv <= 16384 and max_tasks * slot bytes <= 16 MiB - 64 KiB (slot bytes as
 * in pkv_workspace_size: 2080 at G = 4, i.e. max_tasks <= 8034), else
 * PKV_ERR_WORKSPACE with nothing enqueued. Every call on a device shares that device's
 * scratch: calls that overlap in time on one device (different streams, or different
 * host threads) race and give wrong results; calls in order on one stream are safe,
 * whatever their sizes. Outputs are bit-identical to pkv_plan_decode's. */
int pkv_plan_decode_noalloc(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                            int32_t num_pages, const int32_t* block_table, int32_t max_pages_per_row,
                            const int32_t* seq_lens, int32_t B, int32_t Hq, int32_t Hkv, int32_t d,
                            const pkv_plan_params* params, pkv_task* tasks, int32_t max_tasks,
                            int32_t* split_offsets, int32_t* num_tasks, float sm_scale, uint16_t* out,
                            uint32_t* error_bits, hipStream_t stream);

/* pkv_decode and pkv_plan_decode with kernel-execution timestamps, for measurement:
 * start is recorded when the call's first kernel begins executing and stop when its
 * last kernel has finished (the interval a profiler reports, without the queue's own
 * packet latency). start and stop are events created by the caller (hipEventCreate, or
 * a timing event that has been recorded once); either may be NULL. Results and errors
 * as for the untimed calls. */
int pkv_decode_timed(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                     int32_t num_pages, const int32_t* block_table, int32_t max_pages_per_row,
                     const int32_t* seq_lens, int32_t B, int32_t Hq, int32_t Hkv, int32_t d,
                     const pkv_task* tasks, const int32_t* split_offsets, const int32_t* num_tasks,
                     int32_t max_tasks, float sm_scale, int32_t flags, uint16_t* out, void* ws,
                     size_t ws_bytes, hipStream_t stream, hipEvent_t start, hipEvent_t stop);
int pkv_plan_decode_timed(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                          int32_t num_pages, const int32_t* block_table, int32_t max_pages_per_row,
                          const int32_t* seq_lens, int32_t B, int32_t Hq, int32_t Hkv, int32_t d,
                          const pkv_plan_params* params, pkv_task* tasks, int32_t max_tasks,
                          int32_t* split_offsets, int32_t* num_tasks, float sm_scale, uint16_t* out,
                          void* ws, size_t ws_bytes, hipStream_t stream, hipEvent_t start,
                          hipEvent_t stop);

/* Rectangular split grid (Sec. 3.4): rows * Hkv * S split workgroups, then a merge over
 * all S columns (two kernels, no planner). Column s of a row owns the same balanced tile
 * range the planner gives split s when s < min(S, tiles); otherwise it writes the
 * neutral state (-inf, 0, 0) and exits before loading Q (Sec. 3.3). The launch covers
 * rows 0..B-1 when row_ids is NULL, else the n_rows (1..64) rows listed in the HOST
 * array row_ids, reading Q and writing out by index (indexed Q/O, Sec. 4.6). With the
 * same S the output is bit-identical to pkv_decode. 1 <= S <= 65536. ws needs
 * max_tasks >= rows * Hkv * S;
 * tile_tokens as in pkv_plan_params. */
int pkv_decode_rect(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                    int32_t num_pages, const int32_t* block_table, int32_t max_pages_per_row,
                    const int32_t* seq_lens, int32_t B, int32_t Hq, int32_t Hkv, int32_t d,
                    const int32_t* row_ids, int32_t n_rows, int32_t S, int32_t tile_tokens,
                    float sm_scale, uint16_t* out, void* ws, size_t ws_bytes, hipStream_t stream);

/* Length-bucket route (Sec. 3.4, Sec. 4.5): rows grouped on the host by route length
 * and one pkv_decode_rect launch pair per group, on `stream` in order.
 *   host_seq_lens  HOST int32 [B], equal to the device seq_lens
 *   bucket_tokens  0: exact-length buckets (one group per distinct length);
 *                  > 0: coarse buckets, rows grouped by ceil(len / bucket_tokens) and
 *                  masked to their own lengths (row-local bounds, Sec. 3.3)
 *   params         split bounds, target and tile: a group of n rows gets
 *                  S = clamp(ceil(target_tasks / (n * Hkv)), split_min, split_max)
 *   launches       optional host output: kernel launches issued (2 per group)
 * Groups hold at most 64 rows (larger groups are cut). Rows of length 0 form a group
 * whose output is written as zeros. ws needs max_tasks >= max over groups of
 * n * Hkv * S. */
int pkv_decode_buckets(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                       int32_t num_pages, const int32_t* block_table, int32_t max_pages_per_row,
                       const int32_t* seq_lens, const int32_t* host_seq_lens, int32_t B, int32_t Hq,
                       int32_t Hkv, int32_t d, int32_t bucket_tokens, const pkv_plan_params* params,
                       float sm_scale, uint16_t* out, void* ws, size_t ws_bytes, hipStream_t stream,
                       int32_t* launches);

/* Synchronize `stream`, read the workspace error word into *error_bits (may be NULL)
 * and clear it. Returns PKV_OK when no bit was set, PKV_ERR_DEVICE otherwise. */
int pkv_check_device_status(void* ws, hipStream_t stream, uint32_t* error_bits);

/* Static text for a status code. */
const char* pkv_status_string(int status);

/* Streaming copy of `bytes` (a multiple of 16) from src to dst on `stream`: a kernel of
 * known traffic, used to calibrate HBM traffic counters. */
int pkv_stream_copy(const void* src, void* dst, size_t bytes, hipStream_t stream);

/* Streaming read of `bytes` (a multiple of 16) at src on `stream`, with allocating
 * (default-policy) loads: a read-bandwidth probe (the paper's streaming-bandwidth
 * calibration, Sec. 3.5; pkv_stream_read_nt_timed measures it with the decode's load
 * policy) and a way to evict the last-level cache with clean lines between timed
 * steps. `sink` is a device word that is written only if the data hashes to a fixed
 * value. */
int pkv_stream_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream);

/* pkv_stream_read with start/stop events stamped by the launch itself (the kernel's
 * execution interval, as for pkv_decode_timed); either event may be NULL. */
int pkv_stream_read_timed(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream,
                          hipEvent_t start, hipEvent_t stop);

/* pkv_stream_read_timed with non-temporal loads, the cache policy of the decode kernel's
 * K and V page loads (each KV byte is read once per step): the streaming-read ceiling
 * for that policy. Arguments, errors and events as for pkv_stream_read_timed. Not meant
 * for evicting the last-level cache: use pkv_stream_read, whose loads allocate. */
int pkv_stream_read_nt_timed(const void* src, size_t bytes, uint32_t* sink, hipStream_t stream,
                             hipEvent_t start, hipEvent_t stop);

/* Read-only probe of the decode kernel's KV access pattern (the read-bandwidth term of
 * the cost model, Sec. 3.5, measured for the paged layout of Sec. 3.2 instead of a
 * contiguous stream). For each of the first min(*num_tasks, max_tasks) records of
 * `tasks` (as pkv_plan / pkv_plan_decode write them), the K and V bytes of the task's
 * KV heads over the pages of its token range are read with the loads, waves, loads in
 * flight, grid and task-to-workgroup mapping of the one-launch decode kernel:
 * heads_per_workgroup = 1 runs one task per workgroup, 2 the tasks 2p and 2p + 1 (KV
 * heads g, g + 1) together, as the decode's KV-head pairs do. No query is read, nothing
 * is computed or written except `sink`, a device word written only if the data hash to
 * a fixed value. Its duration is the time to read the decode's pages in the decode's
 * pattern: the read ceiling of a decode step with that plan.
 *   k_cache, v_cache  device, [num_pages, 16, Hkv, d] fp16 (16-byte aligned)
 *   block_table       device int32 [B, max_pages_per_row]
 *   tasks, num_tasks  device, a plan's task list and count; records naming a row, head
 *                     or token range outside the arguments' bounds are skipped, and
 *                     page ids outside [0, num_pages) are not read
 *   d                 must be 128 (PKV_ERR_UNSUPPORTED otherwise)
 *   start, stop       events stamped by the launch itself (kernel execution interval);
 *                     either may be NULL
 * Returns PKV_ERR_INVALID_ARG for null or misaligned pointers, non-positive sizes,
 * Hkv > 256, heads_per_workgroup not 1 or 2 or not dividing Hkv. Enqueues one kernel on
 * `stream`; allocates nothing. */
int pkv_stream_read_pages(const uint16_t* k_cache, const uint16_t* v_cache, int32_t num_pages,
                          const int32_t* block_table, int32_t max_pages_per_row, int32_t B, int32_t Hkv, int32_t d,
                          const pkv_task* tasks, const int32_t* num_tasks, int32_t max_tasks,
                          int32_t heads_per_workgroup, uint32_t* sink, hipStream_t stream, hipEvent_t start,
                          hipEvent_t stop);

#ifdef __cplusplus
}
#endif

#endif /* PKV_H */
