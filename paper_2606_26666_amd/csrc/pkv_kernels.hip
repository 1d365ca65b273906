// HIP kernels for paged grouped-query decode attention on CDNA4 (gfx950).
//
//   plan_kernel     compact workqueue of non-empty (row, KV head, split) tasks (Sec. 3.4)
//   split_kernel    online-softmax partial state per task (Sec. 3.2-3.3), optionally
//                   followed by the last-arriver merge (Sec. 3.4); also the rectangular
//                   (B, Hkv, S) grid with neutral empty splits (Sec. 3.3)
//   merge_kernel    exact segmented merge of split states (Sec. 3.3)
//
// Work mapping. One workgroup owns one task: one KV head g of one row and a token
// range [t0, t1). Its W wavefronts take the range's 16-token pages round-robin. A
// wavefront reads one page of one head as four 1 KiB loads: lane (r, c) = (lane/16,
// lane%16) loads 16 bytes (8 halves, dims 8c..8c+7) of token 4i+r, so every load covers
// four whole 256-byte head rows. Each lane keeps the G query vectors' matching 8 dims,
// forms partial dot products with v_dot2_f32_f16 and a 16-lane DPP butterfly completes
// them, so all 16 lanes of a row hold the scores of their token for all G query heads.
// Each of the four lane rows then runs its own online softmax (m, l, acc[G][8 dims]) in
// fp32 over the tokens it saw. At the end of the task a lane butterfly combines the
// four rows of each wavefront and LDS combines the W wavefront states, in a fixed order.
#include <hip/hip_runtime.h>

#include "pkv_internal.h"

namespace pkv {
namespace {

constexpr int D = kHeadDim;
constexpr int P = kPageSize;

typedef _Float16 h2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}

// Sum over the 16 lanes of a DPP row; every lane of the row receives the same value.
__device__ __forceinline__ float row_sum16(float x) {
  x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp<0x141>(x);  // row_half_mirror
  x += dpp<0x140>(x);  // row_mirror
  return x;
}

__device__ __forceinline__ h2 as_h2(unsigned u) { return __builtin_bit_cast(h2, u); }

__device__ __forceinline__ float dot8(const uint4& a, const uint4& b) {
  float s = __builtin_amdgcn_fdot2(as_h2(a.x), as_h2(b.x), 0.0f, false);
  s = __builtin_amdgcn_fdot2(as_h2(a.y), as_h2(b.y), s, false);
  s = __builtin_amdgcn_fdot2(as_h2(a.z), as_h2(b.z), s, false);
  s = __builtin_amdgcn_fdot2(as_h2(a.w), as_h2(b.w), s, false);
  return s;
}

__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint16_t f32_to_f16_bits(float x) {
  return __builtin_bit_cast(uint16_t, static_cast<_Float16>(x));
}

__device__ __forceinline__ void unpack8(const uint4& u, float f[8]) {
  h2 a = as_h2(u.x), b = as_h2(u.y), c = as_h2(u.z), d = as_h2(u.w);
  f[0] = (float)a.x; f[1] = (float)a.y; f[2] = (float)b.x; f[3] = (float)b.y;
  f[4] = (float)c.x; f[5] = (float)c.y; f[6] = (float)d.x; f[7] = (float)d.y;
}

constexpr float kNegInf = -__builtin_inff();

// ---------------------------------------------------------------------------------
// Merge of split states (Sec. 3.3): M = max m_s, L = sum 2^(m_s-M) l_s,
// A = sum 2^(m_s-M) a_s, O = A / L, in split order. States hold m in log2 units.
// l_s < 0 marks a split that met an invalid page; such a (row, KV head) is zeroed.
// Every merge in the library goes through this one function so that all routes round
// identically.
template <int G>
__device__ __forceinline__ float merge_elem(const float* __restrict__ partials, int slot0, int stride,
                                            int nsplit, int h, int dcol) {
  constexpr int SF = 2 * G + G * D;
  float M = kNegInf;
  bool bad = false;
  for (int s = 0; s < nsplit; ++s) {
    const float* st = partials + (size_t)(slot0 + s * stride) * SF;
    M = fmaxf(M, st[h]);
    bad |= st[G + h] < 0.0f;
  }
  if (M == kNegInf || bad) return 0.0f;
  float L = 0.0f, A = 0.0f;
  for (int s = 0; s < nsplit; ++s) {
    const float* st = partials + (size_t)(slot0 + s * stride) * SF;
    const float c = ex2(st[h] - M);
    L = __builtin_fmaf(c, st[G + h], L);
    A = __builtin_fmaf(c, st[2 * G + h * D + dcol], A);
  }
  return A / L;
}

// ---------------------------------------------------------------------------------
// One task: KV head g of `row`, tokens [t0, t1), partial state into `slot`.
template <int G, int W>
__device__ __forceinline__ void run_task(const DecodeArgs& a, int row, int g, int t0, int t1, int slot,
                                         float* lds) {
  constexpr int SF = 2 * G + G * D;
  float* lds_m = lds;                // [W][G]
  float* lds_l = lds + W * G;        // [W][G]
  float* lds_acc = lds + 2 * W * G;  // [W][G][D]
  int* lds_bad = reinterpret_cast<int*>(lds + 2 * W * G + W * G * D);

  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const int r = lane >> 4;
  const int c = lane & 15;
  const int Hkv = a.Hkv;
  const size_t tok_stride = (size_t)Hkv * D;       // halves between consecutive tokens
  const size_t page_stride = (size_t)P * tok_stride;

  uint4 q[G];
  {
    const uint4* qp = reinterpret_cast<const uint4*>(a.q + ((size_t)row * a.Hq + (size_t)g * G) * D) + c;
#pragma unroll
    for (int h = 0; h < G; ++h) q[h] = qp[h * (D / 8)];
  }
  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = kNegInf;
    l[h] = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[h][k] = 0.0f;
  }

  const int pg_begin = t0 / P;
  const int pg_end = (t1 + P - 1) / P;
  const int* bt = a.block_table + (size_t)row * a.max_pages_per_row;
  const size_t lane_off = (size_t)r * tok_stride + (size_t)g * D + (size_t)c * 8;
  const uint16_t* kbase = a.k + lane_off;
  const uint16_t* vbase = a.v + lane_off;
  const int first = pg_begin + wave;                       // this wave's pages: first + k*W
  const int npw = first < pg_end ? (pg_end - first + W - 1) / W : 0;
  bool bad = false;

  // Page ids of this wave's next 64 pages, one per lane, fetched with one load.
  int ids = 0;
  auto fetch_ids = [&](int k0) {
    const int k = k0 + lane;
    ids = k < npw ? bt[first + k * W] : 0;
  };
  auto issue = [&](uint4 (&kr)[4], uint4 (&vr)[4], int k) {
    if ((k & 63) == 0) fetch_ids(k);
    int phys = __builtin_amdgcn_readlane(ids, k & 63);
    if (phys < 0 || phys >= a.num_pages) {
      bad = true;
      phys = 0;
    }
    const uint16_t* kb = kbase + (size_t)phys * page_stride;
    const uint16_t* vb = vbase + (size_t)phys * page_stride;
#pragma unroll
    for (int i = 0; i < 4; ++i) kr[i] = *reinterpret_cast<const uint4*>(kb + (size_t)i * 4 * tok_stride);
#pragma unroll
    for (int i = 0; i < 4; ++i) vr[i] = *reinterpret_cast<const uint4*>(vb + (size_t)i * 4 * tok_stride);
  };
  auto consume = [&](uint4 (&kr)[4], uint4 (&vr)[4], int k) {
    const int pg = first + k * W;
    float x[G][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int h = 0; h < G; ++h) x[h][i] = row_sum16(dot8(q[h], kr[i])) * a.scale_log2;
    }
    if (pg * P + P > t1) {  // the row's last, partial page: mask tokens >= t1
      const int tok = pg * P + r;  // this lane row's token in load i is tok + 4i
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool valid = tok + 4 * i < t1;
#pragma unroll
        for (int h = 0; h < G; ++h) x[h][i] = valid ? x[h][i] : kNegInf;
        if (!valid) vr[i] = make_uint4(0, 0, 0, 0);
      }
    }
    float mt[G];
    bool grow = false;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      mt[h] = fmaxf(fmaxf(x[h][0], x[h][1]), fmaxf(x[h][2], x[h][3]));
      grow |= mt[h] > m[h];
    }
    if (__builtin_amdgcn_ballot_w64(grow)) {  // rescale only when some running max grows
#pragma unroll
      for (int h = 0; h < G; ++h) {
        if (mt[h] > m[h]) {
          const float alpha = ex2(m[h] - mt[h]);
          l[h] *= alpha;
#pragma unroll
          for (int kk = 0; kk < 8; ++kk) acc[h][kk] *= alpha;
          m[h] = mt[h];
        }
      }
    }
    float vf[4][8];
#pragma unroll
    for (int i = 0; i < 4; ++i) unpack8(vr[i], vf[i]);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mref = (m[h] == kNegInf) ? 0.0f : m[h];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float p = ex2(x[h][i] - mref);
        l[h] += p;
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) acc[h][kk] = __builtin_fmaf(p, vf[i][kk], acc[h][kk]);
      }
    }
  };

  // Two register buffers in ping-pong: the next page's loads are in flight while the
  // current page is scored and accumulated.
  uint4 ka[4], va[4], kb2[4], vb2[4];
  if (npw > 0) issue(ka, va, 0);
  for (int k = 0; k < npw; k += 2) {
    if (k + 1 < npw) issue(kb2, vb2, k + 1);
    consume(ka, va, k);
    if (k + 1 < npw) {
      if (k + 2 < npw) issue(ka, va, k + 2);
      consume(kb2, vb2, k + 1);
    }
  }

  // Combine the wave's four lane rows (butterfly over lane xor 16, then xor 32); the
  // lanes of row 0 then hold the wave's state, which goes to LDS for a fixed-order
  // combine of the W wave states into the task's partial state.
#pragma unroll
  for (int sh = 16; sh <= 32; sh <<= 1) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mo = __shfl_xor(m[h], sh);
      const float lo = __shfl_xor(l[h], sh);
      const float M = fmaxf(m[h], mo);
      const float Mref = (M == kNegInf) ? 0.0f : M;
      const float ca = ex2(m[h] - Mref);
      const float cb = ex2(mo - Mref);
      l[h] = __builtin_fmaf(cb, lo, ca * l[h]);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float ao = __shfl_xor(acc[h][k], sh);
        acc[h][k] = __builtin_fmaf(cb, ao, ca * acc[h][k]);
      }
      m[h] = M;
    }
  }
  if (lane < 16) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      float4* dst = reinterpret_cast<float4*>(lds_acc + ((size_t)wave * G + h) * D + c * 8);
      dst[0] = make_float4(acc[h][0], acc[h][1], acc[h][2], acc[h][3]);
      dst[1] = make_float4(acc[h][4], acc[h][5], acc[h][6], acc[h][7]);
    }
  }
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      lds_m[wave * G + h] = m[h];
      lds_l[wave * G + h] = l[h];
    }
    lds_bad[wave] = bad ? 1 : 0;
  }
  __syncthreads();

  bool any_bad = false;
#pragma unroll
  for (int w = 0; w < W; ++w) any_bad |= lds_bad[w] != 0;
  if (any_bad && threadIdx.x == 0) atomicOr(a.err, (unsigned)PKV_DEVERR_PAGE_ID);

  float* st = a.partials + (size_t)slot * SF;
  for (int e = threadIdx.x; e < G * D; e += W * 64) {
    const int h = e / D;
    const int dcol = e % D;
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < W; ++w) M = fmaxf(M, lds_m[w * G + h]);
    const float Mref = (M == kNegInf) ? 0.0f : M;
    float L = 0.0f, A = 0.0f;
#pragma unroll
    for (int w = 0; w < W; ++w) {
      const float cf = ex2(lds_m[w * G + h] - Mref);
      L = __builtin_fmaf(cf, lds_l[w * G + h], L);
      A = __builtin_fmaf(cf, lds_acc[((size_t)w * G + h) * D + dcol], A);
    }
    st[2 * G + h * D + dcol] = A;
    if (dcol == 0) {
      st[h] = M;
      st[G + h] = any_bad ? -1.0f : L;
    }
  }
}

template <int G>
__device__ __forceinline__ void write_neutral(const DecodeArgs& a, int slot) {
  constexpr int SF = 2 * G + G * D;
  float* st = a.partials + (size_t)slot * SF;
  for (int e = threadIdx.x; e < SF; e += blockDim.x) st[e] = (e < G) ? kNegInf : 0.0f;
}

template <int G>
__device__ __forceinline__ void zero_row(const DecodeArgs& a, int row) {
  uint32_t* o = reinterpret_cast<uint32_t*>(a.out + (size_t)row * a.Hq * D);
  for (int e = threadIdx.x; e < a.Hq * D / 2; e += blockDim.x) o[e] = 0u;
}

template <int G, int W>
constexpr int lds_floats() {
  return 2 * W * G + W * G * D + W;
}

// Workqueue split kernel. FUSED: the last split of each (row, KV head) to finish merges
// all of that pair's splits in split order (Sec. 3.4, atomic completion counter).
template <int G, int W, bool FUSED>
__global__ __launch_bounds__(W * 64) void split_kernel(DecodeArgs a) {
  __shared__ float lds[lds_floats<G, W>()];
  __shared__ int lds_last;
  if (FUSED) {
    for (int i = blockIdx.x; i < a.B; i += gridDim.x)
      if (a.split_offsets[i + 1] == a.split_offsets[i]) zero_row<G>(a, i);
  }
  int ntasks = uniform(*a.num_tasks);
  if (ntasks > a.max_tasks) ntasks = a.max_tasks;
  for (int t = blockIdx.x; t < ntasks; t += gridDim.x) {
    const pkv_task task = a.tasks[t];
    const int row = uniform(task.row), g = uniform(task.kvh);
    const int t0 = uniform(task.t_begin), t1 = uniform(task.t_end);
    if (row < 0 || row >= a.B || g < 0 || g >= a.Hkv || t0 < 0 || t1 <= t0 ||
        t1 > a.max_pages_per_row * P) {  // not a task of a valid plan: flag and skip
      if (threadIdx.x == 0) atomicOr(a.err, (unsigned)PKV_DEVERR_TASK);
      continue;
    }
    run_task<G, W>(a, row, g, t0, t1, t, lds);
    if (FUSED) {
      const int off = uniform(a.split_offsets[row]);
      int nsplit = uniform(a.split_offsets[row + 1]) - off;
      if (off < 0 || nsplit < 1 || (long long)(off + nsplit) * a.Hkv > a.max_tasks) {
        if (threadIdx.x == 0) atomicOr(a.err, (unsigned)PKV_DEVERR_TASK);
        nsplit = 0;  // never reached by the counter: no merge from inconsistent offsets
      }
      __threadfence();
      __syncthreads();
      if (threadIdx.x == 0) {
        const int prev = atomicAdd(&a.counters[row * a.Hkv + g], 1);
        lds_last = (prev == nsplit - 1);
      }
      __syncthreads();
      if (lds_last) {
        __threadfence();
        uint16_t* o = a.out + ((size_t)row * a.Hq + (size_t)g * G) * D;
        for (int e = threadIdx.x; e < G * D; e += W * 64)
          o[e] = f32_to_f16_bits(merge_elem<G>(a.partials, off * a.Hkv + g, a.Hkv, nsplit, e / D, e % D));
        if (threadIdx.x == 0) a.counters[row * a.Hkv + g] = 0;
      }
    }
    __syncthreads();
  }
}

// Rectangular grid: workgroup (i, s, g) in slot order (i*S + s)*Hkv + g.
template <int G, int W>
__global__ __launch_bounds__(W * 64) void rect_kernel(DecodeArgs a) {
  __shared__ float lds[lds_floats<G, W>()];
  const int slot = blockIdx.x;
  const int g = slot % a.Hkv;
  const int s = (slot / a.Hkv) % a.S;
  const int row = slot / (a.Hkv * a.S);
  int n = uniform(a.seq_lens[row]);
  if (n < 0 || n > a.max_pages_per_row * P) {
    if (threadIdx.x == 0 && s == 0 && g == 0) atomicOr(a.err, (unsigned)PKV_DEVERR_SEQ_LEN);
    n = 0;
  }
  const int T = a.tile_tokens;
  const int tiles = (n + T - 1) / T;
  const int ns = tiles < a.S ? tiles : a.S;
  if (s >= ns) {  // empty split: neutral state, no Q or KV traffic (Sec. 3.3)
    write_neutral<G>(a, slot);
    return;
  }
  const int b0 = (int)(((long long)s * tiles) / ns);
  const int b1 = (int)(((long long)(s + 1) * tiles) / ns);
  const int t0 = b0 * T;
  const int t1 = min(b1 * T, n);
  run_task<G, W>(a, row, g, t0, t1, slot, lds);
}

// Segmented merge: one workgroup of D threads per (row, query head).
// RECT: slots (row*S + s)*Hkv + g for s < S; else the planner's split_offsets.
template <int G, bool RECT>
__global__ __launch_bounds__(D) void merge_kernel(DecodeArgs a) {
  const int row = blockIdx.x / a.Hq;
  const int hq = blockIdx.x % a.Hq;
  const int g = hq / G;
  const int h = hq % G;
  int slot0, nsplit;
  if (RECT) {
    slot0 = row * a.S * a.Hkv + g;
    nsplit = a.S;
  } else {
    const int off = a.split_offsets[row];
    slot0 = off * a.Hkv + g;
    nsplit = a.split_offsets[row + 1] - off;
    if (off < 0 || nsplit < 0 || (long long)(off + nsplit) * a.Hkv > a.max_tasks) {
      // offsets that do not belong to a plan of this capacity: never read past the slots
      if (threadIdx.x == 0 && h == 0) atomicOr(a.err, (unsigned)PKV_DEVERR_TASK);
      nsplit = 0;
    }
  }
  const float o = merge_elem<G>(a.partials, uniform(slot0), a.Hkv, uniform(nsplit), h, threadIdx.x);
  a.out[((size_t)row * a.Hq + hq) * D + threadIdx.x] = f32_to_f16_bits(o);
}

// ---------------------------------------------------------------------------------
// Planner (Sec. 3.4): one workgroup. Lengths are validated, S follows the active batch
// size, nsplit_i = min(S, ceil(N_i / T)), split_offsets is their exclusive scan, and
// task k = (split_offsets[i] + s) * Hkv + g covers the balanced tile range
// [floor(s*tiles/nsplit), floor((s+1)*tiles/nsplit)) of row i.
constexpr int kPlanThreads = 1024;

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(PlanArgs a) {
  __shared__ int s_len[kMaxPlanBatch];
  __shared__ int s_off[kMaxPlanBatch + 1];
  __shared__ int s_scan[kPlanThreads];
  __shared__ int s_active;
  const int tid = threadIdx.x;
  const int B = a.B;
  const int cap = a.max_pages_per_row * a.page_size;
  if (tid == 0) s_active = 0;
  for (int i = tid; i < B; i += kPlanThreads) {
    int n = a.seq_lens[i];
    if (n < 0 || n > cap) {
      atomicOr(a.err, (unsigned)PKV_DEVERR_SEQ_LEN);
      n = 0;
    }
    s_len[i] = n;
  }
  __syncthreads();
  if (a.block_table) {
    const long long total = (long long)B * a.max_pages_per_row;
    for (long long k = tid; k < total; k += kPlanThreads) {
      const int i = (int)(k / a.max_pages_per_row);
      const int jp = (int)(k % a.max_pages_per_row);
      const int n = s_len[i];
      if (jp < (n + a.page_size - 1) / a.page_size) {
        const int phys = a.block_table[k];
        if (phys < 0 || phys >= a.num_pages) {
          atomicOr(a.err, (unsigned)PKV_DEVERR_PAGE_ID);
          s_len[i] = 0;  // benign race: every writer stores 0
        }
      }
    }
    __syncthreads();
  }
  int act = 0;
  for (int i = tid; i < B; i += kPlanThreads) act += s_len[i] > 0;
  if (act) atomicAdd(&s_active, act);
  __syncthreads();
  const int T = a.tile_tokens;
  const long long denom = (long long)(s_active > 0 ? s_active : 1) * a.Hkv;
  long long Sll = (a.target_tasks + denom - 1) / denom;
  if (Sll < a.split_min) Sll = a.split_min;
  if (Sll > a.split_max) Sll = a.split_max;
  const int S = (int)Sll;

  // exclusive scan of nsplit over rows: thread tid owns rows [tid*per, (tid+1)*per)
  const int per = (B + kPlanThreads - 1) / kPlanThreads;
  const int r0 = tid * per;
  int local = 0;
  for (int i = r0; i < r0 + per && i < B; ++i) {
    const int tiles = (s_len[i] + T - 1) / T;
    local += tiles < S ? tiles : S;
  }
  s_scan[tid] = local;
  __syncthreads();
  for (int off = 1; off < kPlanThreads; off <<= 1) {
    const int v = tid >= off ? s_scan[tid - off] : 0;
    __syncthreads();
    s_scan[tid] += v;
    __syncthreads();
  }
  int run = s_scan[tid] - local;  // exclusive prefix
  for (int i = r0; i < r0 + per && i < B; ++i) {
    s_off[i] = run;
    const int tiles = (s_len[i] + T - 1) / T;
    run += tiles < S ? tiles : S;
  }
  if (tid == kPlanThreads - 1) s_off[B] = s_scan[kPlanThreads - 1];
  __syncthreads();
  for (int i = tid; i <= B; i += kPlanThreads) a.split_offsets[i] = s_off[i];
  long long ntasks = (long long)s_off[B] * a.Hkv;
  if (ntasks > a.max_tasks) {  // excluded by host validation; never write past the buffer
    if (tid == 0) atomicOr(a.err, (unsigned)PKV_DEVERR_SEQ_LEN);
    ntasks = 0;
  }
  if (tid == 0) *a.num_tasks = (int)ntasks;
  for (int k = tid; k < (int)ntasks; k += kPlanThreads) {
    const int sr = k / a.Hkv;
    const int g = k % a.Hkv;
    int lo = 0, hi = B;  // largest i with s_off[i] <= sr
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (s_off[mid] <= sr) lo = mid; else hi = mid;
    }
    const int i = lo;
    const int s = sr - s_off[i];
    const int n = s_len[i];
    const int tiles = (n + T - 1) / T;
    const int ns = s_off[i + 1] - s_off[i];
    const int b0 = (int)(((long long)s * tiles) / ns);
    const int b1 = (int)(((long long)(s + 1) * tiles) / ns);
    pkv_task* t = a.tasks + k;
    t->row = i;
    t->kvh = g;
    t->split = s;
    t->t_begin = b0 * T;
    t->t_end = min(b1 * T, n);
  }
  for (int k = tid; k < B * a.Hkv; k += kPlanThreads) a.counters[k] = 0;
}

__global__ void zero_kernel(uint32_t* p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = 0u;
}

__global__ __launch_bounds__(256) void copy_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

template <int G, int W>
hipError_t launch_decode_g(const DecodeArgs& a, int mode, int grid, hipStream_t s) {
  if (mode == 2) {
    hipLaunchKernelGGL((rect_kernel<G, W>), dim3(a.B * a.Hkv * a.S), dim3(W * 64), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((merge_kernel<G, true>), dim3(a.B * a.Hq), dim3(D), 0, s, a);
    return hipGetLastError();
  }
  if (mode == 1) {
    hipLaunchKernelGGL((split_kernel<G, W, true>), dim3(grid), dim3(W * 64), 0, s, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((split_kernel<G, W, false>), dim3(grid), dim3(W * 64), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((merge_kernel<G, false>), dim3(a.B * a.Hq), dim3(D), 0, s, a);
  return hipGetLastError();
}

}  // namespace

constexpr int kWaves = 4;

hipError_t launch_decode(const DecodeArgs& a, int G, int mode, int grid, hipStream_t s) {
  switch (G) {
    case 1: return launch_decode_g<1, kWaves>(a, mode, grid, s);
    case 2: return launch_decode_g<2, kWaves>(a, mode, grid, s);
    case 4: return launch_decode_g<4, kWaves>(a, mode, grid, s);
    case 8: return launch_decode_g<8, kWaves>(a, mode, grid, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_plan(const PlanArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t s) {
  const size_t n = bytes / 4;
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, (uint32_t*)p, n);
  return hipGetLastError();
}

hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t s) {
  const size_t n = bytes / 16;
  if (n == 0) return hipSuccess;
  size_t blocks = (n + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  hipLaunchKernelGGL(copy_kernel, dim3((unsigned)blocks), dim3(256), 0, s, (const uint4*)src, (uint4*)dst, n);
  return hipGetLastError();
}

}  // namespace pkv
