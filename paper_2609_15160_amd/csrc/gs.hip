// Training-side gather-scatter (Section 3.2, Eq. 6-7) and the router's
// straight-through estimator (Appendix B): the C entry points declared in
// include/tlf.h and their kernels.
//
// The operations are pure data movement plus one add per element, so every
// kernel is bound by HBM bandwidth: rows move as 16-byte vectors, each thread
// keeps four of them in flight.  The active-set planner (integer work over one
// depth per row) runs as a single workgroup, or, with scratch for one count
// per chunk of rows, as one workgroup per chunk in two launches.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"
#include "tlf.h"

namespace {

constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / 64;
constexpr int kPlanPer = 16;  // rows per thread per pass
constexpr int kCopyThreads = 256;
constexpr int kCopyUnroll = 4;  // float4 per thread

struct PlanArgs {
  const int32_t* depth;
  int32_t rows, seq_len, batch, loop;
  int32_t* index;
  int32_t* slot;
  int32_t* offsets;
  int32_t* count;
};

// One workgroup walks the rows in passes of kPlanThreads x kPlanPer.  Within a
// pass, row base + k * kPlanThreads + tid belongs to thread tid (coalesced
// loads); the compact position of an active row is the number of active rows
// before it: the running total of earlier passes, the active rows of earlier
// (k, wave) groups of this pass, and the active lanes below it in its wave.
__global__ __launch_bounds__(kPlanThreads) void k_gs_plan(PlanArgs a) {
  __shared__ int s_cnt[kPlanPer * kPlanWaves];
  __shared__ int s_total;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  if (a.rows == 0) {
    for (int b = tid; b <= a.batch; b += kPlanThreads)
      if (a.offsets) a.offsets[b] = 0;
    if (tid == 0) a.count[0] = 0;
    return;
  }
  int total = 0;
  for (int base = 0; base < a.rows; base += kPlanThreads * kPlanPer) {
    int m[kPlanPer];
#pragma unroll
    for (int k = 0; k < kPlanPer; ++k) {
      const int r = base + k * kPlanThreads + tid;
      m[k] = a.depth[r < a.rows ? r : a.rows - 1];
    }
    uint64_t bal[kPlanPer];
#pragma unroll
    for (int k = 0; k < kPlanPer; ++k) {
      const int r = base + k * kPlanThreads + tid;
      bal[k] = __ballot(r < a.rows && m[k] >= a.loop);
      if (lane == 0) s_cnt[k * kPlanWaves + wave] = __popcll(bal[k]);
    }
    __syncthreads();
    // exclusive scan of the kPlanPer x kPlanWaves group counts by wave 0
    if (wave == 0) {
      constexpr int G = kPlanPer * kPlanWaves / 64;
      int v[G], s = 0;
#pragma unroll
      for (int g = 0; g < G; ++g) { v[g] = s_cnt[lane * G + g]; s += v[g]; }
      int incl = s;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(incl, o);
        if (lane >= o) incl += t;
      }
      int run = incl - s;
#pragma unroll
      for (int g = 0; g < G; ++g) { s_cnt[lane * G + g] = run; run += v[g]; }
      if (lane == 63) s_total = incl;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kPlanPer; ++k) {
      const int r = base + k * kPlanThreads + tid;
      if (r < a.rows) {
        const bool act = m[k] >= a.loop;
        const int pos = total + s_cnt[k * kPlanWaves + wave] + __popcll(bal[k] & below);
        if (act) a.index[pos] = r;
        if (a.slot) a.slot[r] = act ? pos : -1;
        if (a.offsets && r % a.seq_len == 0) a.offsets[r / a.seq_len] = pos;
      }
    }
    total += s_total;
    __syncthreads();  // s_cnt and s_total are rewritten by the next pass
  }
  if (tid == 0) {
    a.count[0] = total;
    if (a.offsets) a.offsets[a.batch] = total;
  }
}

// Multi-workgroup form of the same plan, in two launches that communicate
// through a caller-provided array of per-chunk counts (no workgroup waits
// for another).  Chunk c holds rows [c * kChunkRows, (c + 1) * kChunkRows);
// thread tid of its workgroup takes rows base + k * kChunkThreads + tid.
constexpr int kChunkThreads = 256;
constexpr int kChunkWaves = kChunkThreads / 64;
constexpr int kChunkPer = 8;  // rows per thread
constexpr int kChunkRows = kChunkThreads * kChunkPer;
static_assert(kChunkRows == TLF_GS_PLAN_CHUNK_ROWS, "chunk size in tlf.h");

// Pass 1: counts[c] = active rows of chunk c.
__global__ __launch_bounds__(kChunkThreads) void k_gs_count(const int32_t* __restrict__ depth, int32_t rows,
                                                            int32_t loop, int32_t* __restrict__ counts) {
  __shared__ int s_w[kChunkWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int base = blockIdx.x * kChunkRows;
  int m[kChunkPer];
#pragma unroll
  for (int k = 0; k < kChunkPer; ++k) {
    const int r = base + k * kChunkThreads + tid;
    m[k] = depth[r < rows ? r : rows - 1];
  }
  int n = 0;
#pragma unroll
  for (int k = 0; k < kChunkPer; ++k) {
    const int r = base + k * kChunkThreads + tid;
    n += __popcll(__ballot(r < rows && m[k] >= loop));
  }
  if (lane == 0) s_w[wave] = n;
  __syncthreads();
  if (tid == 0) {
    int t = 0;
#pragma unroll
    for (int w = 0; w < kChunkWaves; ++w) t += s_w[w];
    counts[blockIdx.x] = t;
  }
}

// Pass 2: each chunk starts at the sum of the counts before it and places
// its rows as the single-workgroup planner does; the last chunk writes the
// total.  With no rows, one workgroup writes the empty plan.
__global__ __launch_bounds__(kChunkThreads) void k_gs_place(PlanArgs a, const int32_t* __restrict__ counts,
                                                            int32_t nchunks) {
  __shared__ int s_cnt[kChunkPer * kChunkWaves];
  __shared__ int s_pre[kChunkWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (nchunks == 0) {
    for (int b = tid; b <= a.batch; b += kChunkThreads)
      if (a.offsets) a.offsets[b] = 0;
    if (tid == 0) a.count[0] = 0;
    return;
  }
  const int c = blockIdx.x, base = c * kChunkRows;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int m[kChunkPer];
#pragma unroll
  for (int k = 0; k < kChunkPer; ++k) {
    const int r = base + k * kChunkThreads + tid;
    m[k] = a.depth[r < a.rows ? r : a.rows - 1];
  }
  // rows placed by the chunks before this one
  int pre = 0;
  for (int q = tid; q < c; q += kChunkThreads) pre += counts[q];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) pre += __shfl_xor(pre, o);
  if (lane == 0) s_pre[wave] = pre;
  uint64_t bal[kChunkPer];
#pragma unroll
  for (int k = 0; k < kChunkPer; ++k) {
    const int r = base + k * kChunkThreads + tid;
    bal[k] = __ballot(r < a.rows && m[k] >= a.loop);
    if (lane == 0) s_cnt[k * kChunkWaves + wave] = __popcll(bal[k]);
  }
  __syncthreads();
  // exclusive scan of the kChunkPer x kChunkWaves group counts (32 values) by wave 0
  if (wave == 0) {
    constexpr int G = kChunkPer * kChunkWaves;
    const int v = lane < G ? s_cnt[lane] : 0;
    int incl = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(incl, o);
      if (lane >= o) incl += t;
    }
    if (lane < G) s_cnt[lane] = incl - v;
    if (lane == G - 1 && c == nchunks - 1) {
      int total = incl;
#pragma unroll
      for (int w = 0; w < kChunkWaves; ++w) total += s_pre[w];
      a.count[0] = total;
      if (a.offsets) a.offsets[a.batch] = total;
    }
  }
  __syncthreads();
  int start = 0;
#pragma unroll
  for (int w = 0; w < kChunkWaves; ++w) start += s_pre[w];
#pragma unroll
  for (int k = 0; k < kChunkPer; ++k) {
    const int r = base + k * kChunkThreads + tid;
    if (r < a.rows) {
      const bool act = m[k] >= a.loop;
      const int pos = start + s_cnt[k * kChunkWaves + wave] + __popcll(bal[k] & below);
      if (act) a.index[pos] = r;
      if (a.slot) a.slot[r] = act ? pos : -1;
      if (a.offsets && r % a.seq_len == 0) a.offsets[r / a.seq_len] = pos;
    }
  }
}

// out[r] = h[index[r]] for r < min(count, max_rows); d4 float4 per row.
// Loads are clamped into range rather than guarded, so that all of a thread's
// index loads, then all of its row loads, are in flight together.
__global__ __launch_bounds__(kCopyThreads) void k_gs_gather(const float4* __restrict__ h,
                                                            const int32_t* __restrict__ index,
                                                            const int32_t* __restrict__ count,
                                                            int32_t max_rows, int32_t d4,
                                                            float4* __restrict__ out) {
  const int n = min(count[0], max_rows);
  const int64_t limit = (int64_t)n * d4;
  const int64_t e0 = (int64_t)blockIdx.x * (kCopyThreads * kCopyUnroll) + threadIdx.x;
  if (e0 >= limit) return;
  int src[kCopyUnroll], col[kCopyUnroll];
#pragma unroll
  for (int u = 0; u < kCopyUnroll; ++u) {
    const int64_t e = min(e0 + u * kCopyThreads, limit - 1);
    const int r = (int)(e / d4);
    col[u] = (int)(e - (int64_t)r * d4);
    src[u] = index[r];
  }
  float4 v[kCopyUnroll];
#pragma unroll
  for (int u = 0; u < kCopyUnroll; ++u) v[u] = h[(int64_t)src[u] * d4 + col[u]];
#pragma unroll
  for (int u = 0; u < kCopyUnroll; ++u)
    if (e0 + u * kCopyThreads < limit) out[e0 + u * kCopyThreads] = v[u];
}

// out[r] = prev[r] + y[slot[r]] where slot[r] >= 0, else prev[r] (not read
// or rewritten when out is prev, so an in-place scatter moves only the
// active rows).
template <bool kInPlace>
__global__ __launch_bounds__(kCopyThreads) void k_gs_scatter(const float4* prev, const float4* __restrict__ y,
                                                             const int32_t* __restrict__ slot, int32_t rows,
                                                             int32_t d4, float4* out) {
  const int64_t limit = (int64_t)rows * d4;
  const int64_t e0 = (int64_t)blockIdx.x * (kCopyThreads * kCopyUnroll) + threadIdx.x;
  if (e0 >= limit) return;
  int s[kCopyUnroll], col[kCopyUnroll];
#pragma unroll
  for (int u = 0; u < kCopyUnroll; ++u) {
    const int64_t e = min(e0 + u * kCopyThreads, limit - 1);
    const int r = (int)(e / d4);
    col[u] = (int)(e - (int64_t)r * d4);
    s[u] = slot[r];
  }
  float4 p[kCopyUnroll], q[kCopyUnroll];
#pragma unroll
  for (int u = 0; u < kCopyUnroll; ++u) {
    const int64_t e = min(e0 + u * kCopyThreads, limit - 1);
    if (s[u] >= 0) {
      p[u] = prev[e];
      q[u] = y[(int64_t)s[u] * d4 + col[u]];
    } else if (!kInPlace) {
      p[u] = prev[e];
    }
  }
#pragma unroll
  for (int u = 0; u < kCopyUnroll; ++u) {
    const int64_t e = e0 + u * kCopyThreads;
    if (e < limit && (!kInPlace || s[u] >= 0)) {
      out[e] = s[u] >= 0 ? make_float4(q[u].x + p[u].x, q[u].y + p[u].y, q[u].z + p[u].z, q[u].w + p[u].w)
                         : p[u];
    }
  }
}

__global__ __launch_bounds__(kCopyThreads) void k_ste(const int32_t* __restrict__ depth,
                                                      const float* __restrict__ score,
                                                      const float* __restrict__ grad_value, int32_t n,
                                                      float* __restrict__ value, float* __restrict__ grad_score) {
  const int i = blockIdx.x * kCopyThreads + threadIdx.x;
  if (i >= n) return;
  if (value) value[i] = (float)depth[i];
  if (grad_score) {
    // sigma(s) (1 - sigma(s)) = t / (1 + t)^2 with t = exp(-|s|): no
    // cancellation in 1 - sigma for large |s|
    const float t = expf(-fabsf(score[i]));
    const float u = 1.0f + t;
    grad_score[i] = grad_value[i] * (t / (u * u));
  }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int launch_status() { return hipGetLastError() == hipSuccess ? TLF_OK : TLF_E_HIP; }

int copy_blocks(int64_t elems4) {
  const int64_t per = (int64_t)kCopyThreads * kCopyUnroll;
  return (int)((elems4 + per - 1) / per);
}

}  // namespace

namespace tlf {

int gs_plan_chunked_args(const int32_t* d_depth, int32_t batch, int32_t seq_len, int32_t* d_index,
                         const int32_t* d_count, int64_t max_rows, int64_t* rows_out) {
  if (batch < 0 || seq_len < 0 || !d_count) return TLF_E_INVALID_ARG;
  const int64_t rows = (int64_t)batch * seq_len;
  if (rows > max_rows) return TLF_E_INVALID_ARG;
  if (rows > 0 && (!d_depth || !d_index)) return TLF_E_INVALID_ARG;
  *rows_out = rows;
  return TLF_OK;
}

int launch_gs_plan_chunked(const int32_t* d_depth, int32_t batch, int32_t seq_len, int32_t loop, int32_t* d_index,
                           int32_t* d_slot, int32_t* d_offsets, int32_t* d_count, int32_t* counts, int64_t rows,
                           hipStream_t stream) {
  const int nchunks = (int)((rows + kChunkRows - 1) / kChunkRows);
  PlanArgs a{d_depth, (int32_t)rows, seq_len, batch, loop, d_index, d_slot, d_offsets, d_count};
  if (nchunks > 0)
    hipLaunchKernelGGL(k_gs_count, dim3(nchunks), dim3(kChunkThreads), 0, stream, d_depth, (int32_t)rows, loop,
                       counts);
  hipLaunchKernelGGL(k_gs_place, dim3(nchunks > 0 ? nchunks : 1), dim3(kChunkThreads), 0, stream, a,
                     (const int32_t*)counts, nchunks);
  return launch_status();
}

}  // namespace tlf

extern "C" {

int tlf_gs_plan(const int32_t* d_depth, int32_t batch, int32_t seq_len, int32_t loop, int32_t* d_index,
                int32_t* d_slot, int32_t* d_offsets, int32_t* d_count, void* stream) {
  if (batch < 0 || seq_len < 0 || !d_count) return TLF_E_INVALID_ARG;
  const int64_t rows = (int64_t)batch * seq_len;
  if (rows > INT32_MAX - kPlanThreads * kPlanPer) return TLF_E_INVALID_ARG;
  if (rows > 0 && (!d_depth || !d_index)) return TLF_E_INVALID_ARG;
  PlanArgs a{d_depth, (int32_t)rows, seq_len, batch, loop, d_index, d_slot, d_offsets, d_count};
  hipLaunchKernelGGL(k_gs_plan, dim3(1), dim3(kPlanThreads), 0, (hipStream_t)stream, a);
  return launch_status();
}

int tlf_gs_plan_ws(const int32_t* d_depth, int32_t batch, int32_t seq_len, int32_t loop, int32_t* d_index,
                   int32_t* d_slot, int32_t* d_offsets, int32_t* d_count, void* d_workspace, size_t ws_bytes,
                   void* stream) {
  int64_t rows = 0;
  const int st = tlf::gs_plan_chunked_args(d_depth, batch, seq_len, d_index, d_count, TLF_GS_PLAN_MAX_ROWS, &rows);
  if (st != TLF_OK) return st;
  const size_t need = tlf_gs_plan_ws_bytes(rows);
  if (need > 0 && (!d_workspace || ws_bytes < need || ((uintptr_t)d_workspace & 3u) != 0))
    return TLF_E_INVALID_ARG;
  return tlf::launch_gs_plan_chunked(d_depth, batch, seq_len, loop, d_index, d_slot, d_offsets, d_count,
                                     (int32_t*)d_workspace, rows, (hipStream_t)stream);
}

int tlf_gs_gather(const float* d_h, const int32_t* d_index, const int32_t* d_count, int32_t max_rows,
                  int32_t d, float* d_out, void* stream) {
  if (max_rows < 0 || d <= 0 || d % 4 != 0 || !d_count) return TLF_E_INVALID_ARG;
  if (max_rows == 0) return TLF_OK;
  if (!d_h || !d_index || !d_out || !aligned16(d_h) || !aligned16(d_out)) return TLF_E_INVALID_ARG;
  const int64_t e4 = (int64_t)max_rows * (d / 4);
  if (copy_blocks(e4) > INT32_MAX / 2) return TLF_E_INVALID_ARG;
  hipLaunchKernelGGL(k_gs_gather, dim3(copy_blocks(e4)), dim3(kCopyThreads), 0, (hipStream_t)stream,
                     (const float4*)d_h, d_index, d_count, max_rows, d / 4, (float4*)d_out);
  return launch_status();
}

int tlf_gs_scatter(const float* d_h_prev, const float* d_y, const int32_t* d_slot, int32_t rows, int32_t d,
                   float* d_h_out, void* stream) {
  if (rows < 0 || d <= 0 || d % 4 != 0) return TLF_E_INVALID_ARG;
  if (rows == 0) return TLF_OK;
  if (!d_h_prev || !d_y || !d_slot || !d_h_out) return TLF_E_INVALID_ARG;
  if (!aligned16(d_h_prev) || !aligned16(d_y) || !aligned16(d_h_out)) return TLF_E_INVALID_ARG;
  const int64_t e4 = (int64_t)rows * (d / 4);
  if (copy_blocks(e4) > INT32_MAX / 2) return TLF_E_INVALID_ARG;
  if (d_h_out == d_h_prev)
    hipLaunchKernelGGL(k_gs_scatter<true>, dim3(copy_blocks(e4)), dim3(kCopyThreads), 0, (hipStream_t)stream,
                       (const float4*)d_h_prev, (const float4*)d_y, d_slot, rows, d / 4, (float4*)d_h_out);
  else
    hipLaunchKernelGGL(k_gs_scatter<false>, dim3(copy_blocks(e4)), dim3(kCopyThreads), 0, (hipStream_t)stream,
                       (const float4*)d_h_prev, (const float4*)d_y, d_slot, rows, d / 4, (float4*)d_h_out);
  return launch_status();
}

int tlf_ste(const int32_t* d_depth, const float* d_score, const float* d_grad_value, int32_t n, float* d_value,
            float* d_grad_score, void* stream) {
  if (n < 0) return TLF_E_INVALID_ARG;
  if (n == 0 || (!d_value && !d_grad_score)) return TLF_OK;
  if (d_value && !d_depth) return TLF_E_INVALID_ARG;
  if (d_grad_score && (!d_score || !d_grad_value)) return TLF_E_INVALID_ARG;
  hipLaunchKernelGGL(k_ste, dim3((n + kCopyThreads - 1) / kCopyThreads), dim3(kCopyThreads), 0,
                     (hipStream_t)stream, d_depth, d_score, d_grad_value, n, d_value, d_grad_score);
  return launch_status();
}

}  // extern "C"
