// Training-side gather-scatter (Section 3.2, Eq. 6-7) and the router's
// straight-through estimator (Appendix B): the C entry points declared in
// include/tlf.h and their kernels.
//
// The operations are pure data movement plus one add per element, so every
// kernel is bound by HBM bandwidth: rows move as 16-byte vectors, each thread
// keeps four of them in flight, and only the active-set planner (integer work
// over one depth per row) runs as a single workgroup.
#include <hip/hip_runtime.h>
#include <stdint.h>

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
