// The decode and prefill planners, and utility kernels.
#include "kernels.h"

namespace tlf {

namespace {

// ---------------------------------------------------------------------------
// Decode planner: one workgroup of NT threads (the batch rounded up to whole
// waves, at most kPlanThreads), thread t owning sequences t, t + NT, ...
// Steps:
//   1. depth-sorted order, deepest first and stable in b, by a counting sort
//      whose ranks come from wave ballots: A_i = rows [0, n_i) (Eq. 4-6);
//   2. one new page for every executed (b, i) whose next slot starts a page,
//      numbered by a block prefix sum (deterministic);
//   3. statistics;
//   4. per executed (b, i): the slot's position, cache_len += 1, and the
//      slot's element offset for the QKV epilogue, by compact row.
// All global reads are issued at the start and all slot stores come last,
// after the final barrier (a barrier waits for outstanding stores).
// Dense mode (gather-scatter off): rows stay in batch order and every loop up
// to the deepest token of the step has all B rows; the rows of exited tokens
// get kv_slot -1 (no cache entry) and their attention reads the cache as it
// stands, which the statistics count.
// ---------------------------------------------------------------------------
constexpr int kPlanWaves = kPlanThreads / kWave;

// Running totals of the step statistics: an atomic add returns nothing to
// wait for, where a read-modify-write would cost a memory round trip.
__device__ __forceinline__ void add_stat(long long* p, unsigned long long v) {
  atomicAdd(reinterpret_cast<unsigned long long*>(p), v);
}
constexpr int kPlanChunks = 4;  // kPlanThreads * kPlanChunks >= max batch (NT = kPlanThreads above kPlanThreads sequences)

__global__ __launch_bounds__(kPlanThreads) void k_plan_decode(DecodePlanArgs a) {
  const CacheView& c = a.c;
  const int tid = threadIdx.x, lane = lane_id(), wv = tid >> 6, B = a.B, R = c.R;
  const int NT = blockDim.x, NW = NT / kWave;  // threads (a multiple of the wave) and waves
  __shared__ int cnt[kMaxLoops + 1];
  __shared__ int start[kMaxLoops + 1];
  __shared__ int fill[kMaxLoops + 1];
  __shared__ int wcnt[kPlanWaves][kMaxLoops + 1];
  __shared__ int scan_tmp[kPlanWaves + 1];
  __shared__ unsigned long long s_kvread;
  __shared__ int s_top, s_base;
  __shared__ int s_nact[kMaxLoops];

  // the global reads of the first NT sequences (every batch up to
  // that size) are issued here: depth, sequence length, the R cache lengths
  // and the allocator in one round trip, then the page-table entry of each
  // cache's partly filled last page; sequences beyond (chunks >= 1) read
  // theirs where they are used
  int m_of[kPlanChunks], row_of[kPlanChunks];
#pragma unroll
  for (int ch = 0; ch < kPlanChunks; ++ch) {
    const int b = ch * NT + tid;
    m_of[ch] = b < B ? a.depth[b] : 0;
    row_of[ch] = -1;
  }
  int seq0, len0[kMaxLoops], page0[kMaxLoops];
  {
    const bool in = tid < B;
    seq0 = in ? c.seq_len[tid] : 0;
#pragma unroll
    for (int i = 0; i < kMaxLoops; ++i) len0[i] = in && i < R ? c.cache_len[tid * R + i] : 0;
  }
  const int base0 = tid == 0 ? *c.page_next : 0;
#pragma unroll
  for (int i = 0; i < kMaxLoops; ++i)
    page0[i] = (i < m_of[0] && len0[i] % kPage != 0)
                   ? c.page_table[((int64_t)tid * R + i) * c.pages_per_seq + len0[i] / kPage]
                   : -1;
  auto len_at = [&](int ch, int b, int i) __attribute__((always_inline)) {
    return ch == 0 ? len0[i] : c.cache_len[b * R + i];
  };
  if (tid <= kMaxLoops) { cnt[tid] = 0; fill[tid] = 0; }
  if (tid == 0) { s_kvread = 0ull; s_base = base0; }
  __syncthreads();
#pragma unroll
  for (int ch = 0; ch < kPlanChunks; ++ch)
    if (m_of[ch] > 0) atomicAdd(&cnt[m_of[ch]], 1);
  __syncthreads();
  if (tid == 0) {
    int s = 0, top = 0;
    for (int m = R; m >= 1; --m) { start[m] = s; s += cnt[m]; if (top == 0 && cnt[m] > 0) top = m; }
    for (int i = 1; i <= R; ++i) {
      const int n = a.dense ? (i <= top ? B : 0) : start[i] + cnt[i];  // n_i = #{m >= i}
      a.nact[i - 1] = n;
      s_nact[i - 1] = n;
    }
    s_top = top;
  }
  __syncthreads();
  const int top = s_top;

  // 1. rank of b among the sequences of its depth with smaller b
  const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
  for (int ch = 0; ch < kPlanChunks; ++ch) {
    if (ch * NT >= B) break;  // uniform
    const int m = m_of[ch];
    int rank = 0;
    for (int dv = 1; dv <= R; ++dv) {
      const unsigned long long mask = __ballot(m == dv);
      if (m == dv) rank = __popcll(mask & below);
      if (lane == 0) wcnt[wv][dv] = __popcll(mask);
    }
    __syncthreads();
    if (m > 0) {
      int off = 0;
      for (int w = 0; w < wv; ++w) off += wcnt[w][m];
      const int b = ch * NT + tid;
      const int row = a.dense ? b : start[m] + fill[m] + off + rank;
      row_of[ch] = row;
    }
    __syncthreads();
    if (tid >= 1 && tid <= R) {
      int t = 0;
      for (int w = 0; w < NW; ++w) t += wcnt[w][tid];
      fill[tid] += t;
    }
    __syncthreads();
  }

  // 2. pages needed: (b, i) for i < m_b whose next slot starts a page; each
  // row's first new page follows from a block prefix sum (every thread
  // carries the running total, so no barrier is needed between chunks), and
  // the entries each row's attention reads
  int ex_of[kPlanChunks];
  int total = 0;
  unsigned long long rd_sum = 0ull;
  const int lim_all = a.dense ? top : 0;  // dense: loops every row reads
#pragma unroll
  for (int ch = 0; ch < kPlanChunks; ++ch) {
    ex_of[ch] = 0;
    if (ch * NT >= B) break;  // uniform
    const int b = ch * NT + tid, m = m_of[ch];
    int need = 0;
    unsigned long long rd = 0ull;
#pragma unroll
    for (int i = 0; i < kMaxLoops; ++i) {
      if (m > 0 && i < m) {
        const int len = len_at(ch, b, i);
        need += len % kPage == 0;
        rd += (unsigned long long)(len + 1);
      } else if (m > 0 && i < lim_all) {  // dense: computed and discarded
        rd += (unsigned long long)len_at(ch, b, i);
      }
    }
    rd_sum += rd;
    int tot;
    ex_of[ch] = total + block_exclusive_scan(need, scan_tmp, &tot);
    total += tot;
  }
  // one LDS atomic per wave (a same-address atomic from every lane serialises)
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) rd_sum += shfl_xor(rd_sum, o);
  if (lane == 0 && rd_sum != 0ull) atomicAdd(&s_kvread, rd_sum);
  const int base = s_base;
  const bool oom = (int64_t)base + total > c.max_pages;
  if (tid == 0 && oom) set_err(c.err, kErrOutOfPages);
  __syncthreads();

  // 3. bookkeeping, before any slot is written (a barrier after global
  // stores would wait for them): the depth histogram, the deepest depth and
  // the entries written follow from the per-depth counts
  if (tid == 0 && !oom) *c.page_next = base + total;
  if (tid < R) atomicAdd(&c.depth_hist[tid], (unsigned long long)cnt[tid + 1]);
  if (tid == 0) {
    unsigned long long kvw = 0ull;
    for (int dv = 1; dv <= R; ++dv) kvw += (unsigned long long)dv * cnt[dv];
    if (oom) kvw = 0ull;
    const unsigned long long kvr = oom ? 0ull : s_kvread;
    c.step_stats[kStatKvRead] = (long long)(kvr * (unsigned long long)a.kv_entry_bytes);
    c.step_stats[kStatKvWrite] = (long long)(kvw * (unsigned long long)a.kv_entry_bytes);
    c.step_stats[kStatLoops] = top;
    add_stat(c.step_stats + kStatStepsTotal, 1ull);
    add_stat(c.step_stats + kStatKvWriteTotal, kvw * (unsigned long long)a.kv_entry_bytes);
    add_stat(c.step_stats + kStatLoopsTotal, (unsigned long long)top);
    if (!oom) {
      // each executed (loop, layer) attention reads every valid entry of its
      // cache plus one q row and writes one o row per active token; summed
      // over layers: entry bytes times (entries read + active rows)
      unsigned long long rows = 0;
      for (int i = 0; i < R; ++i)
        rows += (unsigned long long)(a.dense ? (i < top ? B : 0) : start[i + 1] + cnt[i + 1]);
      add_stat(c.step_stats + kStatAttnBytesTotal, (kvr + rows) * (unsigned long long)a.kv_entry_bytes);
    }
  }
  if (tid < R) {
    if (oom) a.nact[tid] = 0;  // the step becomes a no-op: no active rows
    c.step_stats[kStatRows + tid] = oom ? 0 : s_nact[tid];
  }

  // 4. slots of the executed (b, i): positions, cache lengths, new pages and
  // each compact row's slot offset, and the row order; no barrier follows
  // these stores
#pragma unroll
  for (int ch = 0; ch < kPlanChunks; ++ch) {
    if (ch * NT >= B) break;  // uniform
    const int b = ch * NT + tid, m = m_of[ch];
    if (m > 0 && !oom) {
      int len[kMaxLoops], page[kMaxLoops];
      const int lim = a.dense ? top : m;  // loops whose cache this row reads
#pragma unroll
      for (int i = 0; i < kMaxLoops; ++i) {
        len[i] = i < lim ? len_at(ch, b, i) : 0;
        page[i] = ch == 0 ? page0[i] : -1;
      }
      if (ch > 0) {
#pragma unroll
        for (int i = 0; i < kMaxLoops; ++i)
          if (i < m && len[i] % kPage != 0)
            page[i] = c.page_table[((int64_t)b * R + i) * c.pages_per_seq + len[i] / kPage];
      }
      int next = base + ex_of[ch];
      const int t = ch == 0 ? seq0 : c.seq_len[b];
#pragma unroll
      for (int i = 0; i < kMaxLoops; ++i) {
        if (i < m) {
          const int slot = len[i];
          if (slot % kPage == 0) {
            page[i] = next++;
            c.page_table[((int64_t)b * R + i) * c.pages_per_seq + slot / kPage] = page[i];
          }
          c.pos[(int64_t)page[i] * kPage + slot % kPage] = t;
          c.cache_len[b * R + i] = slot + 1;
          a.kv_slot[(int64_t)i * B + row_of[ch]] = (int64_t)page[i] * c.page_elems + slot % kPage;
        } else if (i < lim) {  // dense: computed and discarded
          a.kv_slot[(int64_t)i * B + row_of[ch]] = -1;
        }
      }
    }
    if (m > 0) {
      c.seq_len[b] = (ch == 0 ? seq0 : c.seq_len[b]) + 1;
      a.perm[row_of[ch]] = b;
      if (a.row_depth) a.row_depth[row_of[ch]] = m;
    }
  }
}

// ---------------------------------------------------------------------------
// Prefill planner: workgroup g handles sequence b0 + g.  For each loop i it
// gathers rho^(i) = sort(A_i) over the call's T tokens (Eq. 6) by a block
// prefix sum over the flags m_t >= i, and places those n entries in slots
// [n_old, n_old + n) of cache (b, i): n_old = 0 for a new batch, the current
// length when the call continues the caches (a later prompt chunk).  The
// partly filled last page is used first, then ceil-rounded new pages are
// taken from the pool; every new slot records its original position
// (Section 3.3 address translation).  chunk_len[b][i] = n.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kPlanThreads) void k_plan_prefill(PrefillPlanArgs a) {
  const CacheView& c = a.c;
  const int tid = threadIdx.x, g = blockIdx.x, T = a.T, R = c.R;
  const int b = a.b0 + g;
  const int64_t GT = (int64_t)a.G * T;
  __shared__ int scan_tmp[kPlanThreads / kWave + 1];
  __shared__ int s_carry, s_base, s_tiles[3];
  __shared__ unsigned long long hist[kMaxLoops];
  if (tid < kMaxLoops) hist[tid] = 0ull;
  __syncthreads();
  for (int t = tid; t < T; t += kPlanThreads) atomicAdd(&hist[a.depth[(int64_t)g * T + t] - 1], 1ull);
  for (int i = 0; i < R; ++i) {
    int32_t* idx = a.tok_idx + (int64_t)i * GT + (int64_t)g * T;
    if (tid == 0) s_carry = 0;
    __syncthreads();
    for (int t0 = 0; t0 < T; t0 += kPlanThreads) {
      const int t = t0 + tid;
      const int f = (t < T && a.depth[(int64_t)g * T + t] >= i + 1) ? 1 : 0;
      int tot;
      const int ex = block_exclusive_scan(f, scan_tmp, &tot);
      if (f) idx[s_carry + ex] = g * T + t;
      __syncthreads();
      if (tid == 0) s_carry += tot;
      __syncthreads();
    }
    const int n = s_carry;
    const int bi = b * R + i;
    const int old = a.append ? c.cache_len[bi] : 0;
    const int p_old = (old + kPage - 1) / kPage;        // pages already holding entries
    const int np = (old + n + kPage - 1) / kPage - p_old; // pages to take
    if (tid == 0) {
      int base = np > 0 ? atomicAdd(c.page_next, np) : 0;
      if ((int64_t)base + np > c.max_pages) {
        set_err(c.err, kErrOutOfPages);
        base = -1;
      }
      s_base = base;
    }
    __syncthreads();
    const int base = s_base;
    const int nn = base < 0 ? 0 : n;
    int32_t* pt = c.page_table + (int64_t)bi * c.pages_per_seq;
    if (base >= 0) {
      for (int p = tid; p < np; p += kPlanThreads) pt[p_old + p] = base + p;
      // tail of the partly filled page
      const int tail = p_old * kPage - old;
      if (tid < tail && tid < n) {
        const int s = old + tid;
        c.pos[(int64_t)pt[s / kPage] * kPage + s % kPage] = a.pos0 + idx[tid] - g * T;
      }
      // whole new pages; slots past the last entry are marked empty
      for (int s = tid; s < np * kPage; s += kPlanThreads) {
        const int e = p_old * kPage + s - old;  // entry index within the call
        c.pos[(int64_t)base * kPage + s] = e < n ? a.pos0 + idx[e] - g * T : -1;
      }
    }
    // the cache slot offset of every gathered entry, for the QKV epilogue:
    // entry e goes to slot old + e, on the partly filled last page or on new
    // page base + (page index - p_old)
    int64_t* ks = a.kv_slot + (int64_t)i * GT + (int64_t)g * T;
    for (int e = tid; e < n; e += kPlanThreads) {
      const int s = old + e, pi = s / kPage;
      const int page = base < 0 ? -1 : pi < p_old ? pt[pi] : base + (pi - p_old);
      ks[e] = page < 0 || page >= c.max_pages ? -1 : (int64_t)page * c.page_elems + s % kPage;
    }
    if (a.tile_cnt) {
      // this sequence's active row tiles of loop i: rows g T + k BM, k < ceil(nn / BM)
      const int t64 = (nn + 63) / 64, t128 = (nn + 127) / 128, t256 = (nn + 255) / 256;
      if (tid == 0) {
        s_tiles[0] = atomicAdd(&a.tile_cnt[i * 3 + 0], t64);
        s_tiles[1] = atomicAdd(&a.tile_cnt[i * 3 + 1], t128);
        s_tiles[2] = atomicAdd(&a.tile_cnt[i * 3 + 2], t256);
      }
      __syncthreads();
      for (int k = tid; k < t64; k += kPlanThreads) a.tile_list64[(int64_t)i * (GT / 64) + s_tiles[0] + k] = g * T + k * 64;
      for (int k = tid; k < t128; k += kPlanThreads)
        a.tile_list128[(int64_t)i * (GT / 128) + s_tiles[1] + k] = g * T + k * 128;
      for (int k = tid; k < t256; k += kPlanThreads)
        a.tile_list256[(int64_t)i * (GT / 256) + s_tiles[2] + k] = g * T + k * 256;
    }
    if (tid == 0) {
      c.cache_len[bi] = old + nn;
      c.chunk_len[bi] = nn;
    }
    __syncthreads();
  }
  if (tid == 0) c.seq_len[b] = a.pos0 + T;
  if (tid < R) atomicAdd(&c.depth_hist[tid], hist[tid]);
}

__global__ void k_fill_i32(int32_t* p, int32_t v, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}
__global__ void k_fill_u64(unsigned long long* p, unsigned long long v, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = v;
}
// one wave per row: the largest of its group keys (value, then lowest id)
__global__ void k_argmax_finalize(const unsigned long long* keys, int groups, int32_t* next, int B) {
  const int b = blockIdx.x * (blockDim.x / kWave) + (int)(threadIdx.x / kWave), lane = lane_id();
  if (b >= B) return;
  unsigned long long key = 0ull;
  for (int gi = lane; gi < groups; gi += kWave) {
    const unsigned long long k = keys[(int64_t)b * groups + gi];
    key = k > key ? k : key;
  }
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const unsigned long long other = shfl_xor(key, o);
    key = other > key ? other : key;
  }
  if (lane == 0) next[b] = (int32_t)(0xFFFFFFFFu - (unsigned)(key & 0xFFFFFFFFull));
}

int fill_grid(int64_t n) {
  int64_t g = (n + 255) / 256;
  if (g > 4096) g = 4096;
  return g < 1 ? 1 : (int)g;
}

}  // namespace

hipError_t launch_plan_decode(const DecodePlanArgs& a, hipStream_t s) {
  if (a.B < 0 || a.B > kPlanThreads * kPlanChunks) return hipErrorInvalidValue;
  // fewer threads for a small batch: the planner's many barriers then wait
  // for fewer waves
  const int nt = std::min(kPlanThreads, std::max(kWave, (a.B + kWave - 1) / kWave * kWave));
  hipLaunchKernelGGL(k_plan_decode, dim3(1), dim3(nt), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_plan_prefill(const PrefillPlanArgs& a, hipStream_t s) {
  if (a.G <= 0) return hipSuccess;
  if (a.tile_cnt && (a.T % 256 != 0 || !a.tile_list64 || !a.tile_list128 || !a.tile_list256))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_plan_prefill, dim3(a.G), dim3(kPlanThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_i32, dim3(fill_grid(n)), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}
hipError_t launch_fill_u64(unsigned long long* p, unsigned long long v, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_u64, dim3(fill_grid(n)), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}
hipError_t launch_argmax_finalize(const unsigned long long* keys, int groups, int32_t* next, int B, hipStream_t s) {
  if (B <= 0) return hipSuccess;
  if (B <= 0 || groups <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_argmax_finalize, dim3((B + 3) / 4), dim3(4 * kWave), 0, s, keys, groups, next, B);
  return hipGetLastError();
}

}  // namespace tlf
