// MFMA GEMM for the shared block's projections and the LM head.
//
// out = A W^T on the active rows of a row map, with W [N][K] row-major
// (linear-layer layout) and A either
//   A_NORM: the float residual rows x[src(r)], normalised by RMSNorm without
//           affine (Appendix A).  The row's sum of squares is accumulated
//           while its K tiles stream through, and 1/rms scales the
//           accumulator in the epilogue (RMSNorm commutes with the
//           projection), so the norm costs no extra pass.
//   A_BUF:  storage-dtype rows buf[r] (attention output, SwiGLU activation).
// Epilogues:
//   E_QKV:    q to a buffer; k, v appended to the loop's cache pages (Eq. 11)
//   E_RESID:  x[src(r)] += result (residual of the attention/FFN branch)
//   E_SWIGLU: act = silu(gate) * up, gate/up columns interleaved in 16-column
//             groups so every wave holds matching pairs
//   E_LOGITS: float logits plus a packed (value, -index) atomicMax for greedy
//
// Tiling: 256 threads = 4 waves in a 2x2 grid; each wave owns MT x NT 16x16
// MFMA tiles.  K advances 128 bytes per tile (64 bf16 / 32 f32), staged
// through LDS with the next tile prefetched into registers.
#include "kernels.h"

namespace tlf {

namespace {

__device__ __forceinline__ unsigned int ordered_bits(float v) {
  unsigned int u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int64_t kv_slot_base(const KvDst& kv, int r, int src) {
  const CacheView& c = kv.c;
  int b, slot;
  if (kv.prefill) {
    b = kv.b0 + r / kv.seg;
    slot = r % kv.seg;
  } else {
    b = src;
    slot = c.cache_len[b * c.R + kv.loop] - 1;
  }
  const int page = c.page_table[((int64_t)b * c.R + kv.loop) * c.pages_per_seq + slot / kPage];
  if (page < 0 || page >= c.max_pages) return -1;
  return (int64_t)page * c.page_elems + page_off(c, kv.layer, 0, 0, slot % kPage);
}

template <typename T, int MT, int NT, int AK, int EK>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs g) {
  constexpr int BM = 2 * MT * 16, BN = 2 * NT * 16;
  constexpr int BK = 128 / (int)sizeof(T);
  constexpr int LDK = BK + 16 / (int)sizeof(T);
  using M = Mfma<T>;
  constexpr int KS = M::KS, EPL = M::EPL;
  // A chunks: 16-byte pieces of the source rows
  constexpr int A_ELEM_BYTES = (AK == A_NORM) ? 4 : (int)sizeof(T);
  constexpr int A_CPR = BK * A_ELEM_BYTES / 16;       // chunks per row per K tile
  constexpr int A_EPC = 16 / A_ELEM_BYTES;            // elements per chunk
  constexpr int ACH = BM * A_CPR / 256;               // chunks per thread
  constexpr int B_CPR = 8;
  constexpr int B_EPC = 16 / (int)sizeof(T);
  constexpr int BCH = BN * B_CPR / 256;
  static_assert(ACH >= 1 && BM * A_CPR % 256 == 0, "A tile split");
  static_assert(BCH >= 1 && BN * B_CPR % 256 == 0, "B tile split");

  __shared__ __align__(16) T As[BM * LDK];
  __shared__ __align__(16) T Bs[BN * LDK];
  __shared__ float inv_rms[BM];
  __shared__ int row_src_s[BM];
  __shared__ int64_t kv_base[EK == E_QKV ? BM : 1];
  __shared__ int any_active;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int r0 = blockIdx.y * BM, n0 = blockIdx.x * BN;

  if (tid == 0) any_active = 0;
  __syncthreads();
  for (int i = tid; i < BM; i += 256) {
    const int r = r0 + i;
    int s = -1;
    if (row_active(g.rm, r)) s = row_src(g.rm, r);
    row_src_s[i] = s;
    if (s >= 0) any_active = 1;
    if constexpr (EK == E_QKV) kv_base[i] = (s >= 0) ? kv_slot_base(g.kv, r, s) : -1;
  }
  __syncthreads();
  if (!any_active) return;

  // W row of output column n (clamped; columns >= N are never stored)
  auto w_row = [&](int n) -> int {
    int wr = n;
    if constexpr (EK == E_SWIGLU) {
      const int grp = n >> 5, w = n & 31;
      wr = (w < 16) ? grp * 16 + w : g.F + grp * 16 + (w - 16);
    }
    return wr < g.w_rows ? wr : g.w_rows - 1;
  };

  typedef typename std::conditional<AK == A_NORM, float4, V16<T>>::type AReg;
  AReg ra[ACH];
  V16<T> rb[BCH];
  float ss[ACH];
#pragma unroll
  for (int c = 0; c < ACH; ++c) ss[c] = 0.f;

  const float* Af = reinterpret_cast<const float*>(g.A);
  const T* Ab = reinterpret_cast<const T*>(g.A);
  const T* W = reinterpret_cast<const T*>(g.W);

  auto load_tiles = [&](int kt) {
#pragma unroll
    for (int c = 0; c < ACH; ++c) {
      const int ch = tid + c * 256, row = ch / A_CPR, col = (ch % A_CPR) * A_EPC;
      const int s = row_src_s[row];
      if constexpr (AK == A_NORM) {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (s >= 0) v = *reinterpret_cast<const float4*>(Af + (int64_t)s * g.lda + kt * BK + col);
        ra[c] = v;
      } else {
        V16<T> v;
        v.u = make_uint4(0, 0, 0, 0);
        if (s >= 0) v = ld16(Ab + (int64_t)(r0 + row) * g.lda + kt * BK + col);
        ra[c] = v;
      }
    }
#pragma unroll
    for (int c = 0; c < BCH; ++c) {
      const int ch = tid + c * 256, row = ch / B_CPR, col = (ch % B_CPR) * B_EPC;
      rb[c] = ld16(W + (int64_t)w_row(n0 + row) * g.K + kt * BK + col);
    }
  };
  auto store_tiles = [&]() {
#pragma unroll
    for (int c = 0; c < ACH; ++c) {
      const int ch = tid + c * 256, row = ch / A_CPR, col = (ch % A_CPR) * A_EPC;
      if constexpr (AK == A_NORM) {
        const float4 v = ra[c];
        // explicit fma chain: every row's sum of squares is formed the same way,
        // whichever unrolled slot loads it
        ss[c] = fmaf(v.w, v.w, fmaf(v.z, v.z, fmaf(v.y, v.y, fmaf(v.x, v.x, ss[c]))));
        T* p = &As[row * LDK + col];
        p[0] = from_f<T>(v.x); p[1] = from_f<T>(v.y); p[2] = from_f<T>(v.z); p[3] = from_f<T>(v.w);
      } else {
        st16(&As[row * LDK + col], ra[c]);
      }
    }
#pragma unroll
    for (int c = 0; c < BCH; ++c) {
      const int ch = tid + c * 256, row = ch / B_CPR, col = (ch % B_CPR) * B_EPC;
      st16(&Bs[row * LDK + col], rb[c]);
    }
  };

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int KT = g.K / BK;
  load_tiles(0);
  for (int kt = 0; kt < KT; ++kt) {
    __syncthreads();
    store_tiles();
    __syncthreads();
    if (kt + 1 < KT) load_tiles(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK / KS; ++ks) {
      typename M::frag af[MT], bfr[NT];
#pragma unroll
      for (int i = 0; i < MT; ++i)
        af[i] = M::load(&As[(wm * MT * 16 + i * 16 + (lane & 15)) * LDK + ks * KS + (lane >> 4) * EPL]);
#pragma unroll
      for (int j = 0; j < NT; ++j)
        bfr[j] = M::load(&Bs[(wn * NT * 16 + j * 16 + (lane & 15)) * LDK + ks * KS + (lane >> 4) * EPL]);
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = M::mma(af[i], bfr[j], acc[i][j]);
    }
  }

  if constexpr (AK == A_NORM) {
    // threads sharing a row are A_CPR consecutive lanes of one wave
#pragma unroll
    for (int c = 0; c < ACH; ++c) {
      float v = ss[c];
#pragma unroll
      for (int o = 1; o < A_CPR; o <<= 1) v += shfl_xor(v, o);
      const int ch = tid + c * 256;
      if (ch % A_CPR == 0) inv_rms[ch / A_CPR] = rsqrtf(v / (float)g.K + g.eps);
    }
    __syncthreads();
  }

  const int quad = lane >> 4, col16 = lane & 15;
#pragma unroll
  for (int i = 0; i < MT; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int rl = wm * MT * 16 + i * 16 + quad * 4 + r;
      const int src = row_src_s[rl];
      const int rg = r0 + rl;
      const float sc = (AK == A_NORM) ? inv_rms[rl] : 1.f;
      if constexpr (EK == E_LOGITS) {
        unsigned long long best = 0ull;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const int n = n0 + wn * NT * 16 + j * 16 + col16;
          const float v = acc[i][j][r] * sc;
          if (src >= 0 && n < g.N) {
            reinterpret_cast<float*>(g.out)[(int64_t)(g.out_row_off + rg) * g.ldo + n] = v;
            const unsigned long long key =
                ((unsigned long long)ordered_bits(v) << 32) | (unsigned long long)(0xFFFFFFFFu - (unsigned)n);
            best = key > best ? key : best;
          }
        }
        if (g.argmax_keys) {
#pragma unroll
          for (int o = 1; o < 16; o <<= 1) {
            const unsigned long long other = shfl_xor(best, o);
            best = other > best ? other : best;
          }
          if (col16 == 0 && src >= 0 && best != 0ull) atomicMax(&g.argmax_keys[g.out_row_off + rg], best);
        }
      } else if constexpr (EK == E_SWIGLU) {
#pragma unroll
        for (int j = 0; j < NT; j += 2) {
          const int n = n0 + wn * NT * 16 + j * 16 + col16;  // gate column (n % 32 < 16)
          const int unit = (n >> 5) * 16 + col16;
          if (src >= 0 && unit < g.F) {
            const float gt = acc[i][j][r] * sc, up = acc[i][j + 1][r] * sc;
            const float a = gt / (1.f + __expf(-gt)) * up;
            reinterpret_cast<T*>(g.out)[(int64_t)rg * g.ldo + unit] = from_f<T>(a);
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const int n = n0 + wn * NT * 16 + j * 16 + col16;
          if (src < 0 || n >= g.N) continue;
          const float v = acc[i][j][r] * sc;
          if constexpr (EK == E_RESID) {
            reinterpret_cast<float*>(g.out)[(int64_t)src * g.ldo + n] += v;
          } else {  // E_QKV
            if (n < g.d) {
              reinterpret_cast<T*>(g.out)[(int64_t)rg * g.ldo + n] = from_f<T>(v);
            } else {
              const int64_t base = kv_base[rl];
              if (base >= 0) {
                const int nn = n - g.d, kvsel = nn / g.d, within = nn % g.d;
                const int h = within / g.kv.c.D, e = within % g.kv.c.D;
                T* pool = reinterpret_cast<T*>(g.kv.c.pool);
                pool[base + (int64_t)((kvsel * g.kv.c.H + h) * kPage) * g.kv.c.D + e] = from_f<T>(v);
              }
            }
          }
        }
      }
    }
  }
}

template <typename T, int MT, int NT>
hipError_t launch_tiles(const GemmArgs& a, AKind ak, EKind ek, hipStream_t s) {
  constexpr int BM = 2 * MT * 16, BN = 2 * NT * 16;
  dim3 grid((a.N + BN - 1) / BN, (a.rm.rows + BM - 1) / BM);
  if (grid.x == 0 || grid.y == 0) return hipSuccess;
  if (ak == A_NORM && ek == E_QKV)
    hipLaunchKernelGGL((k_gemm<T, MT, NT, A_NORM, E_QKV>), grid, dim3(256), 0, s, a);
  else if (ak == A_BUF && ek == E_RESID)
    hipLaunchKernelGGL((k_gemm<T, MT, NT, A_BUF, E_RESID>), grid, dim3(256), 0, s, a);
  else if (ak == A_NORM && ek == E_SWIGLU)
    hipLaunchKernelGGL((k_gemm<T, MT, NT, A_NORM, E_SWIGLU>), grid, dim3(256), 0, s, a);
  else if (ak == A_NORM && ek == E_LOGITS)
    hipLaunchKernelGGL((k_gemm<T, MT, NT, A_NORM, E_LOGITS>), grid, dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

template <typename T>
hipError_t launch_gemm(const GemmArgs& a, AKind ak, EKind ek, bool big_tiles, hipStream_t s) {
  constexpr int BK = 128 / (int)sizeof(T);
  if (a.K % BK != 0) return hipErrorInvalidValue;
  if (big_tiles) return launch_tiles<T, 4, 4>(a, ak, ek, s);
  return launch_tiles<T, 1, 2>(a, ak, ek, s);
}

template hipError_t launch_gemm<float>(const GemmArgs&, AKind, EKind, bool, hipStream_t);
template hipError_t launch_gemm<bf16>(const GemmArgs&, AKind, EKind, bool, hipStream_t);

}  // namespace tlf
