// Decode-shaped projections: out = A W^T for the few active rows of one loop
// (at most the batch), with W [N][K] in the storage dtype and A float32.
//
// At these row counts a projection moves 1-6 MB of weights and does little
// arithmetic, so its time is latency: the chain of dependent loads before
// the first product and the number of memory round trips.  Here a workgroup
// of W waves owns a BM x BN output tile; its waves split K between them
// (wave w takes K steps w, w + W, ...), issue all of their loads at once,
// straight into MFMA operand registers (no LDS staging: a lane's operand
// fragment is 8 consecutive k of one row, a 16- or 32-byte load), and sum
// their partial tiles through LDS in a fixed order.  One kernel therefore
// needs one or two load round trips, and every output has one writer, so
// the residual projections add into x directly (deterministic, no split-K
// slabs and no reduction kernel).
//
// The residual stream of a decode step is kept in depth-sorted (compact)
// row order, so that the active rows of every loop are rows [0, n_i) and
// operand rows need no indirection: the step's first projection reads x in
// batch order through the permutation and writes the compact copy, and the
// LM head writes each logits row back to its sequence.
//
// NORM: A is the residual x and the product is taken with RMSNorm(x)
// (no affine): the sum of squares of each row is accumulated from the same
// operand registers and the output row is scaled by 1/rms in the epilogue,
// since (x / rms) W^T = (x W^T) / rms.  This fuses the norm in front of the
// QKV, gate/up and LM-head projections.
//
// With bf16 weights each float32 operand enters the MFMA as bf16 hi + lo
// parts (one product each), as in the prefill GEMM.
//
// Workgroups are numbered so that all row tiles of one column tile run on
// the same XCD (workgroup i runs on XCD i mod 8) and share its L2 copy of
// the weight tile.
#include "kernels.h"

namespace tlf {

namespace {

__device__ __forceinline__ unsigned int ordered_bits(float v) {
  unsigned int u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kXcds = 8;

template <typename T, int RM, int CN, int W, int KB, int AK, int EK, bool NORM>
__global__ __launch_bounds__(W * 64) void k_dgemm(GemmArgs g, int tiles_n, int tiles_m) {
  using M = Mfma<T>;
  typedef typename M::frag Frag;
  constexpr int KS = M::KS, EPL = M::EPL;
  constexpr bool kSplit = sizeof(T) == 2;
  constexpr int BM = RM * 16, BN = CN * 16;
  constexpr int LDR = BN + 1;  // padded LDS row of a partial tile
  constexpr int NT = W * kWave;
  constexpr int EOUT = EK == E_SWIGLU ? BM * BN / 2 : BM * BN;  // epilogue outputs of the tile
  constexpr int EPT = (EOUT + NT - 1) / NT;                     // per thread
  constexpr int SLOTS = W > 8 ? 8 : W;  // partial tiles in LDS (16 waves fold pairwise first)
  static_assert(W == SLOTS || W == 2 * SLOTS, "waves");
  static_assert(EK != E_SWIGLU || CN % 2 == 0, "gate/up pairs");
  static_assert(EK != E_LOGITS || (BN == kWave && EOUT % NT == 0), "one wave per logits row");

  __shared__ float red[SLOTS][BM * LDR];
  __shared__ float s_ss[NORM ? W : 1][BM];
  __shared__ float s_inv[BM];
  __shared__ int s_orow[EK == E_LOGITS ? BM : 1];
  __shared__ int64_t s_kv[EK == E_QKV ? BM : 1];

  const int L = blockIdx.x;
  const int tn = L % kXcds + kXcds * ((L / kXcds) / tiles_m), tm = (L / kXcds) % tiles_m;
  if (tn >= tiles_n) return;
  const int r0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int quad = lane >> 4, c16 = lane & 15;

  // Loads are issued in dependency order: the weight fragments, the
  // epilogue's bookkeeping and residual values, then the activation
  // fragments (after the row permutation for A_SRC).  With g.spec (every
  // row active, e.g. the first loop) they go out before the active-row
  // count arrives; otherwise a tile whose first row has exited returns on
  // the count before loading anything, and activation rows past the count
  // are not loaded.
  const int nact = g.rm.nact ? *g.rm.nact : g.rm.rows;
  if (!g.spec && r0 >= nact) return;
  const int a_rows = g.spec ? g.rm.rows : min(nact, g.rm.rows);  // activation rows worth loading
  // 32-bit element offsets from uniform bases (the weight and activation
  // matrices hold fewer than 2^31 elements)
  const T* Wb = reinterpret_cast<const T*>(g.W);
  int wo[CN];
#pragma unroll
  for (int c = 0; c < CN; ++c) {
    int n = n0 + c * 16 + c16, wr = n;
    if constexpr (EK == E_SWIGLU) {
      // interleaved 32-column groups: 16 gate columns, then the 16 up columns of the same units
      const int grp = n >> 5, k = n & 31;
      wr = (k < 16) ? grp * 16 + k : g.F + grp * 16 + (k - 16);
    }
    wr = min(wr, g.w_rows - 1);
    wo[c] = wr * g.K + quad * EPL;
  }
  if (w == 0 && quad == 0) {
#pragma unroll
    for (int i = 0; i < RM; ++i) {
      const int rl = i * 16 + c16, r = min(r0 + rl, g.rm.rows - 1);
      if constexpr (EK == E_QKV) s_kv[rl] = g.kv.slot_base[r];
      if constexpr (EK == E_LOGITS) s_orow[rl] = g.rm.src ? g.rm.src[r] : g.out_row_off + r;
    }
  }
  float xr[EK == E_RESID ? EPT : 1];
  if constexpr (EK == E_RESID) {
#pragma unroll
    for (int k = 0; k < EPT; ++k) {
      const int e = tid + k * NT, row = e / BN, n = n0 + e % BN;
      xr[k] = (e < EOUT && r0 + row < a_rows && n < g.N) ? g.out[(int64_t)(r0 + row) * g.ldo + n] : 0.f;
    }
  }
  const float* Ab = g.A;
  int ao[RM];
#pragma unroll
  for (int i = 0; i < RM; ++i) {
    const int r = min(r0 + i * 16 + c16, g.rm.rows - 1);
    const int arow = (AK == A_SRC) ? row_src(g.rm, r) : r;
    ao[i] = arow * g.lda + quad * EPL;
  }

  const int S = g.K / KS;              // K steps
  const int NJ = (S - w + W - 1) / W;  // steps of this wave (w, w + W, ...)
  f32x4 acc[RM][CN];
#pragma unroll
  for (int i = 0; i < RM; ++i)
#pragma unroll
    for (int c = 0; c < CN; ++c) acc[i][c] = f32x4{0.f, 0.f, 0.f, 0.f};
  float ss[RM];
#pragma unroll
  for (int i = 0; i < RM; ++i) ss[i] = 0.f;

  for (int jb = 0; jb < (S + W - 1) / W; jb += KB) {
    float av[KB][RM][EPL];
    Frag bw[KB][CN];
    // past this wave's last step the last step is reread (its product is skipped)
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      const int k0 = min(w + W * (jb + j), S - 1) * KS;
#pragma unroll
      for (int c = 0; c < CN; ++c) bw[j][c] = M::load(Wb + (wo[c] + k0));
    }
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      const int k0 = min(w + W * (jb + j), S - 1) * KS;
#pragma unroll
      for (int i = 0; i < RM; ++i) {
#pragma unroll
        for (int e = 0; e < EPL; ++e) av[j][i][e] = 0.f;
        if (r0 + i * 16 >= a_rows) continue;  // uniform: the fragment's rows have exited
        if (r0 + i * 16 + c16 < a_rows) {
          if constexpr (EPL == 8) {
            const float4 lo = *reinterpret_cast<const float4*>(Ab + (ao[i] + k0));
            const float4 hi = *reinterpret_cast<const float4*>(Ab + (ao[i] + k0 + 4));
            av[j][i][0] = lo.x; av[j][i][1] = lo.y; av[j][i][2] = lo.z; av[j][i][3] = lo.w;
            av[j][i][4] = hi.x; av[j][i][5] = hi.y; av[j][i][6] = hi.z; av[j][i][7] = hi.w;
          } else {
            av[j][i][0] = Ab[ao[i] + k0];
          }
        }
      }
    }
    if (jb == 0 && r0 >= nact) return;  // uniform: the tile's rows have all exited
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      if (jb + j >= NJ) break;  // wave-uniform
      const int k0 = (w + W * (jb + j)) * KS;
#pragma unroll
      for (int i = 0; i < RM; ++i) {
        if (g.a_copy && tn == 0) {
          // the compact copy of the operand rows (first projection of a step)
          const int r = r0 + i * 16 + c16;
          if (r < g.rm.rows) {
            float* dst = g.a_copy + (int64_t)r * g.lda + k0 + quad * EPL;
#pragma unroll
            for (int e = 0; e < EPL; ++e) dst[e] = av[j][i][e];
          }
        }
        if constexpr (NORM) {
#pragma unroll
          for (int e = 0; e < EPL; ++e) ss[i] = fmaf(av[j][i][e], av[j][i][e], ss[i]);
        }
        if constexpr (kSplit) {
          uint2 h0, l0, h1, l1;
          split4(make_float4(av[j][i][0], av[j][i][1], av[j][i][2], av[j][i][3]), h0, l0);
          split4(make_float4(av[j][i][4], av[j][i][5], av[j][i][6], av[j][i][7]), h1, l1);
          const bf16x8 ahi = __builtin_bit_cast(bf16x8, make_uint4(h0.x, h0.y, h1.x, h1.y));
          const bf16x8 alo = __builtin_bit_cast(bf16x8, make_uint4(l0.x, l0.y, l1.x, l1.y));
#pragma unroll
          for (int c = 0; c < CN; ++c) {
            acc[i][c] = M::mma(ahi, bw[j][c], acc[i][c]);
            acc[i][c] = M::mma(alo, bw[j][c], acc[i][c]);
          }
        } else {
#pragma unroll
          for (int c = 0; c < CN; ++c) acc[i][c] = M::mma(av[j][i][0], bw[j][c], acc[i][c]);
        }
      }
    }
  }

  // partial tiles into LDS (lane: rows 4 * quad + r of column c16); with 16
  // waves, wave w + 8 first hands its tile to wave w
  if constexpr (W > SLOTS) {
    if (w >= SLOTS) {
#pragma unroll
      for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int c = 0; c < CN; ++c)
#pragma unroll
          for (int r = 0; r < 4; ++r) red[w - SLOTS][(i * 16 + quad * 4 + r) * LDR + c * 16 + c16] = acc[i][c][r];
    }
    __syncthreads();
    if (w < SLOTS) {
#pragma unroll
      for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int c = 0; c < CN; ++c)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[i][c][r] += red[w][(i * 16 + quad * 4 + r) * LDR + c * 16 + c16];
    }
    __syncthreads();
  }
  if (w < SLOTS) {
#pragma unroll
    for (int i = 0; i < RM; ++i)
#pragma unroll
      for (int c = 0; c < CN; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[w][(i * 16 + quad * 4 + r) * LDR + c * 16 + c16] = acc[i][c][r];
  }
  if constexpr (NORM) {
#pragma unroll
    for (int i = 0; i < RM; ++i) {
      float t = ss[i];
      t += shfl_xor(t, 16);
      t += shfl_xor(t, 32);
      if (quad == 0) s_ss[w][i * 16 + c16] = t;
    }
  }
  __syncthreads();
  if constexpr (NORM) {
    if (tid < BM) {
      float t = 0.f;
#pragma unroll
      for (int ww = 0; ww < W; ++ww) t += s_ss[ww][tid];
      s_inv[tid] = rsqrtf(t / (float)g.K + g.eps);
    }
    __syncthreads();
  }
  auto tile_sum = [&](int row, int col) -> float {
    float v = 0.f;
#pragma unroll
    for (int ww = 0; ww < SLOTS; ++ww) v += red[ww][row * LDR + col];
    if constexpr (NORM) v *= s_inv[row];
    return v;
  };
  const int row_end = min(g.rm.rows, nact);  // rows [r0, row_end) are active

#pragma unroll
  for (int k = 0; k < EPT; ++k) {
    const int e = tid + k * NT;
    if (e >= EOUT) break;
    if constexpr (EK == E_SWIGLU) {
      const int row = e / (BN / 2), u = e % (BN / 2);
      const int gcol = (u / 16) * 32 + (u % 16);       // gate column in the tile
      const int unit = ((n0 + gcol) >> 5) * 16 + (u % 16);
      if (r0 + row >= row_end || unit >= g.F) continue;
      const float gt = tile_sum(row, gcol), up = tile_sum(row, gcol + 16);
      g.out[(int64_t)(r0 + row) * g.ldo + unit] = gt / (1.f + __expf(-gt)) * up;
    } else if constexpr (EK == E_LOGITS) {
      const int row = e / BN, n = n0 + e % BN;
      const bool ok = r0 + row < row_end && n < g.N;
      const int orow = s_orow[row];
      unsigned long long key = 0ull;
      if (ok) {
        const float v = tile_sum(row, e % BN);
        g.out[(int64_t)orow * g.ldo + n] = v;
        key = ((unsigned long long)ordered_bits(v) << 32) | (unsigned long long)(0xFFFFFFFFu - (unsigned)n);
      }
      if (g.argmax_keys) {
        // the 64 lanes of a wave hold one row's 64 columns
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
          const unsigned long long other = shfl_xor(key, o);
          key = other > key ? other : key;
        }
        if (lane == 0 && key != 0ull) atomicMax(&g.argmax_keys[orow], key);
      }
    } else {
      const int row = e / BN, col = e % BN, n = n0 + col;
      if (r0 + row >= row_end || n >= g.N) continue;
      const float v = tile_sum(row, col);
      if constexpr (EK == E_RESID) {
        g.out[(int64_t)(r0 + row) * g.ldo + n] = xr[k] + v;
      } else {  // E_QKV
        if (n < g.d) {
          g.out[(int64_t)(r0 + row) * g.ldo + n] = v;
        } else {
          const int64_t base = s_kv[row];
          const int slot = (int)(base & (kPage - 1));
          const int64_t page = base - slot;
          const int nn = n - g.d, kvsel = nn / g.d, within = nn % g.d;
          const int h = within / g.kv.c.D, el = within % g.kv.c.D;
          T* pool = reinterpret_cast<T*>(g.kv.c.pool);
          if (kvsel == 0)
            pool[page + k_block(g.kv.c, g.kv.layer, h) + (int64_t)slot * g.kv.c.D + el] = from_f<T>(v);
          else
            pool[page + v_block(g.kv.c, g.kv.layer, h) + (int64_t)el * kPage + slot] = from_f<T>(v);
        }
      }
    }
  }
}

template <typename T, int RM, int CN, int W, int KB, int AK, int EK, bool NORM>
hipError_t launch_cfg(const GemmArgs& a, hipStream_t s) {
  constexpr int BM = RM * 16, BN = CN * 16;
  const int tiles_n = (a.N + BN - 1) / BN, tiles_m = (a.rm.rows + BM - 1) / BM;
  const int grid = kXcds * ((tiles_n + kXcds - 1) / kXcds) * tiles_m;
  if (tiles_n == 0 || tiles_m == 0) return hipSuccess;
  hipLaunchKernelGGL((k_dgemm<T, RM, CN, W, KB, AK, EK, NORM>), dim3(grid), dim3(W * 64), 0, s, a, tiles_n,
                     tiles_m);
  return hipGetLastError();
}

// K steps per wave in one batch of loads: all of a wave's steps when they
// fit in KBMAX, else batches of KBMAX.
template <typename T, int RM, int CN, int W, int KBMAX, int AK, int EK, bool NORM>
hipError_t launch_w(const GemmArgs& a, hipStream_t s) {
  const int nj = (a.K / Mfma<T>::KS + W - 1) / W;
  if (nj <= 2 || KBMAX == 2) return launch_cfg<T, RM, CN, W, 2, AK, EK, NORM>(a, s);
  if (nj <= 3 || KBMAX == 3) return launch_cfg<T, RM, CN, W, (KBMAX >= 3 ? 3 : 2), AK, EK, NORM>(a, s);
  return launch_cfg<T, RM, CN, W, (KBMAX >= 4 ? 4 : 2), AK, EK, NORM>(a, s);
}

}  // namespace

// Tile shapes (rows x columns, waves), measured on the projections of a
// 256-row batch: the first loop has every row of the batch active (g.spec),
// so its shapes aim at about one workgroup per compute unit over all rows;
// later loops have fewer rows and use narrower tiles.
//   QKV:     first loop 32 x 80,  later 32 x 64   (8 waves)
//   gate/up: first loop 32 x 128, later 32 x 64   (8 waves)
//   O:       32 x 32 (8 waves)
//   down:    first loop 16 x 64 (8 waves), later 16 x 32 (16 waves)  [K > 768 in bf16]
//   LM head: 32 x 64 (8 waves)
template <typename T>
hipError_t launch_dgemm(const GemmArgs& a, AKind ak, EKind ek, bool norm, hipStream_t s) {
  if (a.K % Mfma<T>::KS != 0 || a.rm.rows <= 0) return hipErrorInvalidValue;
  const bool full = a.spec != 0;
  if (ek == E_QKV && norm) {
    if (ak == A_SRC) return launch_w<T, 2, 5, 8, 3, A_SRC, E_QKV, true>(a, s);
    if (full) return launch_w<T, 2, 5, 8, 3, A_CMP, E_QKV, true>(a, s);
    return launch_w<T, 2, 4, 8, 3, A_CMP, E_QKV, true>(a, s);
  }
  if (ak == A_CMP && ek == E_SWIGLU && norm) {
    if (full) return launch_w<T, 2, 8, 8, 3, A_CMP, E_SWIGLU, true>(a, s);
    return launch_w<T, 2, 4, 8, 3, A_CMP, E_SWIGLU, true>(a, s);
  }
  if (ak == A_CMP && ek == E_LOGITS && norm) return launch_w<T, 2, 4, 8, 3, A_CMP, E_LOGITS, true>(a, s);
  if (ak == A_CMP && ek == E_RESID && !norm) {
    if (a.K / Mfma<T>::KS > 3 * 8) {
      if (full) return launch_w<T, 1, 4, 8, 4, A_CMP, E_RESID, false>(a, s);
      return launch_w<T, 1, 2, 16, 4, A_CMP, E_RESID, false>(a, s);
    }
    return launch_w<T, 2, 2, 8, 3, A_CMP, E_RESID, false>(a, s);
  }
  return hipErrorInvalidValue;
}

template hipError_t launch_dgemm<float>(const GemmArgs&, AKind, EKind, bool, hipStream_t);
template hipError_t launch_dgemm<bf16>(const GemmArgs&, AKind, EKind, bool, hipStream_t);

}  // namespace tlf
