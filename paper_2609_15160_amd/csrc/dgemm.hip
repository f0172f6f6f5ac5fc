// Decode-shaped projections: out = A W^T for the few active rows of one loop
// (at most the batch), with W [N][K] in the storage dtype and A float32.
//
// At these row counts a projection moves 1-6 MB of weights and does little
// arithmetic, so its time is latency: the chain of dependent loads before
// the first product and the number of memory round trips.  The weights come
// from a copy in MFMA fragment order (launch_wfrag): one fragment load reads
// 1 KB contiguous instead of 16 rows x 64 bytes, half of each cache line,
// which made the projections 8-24% faster.  Here a workgroup
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
// Only active tiles get workgroups, dealt to the XCDs in equal runs that
// walk the row tiles of a column tile together (shared weight tiles in L2).
#include <algorithm>

#include "kernels.h"

namespace tlf {

namespace {

__device__ __forceinline__ unsigned int ordered_bits(float v) {
  unsigned int u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kXcds = 8;

// Shared-memory scratch of one workgroup, sized by the caller for the larger shape.
struct DgemmShared {
  float* red;       // [SLOTS][BM * (BN + 1)] partial tiles
  float* ss;        // [W][BM] partial sums of squares
  float* inv;       // [BM] 1 / rms per row
  int* orow;        // [BM] logits row of each tile row
  int64_t* kv;      // [BM] cache slot offset of each tile row (-1: no cache entry)
  int* keep;        // [BM] E_RESID: the row's result is stored
  int* moff;        // [BM] E_RESID with a gate: the row's modulation row offset
};

// depth of row r for the AdaLN table (valid for active rows only)
__device__ __forceinline__ int mod_row_depth(const GemmArgs& g, int r) {
  return g.mod_depth[g.mod_by_src ? row_src(g.rm, r) : r];
}

template <typename T, int RM, int CN, int W, int KB, int AK, int EK, bool NORM, bool MOD>
__device__ __forceinline__ void dgemm_tile(const GemmArgs& g, int act_rows, const DgemmShared& sh) {
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

  float* red = sh.red;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int quad = lane >> 4, c16 = lane & 15;
  // Active tiles only (rows past the active count form no tile), dealt to
  // the XCDs in equal contiguous runs: workgroup L runs on XCD L mod 8 and
  // takes tile (L mod 8) * per + L / 8, so no XCD holds more than its share,
  // and a run walks the row tiles of one column tile before the next, which
  // keeps weight tiles shared in that XCD's L2.
  const int tiles_n = (g.N + BN - 1) / BN;
  const int RT = (act_rows + BM - 1) / BM, ntiles = RT * tiles_n, per = (ntiles + kXcds - 1) / kXcds;
  const int L = blockIdx.x, k = L / kXcds, t = (L % kXcds) * per + k;
  if (k >= per || t >= ntiles) return;
  const int tn = t / RT, tm = t % RT;
  const int r0 = tm * BM, n0 = tn * BN;

  // Loads go out before any loaded value is used: the epilogue's bookkeeping
  // and residual values and the weight fragments of the first K batch (they
  // depend on the tile only), then the activation fragments (after the row
  // permutation for A_SRC).  The bookkeeping is kept in registers and written
  // to LDS after the products, so that no use of it makes a wave wait before
  // the weights are in flight.  With g.spec (every row active, e.g. the
  // first loop) the tiles and loads do not wait for the active-row count;
  // otherwise the count decides the tiles first, and activation rows past it
  // are not loaded.
  const int a_rows = act_rows;  // activation rows worth loading
  // 32-bit element offsets from uniform bases (the weight and activation
  // matrices hold fewer than 2^31 elements)
  // weight fragment (c, K step j) at Wb + wo[c] + j * wstep: row-major W, or
  // the fragment-ordered copy, where one load reads 64 x 16 contiguous bytes
  const int S = g.K / KS;  // K steps
  const T* Wb = reinterpret_cast<const T*>(g.Wf ? g.Wf : g.W);
  const int wstep = g.Wf ? kWave * EPL : KS;
  int wo[CN];
#pragma unroll
  for (int c = 0; c < CN; ++c) {
    if (g.Wf) {
      const int blk = min((n0 + c * 16) / 16, (g.N + 15) / 16 - 1);
      wo[c] = (blk * S * kWave + lane) * EPL;
    } else {
      int n = n0 + c * 16 + c16, wr = n;
      if constexpr (EK == E_SWIGLU) {
        // interleaved 32-column groups: 16 gate columns, then the 16 up columns of the same units
        const int grp = n >> 5, k = n & 31;
        wr = (k < 16) ? grp * 16 + k : g.F + grp * 16 + (k - 16);
      }
      wr = min(wr, g.w_rows - 1);
      wo[c] = wr * g.K + quad * EPL;
    }
  }
  // the wave's K steps of batch jb (past the wave's last step the last step
  // is reread; its product is skipped)
  Frag bw[KB][CN];
  auto load_weights = [&](int jb) {
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      const int st = min(w + W * (jb + j), S - 1);
#pragma unroll
      for (int c = 0; c < CN; ++c) bw[j][c] = M::load(Wb + (wo[c] + st * wstep));
    }
  };
  // bookkeeping of the tile's rows (lanes of quad 0 in wave 0, one row per
  // lane and row fragment; rows past the batch read its last row) and the
  // residual value of each output
  const bool bk_lane = w == 0 && quad == 0;
  int64_t bk_kv[EK == E_QKV ? RM : 1];       // cache slot offset (-1: no cache entry)
  int bk_keep[EK == E_RESID ? RM : 1];       // depth the row is kept below (keep_depth)
  int bk_depth[EK == E_RESID ? RM : 1];      // modulation depth
  int bk_orow[EK == E_LOGITS ? RM : 1];      // logits row
  float xr[EK == E_RESID ? EPT : 1];
  int xrow[EK == E_RESID ? EPT : 1];  // residual row of each output (scatter: src(r))
  auto load_epilogue_values = [&]() {
    if (bk_lane) {
#pragma unroll
      for (int i = 0; i < RM; ++i) {
        const int rl = i * 16 + c16, r = min(r0 + rl, g.rm.rows - 1);
        if constexpr (EK == E_QKV) bk_kv[i] = g.kv.slot_base[r];
        if constexpr (EK == E_RESID) {
          bk_keep[i] = g.keep_depth ? g.keep_depth[r] : INT_MAX;
          bk_depth[i] = g.mod_a && r0 + rl < a_rows ? mod_row_depth(g, r) : 1;
        }
        if constexpr (EK == E_LOGITS) bk_orow[i] = g.rm.src ? g.rm.src[r] : g.out_row_off + r;
      }
    }
    if constexpr (EK == E_RESID) {
      // every output's residual value is loaded (rows past those worth
      // loading and columns past the matrix read its last such row or
      // column; the epilogue stores active outputs only), so no load waits on
      // a lane's condition
#pragma unroll
      for (int k = 0; k < EPT; ++k) {
        const int e = tid + k * NT, row = min(r0 + e / BN, a_rows - 1), n = min(n0 + e % BN, g.N - 1);
        xrow[k] = g.scatter ? row_src(g.rm, row) : row;
        xr[k] = g.out[g.out_frag ? frag_index<T>(xrow[k], n, g.N) : (int64_t)xrow[k] * g.ldo + n];
      }
    }
  };
  int nact = g.rm.rows;  // active rows, read with the first K batch
  // the residual projections load these before their weights, the others
  // with their first K batch (measured: each order is the faster one for
  // its projections)
  constexpr bool kEpilogueFirst = EK == E_RESID;
  if constexpr (kEpilogueFirst) load_epilogue_values();
  load_weights(0);

  const float* Ab = g.A;
  int ao[RM];
#pragma unroll
  for (int i = 0; i < RM; ++i) {
    const int r = min(r0 + i * 16 + c16, g.rm.rows - 1);
    const int arow = (AK == A_SRC) ? row_src(g.rm, r) : r;
    ao[i] = g.a_frag ? ((arow >> 4) * S * kWave + quad * 16 + (arow & 15)) * EPL : arow * g.lda + quad * EPL;
  }
  // MOD: the lane's rows are scaled by (1 + gamma) of their modulation rows
  int go[MOD ? RM : 1];
  if constexpr (MOD) {
#pragma unroll
    for (int i = 0; i < RM; ++i) {
      const int r = r0 + i * 16 + c16;
      go[i] = (r < a_rows ? (mod_row_depth(g, r) - 1) * g.mod_ld : 0) + quad * EPL;
    }
  }


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
    float gv[MOD ? KB : 1][RM][EPL];
    if (jb > 0) load_weights(jb);
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      const int stj = min(w + W * (jb + j), S - 1);
      const int k0 = stj * KS, ka = stj * (g.a_frag ? kWave * EPL : KS);
#pragma unroll
      for (int i = 0; i < RM; ++i) {
#pragma unroll
        for (int e = 0; e < EPL; ++e) av[j][i][e] = 0.f;
        if constexpr (MOD) {
#pragma unroll
          for (int e = 0; e < EPL; ++e) gv[j][i][e] = 0.f;
        }
        if (r0 + i * 16 >= a_rows) continue;  // uniform: the fragment's rows have exited
        if (r0 + i * 16 + c16 < a_rows) {
          if constexpr (EPL == 8) {
            const float4 lo = *reinterpret_cast<const float4*>(Ab + (ao[i] + ka));
            const float4 hi = *reinterpret_cast<const float4*>(Ab + (ao[i] + ka + 4));
            av[j][i][0] = lo.x; av[j][i][1] = lo.y; av[j][i][2] = lo.z; av[j][i][3] = lo.w;
            av[j][i][4] = hi.x; av[j][i][5] = hi.y; av[j][i][6] = hi.z; av[j][i][7] = hi.w;
            if constexpr (MOD) {
              const float4 glo = *reinterpret_cast<const float4*>(g.mod_g + (go[i] + k0));
              const float4 ghi = *reinterpret_cast<const float4*>(g.mod_g + (go[i] + k0 + 4));
              gv[j][i][0] = glo.x; gv[j][i][1] = glo.y; gv[j][i][2] = glo.z; gv[j][i][3] = glo.w;
              gv[j][i][4] = ghi.x; gv[j][i][5] = ghi.y; gv[j][i][6] = ghi.z; gv[j][i][7] = ghi.w;
            }
          } else {
            av[j][i][0] = Ab[ao[i] + ka];
            if constexpr (MOD) gv[j][i][0] = g.mod_g[go[i] + k0];
          }
        }
      }
    }
    if (jb == 0) {
      if constexpr (!kEpilogueFirst) load_epilogue_values();
      if (g.rm.nact) nact = *g.rm.nact;
      if (r0 >= nact) return;  // uniform: the tile's rows have all exited
    }
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
            float* dst = g.a_copy + (g.copy_frag ? frag_index<T>(r, k0 + quad * EPL, g.K)
                                                  : (int64_t)r * g.lda + k0 + quad * EPL);
#pragma unroll
            for (int e = 0; e < EPL; ++e) dst[e] = av[j][i][e];
          }
        }
        if constexpr (NORM) {
#pragma unroll
          for (int e = 0; e < EPL; ++e) ss[i] = fmaf(av[j][i][e], av[j][i][e], ss[i]);
        }
        if constexpr (MOD) {
          // RMSNorm(x) (1 + gamma): the norm's sum of squares above takes x itself
#pragma unroll
          for (int e = 0; e < EPL; ++e) av[j][i][e] *= 1.f + gv[j][i][e];
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

  if (bk_lane) {
#pragma unroll
    for (int i = 0; i < RM; ++i) {
      const int rl = i * 16 + c16;
      if constexpr (EK == E_QKV) sh.kv[rl] = bk_kv[i];
      if constexpr (EK == E_RESID) {
        sh.keep[rl] = bk_keep[i] > g.keep_loop;
        sh.moff[rl] = (bk_depth[i] - 1) * g.mod_ld;
      }
      if constexpr (EK == E_LOGITS) sh.orow[rl] = bk_orow[i];
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
          for (int r = 0; r < 4; ++r) red[(w - SLOTS) * BM * LDR + (i * 16 + quad * 4 + r) * LDR + c * 16 + c16] = acc[i][c][r];
    }
    __syncthreads();
    if (w < SLOTS) {
#pragma unroll
      for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int c = 0; c < CN; ++c)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[i][c][r] += red[w * BM * LDR + (i * 16 + quad * 4 + r) * LDR + c * 16 + c16];
    }
    __syncthreads();
  }
  if (w < SLOTS) {
#pragma unroll
    for (int i = 0; i < RM; ++i)
#pragma unroll
      for (int c = 0; c < CN; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[w * BM * LDR + (i * 16 + quad * 4 + r) * LDR + c * 16 + c16] = acc[i][c][r];
  }
  if constexpr (NORM) {
#pragma unroll
    for (int i = 0; i < RM; ++i) {
      float t = ss[i];
      t += shfl_xor(t, 16);
      t += shfl_xor(t, 32);
      if (quad == 0) sh.ss[w * BM + i * 16 + c16] = t;
    }
  }
  __syncthreads();
  if constexpr (NORM) {
    if (tid < BM) {
      float t = 0.f;
#pragma unroll
      for (int ww = 0; ww < W; ++ww) t += sh.ss[ww * BM + tid];
      sh.inv[tid] = rsqrtf(t / (float)g.K + g.eps);
    }
    __syncthreads();
  }
  auto tile_sum = [&](int row, int col) -> float {
    float v = 0.f;
#pragma unroll
    for (int ww = 0; ww < SLOTS; ++ww) v += red[ww * BM * LDR + row * LDR + col];
    if constexpr (NORM) v *= sh.inv[row];
    return v;
  };
  const int row_end = min(g.rm.rows, nact);  // rows [r0, row_end) are active

  if constexpr (EK == E_QKV) {
    // Eight consecutive columns per thread: they lie in one of q, k and v and
    // in one head (d and D are multiples of 16), so the part and head are
    // resolved once per group; q goes out as two 16-byte stores, a bf16 k run
    // as one (eight consecutive dimensions of a slot are adjacent in fragment
    // order), v as eight elements four apart ([slot / 4][D][slot % 4]).
    static_assert(BN % 8 == 0, "column groups");
    T* pool = reinterpret_cast<T*>(g.kv.c.pool);
    for (int e8 = tid; e8 < BM * BN / 8; e8 += NT) {
      const int row = e8 / (BN / 8), col = (e8 % (BN / 8)) * 8, n = n0 + col;
      if (r0 + row >= row_end || n >= g.N) continue;
      float v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = tile_sum(row, col + j);
      if (n < g.d) {
        float* q = g.out + (int64_t)(r0 + row) * g.ldo + n;
        *reinterpret_cast<float4*>(q) = make_float4(v[0], v[1], v[2], v[3]);
        *reinterpret_cast<float4*>(q + 4) = make_float4(v[4], v[5], v[6], v[7]);
        continue;
      }
      const int64_t base = sh.kv[row];
      if (base < 0) continue;
      const int slot = (int)(base & (kPage - 1));
      const int64_t page = base - slot;
      const bool is_v = n - g.d >= g.d;
      const int within = n - g.d - (is_v ? g.d : 0);
      const int h = within / g.kv.c.D, el = within - h * g.kv.c.D;
      if (!is_v) {
        if constexpr (sizeof(T) == 2) {
          *reinterpret_cast<uint4*>(pool + page + k_block(g.kv.c, g.kv.layer, h) + k_frag_off<T>(slot, el)) =
              make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                         pack_bf16x2(v[6], v[7]));
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j)
            pool[page + k_block(g.kv.c, g.kv.layer, h) + k_frag_off<T>(slot, el + j)] = from_f<T>(v[j]);
        }
      } else {
        T* dst = pool + page + v_block(g.kv.c, g.kv.layer, h) + v_frag_off(slot, el, g.kv.c.D);
#pragma unroll
        for (int j = 0; j < 8; ++j) dst[4 * j] = from_f<T>(v[j]);
      }
    }
    return;
  }

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
      const int R = r0 + row;
      const int64_t o = g.out_frag ? ((int64_t)((R >> 4) * (g.F / KS) + unit / KS) * kWave +
                                      (unit % KS) / EPL * 16 + (R & 15)) * EPL + unit % EPL
                                   : (int64_t)R * g.ldo + unit;
      g.out[o] = gt / (1.f + __expf(-gt)) * up;
    } else if constexpr (EK == E_LOGITS) {
      const int row = e / BN, n = n0 + e % BN;
      const bool ok = r0 + row < row_end && n < g.N;
      const int orow = sh.orow[row];
      unsigned long long key = 0ull;
      if (ok) {
        const float v = tile_sum(row, e % BN);
        g.out[(int64_t)orow * g.ldo + n] = v;
        key = ((unsigned long long)ordered_bits(v) << 32) | (unsigned long long)(0xFFFFFFFFu - (unsigned)n);
      }
      if (g.argmax_keys) {
        // the 64 lanes of a wave hold one row's 64 columns: one key per group
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
          const unsigned long long other = shfl_xor(key, o);
          key = other > key ? other : key;
        }
        if (lane == 0 && key != 0ull) g.argmax_keys[(int64_t)orow * g.key_groups + n0 / kWave] = key;
      }
    } else {
      const int row = e / BN, col = e % BN, n = n0 + col;
      if (r0 + row >= row_end || n >= g.N) continue;
      const float v = tile_sum(row, col);
      if constexpr (EK == E_RESID) {
        if (sh.keep[row]) {
          const float gate = g.mod_a ? 1.f + g.mod_a[sh.moff[row] + n] : 1.f;
          g.out[g.out_frag ? frag_index<T>(xrow[k], n, g.N) : (int64_t)xrow[k] * g.ldo + n] = xr[k] + gate * v;
        }
      } else if constexpr (EK == E_HIDDEN) {
        const float u = v + g.bias[n];
        g.out[(int64_t)(r0 + row) * g.ldo + n] = u / (1.f + __expf(-u));
      }
    }
  }
}

// One kernel, two tile shapes: the wide shape when more than `wide_above`
// rows are active (the narrow shape would need more than one workgroup per
// compute unit), the narrow shape otherwise.  The choice is uniform over the
// grid and made from the active-row count the tiles need anyway.
template <int RM, int CN> struct Shape {
  static constexpr int BM = RM * 16, BN = CN * 16;
};

template <typename T, int RMn, int CNn, int RMw, int CNw, int W, int KB, int AK, int EK, bool NORM, bool MOD>
__global__ __launch_bounds__(W * 64) void k_dgemm(GemmArgs g, int wide_above) {
  constexpr int SLOTS = W > 8 ? 8 : W;
  constexpr int BMX = RMn > RMw ? RMn * 16 : RMw * 16;
  constexpr int REDN = SLOTS * RMn * 16 * (CNn * 16 + 1), REDW = SLOTS * RMw * 16 * (CNw * 16 + 1);
  __shared__ float red[REDN > REDW ? REDN : REDW];
  __shared__ float s_ss[NORM ? W * BMX : 1];
  __shared__ float s_inv[BMX];
  __shared__ int s_orow[EK == E_LOGITS ? BMX : 1];
  __shared__ int64_t s_kv[EK == E_QKV ? BMX : 1];
  __shared__ int s_keep[EK == E_RESID ? BMX : 1];
  __shared__ int s_moff[EK == E_RESID ? BMX : 1];
  const DgemmShared sh{red, s_ss, s_inv, s_orow, s_kv, s_keep, s_moff};
  const int act_rows = g.spec ? g.rm.rows : min(g.rm.nact ? *g.rm.nact : g.rm.rows, g.rm.rows);
  if constexpr (RMn != RMw || CNn != CNw) {
    if (act_rows > wide_above) {
      dgemm_tile<T, RMw, CNw, W, KB, AK, EK, NORM, MOD>(g, act_rows, sh);
      return;
    }
  }
  dgemm_tile<T, RMn, CNn, W, KB, AK, EK, NORM, MOD>(g, act_rows, sh);
}

template <typename T, int RMn, int CNn, int RMw, int CNw, int W, int KB, int AK, int EK, bool NORM, bool MOD>
hipError_t launch_cfg(const GemmArgs& a, int cus, hipStream_t s) {
  constexpr int BMn = RMn * 16, BNn = CNn * 16, BMw = RMw * 16, BNw = CNw * 16;
  const int tn_n = (a.N + BNn - 1) / BNn, tm_n = (a.rm.rows + BMn - 1) / BMn;
  const int tn_w = (a.N + BNw - 1) / BNw, tm_w = (a.rm.rows + BMw - 1) / BMw;
  if (tn_n == 0 || tm_n == 0) return hipSuccess;
  // wide above the row count at which the narrow tiles exceed one per compute unit
  const int wide_above = (RMn == RMw && CNn == CNw) ? a.rm.rows : std::max(1, cus / tn_n) * BMn;
  // workgroups for the larger of the two shapes' tile counts; the narrow
  // shape never runs on more than wide_above rows.  No workgroup beyond
  // that: a workgroup past one per compute unit waits for a free one only
  // to find no tile, and the launch is not over until it has run
  const int tiles = std::max(tn_n * std::min(tm_n, (wide_above + BMn - 1) / BMn), tn_w * tm_w);
  const int grid = kXcds * ((tiles + kXcds - 1) / kXcds);
  hipLaunchKernelGGL((k_dgemm<T, RMn, CNn, RMw, CNw, W, KB, AK, EK, NORM, MOD>), dim3(grid), dim3(W * 64), 0, s, a,
                     wide_above);
  return hipGetLastError();
}

// K steps per wave in one batch of loads: all of a wave's steps when they
// fit in KBMAX, else batches of KBMAX.
template <typename T, int RMn, int CNn, int RMw, int CNw, int W, int KBMAX, int AK, int EK, bool NORM,
          bool MOD = false>
hipError_t launch_w(const GemmArgs& a, int cus, hipStream_t s) {
  const int nj = (a.K / Mfma<T>::KS + W - 1) / W;
  if (nj <= 2 || KBMAX == 2) return launch_cfg<T, RMn, CNn, RMw, CNw, W, 2, AK, EK, NORM, MOD>(a, cus, s);
  if (nj <= 3 || KBMAX == 3)
    return launch_cfg<T, RMn, CNn, RMw, CNw, W, (KBMAX >= 3 ? 3 : 2), AK, EK, NORM, MOD>(a, cus, s);
  return launch_cfg<T, RMn, CNn, RMw, CNw, W, (KBMAX >= 4 ? 4 : 2), AK, EK, NORM, MOD>(a, cus, s);
}

}  // namespace

// Tile shapes (rows x columns, waves), measured on the projections of a
// 256-row batch; each kernel holds a narrow shape and a wide one and picks
// the wide one when the narrow tiles would need more than one workgroup per
// compute unit.
//   QKV:     32 x 64 | 32 x 80   (8 waves)
//   gate/up: 32 x 64 | 32 x 128  (8 waves)
//   O:       32 x 32             (8 waves)
//   down:    16 x 32 | 16 x 48   (16 waves)  [K > 768 in bf16; else as O]
//   LM head: 32 x 64             (8 waves)
//   router hidden layer: 32 x 32 (8 waves)
template <typename T>
hipError_t launch_dgemm(const GemmArgs& a, AKind ak, EKind ek, bool norm, int cus, hipStream_t s) {
  if (a.K <= 0 || a.K % Mfma<T>::KS != 0 || a.rm.rows <= 0 || cus <= 0) return hipErrorInvalidValue;
  if (a.a_frag && (ak != A_CMP || a.a_copy)) return hipErrorInvalidValue;
  if (a.copy_frag && !a.a_copy) return hipErrorInvalidValue;
  if (a.out_frag && !((ek == E_SWIGLU && a.F % Mfma<T>::KS == 0) || (ek == E_RESID && !a.scatter)))
    return hipErrorInvalidValue;
  const bool mod = a.mod_g != nullptr;
  if (ek == E_QKV && norm) {
    if (ak == A_SRC)
      return mod ? launch_w<T, 2, 4, 2, 5, 8, 3, A_SRC, E_QKV, true, true>(a, cus, s)
                 : launch_w<T, 2, 4, 2, 5, 8, 3, A_SRC, E_QKV, true>(a, cus, s);
    return mod ? launch_w<T, 2, 4, 2, 5, 8, 3, A_CMP, E_QKV, true, true>(a, cus, s)
               : launch_w<T, 2, 4, 2, 5, 8, 3, A_CMP, E_QKV, true>(a, cus, s);
  }
  if (ek == E_SWIGLU && norm) {
    // with the gamma operands, two K batches in flight (three would spill)
    if (ak == A_SRC)
      return mod ? launch_w<T, 2, 4, 2, 8, 8, 2, A_SRC, E_SWIGLU, true, true>(a, cus, s)
                 : launch_w<T, 2, 4, 2, 8, 8, 3, A_SRC, E_SWIGLU, true>(a, cus, s);
    return mod ? launch_w<T, 2, 4, 2, 8, 8, 2, A_CMP, E_SWIGLU, true, true>(a, cus, s)
               : launch_w<T, 2, 4, 2, 8, 8, 3, A_CMP, E_SWIGLU, true>(a, cus, s);
  }
  if (mod) return hipErrorInvalidValue;  // the operand scale is for the normalised projections
  if (ek == E_LOGITS && norm) {
    if (ak == A_SRC) return launch_w<T, 2, 4, 2, 4, 8, 3, A_SRC, E_LOGITS, true>(a, cus, s);
    return launch_w<T, 2, 4, 2, 4, 8, 3, A_CMP, E_LOGITS, true>(a, cus, s);
  }
  if (ak == A_CMP && ek == E_HIDDEN && !norm) return launch_w<T, 2, 2, 2, 2, 8, 3, A_CMP, E_HIDDEN, false>(a, cus, s);
  if (ak == A_CMP && ek == E_RESID && !norm) {
    if (a.K / Mfma<T>::KS > 3 * 8) return launch_w<T, 1, 2, 1, 3, 16, 4, A_CMP, E_RESID, false>(a, cus, s);
    return launch_w<T, 2, 2, 2, 2, 8, 3, A_CMP, E_RESID, false>(a, cus, s);
  }
  return hipErrorInvalidValue;
}

template hipError_t launch_dgemm<float>(const GemmArgs&, AKind, EKind, bool, int, hipStream_t);
template hipError_t launch_dgemm<bf16>(const GemmArgs&, AKind, EKind, bool, int, hipStream_t);

namespace {

template <typename T>
__global__ __launch_bounds__(256) void k_wfrag(const T* W, T* Wf, int N, int K, int F, int64_t total) {
  constexpr int KS = Mfma<T>::KS, EPL = Mfma<T>::EPL;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;  // (blk, step, lane)
  if (i >= total) return;
  const int S = K / KS;
  const int lane = (int)(i % kWave);
  const int64_t bs = i / kWave;
  const int step = (int)(bs % S), blk = (int)(bs / S);
  const int n = blk * 16 + (lane & 15);
  int row = n;
  if (F > 0) {
    const int grp = n >> 5, k = n & 31;
    row = (k < 16) ? grp * 16 + k : F + grp * 16 + (k - 16);
  }
  const T* src = W + (int64_t)row * K + step * KS + (lane >> 4) * EPL;
  T* dst = Wf + i * EPL;
#pragma unroll
  for (int e = 0; e < EPL; ++e) dst[e] = src[e];
}

}  // namespace

template <typename T>
hipError_t launch_wfrag(const void* W, void* Wf, int N, int K, int swiglu_F, hipStream_t s) {
  if (N <= 0 || N % 16 != 0 || K % Mfma<T>::KS != 0 || (swiglu_F > 0 && N != 2 * swiglu_F)) return hipErrorInvalidValue;
  const int64_t total = (int64_t)(N / 16) * (K / Mfma<T>::KS) * kWave;
  hipLaunchKernelGGL(k_wfrag<T>, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, reinterpret_cast<const T*>(W),
                     reinterpret_cast<T*>(Wf), N, K, swiglu_F, total);
  return hipGetLastError();
}
template hipError_t launch_wfrag<float>(const void*, void*, int, int, int, hipStream_t);
template hipError_t launch_wfrag<bf16>(const void*, void*, int, int, int, hipStream_t);

}  // namespace tlf
