// MFMA GEMM for the prefill projections and LM head (many rows per launch).
//
// out = A W^T on the active rows of a row map, with W [N][K] row-major
// (linear-layer layout) in the storage dtype and A float32, either the
// normalised residual rows y[src(r)] (A_SRC) or compact rows buf[r] (A_CMP).
// With bf16 weights every A tile is split into bf16 hi and lo parts in LDS
// and each product runs once per part, so the activations keep about 16
// significant bits; the weights are exact in bf16.  With a_single the A tile
// is rounded to one bf16 part instead (half the products).
// Epilogues:
//   E_QKV:     q to a buffer; k, v appended to the loop's cache pages (Eq. 11)
//   E_RESID:   x[src(r)] += result (residual of the attention/FFN branch)
//   E_SWIGLU:  act = silu(gate) * up, gate/up columns interleaved in 16-column
//              groups so every wave holds matching pairs
//   E_LOGITS:  float logits plus a packed (value, -index) greedy key per 64 columns;
//              compact rows (A_CMP, the decode LM head) go to row src(r)
//   E_HIDDEN:  silu(result + bias), the MLP router's hidden layer
//
// Tiling: 256 threads = 4 waves in a 2 x 2 grid, a 128 x 256 output tile
// per workgroup (64 x 128 per wave; 128 x 128 when there are few row tiles;
// the down projection of many rows: 8 waves in a 4 x 2 grid, 256 x 256).  K
// advances 32 elements per tile.  Float A: through two LDS stages, the next
// tile's global loads in flight while the current one is multiplied, then
// converted and stored to the other stage (one barrier per tile).  bf16 A
// rows: A and W copied into LDS by the loads themselves, three stages, two
// tiles in flight (one wait and barrier per tile).  LDS rows are
// XOR-swizzled by 16-byte chunk instead of padded, so two workgroups fit on
// a compute unit.
#include "kernels.h"

namespace tlf {

namespace {

// Each wave kGemmMT x NT MFMA tiles of 16 x 16 (64 rows x 128 or 64
// columns), K kGemmBK at a time.
constexpr int kGemmMT = 4, kGemmBK = 32;

__device__ __forceinline__ unsigned int ordered_bits(float v) {
  unsigned int u = __float_as_uint(v);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// 4 x 4 transpose inside each group of four lanes: lane t of the group holds
// v[r] = (row r, column t) of a 4 x 4 block on entry and (row t, column r) on
// return, so an accumulator tile's four consecutive columns of one row meet
// in one lane (one 16-byte access instead of four 4-byte ones).
__device__ __forceinline__ void transpose4(float& v0, float& v1, float& v2, float& v3, int t) {
  float a = (t & 1) ? v0 : v1, b = (t & 1) ? v2 : v3;
  a = shfl_xor(a, 1);
  b = shfl_xor(b, 1);
  if (t & 1) { v0 = a; v2 = b; } else { v1 = a; v3 = b; }
  a = (t & 2) ? v0 : v2;
  b = (t & 2) ? v1 : v3;
  a = shfl_xor(a, 2);
  b = shfl_xor(b, 2);
  if (t & 2) { v0 = a; v1 = b; } else { v2 = a; v3 = b; }
}

// 16-byte chunk c of LDS row `row` is stored at chunk c ^ key(row): the 16
// rows that one MFMA fragment read touches land in distinct banks without
// padding (bf16 rows of 32 elements hold 4 chunks, float rows 8).
template <typename T> __device__ __forceinline__ int swz(int row, int c) {
  if constexpr (sizeof(T) == 2) return c ^ ((row >> 2) & 3);
  else return c ^ (row & 7);
}

// LDS byte address of a shared-memory pointer
__device__ __forceinline__ unsigned lds_addr(void* p) {
  return (unsigned)(uintptr_t)(__attribute__((address_space(3))) void*)p;
}

// 16 bytes from global memory straight into LDS: the wave's 64 lanes fill 64
// consecutive 16-byte chunks from byte `lds` (wave-uniform, passed in M0).
// Written as assembly so that the compiler's wait-count pass, which would
// otherwise wait for every such load before any later LDS read, leaves the
// ordering to wait_loads_barrier; it counts toward vmcnt like any load.
__device__ __forceinline__ void load_lds16(const void* g, unsigned lds) {
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(lds) : "memory");
}

// Waits until at most N vector-memory loads of this wave are outstanding,
// then joins the workgroup barrier.  The memory clobber keeps the compiler
// from moving LDS accesses across it.
template <int N> __device__ __forceinline__ void wait_loads_barrier() {
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(N) : "memory");
}

// MOD: the A rows are scaled by (1 + gamma) of their AdaLN modulation rows.
// NORM: A holds residual rows x and the product is taken with RMSNorm(x): the
// sum of squares of each row is accumulated from the A chunks as they pass
// and the output row is scaled by 1 / rms, since (x / rms) W^T = (x W^T) / rms.
// AMODE (bf16 weights): 0: float A enters the MFMA as hi + lo parts; 1: as
// one bf16 part (round to nearest even), half the products and LDS traffic;
// 2: A is read as bf16 rows (g.A16), half the A bytes as well, and A and W
// are copied into LDS by the loads themselves (global_load_lds: no
// registers, no LDS stores), through NSTD LDS stages so that NSTD - 1 K tiles
// are in flight while one is multiplied.  Float32 weights take float A
// (AMODE 0).
// WM: waves along M (2 or 4; two along N), each wave MT x NT MFMA tiles.
// MT x NT: each wave's 16 x 16 MFMA tiles; BK: K elements per LDS stage.
template <typename T, int MT, int NT, int BK, int AK, int EK, bool MOD, bool NORM, int AMODE, int WM, int NSTD>
__device__ __forceinline__ void gemm_tile(const GemmArgs& g, const int r0, const int n0, void* as_lds, void* bs_lds,
                                          int* row_src_s, int* row_mod_s, float* row_inv_s, int64_t* kv_base) {
  constexpr int NTH = WM * 128;                      // threads: WM x 2 waves
  constexpr int BM = WM * MT * 16, BN = 2 * NT * 16;
  constexpr bool kBf16 = sizeof(T) == 2;             // bf16 weights: A converted to bf16 in LDS
  constexpr bool kSplit = kBf16 && AMODE == 0;       // ... as hi + lo parts
  constexpr bool kDirect = kBf16 && AMODE == 2;      // bf16 A rows; A and W copied to LDS by their loads
  constexpr int NST = kDirect ? NSTD : 2;            // LDS stages
  static_assert(!kDirect || (!MOD && !NORM), "bf16 A rows carry no modulation or norm");
  constexpr int NA = kSplit ? 2 : 1;
  constexpr int CE = 16 / (int)sizeof(T);            // storage elements per 16-byte chunk
  constexpr int WCR = BK / CE;                       // weight chunks per row per K tile
  constexpr int ACR = kDirect ? BK / CE : BK / 4;   // A chunks (8 bf16 or 4 floats) per row per K tile
  using M = Mfma<T>;
  constexpr int KS = M::KS, EPL = M::EPL;
  constexpr int ACH = BM * ACR / NTH;                // A chunks per thread
  constexpr int BCH = BN * WCR / NTH;                // B chunks per thread
  static_assert(ACH >= 1 && BM * ACR % NTH == 0, "A tile split");
  static_assert(BCH >= 1 && BN * WCR % NTH == 0, "B tile split");
  static_assert(BK % KS == 0 && (KS * (int)sizeof(T)) % 16 == 0 || EPL == 1, "K tile");

  // the workgroup's LDS: operand stages, and per tile row its source row,
  // modulation row offset (AdaLN, 0 without), 1 / rms and cache slot
  auto& As = *reinterpret_cast<T (*)[NST][NA][BM * BK]>(as_lds);
  auto& Bs = *reinterpret_cast<T (*)[NST][BN * BK]>(bs_lds);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // decode: a tile whose first row has exited is empty (rows are depth-sorted)
  if (g.rm.nact && r0 >= *g.rm.nact) return;
  // prefill: segments of seg slots with active prefixes; a tile inside one
  // segment that starts past its active count is empty (most tiles of the
  // later loops): leave before resolving rows
  if (g.rm.seg_cnt && r0 % g.rm.seg + BM <= g.rm.seg &&
      r0 % g.rm.seg >= g.rm.seg_cnt[(r0 / g.rm.seg) * g.rm.seg_cnt_stride])
    return;

  // W row of output column n (clamped; columns >= N are never stored)
  auto w_row = [&](int n) -> int {
    int wr = n;
    if constexpr (EK == E_SWIGLU) {
      const int grp = n >> 5, w = n & 31;
      wr = (w < 16) ? grp * 16 + w : g.F + grp * 16 + (w - 16);
    }
    return wr < g.w_rows ? wr : g.w_rows - 1;
  };

  float4 ra[kDirect ? 1 : ACH];
  float4 rg[MOD ? ACH : 1];  // gamma of the A chunks in flight
  V16<T> rb[kDirect ? 1 : BCH];
  const float* A = reinterpret_cast<const float*>(g.A);
  const T* A16 = reinterpret_cast<const T*>(g.A16);
  const T* W = reinterpret_cast<const T*>(g.W);
  const int KT = g.K / BK;

  // chunk u of thread t: A row (t + NTH u) / ACR, floats 4 ((t + NTH u) % ACR)
  // .. + 3; W row (t + NTH u) / WCR, chunk (t + NTH u) % WCR
  auto load_b = [&](int kt) {
    if constexpr (kDirect) return;
    const int kk = kt * BK;
#pragma unroll
    for (int c = 0; c < (kDirect ? 0 : BCH); ++c) {
      const int ch = tid + c * NTH, row = ch / WCR, col = (ch % WCR) * CE;
      rb[c] = ld16(W + (int64_t)w_row(n0 + row) * g.K + kk + col);
    }
  };
  auto load_a = [&](int kt) {
    const int kk = kt * BK;
    if constexpr (kDirect) return;
#pragma unroll
    for (int c = 0; c < ACH; ++c) {
      const int ch = tid + c * NTH, row = ch / ACR, col = (ch % ACR) * 4;
      const int s = row_src_s[row];
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f), gm = v;
      if (s >= 0) {
        const int64_t ar = (AK == A_SRC) ? (int64_t)s : (int64_t)(r0 + row);
        // fragment order (bf16 MFMA): the four floats lie in one run of EPL = 8
        v = *reinterpret_cast<const float4*>(A + (g.a_frag ? frag_index<T>((int)ar, kk + col, g.K)
                                                            : ar * g.lda + kk + col));
        if constexpr (MOD) gm = *reinterpret_cast<const float4*>(g.mod_g + row_mod_s[row] + kk + col);
      }
      ra[c] = v;
      if constexpr (MOD) rg[c] = gm;
    }
  };
  // NORM: this thread's rows are tid / ACR + c * (NTH / ACR), c < ACH
  float ssq[NORM ? ACH : 1];
#pragma unroll
  for (int c = 0; c < (NORM ? ACH : 1); ++c) ssq[c] = 0.f;
  auto store_tiles = [&](int st) {
#pragma unroll
    for (int c = 0; c < (kDirect ? 0 : ACH); ++c) {
      const int ch = tid + c * NTH, row = ch / ACR, f = ch % ACR;  // floats 4f .. 4f + 3 of the row
      float4 av = ra[c];
      if constexpr (NORM) ssq[c] += av.x * av.x + av.y * av.y + av.z * av.z + av.w * av.w;
      if constexpr (MOD)
        av = make_float4(av.x * (1.f + rg[c].x), av.y * (1.f + rg[c].y), av.z * (1.f + rg[c].z),
                         av.w * (1.f + rg[c].w));
      const int e = 4 * f;  // first element: chunk e / CE, offset e % CE
      T* dst = &As[st][0][row * BK + swz<T>(row, e / CE) * CE + e % CE];
      if constexpr (kSplit) {
        uint2 hi, lo;
        split4(av, hi, lo);
        *reinterpret_cast<uint2*>(dst) = hi;
        *reinterpret_cast<uint2*>(dst + BM * BK) = lo;  // As[st][1]
      } else if constexpr (kBf16) {
        *reinterpret_cast<uint2*>(dst) = make_uint2(pack_bf16x2(av.x, av.y), pack_bf16x2(av.z, av.w));
      } else {
        *reinterpret_cast<float4*>(dst) = av;
      }
    }
#pragma unroll
    for (int c = 0; c < (kDirect ? 0 : BCH); ++c) {
      const int ch = tid + c * NTH, row = ch / WCR, cc = ch % WCR;
      st16(&Bs[st][row * BK + swz<T>(row, cc) * CE], rb[c]);
    }
  };

  // AMODE 2: one load instruction of a wave fills 64 consecutive 16-byte
  // chunks of an LDS stage, lane l chunk l; so lane l fetches the chunk whose
  // swizzled place that is (the swizzle is an XOR, its own inverse).  A
  // thread's rows and chunks are the same in every K tile: their sources are
  // resolved once (no LDS read between the loads, which would have to wait
  // for them).  Rows without an active token read row 0 (never stored).
  const T* a_src[kDirect ? ACH : 1];
  const T* b_src[kDirect ? BCH : 1];
  const int wbase = __builtin_amdgcn_readfirstlane(tid & ~(kWave - 1));
  auto issue_b = [&](int kt, int st) __attribute__((always_inline)) {
    if constexpr (kDirect) {
#pragma unroll
      for (int c = 0; c < BCH; ++c)
        load_lds16(b_src[c] + kt * BK, lds_addr(&Bs[st][(c * NTH + wbase) * CE]));
    }
  };
  auto issue_a = [&](int kt, int st) __attribute__((always_inline)) {
    if constexpr (kDirect) {
#pragma unroll
      for (int c = 0; c < ACH; ++c)
        load_lds16(a_src[c] + kt * BK, lds_addr(&As[st][0][(c * NTH + wbase) * CE]));
    }
  };

  // the weight tiles do not depend on which rows are active: they go out
  // first (AMODE 2: those of the first NST - 1 K tiles, straight into their
  // stages)
  load_b(0);
  if constexpr (kDirect) {
#pragma unroll
    for (int c = 0; c < BCH; ++c) {
      const int q = tid + c * NTH, row = q / WCR;
      b_src[c] = W + (int64_t)w_row(n0 + row) * g.K + swz<T>(row, q % WCR) * CE;
    }
#pragma unroll
    for (int t = 0; t < NST - 1; ++t)
      if (t < KT) issue_b(t, t);
  }

  // thread t < BM resolves row r0 + t.  Its source row (and for QKV its
  // cache slot, consumed by the epilogue) is loaded together with the
  // activity test: both are in bounds for every row of the grid and are used
  // only for active rows.
  // The activity test of a tile that lies in one segment takes the
  // segment's count read for the empty-tile test above (uniform, no wait).
  int my_src = -1;
  int64_t my_kv = -1;
  if (tid < BM) {
    const int r = r0 + tid, rc = min(r, g.rm.rows - 1);
    const int src = row_src(g.rm, rc);
    if constexpr (EK == E_QKV) my_kv = g.kv.slot_base[rc];
    bool act;
    if (g.rm.seg_cnt && !g.rm.nact && r0 % g.rm.seg + BM <= g.rm.seg)
      act = r < g.rm.rows && r % g.rm.seg < g.rm.seg_cnt[(r0 / g.rm.seg) * g.rm.seg_cnt_stride];
    else
      act = row_active(g.rm, r);
    my_src = act ? src : -1;
    row_src_s[tid] = my_src;
    row_mod_s[tid] = (g.mod_depth && my_src >= 0)
                         ? (g.mod_depth[g.mod_by_src ? my_src : r] - 1) * g.mod_ld : 0;
  }
  if (!__syncthreads_or(my_src >= 0)) {
    // the weight loads into LDS complete before the workgroup gives up its LDS
    if constexpr (kDirect) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    return;
  }
  load_a(0);

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if constexpr (kDirect) {
#pragma unroll
    for (int c = 0; c < ACH; ++c) {
      const int q = tid + c * NTH, row = q / ACR;
      const int sr = row_src_s[row];
      const int64_t ar = sr < 0 ? 0 : (AK == A_SRC) ? (int64_t)sr : (int64_t)(r0 + row);
      a_src[c] = A16 + ar * g.lda + swz<T>(row, q % ACR) * CE;
    }
  }

  const int frow = lane & 15, quad = lane >> 4;
  auto multiply = [&](int st) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < BK / KS; ++ks) {
      const int k0 = ks * KS + quad * EPL;  // the lane's first element of this K step
      typename M::frag af[NA][MT], bfr[NT];
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const int row = wm * MT * 16 + i * 16 + frow;
        const int off = row * BK + swz<T>(row, k0 / CE) * CE + k0 % CE;
#pragma unroll
        for (int a = 0; a < NA; ++a) af[a][i] = M::load(&As[st][a][off]);
      }
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int row = wn * NT * 16 + j * 16 + frow;
        bfr[j] = M::load(&Bs[st][row * BK + swz<T>(row, k0 / CE) * CE + k0 % CE]);
      }
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
          for (int j = 0; j < NT; ++j) acc[i][j] = M::mma(af[a][i], bfr[j], acc[i][j]);
    }
  };
  if constexpr (kDirect) {
    // NST stages: tile kt + NST - 1 is fetched into the stage tile kt - 1
    // used while tile kt is multiplied.  Before the barrier a thread waits
    // for its own loads of tile kt (those of the up to NST - 2 later tiles,
    // the last LPT each, may stay in flight); after it every thread's tile kt
    // is in LDS and every wave is done reading tile kt - 1.
    // The weight tiles of K tiles 0 and 1 went out before the rows were
    // resolved, so the loads of tile 0 are complete once at most tile 1's A
    // loads are outstanding; from tile 1 on, a tile is complete once at most
    // the next tile's loads are.
    constexpr int LPT = ACH + BCH;  // loads per thread and tile
    static_assert(NST == 3, "stages: the weight tiles of the first two go out ahead");
    static_assert(LPT < 16, "vmcnt field");
#pragma unroll
    for (int t = 0; t < NST - 1; ++t)
      if (t < KT) issue_a(t, t);
    int st = 0;
    for (int kt = 0; kt < KT; ++kt) {
      if (kt + 1 >= KT) wait_loads_barrier<0>();
      else if (kt == 0) wait_loads_barrier<ACH>();
      else wait_loads_barrier<LPT>();
      if (kt + NST - 1 < KT) {
        const int sn = st == 0 ? NST - 1 : st - 1;
        issue_b(kt + NST - 1, sn);
        issue_a(kt + NST - 1, sn);
      }
      multiply(st);
      st = st == NST - 1 ? 0 : st + 1;
    }
    __syncthreads();
  } else {
    // double-buffered LDS: tile kt + 1 loads into registers while tile kt is
    // multiplied, then goes to the other stage; one barrier per tile
    store_tiles(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
      const int st = kt & 1;
      if (kt + 1 < KT) {
        load_b(kt + 1);
        load_a(kt + 1);
      }
      multiply(st);
      if (kt + 1 < KT) store_tiles(st ^ 1);
      __syncthreads();
    }
  }
  if constexpr (EK == E_QKV) {
    if (tid < BM) kv_base[tid] = my_src >= 0 ? my_kv : -1;
    __syncthreads();
  }
  if constexpr (NORM) {
    static_assert(NTH % ACR == 0 && ACR <= kWave, "rows of the A chunks");
    // the ACR threads of a row are consecutive lanes of one wave
#pragma unroll
    for (int c = 0; c < ACH; ++c) {
      float t = ssq[c];
#pragma unroll
      for (int o = 1; o < ACR; o <<= 1) t += shfl_xor(t, o);
      if (tid % ACR == 0) row_inv_s[tid / ACR + c * (NTH / ACR)] = rsqrtf(t / (float)g.K + g.eps);
    }
    __syncthreads();
  }

  const int col16 = lane & 15;
  if constexpr (EK == E_QKV) {
    // q to its buffer; k and v into the cache pages.  A 16-column tile lies
    // in one of q, k and v (d is a multiple of 16).  q and (bf16) k tiles go
    // through an in-group 4 x 4 transpose, after which lane t holds four
    // consecutive columns of row 4 quad + t: one 16-byte q store, or one
    // 8-byte k store (four dimensions of one slot are adjacent in the
    // fragment order).  A v tile keeps the lane's column: when its four rows
    // are consecutive slots of one page from a multiple of 4 (a fresh
    // prefill), their values of that dimension are one aligned run in the V
    // block and go out as one store; otherwise element by element.  The
    // tile's part, head and first dimension are resolved once per tile.
    T* pool = reinterpret_cast<T*>(g.kv.c.pool);
    const int t = col16 & 3;
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      // the 16-column tile's first column (wave-uniform), its part (0: q,
      // 1: k, 2: v), head and first dimension: one division per tile
      const int nt = n0 + wn * NT * 16 + j * 16;
      if (nt >= g.N) continue;
      const int part = nt < g.d ? 0 : nt < 2 * g.d ? 1 : 2;
      const int w0 = nt - part * g.d, h = w0 / g.kv.c.D, e0 = w0 - h * g.kv.c.D;
      const int64_t kvb = part == 2 ? v_block(g.kv.c, g.kv.layer, h) : k_block(g.kv.c, g.kv.layer, h);
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const int rl0 = wm * MT * 16 + i * 16 + quad * 4;
        if (part == 0 || (sizeof(T) == 2 && part == 1)) {
          float v0 = acc[i][j][0], v1 = acc[i][j][1], v2 = acc[i][j][2], v3 = acc[i][j][3];
          transpose4(v0, v1, v2, v3, t);
          const int rl = rl0 + t, cw = col16 & ~3;  // the lane's first column in the tile
          if (part == 0) {
            if (row_src_s[rl] >= 0) {
              if (g.q16) {  // scaled and rounded to bf16 as the attention would on loading q
                const float sc = g.q_scale;
                *reinterpret_cast<uint2*>(g.q16 + (int64_t)(r0 + rl) * g.ldo + nt + cw) =
                    make_uint2(pack_bf16x2(v0 * sc, v1 * sc), pack_bf16x2(v2 * sc, v3 * sc));
              } else {
                *reinterpret_cast<float4*>(reinterpret_cast<float*>(g.out) + (int64_t)(r0 + rl) * g.ldo + nt + cw) =
                    make_float4(v0, v1, v2, v3);
              }
            }
          } else {
            const int64_t base = kv_base[rl];
            if (base >= 0) {
              const int slot = (int)(base & (kPage - 1));
              T* dst = pool + (base - slot) + kvb + k_frag_off<T>(slot, e0 + cw);
              *reinterpret_cast<uint2*>(dst) = make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
            }
          }
          continue;
        }
        const int e = e0 + col16;
        const int64_t b0 = kv_base[rl0];
        const bool run4 = part == 2 && b0 >= 0 && (b0 & 3) == 0 && kv_base[rl0 + 1] == b0 + 1 &&
                          kv_base[rl0 + 2] == b0 + 2 && kv_base[rl0 + 3] == b0 + 3;
        if (run4) {
          const int slot = (int)(b0 & (kPage - 1));
          T* dst = pool + (b0 - slot) + kvb + v_frag_off(slot, e, g.kv.c.D);
          if constexpr (sizeof(T) == 2) {
            *reinterpret_cast<uint2*>(dst) = make_uint2(pack_bf16x2(acc[i][j][0], acc[i][j][1]),
                                                        pack_bf16x2(acc[i][j][2], acc[i][j][3]));
          } else {
            *reinterpret_cast<float4*>(dst) = make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
          }
          continue;
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t base = kv_base[rl0 + r];
          if (base < 0) continue;
          const int slot = (int)(base & (kPage - 1));
          const int64_t page = base - slot;
          const float v = acc[i][j][r];
          if (part == 1)
            pool[page + kvb + k_frag_off<T>(slot, e)] = from_f<T>(v);
          else
            pool[page + kvb + v_frag_off(slot, e, g.kv.c.D)] = from_f<T>(v);
        }
      }
    }
    return;
  }
  if constexpr (EK == E_RESID || EK == E_SWIGLU) {
    // lane t = col16 % 4 of each group of four writes row 4 quad + t of the
    // group's four columns (SwiGLU: four consecutive hidden units) as one
    // 16-byte access (the launcher checks that the widths allow it)
    const int t = col16 & 3;
    if constexpr (EK == E_RESID) {
      // The residual values of one row fragment (NT float4 per lane) are
      // loaded together, so the epilogue waits once per fragment instead of
      // once per 16 x 16 tile.  Inactive rows and columns past N read row 0
      // or the last four columns (in bounds) and store nothing.  With the
      // AdaLN gate (1 + alpha) per column, its values are loaded with them.
      float* out = reinterpret_cast<float*>(g.out);
      auto residual = [&](auto gate_c) __attribute__((always_inline)) {
        constexpr bool kGate = decltype(gate_c)::value;
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          const int rl = wm * MT * 16 + i * 16 + quad * 4 + t;
          const int src = row_src_s[rl];
          const int64_t xo = (int64_t)(src < 0 ? 0 : src) * g.ldo;
          float4 xv[NT], gv[kGate ? NT : 1];
#pragma unroll
          for (int j = 0; j < NT; ++j) {
            const int nb = min(n0 + wn * NT * 16 + j * 16 + (col16 & ~3), g.N - 4);
            xv[j] = *reinterpret_cast<const float4*>(out + xo + nb);
            if constexpr (kGate) gv[j] = *reinterpret_cast<const float4*>(g.mod_a + row_mod_s[rl] + nb);
          }
#pragma unroll
          for (int j = 0; j < NT; ++j) {
            float v0 = acc[i][j][0], v1 = acc[i][j][1], v2 = acc[i][j][2], v3 = acc[i][j][3];
            transpose4(v0, v1, v2, v3, t);
            if constexpr (kGate) { v0 *= 1.f + gv[j].x; v1 *= 1.f + gv[j].y; v2 *= 1.f + gv[j].z; v3 *= 1.f + gv[j].w; }
            const int nb = n0 + wn * NT * 16 + j * 16 + (col16 & ~3);
            if (src >= 0 && nb < g.N)
              *reinterpret_cast<float4*>(out + xo + nb) =
                  make_float4(xv[j].x + v0, xv[j].y + v1, xv[j].z + v2, xv[j].w + v3);
          }
        }
      };
      if (g.mod_a) residual(std::true_type{});
      else residual(std::false_type{});
      return;
    }
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int rl = wm * MT * 16 + i * 16 + quad * 4 + t;
      const int src = row_src_s[rl];
      if constexpr (EK == E_SWIGLU) {
#pragma unroll
        for (int j = 0; j < NT; j += 2) {
          // gate columns j, up columns j + 1 of the same 16 hidden units;
          // silu(g) = g / (1 + e^-g) with the hardware reciprocal (within an
          // ulp of the division, which took ~10 instructions per unit while
          // every workgroup of the round was in its epilogue)
          float h[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float gt = acc[i][j][r], up = acc[i][j + 1][r];
            h[r] = gt * __builtin_amdgcn_rcpf(1.f + __expf(-gt)) * up;
          }
          transpose4(h[0], h[1], h[2], h[3], t);
          const int n = n0 + wn * NT * 16 + j * 16;  // first gate column of the group
          const int unit = (n >> 5) * 16 + (col16 & ~3);
          if (src < 0 || unit >= g.F) continue;
          if (g.out16)
            *reinterpret_cast<uint2*>(g.out16 + (int64_t)(r0 + rl) * g.ldo + unit) =
                make_uint2(pack_bf16x2(h[0], h[1]), pack_bf16x2(h[2], h[3]));
          else
            *reinterpret_cast<float4*>(reinterpret_cast<float*>(g.out) + (int64_t)(r0 + rl) * g.ldo + unit) =
                make_float4(h[0], h[1], h[2], h[3]);
        }
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < MT; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int rl = wm * MT * 16 + i * 16 + quad * 4 + r;
      const int src = row_src_s[rl];
      const int rg = r0 + rl;
      const float rs = NORM ? row_inv_s[rl] : 1.f;
      if constexpr (EK == E_LOGITS) {
        static_assert(NT * 16 % 64 == 0, "whole greedy key groups per wave");
        // compact rows (A_CMP) write their logits to row src(r), the sequence's
        const int orow = AK == A_CMP ? src : g.out_row_off + rg;
#pragma unroll
        for (int j0 = 0; j0 < NT; j0 += 4) {  // one key group: 4 x 16 columns
          unsigned long long best = 0ull;
#pragma unroll
          for (int j = j0; j < j0 + 4; ++j) {
            const int n = n0 + wn * NT * 16 + j * 16 + col16;
            const float v = acc[i][j][r] * rs;
            if (src >= 0 && n < g.N) {
              reinterpret_cast<float*>(g.out)[(int64_t)orow * g.ldo + n] = v;
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
            if (col16 == 0 && src >= 0 && best != 0ull)
              g.argmax_keys[(int64_t)orow * g.key_groups + (n0 + wn * NT * 16 + j0 * 16) / 64] = best;
          }
        }
      } else if constexpr (EK == E_HIDDEN) {  // the other epilogues return above
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          const int n = n0 + wn * NT * 16 + j * 16 + col16;
          if (src < 0 || n >= g.N) continue;
          const float u = acc[i][j][r] + g.bias[n];
          g.out[(int64_t)rg * g.ldo + n] = u / (1.f + __expf(-u));
        }
      }
    }
  }
}

// One output tile per workgroup: tile (blockIdx.y, blockIdx.x).
template <typename T, int MT, int NT, int BK, int AK, int EK, bool MOD, bool NORM, int AMODE, int WM = 2,
          int NSTD = 3>
__global__ __launch_bounds__(WM * 128, WM == 2 ? 2 : 1) void k_gemm(GemmArgs g) {
  constexpr bool kDirect = sizeof(T) == 2 && AMODE == 2;
  constexpr int NST = kDirect ? NSTD : 2, NA = sizeof(T) == 2 && AMODE == 0 ? 2 : 1;
  constexpr int BM = WM * MT * 16, BN = 2 * NT * 16;
  __shared__ __align__(16) T As[NST][NA][BM * BK];
  __shared__ __align__(16) T Bs[NST][BN * BK];
  __shared__ int row_src_s[BM];
  __shared__ int row_mod_s[BM];
  __shared__ float row_inv_s[NORM ? BM : 1];
  __shared__ int64_t kv_base[EK == E_QKV ? BM : 1];
  gemm_tile<T, MT, NT, BK, AK, EK, MOD, NORM, AMODE, WM, NSTD>(g, blockIdx.y * BM, blockIdx.x * BN, As, Bs, row_src_s,
                                                               row_mod_s, row_inv_s, kv_base);
}

// The same with two tile shapes (bf16 A rows): when a loop's active tiles of
// the large shape fill at most half of the workgroup slots (the later
// loops), the workgroups take tiles of the small shape (MT2 x NT2 MFMA tiles
// per wave) from the planner's list instead, about four times as many
// workgroups sharing the loop's K loops.  The small shape uses the large
// one's LDS.
template <typename T, int MT, int NT, int MT2, int NT2, int BK, int AK, int EK, int WM, int NSTD = 3>
__global__ __launch_bounds__(WM * 128, WM == 2 ? 2 : 1) void k_gemm_dual(GemmArgs g) {
  constexpr int BM = WM * MT * 16, BN = 2 * NT * 16, BM2 = WM * MT2 * 16, BN2 = 2 * NT2 * 16;
  static_assert(BM2 < BM && BN2 <= BN && (BM2 == 64 || BM2 == 128), "small shape");
  __shared__ __align__(16) T As[NSTD][1][BM * BK];
  __shared__ __align__(16) T Bs[NSTD][BN * BK];
  __shared__ int row_src_s[BM];
  __shared__ int row_mod_s[BM];
  __shared__ float row_inv_s[1];
  __shared__ int64_t kv_base[EK == E_QKV ? BM : 1];
  if (g.tl.cnt) {
    const int large = g.tl.cnt[BM == 256 ? 2 : 1] * (int)gridDim.x;  // active tiles of the large shape
    const int slots = g.tl.cus * (WM == 2 ? 2 : 1);
    const int tiles_n2 = (g.N + BN2 - 1) / BN2;
    const int small = g.tl.cnt[BM2 == 64 ? 0 : 1] * tiles_n2;
    if (2 * large <= slots && small <= (int)(gridDim.x * gridDim.y)) {
      const int L = (int)(blockIdx.y * gridDim.x + blockIdx.x);
      if (L >= small) return;
      const int32_t* list = BM2 == 64 ? g.tl.list64 : g.tl.list128;
      gemm_tile<T, MT2, NT2, BK, AK, EK, false, false, 2, WM, NSTD>(g, list[L / tiles_n2], (L % tiles_n2) * BN2, As, Bs,
                                                                     row_src_s, row_mod_s, row_inv_s, kv_base);
      return;
    }
    // the large tiles from the list too: the active ones are the grid's first
    // workgroups, in the order of a loop with every row active
    const int L = (int)(blockIdx.y * gridDim.x + blockIdx.x);
    const int32_t* list = BM == 256 ? g.tl.list256 : g.tl.list128;
    // a last round at most half filled: each of its large tiles as four
    // small ones (2 x 2, rows past a segment's count leave at once)
    const int full = large / slots * slots, tail = large - full;
    bool split = false;
    if constexpr (BM2 * 2 == BM && BN2 * 2 == BN) {
      split = full > 0 && 2 * tail <= slots && full + 4 * tail <= (int)(gridDim.x * gridDim.y);
      if (split && L >= full) {
        if (L >= full + 4 * tail) return;
        const int q = (L - full) & 3, t = full + ((L - full) >> 2);
        gemm_tile<T, MT2, NT2, BK, AK, EK, false, false, 2, WM, NSTD>(
            g, list[t / (int)gridDim.x] + (q >> 1) * BM2, (t % (int)gridDim.x) * BN + (q & 1) * BN2, As, Bs,
            row_src_s, row_mod_s, row_inv_s, kv_base);
        return;
      }
    }
    // workgroup L runs on XCD L % 8 (dispatch is round-robin over the XCDs).
    // With at most four column tiles (the O and down projections) the n large
    // tiles go to the XCDs as contiguous runs, so that each XCD's L2 holds a
    // few row tiles at a time rather than a slice of every one; with more
    // columns the plain order, which gives each XCD a subset of the weight
    // columns, measured faster.
    const int n = split ? full : large;
    if (L >= n) return;
    int t = L;
    if (gridDim.x <= 4) {
      const int x = L & 7, per = n >> 3, rem = n & 7;
      t = x * per + min(x, rem) + (L >> 3);
    }
    gemm_tile<T, MT, NT, BK, AK, EK, false, false, 2, WM, NSTD>(g, list[t / (int)gridDim.x], (t % (int)gridDim.x) * BN,
                                                                As, Bs, row_src_s, row_mod_s, row_inv_s, kv_base);
    return;
  }
  gemm_tile<T, MT, NT, BK, AK, EK, false, false, 2, WM, NSTD>(g, blockIdx.y * BM, blockIdx.x * BN, As, Bs, row_src_s,
                                                              row_mod_s, row_inv_s, kv_base);
}

template <typename T, int MT, int NT>
hipError_t launch_tiles(const GemmArgs& a, AKind ak, EKind ek, bool norm, hipStream_t s) {
  constexpr int BM = 2 * MT * 16, BN = 2 * NT * 16;
  const dim3 grid((a.N + BN - 1) / BN, (a.rm.rows + BM - 1) / BM);
  if (grid.x == 0 || grid.y == 0) return hipSuccess;
  const bool mod = a.mod_g != nullptr;
  // operand mode: hi + lo parts, one bf16 part of float A, or bf16 A rows
  // (copied into LDS by their loads)
  const int amode = sizeof(T) != 2 ? 0 : a.A16 ? 2 : a.a_single ? 1 : 0;
  if (amode == 2 && (mod || norm)) return hipErrorInvalidValue;
#define TLF_GEMM_LAUNCH(AKV, EKV, MODV, NORMV, AM) \
  hipLaunchKernelGGL((k_gemm<T, MT, NT, kGemmBK, AKV, EKV, MODV, NORMV, AM>), grid, dim3(256), 0, s, a)
  {
#define TLF_GEMM_CASE(AKV, EKV, MODV, NORMV)                                  \
  if (ak == AKV && ek == EKV && mod == MODV && norm == NORMV) {               \
    if (amode == 0) TLF_GEMM_LAUNCH(AKV, EKV, MODV, NORMV, 0);                \
    else if (amode == 1) TLF_GEMM_LAUNCH(AKV, EKV, MODV, NORMV, 1);           \
    else if constexpr (!MODV && !NORMV) {                                     \
      if constexpr (sizeof(T) == 2 && NT == 8)                                \
        hipLaunchKernelGGL((k_gemm_dual<T, MT, NT, 2, 4, kGemmBK, AKV, EKV, 2>), grid, dim3(256), 0, s, a); \
      else                                                                    \
        TLF_GEMM_LAUNCH(AKV, EKV, false, false, 2);                           \
    }                                                                         \
    return hipGetLastError();                                                 \
  }
  TLF_GEMM_CASE(A_SRC, E_QKV, false, false)
  TLF_GEMM_CASE(A_SRC, E_QKV, true, false)
  TLF_GEMM_CASE(A_SRC, E_SWIGLU, false, false)
  TLF_GEMM_CASE(A_SRC, E_SWIGLU, true, false)
  TLF_GEMM_CASE(A_CMP, E_RESID, false, false)
#undef TLF_GEMM_CASE
  // the LM heads and the router's hidden layer keep the hi + lo parts
  if (amode != 0) return hipErrorInvalidValue;
  if (ak == A_SRC && ek == E_LOGITS && !mod && !norm) { TLF_GEMM_LAUNCH(A_SRC, E_LOGITS, false, false, 0); return hipGetLastError(); }
  if (ak == A_CMP && ek == E_LOGITS && !mod && norm) { TLF_GEMM_LAUNCH(A_CMP, E_LOGITS, false, true, 0); return hipGetLastError(); }
  if (ak == A_CMP && ek == E_HIDDEN && !mod && !norm) { TLF_GEMM_LAUNCH(A_CMP, E_HIDDEN, false, false, 0); return hipGetLastError(); }
  }
#undef TLF_GEMM_LAUNCH
  return hipErrorInvalidValue;
}

// The down projection of many rows (bf16 rows, K = F): 256 x 256 tiles of
// 8 waves (each still 64 x 128), one workgroup per compute unit; at 32768
// rows x 1024 x 2816 it took 204 us against 232 us with 128 x 256 tiles of 4
// waves, while the gate/up, QKV and O projections (K = d) gained nothing.
constexpr int kWideResidMinK = 2048, kWideResidMinRows = 16384;
template <typename T>
hipError_t launch_resid_wide(const GemmArgs& a, hipStream_t s) {
  if constexpr (sizeof(T) == 2) {
    constexpr int WM = 4, BM = WM * kGemmMT * 16, BN = 2 * 8 * 16;
    const dim3 grid((a.N + BN - 1) / BN, (a.rm.rows + BM - 1) / BM);
    hipLaunchKernelGGL((k_gemm_dual<T, kGemmMT, 8, 2, 4, kGemmBK, A_CMP, E_RESID, WM>), grid, dim3(WM * 128), 0, s, a);
    return hipGetLastError();
  }
  return hipErrorInvalidValue;
}

}  // namespace

template <typename T>
hipError_t launch_gemm(const GemmArgs& a, AKind ak, EKind ek, bool norm, hipStream_t s) {
  if (a.K % kGemmBK != 0) return hipErrorInvalidValue;
  // float A in fragment order: bf16 weights (8 consecutive k per run), compact rows
  if (a.a_frag && (sizeof(T) != 2 || ak != A_CMP || a.A16)) return hipErrorInvalidValue;
  // the QKV epilogue takes each 16-column tile as wholly q, k or v
  if (ek == E_QKV && (a.d % 16 != 0 || a.ldo % 4 != 0 || a.kv.c.D % 16 != 0)) return hipErrorInvalidValue;
  // the residual and SwiGLU epilogues write four consecutive columns at once
  if ((ek == E_RESID && (a.N % 4 != 0 || a.ldo % 4 != 0 || (a.mod_a && a.mod_ld % 4 != 0))) ||
      (ek == E_SWIGLU && (a.F % 4 != 0 || a.ldo % 4 != 0)))
    return hipErrorInvalidValue;
  if (sizeof(T) == 2 && ak == A_CMP && ek == E_RESID && !norm && a.A16 && !a.mod_g && a.K >= kWideResidMinK &&
      a.rm.rows >= kWideResidMinRows)
    return launch_resid_wide<T>(a, s);
  // a few row tiles (the decode LM head) take 128-column tiles so the grid
  // still holds about two workgroups per compute unit; prefill takes 256
  const int row_tiles = (a.rm.rows + 2 * kGemmMT * 16 - 1) / (2 * kGemmMT * 16);
  if (row_tiles <= 4) return launch_tiles<T, kGemmMT, 4>(a, ak, ek, norm, s);
  return launch_tiles<T, kGemmMT, 8>(a, ak, ek, norm, s);
}

template hipError_t launch_gemm<float>(const GemmArgs&, AKind, EKind, bool, hipStream_t);
template hipError_t launch_gemm<bf16>(const GemmArgs&, AKind, EKind, bool, hipStream_t);

}  // namespace tlf
