// Attention over the recursion-wise KV cache (Eq. 10).
//
// Decode: a query at loop i reads only cache (b, i), i.e. the earlier tokens
// of its sequence whose depth is >= i plus itself; exited tokens have no
// slot, so the validity mask is implicit.  One workgroup of W waves owns a
// (row, head) of a persistent grid; its page list is staged in LDS, each wave
// streams a contiguous share of the entries in 16-byte K/V loads (G lanes per
// token, 64/G tokens per instruction) with two register batches in flight,
// every lane keeps its own online-softmax state, lanes merge with DPP moves
// and shuffles, and the W waves merge through LDS with a log-sum-exp combine.
// No state crosses workgroups, so no device-scope fence is needed.
//
// Prefill: causal attention among the gathered tokens of each loop (Section
// 3.3), which in compact order is a plain causal mask on the (b, i) slot
// sequence.  One workgroup per (sequence, 64-query tile, head), 16 queries
// per wave, the longest query tiles dispatched first.  Key tiles of four pages are copied into LDS verbatim (the K
// blocks are already in MFMA-fragment order), the next tile loading into
// registers while the current one is in use.  Scores are computed transposed,
// S^T = K q^T, so that the P^T operand of O^T = V^T P^T is exactly the scores
// each lane holds (no data movement between the two products); both run on
// MFMA with an online softmax per query.  Against bf16 keys q enters as hi +
// lo parts, or as one bf16 part when the caller asks for it (q_single).
#include "kernels.h"

namespace tlf {

namespace {

constexpr float kNegInf = -__builtin_inff();

// Streaming loads of cache entries: each K/V byte is read once per launch, so
// the loads are marked non-temporal.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
template <typename F, typename P> __device__ __forceinline__ F ld_stream(const P* p) {
  if constexpr (sizeof(F) == 16) {
    return __builtin_bit_cast(F, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)));
  } else if constexpr (sizeof(F) == 8) {
    return __builtin_bit_cast(F, __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p)));
  } else {
    return __builtin_bit_cast(F, __builtin_nontemporal_load(reinterpret_cast<const unsigned int*>(p)));
  }
}

// Queries per wave and waves per workgroup of the prefill attention.
constexpr int kPreQW = 16, kPreWaves = 8;

__device__ __forceinline__ float4 scale4(float4 v, float s) { return make_float4(v.x * s, v.y * s, v.z * s, v.w * s); }

// 2^x straight from the transcendental unit (v_exp_f32), for softmax
// weights: x is a score less the running maximum (decode) or less a base
// that the tile's weights exceed by at most 2^16 (prefill).  Results below
// the smallest normal float flush to zero; exp2f would rescale around the
// instruction to keep them, five instructions instead of one, for weights
// that are then rounded to bf16 or summed beside a weight of at least 1,
// where they make no difference.
__device__ __forceinline__ float exp2_weight(float x) { return __builtin_amdgcn_exp2f(x); }

// In the decode attention the 16 lanes of a lane row (one quad) hold the
// scores of the same tokens (q fills all 16 columns of the product): the
// four rows' values, read as scalars, give a wave-uniform result without a
// trip through the LDS crossbar.
__device__ __forceinline__ float lane_read(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ float rows_max(float v) {
  return fmaxf(fmaxf(lane_read(v, 0), lane_read(v, 16)), fmaxf(lane_read(v, 32), lane_read(v, 48)));
}
__device__ __forceinline__ float rows_sum(float v) {  // (row 0 + row 1) + (row 2 + row 3)
  return (lane_read(v, 0) + lane_read(v, 16)) + (lane_read(v, 32) + lane_read(v, 48));
}

// Exchanges between lane rows in the VALU instead of the LDS crossbar:
// v_permlane16_swap / v_permlane32_swap of a value with itself hand every
// lane its own and its xor-16 (xor-32) partner's value, the lower row's
// first, so both partners combine the pair in the same order.
__device__ __forceinline__ float max_xor16(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}
__device__ __forceinline__ float max_xor32(float v) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
}
__device__ __forceinline__ float sum_xor16(float v) {
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}
__device__ __forceinline__ float sum_xor32(float v) {
  const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

__device__ __forceinline__ float merge_scale(float m, float mn) {
  return m == kNegInf ? 0.f : exp2_weight(m - mn);
}

// Sum over aligned groups of G lanes (G = 2, 4, 8, 16, 32) with DPP moves
// inside rows of 16 lanes and a shuffle beyond them.
template <typename T, int D, int W>
__global__ __launch_bounds__(W * 64) void k_attn_decode(AttnDecodeArgs a) {
  using M = Mfma<T>;
  constexpr int KS = M::KS, EPL = M::EPL;
  constexpr int PPI = EPL == 8 ? 2 : 1;                    // pages per iteration (4 * PPI slots per lane)
  constexpr int KSTEPS = D / KS;                            // S MFMAs per page
  constexpr int DT = D / 16;                                // output dimension tiles
  constexpr int PVM = 4 * PPI / EPL;                        // P.V MFMAs per iteration
  constexpr int NBUF = D * (int)sizeof(T) <= 128 ? 2 : 1;   // batches in flight
  constexpr int NQ = EPL == 8 ? 2 : 1;                      // parts of q (hi, lo)
  static_assert(KSTEPS >= 1 && D % 16 == 0, "head_dim");
  static_assert(4 * PPI % EPL == 0, "P.V k-slots");
  // V^T fragment per dimension tile: 4 consecutive slots of one dimension from
  // each of the PPI pages (bf16: 2 x 8 bytes; f32: 16 bytes)
  typedef typename M::frag KFrag;
  __shared__ int s_pages[kAttnMaxPages];
  __shared__ float s_red[W][D + 2];

  const CacheView& c = a.c;
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const int quad = lane >> 4, c16 = lane & 15;
  const int H = c.H, R = c.R, i = a.loop;
  const int nunits = *a.nact * H;
  const T* pool = reinterpret_cast<const T*>(c.pool);

  for (int u = blockIdx.x; u < nunits; u += gridDim.x) {
    const int k = u / H, h = u % H;
    const int b = a.perm[k];
    // the row's first W x 64 page-table entries are read together with the
    // cache length (they do not depend on it), the rest once it is known
    const int32_t* pt = c.page_table + ((int64_t)b * R + i) * c.pages_per_seq;
    const int p_first = threadIdx.x < c.pages_per_seq ? pt[threadIdx.x] : 0;
    const int L = c.cache_len[b * R + i];
    const int np = (L + kPage - 1) / kPage;
    __syncthreads();  // the previous unit is done with s_pages and s_red
    if ((int)threadIdx.x < np) s_pages[threadIdx.x] = p_first;
    for (int p = threadIdx.x + W * kWave; p < np; p += W * kWave) s_pages[p] = pt[p];
    __syncthreads();

    // this wave's pages [p0, p1), a multiple of PPI pages each
    const int per = ((np + W - 1) / W + PPI - 1) / PPI * PPI;
    const int p0 = w * per, p1 = min(np, p0 + per);
    const int64_t koff = k_block(c, a.layer, h) + (int64_t)(quad * kPage + c16) * EPL;  // fragment order
    const int64_t voff = v_block(c, a.layer, h) + (int64_t)(quad * D + c16) * 4;  // slots 4 quad .. + 3 of dim c16

    // q (float32) as the B operand of S = K q^T, the same in all 16 columns;
    // against bf16 keys it is split into hi and lo parts, one product each
    KFrag qf[NQ][KSTEPS];
    {
      const float* qp = a.q + (int64_t)k * a.d + h * D + quad * EPL;
#pragma unroll
      for (int ks = 0; ks < KSTEPS; ++ks) {
        if constexpr (NQ == 2) split_frag(qp + ks * KS, qf[0][ks], qf[NQ - 1][ks]);
        else qf[0][ks] = qp[ks * KS];
      }
    }
    f32x4 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m = kNegInf, lsum = 0.f;

    auto load = [&](KFrag (&bk)[PPI][KSTEPS], uint4 (&bv)[DT], int pg) __attribute__((always_inline)) {
      const T* base[PPI];
#pragma unroll
      for (int p = 0; p < PPI; ++p) {
        // past the range: reread the last page (its scores are masked); loads
        // are never skipped so the compiler can count the batch in flight
        const int pp = min(pg + p, p1 - 1);
        base[p] = pool + (int64_t)s_pages[pp] * c.page_elems;
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) bk[p][ks] = ld_stream<KFrag>(base[p] + koff + ks * (4 * kPage * EPL));
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int64_t off = voff + (int64_t)dt * 16 * 4;
        if constexpr (EPL == 8) {
          const u32x2 lo = ld_stream<u32x2>(base[0] + off);
          const u32x2 hi = ld_stream<u32x2>(base[PPI - 1] + off);
          bv[dt] = make_uint4(lo.x, lo.y, hi.x, hi.y);
        } else {
          const u32x4 v = ld_stream<u32x4>(base[0] + off);
          bv[dt] = make_uint4(v.x, v.y, v.z, v.w);
        }
      }
    };
    auto consume = [&](const KFrag (&bk)[PPI][KSTEPS], const uint4 (&bv)[DT], int pg)
                       __attribute__((always_inline)) {
      // scores of this lane's tokens: page p, slot 4 * quad + r
      float sc[PPI][4];
      float mx = m;
      // only a batch that reaches past the wave's pages or the cache's last
      // token is masked (wave-uniform)
      const bool edge = pg + PPI > p1 || (pg + PPI) * kPage > L;
#pragma unroll
      for (int p = 0; p < PPI; ++p) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
          for (int qa = 0; qa < NQ; ++qa) acc = M::mma(bk[p][ks], qf[qa][ks], acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          sc[p][r] = acc[r] * a.scale_log2;
          if (edge) {
            const int t = (pg + p) * kPage + 4 * quad + r;
            if ((pg + p) >= p1 || t >= L) sc[p][r] = kNegInf;
          }
          mx = fmaxf(mx, sc[p][r]);
        }
      }
      mx = rows_max(mx);
      if (mx == kNegInf) return;  // wave-uniform: nothing valid yet
      if (mx != m) {
        // wave-uniform (every lane holds the same query's scores): an
        // unchanged maximum would scale by exactly 1, so the rescale, which
        // moves the accumulators through VGPRs, runs only when it changes
        const float alpha = merge_scale(m, mx);
        lsum *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
      }
      float pr[PPI][4];
#pragma unroll
      for (int p = 0; p < PPI; ++p)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pr[p][r] = exp2_weight(sc[p][r] - mx);  // 0 for masked slots
          lsum += pr[p][r];
        }
      // P.V: MFMA mm takes k-slots (page, r) = mm * EPL .. mm * EPL + EPL - 1 of
      // this lane's tokens, in the same order on both operands
#pragma unroll
      for (int mm = 0; mm < PVM; ++mm) {
        KFrag pa;
        if constexpr (EPL == 8) {
          const uint4 u = make_uint4(pack_bf16x2(pr[0][0], pr[0][1]), pack_bf16x2(pr[0][2], pr[0][3]),
                                     pack_bf16x2(pr[PPI - 1][0], pr[PPI - 1][1]),
                                     pack_bf16x2(pr[PPI - 1][2], pr[PPI - 1][3]));
          pa = __builtin_bit_cast(KFrag, u);
        } else {
          pa = pr[0][mm];
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          KFrag vb;
          if constexpr (EPL == 8) {
            vb = __builtin_bit_cast(KFrag, bv[dt]);
          } else {
            const uint4 u = bv[dt];
            vb = __uint_as_float(mm == 0 ? u.x : mm == 1 ? u.y : mm == 2 ? u.z : u.w);
          }
          o[dt] = M::mma(pa, vb, o[dt]);
        }
      }
      m = mx;
    };
    if (p0 < p1) {
      KFrag ka[PPI][KSTEPS];
      uint4 va[DT];
      if constexpr (NBUF == 2) {
        KFrag kb[PPI][KSTEPS];
        uint4 vb2[DT];
        // batches of PPI pages; every load stays inside the wave's range (a
        // load past it would fetch its last page from memory again), so the
        // last one or two batches are peeled
        load(ka, va, p0);
        int pg = p0;
        for (; pg + 2 * PPI < p1; pg += 2 * PPI) {
          load(kb, vb2, pg + PPI);
          consume(ka, va, pg);
          load(ka, va, pg + 2 * PPI);
          consume(kb, vb2, pg + PPI);
        }
        if (pg + PPI < p1) {
          load(kb, vb2, pg + PPI);
          consume(ka, va, pg);
          consume(kb, vb2, pg + PPI);
        } else {
          consume(ka, va, pg);
        }
      } else {
        for (int pg = p0; pg < p1; pg += PPI) {
          load(ka, va, pg);
          consume(ka, va, pg);
        }
      }
    }
    // the four lane quads hold different tokens: add their softmax sums
    lsum = rows_sum(lsum);
    if (quad == 0) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) s_red[w][2 + dt * 16 + c16] = o[dt][0];
      if (c16 == 0) { s_red[w][0] = m; s_red[w][1] = lsum; }
    }
    __syncthreads();
    // merge the W waves' partial softmax states (log-sum-exp) and write o
    if (w == 0) {
      for (int dim = lane; dim < D; dim += kWave) {
        float Mx = kNegInf, Ls = 0.f, O = 0.f;
#pragma unroll
        for (int ww = 0; ww < W; ++ww) {
          const float mc = s_red[ww][0], lc = s_red[ww][1];
          const float mn = fmaxf(Mx, mc);
          const float a1 = merge_scale(Mx, mn), a2 = merge_scale(mc, mn);
          Ls = Ls * a1 + lc * a2;
          O = O * a1 + s_red[ww][2 + dim] * a2;
          Mx = mn;
        }
        // an empty cache (a discarded row of the dense decode) gives zeros
        const int c = h * D + dim;
        const int64_t oi = a.o_ks > 0 ? ((int64_t)((k >> 4) * (a.d / a.o_ks) + c / a.o_ks) * kWave +
                                         (c % a.o_ks) / a.o_epl * 16 + (k & 15)) * a.o_epl + c % a.o_epl
                                      : (int64_t)k * a.d + c;
        a.o[oi] = Ls > 0.f ? O / Ls : 0.f;
      }
    }
  }
}

template <typename T, int D, bool SPLITQ>
__global__ __launch_bounds__(kPreWaves * 64, 16 / kPreWaves) void k_attn_prefill(AttnPrefillArgs a) {
  using M = Mfma<T>;
  typedef typename M::frag Frag;
  constexpr int KS = M::KS, EPL = M::EPL;
  constexpr int QW = kPreQW;                      // queries per wave
  constexpr int QN = QW / 16;                     // query column tiles per wave
  constexpr int NTH = kPreWaves * kWave;          // threads
  constexpr int BQ = kPreWaves * QW;              // queries per workgroup
  constexpr int BKEY = 4 * kPage;                 // keys per tile: four pages
  constexpr int NT = BKEY / 16;                   // 16-key subtiles
  constexpr int KSTEPS = D / KS;
  constexpr int DT = D / 16;
  constexpr int NQ = EPL == 8 && SPLITQ ? 2 : 1;  // parts of q (hi, lo), or one bf16 part
  constexpr int KBLK = kPage * D;                 // elements of one page's K (or V) block
  constexpr int EPC = 16 / (int)sizeof(T);        // elements per 16-byte chunk
  constexpr int VLD = kPage + (sizeof(T) == 2 ? 4 : 2);  // padded LDS row of one dimension of a V block
  // bf16: one row per dimension holding the tile's 64 slots with the pages
  // paired at 4-slot granularity (slots 4g..4g+3 of page 2m, then those of
  // page 2m + 1), so that a lane's P.V fragment (its four slots of two
  // pages) is one 16-byte read; 144-byte rows keep the 8 or 16 lanes of one
  // LDS pass on distinct banks.  float32: [page][dim] rows of VLD slots.
  constexpr int VDS = 4 * kPage + 8;
  constexpr int VTILE = sizeof(T) == 2 ? D * VDS : 4 * D * VLD;
  auto vidx = [](int p, int d, int slot) {  // element of (page p, dimension d, slot)
    return sizeof(T) == 2 ? d * VDS + (p >> 1) * 32 + (slot >> 2) * 8 + (p & 1) * 4 + (slot & 3)
                          : (p * D + d) * VLD + slot;
  };
  constexpr int CH = 2 * 4 * KBLK / EPC;          // 16-byte chunks of one K + V tile
  static_assert(CH % NTH == 0, "tile chunks per thread");
  constexpr int CPT = CH / NTH;
  static_assert(EPC % 4 == 0 && (4 * D) % EPC == 0, "V chunk: whole 4-slot groups of one slot group");
  // K tile: four pages' K blocks verbatim (fragment order: lane (key, quad) of a
  // K step reads EPL contiguous elements, 64 lanes one contiguous run);
  // V tile: four pages' V blocks rearranged to rows of one dimension (layout at vidx)
  __shared__ __align__(16) T Ks[2][4 * KBLK];
  __shared__ __align__(16) T Vs[2][VTILE];

  const CacheView& c = a.c;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int quad = lane >> 4, c16 = lane & 15;
  const int QT = (a.T + BQ - 1) / BQ;
  // workgroup u = (QT - 1 - qt) * G * H + g * H + h: the last query tiles see
  // the most keys, so they are dispatched first
  const int GH = a.G * c.H, u = blockIdx.x;
  const int qt = QT - 1 - u / GH, g = (u % GH) / c.H, h = u % c.H;
  const int b = a.b0 + g;
  // the call's nq queries are cache entries [n - nq, n) of (b, loop): query
  // row a (compact index n0 + a) sees keys [0, n0 + a]
  const int n = c.cache_len[b * c.R + a.loop];
  const int nq = c.chunk_len[b * c.R + a.loop];
  const int n0 = n - nq;
  const int q0 = qt * BQ;
  if (q0 >= nq) return;
  const int32_t* pt = c.page_table + ((int64_t)b * c.R + a.loop) * c.pages_per_seq;
  const T* pool = reinterpret_cast<const T*>(c.pool);
  const int64_t koff = k_block(c, a.layer, h), voff = v_block(c, a.layer, h);
  const int npages = (n + kPage - 1) / kPage;
  const int nkt = (min(n, n0 + min(nq, q0 + BQ)) + BKEY - 1) / BKEY;  // key tiles of the workgroup
  const int wq0 = n0 + q0 + w * QW;               // compact index of the wave's first query

  // q (float32, scaled by log2(e) / sqrt(D) so scores come out in log2
  // units) as the B operand of S^T = K q^T; against bf16 keys it is split
  // into hi and lo parts, one product each
  Frag qf[QN][NQ][KSTEPS];
#pragma unroll
  for (int qn = 0; qn < QN; ++qn) {
    const int qrow = min(q0 + w * QW + qn * 16 + c16, nq - 1);
    const float* qp = a.q + ((int64_t)g * a.T + qrow) * a.d + h * D + quad * EPL;
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      if constexpr (NQ == 2) {
        const float4 v0 = *reinterpret_cast<const float4*>(qp + ks * KS);
        const float4 v1 = *reinterpret_cast<const float4*>(qp + ks * KS + 4);
        uint2 h0, l0, h1, l1;
        split4(scale4(v0, a.scale_log2), h0, l0);
        split4(scale4(v1, a.scale_log2), h1, l1);
        qf[qn][0][ks] = __builtin_bit_cast(Frag, make_uint4(h0.x, h0.y, h1.x, h1.y));
        qf[qn][1][ks] = __builtin_bit_cast(Frag, make_uint4(l0.x, l0.y, l1.x, l1.y));
      } else if constexpr (EPL == 8) {
        if (a.q16) {  // written scaled and rounded by the QKV projection
          qf[qn][0][ks] = *reinterpret_cast<const Frag*>(a.q16 + (qp - a.q) + ks * KS);
        } else {
          const float4 v0 = scale4(*reinterpret_cast<const float4*>(qp + ks * KS), a.scale_log2);
          const float4 v1 = scale4(*reinterpret_cast<const float4*>(qp + ks * KS + 4), a.scale_log2);
          qf[qn][0][ks] = __builtin_bit_cast(Frag, make_uint4(pack_bf16x2(v0.x, v0.y), pack_bf16x2(v0.z, v0.w),
                                                              pack_bf16x2(v1.x, v1.y), pack_bf16x2(v1.z, v1.w)));
        }
      } else {
        qf[qn][0][ks] = qp[ks * KS] * a.scale_log2;
      }
    }
  }

  // one K + V tile: chunk ci < CH/2 is K chunk ci, else V chunk ci - CH/2;
  // pages past the cache are stored as zeros (their scores are masked).  A
  // page block holds a multiple of 64 chunks, so the 64 chunks of one wave
  // in round u lie in one block: its page and K/V choice are wave-uniform.
  // The tile's table entries are read first (scalar loads), then every data
  // load is issued, from the last page where the tile runs past the cache,
  // so that none waits on another.
  static_assert((KBLK / EPC) % kWave == 0, "a wave's chunks within one page block");
  const int wu = __builtin_amdgcn_readfirstlane(w);
  auto round_page = [&](int u) { return ((wu * kWave + u * NTH) % (CH / 2)) / (KBLK / EPC); };
  uint4 pa[CPT], pb[CPT];  // tiles in flight in registers
  auto load_tile = [&](int kt, uint4 (&pre)[CPT]) __attribute__((always_inline)) {
    int pg[CPT];
#pragma unroll
    for (int u = 0; u < CPT; ++u) pg[u] = pt[min(kt * 4 + round_page(u), npages - 1)];
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      const int ci0 = wu * kWave + u * NTH;  // the wave's first chunk of round u
      const int kv = ci0 / (CH / 2);
      const int off = ((ci0 % (CH / 2)) % (KBLK / EPC) + lane) * EPC;
      pre[u] = *reinterpret_cast<const uint4*>(pool + (int64_t)pg[u] * c.page_elems + (kv ? voff : koff) + off);
    }
  };
  auto store_tile = [&](int kt, int buf, const uint4 (&pre)[CPT]) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
      const int ci = tid + u * NTH;
      const int kv = ci / (CH / 2), cc = ci % (CH / 2);
      const int p = cc / (KBLK / EPC), off = (cc % (KBLK / EPC)) * EPC;
      uint4 v = pre[u];
      if (kt * 4 + round_page(u) >= npages) v = make_uint4(0, 0, 0, 0);
      if (kv == 0) {
        *reinterpret_cast<uint4*>(&Ks[buf][p * KBLK + off]) = v;
      } else {
        // the chunk holds slots 4 g4 .. 4 g4 + 3 of EPC / 4 consecutive dimensions
        const int g4 = off / (4 * D), d0 = (off % (4 * D)) / 4;
        if constexpr (sizeof(T) == 2) {
          *reinterpret_cast<uint2*>(&Vs[buf][vidx(p, d0, 4 * g4)]) = make_uint2(v.x, v.y);
          *reinterpret_cast<uint2*>(&Vs[buf][vidx(p, d0 + 1, 4 * g4)]) = make_uint2(v.z, v.w);
        } else {
          T* dst = &Vs[buf][vidx(p, d0, 4 * g4)];
          *reinterpret_cast<uint2*>(dst) = make_uint2(v.x, v.y);
          *reinterpret_cast<uint2*>(dst + 2) = make_uint2(v.z, v.w);
        }
      }
    }
  };

  f32x4 o[DT][QN];  // O^T: lane holds dims 4 quad + r of tile dt for query c16 of column tile qn
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int qn = 0; qn < QN; ++qn) o[dt][qn] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Online softmax with a lazily moved base per query (column): the score
  // products start from -base, so they come out relative to it, and a
  // tile's weights are exp2 of them directly.  The base is set by the first
  // key tile (key 0 is visible to every query) and moves up, rescaling the
  // running sums, only when a lane's weights in a tile add up to more than
  // kSumMax; weights therefore stay below kSumMax, far inside the range of
  // float32 sums and bf16 operands, and o / l is unchanged by the choice.
  constexpr float kSumMax = 65536.f;
  float nb[QN], lq[QN];  // -base (per query, replicated over quads) and this lane's weight sum
#pragma unroll
  for (int qn = 0; qn < QN; ++qn) { nb[qn] = 0.f; lq[qn] = 0.f; }

  // the products of key tile kt from LDS buffer buf
  auto use_tile = [&](int kt, int buf) __attribute__((always_inline)) {
    // the wave's queries see keys <= their compact index: skip tiles past its last query
    if (kt * BKEY <= wq0 + QW - 1) {
      const T* kb = Ks[buf];
      // mask only a tile that reaches past the wave's first query or the cache end
      const bool edge = kt * BKEY + BKEY - 1 > wq0 || kt * BKEY + BKEY > n;
      // S^T tile (nt, qn) less the base: lane holds keys nt * 16 + 4 quad + r of query c16
      f32x4 s[NT][QN];
      auto scores = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
          for (int qn = 0; qn < QN; ++qn) s[nt][qn] = f32x4{nb[qn], nb[qn], nb[qn], nb[qn]};
#pragma unroll
          for (int ks = 0; ks < KSTEPS; ++ks) {
            const Frag kf = M::load(kb + nt * KBLK + ((ks * 4 + quad) * kPage + c16) * EPL);
#pragma unroll
            for (int qn = 0; qn < QN; ++qn)
#pragma unroll
              for (int qa = 0; qa < NQ; ++qa) s[nt][qn] = M::mma(kf, qf[qn][qa][ks], s[nt][qn]);
          }
        }
        if (edge) {
#pragma unroll
          for (int qn = 0; qn < QN; ++qn) {
            const int qidx = wq0 + qn * 16 + c16;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const int kidx = kt * BKEY + nt * 16 + 4 * quad + r;
                if (kidx > qidx || kidx >= n) s[nt][qn][r] = kNegInf;
              }
          }
        }
      };
      scores();
      float ps[QN];
      bool move = kt == 0;
      if (!move) {
        bool over = false;
#pragma unroll
        for (int qn = 0; qn < QN; ++qn) {
          ps[qn] = 0.f;
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float p = exp2_weight(s[nt][qn][r]);
              s[nt][qn][r] = p;
              ps[qn] += p;
            }
          over |= !(ps[qn] <= kSumMax);
        }
        move = __builtin_amdgcn_ballot_w64(over) != 0;
        if (move) scores();  // rare: the K tile is still in LDS
      }
      if (move) {
        // new base: the column maximum (first tile), else the old base or
        // the column maximum, whichever is larger
#pragma unroll
        for (int qn = 0; qn < QN; ++qn) {
          float mx = kNegInf;
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int r = 0; r < 4; ++r) mx = fmaxf(mx, s[nt][qn][r]);
          mx = max_xor32(max_xor16(mx));
          const float dlt = kt == 0 ? mx : fmaxf(mx, 0.f);
          if (kt > 0) {
            const float alpha = exp2_weight(-dlt);
            lq[qn] *= alpha;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) o[dt][qn] *= alpha;
          }
          nb[qn] -= dlt;
          ps[qn] = 0.f;
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const float p = exp2_weight(s[nt][qn][r] - dlt);
              s[nt][qn][r] = p;
              ps[qn] += p;
            }
        }
      }
#pragma unroll
      for (int qn = 0; qn < QN; ++qn) lq[qn] += ps[qn];
      // O^T += V^T P^T: the k-slots of one MFMA are keys this lane holds
      // scores for, in the same order on both operands
      const T* vb = Vs[buf];
      if constexpr (EPL == 8) {
#pragma unroll
        for (int np = 0; np < NT; np += 2) {  // keys (np, 4 quad + r) and (np + 1, 4 quad + r)
          Frag pf[QN];
#pragma unroll
          for (int qn = 0; qn < QN; ++qn) {
            const uint4 u = make_uint4(pack_bf16x2(s[np][qn][0], s[np][qn][1]), pack_bf16x2(s[np][qn][2], s[np][qn][3]),
                                       pack_bf16x2(s[np + 1][qn][0], s[np + 1][qn][1]),
                                       pack_bf16x2(s[np + 1][qn][2], s[np + 1][qn][3]));
            pf[qn] = __builtin_bit_cast(Frag, u);
          }
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) {
            const int dim = dt * 16 + c16;
            const Frag vf = *reinterpret_cast<const Frag*>(vb + vidx(np, dim, 4 * quad));  // pages np, np + 1
#pragma unroll
            for (int qn = 0; qn < QN; ++qn) o[dt][qn] = M::mma(vf, pf[qn], o[dt][qn]);
          }
        }
      } else {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int r = 0; r < 4; ++r)  // one key (nt, 4 quad + r) per lane per MFMA
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
              const Frag vf = vb[vidx(nt, dt * 16 + c16, 4 * quad + r)];
#pragma unroll
              for (int qn = 0; qn < QN; ++qn) o[dt][qn] = M::mma(vf, s[nt][qn][r], o[dt][qn]);
            }
      }
    }
  };
  if constexpr (sizeof(T) == 2) {
    // tile kt is used from LDS while tile kt + 1 waits in registers and tile
    // kt + 2 is being loaded, so a load has two tiles of work to arrive.
    // Loads past the last tile reread its pages (clamped) and are never
    // skipped, so the wait before a store counts exactly the one tile issued
    // after it.
    load_tile(0, pa);
    load_tile(1, pb);
    store_tile(0, 0, pa);
    __syncthreads();
    for (int kt = 0; kt < nkt; kt += 2) {
      load_tile(kt + 2, pa);
      use_tile(kt, 0);
      if (kt + 1 < nkt) store_tile(kt + 1, 1, pb);
      __syncthreads();
      if (kt + 1 < nkt) {
        load_tile(kt + 3, pb);
        use_tile(kt + 1, 1);
        if (kt + 2 < nkt) store_tile(kt + 2, 0, pa);
        __syncthreads();
      }
    }
  } else {  // float32: one tile ahead (two would spill at D = 128)
    load_tile(0, pa);
    store_tile(0, 0, pa);
    __syncthreads();
    for (int kt = 0; kt < nkt; ++kt) {
      if (kt + 1 < nkt) load_tile(kt + 1, pa);
      use_tile(kt, kt & 1);
      if (kt + 1 < nkt) store_tile(kt + 1, (kt & 1) ^ 1, pa);
      __syncthreads();
    }
  }
  // the four lane quads hold different keys: add their softmax sums, then
  // write o[query][dims 4 quad .. 4 quad + 3] of every dimension tile
#pragma unroll
  for (int qn = 0; qn < QN; ++qn) {
    float lt = lq[qn];
    lt = sum_xor32(sum_xor16(lt));
    const int row = q0 + w * QW + qn * 16 + c16;
    if (row >= nq) continue;
    const int64_t oo = ((int64_t)g * a.T + row) * a.d + h * D + 4 * quad;
    const float inv = 1.f / lt;
    if (a.o16) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        *reinterpret_cast<uint2*>(a.o16 + oo + dt * 16) =
            make_uint2(pack_bf16x2(o[dt][qn][0] * inv, o[dt][qn][1] * inv),
                       pack_bf16x2(o[dt][qn][2] * inv, o[dt][qn][3] * inv));
    } else {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        *reinterpret_cast<float4*>(a.o + oo + dt * 16) =
            make_float4(o[dt][qn][0] * inv, o[dt][qn][1] * inv, o[dt][qn][2] * inv, o[dt][qn][3] * inv);
    }
  }
}

}  // namespace

template <typename T, int D>
hipError_t launch_decode_d(const AttnDecodeArgs& a, hipStream_t s) {
  const dim3 grid(a.grid > 0 ? a.grid : 1);
  switch (a.waves) {
    case 4: hipLaunchKernelGGL((k_attn_decode<T, D, 4>), grid, dim3(256), 0, s, a); break;
    case 8: hipLaunchKernelGGL((k_attn_decode<T, D, 8>), grid, dim3(512), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T, int D>
hipError_t occupancy_d(int waves, int* blocks) {
  switch (waves) {
    case 4: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, k_attn_decode<T, D, 4>, 256, 0);
    case 8: return hipOccupancyMaxActiveBlocksPerMultiprocessor(blocks, k_attn_decode<T, D, 8>, 512, 0);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t launch_attn_decode(const AttnDecodeArgs& a, hipStream_t s) {
  switch (a.c.D) {
    case 16:
      if constexpr (sizeof(T) == 4) return launch_decode_d<T, 16>(a, s);
      return hipErrorInvalidValue;
    case 64: return launch_decode_d<T, 64>(a, s);
    case 128: return launch_decode_d<T, 128>(a, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t attn_decode_blocks_per_cu(int D, int waves, int* blocks) {
  switch (D) {
    case 16:
      if constexpr (sizeof(T) == 4) return occupancy_d<T, 16>(waves, blocks);
      return hipErrorInvalidValue;
    case 64: return occupancy_d<T, 64>(waves, blocks);
    case 128: return occupancy_d<T, 128>(waves, blocks);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t launch_attn_prefill(const AttnPrefillArgs& a, hipStream_t s) {
  const int BQ = kPreWaves * kPreQW;
  const int QT = (a.T + BQ - 1) / BQ;
  const dim3 grid(a.G * QT * a.c.H), block(kPreWaves * kWave);
  if (a.G <= 0) return hipSuccess;
  switch (a.c.D) {
    case 16:
      // a 16-wide head needs the 4-deep f32 MFMA; bf16 models reject head_dim 16
      if constexpr (sizeof(T) == 4) {
        hipLaunchKernelGGL((k_attn_prefill<T, 16, true>), grid, block, 0, s, a);
        break;
      } else {
        return hipErrorInvalidValue;
      }
    case 64:
      if (sizeof(T) == 2 && a.q_single) hipLaunchKernelGGL((k_attn_prefill<T, 64, false>), grid, block, 0, s, a);
      else hipLaunchKernelGGL((k_attn_prefill<T, 64, true>), grid, block, 0, s, a);
      break;
    case 128:
      if (sizeof(T) == 2 && a.q_single) hipLaunchKernelGGL((k_attn_prefill<T, 128, false>), grid, block, 0, s, a);
      else hipLaunchKernelGGL((k_attn_prefill<T, 128, true>), grid, block, 0, s, a);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template hipError_t attn_decode_blocks_per_cu<float>(int, int, int*);
template hipError_t attn_decode_blocks_per_cu<bf16>(int, int, int*);
template hipError_t launch_attn_decode<float>(const AttnDecodeArgs&, hipStream_t);
template hipError_t launch_attn_decode<bf16>(const AttnDecodeArgs&, hipStream_t);
template hipError_t launch_attn_prefill<float>(const AttnPrefillArgs&, hipStream_t);
template hipError_t launch_attn_prefill<bf16>(const AttnPrefillArgs&, hipStream_t);

}  // namespace tlf
