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
// sequence.  One workgroup per (sequence, 64-query tile, head); K tiles and
// transposed V tiles of 64 keys are gathered from the pages into LDS and
// both products run on MFMA with an online softmax.
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

__device__ __forceinline__ float merge_scale(float m, float mn) {
  return m == kNegInf ? 0.f : exp2f(m - mn);
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
    const int L = c.cache_len[b * R + i];
    const int np = (L + kPage - 1) / kPage;
    const int32_t* pt = c.page_table + ((int64_t)b * R + i) * c.pages_per_seq;
    __syncthreads();  // the previous unit is done with s_pages and s_red
    for (int p = threadIdx.x; p < np; p += W * kWave) s_pages[p] = pt[p];
    __syncthreads();

    // this wave's pages [p0, p1), a multiple of PPI pages each
    const int per = ((np + W - 1) / W + PPI - 1) / PPI * PPI;
    const int p0 = w * per, p1 = min(np, p0 + per);
    const int64_t koff = k_block(c, a.layer, h) + (int64_t)(quad * kPage + c16) * EPL;  // fragment order
    const int64_t voff = v_block(c, a.layer, h) + (int64_t)c16 * kPage + quad * 4;

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
        const int64_t off = voff + (int64_t)dt * 16 * kPage;
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
#pragma unroll
      for (int p = 0; p < PPI; ++p) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks)
#pragma unroll
          for (int qa = 0; qa < NQ; ++qa) acc = M::mma(bk[p][ks], qf[qa][ks], acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = (pg + p) * kPage + 4 * quad + r;
          const bool ok = (pg + p) < p1 && t < L;
          sc[p][r] = ok ? acc[r] * a.scale_log2 : kNegInf;
          mx = fmaxf(mx, sc[p][r]);
        }
      }
      mx = fmaxf(mx, shfl_xor(mx, 16));
      mx = fmaxf(mx, shfl_xor(mx, 32));
      if (mx == kNegInf) return;  // wave-uniform: nothing valid yet
      const float alpha = merge_scale(m, mx);
      lsum *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
      float pr[PPI][4];
#pragma unroll
      for (int p = 0; p < PPI; ++p)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pr[p][r] = exp2f(sc[p][r] - mx);  // 0 for masked slots
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
        load(ka, va, p0);
        for (int pg = p0; pg < p1; pg += 2 * PPI) {
          load(kb, vb2, pg + PPI);
          consume(ka, va, pg);
          load(ka, va, pg + 2 * PPI);
          consume(kb, vb2, pg + PPI);
        }
      } else {
        for (int pg = p0; pg < p1; pg += PPI) {
          load(ka, va, pg);
          consume(ka, va, pg);
        }
      }
    }
    // the four lane quads hold different tokens: add their softmax sums
    lsum += shfl_xor(lsum, 16);
    lsum += shfl_xor(lsum, 32);
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
        a.o[(int64_t)k * a.d + h * D + dim] = Ls > 0.f ? O / Ls : 0.f;
      }
    }
  }
}

template <typename T, int D>
__global__ __launch_bounds__(256) void k_attn_prefill(AttnPrefillArgs a) {
  using M = Mfma<T>;
  constexpr int KS = M::KS, EPL = M::EPL;
  constexpr int BQ = 64, BKEY = 64;
  constexpr int PADT = 16 / (int)sizeof(T);
  constexpr int LDK = D + PADT;
  constexpr int LDV = BKEY + PADT;
  constexpr int LDP = BKEY + PADT;
  constexpr int CPK = D * (int)sizeof(T) / 16;  // 16-byte chunks per key row
  constexpr int EPC = 16 / (int)sizeof(T);
  constexpr int DT = D / 16;
  __shared__ __align__(16) T Ks[BKEY * LDK];
  __shared__ __align__(16) T Vt[D * LDV];
  __shared__ __align__(16) T Ps[4 * 16 * LDP];

  const CacheView& c = a.c;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int quad = lane >> 4, c16 = lane & 15;
  const int QT = (a.T + BQ - 1) / BQ;
  const int g = blockIdx.x / QT, qt = blockIdx.x % QT, h = blockIdx.y;
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

  // q (float32) as the A operand of S = Q K^T; against bf16 keys it is split
  // into hi and lo parts, one product each
  constexpr int NQ = EPL == 8 ? 2 : 1;
  typename M::frag qf[NQ][D / KS];
  {
    const int qrow = min(q0 + w * 16 + c16, nq - 1);
    const float* qp = a.q + ((int64_t)g * a.T + qrow) * a.d + h * D + quad * EPL;
#pragma unroll
    for (int ks = 0; ks < D / KS; ++ks) {
      if constexpr (NQ == 2) split_frag(qp + ks * KS, qf[0][ks], qf[NQ - 1][ks]);
      else qf[0][ks] = qp[ks * KS];
    }
  }
  f32x4 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrow[4], lrow[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) { mrow[r] = kNegInf; lrow[r] = 0.f; }

  const int nkt = min((n0 + q0 + BQ + BKEY - 1) / BKEY, (n + BKEY - 1) / BKEY);
  for (int kt = 0; kt < nkt; ++kt) {
    __syncthreads();
    // K rows: key-major, 16-byte pieces
    for (int ci = tid; ci < BKEY * CPK; ci += 256) {
      const int key = ci / CPK, col = (ci % CPK) * EPC;
      const int ka = kt * BKEY + key;
      V16<T> kv;
      kv.u = make_uint4(0, 0, 0, 0);
      if (ka < n) {
        const T* kb = pool + (int64_t)pt[ka / kPage] * c.page_elems + koff;
        if constexpr (EPC == EPL) {
          kv = ld16(kb + k_frag_off<T>(ka % kPage, col));  // one fragment: EPL consecutive elements
        } else {
#pragma unroll
          for (int t = 0; t < EPC; ++t) kv.e[t] = kb[k_frag_off<T>(ka % kPage, col + t)];
        }
      }
      st16(&Ks[key * LDK + col], kv);
    }
    // V^T: each page holds [D][16 slots]; a 16-byte piece is EPC slots of one dimension
    constexpr int VPC = kPage / EPC;  // pieces per (page, dimension)
    for (int ci = tid; ci < (BKEY / kPage) * D * VPC; ci += 256) {
      const int pg = ci / (D * VPC), rem = ci % (D * VPC), dim = rem / VPC, piece = rem % VPC;
      const int pa = kt * (BKEY / kPage) + pg;  // page index within the (b, i) cache
      V16<T> vv;
      vv.u = make_uint4(0, 0, 0, 0);
      // slots past n in the last page hold finite stale values; their P is 0
      if (pa < npages)
        vv = ld16(pool + (int64_t)pt[pa] * c.page_elems + voff + (int64_t)dim * kPage + piece * EPC);
      st16(&Vt[dim * LDV + pg * kPage + piece * EPC], vv);
    }
    __syncthreads();

    f32x4 s[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      s[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / KS; ++ks) {
        const typename M::frag kf = M::load(&Ks[(nt * 16 + c16) * LDK + ks * KS + quad * EPL]);
#pragma unroll
        for (int qa = 0; qa < NQ; ++qa) s[nt] = M::mma(qf[qa][ks], kf, s[nt]);
      }
    }
    float alpha[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = n0 + q0 + w * 16 + quad * 4 + r;
      float mx = kNegInf;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int key = kt * BKEY + nt * 16 + c16;
        float v = s[nt][r] * a.scale_log2;
        if (key > row || key >= n) v = kNegInf;
        s[nt][r] = v;
        mx = fmaxf(mx, v);
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, shfl_xor(mx, off));
      const float mn = fmaxf(mrow[r], mx);
      alpha[r] = (mn == kNegInf) ? 1.f : merge_scale(mrow[r], mn);
      float ps = 0.f;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const float p = (s[nt][r] == kNegInf) ? 0.f : exp2f(s[nt][r] - mn);
        s[nt][r] = p;
        ps += p;
      }
      lrow[r] = lrow[r] * alpha[r] + ps;
      mrow[r] = mn;
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 4; ++r) o[dt][r] *= alpha[r];
    T* pw = Ps + w * 16 * LDP;
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) pw[(quad * 4 + r) * LDP + nt * 16 + c16] = from_f<T>(s[nt][r]);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BKEY / KS; ++kk) {
      const typename M::frag pa = M::load(&pw[c16 * LDP + kk * KS + quad * EPL]);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        o[dt] = M::mma(pa, M::load(&Vt[(dt * 16 + c16) * LDV + kk * KS + quad * EPL]), o[dt]);
    }
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    float lt = lrow[r];
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) lt += shfl_xor(lt, off);
    const int row = q0 + w * 16 + quad * 4 + r;
    if (row >= nq) continue;
    float* op = a.o + ((int64_t)g * a.T + row) * a.d + h * D;
    const float inv = 1.f / lt;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) op[dt * 16 + c16] = o[dt][r] * inv;
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
  const int QT = (a.T + 63) / 64;
  const dim3 grid(a.G * QT, a.c.H), block(256);
  if (a.G <= 0) return hipSuccess;
  switch (a.c.D) {
    case 16:
      // a 16-wide head needs the 4-deep f32 MFMA; bf16 models reject head_dim 16
      if constexpr (sizeof(T) == 4) {
        hipLaunchKernelGGL((k_attn_prefill<T, 16>), grid, block, 0, s, a);
        break;
      } else {
        return hipErrorInvalidValue;
      }
    case 64: hipLaunchKernelGGL((k_attn_prefill<T, 64>), grid, block, 0, s, a); break;
    case 128: hipLaunchKernelGGL((k_attn_prefill<T, 128>), grid, block, 0, s, a); break;
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
