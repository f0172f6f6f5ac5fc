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

__device__ __forceinline__ float merge_scale(float m, float mn) {
  return m == kNegInf ? 0.f : exp2f(m - mn);
}

// Sum over aligned groups of G lanes (G = 2, 4, 8, 16, 32) with DPP moves
// inside rows of 16 lanes and a shuffle beyond them.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

template <int G>
__device__ __forceinline__ float group_sum(float v) {
  if constexpr (G >= 2) v += dpp_mov<0xB1>(v);   // quad_perm [1,0,3,2]: partner lane ^ 1
  if constexpr (G >= 4) v += dpp_mov<0x4E>(v);   // quad_perm [2,3,0,1]: partner lane ^ 2
  if constexpr (G >= 8) v += dpp_mov<0x141>(v);  // row_half_mirror: the other quad of the 8
  if constexpr (G >= 16) v += dpp_mov<0x140>(v); // row_mirror: the other half of the 16
  if constexpr (G >= 32) v += shfl_xor(v, 16);
  return v;
}

template <typename T, int D, int W>
__global__ __launch_bounds__(W * 64) void k_attn_decode(AttnDecodeArgs a) {
  constexpr int EPL = 16 / (int)sizeof(T);  // elements per 16-byte load
  constexpr int G = D / EPL;                // lanes per token
  constexpr int TPI = kWave / G;            // tokens per wave instruction
  constexpr int U = 4;                      // tokens per lane per load batch
  constexpr int STEP = U * TPI;             // tokens per wave per batch
  static_assert(G >= 1 && G <= 32 && kWave % G == 0, "head_dim split");
  __shared__ int s_pages[kAttnMaxPages];
  __shared__ float s_red[W][D + 2];

  const CacheView& c = a.c;
  const int lane = lane_id(), w = threadIdx.x >> 6;
  const int tr = lane / G, gl = lane % G;
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

    // this wave's contiguous share of the L entries
    const int per = ((L + W - 1) / W + TPI - 1) / TPI * TPI;
    const int t0 = w * per, t1 = min(L, t0 + per);
    const int64_t koff = page_off(c, a.layer, 0, h, 0) + gl * EPL;
    const int64_t voff = page_off(c, a.layer, 1, h, 0) + gl * EPL;
    const V16<T> qv = ld16(reinterpret_cast<const T*>(a.q) + (int64_t)k * a.d + h * D + gl * EPL);
    float qf[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) qf[e] = to_f<T>(qv.e[e]) * a.scale_log2;

    float m = kNegInf, l = 0.f, acc[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] = 0.f;

    auto load = [&](V16<T>* kr, V16<T>* vr, int tb) {
#pragma unroll
      for (int uu = 0; uu < U; ++uu) {
        const int t = tb + uu * TPI + tr;
        const int tt = t < t1 ? t : t0;  // lanes past the end read a valid slot
        const int64_t base = (int64_t)s_pages[tt >> 4] * c.page_elems + (tt & (kPage - 1)) * D;
        kr[uu] = ld16(pool + base + koff);
        vr[uu] = ld16(pool + base + voff);
      }
    };
    auto consume = [&](const V16<T>* kr, const V16<T>* vr, int tb) {
      float s[U];
      float mx = m;
#pragma unroll
      for (int uu = 0; uu < U; ++uu) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) d = fmaf(qf[e], to_f<T>(kr[uu].e[e]), d);
        d = group_sum<G>(d);
        s[uu] = (tb + uu * TPI + tr < t1) ? d : kNegInf;
        mx = fmaxf(mx, s[uu]);
      }
      if (mx != kNegInf) {
        const float alpha = merge_scale(m, mx);
        l *= alpha;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] *= alpha;
#pragma unroll
        for (int uu = 0; uu < U; ++uu) {
          const float p = exp2f(s[uu] - mx);  // exp2(-inf) = 0 for masked slots
          l += p;
#pragma unroll
          for (int e = 0; e < EPL; ++e) acc[e] = fmaf(p, to_f<T>(vr[uu].e[e]), acc[e]);
        }
        m = mx;
      }
    };
    if (t0 < t1) {
      // two register batches in flight: the next batch loads while this one is consumed
      V16<T> ka[U], va[U], kb[U], vb[U];
      load(ka, va, t0);
      for (int tb = t0; tb < t1; tb += 2 * STEP) {
        if (tb + STEP < t1) load(kb, vb, tb + STEP);
        consume(ka, va, tb);
        if (tb + STEP >= t1) break;
        if (tb + 2 * STEP < t1) load(ka, va, tb + 2 * STEP);
        consume(kb, vb, tb + STEP);
      }
    }
    // merge the TPI token slots that share this lane's dimension slice
#pragma unroll
    for (int o = G; o < kWave; o <<= 1) {
      const float m2 = shfl_xor(m, o), l2 = shfl_xor(l, o);
      const float mn = fmaxf(m, m2);
      const float a1 = merge_scale(m, mn), a2 = merge_scale(m2, mn);
      l = l * a1 + l2 * a2;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] = acc[e] * a1 + shfl_xor(acc[e], o) * a2;
      m = mn;
    }
    if (tr == 0) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) s_red[w][2 + gl * EPL + e] = acc[e];
      if (gl == 0) { s_red[w][0] = m; s_red[w][1] = l; }
    }
    __syncthreads();
    // merge the W waves' partial softmax states (log-sum-exp) and write o
    if (w == 0 && tr == 0) {
      float M = kNegInf, Ls = 0.f, O[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) O[e] = 0.f;
#pragma unroll
      for (int ww = 0; ww < W; ++ww) {
        const float mc = s_red[ww][0], lc = s_red[ww][1];
        const float mn = fmaxf(M, mc);
        const float a1 = merge_scale(M, mn), a2 = merge_scale(mc, mn);
        Ls = Ls * a1 + lc * a2;
#pragma unroll
        for (int e = 0; e < EPL; ++e) O[e] = O[e] * a1 + s_red[ww][2 + gl * EPL + e] * a2;
        M = mn;
      }
      V16<T> ov;
      const float inv = 1.f / Ls;
#pragma unroll
      for (int e = 0; e < EPL; ++e) ov.e[e] = from_f<T>(O[e] * inv);
      st16(reinterpret_cast<T*>(a.o) + (int64_t)k * a.d + h * D + gl * EPL, ov);
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
  const int n = c.cache_len[b * c.R + a.loop];
  const int q0 = qt * BQ;
  if (q0 >= n) return;
  const int32_t* pt = c.page_table + ((int64_t)b * c.R + a.loop) * c.pages_per_seq;
  const T* pool = reinterpret_cast<const T*>(c.pool);
  const int64_t koff = page_off(c, a.layer, 0, h, 0), voff = page_off(c, a.layer, 1, h, 0);

  typename M::frag qf[D / KS];
  {
    const int qrow = min(q0 + w * 16 + c16, n - 1);
    const T* qp = reinterpret_cast<const T*>(a.q) + ((int64_t)g * a.T + qrow) * a.d + h * D;
#pragma unroll
    for (int ks = 0; ks < D / KS; ++ks) qf[ks] = M::load(qp + ks * KS + quad * EPL);
  }
  f32x4 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrow[4], lrow[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) { mrow[r] = kNegInf; lrow[r] = 0.f; }

  const int nkt = min(qt + 1, (n + BKEY - 1) / BKEY);
  for (int kt = 0; kt < nkt; ++kt) {
    __syncthreads();
    for (int ci = tid; ci < BKEY * CPK; ci += 256) {
      const int key = ci / CPK, col = (ci % CPK) * EPC;
      const int ka = kt * BKEY + key;
      V16<T> kv, vv;
      if (ka < n) {
        const int64_t pb = (int64_t)pt[ka / kPage] * c.page_elems + (ka % kPage) * D + col;
        kv = ld16(pool + pb + koff);
        vv = ld16(pool + pb + voff);
      } else {
        kv.u = make_uint4(0, 0, 0, 0);
        vv.u = make_uint4(0, 0, 0, 0);
      }
      st16(&Ks[key * LDK + col], kv);
#pragma unroll
      for (int e = 0; e < EPC; ++e) Vt[(col + e) * LDV + key] = vv.e[e];
    }
    __syncthreads();

    f32x4 s[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
      s[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < D / KS; ++ks)
        s[nt] = M::mma(qf[ks], M::load(&Ks[(nt * 16 + c16) * LDK + ks * KS + quad * EPL]), s[nt]);
    }
    float alpha[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = q0 + w * 16 + quad * 4 + r;
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
    if (row >= n) continue;
    T* op = reinterpret_cast<T*>(a.o) + ((int64_t)g * a.T + row) * a.d + h * D;
    const float inv = 1.f / lt;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) op[dt * 16 + c16] = from_f<T>(o[dt][r] * inv);
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
