// Attention over the recursion-wise KV cache (Eq. 10).
//
// Decode: a query at loop i reads only cache (b, i), i.e. the earlier tokens
// of its sequence whose depth is >= i plus itself; exited tokens have no
// slot, so the validity mask is implicit.  Each (row, head, chunk of pages)
// is one wave-unit of a persistent grid; K and V stream from HBM in 16-byte
// loads (G lanes per token, 64/G tokens per instruction, U tokens per lane in
// flight), every lane keeps its own online-softmax state, lanes merge with
// shuffles, and chunks of one (row, head) merge through a log-sum-exp
// combine done by the last-arriving wave.
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

template <typename T, int D>
__global__ __launch_bounds__(256) void k_attn_decode(AttnDecodeArgs a) {
  constexpr int EPL = 16 / (int)sizeof(T);  // elements per 16-byte load
  constexpr int G = D / EPL;                // lanes per token
  constexpr int TPI = kWave / G;            // tokens per wave instruction
  constexpr int U = 8;                      // tokens per lane per iteration
  static_assert(G >= 1 && G <= kWave && kWave % G == 0, "head_dim split");

  const CacheView& c = a.c;
  const int lane = lane_id();
  const int tr = lane / G, gl = lane % G;
  const int H = c.H, R = c.R, i = a.loop;
  const int nunits = *a.unit_count * H;
  const int CT = *a.chunk_tokens;
  const int nwaves = gridDim.x * 4;
  const T* pool = reinterpret_cast<const T*>(c.pool);

  for (int u = blockIdx.x * 4 + (threadIdx.x >> 6); u < nunits; u += nwaves) {
    const int ent = a.units[u / H];
    const int h = u % H;
    const int k = ent & 0xFFFF, ch = ent >> 16;
    const int b = a.perm[k];
    const int L = c.cache_len[b * R + i];
    const int t0 = ch * CT;
    const int t1 = min(L, t0 + CT);
    const int32_t* pt = c.page_table + ((int64_t)b * R + i) * c.pages_per_seq;
    const int64_t koff = page_off(c, a.layer, 0, h, 0) + gl * EPL;
    const int64_t voff = page_off(c, a.layer, 1, h, 0) + gl * EPL;

    const V16<T> qv = ld16(reinterpret_cast<const T*>(a.q) + (int64_t)k * a.d + h * D + gl * EPL);
    float qf[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) qf[e] = to_f<T>(qv.e[e]) * a.scale_log2;

    float m = kNegInf, l = 0.f, acc[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[e] = 0.f;

    for (int tb = t0; tb < t1; tb += U * TPI) {
      V16<T> kr[U], vr[U];
      bool ok[U];
#pragma unroll
      for (int uu = 0; uu < U; ++uu) {
        const int t = tb + uu * TPI + tr;
        ok[uu] = t < t1;
        const int tt = ok[uu] ? t : t0;  // masked lanes read a valid slot
        const int64_t base = (int64_t)pt[tt / kPage] * c.page_elems + (tt % kPage) * D;
        kr[uu] = ld16(pool + base + koff);
        vr[uu] = ld16(pool + base + voff);
      }
      float s[U];
#pragma unroll
      for (int uu = 0; uu < U; ++uu) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) d += qf[e] * to_f<T>(kr[uu].e[e]);
#pragma unroll
        for (int o = 1; o < G; o <<= 1) d += shfl_xor(d, o);
        s[uu] = ok[uu] ? d : kNegInf;
      }
      float mx = m;
#pragma unroll
      for (int uu = 0; uu < U; ++uu) mx = fmaxf(mx, s[uu]);
      if (mx == kNegInf) continue;  // nothing valid for this lane yet
      const float alpha = merge_scale(m, mx);
      l *= alpha;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[e] *= alpha;
#pragma unroll
      for (int uu = 0; uu < U; ++uu) {
        const float p = ok[uu] ? exp2f(s[uu] - mx) : 0.f;
        l += p;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] += p * to_f<T>(vr[uu].e[e]);
      }
      m = mx;
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
    const int nc = a.nchunks[k];
    T* orow = reinterpret_cast<T*>(a.o) + (int64_t)k * a.d + h * D + gl * EPL;
    if (nc == 1) {
      if (tr == 0) {
        V16<T> ov;
        const float inv = 1.f / l;
#pragma unroll
        for (int e = 0; e < EPL; ++e) ov.e[e] = from_f<T>(acc[e] * inv);
        st16(orow, ov);
      }
      continue;
    }
    const int64_t pstride = D + 2;
    float* part = a.partial + (((int64_t)k * H + h) * a.max_chunks + ch) * pstride;
    if (tr == 0) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) part[2 + gl * EPL + e] = acc[e];
      if (gl == 0) { part[0] = m; part[1] = l; }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    int old = 0;
    if (lane == 0)
      old = __hip_atomic_fetch_add(&a.counters[k * H + h], 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    old = __shfl(old, 0, kWave);
    if (old != nc - 1) continue;
    // last chunk of this (row, head) to finish: merge all partials
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    if (tr == 0) {
      float M = kNegInf, Ls = 0.f, O[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) O[e] = 0.f;
      const float* pp = a.partial + ((int64_t)k * H + h) * a.max_chunks * pstride;
      for (int cc = 0; cc < nc; ++cc, pp += pstride) {
        const float mc = pp[0], lc = pp[1];
        const float mn = fmaxf(M, mc);
        const float a1 = merge_scale(M, mn), a2 = merge_scale(mc, mn);
        Ls = Ls * a1 + lc * a2;
#pragma unroll
        for (int e = 0; e < EPL; ++e) O[e] = O[e] * a1 + pp[2 + gl * EPL + e] * a2;
        M = mn;
      }
      V16<T> ov;
      const float inv = 1.f / Ls;
#pragma unroll
      for (int e = 0; e < EPL; ++e) ov.e[e] = from_f<T>(O[e] * inv);
      st16(orow, ov);
    }
    if (lane == 0) __hip_atomic_store(&a.counters[k * H + h], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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

template <typename T>
hipError_t launch_attn_decode(const AttnDecodeArgs& a, hipStream_t s) {
  const dim3 grid(a.grid > 0 ? a.grid : 1), block(256);
  switch (a.c.D) {
    case 16:
      if constexpr (sizeof(T) == 4) {
        hipLaunchKernelGGL((k_attn_decode<T, 16>), grid, block, 0, s, a);
        break;
      } else {
        return hipErrorInvalidValue;
      }
    case 64: hipLaunchKernelGGL((k_attn_decode<T, 64>), grid, block, 0, s, a); break;
    case 128: hipLaunchKernelGGL((k_attn_decode<T, 128>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
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

template hipError_t launch_attn_decode<float>(const AttnDecodeArgs&, hipStream_t);
template hipError_t launch_attn_decode<bf16>(const AttnDecodeArgs&, hipStream_t);
template hipError_t launch_attn_prefill<float>(const AttnPrefillArgs&, hipStream_t);
template hipError_t launch_attn_prefill<bf16>(const AttnPrefillArgs&, hipStream_t);

}  // namespace tlf
