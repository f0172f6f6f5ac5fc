// Per-row kernels: embedding + router, and RMSNorm of residual rows.
//
// Both keep the float32 residual row x and write y = RMSNorm(x) (no affine,
// Appendix A), also float32: y is the A operand of the next projection
// (QKV, gate/up, LM head), so the norm is computed once per row instead of
// once per output tile.  Rows of up to 4096 elements stay in
// registers between the sum of squares and the write of y.
#include "kernels.h"

namespace tlf {

namespace {

constexpr int kRowChunks = 16;  // 16 x 256 elements: rows up to 4096 wide
constexpr int kNormChunks = 4;  // 4 x 1024 elements: rows up to 4096 wide (RMSNorm, a workgroup per row)

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Sum over the 64 lanes of a wave; every lane gets the total.
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp<0xB1>(v);   // lane ^ 1
  v += dpp<0x4E>(v);   // lane ^ 2
  v += dpp<0x141>(v);  // other quad of the 8
  v += dpp<0x140>(v);  // other half of the 16
  v += shfl_xor(v, 16);
  v += shfl_xor(v, 32);
  return v;
}

template <typename T> struct V4;  // 4 storage elements
template <> struct V4<float> {
  static __device__ __forceinline__ float4 load(const float* p) { return *reinterpret_cast<const float4*>(p); }
  static __device__ __forceinline__ void store(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
};
template <> struct V4<bf16> {
  static __device__ __forceinline__ float4 load(const bf16* p) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
  }
  static __device__ __forceinline__ void store(bf16* p, float4 v) {
    union { bf16 h[4]; uint2 u; } o;
    o.h[0] = (bf16)v.x; o.h[1] = (bf16)v.y; o.h[2] = (bf16)v.z; o.h[3] = (bf16)v.w;
    *reinterpret_cast<uint2*>(p) = o.u;
  }
};

__device__ __forceinline__ float sumsq(float4 v, float acc) {
  return fmaf(v.w, v.w, fmaf(v.z, v.z, fmaf(v.y, v.y, fmaf(v.x, v.x, acc))));
}
__device__ __forceinline__ float4 scale4(float4 v, float s) { return make_float4(v.x * s, v.y * s, v.z * s, v.w * s); }

// Routed depth m in [1, R] and decision margin from router logits z (Eq. 2-5):
// rule 0 argmax (lowest on ties), 1 cumulative probability with a strict
// threshold and p^(1) = 1, 2 fixed depth.
__device__ void decide_depth(const float* z, int R, int rule, float threshold, int fixed, int* m_out,
                             float* margin_out) {
  int m = 1;
  float margin = __builtin_inff();
  if (rule == 0) {  // argmax, lowest index on ties
    int best = 0;
    for (int i = 1; i < R; ++i)
      if (z[i] > z[best]) best = i;
    float second = -__builtin_inff();
    for (int i = 0; i < R; ++i)
      if (i != best && z[i] > second) second = z[i];
    m = best + 1;
    if (R > 1) margin = z[best] - second;
  } else if (rule == 1) {  // cumulative probability (Eq. 2-5)
    float mx = z[0];
    for (int i = 1; i < R; ++i) mx = fmaxf(mx, z[i]);
    float ex[kMaxLoops];
    float tot = 0.f;
    for (int i = 0; i < R; ++i) { ex[i] = __expf(z[i] - mx); tot += ex[i]; }
    float p_sfx[kMaxLoops + 1];
    p_sfx[R] = 0.f;
    float run = 0.f;
    for (int i = R - 1; i >= 0; --i) { run += ex[i]; p_sfx[i] = run / tot; }
    p_sfx[0] = 1.f;  // p^(1) = 1: every token runs loop 1
    m = 1;
    for (int i = 1; i < R; ++i)
      if (p_sfx[i] > threshold) m = i + 1;
    margin = fminf(p_sfx[m - 1] - threshold, threshold - p_sfx[m]);
  } else {
    m = fixed;
  }
  *m_out = m;
  *margin_out = margin;
}

// Row kernels take the number of 256-element chunks of a row (NC) as a
// template argument and load every chunk unconditionally, the element index
// clamped into the row (the tail's surplus lanes read the row's last four
// elements, finite values, and multiply them by zero: a select would let the
// compiler move each load under a branch again), so all of a row's loads are
// in flight at once instead of one guarded chunk after another.
__device__ __forceinline__ int clamp_k(int k, int n) { return k < n ? k : n - 4; }

// ---------------------------------------------------------------------------
// h0 = E[x] + P[pos] (learned absolute position added once, Section 3.2),
// z = W_r h0 + b_r (Eq. 2's router as a linear map), the depth rule, and
// y = RMSNorm(h0) for the first projection.  One wave per row; lane l holds
// elements 4l + 256c.
// ---------------------------------------------------------------------------
template <typename T, int NC>
__global__ __launch_bounds__(256) void k_embed_route(EmbedArgs a) {
  const int lane = lane_id();
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= a.rows) return;
  // both row reads in one round trip (prefill reads its token twice instead
  // of a branch around the sequence length)
  int tok = a.tokens[row];
  const int sl = (a.prefill_T > 0 ? a.tokens : a.seq_len)[row];
  if (tok < 0 || tok >= a.V) {
    if (lane == 0) set_err(a.err, kErrBadToken);
    tok = 0;
  }
  const int pos = a.prefill_T > 0 ? a.pos0 + row % a.prefill_T : sl;
  const T* e = reinterpret_cast<const T*>(a.tok_emb) + (int64_t)tok * a.d;
  const T* p = reinterpret_cast<const T*>(a.pos_emb) + (int64_t)pos * a.d;
  float* x = a.x + (int64_t)row * a.d;
  float4 h[NC];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int k = 4 * lane + 256 * c, kk = clamp_k(k, a.d);
    const float4 ev = V4<T>::load(e + kk), pv = V4<T>::load(p + kk);
    h[c] = scale4(make_float4(ev.x + pv.x, ev.y + pv.y, ev.z + pv.z, ev.w + pv.w), k < a.d ? 1.f : 0.f);
    ss = sumsq(h[c], ss);
  }
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int k = 4 * lane + 256 * c;
    if (k < a.d) V4<float>::store(x + k, h[c]);
  }
  ss = wave_sum(ss);
  const float inv = rsqrtf(ss / (float)a.d + a.eps);
  if (a.y) {
    float* y = a.y + (int64_t)row * a.d;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int k = 4 * lane + 256 * c;
      if (k < a.d) V4<float>::store(y + k, scale4(h[c], inv));
    }
  }
  if (a.y16) {
    bf16* y = a.y16 + (int64_t)row * a.d;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int k = 4 * lane + 256 * c;
      const float4 v = scale4(h[c], inv);
      if (k < a.d) *reinterpret_cast<uint2*>(y + k) = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
    }
  }
  if (!a.route) return;  // the MLP router runs after this kernel
  float z[kMaxLoops];
#pragma unroll
  for (int i = 0; i < kMaxLoops; ++i) {
    // rows of W_r past R repeat row 0; their sums are never used
    const float* wr = a.Wr + (int64_t)(i < a.R ? i : 0) * a.d;
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const float4 w = V4<float>::load(wr + clamp_k(4 * lane + 256 * c, a.d));
      acc = fmaf(w.w, h[c].w, fmaf(w.z, h[c].z, fmaf(w.y, h[c].y, fmaf(w.x, h[c].x, acc))));
    }
    z[i] = acc;
  }
#pragma unroll
  for (int i = 0; i < kMaxLoops; ++i)
    if (i < a.R) z[i] = wave_sum(z[i]) + a.br[i];
  if (lane != 0) return;
  int m;
  float margin;
  decide_depth(z, a.R, a.rule, a.threshold, a.fixed, &m, &margin);
  a.depth[row] = m;
  if (a.out_depth) a.out_depth[row] = m;
  if (a.out_margin) a.out_margin[row] = margin;
}

// ---------------------------------------------------------------------------
// Output layer of the MLP router on hidden rows (z = W_r h + b_r), then the
// depth rule.  One wave per row; lane l holds elements 4l + 256c.
// ---------------------------------------------------------------------------
template <int NC>
__global__ __launch_bounds__(256) void k_route_rows(RouteArgs a) {
  const int lane = lane_id();
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= a.rows) return;
  const float* h = a.h + (int64_t)row * a.Hr;
  float4 hv[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int k = 4 * lane + 256 * c;
    hv[c] = scale4(V4<float>::load(h + clamp_k(k, a.Hr)), k < a.Hr ? 1.f : 0.f);
  }
  float z[kMaxLoops];
#pragma unroll
  for (int i = 0; i < kMaxLoops; ++i) {
    const float* wr = a.Wr + (int64_t)(i < a.R ? i : 0) * a.Hr;
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const float4 w = V4<float>::load(wr + clamp_k(4 * lane + 256 * c, a.Hr));
      acc = fmaf(w.w, hv[c].w, fmaf(w.z, hv[c].z, fmaf(w.y, hv[c].y, fmaf(w.x, hv[c].x, acc))));
    }
    z[i] = acc;
  }
#pragma unroll
  for (int i = 0; i < kMaxLoops; ++i)
    if (i < a.R) z[i] = wave_sum(z[i]) + a.br[i];
  if (lane != 0) return;
  int m;
  float margin;
  decide_depth(z, a.R, a.rule, a.threshold, a.fixed, &m, &margin);
  a.depth[row] = m;
  if (a.out_depth) a.out_depth[row] = m;
  if (a.out_margin) a.out_margin[row] = margin;
}

// ---------------------------------------------------------------------------
// y[src(r)] = RMSNorm(x[src(r)]) for the active rows of a row map (prefill,
// after each residual projection).  One wave per row, four rows per
// workgroup (most rows of the later loops are inactive, and a row's wave
// leaves at once).  Lane l holds elements 4 (l + 64 v) + 1024 c, v < 4,
// c < NC: those of threads l + 64 v of a 256-thread row.  Its sum of squares
// is taken as such a row would take it: per thread over c, over the 64
// lanes for each v, then the four partials in pairs.
// ---------------------------------------------------------------------------
template <int NC>
__global__ __launch_bounds__(256) void k_resid_norm(ResidNormArgs a) {
  const int lane = lane_id();
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (!row_active(a.rm, r)) return;
  const int src = row_src(a.rm, r);
  const float* x = a.x + (int64_t)src * a.d;
  float4 h[4][NC];
  float ps[4];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    ps[v] = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int k = 4 * (lane + 64 * v) + 1024 * c;
      h[v][c] = scale4(V4<float>::load(x + clamp_k(k, a.d)), k < a.d ? 1.f : 0.f);
      ps[v] = sumsq(h[v][c], ps[v]);
    }
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) ps[v] = wave_sum(ps[v]);
  const float ss = (ps[0] + ps[1]) + (ps[2] + ps[3]);
  const float inv = rsqrtf(ss / (float)a.d + a.eps);
  if (a.y) {
    float* y = a.y + (int64_t)src * a.d;
#pragma unroll
    for (int v = 0; v < 4; ++v)
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int k = 4 * (lane + 64 * v) + 1024 * c;
        if (k < a.d) V4<float>::store(y + k, scale4(h[v][c], inv));
      }
  }
  if (a.y16) {
    bf16* y16 = a.y16 + (int64_t)src * a.d;
#pragma unroll
    for (int v = 0; v < 4; ++v)
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int k = 4 * (lane + 64 * v) + 1024 * c;
        const float4 hv = scale4(h[v][c], inv);
        if (k < a.d) *reinterpret_cast<uint2*>(y16 + k) = make_uint2(pack_bf16x2(hv.x, hv.y), pack_bf16x2(hv.z, hv.w));
      }
  }
}

}  // namespace

// Launches kernel K<NC> for NC = n, 1 <= n <= 16.
#define TLF_NC_SWITCH(n, LAUNCH)                                                                   \
  switch (n) {                                                                                     \
    case 1: LAUNCH(1); break;   case 2: LAUNCH(2); break;   case 3: LAUNCH(3); break;             \
    case 4: LAUNCH(4); break;   case 5: LAUNCH(5); break;   case 6: LAUNCH(6); break;             \
    case 7: LAUNCH(7); break;   case 8: LAUNCH(8); break;   case 9: LAUNCH(9); break;             \
    case 10: LAUNCH(10); break; case 11: LAUNCH(11); break; case 12: LAUNCH(12); break;           \
    case 13: LAUNCH(13); break; case 14: LAUNCH(14); break; case 15: LAUNCH(15); break;           \
    case 16: LAUNCH(16); break;                                                                    \
    default: return hipErrorInvalidValue;                                                          \
  }

template <typename T> hipError_t launch_embed_route(const EmbedArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (a.d <= 0 || a.d % 4 != 0 || a.d > 256 * kRowChunks) return hipErrorInvalidValue;
#define TLF_EMBED(NC) hipLaunchKernelGGL((k_embed_route<T, NC>), dim3((a.rows + 3) / 4), dim3(256), 0, s, a)
  TLF_NC_SWITCH((a.d + 255) / 256, TLF_EMBED)
#undef TLF_EMBED
  return hipGetLastError();
}
template hipError_t launch_embed_route<float>(const EmbedArgs&, hipStream_t);
template hipError_t launch_embed_route<bf16>(const EmbedArgs&, hipStream_t);

template <typename T> hipError_t launch_resid_norm(const ResidNormArgs& a, hipStream_t s) {
  if (a.rm.rows <= 0) return hipSuccess;
  if (a.d <= 0 || a.d % 4 != 0 || a.d > 1024 * kNormChunks) return hipErrorInvalidValue;
#define TLF_NORM(NC) hipLaunchKernelGGL((k_resid_norm<NC>), dim3((a.rm.rows + 3) / 4), dim3(256), 0, s, a)
  switch ((a.d + 1023) / 1024) {
    case 1: TLF_NORM(1); break;
    case 2: TLF_NORM(2); break;
    case 3: TLF_NORM(3); break;
    default: TLF_NORM(4); break;
  }
#undef TLF_NORM
  return hipGetLastError();
}
template hipError_t launch_resid_norm<float>(const ResidNormArgs&, hipStream_t);
template hipError_t launch_resid_norm<bf16>(const ResidNormArgs&, hipStream_t);

hipError_t launch_route_rows(const RouteArgs& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (a.Hr <= 0 || a.Hr > 4 * kWave * kRowChunks || a.Hr % 4 != 0) return hipErrorInvalidValue;
#define TLF_ROUTE(NC) hipLaunchKernelGGL((k_route_rows<NC>), dim3((a.rows + 3) / 4), dim3(256), 0, s, a)
  TLF_NC_SWITCH((a.Hr + 255) / 256, TLF_ROUTE)
#undef TLF_ROUTE
  return hipGetLastError();
}
#undef TLF_NC_SWITCH

}  // namespace tlf
