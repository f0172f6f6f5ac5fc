// AdaLN time/step conditioning tables (Section 3.1, Appendix A), built once
// when a context is created.
//
// A token's modulation depends only on (layer j, loop i, depth m): its
// uniform trajectory gives cumulative time (i - 1) / m and step 1 / m.  So
// every (alpha_msa, alpha_mlp, gamma_msa, gamma_mlp) the block can need is
// tabulated here, [j][i][m][4d] float32 for all R x R (loop, depth) pairs
// (pairs with i > m are computed too and never read), and the decode and
// prefill projections gather one table row per GEMM row.  The table is a few
// MB, computed in float64 accumulation by one thread per output: set-up
// work, not on the decode path.
#include <cmath>

#include "kernels.h"

namespace tlf {

namespace {

constexpr int kFourier = 256;  // Fourier features per conditioning scalar

// Row p < R^2 holds the features of the cumulative time of pair p = i * R + m
// (0-based loop i and depth m + 1): tau = i / (m + 1); row R^2 + p those of
// its step 1 / (m + 1).  Column 2k is cos(tau w_k), 2k + 1 is sin(tau w_k),
// w_k = 10000^(-k / 128) (k 0-based).
__global__ void k_cond_features(float* feat, int R) {
  const int row = blockIdx.x, k = threadIdx.x;
  const int P = R * R, pair = row % P, i = pair / R, m = pair % R + 1;
  const double tau = row < P ? (double)i / m : 1.0 / m;
  const double w = exp(-(double)k / (kFourier / 2) * log(10000.0));
  feat[(int64_t)row * kFourier + 2 * k] = (float)cos(tau * w);
  feat[(int64_t)row * kFourier + 2 * k + 1] = (float)sin(tau * w);
}

__device__ __forceinline__ double silu_d(double x) { return x / (1.0 + exp(-x)); }

// out[p][n] = (acc ? out[p][n] : 0) + g(b[n] + sum_k W[n][k] f(in[p][k])),
// f = silu when silu_in, g = silu when silu_out; W [N][K] storage dtype.
template <typename T>
__global__ void k_cond_linear(const T* W, const float* b, const float* in, float* out, int N, int K,
                              int silu_in, int silu_out, int acc) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x, p = blockIdx.y;
  if (n >= N) return;
  const float* x = in + (int64_t)p * K;
  const T* w = W + (int64_t)n * K;
  double s = b[n];
  for (int k = 0; k < K; ++k) {
    const double v = silu_in ? silu_d((double)x[k]) : (double)x[k];
    s += (double)to_f<T>(w[k]) * v;
  }
  if (silu_out) s = silu_d(s);
  float* o = out + (int64_t)p * N + n;
  *o = (float)(acc ? (double)*o + s : s);
}

template <typename T>
hipError_t linear(const void* W, const float* b, const float* in, float* out, int N, int K, int P,
                  int silu_in, int silu_out, int acc, hipStream_t s) {
  hipLaunchKernelGGL(k_cond_linear<T>, dim3((N + 127) / 128, P), dim3(128), 0, s, reinterpret_cast<const T*>(W), b,
                     in, out, N, K, silu_in, silu_out, acc);
  return hipGetLastError();
}

}  // namespace

size_t cond_scratch_floats(int R, int d) {
  const size_t P = (size_t)R * R;
  return P * (2 * kFourier + 3 * (size_t)d);
}

template <typename T>
hipError_t launch_cond_table(const CondWeights& w, int J, int R, int d, float* table, float* scratch,
                             hipStream_t s) {
  const int P = R * R;
  float* feat = scratch;                      // [2P][256]: time rows, then step rows
  float* ht = feat + (size_t)2 * P * kFourier; // [P][d] hidden of the time embedder
  float* hs = ht + (size_t)P * d;             // [P][d] hidden of the step embedder
  float* e = hs + (size_t)P * d;              // [P][d] e_time + e_step
  hipLaunchKernelGGL(k_cond_features, dim3(2 * P), dim3(kFourier / 2), 0, s, feat, R);
  hipError_t err = hipGetLastError();
  if (err == hipSuccess) err = linear<T>(w.w1[0], w.b1[0], feat, ht, d, kFourier, P, 0, 1, 0, s);
  if (err == hipSuccess) err = linear<T>(w.w1[1], w.b1[1], feat + (size_t)P * kFourier, hs, d, kFourier, P, 0, 1, 0, s);
  if (err == hipSuccess) err = linear<T>(w.w2[0], w.b2[0], ht, e, d, d, P, 0, 0, 0, s);
  if (err == hipSuccess) err = linear<T>(w.w2[1], w.b2[1], hs, e, d, d, P, 0, 0, 1, s);
  for (int j = 0; j < J && err == hipSuccess; ++j)
    err = linear<T>(w.mod_w[j], w.mod_b[j], e, table + (size_t)j * P * 4 * d, 4 * d, d, P, 1, 0, 0, s);
  return err;
}

template hipError_t launch_cond_table<float>(const CondWeights&, int, int, int, float*, float*, hipStream_t);
template hipError_t launch_cond_table<bf16>(const CondWeights&, int, int, int, float*, float*, hipStream_t);

}  // namespace tlf
