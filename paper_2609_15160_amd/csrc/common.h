// Internal definitions shared by libtlf's kernels and host code (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace tlf {

constexpr int kPage = 16;          // tokens per KV page
constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kMaxLoops = 16;
constexpr int kPlanThreads = 1024; // single-workgroup planners
constexpr int kAttnMaxPages = 4096; // page list staged in LDS by the decode attention (max_pos <= 65536)

// Sticky device error bits (reported through tlf_cache_stats).
constexpr int kErrBadToken = 1;
constexpr int kErrOutOfPages = 2;

// Per-step statistics written by the decode planner (int64 slots).
enum StepStat {
  kStatKvRead = 0,
  kStatKvWrite = 1,
  kStatLoops = 2,
  kStatAttnBytesTotal = 3,  // cumulative algorithmic bytes of the decode attention
  kStatStepsTotal = 4,      // cumulative decode steps
  kStatKvWriteTotal = 5,    // cumulative bytes of appended k, v
  kStatLoopsTotal = 6,      // cumulative executed loops (shared block applications)
  kStatRows = 7,            // kStatRows + i: n_i of the step, i < kMaxLoops
  kStatCount = kStatRows + kMaxLoops
};

// Device view of the recursion-wise cache and the bookkeeping around it.
struct CacheView {
  void* pool;             // max_pages pages of page_elems storage elements
  int32_t* pos;           // [max_pages][kPage] original position of every slot (-1 if empty)
  int32_t* page_table;    // [max_batch][R][pages_per_seq] physical page of (b, i, p)
  int32_t* cache_len;     // [max_batch][R] entries n_{b,i}
  int32_t* seq_len;       // [max_batch] tokens of sequence b so far
  int32_t* chunk_len;     // [max_batch][R] entries of (b, i) appended by the latest prefill call
  int32_t* page_next;     // [1] bump allocator: pages in use
  int32_t* err;           // [1] sticky error bits
  unsigned long long* depth_hist; // [R]
  long long* step_stats;  // [kStatCount]
  int64_t page_elems;     // J * 2 * H * kPage * D
  int max_pages, pages_per_seq, R, J, H, D;
};

// Page layout: for each layer j and head h a K block of kPage x D elements
// in MFMA-fragment order (k_frag_off below), followed, after all heads' K
// blocks, by V blocks in groups of four slots, [kPage / 4][D][4] (v_frag_off
// below): one dimension of four consecutive slots is a single 8- or 16-byte
// load, and the D values of one slot lie four elements apart.
//   K(j, h, slot, e) = k_block(j, h) + k_frag_off<T>(slot, e)
//   V(j, h, slot, e) = v_block(j, h) + v_frag_off(slot, e, D)
__device__ __forceinline__ int64_t k_block(const CacheView& c, int j, int h) {
  return (int64_t)((j * 2 + 0) * c.H + h) * kPage * c.D;
}
__device__ __forceinline__ int64_t v_block(const CacheView& c, int j, int h) {
  return (int64_t)((j * 2 + 1) * c.H + h) * kPage * c.D;
}

template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<bf16>(bf16 v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float v) { return (bf16)v; }

// 16-byte vector of storage elements.
template <typename T> struct V16 {
  static constexpr int N = 16 / sizeof(T);
  union { uint4 u; T e[16 / sizeof(T)]; };
};

template <typename T> __device__ __forceinline__ V16<T> ld16(const T* p) {
  V16<T> v;
  v.u = *reinterpret_cast<const uint4*>(p);
  return v;
}
template <typename T> __device__ __forceinline__ void st16(T* p, const V16<T>& v) {
  *reinterpret_cast<uint4*>(p) = v.u;
}

// MFMA traits: one 16x16 output tile per instruction; KS = k per instruction,
// EPL = consecutive k elements held by each lane (lane l holds row/col l%16,
// k = (l/16)*EPL .. +EPL-1 of the step).  Output: lane l holds rows
// 4*(l/16)+r (r = 0..3) of column l%16.
template <typename T> struct Mfma;
template <> struct Mfma<bf16> {
  static constexpr int KS = 32;
  static constexpr int EPL = 8;
  typedef bf16x8 frag;
  static __device__ __forceinline__ frag load(const bf16* p) {
    return *reinterpret_cast<const bf16x8*>(p);
  }
  static __device__ __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma<float> {
  static constexpr int KS = 4;
  static constexpr int EPL = 1;
  typedef float frag;
  static __device__ __forceinline__ frag load(const float* p) { return *p; }
  static __device__ __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// Activations are float32.  A bf16 MFMA takes one as the sum of two bf16
// values, hi = bf16(v) and lo = bf16(v - hi), and runs once per part: the
// product with a bf16 weight is then exact to about 2^-16 of |v| instead of
// the 2^-9 of a single bf16 rounding.
__device__ __forceinline__ void split_bf16(float v, bf16& hi, bf16& lo) {
  hi = (bf16)v;
  lo = (bf16)(v - (float)hi);
}

// Two bf16 values in one 32-bit word, a in the low half.
__device__ __forceinline__ unsigned int pack2(bf16 a, bf16 b) {
  return (unsigned int)__builtin_bit_cast(unsigned short, a) |
         ((unsigned int)__builtin_bit_cast(unsigned short, b) << 16);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two floats rounded to bf16 (nearest even) in one 32-bit word, lo first:
// one two-input conversion instruction (converting the halves one by one
// takes two conversions, a shift and an or).
__device__ __forceinline__ unsigned int pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(unsigned int, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}

// Four float32 values as the packed hi and lo bf16 parts (2 words each):
// hi = bf16(v), lo = bf16(v - hi), each half of a packed word read back as
// the float it is the upper 16 bits of.
__device__ __forceinline__ void split4(float4 v, uint2& hi, uint2& lo) {
  const unsigned int h01 = pack_bf16x2(v.x, v.y), h23 = pack_bf16x2(v.z, v.w);
  const float hx = __uint_as_float(h01 << 16), hy = __uint_as_float(h01 & 0xFFFF0000u);
  const float hz = __uint_as_float(h23 << 16), hw = __uint_as_float(h23 & 0xFFFF0000u);
  hi = make_uint2(h01, h23);
  lo = make_uint2(pack_bf16x2(v.x - hx, v.y - hy), pack_bf16x2(v.z - hz, v.w - hw));
}

// Eight consecutive float32 values as the hi and lo fragments of a bf16 MFMA operand.
__device__ __forceinline__ void split_frag(const float* p, bf16x8& hi, bf16x8& lo) {
  uint2 h0, l0, h1, l1;
  split4(*reinterpret_cast<const float4*>(p), h0, l0);
  split4(*reinterpret_cast<const float4*>(p + 4), h1, l1);
  hi = __builtin_bit_cast(bf16x8, make_uint4(h0.x, h0.y, h1.x, h1.y));
  lo = __builtin_bit_cast(bf16x8, make_uint4(l0.x, l0.y, l1.x, l1.y));
}

// Offset of K(slot, e) inside a K block.  The decode attention takes K as the
// A operand of S = K q^T, one MFMA per K step of KS head dimensions; lane
// (slot, q) of a step holds the EPL consecutive elements e = ks * KS + q * EPL
// + j.  Storing fragment (ks, q, slot) at ((ks * 4 + q) * kPage + slot) * EPL
// makes the 64 lanes of one step read one contiguous run (1 KB in bf16).
template <typename T> __device__ __forceinline__ int k_frag_off(int slot, int e) {
  constexpr int KS = Mfma<T>::KS, EPL = Mfma<T>::EPL;
  static_assert(KS == 4 * EPL, "four lane groups per K step");
  const int ks = e / KS, q = (e % KS) / EPL, j = e % EPL;
  return ((ks * 4 + q) * kPage + slot) * EPL + j;
}

// Offset of V(slot, e) inside a V block: [slot / 4][D][slot % 4].
__device__ __forceinline__ int v_frag_off(int slot, int e, int D) { return ((slot >> 2) * D + e) * 4 + (slot & 3); }

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

template <typename V> __device__ __forceinline__ V shfl_xor(V v, int m) { return __shfl_xor(v, m, kWave); }

__device__ __forceinline__ void set_err(int32_t* err, int bits) { atomicOr(err, bits); }

// Block-wide exclusive prefix sum over blockDim.x (multiple of 64, <= 1024)
// threads.  `tmp` needs blockDim.x / 64 + 1 ints of shared memory.  Returns
// this thread's exclusive prefix; *total receives the block total.  All
// threads must call it.
__device__ __forceinline__ int block_exclusive_scan(int v, int* tmp, int* total) {
  const int lane = lane_id(), wid = threadIdx.x / kWave, nw = blockDim.x / kWave;
  int x = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    int y = __shfl_up(x, o, kWave);
    if (lane >= o) x += y;
  }
  if (lane == kWave - 1) tmp[wid] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
    for (int w = 0; w < nw; ++w) { int t = tmp[w]; tmp[w] = s; s += t; }
    tmp[nw] = s;
  }
  __syncthreads();
  int r = tmp[wid] + x - v;
  *total = tmp[nw];
  __syncthreads();
  return r;
}

}  // namespace tlf
