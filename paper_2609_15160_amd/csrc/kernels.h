// Launch interface between libtlf's host orchestrator and its HIP kernels.
#pragma once

#include "common.h"

namespace tlf {

// ---------------------------------------------------------------------------
// Row maps: which GEMM rows are active and where their residual row lives.
//   decode : row k < n_i is the k-th deepest token of the step, residual row
//            perm[k]; rows >= n_i have exited (Section 3.3 early exit).
//   prefill: rows are G segments of T compact slots; slot a of segment g is
//            active while a < n_{g,i}, and its residual row is tok_idx[r]
//            (the gathered original position, Eq. 6).
//   plain  : rows [0, rows) active, residual row r * src_stride + src_off.
// ---------------------------------------------------------------------------
struct RowMap {
  const int32_t* src = nullptr;   // residual row of row r (nullptr: strided)
  int src_stride = 1, src_off = 0;
  const int32_t* nact = nullptr;  // decode: rows [0, *nact) are active
  const int32_t* seg_cnt = nullptr; // prefill: segment s has seg_cnt[s * seg_cnt_stride] active slots
  int seg = 0, seg_cnt_stride = 0;
  int rows = 0;                   // rows covered by the grid
};

__device__ __forceinline__ bool row_active(const RowMap& m, int r) {
  if (r >= m.rows) return false;
  if (m.nact) return r < *m.nact;
  if (m.seg_cnt) return (r % m.seg) < m.seg_cnt[(r / m.seg) * m.seg_cnt_stride];
  return true;
}
__device__ __forceinline__ int row_src(const RowMap& m, int r) {
  return m.src ? m.src[r] : r * m.src_stride + m.src_off;
}

// Where the QKV epilogue appends k and v (Eq. 11).
struct KvDst {
  CacheView c;
  int loop = 0, layer = 0;
  // element offset of the cache slot that compact row r of this loop writes:
  // its page's offset (a multiple of kPage elements) plus the slot in the
  // low 4 bits, or -1 when the row has no cache entry.  Written by the
  // planners (decode: kv_slot + loop * B; prefill: the loop's gathered
  // entries), so that the projection resolves it with one independent load.
  const int64_t* slot_base = nullptr;
};

// A operand: A_SRC reads rows src(r) of a position-ordered buffer (the
// normalised residual y, or the residual x itself when the GEMM fuses the
// norm); A_CMP reads compact rows buf[r] (attention output, SwiGLU
// activation, the decode residual).  Both are float32.
enum AKind { A_SRC = 0, A_CMP = 1 };
// E_QKV: q to a buffer, k and v appended to the loop's cache pages.
// E_RESID: x[src(r)] += result.  E_SWIGLU: act = silu(gate) * up.
// E_LOGITS: float logits + greedy keys.  E_HIDDEN: out[r] = silu(result + bias)
// (the MLP router's hidden layer).
enum EKind { E_QKV = 0, E_RESID = 1, E_SWIGLU = 3, E_LOGITS = 4, E_HIDDEN = 5 };

// Active row tiles of a prefill loop, listed by the planner (sequences of a
// multiple of 256 tokens): with few of them the many-row GEMM takes smaller
// tiles from the list, so that more workgroups share the K loops of the
// later loops.
struct TileList {
  const int32_t* cnt = nullptr;      // this loop's active row tiles: [0] of 64 rows, [1] of 128, [2] of 256
  const int32_t* list64 = nullptr;   // first rows of the active 64-row tiles (inside one segment)
  const int32_t* list128 = nullptr;  // first rows of the active 128-row tiles
  const int32_t* list256 = nullptr;  // first rows of the active 256-row tiles
  int cus = 0;                       // compute units
};

struct GemmArgs {
  const float* A = nullptr; // float32 rows
  int lda = 0;
  const void* W = nullptr;  // [W rows][K] storage dtype
  const void* Wf = nullptr; // launch_dgemm: the same weights in MFMA fragment order (launch_wfrag), or nullptr
  // launch_dgemm: activations in MFMA fragment order.  For rows R and
  // columns k of a [rows][K] operand, element (R, k) sits at
  //   ((R / 16 * (K / KS) + k / KS) * 64 + (k % KS) / EPL * 16 + R % 16) * EPL + k % EPL
  // (KS, EPL of the model dtype's MFMA; frag_index below), so the 64 lanes'
  // fragments of one K step of 16 rows are one contiguous run.  a_frag: A is
  // stored so (A_CMP).  Buffers hold whole groups of 16 rows.
  int a_frag = 0;
  int out_frag = 0;         // E_SWIGLU: act in fragment order (K = F); E_RESID: the residual rows in
                            // fragment order (K = N), no scatter
  int copy_frag = 0;        // a_copy is written in fragment order (K = K)
  int N = 0;                // output columns (E_SWIGLU: 2F in the interleaved gate/up space)
  int K = 0;
  int w_rows = 0;           // rows of W (loads are clamped below it)
  RowMap rm;
  float* out = nullptr;     // E_QKV: q rows; E_RESID: residual; E_SWIGLU: act rows;
                            // E_LOGITS: logits (all float32)
  int ldo = 0;
  int out_row_off = 0;      // E_LOGITS: output row = out_row_off + r
  unsigned long long* argmax_keys = nullptr;  // E_LOGITS, may be nullptr: [rows][key_groups] greedy keys,
  int key_groups = 0;                         // one per 64-column group of each logits row
  KvDst kv;                 // E_QKV
  int d = 0;                // E_QKV: width of each of q, k, v
  int F = 0;                // E_SWIGLU: hidden width
  float eps = 1e-5f;        // RMSNorm epsilon of the decode projections that fuse the norm
  float* a_copy = nullptr;  // decode: the operand rows are also written here, compact (first projection)
  const float* bias = nullptr;  // E_HIDDEN: [N] float32
  int spec = 0;             // decode: every row is active; loads need not wait for the active count
  int scatter = 0;          // E_RESID: the residual row of row r is src(r) (prefill), not r
  // AdaLN (Section 3.1, Appendix A): row r's modulation row sits at
  // (depth(r) - 1) * mod_ld, depth(r) = mod_depth[mod_by_src ? src(r) : r]
  const float* mod_g = nullptr;  // QKV, gate/up: the operand row is scaled by (1 + mod_g[k])
  const float* mod_a = nullptr;  // E_RESID: out = x + (1 + mod_a[n]) * result
  int mod_ld = 0;
  const int32_t* mod_depth = nullptr;
  int mod_by_src = 0;
  const int32_t* keep_depth = nullptr;  // E_RESID (dense decode): row r is stored only while
  int keep_loop = 0;                    // keep_depth[r] > keep_loop (its token runs this loop)
  int a_single = 0;         // launch_gemm with bf16 weights: A rounded to one bf16 part (not hi + lo)
  const bf16* A16 = nullptr;  // launch_gemm with bf16 weights: A given as bf16 rows (same lda) in place of
                              // A (no norm, no operand modulation)
  bf16* out16 = nullptr;      // launch_gemm E_SWIGLU: act rows written as bf16 instead of float
  bf16* q16 = nullptr;        // launch_gemm E_QKV: q rows written as bf16(q * q_scale) instead of to out
  float q_scale = 1.f;
  TileList tl;                // launch_gemm with A16: the loop's active tiles (tl.cnt set) for the small shape
};

// Offset of element (R, k) of a [rows][K] operand stored in MFMA fragment order.
template <typename T> __device__ __forceinline__ int64_t frag_index(int R, int k, int K) {
  constexpr int KS = Mfma<T>::KS, EPL = Mfma<T>::EPL;
  return ((int64_t)((R >> 4) * (K / KS) + k / KS) * kWave + (k % KS) / EPL * 16 + (R & 15)) * EPL + k % EPL;
}

// Many-row projections (prefill, and the decode LM head of a large batch):
// 128 x 128 MFMA tiles staged through LDS.  norm: A is the residual x and the
// product is taken with RMSNorm(x) (supported for (A_CMP, E_LOGITS), whose
// rows write their logits to row src(r)).
template <typename T>
hipError_t launch_gemm(const GemmArgs& a, AKind ak, EKind ek, bool norm, hipStream_t s);
// Decode-shaped projections (few rows): K split across the waves of a
// workgroup, all loads in flight at once, one writer per output, rows in
// compact order (E_RESID: out[r] += result; E_LOGITS: logits row src(r)).
// norm: A is the residual x and the product is taken with RMSNorm(x).
// Supported: (A_SRC | A_CMP, E_QKV | E_SWIGLU | E_LOGITS, norm),
// (A_CMP, E_RESID | E_HIDDEN, no norm).  The prefill rows of one sequence use
// it too: rows [0, *rm.nact) active, A_SRC through the gathered positions,
// the residual scattered back (scatter) and the prefill cache slots.
// cus: compute units of the device (chooses between a narrow and a wide tile shape).
template <typename T>
hipError_t launch_dgemm(const GemmArgs& a, AKind ak, EKind ek, bool norm, int cus, hipStream_t s);
// Weights in MFMA fragment order for the decode projections: the B operand
// of one 16 x 16 x KS product (16 output columns, one K step) is 64 lanes x
// EPL elements, stored contiguously in lane order, blocks of 16 columns
// outermost and K steps inside them:
//   Wf[((blk * S + step) * 64 + lane) * EPL + e] = W[row(16 blk + lane % 16)][step * KS + (lane / 16) * EPL + e]
// with S = K / KS; row(n) = n, or the SwiGLU interleave (16 gate rows of a
// group of 16 hidden units, then their 16 up rows) when swiglu_F > 0.  One
// fragment load then reads 64 x 16 contiguous bytes (bf16) instead of 16
// rows x 64 bytes.  N must be a multiple of 16 and K of KS.
template <typename T>
hipError_t launch_wfrag(const void* W, void* Wf, int N, int K, int swiglu_F, hipStream_t s);

// ---------------------------------------------------------------------------
// Embedding + router (Section 3.2): h0 = E[x] + P[pos], z = W_r h0 + b_r,
// depth rule, margin, and y = RMSNorm(h0).
// ---------------------------------------------------------------------------
struct EmbedArgs {
  const void* tok_emb = nullptr;
  const void* pos_emb = nullptr;
  const float* Wr = nullptr;
  const float* br = nullptr;
  const int32_t* tokens = nullptr;
  int rows = 0, V = 0, d = 0, R = 0;
  int prefill_T = 0;              // > 0: pos = pos0 + row % T; 0: pos = seq_len[row]
  int pos0 = 0;
  const int32_t* seq_len = nullptr;
  float* x = nullptr;             // [rows][d] float residual
  float* y = nullptr;             // [rows][d] RMSNorm(x), or nullptr
  bf16* y16 = nullptr;            // [rows][d] RMSNorm(x) rounded to bf16, or nullptr
  float eps = 1e-5f;
  int32_t* depth = nullptr;       // [rows]
  int32_t* out_depth = nullptr;   // optional [rows]
  float* out_margin = nullptr;    // optional [rows]
  int rule = 0, fixed = 1;
  float threshold = 0.5f;
  int32_t* err = nullptr;
  int route = 1;                  // 0: the router is an MLP, routed later by launch_route_rows
};
template <typename T> hipError_t launch_embed_route(const EmbedArgs& a, hipStream_t s);

// Output layer of the MLP router and the depth rule: z = W_r h + b_r for the
// hidden rows h [rows][Hr] (float32), depth and margin as in launch_embed_route.
struct RouteArgs {
  const float* h = nullptr;
  int rows = 0, Hr = 0, R = 0;
  const float* Wr = nullptr;      // [R][Hr]
  const float* br = nullptr;      // [R]
  int32_t* depth = nullptr;
  int32_t* out_depth = nullptr;   // optional
  float* out_margin = nullptr;    // optional
  int rule = 0, fixed = 1;
  float threshold = 0.5f;
};
hipError_t launch_route_rows(const RouteArgs& a, hipStream_t s);

// y[src(r)] = RMSNorm(x[src(r)]) on the active rows of a row map.
struct ResidNormArgs {
  RowMap rm;
  const float* x = nullptr;
  float* y = nullptr;       // or nullptr
  bf16* y16 = nullptr;      // also RMSNorm(x) rounded to bf16, or nullptr
  int d = 0;
  float eps = 1e-5f;
};
template <typename T> hipError_t launch_resid_norm(const ResidNormArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// Decode planner (one workgroup): depth-sorted row order, active counts n_i,
// page allocation and slot bookkeeping for every executed (b, i), statistics.
// ---------------------------------------------------------------------------
struct DecodePlanArgs {
  CacheView c;
  int B = 0;
  const int32_t* depth = nullptr;
  int32_t* perm = nullptr;         // [B]
  int32_t* nact = nullptr;         // [R]
  int64_t* kv_slot = nullptr;      // [R][B]: element offset (page * page_elems + slot) of the
                                   // slot that compact row k appends at loop i
  int64_t kv_entry_bytes = 0;      // bytes of one (token, loop) cache entry over all layers
  int32_t* row_depth = nullptr;    // [B] depth of the token of compact row k
  int dense = 0;                   // 1: rows in batch order, every loop up to the deepest token
                                   // runs all B rows; exited rows get kv_slot -1
};
hipError_t launch_plan_decode(const DecodePlanArgs& a, hipStream_t s);

// Prefill planner (one workgroup per sequence of the group): per loop i the
// gathered positions rho^(i) (Eq. 6), n_{b,i}, pages and their positions.
struct PrefillPlanArgs {
  CacheView c;
  int b0 = 0, G = 0, T = 0;
  int append = 0;  // 1: continue every (b, i) cache after its cache_len entries; 0: start it empty
  int pos0 = 0;    // position of the first token of the call
  const int32_t* depth = nullptr;  // [G][T]
  int32_t* tok_idx = nullptr;      // [R][G*T]
  int64_t* kv_slot = nullptr;      // [R][G*T]: cache slot offset of each gathered entry (KvDst)
  // optional (T a multiple of 256): each loop's active row tiles (TileList),
  // appended per sequence; the counts start at 0
  int32_t* tile_cnt = nullptr;     // [R][3]: tiles of 64, 128 and 256 rows
  int32_t* tile_list64 = nullptr;  // [R][G*T / 64]
  int32_t* tile_list128 = nullptr; // [R][G*T / 128]
  int32_t* tile_list256 = nullptr; // [R][G*T / 256]
};
hipError_t launch_plan_prefill(const PrefillPlanArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// Attention over the recursion-wise cache (Eq. 10).
// ---------------------------------------------------------------------------
struct AttnDecodeArgs {
  CacheView c;
  int loop = 0, layer = 0, d = 0;
  const int32_t* perm = nullptr;   // depth-sorted row order
  const int32_t* nact = nullptr;   // n_i of this loop: rows [0, n_i) are active
  const float* q = nullptr;        // [rows][d] compact rows
  float* o = nullptr;              // [rows][d], or in MFMA fragment order (o_ks > 0)
  int o_ks = 0, o_epl = 0;         // o in the fragment order of GemmArgs::a_frag with this KS, EPL
  float scale_log2 = 0.f;          // log2(e) / sqrt(D)
  int grid = 0;                    // persistent workgroups
  int waves = 4;                   // waves per workgroup sharing one (row, head): 4 or 8
};
template <typename T> hipError_t launch_attn_decode(const AttnDecodeArgs& a, hipStream_t s);
// Resident workgroups per compute unit of the decode attention (4 or 8 waves each).
template <typename T> hipError_t attn_decode_blocks_per_cu(int D, int waves, int* blocks);

struct AttnPrefillArgs {
  CacheView c;
  int loop = 0, layer = 0, d = 0;
  int b0 = 0, G = 0, T = 0;
  const float* q = nullptr; // [G*T][d], row g*T + a
  float* o = nullptr;       // [G*T][d]
  float scale_log2 = 0.f;
  int q_single = 0;         // bf16 keys: the scaled q enters the score product as one bf16 part (not hi + lo)
  bf16* o16 = nullptr;      // [G*T][d]: o written as bf16 instead of to o
  const bf16* q16 = nullptr;  // with q_single: [G*T][d] q already scaled and rounded (bf16(q * scale_log2)), read in place of q
};
template <typename T> hipError_t launch_attn_prefill(const AttnPrefillArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// Small utility kernels (no hipMemset inside the step, so a step can be
// captured in a graph).
// ---------------------------------------------------------------------------
hipError_t launch_fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t s);
hipError_t launch_fill_u64(unsigned long long* p, unsigned long long v, int64_t n, hipStream_t s);
// next[b] = the column of the largest key among row b's `groups` keys (lowest id on ties).
hipError_t launch_argmax_finalize(const unsigned long long* keys, int groups, int32_t* next, int B, hipStream_t s);

// ---------------------------------------------------------------------------
// AdaLN conditioning table: modulation of every (layer, loop, depth),
// table[j][i][m][4d] (0-based loop i and depth m + 1), rows alpha_msa |
// alpha_mlp | gamma_msa | gamma_mlp.  Matrices in the storage dtype.
// ---------------------------------------------------------------------------
struct CondWeights {
  const void* w1[2] = {nullptr, nullptr};  // time, step: [d][256]
  const float* b1[2] = {nullptr, nullptr};
  const void* w2[2] = {nullptr, nullptr};  // [d][d]
  const float* b2[2] = {nullptr, nullptr};
  const void* const* mod_w = nullptr;      // host array of J: [4d][d]
  const float* const* mod_b = nullptr;     // host array of J: [4d]
};
size_t cond_scratch_floats(int R, int d);
template <typename T>
hipError_t launch_cond_table(const CondWeights& w, int J, int R, int d, float* table, float* scratch,
                             hipStream_t s);

// Multi-workgroup active-set planner of the training gather-scatter (gs.hip):
// argument checks (host only, no device work; rows <= max_rows) and the two
// launches, with `counts` holding one int32 per chunk of TLF_GS_PLAN_CHUNK_ROWS
// rows.  Both return a TLF_* status.
int gs_plan_chunked_args(const int32_t* d_depth, int32_t batch, int32_t seq_len, int32_t* d_index,
                         const int32_t* d_count, int64_t max_rows, int64_t* rows_out);
int launch_gs_plan_chunked(const int32_t* d_depth, int32_t batch, int32_t seq_len, int32_t loop, int32_t* d_index,
                           int32_t* d_slot, int32_t* d_offsets, int32_t* d_count, int32_t* counts, int64_t rows,
                           hipStream_t stream);

}  // namespace tlf
