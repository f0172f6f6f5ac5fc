// Host side of libtlf: argument validation, workspace layout, the inference
// state machine, and the launch sequences of prefill and decode.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/tlf.h"
#include "kernels.h"

using namespace tlf;

namespace {

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Workspace buffers, in carve order.
enum Buf {
  B_POOL, B_POS, B_PAGE_TABLE, B_CACHE_LEN, B_CHUNK_LEN, B_SEQ_LEN, B_SCALARS, B_DEPTH_HIST, B_STEP_STATS,
  B_X_DEC, B_XC_DEC, B_KVSLOT, B_DEPTH_DEC, B_PERM, B_NACT, B_Q_DEC, B_O_DEC, B_ACT_DEC, B_KEYS,
  B_X_PRE, B_Y_PRE, B_Y16_PRE, B_DEPTH_PRE, B_TOK_IDX, B_KVSLOT_PRE, B_Q_PRE, B_O_PRE, B_ACT_PRE, B_HID,
  B_ROW_DEPTH, B_MOD, B_COND_TMP, B_WFRAG, B_TILES,
  B_COUNT
};

struct Layout {
  size_t off[B_COUNT];
  size_t size[B_COUNT];
  size_t total = 0;
  int64_t page_elems = 0;
  int pages_per_seq = 0, pre_rows = 0, s = 0;
};

bool make_layout(const tlf_config& c, Layout* L) {
  const int64_t s = c.dtype == TLF_DTYPE_BF16 ? 2 : 4;
  const int64_t R = c.max_loops, B = c.max_batch, d = c.d_model, F = c.d_ff, H = c.n_heads, D = c.head_dim;
  L->s = (int)s;
  L->page_elems = (int64_t)c.n_layers * 2 * H * kPage * D;
  L->pages_per_seq = (int)ceil_div(c.max_pos, kPage);
  L->pre_rows = std::max(c.max_prefill_tokens, c.max_pos);
  const int64_t P = L->pre_rows;
  int64_t sz[B_COUNT];
  sz[B_POOL] = (int64_t)c.max_pages * L->page_elems * s;
  sz[B_POS] = (int64_t)c.max_pages * kPage * 4;
  sz[B_PAGE_TABLE] = B * R * L->pages_per_seq * 4;
  sz[B_CACHE_LEN] = B * R * 4;
  sz[B_CHUNK_LEN] = B * R * 4;
  sz[B_SEQ_LEN] = B * 4;
  sz[B_SCALARS] = 2 * 4;  // page_next, err
  sz[B_DEPTH_HIST] = R * 8;
  sz[B_STEP_STATS] = kStatCount * 8;
  sz[B_X_DEC] = B * d * 4;
  sz[B_XC_DEC] = (int64_t)((B + 15) / 16 * 16) * d * 4;  // whole groups of 16 rows (fragment order)
  sz[B_KVSLOT] = R * B * 8;
  sz[B_DEPTH_DEC] = B * 4;
  sz[B_PERM] = B * 4;
  sz[B_NACT] = R * 4;
  sz[B_Q_DEC] = B * d * 4;
  sz[B_O_DEC] = (int64_t)((B + 15) / 16 * 16) * d * 4;  // whole groups of 16 rows (fragment order)
  sz[B_ACT_DEC] = (int64_t)((B + 15) / 16 * 16) * F * 4;  // whole groups of 16 rows (fragment order)
  sz[B_KEYS] = B * ceil_div(c.vocab, kWave) * 8;  // greedy key per 64-column group of each row
  sz[B_X_PRE] = P * d * 4;
  sz[B_Y_PRE] = P * d * 4;
  // one-part bf16 prefill activations: RMSNorm(x) as bf16 rows (o and act
  // are written as bf16 into their own float buffers)
  sz[B_Y16_PRE] = c.prefill_act_bf16 && c.dtype == TLF_DTYPE_BF16 ? P * d * 2 : 0;
  sz[B_DEPTH_PRE] = P * 4;
  sz[B_TOK_IDX] = R * P * 4;
  sz[B_KVSLOT_PRE] = R * P * 8;
  sz[B_Q_PRE] = P * d * 4;
  sz[B_O_PRE] = P * d * 4;
  sz[B_ACT_PRE] = P * F * 4;
  sz[B_HID] = std::max(P, B) * (int64_t)c.router_hidden * 4;  // MLP router hidden rows
  sz[B_ROW_DEPTH] = B * 4;
  // AdaLN: modulation of every (layer, loop, depth), and its set-up scratch
  sz[B_MOD] = c.adaln ? (int64_t)c.n_layers * R * R * 4 * d * 4 : 0;
  sz[B_COND_TMP] = c.adaln ? (int64_t)cond_scratch_floats((int)R, (int)d) * 4 : 0;
  // every layer's block weights in MFMA fragment order (the decode projections' copy)
  sz[B_WFRAG] = (int64_t)c.n_layers * (4 * d * d + 3 * d * F) * s;
  // each prefill loop's active row-tile counts and lists (one-part bf16 activations)
  sz[B_TILES] = c.prefill_act_bf16 && c.dtype == TLF_DTYPE_BF16 ? R * (3 + P / 64 + P / 128 + P / 256) * 4 : 0;
  size_t off = 0;
  for (int i = 0; i < B_COUNT; ++i) {
    if (sz[i] < 0) return false;
    L->off[i] = off;
    L->size[i] = (size_t)sz[i];
    off = align_up(off + (size_t)sz[i], 256);
  }
  L->total = off;
  return true;
}

static_assert(kPlanThreads * 4 >= TLF_MAX_BATCH, "the decode planner covers the batch in 4 chunks");

// TLF_E_INVALID_ARG for a config that describes no valid model or call
// setting, TLF_E_UNSUPPORTED for a valid one outside the shapes and sizes the
// kernels are built for.
int validate_config(const tlf_config* c) {
  if (!c) return TLF_E_INVALID_ARG;
  if (c->abi_version != TLF_ABI_VERSION) return TLF_E_INVALID_ARG;
  if (c->dtype != TLF_DTYPE_F32 && c->dtype != TLF_DTYPE_BF16) return TLF_E_INVALID_ARG;
  if (c->vocab < 1 || c->d_model < 1 || c->head_dim < 1 || c->d_ff < 1) return TLF_E_INVALID_ARG;
  if (c->n_heads < 1 || (int64_t)c->n_heads * c->head_dim != c->d_model) return TLF_E_INVALID_ARG;
  if (c->n_layers < 1 || c->max_loops < 1 || c->max_pos < 1 || c->max_batch < 1) return TLF_E_INVALID_ARG;
  if (c->page_tokens < 1 || c->max_pages < 1 || c->max_prefill_tokens < 1) return TLF_E_INVALID_ARG;
  if (c->route_rule == TLF_ROUTE_CUMPROB) {
    if (!(c->route_threshold > 0.f && c->route_threshold < 1.f)) return TLF_E_INVALID_ARG;
  } else if (c->route_rule == TLF_ROUTE_FIXED) {
    if (c->fixed_depth < 1 || c->fixed_depth > c->max_loops) return TLF_E_INVALID_ARG;
  } else if (c->route_rule != TLF_ROUTE_ARGMAX) {
    return TLF_E_INVALID_ARG;
  }
  if (!(c->rms_eps > 0.f) || !std::isfinite(c->rms_eps)) return TLF_E_INVALID_ARG;
  if (c->decode_graph != 0 && c->decode_graph != 1) return TLF_E_INVALID_ARG;
  if (c->router_hidden < 0) return TLF_E_INVALID_ARG;
  if (c->dense_decode != 0 && c->dense_decode != 1) return TLF_E_INVALID_ARG;
  if (c->adaln != 0 && c->adaln != 1) return TLF_E_INVALID_ARG;
  if (c->prefill_act_bf16 != 0 && c->prefill_act_bf16 != 1) return TLF_E_INVALID_ARG;
  // shapes and sizes of this build's kernels:
  // GEMM K tiles are 256 bytes: 128 bf16 or 64 float32 elements; rows up to 4096 wide
  const int kq = c->dtype == TLF_DTYPE_BF16 ? 128 : 64;
  if (c->d_model < kq || c->d_model % kq != 0 || c->d_model > 4096) return TLF_E_UNSUPPORTED;
  if (c->head_dim != 16 && c->head_dim != 64 && c->head_dim != 128) return TLF_E_UNSUPPORTED;
  if (c->dtype == TLF_DTYPE_BF16 && c->head_dim == 16) return TLF_E_UNSUPPORTED;
  if (c->d_ff < kq || c->d_ff % kq != 0) return TLF_E_UNSUPPORTED;
  if (c->n_layers > TLF_MAX_LAYERS || c->max_loops > TLF_MAX_LOOPS || c->max_batch > TLF_MAX_BATCH)
    return TLF_E_UNSUPPORTED;
  if (c->page_tokens != TLF_PAGE_TOKENS) return TLF_E_UNSUPPORTED;
  if (c->router_hidden > 4096 || c->router_hidden % 64 != 0) return TLF_E_UNSUPPORTED;
  // the decode attention stages one sequence's page list in LDS
  if (ceil_div(c->max_pos, kPage) > kAttnMaxPages) return TLF_E_UNSUPPORTED;
  // the decode projections address weights and activations with 32-bit element offsets
  if ((int64_t)c->vocab * c->d_model >= INT32_MAX || 2 * (int64_t)c->d_ff * c->d_model >= INT32_MAX ||
      (int64_t)TLF_MAX_BATCH * std::max(c->d_ff, 3 * c->d_model) >= INT32_MAX)
    return TLF_E_UNSUPPORTED;
  // positions, row indices and work-list offsets are int32
  if ((int64_t)std::max(c->max_prefill_tokens, c->max_pos) * std::max(c->d_ff, 3 * c->d_model) > INT32_MAX)
    return TLF_E_UNSUPPORTED;
  return TLF_OK;
}

int validate_weights(const tlf_config* c, const tlf_weights* w) {
  if (!w || !w->tok_emb || !w->pos_emb || !w->router_w || !w->router_b) return TLF_E_INVALID_ARG;
  if (w->n_layers != c->n_layers || !w->layers) return TLF_E_INVALID_ARG;
  if ((c->router_hidden > 0) != (w->router_w1 != nullptr && w->router_b1 != nullptr)) return TLF_E_INVALID_ARG;
  for (int j = 0; j < w->n_layers; ++j) {
    const tlf_layer_weights& l = w->layers[j];
    if (!l.w_qkv || !l.w_o || !l.w_gate_up || !l.w_down) return TLF_E_INVALID_ARG;
  }
  if ((c->adaln != 0) != (w->adaln != nullptr)) return TLF_E_INVALID_ARG;
  if (const tlf_adaln_weights* a = w->adaln) {
    if (!a->time_w1 || !a->time_b1 || !a->time_w2 || !a->time_b2 || !a->step_w1 || !a->step_b1 ||
        !a->step_w2 || !a->step_b2 || !a->mod_w || !a->mod_b)
      return TLF_E_INVALID_ARG;
    for (int j = 0; j < w->n_layers; ++j)
      if (!a->mod_w[j] || !a->mod_b[j]) return TLF_E_INVALID_ARG;
  }
  return TLF_OK;
}

}  // namespace

struct tlf_ctx {
  tlf_config cfg;
  tlf_weights w;
  std::vector<tlf_layer_weights> layers;
  Layout L;
  hipStream_t stream = nullptr;
  char* ws = nullptr;
  CacheView cv;
  int batch = 0, seq_len = 0;
  bool prefilled = false, poisoned = false;
  int sticky = TLF_OK;
  int cus = 0;  // compute units of the device
  int attn_blocks[2] = {1, 1};  // resident decode-attention workgroups per CU (4 and 8 waves)
  // measurement: event pairs around decode-attention launches, resolved by tlf_cache_stats
  bool profiling = false;     // decode steps launched eagerly, block region timed
  bool profile_attn = false;  // and every decode-attention launch timed
  std::vector<hipEvent_t> event_pool;
  struct Timed { hipEvent_t start, stop; bool attn; };
  std::vector<Timed> event_pending;
  int64_t attn_launches = 0;
  double attn_ms = 0.0, block_ms = 0.0;

  // decode-step graphs: captured on cap_stream, replayed on stream.  A graph
  // holds the batch and the step's buffer pointers; the last kGraphs distinct
  // ones are kept (greedy decode alternates two token buffers, the output of
  // one step being the input of the next), the least recently used replaced.
  static constexpr int kGraphs = 4;
  hipStream_t cap_stream = nullptr;
  struct GraphKey {
    int batch = -1;
    const void *tokens = nullptr, *logits = nullptr, *next = nullptr, *depths = nullptr, *margin = nullptr;
    bool operator==(const GraphKey& o) const {
      return batch == o.batch && tokens == o.tokens && logits == o.logits && next == o.next &&
             depths == o.depths && margin == o.margin;
    }
  };
  struct CachedGraph {
    GraphKey key;
    hipGraphExec_t exec = nullptr;
    uint64_t used = 0;  // last use (graph_clock)
  } graphs[kGraphs];
  uint64_t graph_clock = 0;

  ~tlf_ctx() {
    recycle_events();
    for (hipEvent_t e : event_pool) (void)hipEventDestroy(e);
    for (CachedGraph& g : graphs)
      if (g.exec) (void)hipGraphExecDestroy(g.exec);
    if (cap_stream) (void)hipStreamDestroy(cap_stream);
  }
  void recycle_events() {
    for (auto& t : event_pending) { event_pool.push_back(t.start); event_pool.push_back(t.stop); }
    event_pending.clear();
  }
  // records the first event of a timed region; the caller records .stop after the work
  hipError_t begin_timed(hipStream_t s, bool attn) {
    Timed t{nullptr, nullptr, attn};
    hipError_t e = take_event(&t.start);
    if (e == hipSuccess) e = take_event(&t.stop);
    if (e == hipSuccess) e = hipEventRecord(t.start, s);
    if (e == hipSuccess) event_pending.push_back(t);
    return e;
  }
  hipError_t end_timed(hipStream_t s) { return hipEventRecord(event_pending.back().stop, s); }
  hipError_t take_event(hipEvent_t* e) {
    if (!event_pool.empty()) { *e = event_pool.back(); event_pool.pop_back(); return hipSuccess; }
    // timing only: no system-scope fence (cache writeback and invalidate) at each record
    return hipEventCreateWithFlags(e, hipEventDisableSystemFence);
  }

  template <typename P> P* buf(Buf b) const { return reinterpret_cast<P*>(ws + L.off[b]); }
  // layer j's weights in fragment order: qkv [3d][d], o [d][d], gate/up [2F][d], down [d][F]
  const void* wfrag(int j, int part) const {
    const int64_t d = cfg.d_model, F = cfg.d_ff;
    const int64_t sizes[4] = {3 * d * d, d * d, 2 * F * d, d * F};
    int64_t off = (int64_t)j * (4 * d * d + 3 * d * F);
    for (int k = 0; k < part; ++k) off += sizes[k];
    return ws + L.off[B_WFRAG] + off * L.s;
  }
};

#define TLF_HIP(expr)                  \
  do {                                 \
    hipError_t e_ = (expr);            \
    if (e_ != hipSuccess) {            \
      ctx->poisoned = true;            \
      return TLF_E_HIP;                \
    }                                  \
  } while (0)

namespace {

int precheck(tlf_ctx* ctx) {
  if (!ctx) return TLF_E_INVALID_ARG;
  if (ctx->poisoned) return TLF_E_STATE;
  if (ctx->sticky != TLF_OK) return ctx->sticky;
  return TLF_OK;
}

// The MLP router (Section 3.2) on `rows` rows of h0: hidden = silu(W_1 h0 + b_1)
// by a projection, then z = W_r hidden + b_r and the depth rule per row.
template <typename T>
int run_mlp_router(tlf_ctx* ctx, hipStream_t s, const float* h0, int rows, bool decode_shape, int32_t* depth,
                   int32_t* out_depth, float* out_margin) {
  const tlf_config& c = ctx->cfg;
  const int Hr = c.router_hidden;
  float* hid = ctx->buf<float>(B_HID);
  GemmArgs g;
  g.A = h0; g.lda = c.d_model; g.W = ctx->w.router_w1; g.N = Hr; g.K = c.d_model; g.w_rows = Hr;
  g.rm.rows = rows; g.out = hid; g.ldo = Hr; g.bias = ctx->w.router_b1; g.spec = 1;
  if (decode_shape) TLF_HIP(launch_dgemm<T>(g, A_CMP, E_HIDDEN, false, ctx->cus, s));
  else TLF_HIP(launch_gemm<T>(g, A_CMP, E_HIDDEN, false, s));
  RouteArgs ra;
  ra.h = hid; ra.rows = rows; ra.Hr = Hr; ra.R = c.max_loops; ra.Wr = ctx->w.router_w; ra.br = ctx->w.router_b;
  ra.depth = depth; ra.out_depth = out_depth; ra.out_margin = out_margin;
  ra.rule = c.route_rule; ra.threshold = c.route_threshold; ra.fixed = c.fixed_depth;
  TLF_HIP(launch_route_rows(ra, s));
  return TLF_OK;
}

// Waves sharing one (row, head) in the decode attention: enough waves in
// flight to cover the device even when batch x heads is small.
int attn_waves(const tlf_ctx* ctx) {
  const int64_t units = (int64_t)ctx->batch * ctx->cfg.n_heads;
  const int64_t slots = (int64_t)ctx->cus * ctx->attn_blocks[0] * 4;  // resident waves with 4-wave groups
  return units * 4 >= slots ? 4 : 8;
}

// Decode batches of at least this many rows run the LM head on the 128 x 128 GEMM.
constexpr int kHeadGemmRows = 128;

// Prefill of a single sequence of at most this many tokens runs its
// projections on the split-K decode GEMM.
constexpr int kPrefillFewRows = 2048;

// AdaLN: point a projection at its rows' modulation at (loop i, layer j):
// part 0..3 = alpha_msa, alpha_mlp, gamma_msa, gamma_mlp of the table
// [j][i][m][4d]; gamma scales the operand rows, alpha gates a residual
// epilogue.  depth(r) = depth[src(r)] (by_src) or depth[r].
void set_mod(const tlf_ctx* ctx, GemmArgs* g, int i, int j, int part, const int32_t* depth, int by_src) {
  const tlf_config& c = ctx->cfg;
  if (!c.adaln) return;
  const int64_t R = c.max_loops, d = c.d_model;
  const float* p = ctx->buf<float>(B_MOD) + ((int64_t)j * R + i) * R * 4 * d + part * d;
  if (part >= 2) g->mod_g = p;
  else g->mod_a = p;
  g->mod_ld = (int)(4 * d);
  g->mod_depth = depth;
  g->mod_by_src = by_src;
}

const void* head_weights(const tlf_ctx* ctx) { return ctx->w.lm_head ? ctx->w.lm_head : ctx->w.tok_emb; }

template <typename T>
int run_prefill(tlf_ctx* ctx, int B, int T_, int pos0, const int32_t* tokens, float* logits, int32_t* depths,
                uint32_t flags) {
  const tlf_config& c = ctx->cfg;
  hipStream_t s = ctx->stream;
  const int d = c.d_model, F = c.d_ff, R = c.max_loops;
  const bool append = (flags & TLF_PREFILL_APPEND) != 0;
  if (!append) {
    TLF_HIP(launch_fill_i32(ctx->cv.page_next, 0, 1, s));
    TLF_HIP(launch_fill_u64(ctx->cv.depth_hist, 0ull, R, s));
  }
  const int G = std::max(1, ctx->L.pre_rows / T_);
  float* x = ctx->buf<float>(B_X_PRE);
  float* y = ctx->buf<float>(B_Y_PRE);
  const int32_t* pre_depth = ctx->buf<int32_t>(B_DEPTH_PRE);  // by residual row
  for (int b0 = 0; b0 < B; b0 += G) {
    const int Gc = std::min(G, B - b0);
    const int rows = Gc * T_;
    // one short sequence: too few rows for the 128 x 128 tiles to fill the
    // device, so the projections take the split-K decode GEMM with the
    // RMSNorm fused (x is read through the gathered positions, no y)
    const bool few = Gc == 1 && T_ <= kPrefillFewRows;
    // one-part bf16 activations (prefill_act_bf16, bf16 weights, the many-row
    // GEMMs): RMSNorm(x), o and act are handed on as bf16 rows; the LM head
    // keeps reading the float32 RMSNorm(x)
    const bool one = c.prefill_act_bf16 && c.dtype == TLF_DTYPE_BF16 && !few;
    // with the normed rows handed on as bf16 and no AdaLN scale to apply to
    // the float rows, RMSNorm(x) in float32 feeds only the LM head: it is
    // written once, for the head's rows, after the last loop
    const bool y32 = !one || c.adaln;
    bf16* y16 = one ? ctx->buf<bf16>(B_Y16_PRE) : nullptr;
    bf16* o16 = one ? ctx->buf<bf16>(B_O_PRE) : nullptr;
    bf16* act16 = one ? ctx->buf<bf16>(B_ACT_PRE) : nullptr;
    EmbedArgs ea;
    ea.tok_emb = ctx->w.tok_emb; ea.pos_emb = ctx->w.pos_emb; ea.Wr = ctx->w.router_w; ea.br = ctx->w.router_b;
    ea.tokens = tokens + (int64_t)b0 * T_;
    ea.rows = rows; ea.V = c.vocab; ea.d = d; ea.R = R; ea.prefill_T = T_; ea.pos0 = pos0;
    ea.x = x; ea.y = few || !y32 ? nullptr : y; ea.y16 = y16; ea.eps = c.rms_eps; ea.depth = ctx->buf<int32_t>(B_DEPTH_PRE);
    ea.out_depth = depths ? depths + (int64_t)b0 * T_ : nullptr;
    ea.rule = c.route_rule; ea.threshold = c.route_threshold; ea.fixed = c.fixed_depth;
    ea.err = ctx->cv.err;
    ea.route = c.router_hidden == 0;
    TLF_HIP(launch_embed_route<T>(ea, s));
    if (c.router_hidden > 0) {
      const int st = run_mlp_router<T>(ctx, s, x, rows, few, ea.depth, ea.out_depth, nullptr);
      if (st != TLF_OK) return st;
    }

    PrefillPlanArgs pa;
    pa.c = ctx->cv; pa.b0 = b0; pa.G = Gc; pa.T = T_; pa.append = append; pa.pos0 = pos0;
    pa.depth = ctx->buf<int32_t>(B_DEPTH_PRE);
    pa.tok_idx = ctx->buf<int32_t>(B_TOK_IDX);
    pa.kv_slot = ctx->buf<int64_t>(B_KVSLOT_PRE);
    // the later loops' projections take smaller tiles from each loop's list
    // of active row tiles (whole tiles per sequence: T a multiple of 256)
    const bool tiles = one && T_ % 256 == 0 && ctx->L.size[B_TILES] > 0;
    int32_t* tile_cnt = ctx->buf<int32_t>(B_TILES);
    int32_t* tile_list64 = tile_cnt + 3 * R;
    int32_t* tile_list128 = tile_list64 + (int64_t)R * (ctx->L.pre_rows / 64);
    int32_t* tile_list256 = tile_list128 + (int64_t)R * (ctx->L.pre_rows / 128);
    if (tiles) {
      TLF_HIP(launch_fill_i32(tile_cnt, 0, 3 * R, s));
      pa.tile_cnt = tile_cnt; pa.tile_list64 = tile_list64; pa.tile_list128 = tile_list128;
      pa.tile_list256 = tile_list256;
    }
    TLF_HIP(launch_plan_prefill(pa, s));

    for (int i = 0; i < R; ++i) {
      // rows: G segments of T compact slots; slot a of segment g is the a-th
      // token of the call in sequence b0 + g with depth >= i + 1 (cache
      // entry n_old + a), residual row tok_idx[r]
      RowMap rm;
      rm.src = ctx->buf<int32_t>(B_TOK_IDX) + (int64_t)i * rows;
      rm.seg_cnt = ctx->cv.chunk_len + (int64_t)b0 * R + i;
      rm.seg = T_; rm.seg_cnt_stride = R; rm.rows = rows;
      if (few) rm.nact = rm.seg_cnt;  // one segment: rows [0, n) active
      TileList tl;
      if (tiles) {
        tl.cnt = tile_cnt + 3 * i;
        tl.list64 = tile_list64 + (int64_t)i * (rows / 64);
        tl.list128 = tile_list128 + (int64_t)i * (rows / 128);
        tl.list256 = tile_list256 + (int64_t)i * (rows / 256);
        tl.cus = ctx->cus;
      }
      ResidNormArgs rn;
      rn.rm = rm; rn.x = x; rn.y = y32 ? y : nullptr; rn.y16 = y16; rn.d = d; rn.eps = c.rms_eps;
      for (int j = 0; j < c.n_layers; ++j) {
        const tlf_layer_weights& lw = ctx->layers[j];
        GemmArgs q;
        q.A = few ? x : y; q.lda = d; q.W = lw.w_qkv; q.Wf = ctx->wfrag(j, 0); q.N = 3 * d; q.K = d; q.w_rows = 3 * d; q.rm = rm;
        q.out = ctx->buf<float>(B_Q_PRE); q.ldo = d; q.d = d; q.eps = c.rms_eps; q.spec = i == 0;
        q.kv.c = ctx->cv; q.kv.loop = i; q.kv.layer = j; q.kv.slot_base = ctx->buf<int64_t>(B_KVSLOT_PRE) + (int64_t)i * rows;
        set_mod(ctx, &q, i, j, 2, pre_depth, 1);
        q.a_single = one;
        if (one && !q.mod_g) q.A16 = y16;  // the AdaLN scale needs the float rows
        const float scale_log2 = 1.4426950408889634f / std::sqrt((float)c.head_dim);
        // one part: q handed on as bf16(q * scale_log2), as the attention rounds it
        bf16* q16 = one ? reinterpret_cast<bf16*>(ctx->buf<float>(B_Q_PRE)) : nullptr;
        q.q16 = q16; q.q_scale = scale_log2; q.tl = tl;
        if (few) TLF_HIP(launch_dgemm<T>(q, A_SRC, E_QKV, true, ctx->cus, s));
        else TLF_HIP(launch_gemm<T>(q, A_SRC, E_QKV, false, s));

        AttnPrefillArgs at;
        at.c = ctx->cv; at.loop = i; at.layer = j; at.d = d; at.b0 = b0; at.G = Gc; at.T = T_;
        at.q = ctx->buf<float>(B_Q_PRE); at.o = ctx->buf<float>(B_O_PRE);
        at.scale_log2 = scale_log2;
        at.q_single = one;
        at.q16 = q16;
        at.o16 = o16;
        TLF_HIP(launch_attn_prefill<T>(at, s));

        GemmArgs o;
        o.A = ctx->buf<float>(B_O_PRE); o.lda = d; o.W = lw.w_o; o.Wf = ctx->wfrag(j, 1); o.N = d; o.K = d; o.w_rows = d; o.rm = rm;
        o.out = x; o.ldo = d; o.scatter = 1; o.spec = i == 0; o.a_single = one; o.A16 = o16; o.tl = tl;
        set_mod(ctx, &o, i, j, 0, pre_depth, 1);
        if (few) {
          TLF_HIP(launch_dgemm<T>(o, A_CMP, E_RESID, false, ctx->cus, s));
        } else {
          TLF_HIP(launch_gemm<T>(o, A_CMP, E_RESID, false, s));
          TLF_HIP(launch_resid_norm<T>(rn, s));
        }

        GemmArgs gu;
        gu.A = few ? x : y; gu.lda = d; gu.W = lw.w_gate_up; gu.Wf = ctx->wfrag(j, 2); gu.N = 2 * F; gu.K = d; gu.w_rows = 2 * F; gu.rm = rm;
        gu.out = ctx->buf<float>(B_ACT_PRE); gu.ldo = F; gu.F = F; gu.eps = c.rms_eps; gu.spec = i == 0;
        gu.a_single = one; gu.out16 = act16; gu.tl = tl;
        set_mod(ctx, &gu, i, j, 3, pre_depth, 1);
        if (one && !gu.mod_g) gu.A16 = y16;
        if (few) TLF_HIP(launch_dgemm<T>(gu, A_SRC, E_SWIGLU, true, ctx->cus, s));
        else TLF_HIP(launch_gemm<T>(gu, A_SRC, E_SWIGLU, false, s));

        GemmArgs dn;
        dn.A = ctx->buf<float>(B_ACT_PRE); dn.lda = F; dn.W = lw.w_down; dn.Wf = ctx->wfrag(j, 3); dn.N = d; dn.K = F; dn.w_rows = d;
        dn.rm = rm; dn.out = x; dn.ldo = d; dn.scatter = 1; dn.spec = i == 0; dn.a_single = one; dn.A16 = act16;
        dn.tl = tl;
        set_mod(ctx, &dn, i, j, 1, pre_depth, 1);
        if (few) {
          TLF_HIP(launch_dgemm<T>(dn, A_CMP, E_RESID, false, ctx->cus, s));
        } else {
          TLF_HIP(launch_gemm<T>(dn, A_CMP, E_RESID, false, s));
          TLF_HIP(launch_resid_norm<T>(rn, s));
        }
      }
    }
    GemmArgs hd;
    hd.A = few ? x : y; hd.lda = d; hd.W = head_weights(ctx); hd.N = c.vocab; hd.K = d; hd.w_rows = c.vocab;
    hd.out = logits; hd.ldo = c.vocab; hd.eps = c.rms_eps; hd.spec = 1;
    if (flags & TLF_PREFILL_ALL_LOGITS) {
      hd.rm.rows = rows; hd.rm.src_stride = 1; hd.rm.src_off = 0;
      hd.out_row_off = b0 * T_;
    } else {
      hd.rm.rows = Gc; hd.rm.src_stride = T_; hd.rm.src_off = T_ - 1;
      hd.out_row_off = b0;
    }
    if (!y32) {
      ResidNormArgs hn;
      hn.rm = hd.rm; hn.x = x; hn.y = y; hn.d = d; hn.eps = c.rms_eps;
      TLF_HIP(launch_resid_norm<T>(hn, s));
    }
    if (few) TLF_HIP(launch_dgemm<T>(hd, A_SRC, E_LOGITS, true, ctx->cus, s));
    else TLF_HIP(launch_gemm<T>(hd, A_SRC, E_LOGITS, false, s));
  }
  return TLF_OK;
}

template <typename T>
int run_decode(tlf_ctx* ctx, hipStream_t s, const int32_t* tokens, float* logits, int32_t* next,
               int32_t* depths, float* margin) {
  const tlf_config& c = ctx->cfg;
  const int d = c.d_model, F = c.d_ff, R = c.max_loops, B = ctx->batch;
  float* x = ctx->buf<float>(B_X_DEC);    // batch order (embedding)
  float* xc = ctx->buf<float>(B_XC_DEC);  // compact order: row k is sequence perm[k]
  int64_t* kv_slot = ctx->buf<int64_t>(B_KVSLOT);
  int32_t* perm = ctx->buf<int32_t>(B_PERM);
  int32_t* nact = ctx->buf<int32_t>(B_NACT);

  EmbedArgs ea;
  ea.tok_emb = ctx->w.tok_emb; ea.pos_emb = ctx->w.pos_emb; ea.Wr = ctx->w.router_w; ea.br = ctx->w.router_b;
  ea.tokens = tokens; ea.rows = B; ea.V = c.vocab; ea.d = d; ea.R = R; ea.prefill_T = 0;
  ea.seq_len = ctx->cv.seq_len; ea.x = x; ea.y = nullptr; ea.eps = c.rms_eps;
  ea.depth = ctx->buf<int32_t>(B_DEPTH_DEC);
  ea.out_depth = depths; ea.out_margin = margin;
  ea.rule = c.route_rule; ea.threshold = c.route_threshold; ea.fixed = c.fixed_depth; ea.err = ctx->cv.err;
  ea.route = c.router_hidden == 0;
  TLF_HIP(launch_embed_route<T>(ea, s));
  if (c.router_hidden > 0) {
    const int st = run_mlp_router<T>(ctx, s, x, B, true, ea.depth, depths, margin);
    if (st != TLF_OK) return st;
  }

  DecodePlanArgs pa;
  pa.c = ctx->cv; pa.B = B; pa.depth = ctx->buf<int32_t>(B_DEPTH_DEC); pa.perm = perm; pa.nact = nact;
  pa.kv_slot = kv_slot;
  pa.kv_entry_bytes = (int64_t)c.n_layers * 2 * c.d_model * ctx->L.s;
  pa.dense = c.dense_decode;
  pa.row_depth = ctx->buf<int32_t>(B_ROW_DEPTH);
  TLF_HIP(launch_plan_decode(pa, s));
  // dense decode: rows are in batch order and a row's result is kept while its
  // token's depth exceeds the loop index
  const int32_t* keep_depth = c.dense_decode ? ctx->buf<int32_t>(B_DEPTH_DEC) : nullptr;
  // bf16 models keep the step's compact residual xc in MFMA fragment order
  // (element (R, k) at frag_index(R, k, d)): the QKV and gate/up projections
  // and the LM head load whole fragments, the O and down epilogues update it
  // in place; float32 fragments hold one element per lane and keep rows
  const bool xfrag = c.dtype == TLF_DTYPE_BF16;

  // the block region (every loop and layer) is timed as a whole when profiling;
  // the attention launches inside it get their own event pairs
  hipEvent_t block_start = nullptr, block_stop = nullptr;
  if (ctx->profiling) {
    TLF_HIP(ctx->take_event(&block_start));
    TLF_HIP(ctx->take_event(&block_stop));
    TLF_HIP(hipEventRecord(block_start, s));
  }
  for (int i = 0; i < R; ++i) {
    // rows [0, n_i) of the depth-sorted order are the tokens still active at
    // loop i; row k is sequence perm[k], its residual xc[k] (dense decode:
    // every row, perm the identity)
    RowMap rm;
    rm.src = perm; rm.nact = nact + i; rm.rows = B;
    for (int j = 0; j < c.n_layers; ++j) {
      const tlf_layer_weights& lw = ctx->layers[j];
      GemmArgs q;  // q, k, v of RMSNorm(x); k, v appended to cache (b, i) of layer j
      const bool first = i == 0 && j == 0;  // reads x through perm and writes xc
      q.A = first ? x : xc; q.lda = d; q.a_copy = first ? xc : nullptr; q.W = lw.w_qkv; q.Wf = ctx->wfrag(j, 0); q.N = 3 * d; q.K = d; q.w_rows = 3 * d; q.rm = rm;
      q.copy_frag = first && xfrag; q.a_frag = !first && xfrag;
      q.out = ctx->buf<float>(B_Q_DEC); q.ldo = d; q.d = d; q.eps = c.rms_eps;
      q.kv.c = ctx->cv; q.kv.loop = i; q.kv.layer = j; q.kv.slot_base = kv_slot + (int64_t)i * B;
      q.spec = i == 0;
      set_mod(ctx, &q, i, j, 2, pa.row_depth, 0);
      TLF_HIP(launch_dgemm<T>(q, first ? A_SRC : A_CMP, E_QKV, true, ctx->cus, s));

      AttnDecodeArgs at;
      at.c = ctx->cv; at.loop = i; at.layer = j; at.d = d; at.perm = perm; at.nact = nact + i;
      at.q = ctx->buf<float>(B_Q_DEC); at.o = ctx->buf<float>(B_O_DEC);
      // o and act in MFMA fragment order for the O and down projections (d and F
      // are multiples of 64 or 128, so of KS: validate_config)
      at.o_ks = Mfma<T>::KS; at.o_epl = Mfma<T>::EPL;
      at.scale_log2 = 1.4426950408889634f / std::sqrt((float)c.head_dim);
      at.waves = attn_waves(ctx);
      at.grid = ctx->cus * ctx->attn_blocks[at.waves == 4 ? 0 : 1];
      if (ctx->profile_attn) {
        TLF_HIP(ctx->begin_timed(s, true));
        TLF_HIP(launch_attn_decode<T>(at, s));
        TLF_HIP(ctx->end_timed(s));
      } else {
        TLF_HIP(launch_attn_decode<T>(at, s));
      }

      GemmArgs o;  // x += o W_o^T
      o.A = ctx->buf<float>(B_O_DEC); o.lda = d; o.W = lw.w_o; o.Wf = ctx->wfrag(j, 1); o.N = d; o.K = d; o.w_rows = d; o.rm = rm;
      o.a_frag = 1;
      o.out = xc; o.ldo = d; o.spec = i == 0; o.keep_depth = keep_depth; o.keep_loop = i; o.out_frag = xfrag;
      set_mod(ctx, &o, i, j, 0, pa.row_depth, 0);
      TLF_HIP(launch_dgemm<T>(o, A_CMP, E_RESID, false, ctx->cus, s));

      GemmArgs gu;  // act = silu(RMSNorm(x) W_g^T) * (RMSNorm(x) W_u^T)
      gu.A = xc; gu.lda = d; gu.W = lw.w_gate_up; gu.Wf = ctx->wfrag(j, 2); gu.N = 2 * F; gu.K = d; gu.w_rows = 2 * F; gu.rm = rm;
      gu.out = ctx->buf<float>(B_ACT_DEC); gu.ldo = F; gu.F = F; gu.eps = c.rms_eps; gu.spec = i == 0;
      gu.out_frag = 1; gu.a_frag = xfrag;
      set_mod(ctx, &gu, i, j, 3, pa.row_depth, 0);
      TLF_HIP(launch_dgemm<T>(gu, A_CMP, E_SWIGLU, true, ctx->cus, s));

      GemmArgs dn;  // x += act W_d^T
      dn.A = ctx->buf<float>(B_ACT_DEC); dn.lda = F; dn.W = lw.w_down; dn.Wf = ctx->wfrag(j, 3); dn.N = d; dn.K = F; dn.w_rows = d;
      dn.a_frag = 1;
      dn.rm = rm; dn.out = xc; dn.ldo = d; dn.spec = i == 0; dn.keep_depth = keep_depth; dn.keep_loop = i;
      dn.out_frag = xfrag;
      set_mod(ctx, &dn, i, j, 1, pa.row_depth, 0);
      TLF_HIP(launch_dgemm<T>(dn, A_CMP, E_RESID, false, ctx->cus, s));
    }
  }
  if (ctx->profiling) {
    TLF_HIP(hipEventRecord(block_stop, s));
    ctx->event_pending.push_back(tlf_ctx::Timed{block_start, block_stop, false});
  }
  // every compact row now holds its sequence's last state h^(m_b):
  // logits[perm[k]] = RMSNorm(xc[k]) E^T
  GemmArgs hd;
  hd.A = xc; hd.lda = d; hd.W = head_weights(ctx); hd.N = c.vocab; hd.K = d; hd.w_rows = c.vocab;
  hd.rm.src = perm; hd.rm.rows = B; hd.out = logits; hd.ldo = c.vocab; hd.eps = c.rms_eps; hd.spec = 1;
  hd.a_frag = xfrag;
  hd.argmax_keys = ctx->buf<unsigned long long>(B_KEYS);
  hd.key_groups = (int)ceil_div(c.vocab, kWave);
  // a large batch makes the head a real GEMM (128 x 128 tiles read each
  // weight row B / 128 times); a small one is the split-K projection
  if (B >= kHeadGemmRows) TLF_HIP(launch_gemm<T>(hd, A_CMP, E_LOGITS, true, s));
  else TLF_HIP(launch_dgemm<T>(hd, A_CMP, E_LOGITS, true, ctx->cus, s));
  if (next) TLF_HIP(launch_argmax_finalize(ctx->buf<unsigned long long>(B_KEYS), hd.key_groups, next, B, s));
  return TLF_OK;
}

int device_status(int err_bits) {
  if (err_bits & kErrOutOfPages) return TLF_E_OUT_OF_PAGES;
  if (err_bits & kErrBadToken) return TLF_E_DEVICE;
  return TLF_OK;
}

}  // namespace

extern "C" {

int tlf_init(const tlf_config* cfg, const tlf_weights* w, void* d_workspace, size_t ws_bytes,
             size_t* ws_needed, void* hip_stream, tlf_ctx** out) {
  int st = validate_config(cfg);
  if (st != TLF_OK) return st;
  Layout L;
  if (!make_layout(*cfg, &L)) return TLF_E_INVALID_ARG;
  if (ws_needed) *ws_needed = L.total;
  if (!d_workspace || ws_bytes < L.total) return TLF_E_NEED_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(d_workspace) % 256 != 0) return TLF_E_INVALID_ARG;
  st = validate_weights(cfg, w);
  if (st != TLF_OK) return st;
  if (!out) return TLF_E_INVALID_ARG;

  tlf_ctx* ctx = new (std::nothrow) tlf_ctx();
  if (!ctx) return TLF_E_INVALID_ARG;
  ctx->cfg = *cfg;
  ctx->w = *w;
  ctx->layers.assign(w->layers, w->layers + w->n_layers);
  ctx->w.layers = ctx->layers.data();
  ctx->L = L;
  ctx->stream = reinterpret_cast<hipStream_t>(hip_stream);
  ctx->ws = reinterpret_cast<char*>(d_workspace);

  CacheView& cv = ctx->cv;
  cv.pool = ctx->buf<void>(B_POOL);
  cv.pos = ctx->buf<int32_t>(B_POS);
  cv.page_table = ctx->buf<int32_t>(B_PAGE_TABLE);
  cv.cache_len = ctx->buf<int32_t>(B_CACHE_LEN);
  cv.seq_len = ctx->buf<int32_t>(B_SEQ_LEN);
  cv.chunk_len = ctx->buf<int32_t>(B_CHUNK_LEN);
  cv.page_next = ctx->buf<int32_t>(B_SCALARS);
  cv.err = ctx->buf<int32_t>(B_SCALARS) + 1;
  cv.depth_hist = ctx->buf<unsigned long long>(B_DEPTH_HIST);
  cv.step_stats = ctx->buf<long long>(B_STEP_STATS);
  cv.page_elems = L.page_elems;
  cv.max_pages = cfg->max_pages;
  cv.pages_per_seq = L.pages_per_seq;
  cv.R = cfg->max_loops;
  cv.J = cfg->n_layers;
  cv.H = cfg->n_heads;
  cv.D = cfg->head_dim;

  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) { delete ctx; return TLF_E_HIP; }
  ctx->cus = std::max(1, cus);
  for (int k = 0; k < 2 && e == hipSuccess; ++k) {
    int blocks = 0;
    e = cfg->dtype == TLF_DTYPE_BF16 ? attn_decode_blocks_per_cu<bf16>(cfg->head_dim, 4 << k, &blocks)
                                     : attn_decode_blocks_per_cu<float>(cfg->head_dim, 4 << k, &blocks);
    ctx->attn_blocks[k] = std::max(1, blocks);
  }
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&ctx->cap_stream, hipStreamNonBlocking);
  if (e != hipSuccess) { delete ctx; return TLF_E_HIP; }

  // The pool starts zeroed: attention kernels read whole 16-slot pages and
  // give zero weight to slots past a cache's length, which must hold finite
  // values (zeros here, or stale entries of an earlier batch).
  hipStream_t s = ctx->stream;
  const int64_t pool_words = (int64_t)(L.size[B_POOL] / 4);
  e = launch_fill_i32(reinterpret_cast<int32_t*>(cv.pool), 0, pool_words, s);
  if (e == hipSuccess) e = launch_fill_i32(cv.pos, -1, (int64_t)cfg->max_pages * kPage, s);
  if (e == hipSuccess) e = launch_fill_i32(cv.page_table, -1, (int64_t)(L.size[B_PAGE_TABLE] / 4), s);
  if (e == hipSuccess) e = launch_fill_i32(cv.cache_len, 0, (int64_t)cfg->max_batch * cfg->max_loops, s);
  if (e == hipSuccess) e = launch_fill_i32(cv.chunk_len, 0, (int64_t)cfg->max_batch * cfg->max_loops, s);
  if (e == hipSuccess) e = launch_fill_i32(cv.seq_len, 0, cfg->max_batch, s);
  if (e == hipSuccess) e = launch_fill_i32(cv.page_next, 0, 2, s);
  if (e == hipSuccess) e = launch_fill_u64(cv.depth_hist, 0ull, cfg->max_loops, s);
  if (e == hipSuccess) e = launch_fill_u64(reinterpret_cast<unsigned long long*>(cv.step_stats), 0ull, kStatCount, s);
  // the decode projections read the block weights in MFMA fragment order
  for (int j = 0; j < cfg->n_layers && e == hipSuccess; ++j) {
    const tlf_layer_weights& lw = ctx->layers[j];
    const int d = cfg->d_model, F = cfg->d_ff;
    const bool bf = cfg->dtype == TLF_DTYPE_BF16;
    auto relayout = [&](const void* W, int part, int N, int K, int sF) {
      void* dst = const_cast<void*>(ctx->wfrag(j, part));
      return bf ? launch_wfrag<bf16>(W, dst, N, K, sF, s) : launch_wfrag<float>(W, dst, N, K, sF, s);
    };
    e = relayout(lw.w_qkv, 0, 3 * d, d, 0);
    if (e == hipSuccess) e = relayout(lw.w_o, 1, d, d, 0);
    if (e == hipSuccess) e = relayout(lw.w_gate_up, 2, 2 * F, d, F);
    if (e == hipSuccess) e = relayout(lw.w_down, 3, d, F, 0);
  }
  if (e == hipSuccess && cfg->adaln) {
    // the modulation of every (layer, loop, depth); the caller's conditioning
    // weights are not read again
    const tlf_adaln_weights& a = *w->adaln;
    CondWeights cw;
    cw.w1[0] = a.time_w1; cw.b1[0] = a.time_b1; cw.w2[0] = a.time_w2; cw.b2[0] = a.time_b2;
    cw.w1[1] = a.step_w1; cw.b1[1] = a.step_b1; cw.w2[1] = a.step_w2; cw.b2[1] = a.step_b2;
    cw.mod_w = a.mod_w; cw.mod_b = a.mod_b;
    float* table = ctx->buf<float>(B_MOD);
    float* tmp = ctx->buf<float>(B_COND_TMP);
    e = cfg->dtype == TLF_DTYPE_BF16
            ? launch_cond_table<bf16>(cw, cfg->n_layers, cfg->max_loops, cfg->d_model, table, tmp, s)
            : launch_cond_table<float>(cw, cfg->n_layers, cfg->max_loops, cfg->d_model, table, tmp, s);
  }
  ctx->w.adaln = nullptr;
  if (e != hipSuccess) { delete ctx; return TLF_E_HIP; }
  *out = ctx;
  return TLF_OK;
}

int tlf_prefill(tlf_ctx* ctx, int32_t batch, int32_t seq_len, const int32_t* d_tokens, float* d_logits,
                int32_t* d_depths, uint32_t flags) {
  int st = precheck(ctx);
  if (st != TLF_OK) return st;
  const tlf_config& c = ctx->cfg;
  if (batch < 1 || batch > c.max_batch || seq_len < 1 || seq_len > c.max_pos) return TLF_E_INVALID_ARG;
  if (!d_tokens || !d_logits || (flags & ~(TLF_PREFILL_ALL_LOGITS | TLF_PREFILL_APPEND))) return TLF_E_INVALID_ARG;
  const bool append = (flags & TLF_PREFILL_APPEND) != 0;
  int pos0 = 0;
  if (append) {
    if (!ctx->prefilled) return TLF_E_STATE;
    if (batch != ctx->batch || seq_len > c.max_pos - ctx->seq_len) return TLF_E_INVALID_ARG;
    pos0 = ctx->seq_len;
  } else {
    // loop 1 alone needs one page per 16 tokens of every sequence
    if ((int64_t)batch * ceil_div(seq_len, kPage) > c.max_pages) return TLF_E_OUT_OF_PAGES;
    ctx->prefilled = false;
  }
  st = c.dtype == TLF_DTYPE_BF16
           ? run_prefill<bf16>(ctx, batch, seq_len, pos0, d_tokens, d_logits, d_depths, flags)
           : run_prefill<float>(ctx, batch, seq_len, pos0, d_tokens, d_logits, d_depths, flags);
  if (st != TLF_OK) return st;
  ctx->batch = batch;
  ctx->seq_len = pos0 + seq_len;
  ctx->prefilled = true;
  return TLF_OK;
}

int tlf_decode_step(tlf_ctx* ctx, const int32_t* d_tokens, float* d_logits, int32_t* d_next,
                    int32_t* d_depths, float* d_margin) {
  int st = precheck(ctx);
  if (st != TLF_OK) return st;
  if (!ctx->prefilled || ctx->seq_len >= ctx->cfg.max_pos) return TLF_E_STATE;
  if (!d_tokens || !d_logits) return TLF_E_INVALID_ARG;
  auto enqueue = [&](hipStream_t s) {
    return ctx->cfg.dtype == TLF_DTYPE_BF16
               ? run_decode<bf16>(ctx, s, d_tokens, d_logits, d_next, d_depths, d_margin)
               : run_decode<float>(ctx, s, d_tokens, d_logits, d_next, d_depths, d_margin);
  };
  if (ctx->cfg.decode_graph && !ctx->profiling) {
    const tlf_ctx::GraphKey key{ctx->batch, d_tokens, d_logits, d_next, d_depths, d_margin};
    tlf_ctx::CachedGraph* g = nullptr;
    for (tlf_ctx::CachedGraph& c : ctx->graphs)
      if (c.exec && c.key == key) g = &c;
    if (!g) {
      // the free or least recently used entry takes the new graph
      g = &ctx->graphs[0];
      for (tlf_ctx::CachedGraph& c : ctx->graphs)
        if (!c.exec || (g->exec && c.used < g->used)) g = &c;
      if (g->exec) {
        (void)hipGraphExecDestroy(g->exec);
        g->exec = nullptr;
      }
      // nothing runs while capturing; the graph is replayed on the context's stream
      if (hipStreamBeginCapture(ctx->cap_stream, hipStreamCaptureModeThreadLocal) != hipSuccess) {
        ctx->poisoned = true;
        return TLF_E_HIP;
      }
      st = enqueue(ctx->cap_stream);
      hipGraph_t graph = nullptr;
      const hipError_t ec = hipStreamEndCapture(ctx->cap_stream, &graph);
      if (st != TLF_OK || ec != hipSuccess || !graph) {
        if (graph) (void)hipGraphDestroy(graph);
        ctx->poisoned = true;
        return st != TLF_OK ? st : TLF_E_HIP;
      }
      const hipError_t ei = hipGraphInstantiate(&g->exec, graph, nullptr, nullptr, 0);
      (void)hipGraphDestroy(graph);
      if (ei != hipSuccess) {
        g->exec = nullptr;
        ctx->poisoned = true;
        return TLF_E_HIP;
      }
      g->key = key;
    }
    g->used = ++ctx->graph_clock;
    if (hipGraphLaunch(g->exec, ctx->stream) != hipSuccess) {
      ctx->poisoned = true;
      return TLF_E_HIP;
    }
  } else {
    st = enqueue(ctx->stream);
    if (st != TLF_OK) return st;
  }
  ctx->seq_len += 1;
  return TLF_OK;
}

int tlf_cache_stats(tlf_ctx* ctx, tlf_cache_stats_t* out, int32_t* h_len, int32_t* h_pos, size_t pos_cap) {
  if (!ctx || !out) return TLF_E_INVALID_ARG;
  if (ctx->poisoned) return TLF_E_STATE;
  const tlf_config& c = ctx->cfg;
  const int B = ctx->batch, R = c.max_loops;
  if (h_pos && !ctx->prefilled) return TLF_E_STATE;
  std::memset(out, 0, sizeof(*out));
  hipError_t e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) { ctx->poisoned = true; return TLF_E_HIP; }
  std::vector<int32_t> len((size_t)std::max(B, 1) * R, 0);
  int32_t scal[2] = {0, 0};
  unsigned long long hist[TLF_MAX_LOOPS] = {0};
  long long stats[kStatCount] = {0};
  if (B > 0) e = hipMemcpy(len.data(), ctx->cv.cache_len, sizeof(int32_t) * B * R, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(scal, ctx->cv.page_next, sizeof(scal), hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(hist, ctx->cv.depth_hist, sizeof(unsigned long long) * R, hipMemcpyDeviceToHost);
  if (e == hipSuccess) e = hipMemcpy(stats, ctx->cv.step_stats, sizeof(stats), hipMemcpyDeviceToHost);
  if (e != hipSuccess) { ctx->poisoned = true; return TLF_E_HIP; }

  const int64_t page_bytes = ctx->L.page_elems * ctx->L.s;
  for (int i = 0; i < R; ++i) {
    for (int b = 0; b < B; ++b) {
      out->slots_per_loop[i] += len[(size_t)b * R + i];
      out->pages_per_loop[i] += ceil_div(len[(size_t)b * R + i], kPage);
    }
    out->depth_hist[i] = (int64_t)hist[i];
    out->last_step_active_rows[i] = stats[kStatRows + i];
  }
  out->pages_used = std::min<int64_t>(scal[0], c.max_pages);
  out->pages_total = c.max_pages;
  out->kv_bytes_resident = out->pages_used * page_bytes;
  out->batch = B;
  out->seq_len = ctx->seq_len;
  out->last_step_kv_read_bytes = stats[kStatKvRead];
  out->last_step_kv_write_bytes = stats[kStatKvWrite];
  out->last_step_loops_executed = stats[kStatLoops];
  const int64_t block_params = 4LL * c.d_model * c.d_model + 3LL * c.d_model * c.d_ff;
  out->last_step_weight_bytes = stats[kStatLoops] * c.n_layers * block_params * ctx->L.s +
                                (int64_t)c.vocab * c.d_model * ctx->L.s + (int64_t)R * c.d_model * 4;
  for (auto& t : ctx->event_pending) {
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, t.start, t.stop);
    if (e != hipSuccess) { ctx->poisoned = true; return TLF_E_HIP; }
    if (t.attn) {
      ctx->attn_ms += ms;
      ctx->attn_launches += 1;
    } else {
      ctx->block_ms += ms;
    }
  }
  ctx->recycle_events();
  out->decode_steps = stats[kStatStepsTotal];
  out->attn_launches = ctx->attn_launches;
  out->attn_algo_bytes = stats[kStatAttnBytesTotal];
  out->attn_ms = ctx->attn_ms;
  out->kv_write_bytes_total = stats[kStatKvWriteTotal];
  out->loops_executed_total = stats[kStatLoopsTotal];
  out->block_ms = ctx->block_ms;
  out->device_error = device_status(scal[1]);
  if (out->device_error != TLF_OK) ctx->sticky = out->device_error;

  if (h_len && B > 0) std::memcpy(h_len, len.data(), sizeof(int32_t) * B * R);
  if (h_pos && B > 0) {
    size_t need = 0;
    for (size_t k = 0; k < (size_t)B * R; ++k) need += (size_t)len[k];
    if (pos_cap < need) return TLF_E_INVALID_ARG;
    const int pps = ctx->L.pages_per_seq;
    std::vector<int32_t> pt((size_t)B * R * pps);
    std::vector<int32_t> pos((size_t)c.max_pages * kPage);
    e = hipMemcpy(pt.data(), ctx->cv.page_table, sizeof(int32_t) * pt.size(), hipMemcpyDeviceToHost);
    if (e == hipSuccess) e = hipMemcpy(pos.data(), ctx->cv.pos, sizeof(int32_t) * pos.size(), hipMemcpyDeviceToHost);
    if (e != hipSuccess) { ctx->poisoned = true; return TLF_E_HIP; }
    size_t o = 0;
    for (int b = 0; b < B; ++b)
      for (int i = 0; i < R; ++i) {
        const int n = len[(size_t)b * R + i];
        for (int t = 0; t < n; ++t) {
          const int page = pt[((size_t)b * R + i) * pps + t / kPage];
          h_pos[o++] = (page >= 0 && page < c.max_pages) ? pos[(size_t)page * kPage + t % kPage] : -1;
        }
      }
  }
  return out->device_error;
}

int tlf_set_profiling(tlf_ctx* ctx, int mode) {
  if (!ctx) return TLF_E_INVALID_ARG;
  if (mode != TLF_PROFILE_OFF && mode != TLF_PROFILE_ATTN && mode != TLF_PROFILE_BLOCK) return TLF_E_INVALID_ARG;
  if (ctx->poisoned) return TLF_E_STATE;
  if (mode != TLF_PROFILE_OFF) {
    // reset the totals: cumulative device counters and the host-side sums
    static_assert(kStatLoopsTotal == kStatAttnBytesTotal + 3, "cumulative counters are contiguous");
    TLF_HIP(launch_fill_u64(reinterpret_cast<unsigned long long*>(ctx->cv.step_stats) + kStatAttnBytesTotal, 0ull,
                            4, ctx->stream));
    ctx->attn_launches = 0;
    ctx->attn_ms = 0.0;
    ctx->block_ms = 0.0;
    ctx->recycle_events();
  }
  ctx->profiling = mode != TLF_PROFILE_OFF;
  ctx->profile_attn = mode == TLF_PROFILE_ATTN;
  return TLF_OK;
}

void tlf_destroy(tlf_ctx* ctx) {
  if (!ctx) return;
  if (!ctx->poisoned) (void)hipStreamSynchronize(ctx->stream);
  delete ctx;
}

const char* tlf_status_str(int status) {
  switch (status) {
    case TLF_OK: return "ok";
    case TLF_E_INVALID_ARG: return "invalid argument";
    case TLF_E_NEED_WORKSPACE: return "workspace needed";
    case TLF_E_OUT_OF_PAGES: return "KV page pool exhausted";
    case TLF_E_STATE: return "invalid state";
    case TLF_E_HIP: return "HIP runtime error";
    case TLF_E_DEVICE: return "device-detected input error";
    case TLF_E_UNSUPPORTED: return "shape or size not supported by this build";
    default: return "unknown status";
  }
}

}  // extern "C"
