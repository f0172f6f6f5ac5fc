/*
 * tlf.h - C ABI of libtlf: routed prefill and decode of a looped, weight-shared
 * transformer with token-level depth and a recursion-wise KV cache
 * (T-LoopFormer, Section 3.2 and Section 3.3), for AMD Instinct MI355X (gfx950).
 *
 * Model
 *   h0 = E[x] + P[pos] (token plus learned absolute position, added once;
 *   Section 3 and Section 3.2).  A router maps h0 to R logits (Eq. 2) and a
 *   depth rule turns them into the token's loop count m in [1, R] (Eq. 3-5, or
 *   argmax, or a fixed depth).  Loop i (1..R) applies the shared block of J
 *   pre-norm layers (RMSNorm without affine, multi-head attention, SwiGLU FFN,
 *   residuals inside each layer; Appendix A) to the tokens with m >= i only
 *   (gather, Eq. 6; scatter, Eq. 7).  Exited tokens keep h^(m).  Logits are
 *   RMSNorm(h^(m)) times the LM head (tied to E unless a head is given).
 *
 * Recursion-wise KV cache (Eq. 8-11)
 *   Every (sequence b, loop i) owns its own cache, shared by the J layers'
 *   K/V planes.  A token that executes loop i writes its k, v there (Eq. 11);
 *   a query at loop i attends only to the entries of that cache (Eq. 10): the
 *   earlier tokens of the sequence whose depth is >= i, and itself.  Entries
 *   are stored compactly in position order in 16-token pages, with the
 *   original position of every entry recorded; tokens that never reached loop
 *   i occupy no slot, so the validity mask of Eq. 10 is implicit.
 *
 * Conventions
 *   - Every function returns an int status (TLF_OK or a negative TLF_E_*
 *     code); no C++ exception crosses this boundary.
 *   - Device pointers ("d_") are HIP device memory on the device that is
 *     current when tlf_init is called.  Host pointers ("h_") are host memory.
 *   - Weights and the workspace are borrowed: the caller keeps them alive and
 *     unchanged until tlf_destroy.  Outputs are caller-allocated.  The context
 *     owns only host-side state.  tlf_init also writes a copy of every
 *     layer's block weights into the workspace, reordered for the decode
 *     projections' matrix-core loads (counted in the workspace size).
 *   - Work is enqueued asynchronously on the stream given to tlf_init; only
 *     tlf_cache_stats waits for the stream.  A context is not thread-safe.
 *   - Arguments are validated on the host before any device work; an argument
 *     error (TLF_E_INVALID_ARG, TLF_E_STATE) leaves the context unchanged.
 *   - A HIP error (TLF_E_HIP) poisons the context: later calls return
 *     TLF_E_STATE.  Errors found on the device (a token id out of range, the
 *     page pool exhausted) are sticky and are returned by tlf_cache_stats and
 *     by every call after it.
 */
#ifndef TLF_H
#define TLF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TLF_ABI_VERSION 5
#define TLF_MAX_LOOPS 16
#define TLF_MAX_LAYERS 8
#define TLF_MAX_BATCH 4096
#define TLF_PAGE_TOKENS 16

/* Status codes. */
#define TLF_OK 0
#define TLF_E_INVALID_ARG (-1)    /* bad argument: no valid model, call or buffer */
#define TLF_E_NEED_WORKSPACE (-2) /* tlf_init size query: *ws_needed is set */
#define TLF_E_OUT_OF_PAGES (-3)   /* the KV page pool (max_pages) is exhausted */
#define TLF_E_STATE (-4)          /* call not valid in this state (e.g. decode before prefill) */
#define TLF_E_HIP (-5)            /* a HIP runtime call failed; the context is poisoned */
#define TLF_E_DEVICE (-6)         /* the device found a bad input (token id out of range) */
#define TLF_E_UNSUPPORTED (-7)    /* a valid config outside this build's shapes and sizes (tlf_init) */

/* Storage dtype of embeddings, block weights and the KV cache.  The residual
 * stream, the activations passed between kernels (normalised rows, q,
 * attention output, SwiGLU output), router, softmax, accumulators and logits
 * are float32 in both cases; with bf16 weights each float32 activation enters
 * a matrix product as the sum of two bf16 parts (hi + lo), so only the weights,
 * the cached k and v, and the attention probabilities are rounded to bf16. */
#define TLF_DTYPE_F32 0
#define TLF_DTYPE_BF16 1

/* Depth rules (Section 3.2). */
#define TLF_ROUTE_ARGMAX 0  /* m = 1 + index of the largest router logit (lowest on ties) */
#define TLF_ROUTE_CUMPROB 1 /* m = max{i : sum_{l>=i} softmax(z)_l > threshold} (Eq. 2-5) */
#define TLF_ROUTE_FIXED 2   /* m = fixed_depth for every token (fixed-depth looped model) */

/* tlf_prefill flags. */
#define TLF_PREFILL_ALL_LOGITS 1u /* logits for every position ([B][T][V]) instead of the last */
#define TLF_PREFILL_APPEND 2u     /* continue the current batch: the tokens are its next positions */

typedef struct tlf_config {
  int32_t abi_version;   /* must be TLF_ABI_VERSION */
  int32_t dtype;         /* TLF_DTYPE_F32 or TLF_DTYPE_BF16 */
  int32_t vocab;         /* V >= 1 */
  int32_t d_model;       /* d <= 4096, multiple of 128 (bf16) or 64 (float32) */
  int32_t n_heads;       /* H, n_heads * head_dim == d_model */
  int32_t head_dim;      /* D: 64 or 128 (16 for float32 models only) */
  int32_t d_ff;          /* F, SwiGLU hidden width, multiple of 128 (bf16) or 64 (float32) */
  int32_t n_layers;      /* J in [1, TLF_MAX_LAYERS], layers of the shared block */
  int32_t max_loops;     /* R = M in [1, TLF_MAX_LOOPS], router width and loop cap */
  int32_t max_pos;       /* rows of the position table, <= 65536; prompt + decode steps <= max_pos */
  int32_t max_batch;     /* sequences per call, in [1, TLF_MAX_BATCH] */
  int32_t page_tokens;   /* tokens per KV page, must be TLF_PAGE_TOKENS */
  int32_t max_pages;     /* KV pages in the pool (all sequences and loops) */
  int32_t max_prefill_tokens; /* activation rows for prefill; larger prefills run in sequence groups */
  int32_t route_rule;    /* TLF_ROUTE_* */
  float route_threshold; /* CUMPROB threshold in (0, 1); the paper uses 0.5 */
  int32_t fixed_depth;   /* FIXED depth in [1, R] */
  float rms_eps;         /* RMSNorm epsilon (> 0) */
  int32_t decode_graph;  /* 1: each decode step replays a captured HIP graph; a graph belongs to
                            the batch and the step's token and output pointers, the graphs of
                            the last 4 distinct ones are kept (a step whose tokens are the
                            previous step's next_tokens alternates between two) and a new one
                            is captured in place of the least recently used;
                            0: kernels are launched one by one */
  int32_t router_hidden; /* 0: linear router z = W_r h0 + b_r; Hr > 0 (<= 4096, multiple of 64): the
                            two-layer MLP router z = W_r silu(W_1 h0 + b_1) + b_r (Section 3.2) */
  int32_t dense_decode;  /* 0: each decode loop runs on the gathered active rows (Eq. 6-7);
                            1: gather-scatter off (the ablation of Section 4's latency study):
                            every loop up to the step's deepest token runs on all rows of the
                            batch, exited rows are computed and discarded at the scatter and
                            write no cache entry, attention keeps the validity mask of Eq. 10.
                            Same results as 0; prefill is not affected */
  int32_t adaln;         /* 0: unconditioned block; 1: AdaLN time/step conditioning (Section 3.1,
                            Appendix A; weights in tlf_weights.adaln): a token of depth m at
                            loop i has cumulative time (i-1)/m and step 1/m, and layer j's
                            modulation (alpha_msa, alpha_mlp, gamma_msa, gamma_mlp) enters as
                            x += (1 + alpha) * F(RMSNorm(x) * (1 + gamma)) */
  int32_t prefill_act_bf16; /* bf16 models, prefills of more than one sequence or longer than 2048
                               tokens: 0: the float32 activations enter the block's matrix products
                               and the attention scores as bf16 hi + lo parts; 1: as one bf16 part
                               (round to nearest even), half the matrix-core work.  Decode steps and
                               every LM head keep the two parts.  An exact bf16 implementation with
                               every activation rounded stays within 1.9e-2 of float64 on the
                               logits at d_model 1024 but reaches 4.1e-2 at 2048 */
} tlf_config;

/* Weights of layer j of the shared block, row-major [out][in] (y = x W^T),
 * in the storage dtype. */
typedef struct tlf_layer_weights {
  const void* w_qkv;     /* [3d][d]: rows q | k | v, each head-major (head h = rows h*D..h*D+D-1) */
  const void* w_o;       /* [d][d] */
  const void* w_gate_up; /* [2F][d]: rows gate | up; FFN(y) = W_down (silu(W_gate y) * (W_up y)) */
  const void* w_down;    /* [d][F] */
} tlf_layer_weights;

/* AdaLN conditioning weights (config.adaln = 1), row-major [out][in]:
 * matrices in the storage dtype, biases float32.  Each conditioning scalar
 * s becomes 256 Fourier features [cos(s w_1), sin(s w_1), ..., cos(s w_128),
 * sin(s w_128)], w_k = 10000^(-(k-1)/128), then phi(s) = W_2 silu(W_1 f + b_1)
 * + b_2; the embedding is phi_time(c) + phi_step(Delta), and layer j's
 * modulation is mod_w[j] silu(embedding) + mod_b[j].  Read by tlf_init only:
 * the modulation of every (layer, loop, depth) is tabulated there. */
typedef struct tlf_adaln_weights {
  const void* time_w1;  /* [d][256] */
  const float* time_b1; /* [d] */
  const void* time_w2;  /* [d][d] */
  const float* time_b2; /* [d] */
  const void* step_w1;  /* [d][256] */
  const float* step_b1; /* [d] */
  const void* step_w2;  /* [d][d] */
  const float* step_b2; /* [d] */
  const void* const* mod_w;  /* host array of n_layers device pointers: [4d][d], output rows
                                alpha_msa | alpha_mlp | gamma_msa | gamma_mlp */
  const float* const* mod_b; /* host array of n_layers device pointers: [4d] */
} tlf_adaln_weights;

typedef struct tlf_weights {
  const void* tok_emb;      /* [V][d] storage dtype; also the LM head when lm_head is NULL */
  const void* pos_emb;      /* [max_pos][d] storage dtype */
  const float* router_w;    /* [R][d] float32 ([R][Hr], the output layer, for an MLP router) */
  const float* router_b;    /* [R] float32 */
  const void* lm_head;      /* [V][d] storage dtype, or NULL for a head tied to tok_emb */
  int32_t n_layers;         /* must equal config.n_layers */
  const tlf_layer_weights* layers; /* host array of n_layers entries (copied by tlf_init) */
  const void* router_w1;    /* MLP router hidden layer [Hr][d] storage dtype; NULL for a linear router */
  const float* router_b1;   /* [Hr] float32; NULL for a linear router */
  const tlf_adaln_weights* adaln; /* host pointer; required when config.adaln = 1, else NULL */
} tlf_weights;

typedef struct tlf_cache_stats_t {
  int64_t slots_per_loop[TLF_MAX_LOOPS];  /* sum over sequences of cache entries of loop i */
  int64_t pages_per_loop[TLF_MAX_LOOPS];  /* pages held by loop i's caches */
  int64_t depth_hist[TLF_MAX_LOOPS];      /* routed depth counts of every token seen (index m-1) */
  int64_t pages_used;                     /* pages in use (free pages: pages_total - pages_used) */
  int64_t pages_total;
  int64_t kv_bytes_resident;              /* pages_used * bytes per page */
  int64_t batch;                          /* sequences in the current batch */
  int64_t seq_len;                        /* tokens per sequence so far */
  /* Algorithmic bytes of the last decode step (exact, from the step's depths):
   * kv_read counts only valid entries (cache entries plus the step's own);
   * kv_write the appended k, v; weight bytes count the shared block once per
   * executed loop plus the LM head and router. */
  int64_t last_step_kv_read_bytes;
  int64_t last_step_kv_write_bytes;
  int64_t last_step_weight_bytes;
  int64_t last_step_loops_executed;       /* #{i : some token of the step has m >= i} */
  int64_t last_step_active_rows[TLF_MAX_LOOPS]; /* rows run at loop i in the last step: n_i = #{b : m_b >= i}
                                                   (dense_decode: the batch, up to the deepest loop) */
  /* Totals since profiling was last enabled (tlf_set_profiling): */
  int64_t decode_steps;                   /* decode steps enqueued */
  int64_t attn_launches;                  /* decode-attention launches timed */
  int64_t attn_algo_bytes;                /* their algorithmic bytes: valid K/V entries read, q read, o written */
  double attn_ms;                         /* their summed duration (HIP events on the context's stream) */
  int64_t kv_write_bytes_total;           /* bytes of appended k, v */
  int64_t loops_executed_total;           /* shared-block applications (each streams the block weights once) */
  double block_ms;                        /* summed duration of the loop-and-layer region of each step */
  int32_t device_error;                   /* sticky device-side status (TLF_OK if none) */
  int32_t reserved;
} tlf_cache_stats_t;

typedef struct tlf_ctx tlf_ctx;

/* Create a context (Section 3.3 inference state).
 *   cfg, w:       model description; w's device pointers are borrowed.
 *   d_workspace:  device memory for the KV page pool, page tables, positions,
 *                 activations and split-K partials; NULL to query the size.
 *   ws_bytes:     size of d_workspace.
 *   ws_needed:    out (may be NULL unless d_workspace is NULL): bytes needed.
 *   hip_stream:   hipStream_t on which all work is enqueued (NULL = default).
 *   out:          receives the context.
 * Returns TLF_E_NEED_WORKSPACE (with *ws_needed set) when d_workspace is NULL
 * or ws_bytes is too small, TLF_E_INVALID_ARG on a bad config or weight set,
 * TLF_E_UNSUPPORTED on a valid config outside the shapes and sizes listed in
 * tlf_config (head_dim, the multiples of d_model and d_ff, the TLF_MAX_* limits,
 * router_hidden, max_pos and the 32-bit offset limits). */
int tlf_init(const tlf_config* cfg, const tlf_weights* w, void* d_workspace, size_t ws_bytes,
             size_t* ws_needed, void* hip_stream, tlf_ctx** out);

/* Batched prefill (Section 3.3; gather-scatter of Eq. 6-7 with K/V written at
 * the gathered original positions, Eq. 11, and causal attention among the
 * gathered tokens of each loop).  Resets every cache and starts a new batch of
 * `batch` sequences of `seq_len` tokens each.
 * With TLF_PREFILL_APPEND the call is a later chunk of the current batch's
 * prompts (chunked prefill; it may also follow decode steps): its tokens take
 * positions [S, S + seq_len) after the S tokens each sequence holds, loop i
 * appends the chunk's tokens of depth >= i to cache (b, i) after its existing
 * entries, and each of them attends over every entry of that cache up to its
 * own position (Eq. 10).  Prefilling a prompt in chunks gives the results of
 * one call on the whole prompt.  Requires a batch (TLF_E_STATE otherwise),
 * the same `batch`, and S + seq_len <= max_pos.
 *   d_tokens: [batch][seq_len] int32 token ids in [0, V).
 *   d_logits: [batch][V] float32 logits of the call's last position, or
 *             [batch][seq_len][V] with TLF_PREFILL_ALL_LOGITS.
 *   d_depths: [batch][seq_len] int32 routed depths, or NULL.
 * Requires 1 <= batch <= max_batch, 1 <= seq_len <= max_pos.  Pages for an
 * appended chunk are taken on the device; running out sets the sticky
 * TLF_E_OUT_OF_PAGES reported by the next synchronizing call. */
int tlf_prefill(tlf_ctx* ctx, int32_t batch, int32_t seq_len, const int32_t* d_tokens,
                float* d_logits, int32_t* d_depths, uint32_t flags);

/* One decode step for every sequence of the current batch (Section 3.3,
 * Eq. 9-11): token b sits at position seq_len, is routed, runs its m_b loops
 * (appending k, v to each loop's cache and attending over it) and exits.
 *   d_tokens: [batch] int32 token ids (the caller picks them, e.g. d_next of
 *             the previous step for greedy decoding).
 *   d_logits: [batch][V] float32.
 *   d_next:   [batch] int32 greedy token (lowest id among maxima), or NULL.
 *   d_depths: [batch] int32 routed depth, or NULL.
 *   d_margin: [batch] float32 depth-decision margin (argmax: top1 - top2
 *             logit; cumprob: min(p^(m) - threshold, threshold - p^(m+1));
 *             fixed: +inf), or NULL.
 * Returns TLF_E_STATE before a prefill or once seq_len == max_pos. */
int tlf_decode_step(tlf_ctx* ctx, const int32_t* d_tokens, float* d_logits, int32_t* d_next,
                    int32_t* d_depths, float* d_margin);

/* Waits for the stream, then fills *out and, optionally, the logical cache
 * index: which original positions each recursion-wise cache (b, i) holds
 * (Eq. 8; each token of depth m appended to the caches of loops 1..m, Eq. 11).
 *   h_len: [batch][R] int32 host array of cache lengths n_{b,i}, or NULL.
 *   h_pos: host array receiving, for b = 0..batch-1 and i = 1..R in that order,
 *          the ascending original positions held by cache (b, i), or NULL.
 *   pos_cap: capacity of h_pos in int32 elements (TLF_E_INVALID_ARG if short).
 * Physical page ids are implementation-defined and are not reported.
 * Returns the sticky device error, if any, after filling *out. */
int tlf_cache_stats(tlf_ctx* ctx, tlf_cache_stats_t* out, int32_t* h_len, int32_t* h_pos,
                    size_t pos_cap);

/* Measurement switch (decode steps are then launched kernel by kernel, not
 * from the captured graph).
 *   TLF_PROFILE_ATTN:  a pair of HIP events on the context's stream around
 *                      every decode-attention launch (attn_ms) and around each
 *                      step's loop-and-layer region (block_ms);
 *   TLF_PROFILE_BLOCK: events around the loop-and-layer region only, so that
 *                      block_ms carries no event overhead from inside it;
 *   TLF_PROFILE_OFF:   no events.
 * Any mode other than OFF resets the totals reported by tlf_cache_stats
 * (decode_steps, attn_*, block_ms, ...).  It launches one small kernel and
 * does not wait for the stream.  TLF_E_INVALID_ARG for an unknown mode. */
#define TLF_PROFILE_OFF 0
#define TLF_PROFILE_ATTN 1
#define TLF_PROFILE_BLOCK 2
int tlf_set_profiling(tlf_ctx* ctx, int mode);

/* Measurement probe (no context): reads `bytes` of device memory at d_buf
 * once with the 16-byte non-temporal vector loads the decode attention
 * streams its cache with, one workgroup per TLF_PROBE_READ_GRAIN bytes, and
 * writes nothing except, with negligible probability, one word of d_sink.
 * The read rate it reaches is the practical ceiling for the decode
 * attention's streaming.  bytes must be a positive multiple of
 * TLF_PROBE_READ_GRAIN and d_buf 16-byte aligned (else TLF_E_INVALID_ARG);
 * enqueued on `d_stream` without waiting. */
#define TLF_PROBE_READ_GRAIN 32768
int tlf_probe_read(const void* d_buf, size_t bytes, unsigned int* d_sink, void* d_stream);

/* Releases the host context (waits for the stream first).  NULL is ignored. */
void tlf_destroy(tlf_ctx* ctx);

/* Static text for a status code. */
const char* tlf_status_str(int status);

/* ---------------------------------------------------------------------------
 * Training-side gather-scatter (Section 3.2, Eq. 6-7) and the router's
 * straight-through estimator (Appendix B).
 *
 * These calls need no context: they work on caller-owned device buffers and
 * enqueue on `stream` (a hipStream_t; NULL is the null stream) without
 * waiting for it.  The tokens of a batch of B sequences of T tokens are the
 * rows b*T + t of one [B*T, d] float32 tensor (row-major, 16-byte aligned,
 * d a multiple of 4).  Token t takes part in loop i exactly when its depth
 * m_t >= i.  Backward passes reuse the same calls: the gradient of the
 * gather is an in-place tlf_gs_scatter of the compact gradient into the row
 * gradients, and the gradient of the scatter is the incoming gradient itself
 * for the previous state plus its tlf_gs_gather for the block output.
 * Argument errors return TLF_E_INVALID_ARG before anything is enqueued; a
 * failed launch returns TLF_E_HIP.  Indices and slots are trusted: they must
 * be what tlf_gs_plan wrote for the same depths.
 * ------------------------------------------------------------------------- */

/* Active set of loop `loop` (Section 3.2 and Eq. 6).
 *   d_depth   [batch*seq_len] int32 depths m_t;
 *   d_index   [batch*seq_len] capacity; receives the active rows in
 *             increasing row order (each sequence's run contiguous and in
 *             causal order), *d_count of them;
 *   d_slot    [batch*seq_len] or NULL; receives each row's position in the
 *             compact tensor, -1 for a row not in the loop;
 *   d_offsets [batch+1] or NULL; receives where each sequence's run starts in
 *             the compact tensor, and the total last;
 *   d_count   [1]; the number of active rows.
 * One workgroup; batch*seq_len may be 0. */
int tlf_gs_plan(const int32_t* d_depth, int32_t batch, int32_t seq_len, int32_t loop, int32_t* d_index,
                int32_t* d_slot, int32_t* d_offsets, int32_t* d_count, void* d_stream);

/* The same plan (same outputs) from many workgroups: one launch counts the
 * active rows of each chunk of TLF_GS_PLAN_CHUNK_ROWS rows into the
 * workspace, a second places every chunk's rows after the counts before it
 * (Section 3.2 and Eq. 6).
 *   d_workspace  device scratch of at least tlf_gs_plan_ws_bytes(batch *
 *                seq_len) bytes, 4-byte aligned, borrowed for the call (it may
 *                be reused once the stream has passed this call); NULL when
 *                that size is 0.  Its contents need no initialisation.
 *   ws_bytes     its size.
 * Other arguments as tlf_gs_plan.  TLF_E_INVALID_ARG for a missing or short
 * workspace or batch * seq_len > TLF_GS_PLAN_MAX_ROWS. */
#define TLF_GS_PLAN_CHUNK_ROWS 2048
#define TLF_GS_PLAN_MAX_ROWS 8388608 /* 4096 chunks */
static inline size_t tlf_gs_plan_ws_bytes(int64_t rows) {
  return rows <= 0 ? 0 : (size_t)((rows + TLF_GS_PLAN_CHUNK_ROWS - 1) / TLF_GS_PLAN_CHUNK_ROWS) * 4u;
}
int tlf_gs_plan_ws(const int32_t* d_depth, int32_t batch, int32_t seq_len, int32_t loop, int32_t* d_index,
                   int32_t* d_slot, int32_t* d_offsets, int32_t* d_count, void* d_workspace, size_t ws_bytes,
                   void* d_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving or training loops, harnesses that forbid
 * hipMalloc): tlf_gs_plan_ws with its per-chunk counts in a fixed array of
 * the library's own device memory (16 KiB on each GPU that runs it, held
 * until the process ends) instead of a caller workspace.  Nothing is
 * allocated, and the array needs no clearing (every count read is written
 * by the same call first).  All calls on one GPU share the array: calls
 * that overlap on that GPU (other streams, other threads) race and must be
 * serialised by the caller.  The stream must belong to the current device.
 * Same arguments and outputs as tlf_gs_plan; TLF_E_INVALID_ARG when
 * batch * seq_len > TLF_GS_PLAN_NOALLOC_MAX_ROWS (checked before any device
 * work), TLF_E_HIP if the array's address cannot be obtained. */
#define TLF_GS_PLAN_NOALLOC_MAX_ROWS 8388608
int tlf_gs_plan_noalloc(const int32_t* d_depth, int32_t batch, int32_t seq_len, int32_t loop, int32_t* d_index,
                        int32_t* d_slot, int32_t* d_offsets, int32_t* d_count, void* d_stream);

/* Gather (Eq. 6): d_out[r] = d_h[d_index[r]] for r < min(*d_count, max_rows).
 * d_out holds max_rows x d floats; rows past the count are not written.  The
 * count stays on the device (no host synchronisation); max_rows bounds the
 * launch. */
int tlf_gs_gather(const float* d_h, const int32_t* d_index, const int32_t* d_count, int32_t max_rows,
                  int32_t d, float* d_out, void* d_stream);

/* Scatter (Eq. 7): d_h_out[r] = d_y[d_slot[r]] + d_h_prev[r] where
 * d_slot[r] >= 0, else d_h_prev[r]; `rows` rows of d floats.  d_h_out may be
 * d_h_prev (in place: rows not in the loop are then neither read nor written);
 * otherwise the two must not overlap, and d_y must overlap neither. */
int tlf_gs_scatter(const float* d_h_prev, const float* d_y, const int32_t* d_slot, int32_t rows, int32_t d,
                   float* d_h_out, void* d_stream);

/* Straight-through estimator of the depth (Appendix B), elementwise over n
 * tokens.  Forward value: d_value[t] = (float)d_depth[t].  Backward: with
 * sigma the logistic function, d_grad_score[t] = d_grad_value[t] *
 * sigma(d_score[t]) * (1 - sigma(d_score[t])).  Either output may be NULL
 * (then its inputs may be NULL too). */
int tlf_ste(const int32_t* d_depth, const float* d_score, const float* d_grad_value, int32_t n, float* d_value,
            float* d_grad_score, void* d_stream);

#ifdef __cplusplus
}
#endif

#endif /* TLF_H */
