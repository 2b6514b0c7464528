/*
 * m2r2.h — C ABI of the MI355X (gfx950) decode path of M2R2, "Mixture of
 * Multi-Rate Residuals" (arXiv 2502.02040).
 *
 * The library runs the autoregressive decode step of a pre-norm decoder-only
 * transformer that carries, in one forward pass, the slow residual stream h
 * (the base model, Eq. 1) and the accelerated residual stream p (Eq. 2):
 * every projection of a layer is streamed from HBM once and applied to both
 * rows; the fast row adds rank-r accelerator adapters (Sec. 2.2) and attends
 * to the slow row's KV cache plus its own key/value (the shared cache of
 * Sec. 2.2); at every layer the cosine between the fast state entering and
 * leaving the layer is computed as the exit signal (the directional shift of
 * Sec. 2.1), and at exit gates the fast row is either re-initialised from the
 * slow row (Fig. 3 caption) or, in exit mode, emits the token (Eq. 4).
 * On top of the step: self-speculative drafting from the fast stream and
 * parallel verification on the slow stream (Sec. 2.3.2), and, for
 * mixture-of-experts models (Sec. 2.3.3), expert prediction from the fast
 * stream driving ahead-of-time copies of expert weights from pinned host
 * memory into a per-layer HBM expert cache.
 *
 * Conventions (all entry points):
 *  - Memory: the caller owns every buffer.  Pointers named *_d are device
 *    pointers, *_h host pointers.  The library never allocates device memory:
 *    the workspace passed to m2r2_create holds a tile-packed copy of every
 *    projection matrix (so that each wave's 16-byte loads form 1 KB contiguous
 *    blocks that are exactly MFMA operands; read by calls with more than two
 *    rows) and all scratch.  Calls with one or two rows (a decode step of one
 *    sequence, a draft, a two-row chunk) stream the caller's row-major
 *    matrices directly, one output row per wave.  Every weight pointer
 *    (matrices, LM head, embedding, norm gains, adapter factors) is therefore
 *    borrowed for the lifetime of the context.  Activations, KV pages and
 *    outputs are borrowed for the duration of a call.
 *  - Layout: matrices are row-major [d_out][d_in] (the reduction dimension is
 *    contiguous).  Adapter factors are A [rank][d_in] and B [d_out][rank]; the
 *    adapter adds (x A^T) B^T to the projection of x.  Matrices and adapters
 *    are stored in the configured weight dtype; norm gains are always float32.
 *  - KV cache: paged, slow stream only.  K and V pages are
 *    [n_layers][num_blocks][n_heads][block_size][head_dim] in the configured
 *    KV dtype; block_table is [batch][max_blocks_per_seq] int32 (physical
 *    block of each logical block, shared by all layers).  Positions outside a
 *    sequence's block table are not read or written (a sticky device error
 *    bit is set instead).
 *  - Streams: every call that takes a hipStream_t only enqueues work on it
 *    (no host synchronisation), so a sequence of calls can be captured into a
 *    HIP graph -- except the decode step of a mixture-of-experts model, which
 *    waits, layer by layer, for the router's choice before it can place the
 *    expert copies (see m2r2_decode_step).  One context must not be used on
 *    two streams at once.
 *  - Errors: no exception or abort crosses the ABI.  Arguments are checked
 *    before anything is enqueued; on failure the call returns a negative
 *    m2r2_status and m2r2_last_error() (thread-local) describes it.  A launch
 *    failure reported by HIP returns M2R2_E_HIP.
 */
#ifndef M2R2_H_
#define M2R2_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define M2R2_API __attribute__((visibility("default")))

typedef enum {
  M2R2_OK = 0,
  M2R2_E_INVALID = -1,      /* NULL pointer, bad enum, bad pointer alignment */
  M2R2_E_SHAPE = -2,        /* a size is out of the supported range */
  M2R2_E_DTYPE = -3,        /* unsupported dtype combination */
  M2R2_E_NOMEM = -4,        /* workspace smaller than m2r2_workspace_size() */
  M2R2_E_HIP = -5,          /* a HIP runtime call failed */
  M2R2_E_STATE = -6,        /* call not valid in the context's current state */
  M2R2_E_UNSUPPORTED = -7   /* valid request the library does not implement */
} m2r2_status;

typedef enum { M2R2_F32 = 0, M2R2_BF16 = 1 } m2r2_dtype;

/* Exit handling at gates (Fig. 3 caption; Eq. 4).
 *  OFF:     no gate is evaluated; p is never re-initialised.
 *  OBSERVE: at each gate b the signal of layer b-1 is compared with tau; the
 *           first gate with signal >= tau is recorded as the exit boundary,
 *           and p <- h at every gate (the full-depth slow token is emitted).
 *  EXIT:    as OBSERVE, but a sequence whose signal reaches tau at a gate
 *           stops there: its token comes from the final norm and LM head on
 *           p at the gate, and the KV entries of its remaining layers are
 *           projected from the slow state h at the gate. */
typedef enum { M2R2_EXIT_OFF = 0, M2R2_EXIT_OBSERVE = 1, M2R2_EXIT_EXIT = 2 } m2r2_exit_mode;

typedef struct {
  int32_t n_layers, d_model, n_heads, head_dim, ffn, vocab, rank;
  int32_t wdtype;           /* m2r2_dtype of matrices, embeddings, adapters */
  int32_t kvdtype;          /* m2r2_dtype of the KV pages */
  float rms_eps;            /* RMSNorm epsilon */
  float rope_theta;         /* rotate-half RoPE base */
  /* Mixture of experts (Sec. 2.3.3); n_experts = 0 for a dense model.  Every
   * layer then has n_experts SwiGLU experts of width expert_ffn, top_k of
   * which are chosen per token, and the HBM cache holds expert_slots experts
   * per layer (top_k <= expert_slots <= n_experts; = n_experts keeps every
   * expert resident). */
  int32_t n_experts, top_k, expert_ffn, expert_slots;
  /* FLOPs-optimised accelerated stream (Sec. 2.5), dense models only; all
   * zero selects the memory-bound form above.
   *  fast_heads:        the fast row keeps heads 0 .. fast_heads-1 (0: all);
   *                     the attention output of the other heads is zero for it.
   *  fast_topk:         fast head j attends to the fast_topk cached positions
   *                     with the largest scores of the slow row's head j at the
   *                     same layer (ties to the lower position; every cached
   *                     position when there are no more), plus its own
   *                     key/value (0: every cached position).
   *  fast_mlp_adapter:  1: the fast row's MLP is the rank-r adapter alone,
   *                     (m A_m^T) B_m^T with m = rms(x) * mlp_norm, from the
   *                     layer's A_m/B_m (the gate/up/down adapters are unused).
   *  head_rank:         a token the fast row emits (an exit in EXIT mode) comes
   *                     from the final norm and the rank-head_rank head
   *                     head_a [head_rank][d], head_b [vocab][head_rank] of
   *                     m2r2_weights (0: the LM head).
   * Supported for one sequence (batch 1) on shapes whose rows are whole
   * multiples of 1 KB (the row-per-wave kernels); m2r2_draft and the exit
   * router are refused with M2R2_E_UNSUPPORTED (a fast-only pass has no
   * slow-row scores to select positions with). */
  int32_t fast_heads, fast_topk, fast_mlp_adapter, head_rank;
} m2r2_config;

/* Per-layer device pointers.  Any adapter pointer may be NULL (adapter
 * absent: that projection of the fast row equals the slow one). */
typedef struct {
  const float* attn_norm;   /* [d] */
  const void* wq;           /* [H*hd][d] */
  const void* wk;           /* [H*hd][d] */
  const void* wv;           /* [H*hd][d] */
  const void* wo;           /* [d][H*hd] */
  const float* mlp_norm;    /* [d] */
  const void* wg;           /* [ffn][d]  gate */
  const void* wu;           /* [ffn][d]  up */
  const void* wd;           /* [d][ffn]  down */
  /* accelerator adapters, index 0..6 = q, k, v, o, gate, up, down */
  const void* A[7];
  const void* B[7];
  /* mixture-of-experts layers: wg, wu, wd and A/B[4..6] are NULL; the router
   * and the fast row's MLP, which is the rank-r adapter alone (Sec. 2.3.3):
   * MLP_fast(x) = (m A_m^T) B_m^T with m = rms(x) * mlp_norm.  A dense model
   * with fast_mlp_adapter set takes its fast MLP from A_m/B_m too (Sec. 2.5). */
  const void* router;       /* [n_experts][d] */
  const void* A_m;          /* [rank][d], may be NULL with B_m (fast MLP absent) */
  const void* B_m;          /* [d][rank] */
} m2r2_layer_weights;

typedef struct {
  const void* embed;                 /* [vocab][d] */
  const float* final_norm;           /* [d] */
  const void* lm_head;               /* [vocab][d] */
  const m2r2_layer_weights* layers;  /* host array of n_layers entries, copied by m2r2_create */
  /* mixture of experts: pinned host memory (hipHostMalloc) holding every
   * expert of every layer, expert e of layer l at byte offset
   * (l * n_experts + e) * m2r2_expert_bytes(), each filled by
   * m2r2_pack_expert.  Borrowed for the lifetime of the context. */
  const void* experts_h;
  /* low-rank head of the FLOPs-optimised fast stream (config head_rank > 0):
   * head_a [head_rank][d], head_b [vocab][head_rank]; NULL otherwise */
  const void* head_a;
  const void* head_b;
} m2r2_weights;

typedef struct {
  void* k_pages;                 /* device, see layout above */
  void* v_pages;
  const int32_t* block_table_d;  /* [batch][max_blocks_per_seq] */
  int32_t* seq_lens_d;           /* [batch]: written with the number of valid cache positions */
  int32_t num_blocks, block_size, max_blocks_per_seq;
} m2r2_kv;

typedef struct {
  const int32_t* gates_h;   /* host array of gate boundaries b in [1, n_layers-1] */
  int32_t n_gates;
  float tau;                /* exit iff signal >= tau */
  int32_t mode;             /* m2r2_exit_mode */
} m2r2_exit;

typedef struct {
  int32_t* next_token_d;    /* [batch] required: greedy token (lowest id on ties) */
  int32_t* exit_boundary_d; /* [batch] optional: first gate whose signal >= tau, n_layers if none */
  float* signal_d;          /* [batch][n_layers] optional: cos(p entering, p leaving) per layer; with
                               the exit router set (m2r2_set_arla), its score at the layer before
                               each gate */
  float* logits_d;          /* [batch][vocab] optional: logits of the emitted row */
  float* h_out_d;           /* [batch][d] optional: slow row fed to the head (gate state on exit) */
  float* p_out_d;           /* [batch][d] optional: fast row at the end of the step */
  int32_t advance;          /* nonzero: positions_d[b] += 1 at the end of the step */
  /* mixture of experts, optional: [batch][n_layers][top_k] experts chosen by
   * the slow row's router (descending probability, lowest id on ties; -1 for
   * layers not run after an exit), and experts predicted for layer l: from
   * the fast row after layer (l-2)/2 (Sec. 2.3.3), or, under the
   * M2R2_MOE_PREVIOUS_LAYER policy, by layer l's router from the slow row
   * entering layer l-1's MLP (-1 where no prediction) */
  int32_t* slow_experts_d;
  int32_t* pred_experts_d;
} m2r2_step_out;

typedef struct m2r2_ctx m2r2_ctx;

/* Workspace bytes a context needs (packed weights plus scratch) for up to
 * max_batch sequences, chunks of up to max_chunk rows (verification/prefill)
 * and max_ctx cache positions per sequence.  max_batch <= 8, max_chunk <= 16.
 * For a mixture-of-experts model it includes the HBM expert cache,
 * n_layers * expert_slots * m2r2_expert_bytes() bytes, and the packed routers;
 * such a model takes max_batch = 1. */
M2R2_API m2r2_status m2r2_workspace_size(const m2r2_config* cfg, int32_t max_batch, int32_t max_chunk,
                                         int32_t max_ctx, size_t* bytes_out);

/* Create a context.  `workspace` is device memory of at least the size above,
 * 256-byte aligned, owned by the caller and used exclusively by this context;
 * it is initialised here, including packing the projection matrices
 * (synchronously, on the null stream) and, for a mixture-of-experts model,
 * the warm start of the expert cache (experts 0..expert_slots-1 of every
 * layer copied from the host store).  Weight pointers must be 16-byte
 * aligned.  Requirements:
 * d_model, H*head_dim and ffn multiples of 32 (bf16) or 16 (f32); head_dim
 * even and <= 128; rank <= 32. */
M2R2_API m2r2_status m2r2_create(const m2r2_config* cfg, const m2r2_weights* w, int32_t max_batch,
                                 int32_t max_chunk, int32_t max_ctx, void* workspace, size_t ws_bytes,
                                 m2r2_ctx** out);
M2R2_API void m2r2_destroy(m2r2_ctx* ctx);

/* One dual-stream decode step (Eq. 1 and Eq. 2 with the shared KV cache,
 * Sec. 2.2) for `batch` sequences.  tokens_d[b] is the input token of
 * sequence b and positions_d[b] its position t; the cache must hold t valid
 * positions.  The slow row's key/value at t are written to the cache and
 * seq_lens_d[b] is set to t+1.  `dual` = 0 runs the slow row alone (plain
 * decoding on the same kernels; exit settings are then ignored).
 * tokens_d may alias out->next_token_d.
 *
 * Mixture-of-experts models (batch 1): in every layer the slow row's router
 * picks top_k experts (softmax over all experts, unrenormalised weights) and
 * the fast row, whose MLP is its adapter alone, predicts the experts of
 * layers 2i+2 and 2i+3 from its state after layer i, each with that layer's
 * norm gain and router (Sec. 2.3.3).  The call then waits until the routing
 * of the layer is known on the host, makes every chosen expert resident in
 * that layer's HBM cache (a miss is copied from the host store on the
 * library's on-demand copy stream), makes `stream` wait for any copy still in
 * flight, and runs the experts from their cache slots.  Under the
 * M2R2_MOE_AHEAD_OF_TIME policy the predicted experts are then copied on the
 * library's prefetch stream; the comparison policies preload their own
 * picks for the next layer on that stream instead (m2r2_moe_policy).  Cache
 * replacement is least-recently-used, with the experts needed now and those
 * predicted for the layer protected from eviction (M2R2_MOE_FIXED: no
 * replacement).  The call returns once the last layer's experts are
 * enqueued.  With as many slots as experts under M2R2_MOE_ON_DEMAND (every
 * expert resident, nothing to decide) the call waits for no routing: the
 * experts are taken from their slots on the device and the whole token is
 * enqueued at once. */
M2R2_API m2r2_status m2r2_decode_step(m2r2_ctx* ctx, int32_t batch, int32_t dual, const int32_t* tokens_d,
                                      int32_t* positions_d, const m2r2_kv* kv, const m2r2_exit* ex,
                                      const m2r2_step_out* out, hipStream_t stream);

/* The decode step of m2r2_decode_step, for callers that cannot allocate
 * device memory or whose memory is fixed before they start (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation).
 * Same arguments, semantics and results; the difference is where the
 * step's per-call scratch lives (residual rows, row statistics, attention
 * and arg-max partials, arrival counters): in a static device array of
 * 32 MiB inside the library, one per GPU, instead of the context's
 * workspace.  The call allocates nothing and clears the scratch's counters
 * itself (with a kernel on `stream`).  Limits: dense models only
 * (M2R2_E_UNSUPPORTED for a mixture-of-experts context); the context's
 * scratch, which grows with max_batch and max_ctx, must fit the 32 MiB
 * (M2R2_E_SHAPE otherwise, e.g. a Phi-3-shaped context with max_batch 1 and
 * max_ctx 1536 needs about 9 MiB); the device that was current at
 * m2r2_create must be current (M2R2_E_STATE).  All such calls on one GPU
 * share the array, which keeps the last call's contents: calls that overlap
 * on one GPU (two streams, or two contexts at once) race. */
M2R2_API m2r2_status m2r2_decode_step_noalloc(m2r2_ctx* ctx, int32_t batch, int32_t dual, const int32_t* tokens_d,
                                              int32_t* positions_d, const m2r2_kv* kv, const m2r2_exit* ex,
                                              const m2r2_step_out* out, hipStream_t stream);

/* Accelerated-residual latent-attention exit router (Sec. 2.3.1, ARLA; Fig.
 * 4a), replacing the cosine signal at the gates of later dual decode steps
 * with the exit settings on.  Weights are borrowed device pointers, read
 * during the steps; block b of each array belongs to boundary b (1 <= b <
 * n_layers; block 0 is not read):
 *   wq, wk, wv: [n_layers][64][d_model] in the weight dtype, row-major;
 *   w_out: [n_layers][64] float; b_out: [n_layers] float.
 * At a gate b the fast states after the layers since the previous gate (or
 * layer 0) through b-1 are scaled to unit RMS (no gain, the model's epsilon),
 * projected to latent keys and values with boundary b's wk, wv; the state
 * after layer b-1 also gives the query (wq).  Single-query softmax attention
 * with scale 1/8 pools the values; the score is sigmoid(w_out . pooled +
 * b_out), and the gate fires iff score >= tau.  A NULL `w` switches the
 * router off.  Dense models, batch 1 (a decode step with batch > 1 and gates
 * on fails with M2R2_E_UNSUPPORTED while the router is set).  Host-only. */
typedef struct {
  const void* wq;
  const void* wk;
  const void* wv;
  const float* w_out;
  const float* b_out;
} m2r2_arla;

M2R2_API m2r2_status m2r2_set_arla(m2r2_ctx* ctx, const m2r2_arla* w);

/* Self-speculative draft (Sec. 2.3.2): gamma greedy tokens from the fast row
 * alone, run through layers 0..exit_layer-1 (a fast stream at rate
 * n_layers/exit_layer), then the final norm and LM head.  Batch 1.  The first
 * draft consumes last_token_d[0] at position positions_d[0] = t; draft j is at
 * position t+j.  The fast row's key/value at those positions are written to
 * cache positions t..t+gamma-1 of layers < exit_layer, where later drafts read
 * them; m2r2_verify overwrites them.  Writes drafts_d[0..gamma).  Dense
 * models only (M2R2_E_UNSUPPORTED for a mixture-of-experts model). */
M2R2_API m2r2_status m2r2_draft(m2r2_ctx* ctx, const int32_t* last_token_d, const int32_t* positions_d,
                                int32_t exit_layer, int32_t gamma, const m2r2_kv* kv, int32_t* drafts_d,
                                hipStream_t stream);

/* Parallel verification on the slow stream (Sec. 2.3.2) of a chunk of n
 * tokens chunk_d[0..n) at positions t..t+n-1 (t = positions_d[0]), causal,
 * batch 1.  Writes the cache at those positions and targets_d[i] = greedy
 * token after chunk row i.  If n_accepted_d is not NULL, the chunk is
 * [last, d_1..d_{n-1}] and n_accepted_d[0] = largest j with
 * d_1..d_j == targets_d[0..j); seq_lens_d[0] = t + j + 1; if
 * bonus_token_d is not NULL it receives targets_d[j]; positions_d[0] is
 * advanced by j + 1.  If n_accepted_d is NULL (prefill) every row is kept:
 * seq_lens_d[0] = t + n and positions_d[0] is advanced by n.  1 <= n <= max_chunk.
 * Dense models only: a mixture-of-experts model is prefilled with slow-only
 * decode steps (dual = 0). */
M2R2_API m2r2_status m2r2_verify(m2r2_ctx* ctx, const int32_t* chunk_d, int32_t n, int32_t* positions_d,
                                 const m2r2_kv* kv, int32_t* targets_d, int32_t* n_accepted_d,
                                 int32_t* bonus_token_d, hipStream_t stream);

/* ---- mixture of experts (Sec. 2.3.3) ----------------------------------- */

/* Expert placement strategies: M2R2's own and the four it is compared with
 * (Sec. 3.3).  Every policy works in the same `slots` slots per layer. */
typedef enum {
  M2R2_MOE_ON_DEMAND = 0,      /* least-recently-used cache, misses loaded when routed */
  M2R2_MOE_AHEAD_OF_TIME = 1,  /* as above, plus copies of the fast stream's predictions for
                                  layers 2i+2 and 2i+3, issued after layer i (dual steps) */
  M2R2_MOE_FIXED = 2,          /* experts 0..slots-top_k-1 resident for good; every other chosen
                                  expert is copied, at every use, into one of top_k staging slots */
  M2R2_MOE_RANDOM_PRELOAD = 3, /* least-recently-used, plus a preload of top_k random experts
                                  (a caller's table) for layer i+1 after layer i */
  M2R2_MOE_PREVIOUS_LAYER = 4  /* least-recently-used, plus a preload of the top_k experts that
                                  layer i+1's router picks from the slow row entering layer i's
                                  MLP, issued after layer i */
} m2r2_moe_policy;

typedef struct {
  int64_t hits, misses;             /* chosen experts resident (or in flight) / not, when routed */
  int64_t prefetch_issued, prefetch_used, prefetch_wasted;   /* wasted: evicted before any use */
  int64_t loads;                    /* host-to-device expert copies */
  int64_t pred_correct, pred_total; /* |P ∩ S| and |P| over predicted layers (preloading policies) */
  int64_t h2d_bytes;                /* bytes copied host to device */
  int64_t copy_waits;               /* times the compute stream was made to wait for a copy */
  int64_t host_wait_ns;             /* host time spent waiting for routing results */
  int64_t copies_failed;            /* copies that could not be enqueued or completed with an error: the
                                       slot is invalidated and the expert loaded on demand when used */
  int64_t layer_misses[128];        /* misses per layer */
} m2r2_moe_counters;

/* Bytes of one packed expert: gate [F_e][d], up [F_e][d] and down [d][F_e],
 * each in the tile-packed layout the expert kernels read.  Requires
 * expert_ffn a multiple of 32 (bf16) or 16 (f32). */
M2R2_API m2r2_status m2r2_expert_bytes(const m2r2_config* cfg, size_t* bytes_out);

/* Host-only: pack one expert's row-major gate, up ([F_e][d]) and down
 * ([d][F_e]) matrices, in the weight dtype, into dst_h (m2r2_expert_bytes
 * bytes of host memory).  No device work. */
M2R2_API m2r2_status m2r2_pack_expert(const m2r2_config* cfg, const void* wg_h, const void* wu_h, const void* wd_h,
                                      void* dst_h);

/* Select the cache policy (m2r2_moe_policy) for later decode steps (default:
 * ahead of time) and restore the warm start as m2r2_moe_reset does
 * (synchronous).  M2R2_E_INVALID for an unknown policy. */
M2R2_API m2r2_status m2r2_moe_set_policy(m2r2_ctx* ctx, int32_t policy);

/* Random draws of the M2R2_MOE_RANDOM_PRELOAD policy: ids_h is
 * [n_tokens][n_layers][top_k] expert ids in [0, n_experts) (-1: no preload),
 * copied into the context.  The decode step that is the t-th since the last
 * reset (counting from 0) preloads row (t mod n_tokens, i+1) for layer i+1
 * after layer i.  Host-only; M2R2_E_SHAPE for ids out of range or
 * n_tokens < 1.  A decode step under that policy without a table fails with
 * M2R2_E_STATE. */
M2R2_API m2r2_status m2r2_moe_set_preload_table(m2r2_ctx* ctx, const int32_t* ids_h, int32_t n_tokens);

/* Make experts ids_h[0..n) of `layer` resident or in flight (Sec. 2.3.3,
 * Appendix B): a resident expert is marked as just used; a missing one
 * replaces the least recently used expert not in ids_h and is copied from the
 * host store on copy_stream (priority != 0: on the library's on-demand copy
 * stream; NULL copy_stream: the library's prefetch stream).  Later decode
 * steps wait for the copy before they use the slot.  Counts as prefetches.
 * A copy that cannot be enqueued invalidates its slot (the expert is loaded
 * on demand when used; counted in copies_failed) instead of failing the call.
 * M2R2_E_STATE under the M2R2_MOE_FIXED policy (its slots never change). */
M2R2_API m2r2_status m2r2_prefetch_experts(m2r2_ctx* ctx, int32_t layer, const int32_t* ids_h, int32_t n,
                                           int32_t priority, hipStream_t copy_stream);

/* Restore the warm start -- experts 0..slots-1 of every layer resident, expert
 * 0 least recently used -- and zero the statistics.  Synchronous. */
M2R2_API m2r2_status m2r2_moe_reset(m2r2_ctx* ctx);

/* Counters since the last reset.  With as many slots as experts under the
 * on-demand policy, tokens are enqueued whole (no host wait for routing) and
 * their hits are counted on the device: the call then waits for the device. */
M2R2_API m2r2_status m2r2_moe_stats(m2r2_ctx* ctx, m2r2_moe_counters* out);

/* Host-only replay of a cache policy on a routing trace, with no copies:
 * slow_h[t][l][top_k] experts chosen at token t, layer l; pred_h (may be
 * NULL) the same shape, predictions (-1 where none).  `policy` is an
 * m2r2_moe_policy: ON_DEMAND ignores pred_h; AHEAD_OF_TIME applies the
 * predictions for layers 2i+2, 2i+3 after layer i; RANDOM_PRELOAD and
 * PREVIOUS_LAYER apply those for layer i+1 after layer i; FIXED ignores
 * pred_h.  Fills the counters of `out` (h2d_bytes, copy_waits and
 * host_wait_ns are 0). */
M2R2_API m2r2_status m2r2_expert_cache_replay(int32_t n_layers, int32_t n_experts, int32_t top_k, int32_t slots,
                                              int32_t n_tokens, const int32_t* slow_h, const int32_t* pred_h,
                                              int32_t policy, m2r2_moe_counters* out);

/* Sticky device error bits set by kernels since the context was created
 * (1: token id out of range, 2: cache position outside the block table,
 * 4: context longer than the workspace was sized for, 8: a position beyond
 * the RoPE table, i.e. at or past max_ctx); waits for `stream`. */
M2R2_API m2r2_status m2r2_device_errors(m2r2_ctx* ctx, hipStream_t stream, int32_t* bits);

/* Report the asynchronous errors of the work enqueued so far: waits for
 * `stream`, then returns M2R2_E_HIP if the stream or an earlier launch
 * failed (the HIP error in m2r2_last_error()), M2R2_E_STATE if a kernel set
 * one of the sticky device error bits above (the bits in m2r2_last_error()),
 * else M2R2_OK.  Entry points check their arguments before they enqueue
 * anything and report launch failures at once; a fault or a device-side
 * range violation inside a kernel can only be seen here (or by the next
 * call's launch).  The error bits stay set once seen. */
M2R2_API m2r2_status m2r2_sync_check(m2r2_ctx* ctx, hipStream_t stream);

/* Description of the last error on this thread ("" if none). */
M2R2_API const char* m2r2_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* M2R2_H_ */
