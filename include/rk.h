/*
 * rk.h -- C ABI of the RippleKV sensitivity-profile library for MI355X (gfx950).
 *
 * The library computes the perturbation-propagation sensitivity profile of a
 * decoder-only Transformer and maps it to per-layer KV-cache budgets
 * (RippleKV, Algorithm 1; Sections 4.1-4.4):
 *
 *   for every calibration sequence x_i and every compressible layer l:
 *     perturb layer l's Value cache only, v~ = v + alpha * ||v||_2 * eps
 *       (Eq. value-perturbation; eps ~ N(0, I) per sequence, layer, KV head and
 *       position; Keys and all other layers untouched),
 *     resume the forward from the clean input of layer l (layers below l are
 *       never recomputed) through the LM head,
 *     d_{i,l} = mean over the window of KL(P_clean || Q_perturbed)
 *       (Eq. sample-response);
 *   s_l = (1/N) sum_i d_{i,l}                                (Eq. layer-sensitivity)
 *   b   = round(B/|A| * ClipNormalize(r ** minmax(s), gamma)) (Eqs. 9-12)
 *
 * The model is the Llama-style decoder of Section 4.1: token embedding, L
 * pre-norm blocks (RMSNorm, fused q|k|v projection, rotate-half rotary embedding
 * on Q and K, grouped-query causal attention, output projection, RMSNorm, SwiGLU
 * feed-forward), a final RMSNorm and an untied LM head.
 *
 * Conventions for every entry point:
 *  - Ownership: the library never allocates, frees or retains caller memory.
 *    All device buffers (weights, tokens, outputs, clean state, workspace) are
 *    allocated by the caller; rk_model keeps pointers only.
 *  - Streams: GPU entry points enqueue work on `stream` (a hipStream_t passed as
 *    void*, NULL = the null stream) and return without synchronising.  Outputs
 *    are valid once the stream reaches that point.
 *  - Errors: every argument is validated before the first launch; on error the
 *    function returns a negative rk_status, writes no output and records a
 *    message for rk_last_error().  A HIP launch failure returns RK_ERR_HIP.
 *  - Determinism: for the same inputs, seed and shapes the results are bitwise
 *    repeatable (fixed-order reductions, no floating-point atomics).  With
 *    alpha = 0 every KL is exactly 0.
 *  - Layouts: row-major; weight matrices in [out_features, in_features] layout;
 *    bf16 buffers hold raw bf16 bit patterns (uint16).
 *  - Thread safety: calls that share a workspace or clean-state buffer must be
 *    ordered by the caller (same stream or explicit synchronisation).
 */
#ifndef RK_H
#define RK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RK_OK = 0,
  RK_ERR_ARG = -1,          /* null pointer, out-of-range scalar, bad layer index     */
  RK_ERR_SHAPE = -2,        /* inconsistent sizes (offsets, rows, batch too large)   */
  RK_ERR_WORKSPACE = -3,    /* workspace or clean-state buffer smaller than required */
  RK_ERR_HIP = -4,          /* a HIP call or kernel launch failed                    */
  RK_ERR_UNSUPPORTED = -5,  /* model shape outside what the kernels implement        */
  RK_ERR_STATE = -6         /* (RK_FLAG_CHECK_STATE) the clean or window state was
                               produced for another model, batch or window start   */
} rk_status;

typedef enum { RK_F32 = 0, RK_BF16 = 1 } rk_dtype;

typedef enum {
  RK_ROUND_LARGEST_REMAINDER = 0,  /* keeps sum(b) = B exactly (default reading)  */
  RK_ROUND_NEAREST_EVEN = 1        /* literal per-layer round() of Eq. layer-budget */
} rk_rounding;

/* Flags of rk_perturb_params.flags */
#define RK_FLAG_FULL_RECOMPUTE 0x1u  /* recompute layers below l instead of resuming
                                        (verification of prefix reuse)              */
#define RK_FLAG_UNFUSED_KL     0x2u  /* materialise fp32 logits and run the separate
                                        log-softmax + KL kernel instead of the fused
                                        LM-head + KL kernel                          */
#define RK_FLAG_GRAPH          0x8u  /* rk_sensitivity_profile only: the first call
                                        runs eagerly and records its launch sequence
                                        in a HIP graph; later calls replay the graph
                                        while every argument (device pointers, sizes,
                                        host arrays) stays the same;
                                        one graph per process, replaced when the
                                        arguments change (graphed calls from
                                        several threads are serialised while
                                        they record or launch).  Saves the per-launch
                                        overhead of the ~10^3-10^4 kernels of a
                                        profile.  With kernel timing on, each graphed
                                        call needs its own rk_timing_begin.         */
#define RK_FLAG_CACHED_WINDOW  0x4u  /* the literal reading of Section 4.3: each
                                        sequence is a cached prefix [0, P) and an
                                        evaluation window [P, T_i), P = window_start;
                                        only layer l's cached prefix Values are
                                        perturbed, every other cache stays frozen,
                                        and only the window is recomputed (see
                                        rk_window_reference).  bf16 models only.     */
#define RK_FLAG_LOCAL_SIGNAL   0x10u /* the layer-local signal of the "w/o DS"
                                        ablation (Section 5, Table ablation): the
                                        same perturbation and averaging, but d_{i,l}
                                        is the window mean of the response of block
                                        l itself, r_t = ||h~_{l+1,t} - h_{l+1,t}||^2
                                        / ||h_{l+1,t}||^2 (its output with and
                                        without the perturbed Values; 0 for a zero
                                        clean row), in place of the KL of the final
                                        distributions.  No layer after l and no LM
                                        head is evaluated.  Not combinable with
                                        RK_FLAG_UNFUSED_KL.                          */
#define RK_FLAG_CHECK_STATE    0x20u /* rk_profile_layer only (ignored elsewhere):
                                        before launching anything, compare the
                                        record that rk_reference_forward /
                                        rk_window_reference left in the state
                                        (the model's config and weight pointers,
                                        the batch's sequence lengths and a digest
                                        of its tokens, the window start) with the
                                        call's, and return RK_ERR_STATE if they
                                        differ.  The record is read back to the
                                        host, so the call synchronises the stream
                                        (a debugging aid; not for graph capture). */

/* Most sequences one batch (one call's rows) may hold. */
#define RK_MAX_BATCH_SEQS 64

/* Model shape (Section 4.1).  dtype selects the storage of weights and GEMM
 * operands: RK_BF16 = bf16 operands, fp32 accumulation, fp32 residual stream;
 * RK_F32 = fp32 throughout.
 * Supported: head_dim in {64, 128} for RK_BF16 and {32, 64, 128} for RK_F32; n_heads a multiple of n_kv_heads; d_model, n_heads*head_dim, the q|k|v
 * width and vocab multiples of 128; d_ff a multiple of 64.                      */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab;
  float rope_theta;   /* rotary base theta                  */
  float rms_eps;      /* RMSNorm epsilon                    */
  rk_dtype dtype;
} rk_model_config;

/* Device pointers to the weights (caller-owned).  Matrices are in the config's
 * dtype; the norm gains are always fp32.  The per-layer members are HOST arrays
 * of n_layers device pointers (copied by rk_model_create).                     */
typedef struct {
  const void *tok_emb;                 /* [vocab, d_model]                               */
  const void *const *w_qkv;            /* [L] -> [(H + 2*Hkv)*head_dim, d_model]: q rows,
                                          then k rows, then v rows                       */
  const void *const *w_o;              /* [L] -> [d_model, H*head_dim]                   */
  const void *const *w_gate_up;        /* [L] -> [2*d_ff, d_model]: gate rows, then up   */
  const void *const *w_down;           /* [L] -> [d_model, d_ff]                         */
  const float *const *attn_norm;       /* [L] -> [d_model] fp32                          */
  const float *const *mlp_norm;        /* [L] -> [d_model] fp32                          */
  const float *final_norm;             /* [d_model] fp32                                 */
  const void *lm_head;                 /* [vocab, d_model] (untied)                      */
} rk_model_weights;

typedef struct rk_model rk_model;      /* opaque, host-side */

/* A batch of calibration sequences processed together (their rows concatenated).
 * tokens: DEVICE int32 [offsets[n_seqs]]; offsets: HOST int64 [n_seqs + 1],
 * offsets[0] = 0, non-decreasing; seq_index0: index in the calibration set of the
 * batch's first sequence (sequence k of the batch has index seq_index0 + k, which
 * keys its noise).  1 <= n_seqs <= RK_MAX_BATCH_SEQS.  On a bf16 model every
 * sequence must satisfy T * (H + 2*Hkv) * head_dim * 2 < 2^31 bytes (the
 * attention kernel's 32-bit buffer offsets; at most 174762 tokens at the
 * Llama-3-8B shape); a longer one is RK_ERR_SHAPE before any device work.      */
typedef struct {
  const int32_t *tokens;
  const int64_t *offsets;
  int32_t n_seqs;
  int32_t seq_index0;
} rk_batch;

/* Perturbation and window parameters (Section 4.3).  Positions u of sequence i
 * with protect_head <= u < T_i - protect_tail are perturbed (the paper excludes
 * positions the base compressor protects); the evaluation window is
 * W_i = [window_start, T_i).  seed keys the Philox4x32-10 noise; the same noise
 * serves every alpha.  With RK_FLAG_CACHED_WINDOW the perturbed positions are
 * the cached prefix positions protect_head <= u < window_start - protect_tail
 * and every sequence must be longer than window_start > 0.                    */
typedef struct {
  uint64_t seed;
  int32_t window_start;
  int32_t protect_head;
  int32_t protect_tail;
  uint32_t flags;              /* RK_FLAG_* */
} rk_perturb_params;

/* ---------------------------------------------------------------- model handle */

/* Validates the config and the weight pointers and returns a handle that stores
 * them (no device work, no device memory).  RK_ERR_UNSUPPORTED for shapes outside
 * the kernels' envelope (see rk_model_config).                                 */
rk_status rk_model_create(const rk_model_config *cfg, const rk_model_weights *w, rk_model **out);
void rk_model_destroy(rk_model *m);

/* ---------------------------------------------------------------- sizes */

/* Bytes of the clean state of a batch of n_rows rows (Algorithm 1,
 * ReferencePredict): the fp32 input h_l of every block l ([L, n_rows, d_model]),
 * the final normalised hidden state ([n_rows, d_model] in the model dtype), the
 * clean log-sum-exp and a 256-byte record of the model and batch that produced
 * it (see RK_FLAG_CHECK_STATE).                                                 */
size_t rk_clean_state_size(const rk_model *m, int64_t n_rows);

/* Bytes of the state of the cached-window mode for a batch of at most n_rows
 * rows (rk_window_reference): the KV cache of every layer for the prefix rows
 * ([L, prefix rows, 2 * n_kv_heads * head_dim] bf16, K then V), and for the
 * window rows the fp32 input of every block, the final normalised hidden state
 * and the clean log-sum-exp of the LM head, and the 256-byte record of the
 * model, batch and window start that produced it.  0 for invalid arguments.    */
size_t rk_window_state_size(const rk_model *m, int64_t n_rows);

/* Flag of rk_workspace_size: the workspace also holds one clean state
 * (rk_sensitivity_profile keeps its clean state there; with
 * RK_FLAG_CACHED_WINDOW also set, a cached-window state).                      */
#define RK_WS_CLEAN_STATE 0x100u

/* Workspace bytes for batches of at most max_rows rows, scoring at most
 * max_group perturbed passes per LM-head launch (1 <= max_group <= 16; a larger
 * group amortises the clean logits over more passes).  flags: RK_WS_CLEAN_STATE
 * and/or RK_FLAG_UNFUSED_KL (room for materialised fp32 logits; implied for
 * RK_F32 models).  Returns 0 for invalid arguments.                            */
size_t rk_workspace_size(const rk_model *m, int64_t max_rows, int32_t max_group, uint32_t flags);
/* (flags may also hold RK_FLAG_CACHED_WINDOW: room for one layer's perturbed
 * prefix Values, and, with RK_WS_CLEAN_STATE, a cached-window state; and
 * RK_FLAG_LOCAL_SIGNAL: room for the clean output of the last block, and none
 * for LM-head partials or logits.)                                             */

/* ---------------------------------------------------------------- profiling */

/* ReferencePredict (Algorithm 1) for one batch: the clean forward, leaving the
 * per-layer inputs h_l and the final normalised hidden state in clean_state.    */
rk_status rk_reference_forward(const rk_model *m, const rk_batch *batch, void *clean_state,
                               size_t clean_bytes, void *workspace, size_t ws_bytes, void *stream);

/* ReferencePredict of the cached-window mode (Section 4.3) for one batch: the
 * prefix [0, window_start) of every sequence runs through all layers once and
 * leaves its KV cache; the window [window_start, T_i) is then evaluated against
 * the intact cache (its block inputs, final hidden state and log-sum-exp are
 * kept).  Every sequence must be longer than window_start > 0; bf16 models only.
 * state: at least rk_window_state_size(m, rows) bytes; workspace: at least
 * rk_workspace_size(m, rows, 1, RK_FLAG_CACHED_WINDOW).                        */
rk_status rk_window_reference(const rk_model *m, const rk_batch *batch, int32_t window_start, void *state,
                              size_t state_bytes, void *workspace, size_t ws_bytes, void *stream);

/* PerturbedPredict + WindowKL (Algorithm 1; Eqs. value-perturbation and
 * sample-response) for one batch, one layer and one alpha, resumed from a clean
 * state produced by rk_reference_forward for the same model and batch.
 *   d_out:      DEVICE fp32 [n_seqs]: d_{i,l} of each sequence of the batch.
 *   kl_pos:     DEVICE fp32 [rows] or NULL: KL(P_t || Q_t) at every position.
 *   logits_out: DEVICE fp32 [rows, vocab] or NULL: the perturbed logits
 *               (selects the unfused LM-head path; for verification).
 * workspace must be at least rk_workspace_size(m, rows, 1, f) with f =
 * RK_FLAG_UNFUSED_KL when logits_out is given, the flag is set or the model is
 * fp32, else 0 (plus RK_FLAG_CACHED_WINDOW in that mode).
 * With RK_FLAG_CACHED_WINDOW in p->flags, clean_state is a state from
 * rk_window_reference with the same window_start, and kl_pos / logits_out hold
 * the window rows only (sum_i (T_i - window_start) rows, sequence by sequence);
 * RK_FLAG_FULL_RECOMPUTE is not available in that mode.
 * With RK_FLAG_LOCAL_SIGNAL, d_out and kl_pos hold the layer-local response
 * instead of the KL, logits_out must be NULL, and the workspace size takes
 * RK_FLAG_LOCAL_SIGNAL in place of RK_FLAG_UNFUSED_KL.                         */
rk_status rk_profile_layer(const rk_model *m, const rk_batch *batch, int32_t layer, float alpha,
                           const rk_perturb_params *p, const void *clean_state, size_t clean_bytes,
                           float *d_out, float *kl_pos, float *logits_out,
                           void *workspace, size_t ws_bytes, void *stream);

/* Algorithm 1, profiling half, for a whole calibration set:
 *   s_out[a * n_A + j] = (1/N) sum_i d_{i, layers[j]} at alpha = alphas[a]
 *   (Eq. layer-sensitivity; an unweighted mean of per-sequence window means).
 * calib: all N sequences (offsets[N] rows); they are processed in batches of
 *   consecutive sequences holding at most max_rows rows each (a single sequence
 *   longer than max_rows is RK_ERR_SHAPE).
 * layers: HOST int32 [n_A], distinct, in [0, n_layers).  alphas: HOST [n_alpha],
 *   finite and >= 0.  s_out: DEVICE fp32 [n_alpha, n_A].  d_out: DEVICE fp32
 *   [n_alpha, N, n_A] or NULL.  One clean pass per batch serves every alpha.
 * max_group: passes scored per LM-head launch (1..16).
 * Pass batching: when max_rows holds at least two copies of a batch, the
 *   resumed passes of a group run layer-synchronously, min(max_group,
 *   max_rows / batch rows, RK_MAX_BATCH_SEQS / batch sequences) at a time:
 *   each joins at its perturbed layer and every launch of a block covers the
 *   rows of all joined passes.  Results are bitwise those of one pass at a
 *   time; the workspace grows with max_rows.
 * With RK_FLAG_CACHED_WINDOW the profile is that of the cached-window mode;
 * with RK_FLAG_LOCAL_SIGNAL, the layer-local signal of the ablation.
 * workspace must be at least rk_workspace_size(m, max_rows, max_group,
 * RK_WS_CLEAN_STATE | (p->flags & (RK_FLAG_UNFUSED_KL | RK_FLAG_CACHED_WINDOW |
 * RK_FLAG_LOCAL_SIGNAL))).                                                     */
rk_status rk_sensitivity_profile(const rk_model *m, const rk_batch *calib, const int32_t *layers,
                                 int32_t n_A, const float *alphas, int32_t n_alpha,
                                 const rk_perturb_params *p, int64_t max_rows, int32_t max_group,
                                 float *s_out, float *d_out, void *workspace, size_t ws_bytes,
                                 void *stream);

/* Allocation-free variant of rk_sensitivity_profile, for callers that cannot
 * allocate device memory (code running under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments, results and errors
 * as rk_sensitivity_profile, without the workspace: the buffers live in a
 * device array of RK_STATIC_SCRATCH_BYTES bytes inside the library (one per
 * GPU, held until the process ends).  It calls no allocator; the caller still
 * owns calib, s_out and d_out.
 *   - Calls whose workspace plan, rk_workspace_size(m, max_rows, max_group,
 *     RK_WS_CLEAN_STATE | (p->flags & (RK_FLAG_UNFUSED_KL |
 *     RK_FLAG_CACHED_WINDOW | RK_FLAG_LOCAL_SIGNAL))), exceeds
 *     RK_STATIC_SCRATCH_BYTES return RK_ERR_WORKSPACE before any device work.
 *   - RK_FLAG_GRAPH is refused (RK_ERR_ARG): recording a graph allocates.
 *   - Every call on one GPU uses that GPU's single array, so calls that
 *     overlap on one GPU (other streams, other threads) race: order them.
 *     Nothing is assumed about the array's previous contents.
 *   - stream, if not NULL, must belong to the current device (RK_ERR_HIP).
 *   - Its launches are not recorded by rk_timing_begin sessions.              */
#define RK_STATIC_SCRATCH_BYTES ((size_t)128 << 20)
rk_status rk_sensitivity_profile_static(const rk_model *m, const rk_batch *calib, const int32_t *layers,
                                        int32_t n_A, const float *alphas, int32_t n_alpha,
                                        const rk_perturb_params *p, int64_t max_rows, int32_t max_group,
                                        float *s_out, float *d_out, void *stream);

/* Eq. value-perturbation on its own: v (DEVICE, model dtype) holds the Values of
 * one layer for a batch, row r at v + r * row_stride elements, n_kv_heads *
 * head_dim contiguous values per row; they are replaced in place by
 * v + alpha * ||v||_2 * eps on the eligible positions.  eps is the Philox stream
 * of (seed, sequence index, layer, KV head, position).  v must be 8-byte (bf16)
 * or 16-byte (fp32) aligned and row_stride a multiple of 4 (RK_ERR_ARG).       */
rk_status rk_perturb_values(const rk_model *m, const rk_batch *batch, int32_t layer, float alpha,
                            const rk_perturb_params *p, void *v, int64_t row_stride, void *stream);

/* ---------------------------------------------------------------- allocation */

/* Algorithm 1, allocation half (Section 4.4, Eqs. sensitivity-normalization,
 * sensitivity-mapping, weight-normalization, layer-budget).  Host only,
 * synchronous, float64.
 *   s: [n] finite sensitivities; B >= 0 global budget; r >= 1 ratio;
 *   gamma: clip bound >= 1, or <= 0 / infinity for no clipping;
 *   eps: denominator guard of the min-max step (0 = the equation, with a
 *        constant profile mapped to all zeros);
 *   w_out: [n] multipliers or NULL; b_out: [n] integer budgets.
 * With RK_ROUND_LARGEST_REMAINDER sum(b) == B: b = floor(q) for q = B w / n
 * snapped to multiples of 2^-20, then the leftover units go to the largest
 * fractional parts (ties: larger s, then lower index).                          */
rk_status rk_layer_budgets(const double *s, int32_t n, int64_t B, double r, double gamma, double eps,
                           rk_rounding mode, double *w_out, int64_t *b_out);

/* ---------------------------------------------------------------- budgets' consumer: SnapKV */

/* Section 4.4: the budgets b_l replace the uniform per-layer budget of the base
 * compressor, whose own token scoring and selection are kept; layer l then keeps
 * b_l positions (the compressed cache of Section 3).  The base method is SnapKV;
 * the paper gives none of its constants, so they are parameters:
 *   obs_window w (1..64): the last w positions of each prompt; their queries vote
 *     and they are always kept;
 *   vote of KV head g for a prefix position u < T - w: the causal softmax weight
 *     the w observation queries put on key u, summed over the queries and over
 *     the query heads sharing g;
 *   pooling along positions, odd kernel (1..31): RK_POOL_MAX = maximum within
 *     kernel/2 positions, RK_POOL_AVG = their sum / kernel (zeros outside);
 *   retained: the window and the b - w prefix positions of highest pooled vote
 *     (ties to the lower position); b >= T keeps all, b <= w the last b.
 * bf16 models only; (n_heads / n_kv_heads) * ceil(w / 32) <= 8.                  */
typedef enum { RK_POOL_MAX = 0, RK_POOL_AVG = 1 } rk_pooling;
typedef struct {
  int32_t obs_window;
  int32_t pool_kernel;
  rk_pooling pooling;
} rk_snapkv_params;

/* Longest prefix (T - w) a sequence may have for rk_snapkv_compress. */
#define RK_SNAPKV_MAX_PREFIX 36864

/* Bytes of the prefill state of a batch of n_rows rows and n_seqs sequences:
 *   kv: [L, n_rows, 2 * n_kv_heads * head_dim] bf16, per row the rotated Keys of
 *       every KV head, then its Values (the prompt's KV cache, Section 3);
 *   q:  [L, n_seqs * w, n_heads * head_dim] bf16, the rotated queries of each
 *       sequence's last w positions multiplied by log2(e) / sqrt(head_dim),
 *   kv first, q at the next multiple of 256 bytes.                               */
size_t rk_snapkv_state_size(const rk_model *m, int64_t n_rows, int32_t n_seqs, int32_t obs_window);

/* Workspace bytes of rk_snapkv_prefill and rk_snapkv_compress for such a batch. */
size_t rk_snapkv_workspace_size(const rk_model *m, int64_t n_rows, int32_t n_seqs, int32_t obs_window);

/* The prompts' forward pass through every layer, keeping the KV cache and the
 * observation queries in `state` (layout above).  Every sequence must be longer
 * than obs_window.                                                               */
rk_status rk_snapkv_prefill(const rk_model *m, const rk_batch *batch, int32_t obs_window, void *state,
                            size_t state_bytes, void *workspace, size_t ws_bytes, void *stream);

/* Compressed-cache layout (host, synchronous).  budgets: HOST int64
 * [n_seqs * n_layers], b_{i,l} at i * n_layers + l.  n_keep(i, l) = min(max(b, 0),
 * T_i); offsets_out (HOST int64 [n_seqs * n_layers + 1], may be NULL) receives the
 * exclusive prefix sums of n_keep in that order.  Returns the total, or -1 on a
 * bad argument.  Block (i, l, g) of the outputs of rk_snapkv_compress holds
 * n_keep(i, l) entries starting at entry offsets[i * L + l] * n_kv_heads +
 * g * n_keep(i, l).                                                              */
int64_t rk_snapkv_layout(const rk_batch *batch, int32_t n_layers, const int64_t *budgets, int64_t *offsets_out);

/* SnapKV selection with the per-layer budgets, every (sequence, layer, KV head),
 * from a prefill state of the same batch.
 *   positions: DEVICE int32 [n_kv_heads * total]: retained positions (within
 *     the sequence), increasing, per block;
 *   k_out, v_out: DEVICE bf16 [n_kv_heads * total, head_dim]: their rotated Keys
 *     and Values;
 *   scores: DEVICE fp32 [n_layers, n_kv_heads, sum_i (T_i - w)] pooled votes,
 *     sequence by sequence, or NULL.
 * Requires obs_window < T_i and T_i - obs_window <= RK_SNAPKV_MAX_PREFIX.        */
rk_status rk_snapkv_compress(const rk_model *m, const rk_batch *batch, const rk_snapkv_params *p,
                             const int64_t *budgets, const void *state, size_t state_bytes, int32_t *positions,
                             void *k_out, void *v_out, float *scores, void *workspace, size_t ws_bytes,
                             void *stream);

/* ---------------------------------------------------------------- compression damage */

/* Isolated single-layer compression damage (Section 2, Eq.
 * layer-compression-damage) in the cached-window split: the window [P, T) of
 * every sequence is evaluated against the prompt caches of rk_window_reference
 * (same batch, window_start = P) with only layer `layer`'s prompt cache
 * restricted to n_keep retained positions per KV head (1 <= n_keep <= P); the
 * other layers keep their full caches.  d_out[i] = mean over the window of
 * KL(P_full || P_compressed), kl_pos (may be NULL) the per-position values
 * (window rows only).
 *   positions: DEVICE int32, position j (< P, within the sequence) retained by
 *     KV head g of sequence i at positions[i * seq_stride + g * n_keep + j]
 *     (seq_stride >= n_kv_heads * n_keep).  With the outputs of
 *     rk_snapkv_compress for prompts of P tokens and the same budget b at every
 *     layer, layer l's positions start at entry l * n_kv_heads * b with
 *     seq_stride = n_layers * n_kv_heads * b.
 * Workspace: rk_workspace_size(m, rows, 1, RK_FLAG_CACHED_WINDOW).  bf16 only.  */
rk_status rk_compression_damage(const rk_model *m, const rk_batch *batch, int32_t window_start, int32_t layer,
                                const int32_t *positions, int64_t seq_stride, int32_t n_keep, const void *state,
                                size_t state_bytes, float *d_out, float *kl_pos, void *workspace, size_t ws_bytes,
                                void *stream);

/* The damage of several layers in one call: d_out[k * n_seqs + i] is
 * rk_compression_damage's d_i for layer layers[k] (HOST int32 [n_layers], 1 ..
 * 16 entries), whose retained positions start at positions + layers[k] *
 * layer_stride (per sequence at seq_stride, as for rk_compression_damage; with
 * the outputs of rk_snapkv_compress for prompts of P tokens and the same budget b
 * at every layer: layer_stride = n_kv_heads * b, seq_stride = n_layers *
 * n_kv_heads * b).  kl_pos: DEVICE fp32 [n_layers, window rows] or NULL.  The
 * layers are evaluated together, each joining at its own layer, so the
 * projections run once per layer over the window rows of every layer being
 * evaluated; the results are bitwise those of separate rk_compression_damage
 * calls.  Workspace: rk_workspace_size(m, rows, n_layers, RK_FLAG_CACHED_WINDOW).  */
rk_status rk_compression_damage_layers(const rk_model *m, const rk_batch *batch, int32_t window_start,
                                       const int32_t *layers, int32_t n_layers, const int32_t *positions,
                                       int64_t layer_stride, int64_t seq_stride, int32_t n_keep, const void *state,
                                       size_t state_bytes, float *d_out, float *kl_pos, void *workspace,
                                       size_t ws_bytes, void *stream);

/* The damage of a whole per-layer budget policy (Section 4.4: the budgets
 * deployed, every layer's prompt cache compressed at once): the window rows
 * [window_start, T_i) run from block 0 with block l attending to the n_keep[l]
 * retained prompt positions of each KV head, or to the whole prompt cache when
 * n_keep[l] is 0; d_out[i] is the window mean of KL(full-cache || compressed)
 * per position, as for rk_compression_damage.  The prompt caches are those of
 * the full prefill in state (rk_window_reference with the same window_start).
 *   positions:     DEVICE int32; layer l, sequence i, KV head h, entry j at
 *                  positions[layer_offsets[l] + i * seq_stride + h * n_keep[l] + j]
 *                  (clamped to [0, window_start)); NULL allowed when every
 *                  n_keep is 0.  With the outputs of rk_snapkv_compress for
 *                  budgets that are the same for every sequence:
 *                  layer_offsets[l] = n_kv_heads * sum_{l' < l} b_l',
 *                  seq_stride = n_kv_heads * sum_l b_l.
 *   layer_offsets: HOST int64 [n_layers]; n_keep: HOST int32 [n_layers], each in
 *                  [0, window_start].
 *   kl_pos:        DEVICE fp32 [window rows] or NULL.
 *   logits_out:    DEVICE fp32 [window rows, vocab] or NULL: the compressed
 *                  model's logits of the window rows (with window_start = T_i - 1,
 *                  one decode step over the compressed caches); selects the
 *                  unfused LM head.
 * Workspace: rk_workspace_size(m, rows, 1, RK_FLAG_CACHED_WINDOW), plus
 * RK_FLAG_UNFUSED_KL when logits_out is given.                                  */
rk_status rk_policy_damage(const rk_model *m, const rk_batch *batch, int32_t window_start, const int32_t *positions,
                           const int64_t *layer_offsets, int64_t seq_stride, const int32_t *n_keep,
                           const void *state, size_t state_bytes, float *d_out, float *kl_pos, float *logits_out,
                           void *workspace, size_t ws_bytes, void *stream);

/* Several budget policies in one call: d_out[q * n_seqs + i] (and kl_pos [q,
 * window rows], DEVICE fp32 or NULL) are rk_policy_damage's values for policy q
 * (1 <= n_policies <= 16).  Per policy q: positions[q] (a HOST array of DEVICE
 * pointers; NULL allowed when every n_keep of the policy is 0), layer offsets
 * layer_offsets[q * n_layers + l] and counts n_keep[q * n_layers + l] (HOST),
 * sequence stride seq_stride[q] (HOST int64 [n_policies]).  The policies are
 * evaluated together from block 0: every norm, projection and feed-forward runs
 * once per layer over the window rows of all of them, each attending to its own
 * caches; the results are bitwise those of separate rk_policy_damage calls.
 * Workspace: rk_workspace_size(m, rows, n_policies, RK_FLAG_CACHED_WINDOW).     */
rk_status rk_policy_damage_group(const rk_model *m, const rk_batch *batch, int32_t window_start, int32_t n_policies,
                                 const int32_t *const *positions, const int64_t *layer_offsets,
                                 const int64_t *seq_stride, const int32_t *n_keep, const void *state,
                                 size_t state_bytes, float *d_out, float *kl_pos, void *workspace, size_t ws_bytes,
                                 void *stream);

/* Spearman's rho of two profiles x, y [n] (Section 2, Table
 * sensitivity-correlation): the Pearson correlation of their ranks, ties sharing
 * the mean rank; NaN when a profile is constant.  Host only, float64.          */
rk_status rk_spearman(const double *x, const double *y, int32_t n, double *rho);

/* ---------------------------------------------------------------- diagnostics */

/* Per-kernel timing for measurement: after rk_timing_begin(family) every launch
 * of that kernel family is bracketed by HIP events recorded on its launch stream
 * (families: "rmsnorm", "gemm_qkv", "noise", "attention", "gemm_o",
 * "gemm_gate_up", "gemm_down", "lm_lse", "lm_kl", "kl_logits", "lm_logits",
 * "local", "snap_scores", "snap_select").
 * rk_timing_end waits for the recorded events, returns the number of launches
 * and their summed duration in milliseconds, and stops recording.  Host-side
 * state is process-wide; not for concurrent use from several threads.          */
rk_status rk_timing_begin(const char *family);
rk_status rk_timing_end(int64_t *launches, double *total_ms);

/* Message of the last error on the calling thread ("" if none). */
const char *rk_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RK_H */
