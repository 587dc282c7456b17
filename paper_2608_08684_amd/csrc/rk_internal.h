// Internal declarations shared by the HIP kernels and the host scheduler.
// Everything here is private to librk; the public surface is include/rk.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "rk.h"

namespace rk {

typedef uint16_t bf16_t;  // raw bf16 bit pattern in memory
// 16-byte native vector (promotes to registers, unlike HIP's union-based uint4)
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// Row layout of one batch: sequence k owns rows [off[k], off[k+1]).  Passed to
// kernels by value (fits easily in the kernel-argument segment).
struct SeqTable {
  int32_t n;            // sequences in the batch
  int32_t seq_index0;   // calibration index of sequence 0 (keys the noise)
  int32_t max_len;      // longest sequence of the batch
  int32_t rows;         // off[n]
  int32_t off[RK_MAX_BATCH_SEQS + 1];
};

// Work list of the bf16 attention kernel.  A work item is a pair of q-blocks of
// one sequence, (nqb - 1 - x, x), so every item of a sequence costs about the
// same; sequences are visited longest first.
struct AttnWork {
  int32_t total;                          // work items (pairs) over all sequences
  int32_t order[RK_MAX_BATCH_SEQS];       // sequence indices by decreasing length
  int32_t cum[RK_MAX_BATCH_SEQS + 1];     // cum[j] = pairs of sequences order[0..j)
};

// --------------------------------------------------------------------------- device helpers
#if defined(__HIPCC__)
__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// fp32 -> bf16, round to nearest even (gfx950 v_cvt_pk_bf16_f32; NaN stays NaN).
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

__device__ __forceinline__ int seq_of_row(const SeqTable& st, int r) {
  int lo = 0, hi = st.n - 1;
  while (lo < hi) {  // largest k with off[k] <= r
    int mid = (lo + hi + 1) >> 1;
    if (st.off[mid] <= r) lo = mid; else hi = mid - 1;
  }
  return lo;
}

template <typename T> struct Act;
template <> struct Act<float> {
  static __device__ __forceinline__ float load(const float* p) { return *p; }
  static __device__ __forceinline__ void store(float* p, float v) { *p = v; }
};
template <> struct Act<bf16_t> {
  static __device__ __forceinline__ float load(const bf16_t* p) { return bf2f(*p); }
  static __device__ __forceinline__ void store(bf16_t* p, float v) { *p = f2bf(v); }
};
#endif

// Device address of this device's RK_STATIC_SCRATCH_BYTES-byte scratch array
// (looked up once per device).  A non-null stream must belong to the current
// device (hipErrorInvalidDevice otherwise).
hipError_t static_scratch(hipStream_t stream, void** out);

// --------------------------------------------------------------------------- launchers
// Each returns hipSuccess or the launch error.  `act_bf16` selects the element type
// of activation buffers (bf16 when true, fp32 otherwise).

hipError_t launch_embed(const void* emb, bool emb_bf16, const int32_t* tokens, float* h, int rows, int d,
                        hipStream_t s);
hipError_t launch_rmsnorm(const float* h, const float* g, void* out, bool out_bf16, int rows, int d,
                          float eps, hipStream_t s);
// Rotary table of a batch: tab[t * head_dim/2 + j] = (cos, sin)(t * theta^(-2j/head_dim)) for
// t < max_len, and pos[r] = position of row r inside its sequence.
// Rotary table for positions [0, pos0 + max_len) and the position of every row:
// pos0 + its index within its sequence.
hipError_t launch_rope_table(float2* tab, int32_t* pos, const SeqTable& st, int head_dim, float theta, hipStream_t s,
                             int pos0 = 0);
hipError_t launch_embed_gather(const void* emb, bool emb_bf16, const int32_t* tokens, const SeqTable& src,
                               const SeqTable& dst, int pos0, float* h, int d, hipStream_t s);
hipError_t launch_copy_cols(const void* src, int64_t ld_src_bytes, int64_t off_bytes, void* dst, int64_t ld_dst_bytes,
                            int64_t nbytes, int rows, hipStream_t s);
hipError_t launch_value_noise(void* v, bool bf16, int64_t row_stride, const SeqTable& st, int n_kv_heads,
                              int head_dim, int layer, float alpha, uint64_t seed, int protect_head,
                              int protect_tail, hipStream_t s);

// GEMM family: C[M, N] = A[M, K] * B[N, K]^T with a fused epilogue.
enum class Epi { kStoreRope, kResidual, kSwiGLU, kStoreF32 };
struct GemmArgs {
  const void* A; int64_t lda;
  const void* B; int64_t ldb;
  int M, N, K;           // N = columns of B used (for kSwiGLU: 2 * d_ff)
  Epi epi;
  void* out; int64_t ldo;         // output (act type, or fp32 for kResidual/kStoreF32)
  const float* res; int64_t ldr;  // kResidual: out = res + C (res may alias out)
  // kStoreRope: columns < rope_cols are rotated (pairs j, j + head_dim/2) with
  // rope_tab[pos * head_dim/2 + j] = (cos, sin), pos = rope_pos[row]
  int rope_cols; int head_dim; const float2* rope_tab; const int32_t* rope_pos;
  // kStoreRope: columns < q_cols (the queries) are multiplied by q_scale after the
  // rotation, before rounding (q_cols = 0: no scaling)
  int q_cols; float q_scale;
  int d_ff;                        // kSwiGLU: gate rows [0, d_ff), up rows [d_ff, 2 d_ff)
  int tile_m, tile_n, tile_k;      // 0: automatic tile choice (bf16 path)
  int tile_waves;                  // waves per workgroup of an explicit tile (4 or 8)
  int tile_stages;                 // LDS pipeline stages of an explicit tile (0: 2)
  int group_m;                     // tile-rows per L2 group (0: default)
};
hipError_t launch_gemm(const GemmArgs& a, bool bf16, hipStream_t s);

// Cached prefix of the cached-window mode: every sequence k of the batch has P
// cached positions, rows k * P .. k * P + P - 1 of the K cache (row stride ldk,
// KV head h at columns h * d_h) and of the V cache (row stride ldv, same columns);
// the attention rows of the batch are the positions P.. of each sequence and see
// every cached position before their own causal keys.
struct KvPrefix {
  const bf16_t* k;
  const bf16_t* v;
  int64_t ldk, ldv;
  int32_t P;
  // Several passes' window rows in one launch (n_seq > 0): sequence s of the table
  // reads the cached prefix of sequence s % n_seq, and the sequences of pass
  // alt_pass (s / n_seq == alt_pass; -1 for none) read their Values from v_alt
  // (row stride ldv_alt) instead of v.  n_seq = 0: sequence s reads prefix s.
  const bf16_t* v_alt;
  int64_t ldv_alt;
  int32_t n_seq;
  int32_t alt_pass;
};

hipError_t launch_attention(const void* qkv, int64_t ldq, void* out, int64_t ldo, const SeqTable& st,
                            int n_heads, int n_kv_heads, int head_dim, bool bf16, hipStream_t s,
                            const KvPrefix* prefix = nullptr);

// Clean log-sum-exp of the LM head, fused (bf16): lse[r] = logsumexp_v (x[r] . W[v]).
int lm_chunks(int rows, int vocab);      // vocab chunks of lm_lse (partials: chunks * rows float2)
int lm_kl_chunks(int rows, int vocab);   // vocab chunks of lm_kl (partials: chunks * G * rows float2)
hipError_t launch_lm_lse(const bf16_t* x, const bf16_t* W, int rows, int d, int vocab, float2* part,
                         float* lse, hipStream_t s);
// Fused LM head + KL (bf16): for pass g, kl[g][r] = KL(softmax(x_c W^T) || softmax(x_g W^T)).
hipError_t launch_lm_kl(const bf16_t* xc, const bf16_t* xp, int64_t pass_stride, int G, const bf16_t* W,
                        int rows, int d, int vocab, const float* lse, float2* part, float* kl,
                        hipStream_t s);
// Unfused KL over materialised fp32 logits: kl[g][r] = KL(softmax(lc[r]) || softmax(lp[g][r])).
hipError_t launch_kl_logits(const float* lc, const float* lp, int64_t pass_stride, int G, int rows, int vocab,
                            float* kl, hipStream_t s);

// Layer-local response of one block: r[row] = ||hp[row] - hc[row]||^2 / ||hc[row]||^2
// (fp32 rows of d values, d a multiple of 4; 0 for a zero clean row).
hipError_t launch_local_response(const float* hp, const float* hc, int rows, int d, float* r, hipStream_t s);

// dbatch[g * n_seqs + k] = mean of kl[g * kl_stride + r] over r in [off[k] + window_start, off[k+1]).
// {magic, host, digest of tokens[0, rows), rows} into out[0..3] (one block)
hipError_t launch_state_tag(const int32_t* tokens, int64_t rows, uint64_t magic, uint64_t host, uint64_t* out,
                            hipStream_t s);
hipError_t launch_window_mean(const float* kl, int64_t kl_stride, int G, const SeqTable& st, int window_start,
                              float* dbatch, hipStream_t s);

// Where the d values of a group of passes go: pass g of the group writes
// d_out[d_base[g] + seq * d_seq_stride] and accumulates into s_acc[s_index[g]].
#define RK_MAX_GROUP 16
struct PassMap {
  int32_t G;
  int32_t seq_index0;
  int64_t d_seq_stride;
  int64_t d_base[RK_MAX_GROUP];
  int32_t s_index[RK_MAX_GROUP];
};
hipError_t launch_accumulate(const float* dbatch, int n_seqs, const PassMap& pm, float* d_out, double* s_acc,
                             hipStream_t s);

// SnapKV selection with per-layer budgets (bf16).  One layer per call.
// Observation queries of the prefill: dst[i * w + j] = qkv row off[i + 1] - w + j, first qcols columns.
hipError_t launch_snap_qobs(const void* qkv, int64_t ldq, const SeqTable& st, int w, int qcols, void* dst,
                            hipStream_t s);
constexpr int kSnapMaxPrefix = RK_SNAPKV_MAX_PREFIX;   // prefix positions held in LDS by the selection
constexpr int kSnapMaxCombos = 8;                      // (query heads per KV head) x ceil(w / 32)
int snap_chunks(int max_len);                          // key chunks of the scoring kernels
// Votes of every layer: votes[(l * n_kv + g) * prefix_rows + (off[i] - i w) + u] for prefix keys
// u < T_i - w; layer l's cache at kv + l * kv_layer_stride and queries at qobs + l * q_layer_stride
// (elements); part: L * n * H * w * chunks float2, cnorm: L * n * H * w floats.
hipError_t launch_snap_scores(const void* kv, int64_t ldkv, int64_t kv_layer_stride, const void* qobs,
                              int64_t q_layer_stride, int n_layers, const SeqTable& st, int w, int n_heads, int n_kv,
                              int head_dim, float2* part, float* cnorm, float* votes, int64_t prefix_rows,
                              hipStream_t s);
// A prompt cache of b rows per sequence from the retained positions (per KV head) of a
// full prompt cache of P rows per sequence: row i * b + j, head g <- position
// pos[i * seq_stride + g * b + j].
hipError_t launch_prefix_gather(const void* kv, int64_t ldkv, int n_seqs, int P, int n_kv, int head_dim,
                                const int32_t* pos, int64_t seq_stride, int b, void* out, hipStream_t s);
// Pooling, selection and gather for n_items (sequence, layer) items (host arrays);
// votes and scores [layer][n_kv][prefix_rows], kv of layer l at kv + l * kv_layer_stride.
hipError_t launch_snap_select(const float* votes, int64_t prefix_rows, const void* kv, int64_t ldkv,
                              int64_t kv_layer_stride, const SeqTable& st, int w, int n_kv, int head_dim,
                              int pool_kernel, bool pool_avg, int n_items, const int16_t* seq, const int16_t* layer,
                              const int32_t* keep, const int64_t* entry0, int32_t* positions, void* k_out, void* v_out,
                              float* scores, hipStream_t s);
hipError_t launch_finalize(const double* s_acc, int n, double inv_n, float* s_out, hipStream_t s);
hipError_t launch_zero_f64(double* p, int n, hipStream_t s);

}  // namespace rk
