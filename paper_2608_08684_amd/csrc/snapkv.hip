// SnapKV token selection with per-layer budgets: the consumer of the budgets b_l
// (Section 4.4 keeps the base compressor's scoring and selection and replaces
// only its uniform per-layer budget; Section 3 defines the compressed cache of
// b_l positions per layer).
//
// Per layer l, sequence i (T_i positions, observation window w = its last w
// positions) and KV head g:
//   vote(u)  = sum over the query heads of g and the w observation queries t of
//              softmax_t(q_t . k_u / sqrt(d_h)) (causal), for prefix keys u < T_i - w;
//   pooled   = max (or mean, zeros outside) of the votes within kernel/2 positions;
//   retained = the window plus the b - w prefix positions of highest pooled vote
//              (ties to the lower position), in increasing order;
//   the compressed cache holds those positions' rotated Keys and Values.
//
// Kernels (one layer per launch):
//   snap_stats_kernel   per (key chunk, KV head, sequence): running max / sum of
//                       exp2 of the observation queries' scores over the chunk's
//                       keys (S^T = K Q^T on MFMA, one query per lane);
//   snap_norm_kernel    fixed-order merge over chunks -> log2 normalizer c_t;
//   snap_votes_kernel   per (prefix chunk, KV head, sequence): S = Q K^T on MFMA
//                       with the accumulator started at -c_t, so exp2 of the
//                       result is the probability; each lane owns one key and
//                       sums its probabilities over queries and heads;
//   snap_select_kernel  per (KV head, sequence): pooling into LDS, radix select
//                       of the (b - w)-th largest pooled vote, compaction in
//                       position order, gather of the K and V rows.
// Queries arrive multiplied by log2(e) / sqrt(d_h) (the attention kernels' form),
// so all exponentials are exp2.
#include <math.h>

#include <algorithm>

#include "mfma_tile.h"

namespace rk {

constexpr int kSnapChunk = 256;   // keys per workgroup of the scoring kernels (4 waves x 64)

// Observation-query tile in LDS: row r (combination c = r / 32 of query head and
// 32-query block, query j = r % 32) holds CH = d_h / 8 16-byte chunks padded to
// CH + 1 slots, which spreads 16 consecutive rows over all 64 banks.
template <int DH>
__device__ __forceinline__ bf16x8_t qfrag(const v4u* qt, int row, int ks, int lane) {
  constexpr int CH = DH / 8;
  return __builtin_bit_cast(bf16x8_t, qt[row * (CH + 1) + ks * 2 + (lane >> 5)]);
}

// The K fragment of one cache row, k-slice ks, straight from global memory.
__device__ __forceinline__ bf16x8_t kfrag(const bf16_t* krow, int ks, int lane) {
  return *reinterpret_cast<const bf16x8_t*>(krow + ks * 16 + (lane >> 5) * 8);
}

// Stage the observation queries of KV head g of sequence i into LDS: combos =
// group * nqb rows of 32 queries (rows past w are zero).
template <int DH>
__device__ __forceinline__ void load_qobs(v4u* qt, const bf16_t* qobs, int64_t ldq, int i, int g, int w, int group,
                                          int nqb) {
  constexpr int CH = DH / 8;
  const int rows = group * nqb * 32;
  for (int slot = threadIdx.x; slot < rows * CH; slot += blockDim.x) {
    const int r = slot / CH, ch = slot % CH;
    const int combo = r >> 5, jj = (combo % nqb) * 32 + (r & 31);
    const int h = g * group + combo / nqb;
    v4u val = {0u, 0u, 0u, 0u};
    if (jj < w) val = *reinterpret_cast<const v4u*>(qobs + ((int64_t)i * w + jj) * ldq + h * DH + ch * 8);
    qt[r * (CH + 1) + ch] = val;
  }
}

// Bytes of the observation-query tile (dynamic LDS of the scoring kernels).
__host__ __device__ constexpr int qtile_bytes(int head_dim, int combos) { return combos * 32 * (head_dim / 8 + 1) * 16; }

// Layer l of the batched launches: blockIdx.z = l * n + i; the layer's K|V cache
// at kv + l * kv_stride, its observation queries at qobs + l * q_stride.
struct SnapLayers {
  int64_t kv_stride, q_stride;   // elements
};

template <int DH>
__global__ __launch_bounds__(256) void snap_stats_kernel(const bf16_t* __restrict__ kv, int64_t ldkv,
                                                         const bf16_t* __restrict__ qobs, int64_t ldq, SeqTable st,
                                                         int w, int n_heads, int n_kv, int nchunks, SnapLayers ly,
                                                         float2* __restrict__ part) {
  constexpr int NKS = DH / 16, MAXC = 8;
  extern __shared__ v4u qt[];
  __shared__ float2 red[4][MAXC][32];
  const int c = blockIdx.x, g = blockIdx.y, l = blockIdx.z / st.n, i = blockIdx.z % st.n;
  const int T = st.off[i + 1] - st.off[i], row0 = st.off[i];
  if (c * kSnapChunk >= T) return;
  kv += l * ly.kv_stride;
  qobs += l * ly.q_stride;
  part += (int64_t)l * st.n * n_heads * w * nchunks;
  const int group = n_heads / n_kv, nqb = (w + 31) >> 5, combos = group * nqb;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, l32 = lane & 31;
  // this wave's 64 keys, both 32-key blocks in flight before the MFMAs
  const int ub0 = c * kSnapChunk + wv * 64;
  bf16x8_t kf2[2][NKS];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int uc = min(ub0 + kb * 32 + l32, T - 1);
    const bf16_t* krow = kv + (int64_t)(row0 + uc) * ldkv + (int64_t)g * DH;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) kf2[kb][ks] = kfrag(krow, ks, lane);
  }
  load_qobs<DH>(qt, qobs, ldq, i, g, w, group, nqb);
  __syncthreads();
  float m[MAXC], z[MAXC];
#pragma unroll
  for (int q = 0; q < MAXC; ++q) { m[q] = -INFINITY; z[q] = 0.f; }
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int ub = ub0 + kb * 32;
    if (ub >= T) break;
    const bf16x8_t* kf = kf2[kb];
#pragma unroll
    for (int q = 0; q < MAXC; ++q) {
      if (q >= combos) break;
      f32x16_t acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks], qfrag<DH>(qt, q * 32 + l32, ks, lane), acc, 0, 0, 0);
      // element r: key ub + 8 (r / 4) + 4 (lane / 32) + r % 4, query t (this lane's column)
      const int jj = (q % nqb) * 32 + l32;
      const int t = T - w + jj;
      float mx = -INFINITY;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int u = ub + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (u >= T || u > t || jj >= w) acc[r] = -INFINITY;
        mx = fmaxf(mx, acc[r]);
      }
      const float mn = fmaxf(m[q], mx);
      if (mn != -INFINITY) {
        float sum = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) sum += exp2f(acc[r] - mn);
        z[q] = z[q] * exp2f(m[q] - mn) + sum;
        m[q] = mn;
      }
    }
  }
  // the two half-waves hold the same queries (different keys); then the 4 waves
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    if (q >= combos) break;
    const float m2 = __shfl_xor(m[q], 32, 64), z2 = __shfl_xor(z[q], 32, 64);
    const float mm = fmaxf(m[q], m2);
    const float zz = mm == -INFINITY ? 0.f : z[q] * exp2f(m[q] - mm) + z2 * exp2f(m2 - mm);
    if (lane < 32) red[wv][q][l32] = make_float2(mm, zz);
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < combos * 32; idx += blockDim.x) {
    const int q = idx >> 5, j = idx & 31;
    const int jj = (q % nqb) * 32 + j;
    if (jj >= w) continue;
    float mm = -INFINITY;
    for (int k = 0; k < 4; ++k) mm = fmaxf(mm, red[k][q][j].x);
    float zz = 0.f;
    if (mm != -INFINITY)
      for (int k = 0; k < 4; ++k) zz += red[k][q][j].y * exp2f(red[k][q][j].x - mm);
    const int h = g * group + q / nqb;
    part[(((int64_t)i * n_heads + h) * w + jj) * nchunks + c] = make_float2(mm, zz);
  }
}

// c_t = log2 of the softmax denominator of query t (in the scores' log2 units),
// for every layer: index l * n * H * w + (i * H + h) * w + j.
__global__ void snap_norm_kernel(const float2* __restrict__ part, SeqTable st, int w, int n_heads, int nchunks,
                                 int n_layers, float* __restrict__ cnorm) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n_layers * st.n * n_heads * w) return;
  const int i = (idx / (n_heads * w)) % st.n;
  const int T = st.off[i + 1] - st.off[i];
  const int nc = (T + kSnapChunk - 1) / kSnapChunk;
  const float2* p = part + (int64_t)idx * nchunks;
  float M = -INFINITY;
  for (int c = 0; c < nc; ++c) M = fmaxf(M, p[c].x);
  double Z = 0.0;
  for (int c = 0; c < nc; ++c)
    if (p[c].y > 0.f) Z += (double)p[c].y * exp2((double)p[c].x - (double)M);
  cnorm[idx] = (float)((double)M + log2(Z));
}

template <int DH>
__global__ __launch_bounds__(256) void snap_votes_kernel(const bf16_t* __restrict__ kv, int64_t ldkv,
                                                         const bf16_t* __restrict__ qobs, int64_t ldq, SeqTable st,
                                                         int w, int n_heads, int n_kv, SnapLayers ly,
                                                         const float* __restrict__ cnorm, float* __restrict__ votes,
                                                         int64_t prefix_rows) {
  constexpr int NKS = DH / 16, MAXC = 8;
  extern __shared__ v4u qt[];
  __shared__ float cinit[MAXC * 32];
  const int c = blockIdx.x, g = blockIdx.y, l = blockIdx.z / st.n, i = blockIdx.z % st.n;
  const int T = st.off[i + 1] - st.off[i], row0 = st.off[i], npre = T - w;
  if (c * kSnapChunk >= npre) return;
  kv += l * ly.kv_stride;
  qobs += l * ly.q_stride;
  cnorm += (int64_t)l * st.n * n_heads * w;
  votes += (int64_t)l * n_kv * prefix_rows;
  const int group = n_heads / n_kv, nqb = (w + 31) >> 5, combos = group * nqb;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, l32 = lane & 31;
  const int ub0 = c * kSnapChunk + wv * 64;
  bf16x8_t kf2[2][NKS];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const bf16_t* krow = kv + (int64_t)(row0 + min(ub0 + kb * 32 + l32, npre - 1)) * ldkv + (int64_t)g * DH;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) kf2[kb][ks] = kfrag(krow, ks, lane);
  }
  load_qobs<DH>(qt, qobs, ldq, i, g, w, group, nqb);
  for (int idx = threadIdx.x; idx < combos * 32; idx += blockDim.x) {
    const int q = idx >> 5, jj = (q % nqb) * 32 + (idx & 31);
    const int h = g * group + q / nqb;
    cinit[idx] = jj < w ? -cnorm[((int64_t)i * n_heads + h) * w + jj] : -INFINITY;
  }
  __syncthreads();
  const int64_t pre0 = (int64_t)row0 - (int64_t)i * w;   // first prefix row of sequence i in the votes
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int ub = ub0 + kb * 32;
    if (ub >= npre) break;
    const int u = ub + l32;
    const bf16x8_t* kf = kf2[kb];
    float vote = 0.f;
#pragma unroll
    for (int q = 0; q < MAXC; ++q) {
      if (q >= combos) break;
      // element r: query row 8 (r / 4) + 4 (lane / 32) + r % 4 of block q, key u
      f32x16_t acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = cinit[q * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)];
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qfrag<DH>(qt, q * 32 + l32, ks, lane), kf[ks], acc, 0, 0, 0);
#pragma unroll
      for (int r = 0; r < 16; ++r) vote += exp2f(acc[r]);
    }
    vote += __shfl_xor(vote, 32, 64);
    if (lane < 32 && u < npre) votes[(int64_t)g * prefix_rows + pre0 + u] = vote;
  }
}

// Selection work of one launch: items (sequence i, layer l) with their kept
// count and first output entry; the table travels in the kernel arguments.
constexpr int kSelItems = 192;   // keeps the argument block (with the row table) under 4 KB
struct SnapSel {
  int32_t n;
  int16_t seq[kSelItems];
  int16_t layer[kSelItems];
  int32_t keep[kSelItems];     // n_keep = min(max(b, 0), T_i)
  int64_t entry0[kSelItems];   // first output entry of (i, l): offset(i, l) * n_kv_heads
};

constexpr int kSelThreads = 512;

__device__ __forceinline__ int block_exclusive_scan(int v, int* s) {
  const int tid = threadIdx.x;
  s[tid] = v;
  __syncthreads();
  for (int off = 1; off < kSelThreads; off <<= 1) {
    const int t = tid >= off ? s[tid - off] : 0;
    __syncthreads();
    s[tid] += t;
    __syncthreads();
  }
  const int incl = s[tid];
  __syncthreads();
  return incl - v;
}

// votes / scores: [layer][n_kv][prefix_rows]; kv: [layer][rows][ldkv].
template <int DH>
__global__ __launch_bounds__(kSelThreads) void snap_select_kernel(
    const float* __restrict__ votes, int64_t prefix_rows, const bf16_t* __restrict__ kv, int64_t ldkv,
    int64_t kv_layer_stride, SeqTable st, int w, int n_kv, int pool_kernel, int pool_avg, SnapSel sel,
    int32_t* __restrict__ positions, bf16_t* __restrict__ k_out, bf16_t* __restrict__ v_out,
    float* __restrict__ scores) {
  __shared__ float sc[kSnapMaxPrefix];
  __shared__ int hist[256];
  __shared__ int scan[kSelThreads];
  __shared__ int bcast[2];
  const int g = blockIdx.x, item = blockIdx.y, tid = threadIdx.x;
  const int i = sel.seq[item], l = sel.layer[item];
  const int T = st.off[i + 1] - st.off[i], row0 = st.off[i], npre = T - w;
  const int keep = sel.keep[item];
  const int64_t e0 = sel.entry0[item] + (int64_t)g * keep;
  const int64_t pre0 = (int64_t)row0 - (int64_t)i * w;
  const int64_t vbase = ((int64_t)l * n_kv + g) * prefix_rows + pre0;
  const float* vg = votes + vbase;
  kv += (int64_t)l * kv_layer_stride;
  // pooled votes
  const int r = pool_kernel >> 1;
  for (int u = tid; u < npre; u += kSelThreads) {
    const int lo = max(0, u - r), hi = min(npre - 1, u + r);
    float p = pool_avg ? 0.f : -INFINITY;
    for (int x = lo; x <= hi; ++x) p = pool_avg ? p + vg[x] : fmaxf(p, vg[x]);
    if (pool_avg) p /= (float)pool_kernel;
    sc[u] = p;
    if (scores) scores[vbase + u] = p;
  }
  __syncthreads();
  int k = keep - w;   // prefix positions to keep
  if (keep >= T) {
    for (int u = tid; u < T; u += kSelThreads) positions[e0 + u] = u;
  } else if (k <= 0) {
    for (int j = tid; j < keep; j += kSelThreads) positions[e0 + j] = T - keep + j;
  } else {
    // radix select: tau = the k-th largest pooled vote (non-negative floats order as their bits)
    uint32_t prefix = 0, mask = 0;
    int rem = k;
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int j = tid; j < 256; j += kSelThreads) hist[j] = 0;
      __syncthreads();
      for (int u = tid; u < npre; u += kSelThreads) {
        const uint32_t x = __float_as_uint(sc[u]);
        if ((x & mask) == prefix) atomicAdd(&hist[(x >> shift) & 255], 1);
      }
      __syncthreads();
      if (tid == 0) {
        int cum = 0, d = 255;
        for (; d > 0; --d) {
          if (cum + hist[d] >= rem) break;
          cum += hist[d];
        }
        bcast[0] = d;
        bcast[1] = rem - cum;
      }
      __syncthreads();
      prefix |= (uint32_t)bcast[0] << shift;
      mask |= 255u << shift;
      rem = bcast[1];
      __syncthreads();
    }
    // keep everything above tau and the first `rem` positions equal to tau
    const int seg = (npre + kSelThreads - 1) / kSelThreads;
    const int u0 = min(npre, tid * seg), u1 = min(npre, u0 + seg);
    int gt = 0, eq = 0;
    for (int u = u0; u < u1; ++u) {
      const uint32_t x = __float_as_uint(sc[u]);
      gt += x > prefix;
      eq += x == prefix;
    }
    const int eq_before = block_exclusive_scan(eq, scan);
    const int take = min(eq, max(0, rem - eq_before));
    int out = block_exclusive_scan(gt + take, scan);
    int seen = 0;
    for (int u = u0; u < u1; ++u) {
      const uint32_t x = __float_as_uint(sc[u]);
      bool keep_u = x > prefix;
      if (x == prefix) keep_u = seen++ < take;
      if (keep_u) positions[e0 + out++] = u;
    }
    for (int j = tid; j < w; j += kSelThreads) positions[e0 + k + j] = npre + j;
  }
  __syncthreads();
  // gather the retained rows' Keys and Values
  constexpr int CH = DH / 8;
  const int64_t voff = (int64_t)n_kv * DH;
  for (int idx = tid; idx < keep * CH; idx += kSelThreads) {
    const int j = idx / CH, ch = idx % CH;
    const int p = min(max(positions[e0 + j], 0), T - 1);   // always a row of this sequence
    const bf16_t* src = kv + (int64_t)(row0 + p) * ldkv + (int64_t)g * DH + ch * 8;
    *reinterpret_cast<v4u*>(k_out + (e0 + j) * DH + ch * 8) = *reinterpret_cast<const v4u*>(src);
    *reinterpret_cast<v4u*>(v_out + (e0 + j) * DH + ch * 8) = *reinterpret_cast<const v4u*>(src + voff);
  }
}

// Observation queries of the prefill: row i * w + j <- row off[i + 1] - w + j of
// the q|k|v buffer, the first qcols columns.
__global__ void snap_qobs_kernel(const bf16_t* __restrict__ qkv, int64_t ldq, SeqTable st, int w, int qcols,
                                 bf16_t* __restrict__ dst) {
  const int row = blockIdx.x, i = row / w, j = row % w;
  const int64_t src_row = (int64_t)st.off[i + 1] - w + j;
  for (int c = threadIdx.x * 8; c < qcols; c += blockDim.x * 8)
    *reinterpret_cast<v4u*>(dst + (int64_t)row * qcols + c) = *reinterpret_cast<const v4u*>(qkv + src_row * ldq + c);
}

// Layer l's prompt cache restricted to retained positions, laid out as a prompt
// cache of b rows per sequence: row i * b + j holds, for KV head g, the Key and
// Value of position pos[i * seq_stride + g * b + j] of sequence i (prompt rows
// i * P ..).  Used to evaluate the window with only that layer compressed.
__global__ void prefix_gather_kernel(const bf16_t* __restrict__ kv, int64_t ldkv, int P, int n_kv, int head_dim,
                                     const int32_t* __restrict__ pos, int64_t seq_stride, int b,
                                     bf16_t* __restrict__ out) {
  const int row = blockIdx.x, i = row / b, j = row % b;
  const int cpr = head_dim / 8;                       // 16-byte chunks per head
  for (int c = threadIdx.x; c < 2 * n_kv * cpr; c += blockDim.x) {
    const int kvh = c / cpr, g = kvh % n_kv, ch = c % cpr;   // kvh < n_kv: Keys, else Values
    const int u = min(max(pos[(int64_t)i * seq_stride + (int64_t)g * b + j], 0), P - 1);
    const int64_t col = (int64_t)kvh * head_dim + ch * 8;
    *reinterpret_cast<v4u*>(out + (int64_t)row * ldkv + col) =
        *reinterpret_cast<const v4u*>(kv + ((int64_t)i * P + u) * ldkv + col);
  }
}

// --------------------------------------------------------------------------- launchers
hipError_t launch_prefix_gather(const void* kv, int64_t ldkv, int n_seqs, int P, int n_kv, int head_dim,
                                const int32_t* pos, int64_t seq_stride, int b, void* out, hipStream_t s) {
  if (n_seqs * b == 0) return hipSuccess;
  prefix_gather_kernel<<<n_seqs * b, 128, 0, s>>>((const bf16_t*)kv, ldkv, P, n_kv, head_dim, pos, seq_stride, b,
                                                  (bf16_t*)out);
  return hipGetLastError();
}

hipError_t launch_snap_qobs(const void* qkv, int64_t ldq, const SeqTable& st, int w, int qcols, void* dst,
                            hipStream_t s) {
  snap_qobs_kernel<<<st.n * w, 128, 0, s>>>((const bf16_t*)qkv, ldq, st, w, qcols, (bf16_t*)dst);
  return hipGetLastError();
}

int snap_chunks(int max_len) { return (max_len + kSnapChunk - 1) / kSnapChunk; }

hipError_t launch_snap_scores(const void* kv, int64_t ldkv, int64_t kv_layer_stride, const void* qobs,
                              int64_t q_layer_stride, int n_layers, const SeqTable& st, int w, int n_heads, int n_kv,
                              int head_dim, float2* part, float* cnorm, float* votes, int64_t prefix_rows,
                              hipStream_t s) {
  const int nchunks = snap_chunks(st.max_len);
  const int64_t ldq = (int64_t)n_heads * head_dim;
  const int combos = (n_heads / n_kv) * ((w + 31) / 32);
  const size_t lds = qtile_bytes(head_dim, combos);
  const SnapLayers ly{kv_layer_stride, q_layer_stride};
  dim3 grid(nchunks, n_kv, st.n * n_layers);
  if (head_dim == 64)
    snap_stats_kernel<64><<<grid, 256, lds, s>>>((const bf16_t*)kv, ldkv, (const bf16_t*)qobs, ldq, st, w, n_heads,
                                                 n_kv, nchunks, ly, part);
  else if (head_dim == 128)
    snap_stats_kernel<128><<<grid, 256, lds, s>>>((const bf16_t*)kv, ldkv, (const bf16_t*)qobs, ldq, st, w, n_heads,
                                                  n_kv, nchunks, ly, part);
  else
    return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nq = n_layers * st.n * n_heads * w;
  snap_norm_kernel<<<(nq + 255) / 256, 256, 0, s>>>(part, st, w, n_heads, nchunks, n_layers, cnorm);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (head_dim == 64)
    snap_votes_kernel<64><<<grid, 256, lds, s>>>((const bf16_t*)kv, ldkv, (const bf16_t*)qobs, ldq, st, w, n_heads,
                                                 n_kv, ly, cnorm, votes, prefix_rows);
  else
    snap_votes_kernel<128><<<grid, 256, lds, s>>>((const bf16_t*)kv, ldkv, (const bf16_t*)qobs, ldq, st, w, n_heads,
                                                  n_kv, ly, cnorm, votes, prefix_rows);
  return hipGetLastError();
}

hipError_t launch_snap_select(const float* votes, int64_t prefix_rows, const void* kv, int64_t ldkv,
                              int64_t kv_layer_stride, const SeqTable& st, int w, int n_kv, int head_dim,
                              int pool_kernel, bool pool_avg, int n_items, const int16_t* seq, const int16_t* layer,
                              const int32_t* keep, const int64_t* entry0, int32_t* positions, void* k_out, void* v_out,
                              float* scores, hipStream_t s) {
  for (int first = 0; first < n_items; first += kSelItems) {
    SnapSel sel;
    sel.n = std::min(kSelItems, n_items - first);
    for (int j = 0; j < sel.n; ++j) {
      sel.seq[j] = seq[first + j];
      sel.layer[j] = layer[first + j];
      sel.keep[j] = keep[first + j];
      sel.entry0[j] = entry0[first + j];
    }
    dim3 grid(n_kv, sel.n);
    if (head_dim == 64)
      snap_select_kernel<64><<<grid, kSelThreads, 0, s>>>(votes, prefix_rows, (const bf16_t*)kv, ldkv, kv_layer_stride,
                                                          st, w, n_kv, pool_kernel, pool_avg ? 1 : 0, sel, positions,
                                                          (bf16_t*)k_out, (bf16_t*)v_out, scores);
    else if (head_dim == 128)
      snap_select_kernel<128><<<grid, kSelThreads, 0, s>>>(votes, prefix_rows, (const bf16_t*)kv, ldkv,
                                                           kv_layer_stride, st, w, n_kv, pool_kernel,
                                                           pool_avg ? 1 : 0, sel, positions, (bf16_t*)k_out,
                                                           (bf16_t*)v_out, scores);
    else
      return hipErrorInvalidValue;
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace rk
