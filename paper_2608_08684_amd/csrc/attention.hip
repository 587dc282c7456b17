// Causal grouped-query attention of one decoder block (Section 4.1), reading the
// (possibly perturbed) Values of the q|k|v buffer: o = softmax(q k^T / sqrt(d_h)) v
// with key u visible from query t iff u <= t; query head hq reads KV head
// hq / (H / H_kv).  With the Keys fixed the attention weights of the perturbed
// layer equal the clean ones (Section 4.3); only the aggregated Values change.
//
// bf16 kernel (flash attention, fp32 online softmax):
//   * one workgroup = 128 queries of one head (4 waves x 32 queries), keys in
//     tiles of 64 staged in LDS (K row-major, V transposed), double-buffered;
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16, so each lane owns one query
//     column: the row max and row sum of the softmax are lane-local plus one
//     exchange with the partner half-wave;
//   * O^T = V^T P^T: the P^T operand is the lane's own S^T registers rounded to
//     bf16 (keys 4h..4h+3 and 8+4h..8+4h+3 of each 16-key step); V^T is written
//     to LDS as key pairs and read as two 8-byte pieces that match those keys;
//   * masks only on diagonal / ragged tiles; the softmax scale is folded into
//     one FMA before exp2; the running max is raised lazily (rescaling O only
//     when a tile's max grows by more than 2^8);
//   * work items run heaviest (latest q-block) first.
// fp32 kernel: one thread per (row, head), streaming keys; for the small fp32
// model only.
#include <math.h>

#include "rk_internal.h"

namespace rk {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));

// Raw scores are kept unscaled; p = 2^((s - m) * c) with c = log2(e) / sqrt(d_h).
// The running max m is only raised when a tile's max exceeds it by more than
// kLazy / c (2^8 headroom in P), so most tiles skip the rescale of O and l.
constexpr float kLazyLog2 = 8.0f;

// XOR swizzle of the 16-byte chunks of V^T row dd: lanes that write one element of
// eight rows dd = 8 c + e (c = 0..7) and lanes that read eight consecutive rows both
// land on distinct chunks.
__device__ __forceinline__ int vsw(int dd) { return (dd ^ (dd >> 3)) & 7; }

template <int DH>
__global__ __launch_bounds__(256) void attn_bf16_kernel(const bf16_t* __restrict__ qkv, int64_t ldq,
                                                        bf16_t* __restrict__ out, int64_t ldo, SeqTable st,
                                                        AttnWork wk, int H, int Hkv, float c_log2) {
  constexpr int BQ = 128, BKV = 64;
  constexpr int KCH = DH / 8;               // 16-byte chunks per K row
  constexpr int NKS = DH / 16;              // k-steps of S^T
  constexpr int NDB = DH / 32;              // 32-row blocks of O^T
  constexpr int NLK = BKV * KCH / 256;      // K chunks loaded per thread
  constexpr int NLV = BKV * KCH / 512;      // V key-pair chunks loaded per thread
  __shared__ __attribute__((aligned(16))) v4u Ks[2][BKV * KCH];
  __shared__ __attribute__((aligned(16))) v4u Vt[2][DH * 8];   // [d][64 keys], 16-byte chunks XOR-swizzled (vsw)

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l32 = lane & 31, hf = lane >> 5;
  const int item = wk.total - 1 - (int)blockIdx.x;
  int k = 0;
  {
    int lo = 0, hi = st.n - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (wk.cum[mid] <= item) lo = mid; else hi = mid - 1;
    }
    k = lo;
  }
  const int qb = item - wk.cum[k];
  const int row0 = st.off[k], T = st.off[k + 1] - row0;
  const int q0 = qb * BQ;
  const int hq = blockIdx.y, hk = hq / (H / Hkv);
  const int64_t kcol = (int64_t)H * DH + (int64_t)hk * DH;
  const int64_t vcol = (int64_t)(H + Hkv) * DH + (int64_t)hk * DH;
  const int my_q = q0 + w * 32 + l32;

  bf16x8_t qf[NKS];
  {
    const bf16_t* qp = qkv + (int64_t)(row0 + min(my_q, T - 1)) * ldq + (int64_t)hq * DH + hf * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) qf[ks] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const v4u*>(qp + ks * 16));
  }

  const int kv_end = min(T, q0 + BQ);
  const int n_tiles = (kv_end + BKV - 1) / BKV;

  v4u rk[NLK], rv[2 * NLV];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < NLK; ++i) {
      const int c = tid + 256 * i, key = c / KCH, ch = c % KCH;
      const int64_t r = row0 + min(k0 + key, T - 1);
      rk[i] = *reinterpret_cast<const v4u*>(qkv + r * ldq + kcol + ch * 8);
    }
#pragma unroll
    for (int i = 0; i < NLV; ++i) {
      const int c = tid + 256 * i, kp = c / KCH, ch = c % KCH;   // key pair kp: keys 2kp, 2kp+1
      const int64_t r0 = row0 + min(k0 + 2 * kp, T - 1), r1 = row0 + min(k0 + 2 * kp + 1, T - 1);
      rv[2 * i] = *reinterpret_cast<const v4u*>(qkv + r0 * ldq + vcol + ch * 8);
      rv[2 * i + 1] = *reinterpret_cast<const v4u*>(qkv + r1 * ldq + vcol + ch * 8);
    }
  };
  auto lstore = [&](int b) {
#pragma unroll
    for (int i = 0; i < NLK; ++i) {
      const int c = tid + 256 * i, key = c / KCH, ch = c % KCH;
      Ks[b][key * KCH + (ch ^ (key & 7))] = rk[i];
    }
    uint32_t* vt = reinterpret_cast<uint32_t*>(Vt[b]);
#pragma unroll
    for (int i = 0; i < NLV; ++i) {
      const int c = tid + 256 * i, kp = c / KCH, ch = c % KCH;
      const int key = 2 * kp;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int dd = ch * 8 + e;
        const uint32_t lo = (rv[2 * i][e >> 1] >> ((e & 1) * 16)) & 0xffffu;
        const uint32_t hi = (rv[2 * i + 1][e >> 1] >> ((e & 1) * 16)) & 0xffffu;
        // word index: row dd (32 words), chunk key/8 swizzled, word (key%8)/2 inside the chunk
        vt[dd * 32 + (((key >> 3) ^ vsw(dd)) << 2) + ((key & 7) >> 1)] = lo | (hi << 16);
      }
    }
  };

  float m_run = -INFINITY, l_run = 0.f;
  f32x16_t o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[db][i] = 0.f;

  gload(0);
  lstore(0);
  __syncthreads();
  const int wave_qmin = q0 + w * 32, wave_qmax = wave_qmin + 31;
  const float lazy = kLazyLog2 / c_log2;
  for (int t = 0; t < n_tiles; ++t) {
    const int buf = t & 1, k0 = t * BKV;
    if (t + 1 < n_tiles) gload(k0 + BKV);
    if (k0 <= wave_qmax) {
      f32x16_t s[2];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) s[rb][i] = 0.f;
        const int key = rb * 32 + l32;
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
          const bf16x8_t a = __builtin_bit_cast(bf16x8_t, Ks[buf][key * KCH + ((2 * ks + hf) ^ (key & 7))]);
          s[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s[rb], 0, 0, 0);
        }
      }
      // masks only where a key can exceed the query or the sequence (wave-uniform test)
      if (k0 + BKV - 1 > wave_qmin || k0 + BKV > T) {
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = k0 + rb * 32 + (i >> 2) * 8 + hf * 4 + (i & 3);
            if (key > my_q || key >= T) s[rb][i] = -INFINITY;
          }
      }
      float mx = s[0][0];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[rb][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      if (__any(mx > m_run + lazy)) {
        const float m_new = fmaxf(m_run, mx);
        const float corr = __builtin_amdgcn_exp2f((m_run - m_new) * c_log2);
        l_run *= corr;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int i = 0; i < 16; ++i) o[db][i] *= corr;
        m_run = m_new;
      }
      const float mc = m_run * c_log2;
      float rs = 0.f;
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s[rb][i], c_log2, -mc));
          s[rb][i] = p;
          rs += p;
        }
      l_run += rs;
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int ss = 0; ss < 2; ++ss) {
          bf16x8_t pb;
#pragma unroll
          for (int e = 0; e < 8; ++e) pb[e] = (__bf16)s[rb][8 * ss + e];
          // this lane's k-slots: keys 16*(2rb+ss) + 4hf + {0..3} and the same + 8
          const int kb = rb * 32 + ss * 16 + hf * 4;
#pragma unroll
          for (int db = 0; db < NDB; ++db) {
            const int dd = db * 32 + l32;
            const v2u* row = reinterpret_cast<const v2u*>(Vt[buf]) + dd * 16;
            const v2u lo = row[(((kb >> 3) ^ vsw(dd)) << 1) + ((kb & 7) >> 2)];
            const v2u hi = row[((((kb + 8) >> 3) ^ vsw(dd)) << 1) + ((kb & 7) >> 2)];
            const v4u vv = {lo[0], lo[1], hi[0], hi[1]};
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, vv), pb, o[db], 0, 0, 0);
          }
        }
    }
    if (t + 1 < n_tiles) lstore(buf ^ 1);
    __syncthreads();
  }

  const float l = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l;
  if (my_q < T) {
    bf16_t* op = out + (int64_t)(row0 + my_q) * ldo + (int64_t)hq * DH;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4_t u;
#pragma unroll
        for (int e = 0; e < 4; ++e) u[e] = (__bf16)(o[db][g * 4 + e] * inv);
        *reinterpret_cast<bf16x4_t*>(op + db * 32 + g * 8 + hf * 4) = u;
      }
  }
}

template <int DH>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ qkv, int64_t ldq,
                                                      float* __restrict__ out, int64_t ldo, SeqTable st, int H,
                                                      int Hkv, float scale) {
  const int r = blockIdx.x * 64 + threadIdx.x;
  if (r >= st.rows) return;
  const int hq = blockIdx.y, hk = hq / (H / Hkv);
  const int k = seq_of_row(st, r), row0 = st.off[k], q = r - row0;
  float qv[DH], acc[DH];
  const float* qp = qkv + (int64_t)r * ldq + (int64_t)hq * DH;
#pragma unroll
  for (int j = 0; j < DH; ++j) { qv[j] = qp[j]; acc[j] = 0.f; }
  float m = -INFINITY, l = 0.f;
  for (int u = 0; u <= q; ++u) {
    const float* kp = qkv + (int64_t)(row0 + u) * ldq + (int64_t)H * DH + (int64_t)hk * DH;
    const float* vp = qkv + (int64_t)(row0 + u) * ldq + (int64_t)(H + Hkv) * DH + (int64_t)hk * DH;
    float sdot = 0.f;
#pragma unroll
    for (int j = 0; j < DH; ++j) sdot = fmaf(qv[j], kp[j], sdot);
    sdot *= scale;
    const float m_new = fmaxf(m, sdot);
    const float corr = expf(m - m_new), p = expf(sdot - m_new);
    l = l * corr + p;
#pragma unroll
    for (int j = 0; j < DH; ++j) acc[j] = fmaf(p, vp[j], acc[j] * corr);
    m = m_new;
  }
  float* op = out + (int64_t)r * ldo + (int64_t)hq * DH;
  const float inv = 1.0f / l;
#pragma unroll
  for (int j = 0; j < DH; ++j) op[j] = acc[j] * inv;
}

hipError_t launch_attention(const void* qkv, int64_t ldq, void* out, int64_t ldo, const SeqTable& st, int n_heads,
                            int n_kv_heads, int head_dim, bool bf16, hipStream_t s) {
  if (st.rows <= 0) return hipSuccess;
  if (bf16) {
    AttnWork wk;
    wk.cum[0] = 0;
    for (int k = 0; k < st.n; ++k) wk.cum[k + 1] = wk.cum[k] + (st.off[k + 1] - st.off[k] + 127) / 128;
    wk.total = wk.cum[st.n];
    if (wk.total == 0) return hipSuccess;
    const float c_log2 = (float)(1.4426950408889634 / sqrt((double)head_dim));
    dim3 grid(wk.total, n_heads);
    if (head_dim == 128)
      attn_bf16_kernel<128><<<grid, 256, 0, s>>>((const bf16_t*)qkv, ldq, (bf16_t*)out, ldo, st, wk, n_heads,
                                                 n_kv_heads, c_log2);
    else if (head_dim == 64)
      attn_bf16_kernel<64><<<grid, 256, 0, s>>>((const bf16_t*)qkv, ldq, (bf16_t*)out, ldo, st, wk, n_heads,
                                                n_kv_heads, c_log2);
    else
      return hipErrorInvalidValue;
  } else {
    const float scale = (float)(1.0 / sqrt((double)head_dim));
    dim3 grid((st.rows + 63) / 64, n_heads);
    if (head_dim == 32)
      attn_f32_kernel<32><<<grid, 64, 0, s>>>((const float*)qkv, ldq, (float*)out, ldo, st, n_heads, n_kv_heads, scale);
    else if (head_dim == 64)
      attn_f32_kernel<64><<<grid, 64, 0, s>>>((const float*)qkv, ldq, (float*)out, ldo, st, n_heads, n_kv_heads, scale);
    else if (head_dim == 128)
      attn_f32_kernel<128><<<grid, 64, 0, s>>>((const float*)qkv, ldq, (float*)out, ldo, st, n_heads, n_kv_heads, scale);
    else
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace rk
