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
//     bf16; V^T is written to LDS with the key order permuted inside each group
//     of 16 so that the matching V^T fragment is one 16-byte read;
//   * work items run heaviest (latest q-block) first.
// fp32 kernel: one thread per (row, head), streaming keys; for the small fp32
// model only.
#include <math.h>

#include "rk_internal.h"

namespace rk {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Physical position of key w (0..63) of a tile inside the transposed V tile.
__device__ __forceinline__ int vt_perm(int key) {
  const int grp = key >> 4, w = key & 15;
  const int a = w >> 3, hh = (w >> 2) & 1, j = w & 3;
  return grp * 16 + hh * 8 + a * 4 + j;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)f2bf(lo) | ((uint32_t)f2bf(hi) << 16);
}

template <int DH>
__global__ __launch_bounds__(256) void attn_bf16_kernel(const bf16_t* __restrict__ qkv, int64_t ldq,
                                                        bf16_t* __restrict__ out, int64_t ldo, SeqTable st,
                                                        AttnWork wk, int H, int Hkv, float scale_log2) {
  constexpr int BQ = 128, BKV = 64;
  constexpr int KCH = DH / 8;               // 16-byte chunks per K row
  constexpr int NKS = DH / 16;              // k-steps of S^T
  constexpr int NDB = DH / 32;              // 32-row blocks of O^T
  constexpr int NLD = BKV * KCH / 256;      // K (and V) chunks loaded per thread
  __shared__ __attribute__((aligned(16))) v4u Ks[2][BKV * KCH];
  __shared__ __attribute__((aligned(16))) v4u Vt[2][DH * 8];

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

  v4u rk[NLD], rv[NLD];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int c = tid + 256 * i, key = c / KCH, ch = c % KCH;
      const int64_t r = row0 + min(k0 + key, T - 1);
      rk[i] = *reinterpret_cast<const v4u*>(qkv + r * ldq + kcol + ch * 8);
      rv[i] = *reinterpret_cast<const v4u*>(qkv + r * ldq + vcol + ch * 8);
    }
  };
  auto lstore = [&](int b) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int c = tid + 256 * i, key = c / KCH, ch = c % KCH;
      Ks[b][key * KCH + (ch ^ (key & 7))] = rk[i];
      const int pk = vt_perm(key);
      bf16_t* vt = reinterpret_cast<bf16_t*>(Vt[b]);
      const uint32_t words[4] = {rv[i].x, rv[i].y, rv[i].z, rv[i].w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int dd = ch * 8 + e;
        const bf16_t val = (bf16_t)((e & 1) ? (words[e >> 1] >> 16) : (words[e >> 1] & 0xffffu));
        vt[(dd * 8 + ((pk >> 3) ^ (dd & 7))) * 8 + (pk & 7)] = val;
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
  const int wave_qmax = q0 + w * 32 + 31;
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
      float mx = -INFINITY;
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = k0 + rb * 32 + (i >> 2) * 8 + hf * 4 + (i & 3);
          float v = s[rb][i] * scale_log2;
          if (key > my_q || key >= T) v = -INFINITY;
          s[rb][i] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);
      const float corr = exp2f(m_run - m_new);
      float rs = 0.f;
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float p = exp2f(s[rb][i] - m_new);
          s[rb][i] = p;
          rs += p;
        }
      l_run = l_run * corr + rs;
      m_run = m_new;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[db][i] *= corr;
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int ss = 0; ss < 2; ++ss) {
          v4u pw;
          pw.x = pack_bf16x2(s[rb][8 * ss + 0], s[rb][8 * ss + 1]);
          pw.y = pack_bf16x2(s[rb][8 * ss + 2], s[rb][8 * ss + 3]);
          pw.z = pack_bf16x2(s[rb][8 * ss + 4], s[rb][8 * ss + 5]);
          pw.w = pack_bf16x2(s[rb][8 * ss + 6], s[rb][8 * ss + 7]);
          const bf16x8_t pb = __builtin_bit_cast(bf16x8_t, pw);
          const int ch = rb * 4 + 2 * ss + hf;
#pragma unroll
          for (int db = 0; db < NDB; ++db) {
            const int dd = db * 32 + l32;
            const bf16x8_t va = __builtin_bit_cast(bf16x8_t, Vt[buf][dd * 8 + (ch ^ (dd & 7))]);
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[db], 0, 0, 0);
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
        uint2 u;
        u.x = pack_bf16x2(o[db][g * 4 + 0] * inv, o[db][g * 4 + 1] * inv);
        u.y = pack_bf16x2(o[db][g * 4 + 2] * inv, o[db][g * 4 + 3] * inv);
        *reinterpret_cast<uint2*>(op + db * 32 + g * 8 + hf * 4) = u;
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
    const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)head_dim));
    dim3 grid(wk.total, n_heads);
    if (head_dim == 128)
      attn_bf16_kernel<128><<<grid, 256, 0, s>>>((const bf16_t*)qkv, ldq, (bf16_t*)out, ldo, st, wk, n_heads,
                                                 n_kv_heads, scale_log2);
    else if (head_dim == 64)
      attn_bf16_kernel<64><<<grid, 256, 0, s>>>((const bf16_t*)qkv, ldq, (bf16_t*)out, ldo, st, wk, n_heads,
                                                n_kv_heads, scale_log2);
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
