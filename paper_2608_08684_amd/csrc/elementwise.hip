// HBM-bound kernels of the profiling path: embedding gather, RMSNorm, the rotary
// table, the norm-adaptive Value noise (Eq. value-perturbation) and the window /
// calibration means (Eqs. sample-response and layer-sensitivity).
#include <algorithm>

#include "rk_internal.h"

namespace rk {

// --------------------------------------------------------------------------- embedding
template <typename E>
__global__ void embed_kernel(const E* __restrict__ emb, const int32_t* __restrict__ tok, float* __restrict__ h,
                             int rows, int d) {
  const int64_t total = (int64_t)rows * d;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / d, c = i - r * d;
    h[i] = Act<E>::load(emb + (int64_t)tok[r] * d + c);
  }
}

hipError_t launch_embed(const void* emb, bool emb_bf16, const int32_t* tokens, float* h, int rows, int d,
                        hipStream_t s) {
  const int64_t total = (int64_t)rows * d;
  int blocks = (int)((total + 255) / 256);
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  if (emb_bf16)
    embed_kernel<bf16_t><<<blocks, 256, 0, s>>>((const bf16_t*)emb, tokens, h, rows, d);
  else
    embed_kernel<float><<<blocks, 256, 0, s>>>((const float*)emb, tokens, h, rows, d);
  return hipGetLastError();
}

// Row r of table dst (sequence k, local index j) takes token src.off[k] + pos0 + j.
template <typename E>
__global__ void embed_gather_kernel(const E* __restrict__ emb, const int32_t* __restrict__ tok, SeqTable src,
                                    SeqTable dst, int pos0, float* __restrict__ h, int d) {
  for (int r = blockIdx.x; r < dst.rows; r += gridDim.x) {
    const int k = seq_of_row(dst, r);
    const int64_t t = tok[src.off[k] + pos0 + (r - dst.off[k])];
    for (int c = threadIdx.x; c < d; c += blockDim.x) h[(int64_t)r * d + c] = Act<E>::load(emb + t * d + c);
  }
}

hipError_t launch_embed_gather(const void* emb, bool emb_bf16, const int32_t* tokens, const SeqTable& src,
                               const SeqTable& dst, int pos0, float* h, int d, hipStream_t s) {
  if (dst.rows <= 0) return hipSuccess;
  const int blocks = std::min(dst.rows, 65536);
  if (emb_bf16)
    embed_gather_kernel<bf16_t><<<blocks, 256, 0, s>>>((const bf16_t*)emb, tokens, src, dst, pos0, h, d);
  else
    embed_gather_kernel<float><<<blocks, 256, 0, s>>>((const float*)emb, tokens, src, dst, pos0, h, d);
  return hipGetLastError();
}

// dst[r][0 .. nbytes) = src[r][off .. off + nbytes), rows of ld_src / ld_dst bytes;
// all byte counts multiples of 16.
__global__ void copy_cols_kernel(const char* __restrict__ src, int64_t ld_src, int64_t off, char* __restrict__ dst,
                                 int64_t ld_dst, int nvec, int rows) {
  const int64_t total = (int64_t)rows * nvec;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / nvec, c = i - r * nvec;
    reinterpret_cast<v4u*>(dst + r * ld_dst)[c] = reinterpret_cast<const v4u*>(src + r * ld_src + off)[c];
  }
}

hipError_t launch_copy_cols(const void* src, int64_t ld_src_bytes, int64_t off_bytes, void* dst, int64_t ld_dst_bytes,
                            int64_t nbytes, int rows, hipStream_t s) {
  if (rows <= 0 || nbytes <= 0) return hipSuccess;
  if ((ld_src_bytes | off_bytes | ld_dst_bytes | nbytes) & 15) return hipErrorInvalidValue;
  const int nvec = (int)(nbytes / 16);
  const int64_t total = (int64_t)rows * nvec;
  int blocks = (int)std::min<int64_t>((total + 255) / 256, 16384);
  copy_cols_kernel<<<blocks, 256, 0, s>>>((const char*)src, ld_src_bytes, off_bytes, (char*)dst, ld_dst_bytes, nvec,
                                          rows);
  return hipGetLastError();
}

// --------------------------------------------------------------------------- RMSNorm
// One wave per row: out = h / sqrt(mean(h^2) + eps) * g.  fp32 in, act out.  With
// NV > 0 the row stays in registers (NV float4 per lane) between the sum of
// squares and the scaled store, and each lane writes its four outputs with one
// 16-byte (fp32) or 8-byte (bf16) store; NV = 0 streams the row twice (any d).
__device__ __forceinline__ void store4v(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
__device__ __forceinline__ void store4v(bf16_t* p, float a, float b, float c, float d) {
  uint2 u;
  u.x = (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
  u.y = (uint32_t)f2bf(c) | ((uint32_t)f2bf(d) << 16);
  *reinterpret_cast<uint2*>(p) = u;
}

template <typename O, int NV>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ h, const float* __restrict__ g,
                                                      O* __restrict__ out, int rows, int d, float eps) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const float4* hr = reinterpret_cast<const float4*>(h + (int64_t)row * d);
  const float4* g4 = reinterpret_cast<const float4*>(g);
  O* orow = out + (int64_t)row * d;
  const int n4 = d >> 2;
  float ss = 0.f;
  if constexpr (NV > 0) {
    float4 v[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int i = lane + 64 * j;
      v[j] = i < n4 ? hr[i] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int j = 0; j < NV; ++j) ss += v[j].x * v[j].x + v[j].y * v[j].y + v[j].z * v[j].z + v[j].w * v[j].w;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int i = lane + 64 * j;
      if (i < n4) {
        const float4 w = g4[i];
        store4v(orow + 4 * i, v[j].x * inv * w.x, v[j].y * inv * w.y, v[j].z * inv * w.z, v[j].w * inv * w.w);
      }
    }
  } else {
    for (int i = lane; i < n4; i += 64) {
      const float4 v = hr[i];
      ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
    const float inv = 1.0f / sqrtf(ss / (float)d + eps);
    for (int i = lane; i < n4; i += 64) {
      const float4 v = hr[i], w = g4[i];
      store4v(orow + 4 * i, v.x * inv * w.x, v.y * inv * w.y, v.z * inv * w.z, v.w * inv * w.w);
    }
  }
}

template <typename O>
static void rmsnorm_go(const float* h, const float* g, O* out, int rows, int d, float eps, hipStream_t s) {
  const int blocks = (rows + 3) / 4;
  const int nv = (d / 4 + 63) / 64;   // float4 per lane
  switch (nv) {
    case 1: rmsnorm_kernel<O, 1><<<blocks, 256, 0, s>>>(h, g, out, rows, d, eps); break;
    case 2: rmsnorm_kernel<O, 2><<<blocks, 256, 0, s>>>(h, g, out, rows, d, eps); break;
    case 3: rmsnorm_kernel<O, 3><<<blocks, 256, 0, s>>>(h, g, out, rows, d, eps); break;
    case 4: rmsnorm_kernel<O, 4><<<blocks, 256, 0, s>>>(h, g, out, rows, d, eps); break;
    case 5: case 6: rmsnorm_kernel<O, 6><<<blocks, 256, 0, s>>>(h, g, out, rows, d, eps); break;
    case 7: case 8: rmsnorm_kernel<O, 8><<<blocks, 256, 0, s>>>(h, g, out, rows, d, eps); break;
    case 9: case 10: case 11: case 12: rmsnorm_kernel<O, 12><<<blocks, 256, 0, s>>>(h, g, out, rows, d, eps); break;
    case 13: case 14: case 15: case 16: rmsnorm_kernel<O, 16><<<blocks, 256, 0, s>>>(h, g, out, rows, d, eps); break;
    default: rmsnorm_kernel<O, 0><<<blocks, 256, 0, s>>>(h, g, out, rows, d, eps); break;
  }
}

hipError_t launch_rmsnorm(const float* h, const float* g, void* out, bool out_bf16, int rows, int d, float eps,
                          hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d & 3) return hipErrorInvalidValue;
  if (out_bf16)
    rmsnorm_go<bf16_t>(h, g, (bf16_t*)out, rows, d, eps, s);
  else
    rmsnorm_go<float>(h, g, (float*)out, rows, d, eps, s);
  return hipGetLastError();
}

// --------------------------------------------------------------------------- layer-local response
// The layer-local signal of the "w/o DS" ablation: r[row] = ||hp - hc||^2 / ||hc||^2
// for the perturbed and clean outputs of one block (fp32 rows of d values), 0 for a
// zero clean row.  One wave per row; each lane sums its float4 columns in order,
// then a fixed butterfly combines the lanes, so the result is repeatable.
__global__ __launch_bounds__(256) void local_response_kernel(const float* __restrict__ hp,
                                                             const float* __restrict__ hc, int rows, int d,
                                                             float* __restrict__ r) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const float4* a = reinterpret_cast<const float4*>(hp + (int64_t)row * d);
  const float4* c = reinterpret_cast<const float4*>(hc + (int64_t)row * d);
  const int n4 = d >> 2;
  float num = 0.f, den = 0.f;
  for (int i = lane; i < n4; i += 64) {
    const float4 x = a[i], y = c[i];
    const float e0 = x.x - y.x, e1 = x.y - y.y, e2 = x.z - y.z, e3 = x.w - y.w;
    num += e0 * e0 + e1 * e1 + e2 * e2 + e3 * e3;
    den += y.x * y.x + y.y * y.y + y.z * y.z + y.w * y.w;
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    num += __shfl_xor(num, m, 64);
    den += __shfl_xor(den, m, 64);
  }
  if (lane == 0) r[row] = den > 0.f ? num / den : 0.f;
}

hipError_t launch_local_response(const float* hp, const float* hc, int rows, int d, float* r, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  if (d & 3) return hipErrorInvalidValue;
  local_response_kernel<<<(rows + 3) / 4, 256, 0, s>>>(hp, hc, rows, d, r);
  return hipGetLastError();
}

// --------------------------------------------------------------------------- rotary table
// tab[t * (dh/2) + j] = (cos, sin)(t * theta^(-2j/dh)) for t < max_len; the angle is
// formed and reduced modulo 2*pi in double precision before the fp32 rounding.
// pos[r] = position of row r inside its sequence.
__global__ void rope_table_kernel(float2* tab, int32_t* pos, SeqTable st, int half, int dh, double log2_theta,
                                  int pos0) {
  const int64_t total = (int64_t)(pos0 + st.max_len) * half;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int t = (int)(i / half), j = (int)(i - (int64_t)t * half);
    const double inv_freq = exp2(-(2.0 * j / dh) * log2_theta);
    double ang = (double)t * inv_freq;
    const double two_pi = 6.283185307179586476925;
    ang -= two_pi * floor(ang / two_pi);
    double sv, cv;
    sincos(ang, &sv, &cv);
    tab[i] = make_float2((float)cv, (float)sv);
  }
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < st.rows; r += stride)
    pos[r] = (int32_t)(pos0 + r - st.off[seq_of_row(st, (int)r)]);
}

hipError_t launch_rope_table(float2* tab, int32_t* pos, const SeqTable& st, int head_dim, float theta, hipStream_t s,
                             int pos0) {
  const int half = head_dim / 2;
  const int64_t total = std::max((int64_t)(pos0 + st.max_len) * half, (int64_t)st.rows);
  int blocks = (int)((total + 255) / 256);
  if (blocks > 16384) blocks = 16384;
  if (blocks < 1) blocks = 1;
  rope_table_kernel<<<blocks, 256, 0, s>>>(tab, pos, st, half, head_dim, log2((double)theta), pos0);
  return hipGetLastError();
}

// --------------------------------------------------------------------------- Value noise
// Philox4x32-10 (Salmon et al., SC'11): counter (c0..c3), key (k0, k1), ten rounds.
__device__ __forceinline__ void philox10(uint32_t& c0, uint32_t& c1, uint32_t& c2, uint32_t& c3, uint32_t k0,
                                         uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    // one 32 x 32 -> 64-bit product per multiplier (v_mad_u64_u32) gives both halves
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t lo0 = (uint32_t)p0, hi0 = (uint32_t)(p0 >> 32);
    const uint32_t lo1 = (uint32_t)p1, hi1 = (uint32_t)(p1 >> 32);
    const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;
  }
}

// 32-bit word -> uniform in (0, 1): (2 * (x >> 9) + 1) * 2^-24, exact in fp32.
__device__ __forceinline__ float to_uniform(uint32_t x) {
  return (float)(2u * (x >> 9) + 1u) * 5.9604644775390625e-8f;
}

// Four consecutive values as one 16-byte (fp32) or 8-byte (bf16) access.
__device__ __forceinline__ void load4v(const float* p, float& a, float& b, float& c, float& d) {
  const float4 v = *reinterpret_cast<const float4*>(p);
  a = v.x; b = v.y; c = v.z; d = v.w;
}
__device__ __forceinline__ void load4v(const bf16_t* p, float& a, float& b, float& c, float& d) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  a = __uint_as_float(u.x << 16); b = __uint_as_float(u.x & 0xffff0000u);
  c = __uint_as_float(u.y << 16); d = __uint_as_float(u.y & 0xffff0000u);
}

// One thread owns four consecutive coordinates j = 4g..4g+3 of one (row, KV head)
// Value vector; TPV = head_dim / 4 threads cooperate on the vector's norm.
template <typename T, int TPV>
__global__ __launch_bounds__(256) void value_noise_kernel(T* __restrict__ v, int64_t row_stride, SeqTable st,
                                                          int n_kv_heads, int layer, float alpha, uint32_t key0,
                                                          uint32_t key1, int protect_head, int protect_tail) {
  constexpr int VPB = 256 / TPV;  // vectors per block
  const int sub = threadIdx.x % TPV;
  const int64_t vec = (int64_t)blockIdx.x * VPB + threadIdx.x / TPV;
  const int64_t n_vec = (int64_t)st.rows * n_kv_heads;
  const bool live = vec < n_vec;
  const int row = live ? (int)(vec / n_kv_heads) : 0;
  const int head = live ? (int)(vec - (int64_t)row * n_kv_heads) : 0;
  const int k = seq_of_row(st, row);
  const int u = row - st.off[k];
  const int len = st.off[k + 1] - st.off[k];
  T* p = v + (int64_t)row * row_stride + (int64_t)head * (TPV * 4) + sub * 4;
  float x0 = 0.f, x1 = 0.f, x2 = 0.f, x3 = 0.f;
  if (live) load4v(p, x0, x1, x2, x3);
  float ss = x0 * x0 + x1 * x1 + x2 * x2 + x3 * x3;
#pragma unroll
  for (int m = TPV / 2; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
  const bool eligible = live && u >= protect_head && u < len - protect_tail;
  if (!eligible) return;
  const float an = alpha * sqrtf(ss);
  uint32_t c0 = (uint32_t)u, c1 = (uint32_t)sub | ((uint32_t)head << 16), c2 = (uint32_t)layer,
           c3 = (uint32_t)(st.seq_index0 + k);
  philox10(c0, c1, c2, c3, key0, key1);
  const float r0 = sqrtf(-2.0f * logf(to_uniform(c0)));
  const float r1 = sqrtf(-2.0f * logf(to_uniform(c2)));
  float s0, co0, s1, co1;
  sincospif(2.0f * to_uniform(c1), &s0, &co0);
  sincospif(2.0f * to_uniform(c3), &s1, &co1);
  store4v(p, fmaf(an, r0 * co0, x0), fmaf(an, r0 * s0, x1), fmaf(an, r1 * co1, x2), fmaf(an, r1 * s1, x3));
}

template <typename T>
static hipError_t noise_dispatch(T* v, int64_t row_stride, const SeqTable& st, int hkv, int dh, int layer,
                                 float alpha, uint64_t seed, int ph, int pt, hipStream_t s) {
  const int64_t n_vec = (int64_t)st.rows * hkv;
  const uint32_t k0 = (uint32_t)(seed & 0xffffffffu), k1 = (uint32_t)(seed >> 32);
  const int tpv = dh / 4;
  const int64_t blocks = (n_vec * tpv + 255) / 256;
  if (blocks <= 0) return hipSuccess;
  switch (tpv) {
    case 8:  value_noise_kernel<T, 8><<<(unsigned)blocks, 256, 0, s>>>(v, row_stride, st, hkv, layer, alpha, k0, k1, ph, pt); break;
    case 16: value_noise_kernel<T, 16><<<(unsigned)blocks, 256, 0, s>>>(v, row_stride, st, hkv, layer, alpha, k0, k1, ph, pt); break;
    case 32: value_noise_kernel<T, 32><<<(unsigned)blocks, 256, 0, s>>>(v, row_stride, st, hkv, layer, alpha, k0, k1, ph, pt); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_value_noise(void* v, bool bf16, int64_t row_stride, const SeqTable& st, int n_kv_heads,
                              int head_dim, int layer, float alpha, uint64_t seed, int protect_head,
                              int protect_tail, hipStream_t s) {
  if (bf16)
    return noise_dispatch<bf16_t>((bf16_t*)v, row_stride, st, n_kv_heads, head_dim, layer, alpha, seed,
                                  protect_head, protect_tail, s);
  return noise_dispatch<float>((float*)v, row_stride, st, n_kv_heads, head_dim, layer, alpha, seed, protect_head,
                               protect_tail, s);
}

// --------------------------------------------------------------------------- state tag
// The identity record of a clean or window state: {magic, host identity, token
// digest, rows}.  The digest is a wrapping sum over positions i of
// splitmix64((i << 32) | token_i) (the splitmix64 finaliser of Steele, Lea and
// Flood), so it depends on every token and its position and not on the order of
// the summation.
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__global__ __launch_bounds__(256) void state_tag_kernel(const int32_t* __restrict__ tok, int64_t rows,
                                                        uint64_t magic, uint64_t host, uint64_t* __restrict__ out) {
  __shared__ uint64_t part[256];
  uint64_t acc = 0;
  for (int64_t i = threadIdx.x; i < rows; i += 256) acc += mix64(((uint64_t)i << 32) | (uint32_t)tok[i]);
  part[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x < 4) {
    const uint64_t v[4] = {magic, host, part[0], (uint64_t)rows};
    out[threadIdx.x] = v[threadIdx.x];
  }
}

hipError_t launch_state_tag(const int32_t* tokens, int64_t rows, uint64_t magic, uint64_t host, uint64_t* out,
                            hipStream_t s) {
  state_tag_kernel<<<1, 256, 0, s>>>(tokens, rows, magic, host, out);
  return hipGetLastError();
}

// --------------------------------------------------------------------------- means
// d[g * n + k] = mean of kl[g * kl_stride + r] for r in [off[k] + window_start, off[k+1]);
// 0 for an empty window.  Fixed-order double accumulation.
__global__ __launch_bounds__(256) void window_mean_kernel(const float* __restrict__ kl, int64_t kl_stride,
                                                          SeqTable st, int window_start, float* __restrict__ d) {
  const int k = blockIdx.x, g = blockIdx.y;
  const int r0 = st.off[k] + window_start, r1 = st.off[k + 1];
  __shared__ double part[256];
  double acc = 0.0;
  for (int r = r0 + (int)threadIdx.x; r < r1; r += 256) acc += (double)kl[(int64_t)g * kl_stride + r];
  part[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) d[g * st.n + k] = r1 > r0 ? (float)(part[0] / (double)(r1 - r0)) : 0.0f;
}

hipError_t launch_window_mean(const float* kl, int64_t kl_stride, int G, const SeqTable& st, int window_start,
                              float* d, hipStream_t s) {
  window_mean_kernel<<<dim3(st.n, G), 256, 0, s>>>(kl, kl_stride, st, window_start, d);
  return hipGetLastError();
}

// One thread per pass of the group: copies the batch's d values to the caller's
// d matrix and adds their sum (in sequence order) to the profile accumulator.
__global__ void accumulate_kernel(const float* __restrict__ dbatch, int n_seqs, PassMap pm, float* __restrict__ d_out,
                                  double* __restrict__ s_acc) {
  const int g = threadIdx.x;
  if (g >= pm.G) return;
  double acc = 0.0;
  for (int k = 0; k < n_seqs; ++k) {
    const float x = dbatch[g * n_seqs + k];
    acc += (double)x;
    if (d_out) d_out[pm.d_base[g] + (int64_t)(pm.seq_index0 + k) * pm.d_seq_stride] = x;
  }
  s_acc[pm.s_index[g]] += acc;
}

hipError_t launch_accumulate(const float* dbatch, int n_seqs, const PassMap& pm, float* d_out, double* s_acc,
                             hipStream_t s) {
  accumulate_kernel<<<1, 64, 0, s>>>(dbatch, n_seqs, pm, d_out, s_acc);
  return hipGetLastError();
}

__global__ void finalize_kernel(const double* __restrict__ s_acc, int n, double inv_n, float* __restrict__ s_out) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    s_out[i] = (float)(s_acc[i] * inv_n);
}

__global__ void zero_f64_kernel(double* p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0.0;
}

hipError_t launch_finalize(const double* s_acc, int n, double inv_n, float* s_out, hipStream_t s) {
  finalize_kernel<<<(n + 255) / 256, 256, 0, s>>>(s_acc, n, inv_n, s_out);
  return hipGetLastError();
}

hipError_t launch_zero_f64(double* p, int n, hipStream_t s) {
  zero_f64_kernel<<<(n + 255) / 256, 256, 0, s>>>(p, n);
  return hipGetLastError();
}

}  // namespace rk
