// LM head + log-softmax + KL (Algorithm 1, WindowKL; Eq. sample-response).
//
// KL_t = sum_v P_v (log P_v - log Q_v) with P = softmax(a), Q = softmax(b),
// a = x_clean W^T, b = x_pert W^T.  With delta = a - b, A_t = logsumexp(a) and
// p_v = exp(a_v - A_t):
//   KL_t = sum_v p_v delta_v + log(sum_v p_v e^{-delta_v})
//        = sum_v p_v delta_v + log1p(S_t),  S_t = sum_v p_v (e^{-delta_v} - 1)
//        = sum_v p_v f(delta_v) - g(S_t),  f(x) = x + expm1(-x), g(y) = y - log1p(y).
// The fused kernel accumulates the first form (cheap: no clean max or sums
// beyond A_t, delta = 0 gives exactly 0); the unfused kernel uses the last form,
// whose terms are all non-negative (f and g by series near 0), as a cross-check.
//
// Fused path (bf16): logits never reach HBM.  The clean pass runs lm_lse once per
// batch (A_t).  lm_kl then computes, per 128-token x 128-vocab tile, the clean
// logits once and the logits of G perturbed passes against the same W tile, and
// folds each into per-lane (F, S) partials.  The tile is computed transposed
// (vocab rows = MFMA M, tokens = MFMA N), so a lane owns one token and all its
// vocab reductions are lane-local.  Vocab is split into chunks across
// workgroups; a fixed-order merge kernel combines the chunk partials.
// Unfused path (any dtype): KL over two materialised fp32 logit tensors.
#include <math.h>

#include "mfma_tile.h"

#include <type_traits>

namespace rk {

// f(x) = x + expm1(-x) = x^2/2 - x^3/6 + ...  (>= 0)
__device__ __forceinline__ float kl_f(float x) {
  if (fabsf(x) < 0.25f) {
    float p = x * (1.0f / 40320.0f) - (1.0f / 5040.0f);
    p = fmaf(p, x, 1.0f / 720.0f);
    p = fmaf(p, x, -1.0f / 120.0f);
    p = fmaf(p, x, 1.0f / 24.0f);
    p = fmaf(p, x, -1.0f / 6.0f);
    p = fmaf(p, x, 0.5f);
    return p * x * x;
  }
  return (expf(-fmaxf(x, -80.0f)) - 1.0f) + x;
}

// --------------------------------------------------------------------------- shared tile GEMM
// acc[vb] (vb = 0..3) = W[v0 + 32 vb + ..] . X[t0 + 32 w + l32]: the 128 x 128 logit
// tile, transposed, wave w owning tokens 32w..32w+31.  X is padded to whole
// 128-row tiles by the caller.  Leaves LDS free on return.
__device__ __forceinline__ void logit_tile(const bf16_t* __restrict__ W, const bf16_t* __restrict__ X, int v0,
                                           int t0, int d, v4u* As, v4u* Bs, f32x16_t acc[4]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, l32 = lane & 31;
  TileSrc sw, sx;
  sw.init(W + (int64_t)v0 * d, d, w, lane);
  sx.init(X + (int64_t)t0 * d, d, w, lane);
#pragma unroll
  for (int vb = 0; vb < 4; ++vb)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[vb][i] = 0.f;
  const int nk = d / kBK;
  sw.load<128>(0, As, w);
  sx.load<128>(0, Bs, w);
  wait_vmem();
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      sw.load<128>(kt + 1, As + (cur ^ 1) * 1024, w);
      sx.load<128>(kt + 1, Bs + (cur ^ 1) * 1024, w);
    }
    const v4u* At = As + cur * 1024;
    const v4u* Bt = Bs + cur * 1024;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bf16x8_t bx = frag(Bt, w * 32 + l32, ks, lane);
#pragma unroll
      for (int vb = 0; vb < 4; ++vb)
        acc[vb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag(At, vb * 32 + l32, ks, lane), bx, acc[vb], 0, 0, 0);
    }
    wait_vmem();
    __syncthreads();
  }
}

// --------------------------------------------------------------------------- clean log-sum-exp
__global__ __launch_bounds__(256) void lm_lse_kernel(const bf16_t* __restrict__ X, const bf16_t* __restrict__ W,
                                                     int rows, int d, int n_vt, int vt_per_chunk,
                                                     float2* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) v4u smem[4096];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int t0 = blockIdx.x * 128, chunk = blockIdx.y;
  const int vt0 = chunk * vt_per_chunk, vt1 = min(n_vt, vt0 + vt_per_chunk);
  float m = -INFINITY, z = 0.f;
  f32x16_t acc[4];
  for (int vt = vt0; vt < vt1; ++vt) {
    logit_tile(W, X, vt * 128, t0, d, smem, smem + 2048, acc);
    float mx = -INFINITY;
#pragma unroll
    for (int vb = 0; vb < 4; ++vb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, acc[vb][i]);
    const float m_new = fmaxf(m, mx);
    float sum = 0.f;
#pragma unroll
    for (int vb = 0; vb < 4; ++vb)
#pragma unroll
      for (int i = 0; i < 16; ++i) sum += expf(acc[vb][i] - m_new);
    z = z * expf(m - m_new) + sum;
    m = m_new;
  }
  // merge the two half-waves that share a token
  const float m2 = __shfl_xor(m, 32, 64), z2 = __shfl_xor(z, 32, 64);
  const float mm = fmaxf(m, m2);
  const float zz = (mm == -INFINITY) ? 0.f : z * expf(m - mm) + z2 * expf(m2 - mm);
  const int token = t0 + w * 32 + (lane & 31);
  if ((lane >> 5) == 0 && token < rows) part[(int64_t)chunk * rows + token] = make_float2(mm, zz);
}

__global__ void lse_merge_kernel(const float2* __restrict__ part, int n_chunks, int rows, float* __restrict__ lse) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows) return;
  float M = -INFINITY;
  for (int c = 0; c < n_chunks; ++c) M = fmaxf(M, part[(int64_t)c * rows + r].x);
  double z = 0.0;
  for (int c = 0; c < n_chunks; ++c) {
    const float2 p = part[(int64_t)c * rows + r];
    if (p.y > 0.f) z += (double)p.y * exp((double)p.x - (double)M);
  }
  lse[r] = (float)((double)M + log(z));
}

// --------------------------------------------------------------------------- fused KL
// Per (token t, pass g): T1 = sum_v p_v delta_v and S = sum_v p_v (e^{-delta_v} - 1)
// with p_v = exp(a_v - A_t), so KL_t = T1 + log1p(S) (= sum p (a - b) - A + B
// without forming A and B).  delta = 0 gives exactly T1 = S = 0.  p is recomputed
// per pass instead of being held, which keeps the kernel at two waves per SIMD.
//
// A workgroup of 8 waves owns 256 tokens and a chunk of 128-wide vocab tiles.  For
// each vocab tile it computes the clean logit tile (kept in registers as `a`) and
// then the G perturbed tiles against the same W rows, folding each into the
// per-lane (T1, S) of its pass.  All the k-steps of all these tiles form one
// stream through a 3-stage LDS ring, so the copies run ahead across tile
// boundaries.  Wave w owns tokens 32 w .. 32 w + 31 (the MFMA N side) and all 128
// vocab rows of the tile (M side): its reductions over vocab stay in its lanes.
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kKlTok = 256;     // tokens per workgroup

// One 16-byte global->LDS copy per lane through a raw buffer descriptor over
// [base, base + nrec): lanes whose offset falls outside read zeros.
__device__ __forceinline__ void dma16_rows(const void* base, uint32_t nrec, uint32_t voff, int32_t soff,
                                           uint32_t lds) {
  const uint64_t b = (uint64_t)base;
  i32x4_t rsrc;
  rsrc[0] = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)b);
  rsrc[1] = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)(b >> 32));
  rsrc[2] = __builtin_amdgcn_readfirstlane((int32_t)nrec);
  rsrc[3] = 0x00020000;   // raw buffer, 32-bit data format
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               :
               : "v"(voff), "s"(rsrc), "s"(soff), "{m0}"(lds)
               : "memory");
}

// Wait until at most `ahead` k-steps of NL copies each (those issued after the
// one about to be consumed) are still in flight; ahead <= K.
template <int NL, int K>
__device__ __forceinline__ void wait_steps_ahead(int ahead) {
  if constexpr (K <= 0) {
    wait_vmem();
  } else {
    if (ahead >= K) wait_vmem_le<NL * K>();
    else wait_steps_ahead<NL, K - 1>(ahead);
  }
}

template <int GMAX, int BK, int ST>
__global__ __launch_bounds__(512) void lm_kl_kernel(const bf16_t* __restrict__ Xc, const bf16_t* __restrict__ Xp,
                                                    int64_t pass_stride, int G, const bf16_t* __restrict__ W,
                                                    int rows, int d, int n_vt, int n_chunks,
                                                    const float* __restrict__ lse, float2* __restrict__ part) {
  constexpr int CH = BK / 8;                     // 16-byte chunks per k row of a stage
  constexpr int RPI = 64 / CH;                   // rows per wave copy instruction
  constexpr int WS = 128 * CH, XS = kKlTok * CH, SS = WS + XS;   // 16-byte slots per stage
  constexpr int NLW = WS / 512, NLX = XS / 512, NL = NLW + NLX;  // copies per thread and stage
  constexpr int NKS = BK / 16;                   // k-slices per k-step
  static_assert(WS % 512 == 0 && (ST - 2) * NL < 16 && ST * SS * 16 <= 160 * 1024, "stage geometry");
  __shared__ __attribute__((aligned(16))) v4u smem[ST * SS];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l32 = lane & 31;
  // Workgroup -> (token block, vocab chunk): the 32 workgroups an XCD runs at once
  // cover 4 token blocks x 8 chunks, so one pass's X rows (4 x 384 KB at d = 768)
  // and the W tiles in use (8 x 192 KB) stay in that XCD's L2 through the passes.
  int tb, chunk;
  xcd_tile((int)blockIdx.x, (rows + kKlTok - 1) / kKlTok, n_chunks, 4, &tb, &chunk);
  const int t0 = tb * kKlTok;
  const int vt0 = (int)((int64_t)chunk * n_vt / n_chunks), vt1 = (int)((int64_t)(chunk + 1) * n_vt / n_chunks);
  const int nk = d / BK;
  const int nsteps = (vt1 - vt0) * (G + 1) * nk;
  const int token = t0 + w * 32 + l32;
  float Ac = lse[min(token, rows - 1)] * kLog2e;
  asm volatile("" : "+v"(Ac));   // loaded before the copies start: no vector-memory wait inside the loop

  // Copy geometry: in round j a wave instruction fills rows 8 RPI j + RPI w ..
  // + RPI - 1 of a tile, lane -> (row 8 RPI j + RPI w + lane / CH, swizzled chunk);
  // rounds advance by a multiple of 16 rows, which leaves the row swizzle unchanged.
  const int r0 = w * RPI + lane / CH;
  const uint32_t voff0 = (uint32_t)(r0 * d * 2 + (((lane % CH) ^ swz<CH>(r0)) * 16));
  const uint32_t round_bytes = (uint32_t)(8 * RPI * d * 2);
  const uint32_t x_nrec = (uint32_t)(max(0, min(rows - t0, kKlTok)) * d * 2);
  const uint32_t w_nrec = (uint32_t)(128 * d * 2);
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) v4u*)smem;

  // producer position: the next k-step to copy
  int p_kt = 0, p_g = -1, p_vt = vt0, issued = 0;
  auto issue_one = [&](int j, int slot) {
    const uint32_t lds = lds0 + (uint32_t)(slot * SS * 16);
    const int32_t soff = p_kt * BK * 2;
    if (j < NLW) {
      dma16_rows(W + (int64_t)p_vt * 128 * d, w_nrec, voff0 + j * round_bytes, soff,
                 lds + (uint32_t)((j * 8 + w) * 64 * 16));
    } else {
      const int jx = j - NLW;
      const bf16_t* xb = (p_g < 0 ? Xc : Xp + (int64_t)p_g * pass_stride) + (int64_t)t0 * d;
      dma16_rows(xb, x_nrec, voff0 + jx * round_bytes, soff, lds + (uint32_t)((WS + (jx * 8 + w) * 64) * 16));
    }
  };
  auto advance = [&]() {
    ++issued;
    if (++p_kt == nk) {
      p_kt = 0;
      if (++p_g == G) { p_g = -1; ++p_vt; }
    }
  };
#pragma unroll
  for (int q = 0; q < ST - 1; ++q)
    if (issued < nsteps) {
#pragma unroll
      for (int j = 0; j < NL; ++j) issue_one(j, q);
      advance();
    }

  float T1[GMAX], S[GMAX];
#pragma unroll
  for (int g = 0; g < GMAX; ++g) { T1[g] = 0.f; S[g] = 0.f; }
  f32x16_t a[4], b[4];
  int kt = 0, g = -1, slot = 0, pslot = ST - 1;
  constexpr int PER = (NL + NKS - 1) / NKS;   // copies issued per k-slice
  // One k-step of the stream from LDS slot `slot`; COPY: it also issues its share
  // of the copies of the step ST - 1 ahead.  The copying steps and the last ST - 1
  // (which copy nothing) run as two loops, so each k-slice's reads, copies and
  // MFMAs form one basic block.
  int s = 0;
  auto kstep = [&](auto COPY) {
    constexpr bool CP = decltype(COPY)::value;
    if constexpr (CP) wait_vmem_le<(ST - 2) * NL>(); else wait_steps_ahead<NL, ST - 2>(issued - 1 - s);
    __syncthreads();   // k-step s is in LDS for every wave; the slot of s - 1 is free
    if (kt == 0) {
#pragma unroll
      for (int vb = 0; vb < 4; ++vb)
#pragma unroll
        for (int i = 0; i < 16; ++i) b[vb][i] = 0.f;
    }
    const v4u* Wt = smem + slot * SS;
    const v4u* Xt = Wt + WS;
    bf16x8_t wf[2][4], xf[2];
#pragma unroll
    for (int vb = 0; vb < 4; ++vb) wf[0][vb] = frag<CH>(Wt, vb * 32 + l32, 0, lane);
    xf[0] = frag<CH>(Xt, w * 32 + l32, 0, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      const int c = ks & 1;
      if (ks + 1 < NKS) {
#pragma unroll
        for (int vb = 0; vb < 4; ++vb) wf[c ^ 1][vb] = frag<CH>(Wt, vb * 32 + l32, ks + 1, lane);
        xf[c ^ 1] = frag<CH>(Xt, w * 32 + l32, ks + 1, lane);
      }
      if constexpr (CP) {
#pragma unroll
        for (int j = ks * PER; j < (ks + 1) * PER; ++j)
          if (j < NL) issue_one(j, pslot);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int vb = 0; vb < 4; ++vb)
        b[vb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[c][vb], xf[c], b[vb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (CP) {
      advance();
      pslot = pslot == ST - 1 ? 0 : pslot + 1;
    }
    slot = slot == ST - 1 ? 0 : slot + 1;
  };
  // after each k-step: a complete logit tile is kept (clean) or folded (a pass)
  auto tile_done = [&]() {
    if (++kt < nk) return;
    kt = 0;
    if (g < 0) {
#pragma unroll
      for (int vb = 0; vb < 4; ++vb) a[vb] = b[vb];
    } else {
      float t1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int vb = 0; vb < 4; ++vb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float av = a[vb][i];
          const float p = __builtin_amdgcn_exp2f(fmaf(av, kLog2e, -Ac));
          const float dl = av - b[vb][i];
          const float e = __builtin_amdgcn_exp2f(-dl * kLog2e) - 1.0f;
          t1 = fmaf(p, dl, t1);
          s2 = fmaf(p, e, s2);
        }
#pragma unroll
      for (int j = 0; j < GMAX; ++j)
        if (j == g) { T1[j] += t1; S[j] += s2; }
    }
    if (++g == G) g = -1;
  };
  for (; s < nsteps - (ST - 1); ++s) {
    kstep(std::true_type{});
    tile_done();
  }
  for (; s < nsteps; ++s) {
    kstep(std::false_type{});
    tile_done();
  }
#pragma unroll
  for (int g2 = 0; g2 < GMAX; ++g2) {
    if (g2 < G) {
      const float x = T1[g2] + __shfl_xor(T1[g2], 32, 64);
      const float y = S[g2] + __shfl_xor(S[g2], 32, 64);
      if ((lane >> 5) == 0 && token < rows) part[((int64_t)chunk * G + g2) * rows + token] = make_float2(x, y);
    }
  }
}

// kl[g * rows + r] = sum_c T1 + log1p(sum_c S), fixed chunk order, double.
__global__ void kl_merge_kernel(const float2* __restrict__ part, int n_chunks, int G, int rows, float* __restrict__ kl) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x, g = blockIdx.y;
  if (r >= rows) return;
  double t1 = 0.0, s = 0.0;
  for (int c = 0; c < n_chunks; ++c) {
    const float2 v = part[((int64_t)c * G + g) * rows + r];
    t1 += v.x;
    s += v.y;
  }
  kl[(int64_t)g * rows + r] = (float)(t1 + log1p(s));
}

int lm_chunks(int rows, int vocab) {
  const int n_vt = vocab / 128, n_tt = (rows + 127) / 128;
  int chunks = (2048 + n_tt - 1) / n_tt;
  if (chunks > n_vt) chunks = n_vt;
  if (chunks < 1) chunks = 1;
  const int per = (n_vt + chunks - 1) / chunks;
  return (n_vt + per - 1) / per;
}

// chunks of the fused KL kernel: about 1024 workgroups of 256 tokens; chunk c
// takes vocab tiles [c n_vt / chunks, (c + 1) n_vt / chunks)
int lm_kl_chunks(int rows, int vocab) {
  const int n_vt = vocab / 128, n_tb = (rows + kKlTok - 1) / kKlTok;
  const int chunks = (1024 + n_tb - 1) / n_tb;
  return chunks > n_vt ? n_vt : (chunks < 1 ? 1 : chunks);
}

static int vt_per_chunk(int vocab, int chunks) {
  const int n_vt = vocab / 128;
  return (n_vt + chunks - 1) / chunks;
}

hipError_t launch_lm_lse(const bf16_t* x, const bf16_t* W, int rows, int d, int vocab, float2* part, float* lse,
                         hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const int chunks = lm_chunks(rows, vocab);
  dim3 grid((rows + 127) / 128, chunks);
  lm_lse_kernel<<<grid, 256, 0, s>>>(x, W, rows, d, vocab / 128, vt_per_chunk(vocab, chunks), part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  lse_merge_kernel<<<(rows + 255) / 256, 256, 0, s>>>(part, chunks, rows, lse);
  return hipGetLastError();
}

hipError_t launch_lm_kl(const bf16_t* xc, const bf16_t* xp, int64_t pass_stride, int G, const bf16_t* W, int rows,
                        int d, int vocab, const float* lse, float2* part, float* kl, hipStream_t s) {
  if (rows <= 0 || G <= 0) return hipSuccess;
  if (d % 64 != 0 || vocab % 128 != 0 || (int64_t)kKlTok * d * 2 > 0x7fffffff) return hipErrorInvalidValue;
  const int chunks = lm_kl_chunks(rows, vocab);
  const int grid = (rows + kKlTok - 1) / kKlTok * chunks;
#ifndef RK_KL_BK
#define RK_KL_BK 64
#define RK_KL_ST 3
#endif
  constexpr int BK = RK_KL_BK, ST = RK_KL_ST;
  if (d % BK != 0) return hipErrorInvalidValue;
  if (G <= 4)
    lm_kl_kernel<4, BK, ST><<<grid, 512, 0, s>>>(xc, xp, pass_stride, G, W, rows, d, vocab / 128, chunks, lse, part);
  else if (G <= 8)
    lm_kl_kernel<8, BK, ST><<<grid, 512, 0, s>>>(xc, xp, pass_stride, G, W, rows, d, vocab / 128, chunks, lse, part);
  else if (G <= RK_MAX_GROUP)
    lm_kl_kernel<RK_MAX_GROUP, BK, ST><<<grid, 512, 0, s>>>(xc, xp, pass_stride, G, W, rows, d, vocab / 128, chunks, lse,
                                                             part);
  else
    return hipErrorInvalidValue;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  kl_merge_kernel<<<dim3((rows + 255) / 256, G), 256, 0, s>>>(part, chunks, G, rows, kl);
  return hipGetLastError();
}

// --------------------------------------------------------------------------- unfused KL
// One workgroup (16 waves) per row scores every pass of the group: one sweep over
// the clean row gives its log-sum-exp A (running max and rescaled sum per thread,
// merged in a fixed order); when the row fits (vocab <= kKlLdsRow) it stays in
// LDS, so every pass reads only its own row from memory, once (p_v =
// 2^(a_v log2 e - A log2 e) with the hardware exp2, as in the fused kernel).  Per
// thread F and S are summed in fp32 over its vocab / 1024 entries, then across
// the workgroup in double, in a fixed order (lane tree, then waves in order).
constexpr int kKlThreads = 1024;
constexpr int kKlLdsRow = 36864;   // longest row kept in LDS (144 KB of fp32)

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// sum over the workgroup: every thread gets the same value
__device__ __forceinline__ double block_sum(double v, double* red) {
  const int w = threadIdx.x >> 6;
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  double r = 0.0;
  for (int i = 0; i < kKlThreads / 64; ++i) r += red[i];
  __syncthreads();
  return r;
}

// merge of two (max, sum of exp(x - max)) pairs
__device__ __forceinline__ void lse_merge(float& m, double& z, float m2, double z2) {
  if (m2 == -INFINITY) return;
  if (m == -INFINITY) { m = m2; z = z2; return; }
  const float mn = fmaxf(m, m2);
  z = z * (double)expf(m - mn) + z2 * (double)expf(m2 - mn);
  m = mn;
}

// one step of the running (max, sum) of a thread
__device__ __forceinline__ void lse_add(float& m, double& z, float x) {
  if (x > m) { z = z * (double)expf(m - x) + 1.0; m = x; }   // expf(-inf) = 0 on the first element
  else z += (double)expf(x - m);
}

__device__ __forceinline__ float block_lse(float m, double z, double* red, float* redm) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) lse_merge(m, z, __shfl_xor(m, d, 64), __shfl_xor(z, d, 64));
  if (lane == 0) { redm[w] = m; red[w] = z; }
  __syncthreads();
  float M = -INFINITY;
  double Z = 0.0;
  for (int i = 0; i < kKlThreads / 64; ++i) lse_merge(M, Z, redm[i], red[i]);
  __syncthreads();
  return (float)((double)M + log(Z));
}

// F and S terms of one entry: clean logit x, pass logit y
__device__ __forceinline__ void kl_terms(float x, float y, float Al, float& f1, float& s1) {
  const float p = __builtin_amdgcn_exp2f(fmaf(x, kLog2e, -Al));
  const float dl = x - y;
  const float f = kl_f(dl);
  f1 = fmaf(p, f, f1);
  s1 = fmaf(p, f - dl, s1);
}

// Rows are read as 16-byte groups of four entries (vocab is a multiple of 128),
// four groups per thread in flight.
template <bool IN_LDS>
__global__ __launch_bounds__(kKlThreads) void kl_logits_kernel(const float* __restrict__ lc,
                                                               const float* __restrict__ lp, int64_t pass_stride,
                                                               int G, int rows, int vocab, float* __restrict__ kl) {
  __shared__ float4 row[IN_LDS ? kKlLdsRow / 4 : 1];
  __shared__ double red[kKlThreads / 64];
  __shared__ float redm[kKlThreads / 64];
  constexpr int U = 4;
  const int r = blockIdx.x, t = threadIdx.x, n4 = vocab / 4;
  const float4* a = reinterpret_cast<const float4*>(lc + (int64_t)r * vocab);
  float m = -INFINITY;
  double z = 0.0;
  for (int q0 = t; q0 < n4; q0 += U * kKlThreads) {
    float4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int q = q0 + u * kKlThreads;
      if (q < n4) x[u] = a[q];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int q = q0 + u * kKlThreads;
      if (q < n4) {
        if (IN_LDS) row[q] = x[u];
        lse_add(m, z, x[u].x);
        lse_add(m, z, x[u].y);
        lse_add(m, z, x[u].z);
        lse_add(m, z, x[u].w);
      }
    }
  }
  const float A = block_lse(m, z, red, redm);   // its barriers also publish the LDS row
  const float Al = A * kLog2e;
  for (int g = 0; g < G; ++g) {
    const float4* b = reinterpret_cast<const float4*>(lp + (int64_t)g * pass_stride + (int64_t)r * vocab);
    float f1 = 0.f, s1 = 0.f;
    for (int q0 = t; q0 < n4; q0 += U * kKlThreads) {
      float4 y[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int q = q0 + u * kKlThreads;
        if (q < n4) y[u] = b[q];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int q = q0 + u * kKlThreads;
        if (q < n4) {
          const float4 x = IN_LDS ? row[q] : a[q];
          kl_terms(x.x, y[u].x, Al, f1, s1);
          kl_terms(x.y, y[u].y, Al, f1, s1);
          kl_terms(x.z, y[u].z, Al, f1, s1);
          kl_terms(x.w, y[u].w, Al, f1, s1);
        }
      }
    }
    const double F = block_sum((double)f1, red);
    const double S = block_sum((double)s1, red);
    if (t == 0) kl[(int64_t)g * rows + r] = (float)(F - (S - log1p(S)));
  }
}

hipError_t launch_kl_logits(const float* lc, const float* lp, int64_t pass_stride, int G, int rows, int vocab,
                            float* kl, hipStream_t s) {
  if (rows <= 0 || G <= 0) return hipSuccess;
  if (vocab % 4 != 0 || pass_stride % 4 != 0 || ((uintptr_t)lc | (uintptr_t)lp) % 16 != 0) return hipErrorInvalidValue;
  if (vocab <= kKlLdsRow)
    kl_logits_kernel<true><<<rows, kKlThreads, 0, s>>>(lc, lp, pass_stride, G, rows, vocab, kl);
  else
    kl_logits_kernel<false><<<rows, kKlThreads, 0, s>>>(lc, lp, pass_stride, G, rows, vocab, kl);
  return hipGetLastError();
}

}  // namespace rk
