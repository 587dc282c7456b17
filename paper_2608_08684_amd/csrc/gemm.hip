// Projection GEMMs of the decoder block, C[M, N] = A[M, K] * B[N, K]^T, with the
// block's elementwise work fused into the epilogue:
//   q|k|v projection  -> rotate-half rotary embedding on the q and k columns,
//   output / down     -> residual add into the fp32 stream,
//   gate|up           -> SwiGLU (silu(gate) * up), written as one [M, d_ff] tile,
//   LM head (unfused) -> plain fp32 logits.
// bf16 path: 128x128 block tile, 4 waves of 64x64, v_mfma_f32_32x32x16_bf16,
// K-step 64 double-buffered through LDS with an XOR swizzle of 16-byte chunks.
// fp32 path: a VALU kernel with the same epilogues (64x128 tile).
// Both stage the finished tile through LDS so each epilogue sees whole rows
// (a rotary pair j, j + d_h/2 or a gate/up pair lies inside one tile).
#include "rk_internal.h"

namespace rk {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kCsStride = 132;  // staged tile row stride in floats (128 + pad)

// --------------------------------------------------------------------------- stores of 8 values
__device__ __forceinline__ void store8(float* p, const float* v) {
  reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ void store8(bf16_t* p, const float* v) {
  v4u u;
  u.x = (uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16);
  u.y = (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16);
  u.z = (uint32_t)f2bf(v[4]) | ((uint32_t)f2bf(v[5]) << 16);
  u.w = (uint32_t)f2bf(v[6]) | ((uint32_t)f2bf(v[7]) << 16);
  *reinterpret_cast<v4u*>(p) = u;
}

// --------------------------------------------------------------------------- epilogues
// Called per (row, 8 consecutive tile columns starting at c0) with cs = the staged
// fp32 row of the tile.  kOutCols = output columns one tile produces.
template <typename O>
struct EpiRope {
  static constexpr int kOutCols = 128;
  O* out; int64_t ldo; int rope_cols; int head_dim; const float2* tab; SeqTable seq;
  __device__ void operator()(int row, int bn, int c0, const float* cs) const {
    const int n0 = bn * 128;
    const int pos = row - seq.off[seq_of_row(seq, row)];
    const int half = head_dim >> 1;
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = c0 + j, gc = n0 + c;
      float x = cs[c];
      if (gc < rope_cols) {
        const int jh = gc & (head_dim - 1);
        if (jh < half) {
          const float2 t = tab[(int64_t)pos * half + jh];
          x = cs[c] * t.x - cs[c + half] * t.y;
        } else {
          const float2 t = tab[(int64_t)pos * half + (jh - half)];
          x = cs[c] * t.x + cs[c - half] * t.y;
        }
      }
      v[j] = x;
    }
    store8(out + (int64_t)row * ldo + n0 + c0, v);
  }
};

struct EpiResidual {
  static constexpr int kOutCols = 128;
  float* out; int64_t ldo; const float* res; int64_t ldr;
  __device__ void operator()(int row, int bn, int c0, const float* cs) const {
    const int64_t n = (int64_t)bn * 128 + c0;
    const float4* r4 = reinterpret_cast<const float4*>(res + (int64_t)row * ldr + n);
    const float4 a = r4[0], b = r4[1];
    float v[8] = {a.x + cs[c0 + 0], a.y + cs[c0 + 1], a.z + cs[c0 + 2], a.w + cs[c0 + 3],
                  b.x + cs[c0 + 4], b.y + cs[c0 + 5], b.z + cs[c0 + 6], b.w + cs[c0 + 7]};
    store8(out + (int64_t)row * ldo + n, v);
  }
};

template <typename O>
struct EpiSwiGLU {
  static constexpr int kOutCols = 64;   // tile columns [0,64) gate, [64,128) up
  O* out; int64_t ldo;
  __device__ void operator()(int row, int bn, int c0, const float* cs) const {
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float g = cs[c0 + j], u = cs[64 + c0 + j];
      v[j] = g / (1.0f + expf(-g)) * u;
    }
    store8(out + (int64_t)row * ldo + (int64_t)bn * 64 + c0, v);
  }
};

struct EpiStoreF32 {
  static constexpr int kOutCols = 128;
  float* out; int64_t ldo;
  __device__ void operator()(int row, int bn, int c0, const float* cs) const {
    store8(out + (int64_t)row * ldo + (int64_t)bn * 128 + c0, cs + c0);
  }
};

template <class E>
__device__ __forceinline__ void run_epilogue(const E& e, const float* Cs, int row0, int M, int bn) {
  constexpr int TPR = E::kOutCols / 8;
  constexpr int RPP = 256 / TPR;
  const int t = threadIdx.x;
  const int c0 = (t % TPR) * 8;
  for (int r = t / TPR; r < 64; r += RPP) {
    const int row = row0 + r;
    if (row < M) e(row, bn, c0, Cs + r * kCsStride);
  }
}

// Row of B feeding tile column n of column-block bn.
template <bool SWIGLU>
__device__ __forceinline__ int b_row(int bn, int n, int d_ff) {
  if (SWIGLU) return n < 64 ? bn * 64 + n : d_ff + bn * 64 + (n - 64);
  return bn * 128 + n;
}

// --------------------------------------------------------------------------- bf16 MFMA kernel
template <class E, bool SWIGLU>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(const bf16_t* __restrict__ A, int64_t lda,
                                                        const bf16_t* __restrict__ B, int64_t ldb, int M, int K,
                                                        int d_ff, E e) {
  __shared__ __attribute__((aligned(16))) v4u smem[4096];  // 2 x (A 128x64 + B 128x64) bf16 = 64 KB
  v4u* As = smem;
  v4u* Bs = smem + 2048;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int bn = blockIdx.x, m0 = blockIdx.y * 128;

  const v4u* ga[4];
  const v4u* gb[4];
  int so[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i, row = c >> 3, kc = c & 7;
    const int ar = min(m0 + row, M - 1);
    ga[i] = reinterpret_cast<const v4u*>(A + (int64_t)ar * lda) + kc;
    gb[i] = reinterpret_cast<const v4u*>(B + (int64_t)b_row<SWIGLU>(bn, row, d_ff) * ldb) + kc;
    so[i] = row * 8 + (kc ^ (row & 7));
  }
  const int nk = K / 64;
  v4u ra[4], rb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) { ra[i] = ga[i][0]; rb[i] = gb[i][0]; }
#pragma unroll
  for (int i = 0; i < 4; ++i) { As[so[i]] = ra[i]; Bs[so[i]] = rb[i]; }
  __syncthreads();

  f32x16_t acc[2][2];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[mi][ni][i] = 0.f;

  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) {
#pragma unroll
      for (int i = 0; i < 4; ++i) { ra[i] = ga[i][(kt + 1) * 8]; rb[i] = gb[i][(kt + 1) * 8]; }
    }
    const v4u* Ab = As + buf * 1024;
    const v4u* Bb = Bs + buf * 1024;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int ch = ks * 2 + (lane >> 5);
      bf16x8_t af[2], bfr[2];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi) {
        const int row = wm * 64 + mi * 32 + (lane & 31);
        af[mi] = __builtin_bit_cast(bf16x8_t, Ab[row * 8 + (ch ^ (row & 7))]);
      }
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int row = wn * 64 + ni * 32 + (lane & 31);
        bfr[ni] = __builtin_bit_cast(bf16x8_t, Bb[row * 8 + (ch ^ (row & 7))]);
      }
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[mi], bfr[ni], acc[mi][ni], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      const int nb = (kt + 1) & 1;
#pragma unroll
      for (int i = 0; i < 4; ++i) { As[nb * 1024 + so[i]] = ra[i]; Bs[nb * 1024 + so[i]] = rb[i]; }
    }
    __syncthreads();
  }

  // Stage 64 rows at a time (the two wave rows) and run the epilogue on whole rows.
  float* Cs = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    if (wm == half) {
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int r = mi * 32 + (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
            const int c = wn * 64 + ni * 32 + (lane & 31);
            Cs[r * kCsStride + c] = acc[mi][ni][i];
          }
    }
    __syncthreads();
    run_epilogue(e, Cs, m0 + half * 64, M, bn);
    __syncthreads();
  }
}

// --------------------------------------------------------------------------- fp32 VALU kernel
template <class E, bool SWIGLU>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, int64_t lda,
                                                       const float* __restrict__ B, int64_t ldb, int M, int K,
                                                       int d_ff, E e) {
  __shared__ __attribute__((aligned(16))) float smem[64 * kCsStride];
  float* As = smem;             // [16][68]  k-major
  float* Bs = smem + 16 * 68;   // [16][132] k-major
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const int bn = blockIdx.x, m0 = blockIdx.y * 64;
  const int lrow = tid >> 2, kq = (tid & 3) * 4;
  const float* pa = A + (int64_t)min(m0 + lrow, M - 1) * lda + kq;
  const float* pb0 = B + (int64_t)b_row<SWIGLU>(bn, lrow, d_ff) * ldb + kq;
  const float* pb1 = B + (int64_t)b_row<SWIGLU>(bn, lrow + 64, d_ff) * ldb + kq;
  float acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < K; k0 += 16) {
    const float4 a = *reinterpret_cast<const float4*>(pa + k0);
    const float4 b0 = *reinterpret_cast<const float4*>(pb0 + k0);
    const float4 b1 = *reinterpret_cast<const float4*>(pb1 + k0);
    __syncthreads();
    As[(kq + 0) * 68 + lrow] = a.x; As[(kq + 1) * 68 + lrow] = a.y;
    As[(kq + 2) * 68 + lrow] = a.z; As[(kq + 3) * 68 + lrow] = a.w;
    Bs[(kq + 0) * 132 + lrow] = b0.x; Bs[(kq + 1) * 132 + lrow] = b0.y;
    Bs[(kq + 2) * 132 + lrow] = b0.z; Bs[(kq + 3) * 132 + lrow] = b0.w;
    Bs[(kq + 0) * 132 + lrow + 64] = b1.x; Bs[(kq + 1) * 132 + lrow + 64] = b1.y;
    Bs[(kq + 2) * 132 + lrow + 64] = b1.z; Bs[(kq + 3) * 132 + lrow + 64] = b1.w;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      float av[4], bv[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[k * 68 + ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 8; ++j) bv[j] = Bs[k * 132 + tx * 8 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
  }
  __syncthreads();
  float* Cs = smem;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) Cs[(ty * 4 + i) * kCsStride + tx * 8 + j] = acc[i][j];
  __syncthreads();
  run_epilogue(e, Cs, m0, M, bn);
}

// --------------------------------------------------------------------------- dispatch
template <class E, bool SWIGLU>
static hipError_t go(const GemmArgs& a, bool bf16, const E& e, hipStream_t s) {
  const int nbn = SWIGLU ? a.d_ff / 64 : a.N / 128;
  if (bf16) {
    dim3 grid(nbn, (a.M + 127) / 128);
    gemm_bf16_kernel<E, SWIGLU><<<grid, 256, 0, s>>>((const bf16_t*)a.A, a.lda, (const bf16_t*)a.B, a.ldb, a.M,
                                                     a.K, a.d_ff, e);
  } else {
    dim3 grid(nbn, (a.M + 63) / 64);
    gemm_f32_kernel<E, SWIGLU><<<grid, 256, 0, s>>>((const float*)a.A, a.lda, (const float*)a.B, a.ldb, a.M, a.K,
                                                    a.d_ff, e);
  }
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs& a, bool bf16, hipStream_t s) {
  if (a.M <= 0) return hipSuccess;
  switch (a.epi) {
    case Epi::kStoreRope:
      if (bf16) {
        EpiRope<bf16_t> e{(bf16_t*)a.out, a.ldo, a.rope_cols, a.head_dim, a.rope_tab, a.seq};
        return go<EpiRope<bf16_t>, false>(a, true, e, s);
      } else {
        EpiRope<float> e{(float*)a.out, a.ldo, a.rope_cols, a.head_dim, a.rope_tab, a.seq};
        return go<EpiRope<float>, false>(a, false, e, s);
      }
    case Epi::kResidual: {
      EpiResidual e{(float*)a.out, a.ldo, a.res, a.ldr};
      return go<EpiResidual, false>(a, bf16, e, s);
    }
    case Epi::kSwiGLU:
      if (bf16) {
        EpiSwiGLU<bf16_t> e{(bf16_t*)a.out, a.ldo};
        return go<EpiSwiGLU<bf16_t>, true>(a, true, e, s);
      } else {
        EpiSwiGLU<float> e{(float*)a.out, a.ldo};
        return go<EpiSwiGLU<float>, true>(a, false, e, s);
      }
    case Epi::kStoreF32: {
      EpiStoreF32 e{(float*)a.out, a.ldo};
      return go<EpiStoreF32, false>(a, bf16, e, s);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace rk
