// Projection GEMMs of the decoder block, C[M, N] = A[M, K] * B[N, K]^T, with the
// block's elementwise work fused into the epilogue:
//   q|k|v projection  -> rotate-half rotary embedding on the q and k columns,
//   output / down     -> residual add into the fp32 stream,
//   gate|up           -> SwiGLU (silu(gate) * up), written as one [M, d_ff] tile,
//   LM head (unfused) -> plain fp32 logits.
// bf16 path: BM x BN block tile (256x256 or 256x192 on 8 waves, whichever wastes
// less of the last round of workgroups; 128x128 on 4 for small M),
// v_mfma_f32_32x32x16_bf16, K-steps streamed global -> LDS by buffer loads into a
// ring of LDS stages (see mfma_tile.h).  The finished tile leaves through LDS so
// the global accesses are whole rows; a rotary pair j, j + d_h/2 or a gate/up pair
// always lies inside one tile.
// fp32 path: a VALU kernel with the same epilogues (64x128 tile), staged 64 rows
// at a time.
#include "mfma_tile.h"

#include <algorithm>
#include <cstdint>
#include <type_traits>

namespace rk {

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

// 4 values to 4 consecutive elements (16 bytes fp32, 8 bytes bf16)
__device__ __forceinline__ void store4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
__device__ __forceinline__ void store4(bf16_t* p, float4 v) {
  uint2 u;
  u.x = (uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16);
  u.y = (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16);
  *reinterpret_cast<uint2*>(p) = u;
}
// 16 bytes between LDS and global memory (the LDS side 8-byte aligned for bf16 rows)
__device__ __forceinline__ void copy16(float* dst, const float* src) {
  *reinterpret_cast<float4*>(dst) = *reinterpret_cast<const float4*>(src);
}
__device__ __forceinline__ void copy16(bf16_t* dst, const bf16_t* src) {
  const uint2 a = reinterpret_cast<const uint2*>(src)[0], b = reinterpret_cast<const uint2*>(src)[1];
  *reinterpret_cast<uint4*>(dst) = make_uint4(a.x, a.y, b.x, b.y);
}

// --------------------------------------------------------------------------- epilogues
// Called per (row, 8 consecutive output columns starting at c0) with cs = the
// staged fp32 row of a BN-wide tile.  out_cols(BN) = output columns per tile.
template <typename O>
struct EpiRope {
  static constexpr int out_cols(int BN) { return BN; }
  static constexpr bool kPaired = true;
  static constexpr int pair_dist(int, int head_dim) { return head_dim / 2; }
  // tab[pos * head_dim/2 + j] = (cos, sin) of position pos, pair j; pos[row] = position of the row
  O* out; int64_t ldo; int rope_cols; int head_dim; const float2* tab; const int32_t* pos; int q_cols; float q_scale;
  template <int BN>
  __device__ void apply(int row, int bn, int c0, const float* cs) const {
    const int gc0 = bn * BN + c0;
    O* dst = out + (int64_t)row * ldo + gc0;
    if (gc0 >= rope_cols) {  // value columns: no rotation
      store8(dst, cs + c0);
      return;
    }
    // the 8 columns lie in one half of one head: pairs jh0..jh0+7 with partners at +-half
    const int half = head_dim >> 1;
    const int jh = gc0 & (head_dim - 1);
    const bool lo = jh < half;
    const int j0 = lo ? jh : jh - half;
    const float4* t4 = reinterpret_cast<const float4*>(tab + (int64_t)pos[row] * half + j0);
    const float* x = cs + c0;
    const float* y = cs + c0 + (lo ? half : -half);
    const float sg = lo ? -1.0f : 1.0f;
    const float sc = gc0 < q_cols ? q_scale : 1.0f;
    float v[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 t = t4[q];  // (cos, sin) of pairs 2q and 2q+1
      v[2 * q] = fmaf(sg * y[2 * q], t.y, x[2 * q] * t.x) * sc;
      v[2 * q + 1] = fmaf(sg * y[2 * q + 1], t.w, x[2 * q + 1] * t.z) * sc;
    }
    store8(dst, v);
  }
  // register form: x = tile columns tc..tc+3 (first half of a head), y = their
  // partners head_dim/2 further on; o0, o1 = the outputs at the same columns
  using stage_t = O;
  static constexpr int kOut = 2;
  template <int BN>
  __device__ __forceinline__ void pair(int row, int bn, int tc, float4 x, float4 y, float4& o0, float4& o1) const {
    const int gc = bn * BN + tc, half = head_dim >> 1;
    if (gc >= rope_cols) {  // value columns: no rotation
      o0 = x;
      o1 = y;
      return;
    }
    const float4* t4 = reinterpret_cast<const float4*>(tab + (int64_t)pos[row] * half + (gc & (head_dim - 1)));
    const float4 t01 = t4[0], t23 = t4[1];   // (cos, sin) of pairs j .. j+3
    const float sc = gc < q_cols ? q_scale : 1.0f;
    o0 = make_float4(fmaf(-y.x, t01.y, x.x * t01.x) * sc, fmaf(-y.y, t01.w, x.y * t01.z) * sc,
                     fmaf(-y.z, t23.y, x.z * t23.x) * sc, fmaf(-y.w, t23.w, x.w * t23.z) * sc);
    o1 = make_float4(fmaf(x.x, t01.y, y.x * t01.x) * sc, fmaf(x.y, t01.w, y.y * t01.z) * sc,
                     fmaf(x.z, t23.y, y.z * t23.x) * sc, fmaf(x.w, t23.w, y.w * t23.z) * sc);
  }
};

struct EpiResidual {
  static constexpr int out_cols(int BN) { return BN; }
  static constexpr bool kPaired = false;
  float* out; int64_t ldo; const float* res; int64_t ldr;
  using stage_t = float;
  template <int BN>
  __device__ void apply(int row, int bn, int c0, const float* cs) const {
    const int64_t n = (int64_t)bn * BN + c0;
    const float4* r4 = reinterpret_cast<const float4*>(res + (int64_t)row * ldr + n);
    const float4 a = r4[0], b = r4[1];
    float v[8] = {a.x + cs[c0 + 0], a.y + cs[c0 + 1], a.z + cs[c0 + 2], a.w + cs[c0 + 3],
                  b.x + cs[c0 + 4], b.y + cs[c0 + 5], b.z + cs[c0 + 6], b.w + cs[c0 + 7]};
    store8(out + (int64_t)row * ldo + n, v);
  }
};

template <typename O>
struct EpiSwiGLU {
  static constexpr int out_cols(int BN) { return BN / 2; }  // tile columns [0, BN/2) gate, [BN/2, BN) up
  static constexpr bool kPaired = true;
  static constexpr int pair_dist(int BN, int) { return BN / 2; }
  O* out; int64_t ldo;
  static __device__ __forceinline__ float silu_mul(float g, float u) {
    return g * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-g * 1.4426950408889634f)) * u;
  }
  // register form: gate = tile columns tc..tc+3 (< BN/2), up = the same columns + BN/2;
  // o0 = output columns tc..tc+3 of this tile
  using stage_t = O;
  static constexpr int kOut = 1;
  template <int BN>
  __device__ __forceinline__ void pair(int, int, int, float4 g, float4 u, float4& o0, float4&) const {
    o0 = make_float4(silu_mul(g.x, u.x), silu_mul(g.y, u.y), silu_mul(g.z, u.z), silu_mul(g.w, u.w));
  }
  template <int BN>
  __device__ void apply(int row, int bn, int c0, const float* cs) const {
    // silu(g) = g / (1 + e^-g) with the hardware exp2 and reciprocal (about 1 ulp
    // each); the product is rounded to bf16 (or stored fp32 on the fp32 path).
    float v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float g = cs[c0 + j], u = cs[BN / 2 + c0 + j];
      const float sig = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-g * 1.4426950408889634f));
      v[j] = g * sig * u;
    }
    store8(out + (int64_t)row * ldo + (int64_t)bn * (BN / 2) + c0, v);
  }
};

struct EpiStoreF32 {
  static constexpr int out_cols(int BN) { return BN; }
  static constexpr bool kPaired = false;
  float* out; int64_t ldo;
  using stage_t = float;
  template <int BN>
  __device__ void apply(int row, int bn, int c0, const float* cs) const {
    store8(out + (int64_t)row * ldo + (int64_t)bn * BN + c0, cs + c0);
  }
};

// Run the epilogue over 64 staged rows (row stride BN + 4 floats) with NT threads.
template <int BN, class E, int NT = 256>
__device__ __forceinline__ void run_epilogue(const E& e, const float* Cs, int row0, int M, int bn) {
  constexpr int TPR = E::out_cols(BN) / 8;
  constexpr int RPP = NT / TPR;
  const int t = threadIdx.x;
  const int c0 = (t % TPR) * 8;
  for (int r = t / TPR; r < 64; r += RPP) {
    const int row = row0 + r;
    if (row < M) e.template apply<BN>(row, bn, c0, Cs + r * (BN + 4));
  }
}

// Row of B feeding tile column n of column-block bn (fp32 path, 128-wide tiles).
template <bool SWIGLU>
__device__ __forceinline__ int b_row(int bn, int n, int d_ff) {
  if (SWIGLU) return n < 64 ? bn * 64 + n : d_ff + bn * 64 + (n - 64);
  return bn * 128 + n;
}

// --------------------------------------------------------------------------- bf16 MFMA kernels
// Wave layout.  PD: distance in tile columns between the two values an epilogue
// combines (a rotary pair, gate/up).  A wave with NI = 2 P column blocks (P = 1 or
// 2) holds P pairs: pair p is the blocks at c_p and c_p + PD, so each lane holds
// both values in registers.  With PD >= 32 P the first members are contiguous, c_p
// = wcol + 32 p with wcol = (wn / (PD / 32P)) * 2 PD + (wn % (PD / 32P)) * 32 P;
// with PD = 32 < 32 P the pairs are adjacent, c_p = wcol + 64 p, wcol = 128 wn.
// PD = 32 with P = 1 is the plain layout (wave wn: columns 64 wn ..).  Waves with
// three column blocks (NI = 3) take the plain layout, and paired epilogues then
// combine their values from the staged fp32 tile instead.
template <int BM_, int BN_, int BK_, int NWM_, int NWN_, int PD_, class E>
struct TileGeom {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, NWM = NWM_, NWN = NWN_, PD = PD_;
  static constexpr int NW = NWM * NWN, NT = 64 * NW;
  static constexpr int WTM = BM / NWM, WTN = BN / NWN;   // wave tile
  static constexpr int MI = WTM / 32, NI = WTN / 32;     // 32x32 blocks per wave
  static constexpr int CH = BK / 8;                      // 16-byte chunks per tile row
  static constexpr int AS = BM * CH, BS = BN * CH;       // 16-byte slots of one stage's A and B tiles
  static constexpr bool REG_PAIR = E::kPaired && (NI == 2 || NI == 4);   // pairs combined in registers
  static constexpr int NP = NI == 3 ? 1 : NI / 2;                        // pairs per wave
  static constexpr int PSTEP = PD >= 32 * NP ? 32 : 2 * PD;              // column step between pairs
  static_assert(((NI == 2 || NI == 4) && BN % (2 * PD) == 0 && PD % 32 == 0 && (PD >= 32 * NP || PD == 32)) ||
                    (NI == 3 && PD == 32),
                "column blocks");
  // Epilogue staging: register-paired epilogues stage their outputs (type O), the
  // others the fp32 accumulators; rows padded by 4 elements.
  using SO = typename std::conditional<REG_PAIR, typename E::stage_t, float>::type;
  static constexpr int OC = REG_PAIR ? E::out_cols(BN) : BN, SP = OC + 4;
  static constexpr int ROW_BYTES = SP * (int)sizeof(SO);
  // fewest staging rounds (1, 2 or 4, each a whole number of every wave's 32-row
  // blocks) whose rows fit in `bytes`; 0 if none does
  static constexpr int rounds_for(int bytes) {
    return BM * ROW_BYTES <= bytes                        ? 1
           : (MI % 2 == 0 && BM / 2 * ROW_BYTES <= bytes) ? 2
           : (MI % 4 == 0 && BM / 4 * ROW_BYTES <= bytes) ? 4
                                                          : 0;
  }
  // copy instructions per thread and stage (A tile, then B tile or its gate and up halves)
  static constexpr int NA = BM * CH / (64 * NW), NB = BN * CH / (64 * NW), NL = NA + NB;
  static constexpr int NKS = BK / 16;   // k-slices per k-step
  static __device__ __forceinline__ int wave_col(int wn) {
    return NI == 3 ? wn * WTN
                   : (PD >= 32 * NP ? (wn / (PD / (32 * NP))) * (2 * PD) + (wn % (PD / (32 * NP))) * (32 * NP)
                                    : wn * WTN);
  }
  // tile column of column block ni (blocks ni < NP: first members, ni >= NP: partners)
  static __device__ __forceinline__ int colblk(int wcol, int ni) {
    return NI == 3 ? wcol + ni * 32 : wcol + (ni % NP) * PSTEP + (ni / NP) * PD;
  }
};

// The global -> LDS copy sources of one tile: A rows m0.., B rows (or gate and up
// rows) of column block bn.
template <class G, bool SWIGLU>
struct TileCopies {
  TileSrcT<G::BK, G::NW> sa, sb, su;
  __device__ __forceinline__ void init(const bf16_t* A, int64_t lda, const bf16_t* B, int64_t ldb, int d_ff, int m0,
                                       int bn, int w, int lane) {
    sa.init(A + (int64_t)m0 * lda, lda, w, lane);
    if (SWIGLU) {
      sb.init(B + (int64_t)bn * (G::BN / 2) * ldb, ldb, w, lane);
      su.init(B + ((int64_t)d_ff + (int64_t)bn * (G::BN / 2)) * ldb, ldb, w, lane);
    } else {
      sb.init(B + (int64_t)bn * G::BN * ldb, ldb, w, lane);
    }
  }
  // copy j (of NL) of k-step kt into the stage whose A tile is at As and B tile at Bs
  __device__ __forceinline__ void issue_one(int kt, v4u* As, v4u* Bs, int j, int w) const {
    if (j < G::NA) {
      sa.load_round(kt, j, As, w);
    } else if (SWIGLU) {
      const int jb = j - G::NA;
      if (jb < G::NB / 2) sb.load_round(kt, jb, Bs, w);
      else su.load_round(kt, jb - G::NB / 2, Bs + (G::BN / 2) * G::CH, w);
    } else {
      sb.load_round(kt, j - G::NA, Bs, w);
    }
  }
};

// One k-step from the stage (At, Bt): fragments double-buffered in registers; the
// LDS reads of k-slice ks + 1 and this k-step's share of the next copies
// (copy(ks)) are issued ahead of the MFMAs of slice ks.
template <class G, class Copy>
__device__ __forceinline__ void mfma_kstep(f32x16_t (&acc)[G::MI][G::NI], const v4u* At, const v4u* Bt, int wm,
                                           int wcol, int lane, const Copy& copy) {
  constexpr int MI = G::MI, NI = G::NI, CH = G::CH;
  const int l32 = lane & 31;
  bf16x8_t af[2][MI], bfr[2][NI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) af[0][mi] = frag<CH>(At, wm * G::WTM + mi * 32 + l32, 0, lane);
#pragma unroll
  for (int ni = 0; ni < NI; ++ni) bfr[0][ni] = frag<CH>(Bt, G::colblk(wcol, ni) + l32, 0, lane);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int ks = 0; ks < G::NKS; ++ks) {
    const int c = ks & 1;
    if (ks + 1 < G::NKS) {
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) af[c ^ 1][mi] = frag<CH>(At, wm * G::WTM + mi * 32 + l32, ks + 1, lane);
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) bfr[c ^ 1][ni] = frag<CH>(Bt, G::colblk(wcol, ni) + l32, ks + 1, lane);
    }
    copy(ks);
    if constexpr (G::NW != 4) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
        acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[c][ni], af[c][mi], acc[mi][ni], 0, 0, 0);
    if constexpr (G::NW == 4) {
      // one wave per SIMD (no second wave to cover the reads): the next slice's
      // fragment reads go between this slice's MFMAs (scheduling groups)
      if (ks + 1 < G::NKS) {
#pragma unroll
        for (int r = 0; r < MI + NI; ++r) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, MI * NI - (MI + NI), 0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Epilogue of one tile, staged in ROUNDS passes through the LDS at `stage`.  The
// MFMAs take B as the first operand, so acc[mi][ni] is the transposed 32x32 block:
// lane l holds row l % 32 and, in elements 4g..4g+3, the four consecutive columns
// 8 g + 4 (l / 32) .. +3 of the block.  Paired epilogues combine their two blocks
// in registers; the results go through LDS so the global accesses are whole
// rows.  The caller has freed the staging area (barrier) and must place a barrier
// before the area is written again.
template <class G, int ROUNDS, class E>
__device__ __forceinline__ void tile_epilogue(const f32x16_t (&acc)[G::MI][G::NI], v4u* stage, int m0, int bn, int M,
                                              const E& e, int wm, int wcol, int tid) {
  using SO = typename G::SO;
  constexpr int MI = G::MI, NI = G::NI, NP = G::NP, OC = G::OC, SP = G::SP, NT = G::NT, BN = G::BN;
  static_assert(ROUNDS >= 1 && MI % ROUNDS == 0, "staging rounds split each wave's rows evenly");
  const int lane = tid & 63, l32 = lane & 31;
  SO* Cs = reinterpret_cast<SO*>(stage);
  constexpr int WR = G::WTM / ROUNDS, MIR = MI / ROUNDS;   // rows per wave and round, blocks per round
#pragma unroll
  for (int h = 0; h < ROUNDS; ++h) {
    if (h) __syncthreads();   // the previous round has been written out
#pragma unroll
    for (int q = 0; q < MIR; ++q) {
      const int mi = h * MIR + q;
      const int row = m0 + wm * G::WTM + mi * 32 + l32;
      SO* cs = Cs + (wm * WR + q * 32 + l32) * SP;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int q4 = g * 8 + (lane >> 5) * 4;
        if constexpr (G::REG_PAIR) {
#pragma unroll
          for (int pp = 0; pp < NP; ++pp) {
            const int tc = G::colblk(wcol, pp) + q4;
            const f32x16_t& ax = acc[mi][pp];
            const f32x16_t& ay = acc[mi][pp + NP];
            const float4 x = make_float4(ax[4 * g], ax[4 * g + 1], ax[4 * g + 2], ax[4 * g + 3]);
            const float4 y = make_float4(ay[4 * g], ay[4 * g + 1], ay[4 * g + 2], ay[4 * g + 3]);
            float4 o0 = make_float4(0.f, 0.f, 0.f, 0.f), o1 = o0;
            if (row < M) e.template pair<BN>(row, bn, tc, x, y, o0, o1);
            store4(cs + tc, o0);   // SwiGLU: gate columns [0, PD) are the output columns
            if constexpr (E::kOut == 2) store4(cs + tc + G::PD, o1);
          }
        } else {
#pragma unroll
          for (int ni = 0; ni < NI; ++ni)
            store4(cs + G::colblk(wcol, ni) + q4, make_float4(acc[mi][ni][4 * g], acc[mi][ni][4 * g + 1],
                                                              acc[mi][ni][4 * g + 2], acc[mi][ni][4 * g + 3]));
        }
      }
    }
    __syncthreads();
    // staged row r is tile row (r / WR) * WTM + h * WR + r % WR
    if constexpr (G::REG_PAIR) {
      constexpr int CE = 16 / (int)sizeof(SO), CPR = OC / CE, RPP = NT / CPR;
      const int c = (tid % CPR) * CE;
      if (tid < RPP * CPR)
        for (int r = tid / CPR; r < G::BM / ROUNDS; r += RPP) {
          const int row = m0 + (r / WR) * G::WTM + h * WR + r % WR;
          if (row < M) copy16(e.out + (int64_t)row * e.ldo + (int64_t)bn * OC + c, Cs + r * SP + c);
        }
    } else {
      constexpr int TPR = E::out_cols(BN) / 8, RPP = NT / TPR;
      const int c0 = (tid % TPR) * 8;
      if (tid < RPP * TPR)
        for (int r = tid / TPR; r < G::BM / ROUNDS; r += RPP) {
          const int row = m0 + (r / WR) * G::WTM + h * WR + r % WR;
          if (row < M) e.template apply<BN>(row, bn, c0, Cs + r * SP);
        }
    }
  }
}

// One tile per workgroup, a ring of STAGES LDS stages: k-step kt + STAGES - 1 is in
// flight while kt is consumed; the copies of a stage are spread over the k-slices
// of the k-step before it.
template <int BM, int BN, int BK, int NWM, int NWN, int STAGES, int PD, class E, bool SWIGLU>
__global__ __launch_bounds__(64 * NWM * NWN) void gemm_bf16_kernel(const bf16_t* __restrict__ A, int64_t lda,
                                                                  const bf16_t* __restrict__ B, int64_t ldb, int M,
                                                                  int K, int d_ff, int n_bn, int group_m, E e) {
  using G = TileGeom<BM, BN, BK, NWM, NWN, PD, E>;
  constexpr int PIPE = STAGES * (G::AS + G::BS);
  constexpr int ROUNDS = G::rounds_for(160 * 1024);
  static_assert(ROUNDS > 0, "staging");
  constexpr int STG = G::BM / ROUNDS * G::ROW_BYTES / 16;
  static_assert(PIPE * 16 <= 160 * 1024 && STG * 16 <= 160 * 1024, "LDS");
  static_assert(!SWIGLU || G::REG_PAIR, "SwiGLU tiles pair gate and up in registers");
  constexpr int NL = G::NL;
  static_assert(STAGES >= 2 && (STAGES - 2) * NL < 16, "ring depth");
  __shared__ __attribute__((aligned(16))) v4u smem[PIPE > STG ? PIPE : STG];
  v4u* As = smem;
  v4u* Bs = smem + STAGES * G::AS;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w / NWN, wn = w % NWN;
  const int wcol = G::wave_col(wn);
  int bm_, bn;
  xcd_tile((int)blockIdx.x, (M + BM - 1) / BM, n_bn, group_m, &bm_, &bn);
  const int m0 = bm_ * BM;
  TileCopies<G, SWIGLU> src;
  src.init(A, lda, B, ldb, d_ff, m0, bn, w, lane);
  constexpr int PER = (NL + 1) / 2;   // copies issued per k-slice: over the first two slices

  f32x16_t acc[G::MI][G::NI];
#pragma unroll
  for (int mi = 0; mi < G::MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < G::NI; ++ni)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[mi][ni][i] = 0.f;

  const int nk = K / BK;
#pragma unroll
  for (int p = 0; p < STAGES - 1; ++p)
    if (p < nk)
#pragma unroll
      for (int j = 0; j < NL; ++j) src.issue_one(p, As + p * G::AS, Bs + p * G::BS, j, w);
  int cur = 0, nxt = STAGES - 1;
  // The copying k-steps and the last STAGES - 1 (which copy nothing) run as two
  // loops, so each k-slice's reads, copies and MFMAs form one basic block that
  // the compiler schedules as a whole (+2-3% at the Llama-3-8B shapes against a
  // per-k-step test of whether to copy).
  int kt = 0;
  for (; kt + STAGES - 1 < nk; ++kt) {   // steady state: each k-step copies k-step kt + STAGES - 1
    wait_vmem_le<(STAGES - 2) * NL>();
    __syncthreads();   // k-step kt is in LDS for every wave; the slot of kt - 1 is free
    mfma_kstep<G>(acc, As + cur * G::AS, Bs + cur * G::BS, wm, wcol, lane, [&](int ks) {
#pragma unroll
      for (int j = ks * PER; j < (ks + 1) * PER; ++j)
        if (j < NL) src.issue_one(kt + STAGES - 1, As + nxt * G::AS, Bs + nxt * G::BS, j, w);
    });
    cur = cur == STAGES - 1 ? 0 : cur + 1;
    nxt = nxt == STAGES - 1 ? 0 : nxt + 1;
  }
  for (; kt < nk; ++kt) {   // the last STAGES - 1 k-steps copy nothing
    wait_vmem();
    __syncthreads();
    mfma_kstep<G>(acc, As + cur * G::AS, Bs + cur * G::BS, wm, wcol, lane, [&](int) {});
    cur = cur == STAGES - 1 ? 0 : cur + 1;
  }
  __syncthreads();   // the staging area overlaps the ring
  tile_epilogue<G, ROUNDS>(acc, smem, m0, bn, M, e, wm, wcol, tid);
}

// --------------------------------------------------------------------------- fp32 VALU kernel
template <class E, bool SWIGLU>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, int64_t lda,
                                                       const float* __restrict__ B, int64_t ldb, int M, int K,
                                                       int d_ff, E e) {
  __shared__ __attribute__((aligned(16))) float smem[64 * kCsStride];
  static_assert(kCsStride == 128 + 4, "fp32 path stages 128-wide tiles");
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
    // blocked summation: each 16-wide k-chunk in a fresh partial, then added to
    // the running sum, so the rounding error grows with K / 16 + 16 terms, not K
    float part[4][8];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) part[i][j] = 0.f;
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
        for (int j = 0; j < 8; ++j) part[i][j] = fmaf(av[i], bv[j], part[i][j]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[i][j] += part[i][j];
  }
  __syncthreads();
  float* Cs = smem;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) Cs[(ty * 4 + i) * kCsStride + tx * 8 + j] = acc[i][j];
  __syncthreads();
  run_epilogue<128>(e, Cs, m0, M, bn);
}

// --------------------------------------------------------------------------- dispatch
// Tile choice (measured on MI355X over the decoder's projection shapes): a
// 256x256 tile on 8 waves (2x4, 128x64 per wave) wherever it divides N and
// yields at least half a wave of tiles; otherwise 128x128 on 4 waves.
static int cu_count() {
  static int n = 0;
  if (n == 0) {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) == hipSuccess && hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
      n = v;
    else
      n = 256;
  }
  return n;
}

static void pick_tile(const GemmArgs& a, bool swiglu, int* bm, int* bn_, int* bk, int* waves, int* stages) {
  const int ncu = cu_count();
  const int64_t nm = (a.M + 255) / 256;
  const bool fits256 = swiglu ? (a.d_ff % 128 == 0) : (a.N % 256 == 0);
  // 192-wide tiles have three column blocks per wave, so their rotary pairs would
  // go through the staged tile: measured slower than 256-wide tiles for q|k|v
  const bool fits192 = !swiglu && a.N % 192 == 0 && a.epi != Epi::kStoreRope;
  const int64_t tiles256 = fits256 ? nm * (a.N / 256) : 0, tiles192 = fits192 ? nm * (a.N / 192) : 0;
  // fewer than half a wave of large tiles on the CUs (small M, e.g. window rows): 128x128 tiles
  if (a.K % 64 == 0 && std::max(tiles256, tiles192) >= ncu / 2) {
    // the 256-row tile whose last round of workgroups wastes least: cost = rounds x tile area
    const int64_t c256 = fits256 ? (tiles256 + ncu - 1) / ncu * 256 : INT64_MAX;
    const int64_t c192 = fits192 ? (tiles192 + ncu - 1) / ncu * 192 : INT64_MAX;
    *bm = 256; *bn_ = c192 < c256 ? 192 : 256; *bk = 64; *waves = 8; *stages = 2;
    return;
  }
  *bm = 128; *bn_ = 128; *bk = 64; *waves = 4; *stages = 2;
}

template <int BM, int BN, int BK, int ST, int PD, class E, bool SWIGLU, int NWM, int NWN>
static void go_pd(const GemmArgs& a, const E& e, hipStream_t s) {
  const int nbn = SWIGLU ? a.d_ff / (BN / 2) : a.N / BN;
  const int nbm = (a.M + BM - 1) / BM;
  // tile-rows per L2 group: 4 for the long-K projections of the 8B-scale models
  // (1-2% faster than 8 on q|k|v, output and down at 32768 rows, equal on
  // gate|up), 8 for short K
  const int group_m = a.group_m > 0 ? a.group_m : (a.K >= 4096 ? 4 : 8);
  gemm_bf16_kernel<BM, BN, BK, NWM, NWN, ST, PD, E, SWIGLU><<<nbm * nbn, 64 * NWM * NWN, 0, s>>>(
      (const bf16_t*)a.A, a.lda, (const bf16_t*)a.B, a.ldb, a.M, a.K, a.d_ff, nbn, group_m, e);
}

// the pair distance each epilogue needs (plain layout when it pairs nothing)
template <int BM, int BN, int BK, int ST, class E, bool SWIGLU, int NWM = 2, int NWN = 2>
static hipError_t go_bf16(const GemmArgs& a, const E& e, hipStream_t s) {
  constexpr int WTN = BN / NWN;
  if constexpr (WTN != 64 && WTN != 128) {   // three column blocks per wave: pairs via the staged tile
    if constexpr (SWIGLU) {
      return hipErrorInvalidValue;   // SwiGLU needs the paired layout
    } else {
      if (E::kPaired && BN % a.head_dim != 0) return hipErrorInvalidValue;   // rotary pairs inside the tile
      go_pd<BM, BN, BK, ST, 32, E, SWIGLU, NWM, NWN>(a, e, s);
    }
  } else if constexpr (!E::kPaired) {
    go_pd<BM, BN, BK, ST, 32, E, SWIGLU, NWM, NWN>(a, e, s);
  } else if constexpr (SWIGLU) {
    go_pd<BM, BN, BK, ST, BN / 2, E, SWIGLU, NWM, NWN>(a, e, s);
  } else {
    if (a.head_dim == 64) go_pd<BM, BN, BK, ST, 32, E, SWIGLU, NWM, NWN>(a, e, s);
    else if (a.head_dim == 128) go_pd<BM, BN, BK, ST, 64, E, SWIGLU, NWM, NWN>(a, e, s);
    else return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class E, bool SWIGLU>
static hipError_t go(const GemmArgs& a, bool bf16, const E& e, hipStream_t s) {
  if (bf16) {
    int bm, bn, bk, waves, st;
    pick_tile(a, SWIGLU, &bm, &bn, &bk, &waves, &st);
    if (a.tile_m) {
      bm = a.tile_m; bn = a.tile_n; bk = a.tile_k ? a.tile_k : 64; waves = a.tile_waves ? a.tile_waves : 4;
      st = a.tile_stages ? a.tile_stages : 2;
    }
#define RK_TILE(BM_, BN_, BK_, W_, ST_, NWM_, NWN_)                                     \
  if (bm == BM_ && bn == BN_ && bk == BK_ && waves == W_ && st == ST_)                  \
    return go_bf16<BM_, BN_, BK_, ST_, E, SWIGLU, NWM_, NWN_>(a, e, s);
    // each wave: two 32-column blocks (BN = 64 NWN) or three (BN = 96 NWN, not SwiGLU)
    RK_TILE(256, 256, 64, 8, 2, 2, 4)
    RK_TILE(256, 192, 64, 8, 2, 4, 2)
    RK_TILE(256, 256, 32, 8, 3, 2, 4)
    RK_TILE(256, 256, 32, 8, 4, 2, 4)
    RK_TILE(128, 128, 64, 4, 2, 2, 2)
    RK_TILE(128, 128, 64, 4, 3, 2, 2)
#undef RK_TILE
    return hipErrorInvalidValue;
  } else {
    const int nbn = SWIGLU ? a.d_ff / 64 : a.N / 128;
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
        EpiRope<bf16_t> e{(bf16_t*)a.out, a.ldo, a.rope_cols, a.head_dim, a.rope_tab, a.rope_pos, a.q_cols, a.q_scale};
        return go<EpiRope<bf16_t>, false>(a, true, e, s);
      } else {
        EpiRope<float> e{(float*)a.out, a.ldo, a.rope_cols, a.head_dim, a.rope_tab, a.rope_pos, a.q_cols, a.q_scale};
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
