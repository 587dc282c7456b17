// Causal grouped-query attention of one decoder block (Section 4.1), reading the
// (possibly perturbed) Values of the q|k|v buffer: o = softmax(q k^T / sqrt(d_h)) v
// with key u visible from query t iff u <= t; query head hq reads KV head
// hq / (H / H_kv).  With the Keys fixed the attention weights of the perturbed
// layer equal the clean ones (Section 4.3); only the aggregated Values change.
//
// bf16 kernel (flash attention, fp32 online softmax in base 2):
//   * the queries arrive pre-multiplied by log2(e) / sqrt(d_h) (the q|k|v
//     projection's epilogue does it before rounding), so a score is already
//     the exponent of 2;
//   * one workgroup = 4 waves (d_h 64) or 8 waves (d_h 128) x 32 queries of one
//     head; it runs a pair of query blocks (nqb - 1 - x, then x) so all pairs of
//     a sequence cost the same, longest sequences first (one block per workgroup
//     when the rows sit behind a cached prefix, which every block reads in full);
//   * 64-key tiles of K and V go global -> LDS by buffer_load ... lds (no
//     staging registers; rows past the sequence read as zero) through a
//     ring of 2-3 stages;
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16 with the accumulator started at
//     -m (the running max), so each lane owns one query column and exp2 is
//     applied to the MFMA result directly; m is raised lazily (only when a
//     tile's max exceeds it by 2^8), with one exchange with the partner
//     half-wave (v_permlane32_swap); the two 32-key halves of a tile run as two
//     interleaved accumulator chains;
//   * O^T = V^T P^T: P^T is the lane's own S^T registers rounded to bf16, and
//     the V^T operand comes from the row-major V tile through ds_read_b64_tr_b16
//     in the same key order; the softmax denominator is summed from the rounded
//     P with v_dot2_f32_bf16, so the weights applied to V sum to one;
//   * masks only on diagonal / ragged tiles;
//   * the K fragment reads of a tile are issued up to six ahead of the MFMAs
//     that consume them (scheduling groups), not each right before its use.
// fp32 kernel: one thread per (row, head), streaming keys; for the small fp32
// model only.
#include <math.h>

#include <algorithm>

#include "rk_internal.h"

namespace rk {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4;

// A score may exceed the running max by up to 2^kLazy before m is raised.
constexpr float kLazy = 8.0f;

typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));

// 16-byte global -> LDS copy of one wave (lane l lands at lds_base + 16 l); rows
// past the descriptor's range read as zero.  Issued as inline assembly so the
// compiler does not tie later LDS reads of the other buffer to it: the caller
// waits with s_waitcnt vmcnt(0) and a barrier before the data is read.
__device__ __forceinline__ void dma16(i32x4_t rsrc, uint32_t lds_base, uint32_t voff, int32_t soff) {
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               :
               : "v"(voff), "s"(rsrc), "s"(soff), "{m0}"(lds_base)
               : "memory");
}

// s_waitcnt vmcnt(0) (gfx9 encoding: expcnt and lgkmcnt fields at their maximum)
// as a builtin, so the compiler also knows that its own earlier loads are done
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }
// s_waitcnt vmcnt(N), N < 16
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

// 16-byte chunk swizzles that keep the LDS reads free of bank conflicts (64
// banks of 4 bytes): the K tile is read as 16 rows x one chunk per quarter-wave,
// the V tile by ds_read_b64_tr_b16 as 4 rows x 4 chunks per half-wave.
template <int DH>
__device__ __forceinline__ int k_swz(int row) { return DH == 128 ? (row & 15) : ((row >> 1) & 7); }
template <int DH>
__device__ __forceinline__ int v_swz(int row) { return DH == 128 ? ((row & 3) << 2) : (((row >> 1) & 1) << 2); }

// max / sum of a lane's value and that of lane l ^ 32 (the other half-wave):
// v_permlane32_swap with both operands x hands lanes 0-31 the upper half's x and
// lanes 32-63 the lower half's, each keeping its own in the other result.
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Workgroup shape per head size.  d_h = 64: 4 waves (128 queries), a three-stage
// K/V ring (prefetch two tiles ahead), three workgroups per CU.  d_h = 128: 8 waves
// (256 queries) share one two-stage ring, one workgroup per CU (two waves per SIMD
// either way; the wider group halves the copies per query).
template <int DH>
struct AttnTraits {
  static constexpr int kWaves = DH == 64 ? 4 : 8;
  static constexpr int kStages = DH == 64 ? 3 : 2;
  static constexpr int kMinBlocks = DH == 64 ? 3 : 1;
};

template <int DH, bool PREFIX>
__global__ __launch_bounds__(64 * AttnTraits<DH>::kWaves, AttnTraits<DH>::kMinBlocks) void attn_bf16_kernel(const bf16_t* __restrict__ qkv, int64_t ldq,
                                                        bf16_t* __restrict__ out, int64_t ldo, SeqTable st,
                                                        AttnWork wk, int H, int Hkv, int n_items, KvPrefix pk) {
  constexpr int NW = AttnTraits<DH>::kWaves;
  constexpr int BQ = 32 * NW, BKV = 64;
  constexpr int CH = DH / 8;                // 16-byte chunks per row
  constexpr int NKS = DH / 16;              // k-steps of S^T
  constexpr int NDB = DH / 32;              // 32-row blocks of O^T
  constexpr int SLOTS = BKV * CH;           // 16-byte slots per tile
  constexpr int NLD = SLOTS / (64 * NW);    // DMA instructions per thread, per tile and matrix
  constexpr int ROWB = DH * 2;              // bytes per tile row
  constexpr int S = AttnTraits<DH>::kStages;
  __shared__ __attribute__((aligned(16))) v4u Ks[S][SLOTS];
  __shared__ __attribute__((aligned(16))) v4u Vs[S][SLOTS];

  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hf = lane >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  // ---- work item: XCD-grouped so the query heads of one KV head share an L2
  const int grp = H / Hkv;
  int t_item;
  {
    const int g = blockIdx.x, x = g & 7, n = g >> 3;
    t_item = (n / grp) * (8 * grp) + x * grp + n % grp;
  }
  if (t_item >= n_items) return;
  const int item = t_item / H, hq = t_item - item * H, hk = hq / grp;
  int j = 0;
  {
    int lo = 0, hi = st.n - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (wk.cum[mid] <= item) lo = mid; else hi = mid - 1;
    }
    j = lo;
  }
  const int k = wk.order[j], x = item - wk.cum[j];
  const int row0 = st.off[k], T = st.off[k + 1] - row0;
  const int nqb = (T + BQ - 1) / BQ;

  // buffer descriptor over this sequence's rows (raw, stride 0): reads past row T - 1 return zero
  auto make_rsrc = [](const bf16_t* base_ptr, int64_t bytes) {
    i32x4_t r;
    const uint64_t base = (uint64_t)base_ptr;
    r[0] = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)base);
    r[1] = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)(base >> 32));
    r[2] = __builtin_amdgcn_readfirstlane((int32_t)bytes);
    r[3] = 0x00020000;
    return r;
  };
  const i32x4_t rsrc = make_rsrc(qkv + (int64_t)row0 * ldq, (int64_t)T * ldq * 2);
  const int kcol = (H + hk) * DH, vcol = (H + Hkv + hk) * DH;
  uint32_t koff[NLD], voff[NLD];
#pragma unroll
  for (int i = 0; i < NLD; ++i) {
    const int slot = (i * NW + w) * 64 + lane, r = slot / CH, ph = slot % CH;
    koff[i] = (uint32_t)(r * ldq * 2 + (kcol + (ph ^ k_swz<DH>(r)) * 8) * 2);
    voff[i] = (uint32_t)(r * ldq * 2 + (vcol + (ph ^ v_swz<DH>(r)) * 8) * 2);
  }
  // cached prefix of this sequence (PREFIX): rows k * P .. k * P + P - 1 of the K and V caches
  const int P = PREFIX ? pk.P : 0;
  i32x4_t rk_p = rsrc, rv_p = rsrc;
  uint32_t koff_p[PREFIX ? NLD : 1], voff_p[PREFIX ? NLD : 1];
  int64_t ldv_p = pk.ldv;
  if constexpr (PREFIX) {
    // the prefix of this sequence (of sequence k % n_seq when several passes share a launch)
    const int ps = pk.n_seq > 0 ? k % pk.n_seq : k;
    const bool alt = pk.n_seq > 0 && k / pk.n_seq == pk.alt_pass;
    const bf16_t* vb = alt ? pk.v_alt : pk.v;
    ldv_p = alt ? pk.ldv_alt : pk.ldv;
    rk_p = make_rsrc(pk.k + (int64_t)ps * P * pk.ldk, (int64_t)P * pk.ldk * 2);
    rv_p = make_rsrc(vb + (int64_t)ps * P * ldv_p, (int64_t)P * ldv_p * 2);
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int slot = (i * NW + w) * 64 + lane, r = slot / CH, ph = slot % CH;
      koff_p[i] = (uint32_t)(r * pk.ldk * 2 + (hk * DH + (ph ^ k_swz<DH>(r)) * 8) * 2);
      voff_p[i] = (uint32_t)(r * ldv_p * 2 + (hk * DH + (ph ^ v_swz<DH>(r)) * 8) * 2);
    }
  }
  const int n_pre = (P + BKV - 1) / BKV;   // prefix tiles, visited before the window's own
  const uint32_t ks_lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) v4u*)&Ks[0][0];
  const uint32_t vs_lds = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) v4u*)&Vs[0][0];
  // tile t: prefix tile t (t < n_pre), else the sequence's own tile t - n_pre
  auto issue = [&](int t, int b) {
    if (PREFIX && t < n_pre) {
      const int sk = __builtin_amdgcn_readfirstlane(t * BKV * (int)pk.ldk * 2);
      const int sv = __builtin_amdgcn_readfirstlane(t * BKV * (int)ldv_p * 2);
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        const uint32_t o = (uint32_t)((b * SLOTS + (i * NW + w) * 64) * 16);
        dma16(rk_p, __builtin_amdgcn_readfirstlane(ks_lds + o), koff_p[i], sk);
        dma16(rv_p, __builtin_amdgcn_readfirstlane(vs_lds + o), voff_p[i], sv);
      }
    } else {
      const int so = __builtin_amdgcn_readfirstlane((t - n_pre) * BKV * (int)ldq * 2);
#pragma unroll
      for (int i = 0; i < NLD; ++i) {
        const uint32_t o = (uint32_t)((b * SLOTS + (i * NW + w) * 64) * 16);
        dma16(rsrc, __builtin_amdgcn_readfirstlane(ks_lds + o), koff[i], so);
        dma16(rsrc, __builtin_amdgcn_readfirstlane(vs_lds + o), voff[i], so);
      }
    }
  };

  // per-lane LDS byte offsets of the K fragments (row l32 of a 32-row block, chunk 2 ks + hf)
  // and of the V^T fragments (ds_read_b64_tr_b16: lane (G, jj) reads row 4 (G / 2) + jj / 4
  // of an 8-row group, columns db * 32 + 16 (G % 2) + 4 (jj % 4))
  int kfo[NKS];
#pragma unroll
  for (int ks = 0; ks < NKS; ++ks) kfo[ks] = l32 * ROWB + (((2 * ks + hf) ^ k_swz<DH>(l32)) << 4);
  int vfo[NDB];
  {
    const int G = lane >> 4, jj = lane & 15, r = 4 * (G >> 1) + (jj >> 2);
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int ch = 4 * db + 2 * (G & 1) + ((jj & 3) >> 1);
      vfo[db] = r * ROWB + ((ch ^ v_swz<DH>(r)) << 4) + (jj & 1) * 8;
    }
  }

  const bf16x2_t ones = {(__bf16)1.0f, (__bf16)1.0f};
  // causal rows: the pair (nqb - 1 - x, x); behind a cached prefix every q-block
  // costs about the same, so one q-block per item
  const int n_blocks = PREFIX ? 1 : ((x == nqb - 1 - x) ? 1 : 2);
  for (int bi = 0; bi < n_blocks; ++bi) {
    const int qb = (PREFIX || bi == 0) ? nqb - 1 - x : x;
    const int q0 = qb * BQ;
    const int my_q = min(q0 + w * 32 + l32, T - 1);   // rows past T duplicate row T - 1
    bf16x8_t qf[NKS];
    {
      const bf16_t* qp = qkv + (int64_t)(row0 + my_q) * ldq + (int64_t)hq * DH + hf * 8;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks)
        qf[ks] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const v4u*>(qp + ks * 16));
    }
    const int kv_end = min(T, q0 + BQ);
    const int n_tiles = n_pre + (kv_end + BKV - 1) / BKV;
    const int wave_qmin = q0 + w * 32, wave_qmax = wave_qmin + 31;

    f32x16_t o[NDB], negm;
#pragma unroll
    for (int i = 0; i < 16; ++i) negm[i] = 0.f;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[db][i] = 0.f;
    float l_run = 0.f;

    wait_vm0();   // the query fragments are in registers before the ring starts
#pragma unroll
    for (int p = 0; p < S - 1; ++p)
      if (p < n_tiles) issue(p, p);
    int buf = 0, nbuf = S - 1;   // ring slots of tile t and of tile t + S - 1
    for (int t = 0; t < n_tiles; ++t) {
      const bool pre = PREFIX && t < n_pre;
      const int k0 = (pre ? t : t - n_pre) * BKV;   // first key of the tile within its segment
      // tile t has landed once at most the S - 2 later tiles are in flight
      if (t + S - 2 < n_tiles) wait_vm<(S - 2) * 2 * NLD>(); else wait_vm0();
      __syncthreads();   // ... for every wave; and tile t - 1's slot is free again
      if (t + S - 1 < n_tiles) issue(t + S - 1, nbuf);
      if (pre || k0 <= wave_qmax) {
        const char* kt = reinterpret_cast<const char*>(Ks[buf]);
        f32x16_t s[2] = {negm, negm};
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks)
#pragma unroll
          for (int rb = 0; rb < 2; ++rb) {
            const bf16x8_t a = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const v4u*>(kt + rb * 32 * ROWB + kfo[ks]));
            s[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[ks], s[rb], 0, 0, 0);
          }
        {
          // schedule: the K fragment reads run up to three MFMA pairs ahead of their
          // MFMAs (the compiler's own order waits on each read right before its use)
          constexpr int AHEAD = NKS >= 8 ? 6 : 4, N = 2 * NKS;
          __builtin_amdgcn_sched_group_barrier(0x100, AHEAD, 0);   // LDS reads
#pragma unroll
          for (int p = 0; p < (N - AHEAD) / 2; ++p) {
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);     // MFMAs
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
          }
          __builtin_amdgcn_sched_group_barrier(0x008, AHEAD, 0);
        }
        // masks only where a key can exceed the query or the segment (wave-uniform test);
        // every cached prefix key precedes every query of the sequence's own rows
        if (pre ? (k0 + BKV > P) : (k0 + BKV - 1 > wave_qmin || k0 + BKV > T)) {
          const int qlim = pre ? P - 1 : my_q, klim = pre ? P : T;
#pragma unroll
          for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
              const int key = k0 + rb * 32 + (i >> 2) * 8 + hf * 4 + (i & 3);
              if (key > qlim || key >= klim) s[rb][i] = -INFINITY;
            }
        }
        float mx = fmaxf(s[0][0], s[0][1]);
#pragma unroll
        for (int i = 2; i < 16; i += 2) mx = fmaxf(mx, fmaxf(s[0][i], s[0][i + 1]));
#pragma unroll
        for (int i = 0; i < 16; i += 2) mx = fmaxf(mx, fmaxf(s[1][i], s[1][i + 1]));
        mx = max_halves(mx);
        if (t == 0 || __any(mx > kLazy)) {
          // raise the running max: by the tile max on the first tile, else where it grew past 2^kLazy
          const float dm = (t == 0 || mx > kLazy) ? mx : 0.f;
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            s[0][i] -= dm;
            s[1][i] -= dm;
            negm[i] -= dm;
          }
          if (t != 0) {
            const float corr = __builtin_amdgcn_exp2f(-dm);
            l_run *= corr;
#pragma unroll
            for (int db = 0; db < NDB; ++db)
#pragma unroll
              for (int i = 0; i < 16; ++i) o[db][i] *= corr;
          }
        }
        const char* vt = reinterpret_cast<const char*>(Vs[buf]);
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
          for (int ss = 0; ss < 2; ++ss) {
            bf16x8_t pb;
#pragma unroll
            for (int e = 0; e < 8; ++e) pb[e] = (__bf16)__builtin_amdgcn_exp2f(s[rb][8 * ss + e]);
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
              const bf16x2_t pr = {pb[e], pb[e + 1]};
              l_run = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, l_run, false);
            }
            // k-slot hf * 8 + e of this MFMA is key rb*32 + ss*16 + 8 (e / 4) + 4 hf + e % 4
            const int kr = (rb * 32 + ss * 16) * ROWB;
#pragma unroll
            for (int db = 0; db < NDB; ++db) {
              const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vt + kr + vfo[db]));
              const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(vt + kr + 8 * ROWB + vfo[db]));
              const v4u vv = {__builtin_bit_cast(v2u, lo)[0], __builtin_bit_cast(v2u, lo)[1],
                              __builtin_bit_cast(v2u, hi)[0], __builtin_bit_cast(v2u, hi)[1]};
              o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, vv), pb, o[db], 0, 0, 0);
            }
          }
      }
      buf = buf == S - 1 ? 0 : buf + 1;
      nbuf = nbuf == S - 1 ? 0 : nbuf + 1;
    }
    __syncthreads();   // the next q-block refills the ring

    const float l = sum_halves(l_run);
    const float inv = 1.0f / l;
    const int q_out = q0 + w * 32 + l32;
    if (q_out < T) {
      bf16_t* op = out + (int64_t)(row0 + q_out) * ldo + (int64_t)hq * DH;
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
                            int n_kv_heads, int head_dim, bool bf16, hipStream_t s, const KvPrefix* prefix) {
  if (st.rows <= 0) return hipSuccess;
  if (bf16) {
    // sequences by decreasing length; items = pairs of q-blocks
    AttnWork wk;
    for (int k = 0; k < st.n; ++k) wk.order[k] = k;
    for (int a = 1; a < st.n; ++a) {  // insertion sort, stable
      const int v = wk.order[a], len = st.off[v + 1] - st.off[v];
      int b = a;
      while (b > 0 && st.off[wk.order[b - 1] + 1] - st.off[wk.order[b - 1]] < len) {
        wk.order[b] = wk.order[b - 1];
        --b;
      }
      wk.order[b] = v;
    }
    const bool pre = prefix && prefix->P > 0;
    const int bq = 32 * (head_dim == 64 ? AttnTraits<64>::kWaves : AttnTraits<128>::kWaves);   // queries per block
    wk.cum[0] = 0;
    for (int j = 0; j < st.n; ++j) {
      const int k = wk.order[j], nqb = (st.off[k + 1] - st.off[k] + bq - 1) / bq;
      wk.cum[j + 1] = wk.cum[j] + (pre ? nqb : (nqb + 1) / 2);
    }
    wk.total = wk.cum[st.n];
    if (wk.total == 0) return hipSuccess;
    // the buffer descriptor covers one sequence's rows with 32-bit byte offsets
    if ((int64_t)st.max_len * ldq * 2 >= ((int64_t)1 << 31) || n_heads % n_kv_heads != 0) return hipErrorInvalidValue;
    const int grp = n_heads / n_kv_heads;
    const int n_items = wk.total * n_heads;
    const int grid = (n_items + 8 * grp - 1) / (8 * grp) * (8 * grp);
    KvPrefix pk{};
    if (pre) {
      pk = *prefix;
      // one descriptor per sequence's cached prefix, also with 32-bit byte offsets
      const int64_t ld = std::max(std::max(pk.ldk, pk.ldv), pk.alt_pass >= 0 && pk.n_seq > 0 ? pk.ldv_alt : 0);
      if ((int64_t)pk.P * ld * 2 >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
      if (pk.n_seq > 0 && (st.n % pk.n_seq != 0 || (pk.alt_pass >= 0 && !pk.v_alt))) return hipErrorInvalidValue;
    }
#define RK_ATTN(D, PRE)                                                                                      \
  attn_bf16_kernel<D, PRE><<<grid, 64 * AttnTraits<D>::kWaves, 0, s>>>((const bf16_t*)qkv, ldq, (bf16_t*)out, ldo, \
                                                                      st, wk, n_heads, n_kv_heads, n_items, pk)
    if (head_dim == 128) { if (pre) RK_ATTN(128, true); else RK_ATTN(128, false); }
    else if (head_dim == 64) { if (pre) RK_ATTN(64, true); else RK_ATTN(64, false); }
    else return hipErrorInvalidValue;
#undef RK_ATTN
  } else {
    if (prefix && prefix->P > 0) return hipErrorInvalidValue;   // cached prefixes: bf16 path only
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
