// Block-tile machinery shared by the bf16 GEMM-shaped kernels (projections and
// the LM head): tiles of A[M, K] and B[N, K] (K contiguous) are streamed straight
// from global memory into LDS with buffer_load_dwordx4 ... lds (no staging registers)
// and consumed by v_mfma_f32_32x32x16_bf16.
//
// LDS tile layout: a BR x BK bf16 tile is BR rows of CH = BK / 8 16-byte chunks;
// chunk kc of row r sits at slot r*CH + (kc ^ swz<CH>(r)).  A fragment read
// (32 lanes reading one k-chunk of 32 consecutive rows) is serviced 16 lanes at
// a time by 64 banks of 4 bytes, so the 16 rows of a quarter-wave must cover
// all 16 bank quads: with 128-byte rows (CH = 8) two rows share a bank line and
// the chunk is XORed with bits 1-3 of the row, with 64-byte rows (CH = 4) four
// rows share it and bits 2-3 are used.  One wave instruction fills 64
// consecutive slots (lane l -> slot base + l, as the hardware places them).
//
// Callers guarantee that all BR rows of every tile are readable (activation
// buffers are padded to a multiple of 256 rows; weight row counts are multiples
// of the tile), so the loads need no clamping.
#pragma once

#include "rk_internal.h"

namespace rk {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_void;
typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));

constexpr int kBK = 64;  // default K elements per pipeline stage


__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// s_waitcnt vmcnt(N) for N < 64 (gfx9 encoding: vmcnt bits 3:0 and 15:14; expcnt and
// lgkmcnt left at their maximum)
template <int N>
__device__ __forceinline__ void wait_vmem_le() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// Chunk swizzle of a tile row with CH 16-byte chunks (CH = BK / 8).
template <int CH>
__device__ __forceinline__ int swz(int row) {
  return CH == 8 ? ((row >> 1) & 7) : ((row >> 2) & 3);
}

// Per-lane source of a BR x BK tile whose rows start at `rows0` (row stride ld
// elements).  One wave instruction fills 64 consecutive slots = 64 / CH rows;
// round j of wave w covers rows (NW j + w) * (64 / CH) ...  The copies are
// buffer_load_dwordx4 ... lds with the tile's base in an SGPR descriptor, a
// per-lane 32-bit offset fixed at init, and the k-step and round in the scalar
// offset, so issuing one costs no vector ALU work.  They are inline assembly:
// the compiler neither counts them in its own waits nor orders later LDS reads
// behind them, so callers wait with s_waitcnt vmcnt and a barrier themselves.
template <int BK = kBK, int NW = 4>
struct TileSrcT {
  static constexpr int CH = BK / 8;
  static constexpr int RPI = 64 / CH;  // rows per wave instruction
  i32x4_t rsrc;
  uint32_t voff;
  int32_t round_bytes;
  __device__ __forceinline__ void init(const bf16_t* rows0, int64_t ld, int w, int lane) {
    const int r = w * RPI + lane / CH;
    const int kc = (lane % CH) ^ swz<CH>(r);   // rounds add multiples of 16 rows: same swizzle
    const uint64_t base = (uint64_t)rows0;
    rsrc[0] = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)base);
    rsrc[1] = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)(base >> 32));
    rsrc[2] = -1;            // no range limit: callers keep every row readable
    rsrc[3] = 0x00020000;    // raw buffer, 32-bit data format (gfx9 word 3)
    voff = (uint32_t)(r * ld * 2 + kc * 16);
    round_bytes = __builtin_amdgcn_readfirstlane((int32_t)(NW * RPI * ld * 2));
  }
  // round j (j < BR * CH / (64 NW)) of k-step kt into the tile at dst
  __device__ __forceinline__ void load_round(int kt, int j, v4u* dst, int w) const {
    const uint32_t lds = __builtin_amdgcn_readfirstlane(
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) v4u*)(dst + (j * NW + w) * 64));
    const int32_t soff = __builtin_amdgcn_readfirstlane(kt * (BK * 2) + j * round_bytes);
    asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
                 :
                 : "v"(voff), "s"(rsrc), "s"(soff), "{m0}"(lds)
                 : "memory");
  }
  // issue the k-step kt of a BR-row tile (NW waves, BR * CH / (64 NW) rounds)
  template <int BR>
  __device__ __forceinline__ void load(int kt, v4u* dst, int w) const {
    static_assert(BR * CH % (64 * NW) == 0, "tile rows must fill whole rounds");
#pragma unroll
    for (int j = 0; j < BR * CH / (64 * NW); ++j) load_round(kt, j, dst, w);
  }
};
typedef TileSrcT<kBK, 4> TileSrc;

// One 32x16 (or 16x32) bf16 fragment of row `row`, k-slice ks, from a swizzled tile.
template <int CH = 8>
__device__ __forceinline__ bf16x8_t frag(const v4u* tile, int row, int ks, int lane) {
  const int ch = ks * 2 + (lane >> 5);
  return __builtin_bit_cast(bf16x8_t, tile[row * CH + (ch ^ swz<CH>(row))]);
}

// Tile order for a 1-D grid of n_m x n_n tiles on 8 XCDs.  The dispatcher hands
// workgroup g to XCD g % 8, so g is first renumbered to make each XCD's
// workgroups a contiguous run of tile ids, and tile ids are then laid out in
// groups of `group_m` tile-rows (column-major inside a group): the tiles one XCD
// runs at the same time share a few A row-panels and B column-panels in its L2.
__device__ __forceinline__ void xcd_tile(int g, int n_m, int n_n, int group_m, int* bm, int* bn) {
  const int total = n_m * n_n;
  const int q = total >> 3, r = total & 7;
  const int xcd = g & 7, local = g >> 3;
  const int t = xcd < r ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
  const int per_group = group_m * n_n;
  const int first = (t / per_group) * group_m;
  const int gm = min(group_m, n_m - first);
  const int in = t - (t / per_group) * per_group;
  *bm = first + in % gm;
  *bn = in / gm;
}

}  // namespace rk
