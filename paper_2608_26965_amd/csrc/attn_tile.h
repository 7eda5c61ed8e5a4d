// Device building blocks shared by the block-sparse attention kernel and the
// compensation kernel: one wavefront owns 32 queries and streams 32*MT-key tiles
// through an online softmax on bf16 MFMA (v_mfma_f32_32x32x16_bf16).
//
// Products are formed transposed: S^T = K Q^T (keys on the MFMA rows, queries
// on the columns), so a lane's accumulators hold many keys of ONE query and the
// softmax max/sum stay in the lane (plus one exchange with lane^32). The value
// product is O^T = V^T P^T, whose output again puts one query per lane, so the
// rescale by the running max needs no cross-lane traffic either.
//
// MFMA 32x32 output layout (per lane l, accumulator r = 0..15):
//   row = 8*(r/4) + 4*(l/32) + r%4,   column = l%32.
// For the P^T operand of the value product a lane must own 8 keys that are
// consecutive in the V^T tile. The rows a lane owns in one 16-row half are
// {4h..4h+3, 8+4h..8+4h+3} (h = l/32); feeding K row kswz(i) to MFMA row i,
// with kswz swapping the middle two groups of four in every 16, maps them to
// the consecutive keys 8h..8h+7.
#pragma once

#include "common.h"

namespace ca {

__device__ __forceinline__ int kswz(int i) {
  int o = i & 15;
  int g = o >> 2;
  int g2 = (g == 1) ? 2 : (g == 2 ? 1 : g);
  return (i & ~15) | (g2 << 2) | (o & 3);
}

// Physical key (within the tile) held by accumulator r of row-tile mt in a lane
// of half h.
__device__ __forceinline__ int acc_key(int mt, int r, int h) {
  int rho = 8 * (r >> 2) + 4 * h + (r & 3);
  return 32 * mt + kswz(rho);
}

__device__ __forceinline__ float wave_xor32(float x) {
  return __shfl_xor(x, 32, 64);
}

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;

// Eight floats to bf16 with the hardware round-to-nearest-even conversion.
__device__ __forceinline__ bf16x8 pack8(const float* v) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const f32x2 f = {v[i], v[i + 1]};
    const bf16x2 b = __builtin_convertvector(f, bf16x2);
    r[i] = b[0];
    r[i + 1] = b[1];
  }
  return r;
}

// Sum of the eight bf16 values of a packed operand, accumulated in fp32.
__device__ __forceinline__ float sum8(bf16x8 p, float acc) {
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const bf16x2 q = {p[i], p[i + 1]};
    acc = __builtin_amdgcn_fdot2_f32_bf16(q, one, acc, false);
  }
  return acc;
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void wait_lgkm() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void raw_barrier() { asm volatile("s_barrier" ::: "memory"); }

// One direct global-to-LDS copy of 16 bytes per lane (global_load_lds_dwordx4
// with an SGPR base and a 32-bit per-lane byte offset): lane i writes LDS bytes
// [lds + 16 i, lds + 16 i + 16). Issued as inline assembly so that the compiler
// does not treat later LDS reads of the other pipeline stage as dependent on
// it; completion is awaited explicitly with s_waitcnt vmcnt. M0 (the LDS base
// of the copy) is saved and restored, with one wait state between writing M0
// and the copy.
__device__ __forceinline__ void lds_dma16(const void* gbase, uint32_t voff, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %2\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(voff), "s"(gbase), "s"(lds)
      : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const void __attribute__((address_space(3)))*)p);
}

// XOR swizzle of the 16-byte chunks of an LDS tile row, chosen so that the
// operand reads of the MFMA kernels (32 rows in the K-row order of kswz, or 32
// consecutive rows) hit distinct banks whether the hardware serves a
// ds_read_b128 in groups of 8 lanes over 128 bytes or of 16 lanes over 256
// bytes. Row r stores its logical chunk lc at chunk lc ^ swz_key(r).
template <int ROWBYTES>
__device__ __forceinline__ int swz_key(int r) {
  static_assert(ROWBYTES == 128 || ROWBYTES == 256, "row width");
  constexpr uint64_t tbl = ROWBYTES == 128 ? 0x1706352453427160ull : 0xba987654fedc3210ull;
  return (int)((tbl >> ((r & 15) * 4)) & 15);
}

// Byte offset of logical 16-byte chunk lc of row r in a swizzled LDS tile.
template <int ROWBYTES>
__device__ __forceinline__ int swz_off(int r, int lc) {
  return r * ROWBYTES + ((lc ^ swz_key<ROWBYTES>(r)) << 4);
}

// Per-lane global byte offsets of a tile copy: wavefront w's instruction i
// fills LDS bytes [(i*NW + w)*1024, +1024); lane l writes 16 of them, which
// belong to row r, LDS chunk pc, i.e. to the row's logical chunk
// pc ^ swz_key(r) in global memory, where rows are GROWBYTES apart (a tile
// may be a column range of wider rows).
template <int ROWBYTES, int NINSTR, int NW, int GROWBYTES = ROWBYTES>
struct TileCopy {
  uint32_t off[NINSTR];
  __device__ __forceinline__ TileCopy(int w, int lane) {
    constexpr int NCH = ROWBYTES / 16;
#pragma unroll
    for (int i = 0; i < NINSTR; ++i) {
      const int g = (i * NW + w) * 64 + lane;
      const int r = g / NCH, pc = g % NCH;
      off[i] = (uint32_t)(r * GROWBYTES + ((pc ^ swz_key<ROWBYTES>(r)) << 4));
    }
  }
  __device__ __forceinline__ void issue(const void* src, uint32_t lds, int w) const {
#pragma unroll
    for (int i = 0; i < NINSTR; ++i)
      lds_dma16(src, off[i], __builtin_amdgcn_readfirstlane(lds + (uint32_t)((i * NW + w) * 1024)));
  }
};

}  // namespace ca
