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

__device__ __forceinline__ bf16x8 pack8(const float* v) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = f2bf(v[i]);
  return r;
}

}  // namespace ca
