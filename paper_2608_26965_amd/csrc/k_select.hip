// Cluster assignment (paper: Method, Cluster assignment - scoring and top-k
// selection).
//
// scores[a][b] = qbar_a . kbar_b in fp32 (fixed summation order, so scores are
// reproducible); lists[a] = the k key clusters of largest score, ties to the
// lower index, in ascending order. The selection is an exact radix select on
// order-preserving integer images of the scores (four 8-bit digit passes),
// followed by an order-keeping compaction; it makes no floating-point
// decision of its own, so given the scores the lists are exact.
#include "common.h"

namespace ca {

namespace {

constexpr int kTileS = 64;  // score tile edge

// S tile of 64 x 64 for one head: each thread accumulates a 4 x 4 block over d.
__global__ __launch_bounds__(256) void scores_kernel(const float* __restrict__ cq,
                                                     const float* __restrict__ ck, int nqc,
                                                     int nkc, int d, float* __restrict__ S) {
  __shared__ float A[kTileS][kMaxD + 1];
  __shared__ float B[kTileS][kMaxD + 1];
  const int bh = blockIdx.z, a0 = blockIdx.y * kTileS, b0 = blockIdx.x * kTileS;
  const float* qh = cq + (size_t)bh * nqc * d;
  const float* kh = ck + (size_t)bh * nkc * d;
  for (int e = threadIdx.x; e < kTileS * d; e += 256) {
    const int r = e / d, t = e % d;
    A[r][t] = (a0 + r < nqc) ? qh[(size_t)(a0 + r) * d + t] : 0.f;
    B[r][t] = (b0 + r < nkc) ? kh[(size_t)(b0 + r) * d + t] : 0.f;
  }
  __syncthreads();
  const int tr = (threadIdx.x / 16) * 4, tc = (threadIdx.x % 16) * 4;
  float acc[4][4] = {};
  for (int t = 0; t < d; ++t) {
    float x[4], y[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[i] = A[tr + i][t];
      y[i] = B[tc + i][t];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fmaf(x[i], y[j], acc[i][j]);
  }
  float* Sh = S + (size_t)bh * nqc * nkc;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int a = a0 + tr + i, b = b0 + tc + j;
      if (a < nqc && b < nkc) Sh[(size_t)a * nkc + b] = acc[i][j];
    }
}

// Key that orders scores descending: the largest score gets the smallest key.
__device__ __forceinline__ uint32_t desc_key(float s) { return ~ordered_bits(s); }

// Exclusive scan of one int per thread over a 256-thread block; returns the
// exclusive prefix and writes the block total.
__device__ __forceinline__ int block_scan_256(int x, int* sh_warp, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int v = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(v, o, 64);
    if (lane >= o) v += y;
  }
  if (lane == 63) sh_warp[w] = v;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (i < w) base += sh_warp[i];
    tot += sh_warp[i];
  }
  __syncthreads();
  *total = tot;
  return base + v - x;
}

// One row (head, query cluster) per block: exact top-k of S[row][0..nkc).
__global__ __launch_bounds__(256) void topk_kernel(const float* __restrict__ S, int nkc, int k,
                                                   int32_t* __restrict__ lists) {
  __shared__ int hist[256];
  __shared__ int sh_warp[4];
  __shared__ uint32_t sh_prefix;
  __shared__ int sh_rank;
  const size_t row = blockIdx.x;
  const float* s = S + row * nkc;
  const int tid = threadIdx.x;

  // Radix select of the k-th smallest key (rank k-1), most significant digit first.
  uint32_t prefix = 0;
  int rank = k - 1;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    const uint32_t hmask = pass == 0 ? 0u : (0xFFFFFFFFu << (shift + 8));
    hist[tid] = 0;
    __syncthreads();
    for (int b = tid; b < nkc; b += 256) {
      const uint32_t u = desc_key(s[b]);
      if ((u & hmask) == prefix) atomicAdd(&hist[(u >> shift) & 255], 1);
    }
    __syncthreads();
    if (tid < 64) {
      // Wave 0 finds the digit whose cumulative count passes `rank`.
      int c[4], sum = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        c[i] = hist[4 * tid + i];
        sum += c[i];
      }
      int incl = sum;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        int y = __shfl_up(incl, o, 64);
        if (tid >= o) incl += y;
      }
      int before = incl - sum;
      if (rank >= before && rank < incl) {
        int acc = before;
        for (int i = 0; i < 4; ++i) {
          if (rank < acc + c[i]) {
            sh_prefix = prefix | ((uint32_t)(4 * tid + i) << shift);
            sh_rank = rank - acc;
            break;
          }
          acc += c[i];
        }
      }
    }
    __syncthreads();
    prefix = sh_prefix;
    rank = sh_rank;
  }
  // prefix = threshold key; `rank` equal keys precede the k-th in index order,
  // so the first rank+1 keys equal to the threshold are taken.
  const uint32_t thr = prefix;
  const int need_eq = rank + 1;
  const int per = (nkc + 255) / 256;
  const int lo = min(nkc, tid * per), hi = min(nkc, lo + per);
  int eq = 0;
  for (int b = lo; b < hi; ++b) eq += desc_key(s[b]) == thr;
  int tot;
  const int eq_before = block_scan_256(eq, sh_warp, &tot);
  int sel = 0, er = eq_before;
  for (int b = lo; b < hi; ++b) {
    const uint32_t u = desc_key(s[b]);
    if (u < thr) {
      ++sel;
    } else if (u == thr) {
      sel += er < need_eq;
      ++er;
    }
  }
  const int sel_before = block_scan_256(sel, sh_warp, &tot);
  int32_t* out = lists + row * k;
  int pos = sel_before;
  er = eq_before;
  for (int b = lo; b < hi; ++b) {
    const uint32_t u = desc_key(s[b]);
    bool take = false;
    if (u < thr) {
      take = true;
    } else if (u == thr) {
      take = er < need_eq;
      ++er;
    }
    if (take && pos < k) out[pos++] = b;
  }
}

}  // namespace

hipError_t launch_select(const Prob& P, const float* cq, const float* ck, const float* scores_in,
                         float* scores, int k, int32_t* lists, hipStream_t st) {
  const float* S = scores_in;
  if (!S) {
    dim3 grid((P.nkc + kTileS - 1) / kTileS, (P.nqc + kTileS - 1) / kTileS, P.BH);
    hipLaunchKernelGGL(scores_kernel, grid, dim3(256), 0, st, cq, ck, P.nqc, P.nkc, P.d, scores);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    S = scores;
  } else if (scores && scores != scores_in) {
    hipError_t e = hipMemcpyAsync(scores, scores_in, (size_t)P.BH * P.nqc * P.nkc * 4,
                                  hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(topk_kernel, dim3((unsigned)((size_t)P.BH * P.nqc)), dim3(256), 0, st, S,
                     P.nkc, k, lists);
  return hipGetLastError();
}

}  // namespace ca
