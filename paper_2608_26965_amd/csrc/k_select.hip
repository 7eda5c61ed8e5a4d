// Cluster assignment (paper: Method, Cluster assignment - scoring, top-k
// selection and the two-pass histogram selection).
//
// scores[a][b] = qbar_a . kbar_b in fp32 (fixed summation order, so scores are
// reproducible; bf16 problems with d = 64 or 128 form them on the matrix
// cores from a three-term bf16 split of the fp32 centroids); lists[a] = the k key clusters of largest score, ties to the
// lower index, in ascending order. The selection is an exact radix select on
// order-preserving integer images of the scores (four 8-bit digit passes),
// followed by an order-keeping compaction; it makes no floating-point
// decision of its own, so given the scores the lists are exact.
#include <algorithm>

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

// Centroid scores on the matrix cores (bf16 problems, d = 64 or 128). Each
// fp32 operand x is split into hi = bf16(x) and lo = bf16(x - hi), and
// S = lo_q hi_k + hi_q lo_k + hi_q hi_k is accumulated in fp32 (the dropped
// lo_q lo_k term is about 2^-16 of each product), so the scores keep close to
// fp32 accuracy at the bf16 MFMA rate. Per 128 x 128 tile of one head: wave
// w owns query rows 32 w .. 32 w + 31 and takes the four 32-column key blocks
// in turn. v_mfma_f32_32x32x16_bf16 with the query rows
// as the A operand and the key rows as B: lane l holds key column l % 32 of
// the output block and query rows 8 (r / 4) + 4 (l / 32) + r % 4, so each
// store instruction writes two 128-byte row segments.
__device__ __forceinline__ void split_hilo(const float4 x0, const float4 x1, bf16x8& hi,
                                           bf16x8& lo) {
  const float v[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const bf16 h = (bf16)v[i];
    hi[i] = h;
    lo[i] = (bf16)(v[i] - (float)h);
  }
}

// A workgroup takes 128 query clusters against up to eight blocks of 128
// key clusters (jb_per_wg). Each key block is split into bf16 hi / lo once
// per workgroup and staged in LDS (rows padded by 16 bytes, so the 32 rows
// one operand read touches fall in distinct banks) while the next block's
// fp32 rows are loaded into registers.
template <int D>
__global__ __launch_bounds__(256) void scores_lds_kernel(const float* __restrict__ cq,
                                                         const float* __restrict__ ck, int nqc,
                                                         int nkc, int jb_per_wg,
                                                         float* __restrict__ S) {
  constexpr int KS = D / 16;
  constexpr int RW = 2 * D + 8;  // bf16 per LDS row: hi, lo, padding
  constexpr int NF4 = D / 8;     // float4 loads per thread and block (half a row)
  __shared__ __attribute__((aligned(16))) __bf16 kt[128 * RW];
  const int bh = blockIdx.z, a0 = blockIdx.y * 128;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const float* qh = cq + (size_t)bh * nqc * D;
  const float* kh = ck + (size_t)bh * nkc * D;
  const int arow = a0 + 32 * w + l32;
  bf16x8 qhi[KS], qlo[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    float4 x0 = make_float4(0.f, 0.f, 0.f, 0.f), x1 = x0;
    if (arow < nqc) {
      const float4* src = (const float4*)(qh + (size_t)arow * D + 16 * ks + 8 * h);
      x0 = src[0];
      x1 = src[1];
    }
    split_hilo(x0, x1, qhi[ks], qlo[ks]);
  }
  // thread t stages half hf of key row r of a block
  const int r = tid >> 1, hf = tid & 1;
  float4 pf[NF4];
  auto load_block = [&](int b0) __attribute__((always_inline)) {
    const int row = b0 + r;
#pragma unroll
    for (int i = 0; i < NF4; ++i) {
      pf[i] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (row < nkc) pf[i] = *(const float4*)(kh + (size_t)row * D + hf * (D / 2) + 4 * i);
    }
  };
  float* Sh = S + (size_t)bh * nqc * nkc;
  const int bfirst = blockIdx.x * jb_per_wg * 128;
  const int bend = min(nkc, bfirst + jb_per_wg * 128);
  load_block(bfirst);
  for (int b0 = bfirst; b0 < bend; b0 += 128) {
    __syncthreads();  // every wavefront is done with the previous block
#pragma unroll
    for (int i = 0; i < NF4; i += 2) {
      bf16x8 hi8, lo8;
      split_hilo(pf[i], pf[i + 1], hi8, lo8);
      *(bf16x8*)&kt[r * RW + hf * (D / 2) + 4 * i] = hi8;
      *(bf16x8*)&kt[r * RW + D + hf * (D / 2) + 4 * i] = lo8;
    }
    __syncthreads();
    if (b0 + 128 < bend) load_block(b0 + 128);
#pragma unroll 1
    for (int j = 0; j < 4; ++j) {
      if (b0 + 32 * j >= nkc) break;  // uniform
      const int bcol = b0 + 32 * j + l32;
      const __bf16* kr = &kt[(32 * j + l32) * RW];
      bf16x8 khi[KS], klo[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        khi[ks] = *(const bf16x8*)(kr + 16 * ks + 8 * h);
        klo[ks] = *(const bf16x8*)(kr + D + 16 * ks + 8 * h);
      }
      f32x16 acc;
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[q] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qlo[ks], khi[ks], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qhi[ks], klo[ks], acc, 0, 0, 0);
      }
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qhi[ks], khi[ks], acc, 0, 0, 0);
      if (bcol < nkc) {
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int a = a0 + 32 * w + 8 * (q >> 2) + 4 * h + (q & 3);
          if (a < nqc) Sh[(size_t)a * nkc + bcol] = acc[q];
        }
      }
    }
  }
}

// Scores of every (query cluster, key cluster) pair of every head.
hipError_t launch_scores(const Prob& P, const float* cq, const float* ck, float* scores,
                         hipStream_t st) {
  const bool aligned = (((uintptr_t)cq | (uintptr_t)ck) & 15) == 0;
  if (P.dtype == CA_BF16 && (P.d == 64 || P.d == 128) && aligned) {
    // key blocks per workgroup: up to eight, while the launch keeps at
    // least 2048 workgroups
    const int nb = (P.nkc + 127) / 128, nr = (P.nqc + 127) / 128;
    const long wgs = (long)nb * nr * P.BH;
    const int jb = (int)std::max(1L, std::min(8L, wgs / 2048));
    const dim3 grid((nb + jb - 1) / jb, nr, P.BH);
    if (P.d == 64)
      hipLaunchKernelGGL(scores_lds_kernel<64>, grid, dim3(256), 0, st, cq, ck, P.nqc, P.nkc, jb,
                         scores);
    else
      hipLaunchKernelGGL(scores_lds_kernel<128>, grid, dim3(256), 0, st, cq, ck, P.nqc, P.nkc, jb,
                         scores);
  } else {
    const dim3 grid((P.nkc + kTileS - 1) / kTileS, (P.nqc + kTileS - 1) / kTileS, P.BH);
    hipLaunchKernelGGL(scores_kernel, grid, dim3(256), 0, st, cq, ck, P.nqc, P.nkc, P.d, scores);
  }
  return hipGetLastError();
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

__device__ __forceinline__ float block_min_max(float v, bool want_max, float* sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float y = __shfl_xor(v, o, 64);
    v = want_max ? fmaxf(v, y) : fminf(v, y);
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) sh[w] = v;
  __syncthreads();
  float r = sh[0];
#pragma unroll
  for (int i = 1; i < 4; ++i) r = want_max ? fmaxf(r, sh[i]) : fminf(r, sh[i]);
  __syncthreads();
  return r;
}

constexpr int kTopBins = 2048;  // linear bins of the top-k pre-pass

// One row (head, query cluster) per block: exact top-k of S[row][0..nkc).
// A pre-pass counts the row into linear bins over [min, max] (descending
// score; the map is monotone, so the k-th largest lies in one bin and every
// key of a lower bin precedes it); the radix select then only counts that
// bin's keys, which keeps the LDS atomics of long rows from piling onto the
// few digits a narrow score range has in common. Rows longer than 8192
// scores take this kernel; shorter ones the wave and block kernels below.
__global__ __launch_bounds__(256) void topk_kernel(const float* __restrict__ S, int nkc, int k,
                                                   int32_t* __restrict__ lists) {
  __shared__ int hist[256];
  __shared__ int bins[kTopBins];
  __shared__ int sh_warp[4];
  __shared__ float sh_f[4];
  __shared__ uint32_t sh_prefix;
  __shared__ int sh_rank, sh_bin;
  const size_t row = blockIdx.x;
  const int tid = threadIdx.x;
  const float* s = S + row * nkc;

  float lo = INFINITY, hi = -INFINITY;
  for (int b = tid; b < nkc; b += 256) {
    lo = fminf(lo, s[b]);
    hi = fmaxf(hi, s[b]);
  }
  lo = block_min_max(lo, false, sh_f);
  hi = block_min_max(hi, true, sh_f);
  // (a range too narrow for a finite bin scale puts every score in bin 0)
  const float inv0 = (float)kTopBins / (hi - lo);
  const float inv = hi > lo && inv0 < INFINITY ? inv0 : 0.f;
  auto bin_of = [&](float v) {
    const float t = (hi - v) * inv;  // 0 for the largest score
    return t < (float)kTopBins ? (t > 0.f ? (int)t : 0) : kTopBins - 1;
  };
  for (int i = tid; i < kTopBins; i += 256) bins[i] = 0;
  __syncthreads();
  for (int b = tid; b < nkc; b += 256) atomicAdd(&bins[bin_of(s[b])], 1);
  __syncthreads();
  {
    constexpr int PB = kTopBins / 256;
    int c[PB], sum = 0;
#pragma unroll
    for (int i = 0; i < PB; ++i) {
      c[i] = bins[PB * tid + i];
      sum += c[i];
    }
    int tot;
    int before = block_scan_256(sum, sh_warp, &tot);
    if (k - 1 >= before && k - 1 < before + sum) {
#pragma unroll
      for (int i = 0; i < PB; ++i) {
        if (k - 1 < before + c[i]) {
          sh_bin = PB * tid + i;
          sh_rank = k - 1 - before;
          break;
        }
        before += c[i];
      }
    }
    __syncthreads();
  }
  const int B = sh_bin;

  // Radix select of the wanted key inside bin B, most significant digit first.
  uint32_t prefix = 0;
  int rank = sh_rank;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    const uint32_t hmask = pass == 0 ? 0u : (0xFFFFFFFFu << (shift + 8));
    hist[tid] = 0;
    __syncthreads();
    for (int b = tid; b < nkc; b += 256) {
      const float v = s[b];
      if (bin_of(v) != B) continue;
      const uint32_t u = desc_key(v);
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
  const int b_lo = min(nkc, tid * per), b_hi = min(nkc, b_lo + per);
  int eq = 0;
  for (int b = b_lo; b < b_hi; ++b) eq += desc_key(s[b]) == thr;
  int tot;
  const int eq_before = block_scan_256(eq, sh_warp, &tot);
  int sel = 0, er = eq_before;
  for (int b = b_lo; b < b_hi; ++b) {
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
  for (int b = b_lo; b < b_hi; ++b) {
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

// Exact top-k of rows of at most 64 * VPL scores, one row per wavefront, the
// row held in registers (lane l owns the VPL consecutive scores from VPL * l),
// so no block barrier is needed. The same selection as topk_kernel: linear
// bins over [min, max] locate the bin holding the k-th largest score; that
// bin's scores are compacted into a per-wave LDS list (ballot positions) and
// an 8-bit radix select finds the k-th key among them (or among the bin's
// scores in registers when more than kWaveCand fall in it); the first rank+1
// keys equal to it in index order are kept.
constexpr int kWaveBins = 1024;
constexpr int kWaveCand = 512;

__device__ __forceinline__ void wave_lds_sync() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// Radix passes a candidate set can skip: every key between the smallest and
// the largest shares their common leading bytes, so the byte passes over
// those would only confirm them. Returns how many leading bytes are common
// (4: all keys equal) and sets prefix to them.
__device__ __forceinline__ int common_bytes(uint32_t kmin, uint32_t kmax, uint32_t* prefix) {
  const uint32_t x = kmin ^ kmax;
  const int n = x == 0u ? 4 : __builtin_clz(x) / 8;
  *prefix = n == 0 ? 0u : (n == 4 ? kmin : kmin & (0xFFFFFFFFu << (32 - 8 * n)));
  return n;
}

__device__ __forceinline__ int wave_incl_scan(int x, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

template <int VPL>
__global__ __launch_bounds__(256) void topk_wave_kernel(const float* __restrict__ S, int nkc, int k,
                                                        int nrows, int vec4,
                                                        int32_t* __restrict__ lists) {
  __shared__ int bins_all[4][kWaveBins];
  __shared__ int hist_all[4][256];
  __shared__ uint32_t ckey_all[4][kWaveCand];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const size_t row = (size_t)blockIdx.x * 4 + w;
  if (row >= (size_t)nrows) return;  // whole wavefront; no block barrier follows
  int* bins = bins_all[w];
  int* hist = hist_all[w];
  uint32_t* ckey = ckey_all[w];
  const float* s = S + row * nkc;
  const int b0 = VPL * lane;
  float v[VPL];
  if (vec4 && VPL >= 4) {
#pragma unroll
    for (int j = 0; j < VPL; j += 4) {
      float4 x = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      if (b0 + j < nkc) x = *(const float4*)(s + b0 + j);  // nkc % 4 == 0: whole float4
      v[j] = x.x;
      v[j + 1] = x.y;
      v[j + 2] = x.z;
      v[j + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < VPL; ++j) v[j] = b0 + j < nkc ? s[b0 + j] : -INFINITY;
  }
  // Positions past the row hold -inf: they sort after every score (last bin,
  // largest key, and indices after the row's), so with k <= nkc they are never
  // taken; only the range below has to leave them out.
  float lo = INFINITY, hi = -INFINITY;
#pragma unroll
  for (int j = 0; j < VPL; ++j)
    if (b0 + j < nkc) {
      lo = fminf(lo, v[j]);
      hi = fmaxf(hi, v[j]);
    }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    lo = fminf(lo, __shfl_xor(lo, o, 64));
    hi = fmaxf(hi, __shfl_xor(hi, o, 64));
  }
  const float inv0 = (float)kWaveBins / (hi - lo);
  const float inv = hi > lo && inv0 < INFINITY ? inv0 : 0.f;  // too narrow: one bin
  auto bin_of = [&](float x) {
    const float t = (hi - x) * inv;  // 0 for the largest score
    return t < (float)kWaveBins ? (t > 0.f ? (int)t : 0) : kWaveBins - 1;
  };
  for (int i = lane; i < kWaveBins; i += 64) bins[i] = 0;
  wave_lds_sync();
#pragma unroll
  for (int j = 0; j < VPL; ++j) atomicAdd(&bins[bin_of(v[j])], 1);
  wave_lds_sync();
  // Each pass recomputes bins and keys from the scores: keeping them from an
  // earlier pass would hold two more registers per score.
  auto fence_row = [&]() {
#pragma unroll
    for (int j = 0; j < VPL; ++j) asm volatile("" : "+v"(v[j]));
  };
  fence_row();
  // the bin holding rank k - 1 (bins in descending score order)
  int B, rank;
  {
    constexpr int PB = kWaveBins / 64;
    int sum = 0;
#pragma unroll
    for (int i = 0; i < PB; ++i) sum += bins[PB * lane + i];
    const int incl = wave_incl_scan(sum, lane);
    const bool mine = k - 1 >= incl - sum && k - 1 < incl;
    const int owner = __ffsll((long long)__ballot(mine)) - 1;
    int fb = 0, fr = 0;
    if (mine) {
      int acc = incl - sum;
      for (int i = 0; i < PB; ++i) {
        const int c = bins[PB * lane + i];
        if (k - 1 < acc + c) {
          fb = PB * lane + i;
          fr = k - 1 - acc;
          break;
        }
        acc += c;
      }
    }
    B = __builtin_amdgcn_readlane(fb, owner);
    rank = __builtin_amdgcn_readlane(fr, owner);
  }
  // candidates: the keys of bin B (and their smallest and largest key)
  int ncand = 0;
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const bool hit = bin_of(v[j]) == B;
    const uint64_t m = __ballot(hit);
    const int pos = ncand + (int)__popcll(m & ((1ull << lane) - 1ull));
    const uint32_t u = desc_key(v[j]);
    if (hit) {
      if (pos < kWaveCand) ckey[pos] = u;
      kmin = min(kmin, u);
      kmax = max(kmax, u);
    }
    ncand += (int)__popcll(m);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, o, 64));
    kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, o, 64));
  }
  wave_lds_sync();
  fence_row();
  const bool in_lds = ncand <= kWaveCand;
  uint32_t prefix;
  const int p0 = common_bytes(kmin, kmax, &prefix);
  for (int pass = p0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    const uint32_t hmask = pass == 0 ? 0u : (0xFFFFFFFFu << (shift + 8));
    for (int i = lane; i < 256; i += 64) hist[i] = 0;
    wave_lds_sync();
    if (in_lds) {
      for (int i = lane; i < ncand; i += 64) {
        const uint32_t u = ckey[i];
        if ((u & hmask) == prefix) atomicAdd(&hist[(u >> shift) & 255], 1);
      }
    } else {
#pragma unroll
      for (int j = 0; j < VPL; ++j)
        if (bin_of(v[j]) == B) {
          const uint32_t u = desc_key(v[j]);
          if ((u & hmask) == prefix) atomicAdd(&hist[(u >> shift) & 255], 1);
        }
    }
    wave_lds_sync();
    int c[4], sum = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      c[i] = hist[4 * lane + i];
      sum += c[i];
    }
    const int incl = wave_incl_scan(sum, lane);
    const bool mine = rank >= incl - sum && rank < incl;
    const int owner = __ffsll((long long)__ballot(mine)) - 1;
    int fd = 0, fr = 0;
    if (mine) {
      int acc = incl - sum;
      for (int i = 0; i < 4; ++i) {
        if (rank < acc + c[i]) {
          fd = 4 * lane + i;
          fr = rank - acc;
          break;
        }
        acc += c[i];
      }
    }
    prefix |= (uint32_t)__builtin_amdgcn_readlane(fd, owner) << shift;
    rank = __builtin_amdgcn_readlane(fr, owner);
    wave_lds_sync();  // hist is cleared again by the next pass
    fence_row();
  }
  // keys below the threshold, and the first rank + 1 equal ones in index order
  fence_row();
  const uint32_t thr = prefix;
  const int need_eq = rank + 1;
  int less = 0, eq = 0;
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const uint32_t u = desc_key(v[j]);
    less += u < thr;
    eq += u == thr;
  }
  fence_row();
  const int eq_before = wave_incl_scan(eq, lane) - eq;
  const int sel = less + min(max(need_eq - eq_before, 0), eq);
  int pos = wave_incl_scan(sel, lane) - sel;
  int er = eq_before;
  int32_t* out = lists + row * k;
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const uint32_t u = desc_key(v[j]);
    bool take = u < thr;
    if (u == thr) take = er++ < need_eq;
    if (take && pos < k) out[pos++] = b0 + j;
  }
}

// Exact top-k of rows of up to 64 * VPL * NWV scores, one row per block of NWV
// wavefronts (for rows too wide for one wavefront's registers). Wave w owns
// the contiguous range [64 VPL w, 64 VPL (w + 1)) of the row, read as
// float4s interleaved over the lanes (lane l holds positions
// 64 VPL w + 256 g + 4 l + e, g < VPL / 4, e < 4), so every load instruction
// reads 1 KB of consecutive scores. The selection is that of topk_wave_kernel
// (linear bins over [min, max], candidates of the k-th's bin, 8-bit radix
// select on order-preserving keys, ties to the lower index) with the
// histograms shared by the block; the output is written in index order.
template <int VPL, int NWV>
__global__ __launch_bounds__(64 * NWV, 4) void topk_block_kernel(const float* __restrict__ S, int nkc,
                                                              int k, int vec4,
                                                              int32_t* __restrict__ lists) {
  constexpr int NT = 64 * NWV, G = VPL / 4;
  static_assert(VPL % 4 == 0, "float4 groups");
  __shared__ int bins[kWaveBins];
  __shared__ int hist[256];
  __shared__ uint32_t ckey[NWV][kWaveCand];
  __shared__ float red_lo[NWV], red_hi[NWV];
  __shared__ int wcnt[2][NWV];
  __shared__ uint32_t wkey[2][NWV];
  __shared__ int sh_over;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, tid = threadIdx.x;
  const size_t row = blockIdx.x;
  const float* s = S + row * nkc;
  const int wbase = 64 * VPL * w;
  auto pos_of = [&](int g, int e) { return wbase + 256 * g + 4 * lane + e; };
  float v[VPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int p0 = pos_of(g, 0);
    if (vec4) {
      float4 x = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      if (p0 < nkc) x = *(const float4*)(s + p0);  // nkc % 4 == 0: whole float4
      v[4 * g] = x.x;
      v[4 * g + 1] = x.y;
      v[4 * g + 2] = x.z;
      v[4 * g + 3] = x.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[4 * g + e] = p0 + e < nkc ? s[p0 + e] : -INFINITY;
    }
  }
  // Positions past the row hold -inf (sorted after every score); only the
  // range below leaves them out.
  float lo = INFINITY, hi = -INFINITY;
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (pos_of(g, e) < nkc) {
        lo = fminf(lo, v[4 * g + e]);
        hi = fmaxf(hi, v[4 * g + e]);
      }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    lo = fminf(lo, __shfl_xor(lo, o, 64));
    hi = fmaxf(hi, __shfl_xor(hi, o, 64));
  }
  if (lane == 0) {
    red_lo[w] = lo;
    red_hi[w] = hi;
  }
  for (int i = tid; i < kWaveBins; i += NT) bins[i] = 0;
  __syncthreads();
#pragma unroll
  for (int i = 0; i < NWV; ++i) {
    lo = fminf(lo, red_lo[i]);
    hi = fmaxf(hi, red_hi[i]);
  }
  const float inv0 = (float)kWaveBins / (hi - lo);
  const float inv = hi > lo && inv0 < INFINITY ? inv0 : 0.f;  // too narrow: one bin
  auto bin_of = [&](float x) {
    const float t = (hi - x) * inv;  // 0 for the largest score
    return t < (float)kWaveBins ? (t > 0.f ? (int)t : 0) : kWaveBins - 1;
  };
#pragma unroll
  for (int j = 0; j < VPL; ++j) atomicAdd(&bins[bin_of(v[j])], 1);
  __syncthreads();
  // the bin holding rank k - 1 (every wavefront finds the same)
  int B, rank;
  {
    constexpr int PB = kWaveBins / 64;
    int sum = 0;
#pragma unroll
    for (int i = 0; i < PB; ++i) sum += bins[PB * lane + i];
    const int incl = wave_incl_scan(sum, lane);
    const bool mine = k - 1 >= incl - sum && k - 1 < incl;
    const int owner = __ffsll((long long)__ballot(mine)) - 1;
    int fb = 0, fr = 0;
    if (mine) {
      int acc = incl - sum;
      for (int i = 0; i < PB; ++i) {
        const int c = bins[PB * lane + i];
        if (k - 1 < acc + c) {
          fb = PB * lane + i;
          fr = k - 1 - acc;
          break;
        }
        acc += c;
      }
    }
    B = __builtin_amdgcn_readlane(fb, owner);
    rank = __builtin_amdgcn_readlane(fr, owner);
  }
  // candidates of bin B: each wavefront compacts its own into its segment
  // (and finds their smallest and largest key)
  int ncand = 0;
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const bool hit = bin_of(v[j]) == B;
    const uint64_t m = __ballot(hit);
    const int pos = ncand + (int)__popcll(m & ((1ull << lane) - 1ull));
    const uint32_t u = desc_key(v[j]);
    if (hit) {
      if (pos < kWaveCand) ckey[w][pos] = u;
      kmin = min(kmin, u);
      kmax = max(kmax, u);
    }
    ncand += (int)__popcll(m);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, o, 64));
    kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, o, 64));
  }
  if (tid == 0) sh_over = 0;
  __syncthreads();
  if (lane == 0) {
    if (ncand > kWaveCand) sh_over = 1;
    wkey[0][w] = kmin;
    wkey[1][w] = kmax;
  }
  __syncthreads();
  const bool in_lds = sh_over == 0;
#pragma unroll
  for (int i = 0; i < NWV; ++i) {
    kmin = min(kmin, wkey[0][i]);
    kmax = max(kmax, wkey[1][i]);
  }
  uint32_t prefix;
  const int p0 = common_bytes(kmin, kmax, &prefix);
  for (int pass = p0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    const uint32_t hmask = pass == 0 ? 0u : (0xFFFFFFFFu << (shift + 8));
    for (int i = tid; i < 256; i += NT) hist[i] = 0;
    __syncthreads();
    if (in_lds) {
      for (int i = lane; i < ncand; i += 64) {
        const uint32_t u = ckey[w][i];
        if ((u & hmask) == prefix) atomicAdd(&hist[(u >> shift) & 255], 1);
      }
    } else {
#pragma unroll
      for (int j = 0; j < VPL; ++j)
        if (bin_of(v[j]) == B) {
          const uint32_t u = desc_key(v[j]);
          if ((u & hmask) == prefix) atomicAdd(&hist[(u >> shift) & 255], 1);
        }
    }
    __syncthreads();
    int c[4], sum = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      c[i] = hist[4 * lane + i];
      sum += c[i];
    }
    const int incl = wave_incl_scan(sum, lane);
    const bool mine = rank >= incl - sum && rank < incl;
    const int owner = __ffsll((long long)__ballot(mine)) - 1;
    int fd = 0, fr = 0;
    if (mine) {
      int acc = incl - sum;
      for (int i = 0; i < 4; ++i) {
        if (rank < acc + c[i]) {
          fd = 4 * lane + i;
          fr = rank - acc;
          break;
        }
        acc += c[i];
      }
    }
    prefix |= (uint32_t)__builtin_amdgcn_readlane(fd, owner) << shift;
    rank = __builtin_amdgcn_readlane(fr, owner);
    __syncthreads();  // hist is cleared again by the next pass
  }
  // keys below the threshold, and the first rank + 1 equal ones in index
  // order: counts per wavefront first, then per float4 group in lane order
  const uint32_t thr = prefix;
  const int need_eq = rank + 1;
  // Per wavefront: keys equal to the threshold and keys below it; it selects
  // those below and its share of the first need_eq equal ones in index order
  // (equal ranks eq_run .. eq_run + eq_w - 1), so one exchange of the two
  // counts gives every wavefront its base in the list.
  int eq_w = 0, lt_w = 0;
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const uint32_t u = desc_key(v[j]);
    eq_w += u == thr;
    lt_w += u < thr;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    eq_w += __shfl_xor(eq_w, o, 64);
    lt_w += __shfl_xor(lt_w, o, 64);
  }
  if (lane == 0) {
    wcnt[0][w] = eq_w;
    wcnt[1][w] = lt_w;
  }
  __syncthreads();
  int eq_run = 0, sel_base = 0;  // equal keys and selected keys before this wavefront's range
  for (int i = 0; i < w; ++i) {
    sel_base += wcnt[1][i] + min(max(need_eq - eq_run, 0), wcnt[0][i]);
    eq_run += wcnt[0][i];
  }
  // the selected positions, per float4 group in lane order, written from
  // the wavefront's base (the totals of the wavefronts before it)
  auto walk = [&](int32_t* out) {
    int er = eq_run, pos_run = sel_base;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      uint32_t u[4];
      int eq = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        u[e] = desc_key(v[4 * g + e]);
        eq += u[e] == thr;
      }
      const int eq_incl = wave_incl_scan(eq, lane);
      int ebefore = er + eq_incl - eq;
      bool take[4];
      int sel = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        take[e] = u[e] < thr;
        if (u[e] == thr) take[e] = ebefore++ < need_eq;
        sel += take[e];
      }
      const int sel_incl = wave_incl_scan(sel, lane);
      {
        int p = pos_run + sel_incl - sel;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (take[e] && p < k) out[p++] = pos_of(g, e);
      }
      er += __builtin_amdgcn_readlane(eq_incl, 63);
      const int gsel = __builtin_amdgcn_readlane(sel_incl, 63);
      pos_run += gsel;
    }
  };
  walk(lists + row * k);
}

// ---------------------------------------------------------------------------
// Two-pass histogram selection (paper: Method, Cluster assignment -
// selection). One block per row: the grid position g of every score on a
// 128 x 128 grid over [min, max] of the row (fp32), coarse counts and masses
// (the estimated attention mass count_b * exp(tau (S_b - max)) in 2^-32
// fixed point, so the sums are exact), the highest coarse bin whose lower
// edge keeps both thresholds, the same on the 128 fine bins inside it, then
// every b with g_b at or above that edge, in ascending order.
// ---------------------------------------------------------------------------

constexpr int kHistBins = 128;
constexpr int kHistGrid = kHistBins * kHistBins;

__device__ __forceinline__ unsigned long long block_sum_u64(unsigned long long v,
                                                            unsigned long long* sh) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) sh[w] = v;
  __syncthreads();
  const unsigned long long r = sh[0] + sh[1] + sh[2] + sh[3];
  __syncthreads();
  return r;
}

// Estimated mass of one key cluster in 2^-32 units (fp64 arithmetic).
__device__ __forceinline__ unsigned long long mass_units(float s, float hi, int count, float tau) {
  const double m = (double)count * exp((double)tau * ((double)s - (double)hi));
  return (unsigned long long)floor(m * 4294967296.0 + 0.5);
}

// Wavefront 0: the highest bin b whose suffix (bins >= b, plus the given
// count and mass above them) holds both thresholds; also the suffix just
// above b. The condition only grows as b decreases, so b = (number of bins
// that hold it) - 1. Bin 0 always holds it for the thresholds this kernel is
// given.
__device__ __forceinline__ void hist_crossing(const int* cnt, const unsigned long long* ms,
                                              int above_c, unsigned long long above_m,
                                              int min_count, unsigned long long need, int* bin,
                                              int* next_c, unsigned long long* next_m) {
  const int l = threadIdx.x;  // 0..63, bins 2l and 2l + 1
  const int c0 = cnt[2 * l], c1 = cnt[2 * l + 1];
  const unsigned long long m0 = ms[2 * l], m1 = ms[2 * l + 1];
  int vc = c0 + c1;
  unsigned long long vm = m0 + m1;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {  // suffix sums over lanes >= l
    const int yc = __shfl_down(vc, o, 64);
    const unsigned long long ym = __shfl_down(vm, o, 64);
    if (l + o < 64) {
      vc += yc;
      vm += ym;
    }
  }
  const int suf0c = above_c + vc, suf1c = suf0c - c0;  // from bin 2l, from bin 2l + 1
  const unsigned long long suf0m = above_m + vm, suf1m = suf0m - m0;
  const bool ok0 = suf0c >= min_count && suf0m >= need;
  const bool ok1 = suf1c >= min_count && suf1m >= need;
  const int nok = __popcll(__ballot(ok0)) + __popcll(__ballot(ok1));
  const int b = nok > 0 ? nok - 1 : 0;
  // the suffix strictly above b, held by the lane of bin b + 1
  if (b + 1 < kHistBins && ((b + 1) >> 1) == l) {
    const bool odd = (b + 1) & 1;
    *next_c = odd ? suf1c : suf0c;
    *next_m = odd ? suf1m : suf0m;
  }
  if (b + 1 == kHistBins && l == 0) {
    *next_c = above_c;
    *next_m = above_m;
  }
  if (l == 0) *bin = b;
}

__global__ __launch_bounds__(256) void hist_select_kernel(const float* __restrict__ S,
                                                          const int32_t* __restrict__ count_k,
                                                          int nqc, int nkc, int min_count,
                                                          float recall, float tau,
                                                          int32_t* __restrict__ lists,
                                                          int32_t* __restrict__ lens) {
  __shared__ int cnt[kHistBins];
  __shared__ unsigned long long ms[kHistBins];
  __shared__ float sh_f[4];
  __shared__ unsigned long long sh_u[4];
  __shared__ int sh_warp[4];
  __shared__ int sh_bin, sh_above_c;
  __shared__ unsigned long long sh_above_m;
  const size_t row = blockIdx.x;
  const int bh = (int)(row / nqc);
  const float* s = S + row * nkc;
  const int32_t* cntk = count_k + (size_t)bh * nkc;
  int32_t* out = lists + row * nkc;
  const int tid = threadIdx.x;

  float lo = INFINITY, hi = -INFINITY;
  for (int b = tid; b < nkc; b += 256) {
    lo = fminf(lo, s[b]);
    hi = fmaxf(hi, s[b]);
  }
  lo = block_min_max(lo, false, sh_f);
  hi = block_min_max(hi, true, sh_f);
  if (!(hi > lo) || min_count >= nkc) {  // nothing to bin, or the floor takes all
    for (int b = tid; b < nkc; b += 256) out[b] = b;
    if (tid == 0) lens[row] = nkc;
    return;
  }
  const float inv = (float)kHistGrid / (hi - lo);
  auto grid = [&](float v) {
    const int g = (int)floorf((v - lo) * inv);
    return g < 0 ? 0 : (g >= kHistGrid ? kHistGrid - 1 : g);
  };
  const bool use_mass = recall > 0.f;

  // pass 1: coarse counts and masses
  for (int i = tid; i < kHistBins; i += 256) {
    cnt[i] = 0;
    ms[i] = 0ull;
  }
  __syncthreads();
  unsigned long long tot = 0ull;
  for (int b = tid; b < nkc; b += 256) {
    const int g = grid(s[b]);
    atomicAdd(&cnt[g / kHistBins], 1);
    if (use_mass) {
      const unsigned long long u = mass_units(s[b], hi, cntk[b], tau);
      atomicAdd(&ms[g / kHistBins], u);
      tot += u;
    }
  }
  unsigned long long need = 0ull;
  if (use_mass) {
    tot = block_sum_u64(tot, sh_u);
    need = (unsigned long long)ceil((double)tot * (double)recall);
    need = need < tot ? need : tot;
  } else {
    __syncthreads();
  }
  if (tid < 64)
    hist_crossing(cnt, ms, 0, 0ull, min_count, need, &sh_bin, &sh_above_c, &sh_above_m);
  __syncthreads();
  const int B = sh_bin;
  const int above_c = sh_above_c;
  const unsigned long long above_m = sh_above_m;
  // pass 2: fine counts and masses inside coarse bin B
  for (int i = tid; i < kHistBins; i += 256) {
    cnt[i] = 0;
    ms[i] = 0ull;
  }
  __syncthreads();
  for (int b = tid; b < nkc; b += 256) {
    const int g = grid(s[b]);
    if (g / kHistBins != B) continue;
    atomicAdd(&cnt[g % kHistBins], 1);
    if (use_mass) atomicAdd(&ms[g % kHistBins], mass_units(s[b], hi, cntk[b], tau));
  }
  __syncthreads();
  if (tid < 64)
    hist_crossing(cnt, ms, above_c, above_m, min_count, need, &sh_bin, &sh_above_c, &sh_above_m);
  __syncthreads();
  const int G = B * kHistBins + sh_bin;

  // ascending compaction of {b : g_b >= G}
  const int per = (nkc + 255) / 256;
  const int b0 = min(nkc, tid * per), b1 = min(nkc, b0 + per);
  int n = 0;
  for (int b = b0; b < b1; ++b) n += grid(s[b]) >= G;
  int total;
  int pos = block_scan_256(n, sh_warp, &total);
  for (int b = b0; b < b1; ++b)
    if (grid(s[b]) >= G) out[pos++] = b;
  if (tid == 0) lens[row] = total;
}

}  // namespace

hipError_t launch_select(const Prob& P, const float* cq, const float* ck, const float* scores_in,
                         float* scores, int k, int32_t* lists, hipStream_t st) {
  const float* S = scores_in;
  if (!S) {
    hipError_t e = launch_scores(P, cq, ck, scores, st);
    if (e != hipSuccess) return e;
    S = scores;
  } else if (scores && scores != scores_in) {
    hipError_t e = hipMemcpyAsync(scores, scores_in, (size_t)P.BH * P.nqc * P.nkc * 4,
                                  hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return e;
  }
  const size_t nrows = (size_t)P.BH * P.nqc;
  if (P.nkc <= 64 * 128) {
    const int vec4 = (P.nkc % 4 == 0) && (((uintptr_t)S & 15) == 0);
    const dim3 grid((unsigned)((nrows + 3) / 4));
#define CA_TOPK_WAVE(V)                                                                        \
  if (P.nkc <= 64 * V) {                                                                       \
    hipLaunchKernelGGL(topk_wave_kernel<V>, grid, dim3(256), 0, st, S, P.nkc, k, (int)nrows, \
                       vec4, lists);                                                           \
    return hipGetLastError();                                                                  \
  }
    CA_TOPK_WAVE(4)
    CA_TOPK_WAVE(8)
    CA_TOPK_WAVE(16)
    CA_TOPK_WAVE(32)
#undef CA_TOPK_WAVE
    // wider rows: one row per block of four wavefronts (more rows in flight
    // than with a whole row in one wavefront's registers)
#define CA_TOPK_BLOCK(V)                                                                      \
  if (P.nkc <= 256 * V) {                                                                     \
    hipLaunchKernelGGL((topk_block_kernel<V, 4>), dim3((unsigned)nrows), dim3(256), 0, st, S, \
                       P.nkc, k, vec4, lists);                                                \
    return hipGetLastError();                                                                 \
  }
    CA_TOPK_BLOCK(16)
    CA_TOPK_BLOCK(32)
#undef CA_TOPK_BLOCK
  }
  hipLaunchKernelGGL(topk_kernel, dim3((unsigned)nrows), dim3(256), 0, st, S, P.nkc, k, lists);
  return hipGetLastError();
}

}  // namespace ca

namespace ca {

hipError_t launch_select_hist(const Prob& P, const float* cq, const float* ck,
                              const int32_t* count_k, const float* scores_in, float* scores,
                              int min_count, float recall, float scale, int32_t* lists,
                              int32_t* lens, hipStream_t st) {
  const float* S = scores_in;
  if (!S) {
    hipError_t e = launch_scores(P, cq, ck, scores, st);
    if (e != hipSuccess) return e;
    S = scores;
  } else if (scores && scores != scores_in) {
    hipError_t e = hipMemcpyAsync(scores, scores_in, (size_t)P.BH * P.nqc * P.nkc * 4,
                                  hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(hist_select_kernel, dim3((unsigned)((size_t)P.BH * P.nqc)), dim3(256), 0, st,
                     S, count_k, P.nqc, P.nkc, min_count, recall, scale, lists, lens);
  return hipGetLastError();
}

}  // namespace ca
