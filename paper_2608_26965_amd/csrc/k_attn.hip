// Block-sparse attention over selected key clusters (paper: Method, Overview -
// attention over the selected clusters, returning the softmax denominator).
//
// One workgroup per (head, query cluster); the workgroup streams the k
// selected key-cluster tiles through LDS (double-buffered) and runs an online
// softmax. bf16: MFMA 32x32x16 with fp32 accumulation, one wavefront per 32
// queries. fp32: plain FMA, one thread per query.
#include <math.h>

#include "attn_tile.h"

namespace ca {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Workgroup w of a 1-D grid runs on XCD w % 8. Renumber so that each XCD gets
// one contiguous range of (head, query cluster) items: neighbouring query
// clusters of one head share most selected key tiles, which then stay in that
// XCD's L2.
__device__ __forceinline__ int xcd_remap(int wg, int total) {
  int per = total >> 3, rem = total & 7;
  int xcd = wg & 7, loc = wg >> 3;
  return xcd < rem ? xcd * (per + 1) + loc : rem * (per + 1) + (xcd - rem) * per + loc;
}

template <int D, int CQ, int CK>
__global__ __launch_bounds__(CQ * 2) void attn_bf16_kernel(
    const bf16* __restrict__ qp, const bf16* __restrict__ kp, const bf16* __restrict__ vp,
    const int32_t* __restrict__ count_k, const int32_t* __restrict__ lists, int nqc, int nkc,
    int k, float sl2, bf16* __restrict__ op, float* __restrict__ lse, int total) {
  constexpr int NW = CQ / 32;
  constexpr int T = NW * 64;
  constexpr int MT = CK / 32;
  constexpr int KS = D / 16;
  constexpr int DT = D / 32;
  constexpr int KP = D + 8;   // LDS pitch of a K row (bf16), +16 bytes against bank conflicts
  constexpr int VP = CK + 8;  // LDS pitch of a V^T row
  constexpr int KCH = CK * D / 8 / T;  // 16-byte chunks per thread per tile
  constexpr int VCH = D * CK / 8 / T;
  static_assert(KCH * T * 8 == CK * D && VCH * T * 8 == D * CK, "tile split");
  __shared__ __attribute__((aligned(16))) bf16 Ks[2][CK * KP];
  __shared__ __attribute__((aligned(16))) bf16 Vs[2][D * VP];

  const int item = xcd_remap(blockIdx.x, total);
  const int bh = item / nqc, a = item - bh * nqc;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const size_t nq_pad = (size_t)nqc * CQ, nk_pad = (size_t)nkc * CK;
  const size_t qrow = (size_t)bh * nq_pad + (size_t)a * CQ + 32 * w + l32;

  bf16x8 qreg[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    qreg[ks] = *(const bf16x8*)(qp + qrow * D + 16 * ks + 8 * h);

  const int32_t* lst = lists + ((size_t)bh * nqc + a) * k;
  auto tile_id = [&](int t) {
    int b = lst[t];
    return b < 0 ? 0 : (b >= nkc ? nkc - 1 : b);
  };

  uint4 kreg[KCH], vreg[VCH];
  auto fetch = [&](int b) {
    const bf16* kt = kp + ((size_t)bh * nk_pad + (size_t)b * CK) * D;
    const bf16* vt = vp + ((size_t)bh * nkc + b) * (size_t)D * CK;
#pragma unroll
    for (int i = 0; i < KCH; ++i) kreg[i] = ((const uint4*)kt)[tid + i * T];
#pragma unroll
    for (int i = 0; i < VCH; ++i) vreg[i] = ((const uint4*)vt)[tid + i * T];
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      int c = tid + i * T, row = c / (D / 8), c8 = c % (D / 8);
      *(uint4*)&Ks[buf][row * KP + c8 * 8] = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < VCH; ++i) {
      int c = tid + i * T, row = c / (CK / 8), c8 = c % (CK / 8);
      *(uint4*)&Vs[buf][row * VP + c8 * 8] = vreg[i];
    }
  };

  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[dt][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  fetch(tile_id(0));
  stash(0);
  __syncthreads();

  for (int t = 0; t < k; ++t) {
    const int cur = t & 1;
    if (t + 1 < k) fetch(tile_id(t + 1));
    const int cnt = count_k[(size_t)bh * nkc + tile_id(t)];

    f32x16 sacc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[mt][r] = 0.f;
      const bf16* krow = &Ks[cur][(32 * mt + kswz(l32)) * KP + 8 * h];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        bf16x8 av = *(const bf16x8*)(krow + 16 * ks);
        sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qreg[ks], sacc[mt], 0, 0, 0);
      }
    }
    if (cnt < CK) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (acc_key(mt, r, h) >= cnt) sacc[mt][r] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[mt][r]);
    mx = fmaxf(mx, wave_xor32(mx));
    const float m_new = fmaxf(m_run, mx * sl2);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float lsum = 0.f;
    bf16x8 pb[MT][2];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        float pv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          pv[j] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[mt][8 * s + j], sl2, -m_new));
          lsum += pv[j];
        }
        pb[mt][s] = pack8(pv);
      }
    l_run = l_run * alpha + lsum;
    m_run = m_new;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
      const bf16* vrow = &Vs[cur][(32 * dt + l32) * VP + 8 * h];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          bf16x8 av = *(const bf16x8*)(vrow + 32 * mt + 16 * s);
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb[mt][s], oacc[dt], 0, 0, 0);
        }
    }
    if (t + 1 < k) stash(cur ^ 1);
    __syncthreads();
  }

  const float l_tot = l_run + wave_xor32(l_run);
  const float inv = 1.f / l_tot;
  bf16* orow = op + qrow * D;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 v4;
#pragma unroll
      for (int j = 0; j < 4; ++j) v4[j] = f2bf(oacc[dt][4 * g + j] * inv);
      *(bf16x4*)(orow + 32 * dt + 8 * g + 4 * h) = v4;
    }
  if (h == 0) lse[qrow] = (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2;
}

// fp32 path: one thread per query, keys streamed through LDS 32 at a time.
template <int DP>
__global__ __launch_bounds__(256) void attn_f32_kernel(
    const float* __restrict__ qp, const float* __restrict__ kp, const float* __restrict__ vp,
    const int32_t* __restrict__ count_k, const int32_t* __restrict__ lists, int nqc, int nkc,
    int cq, int ck, int d, int k, float scale, float* __restrict__ op, float* __restrict__ lse) {
  constexpr int KC = 32;
  __shared__ float Ksh[KC][DP + 1];
  __shared__ float Vsh[KC][DP + 1];
  const int a = blockIdx.x, bh = blockIdx.y, i = threadIdx.x;
  const bool active = i < cq;
  const size_t qrow = ((size_t)bh * nqc + a) * cq + (active ? i : 0);
  const size_t nk_pad = (size_t)nkc * ck;
  float q[DP], o[DP];
#pragma unroll
  for (int t = 0; t < DP; ++t) {
    q[t] = (active && t < d) ? qp[qrow * d + t] : 0.f;
    o[t] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int32_t* lst = lists + ((size_t)bh * nqc + a) * k;
  for (int tt = 0; tt < k; ++tt) {
    int b = lst[tt];
    b = b < 0 ? 0 : (b >= nkc ? nkc - 1 : b);
    const int cnt = count_k[(size_t)bh * nkc + b];
    for (int k0 = 0; k0 < cnt; k0 += KC) {
      const int nk = min(KC, cnt - k0);
      __syncthreads();
      for (int e = threadIdx.x; e < KC * DP; e += blockDim.x) {
        int kk = e / DP, t = e % DP;
        Ksh[kk][t] = (kk < nk && t < d) ? kp[((size_t)bh * nk_pad + (size_t)b * ck + k0 + kk) * d + t]
                                        : 0.f;
      }
      for (int e = threadIdx.x; e < KC * DP; e += blockDim.x) {
        int kk = e % KC, t = e / KC;
        Vsh[kk][t] = (kk < nk && t < d) ? vp[(((size_t)bh * nkc + b) * d + t) * ck + k0 + kk] : 0.f;
      }
      __syncthreads();
      for (int kk = 0; kk < nk; ++kk) {
        float s = 0.f;
#pragma unroll
        for (int t = 0; t < DP; ++t) s = __builtin_fmaf(q[t], Ksh[kk][t], s);
        s *= scale;
        if (s > m) {
          const float al = expf(m - s);
#pragma unroll
          for (int t = 0; t < DP; ++t) o[t] *= al;
          l *= al;
          m = s;
        }
        const float pw = expf(s - m);
        l += pw;
#pragma unroll
        for (int t = 0; t < DP; ++t) o[t] = __builtin_fmaf(pw, Vsh[kk][t], o[t]);
      }
    }
  }
  if (active) {
    const float inv = 1.f / l;
    for (int t = 0; t < d; ++t) op[qrow * d + t] = o[t] * inv;
    lse[qrow] = m + logf(l);
  }
}

template <int D, int CQ, int CK>
hipError_t run_bf16(const Prob& P, const void* qp, const void* kp, const void* vp,
                    const int32_t* count_k, const int32_t* lists, int k, float scale, void* op,
                    float* lse, hipStream_t st) {
  int total = P.BH * P.nqc;
  hipLaunchKernelGGL((attn_bf16_kernel<D, CQ, CK>), dim3(total), dim3(CQ * 2), 0, st,
                     (const bf16*)qp, (const bf16*)kp, (const bf16*)vp, count_k, lists, P.nqc,
                     P.nkc, k, scale * kLog2e, (bf16*)op, lse, total);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const Prob& P, const void* qp, const void* kp, const void* vp,
                       const int32_t* count_k, const int32_t* lists, int k, float scale, void* op,
                       float* lse, hipStream_t st) {
  if (P.dtype == CA_BF16) {
#define CA_ATTN_CASE(D, CQ, CK) \
  if (P.d == D && P.cq == CQ && P.ck == CK) \
    return run_bf16<D, CQ, CK>(P, qp, kp, vp, count_k, lists, k, scale, op, lse, st);
    CA_ATTN_CASE(64, 64, 64)
    CA_ATTN_CASE(64, 64, 128)
    CA_ATTN_CASE(64, 128, 64)
    CA_ATTN_CASE(64, 128, 128)
    CA_ATTN_CASE(128, 64, 64)
    CA_ATTN_CASE(128, 64, 128)
    CA_ATTN_CASE(128, 128, 64)
    CA_ATTN_CASE(128, 128, 128)
#undef CA_ATTN_CASE
    return hipErrorInvalidValue;
  }
  dim3 grid(P.nqc, P.BH);
  int threads = ((P.cq + 63) / 64) * 64;
  if (P.d <= 32) {
    hipLaunchKernelGGL(attn_f32_kernel<32>, grid, dim3(threads), 0, st, (const float*)qp,
                       (const float*)kp, (const float*)vp, count_k, lists, P.nqc, P.nkc, P.cq,
                       P.ck, P.d, k, scale, (float*)op, lse);
  } else if (P.d <= 64) {
    hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(threads), 0, st, (const float*)qp,
                       (const float*)kp, (const float*)vp, count_k, lists, P.nqc, P.nkc, P.cq,
                       P.ck, P.d, k, scale, (float*)op, lse);
  } else {
    hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(threads), 0, st, (const float*)qp,
                       (const float*)kp, (const float*)vp, count_k, lists, P.nqc, P.nkc, P.cq,
                       P.ck, P.d, k, scale, (float*)op, lse);
  }
  return hipGetLastError();
}

}  // namespace ca
