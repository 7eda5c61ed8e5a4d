// Striped mean-compensation (paper: Preliminaries, error in sparse attention;
// App. A) fused with the merge into the block-sparse result and the return to
// the original token order.
//
// Every key cluster b that query cluster a did not select contributes to each
// query of a through its centroid key and value with the logit
// scale*q.kbar_b + ln|b|. These centroid logits form a second softmax whose
// (lse_c, o_c) is merged with the sparse part (lse_s, o_s) in log-sum-exp form.
// bf16: centroids are rounded to bf16 in LDS and contracted on MFMA exactly like
// key tiles, 128 centroids per tile. fp32: one thread per query.
#include <math.h>

#include "attn_tile.h"

namespace ca {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kMaskWords = 2048;  // up to 65536 key clusters

__device__ __forceinline__ int xcd_remap(int wg, int total) {
  int per = total >> 3, rem = total & 7;
  int xcd = wg & 7, loc = wg >> 3;
  return xcd < rem ? xcd * (per + 1) + loc : rem * (per + 1) + (xcd - rem) * per + loc;
}

__device__ __forceinline__ size_t out_row(int bh, int i, int nq, int H, int d, int layout) {
  return row_off(bh, i, nq, H, d, layout);
}

template <int D, int CQ>
__global__ __launch_bounds__(CQ * 2, (D == 64 ? 2 : 1)) void comp_bf16_kernel(
    const bf16* __restrict__ qp, const float* __restrict__ cent_k,
    const float* __restrict__ cent_v, const int32_t* __restrict__ count_k,
    const int32_t* __restrict__ lists, int nq, int H, int nqc, int nkc, int k, float sl2,
    int enable, const bf16* __restrict__ op, const float* __restrict__ lse_s,
    const int32_t* __restrict__ perm_q, bf16* __restrict__ out, float* __restrict__ lse_out,
    int layout, int total) {
  constexpr int NW = CQ / 32;
  constexpr int T = NW * 64;
  constexpr int CT = 128;  // centroids per tile
  constexpr int MT = CT / 32;
  constexpr int KS = D / 16;
  constexpr int DT = D / 32;
  constexpr int KP = D + 8;
  constexpr int VP = CT + 8;
  __shared__ __attribute__((aligned(16))) bf16 Ks[CT * KP];
  __shared__ __attribute__((aligned(16))) bf16 Vs[D * VP];
  __shared__ __attribute__((aligned(16))) float bias[CT];
  __shared__ uint32_t selmask[kMaskWords];

  const int item = xcd_remap(blockIdx.x, total);
  const int bh = item / nqc, a = item - bh * nqc;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const size_t nq_pad = (size_t)nqc * CQ;
  const int prow = a * CQ + 32 * w + l32;  // row inside this head's permuted order
  const size_t qrow = (size_t)bh * nq_pad + prow;
  const int nwords = (nkc + 31) >> 5;

  float m_run = -INFINITY, l_run = 0.f;
  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[dt][r] = 0.f;

  const bool do_comp = enable && k < nkc;
  if (do_comp) {
    for (int i = tid; i < nwords; i += T) selmask[i] = 0u;
    __syncthreads();
    const int32_t* lst = lists + ((size_t)bh * nqc + a) * k;
    for (int i = tid; i < k; i += T) {
      int b = lst[i];
      if (b >= 0 && b < nkc) atomicOr(&selmask[b >> 5], 1u << (b & 31));
    }
    bf16x8 qreg[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qreg[ks] = *(const bf16x8*)(qp + qrow * D + 16 * ks + 8 * h);

    const float* ckh = cent_k + (size_t)bh * nkc * D;
    const float* cvh = cent_v + (size_t)bh * nkc * D;
    const int32_t* cnth = count_k + (size_t)bh * nkc;
    // Staging tasks: K rows as 8-column chunks (one 16-byte LDS store each);
    // V as 8-centroid x 4-column blocks, transposed in registers into four
    // 16-byte stores. The global loads of tile t+1 are issued before the
    // products of tile t, so their latency hides behind the matrix work.
    constexpr int NKT = CT * (D / 8) / T;
    constexpr int NVT = (CT / 8) * (D / 4) / T;
    constexpr int NBT = (CT + T - 1) / T;
    static_assert(NKT * T == CT * (D / 8) && NVT * T == (CT / 8) * (D / 4), "staging split");
    // (without registers to spare, a tile is loaded just before it is staged)
    constexpr bool kPrefetch = NKT * 2 + NVT * 8 <= 16;
    float4 kv[NKT][2], vv[NVT][8];
    int cv[NBT];
    __syncthreads();  // selmask complete
    // Tiles holding at least one unselected centroid, in order.
    auto tile_live = [&](int b0) {
      int any = 0;
      for (int e = b0 >> 5; e < ((b0 + CT) >> 5) && e < nwords; ++e) {
        const uint32_t wmask = e == nwords - 1 && (nkc & 31) ? (1u << (nkc & 31)) - 1u : ~0u;
        any |= (~selmask[e] & wmask) != 0u;
      }
      return any;
    };
    auto next_live = [&](int b0) {
      while (b0 < nkc && !tile_live(b0)) b0 += CT;
      return b0;
    };
    auto load_k = [&](int b0) {
#pragma unroll
      for (int u = 0; u < NKT; ++u) {
        const int i = tid + T * u, row = i / (D / 8), c8 = i % (D / 8), b = b0 + row;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
          kv[u][hh] = b < nkc ? *(const float4*)(ckh + (size_t)b * D + 8 * c8 + 4 * hh)
                              : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < NBT; ++u) {
        const int e = tid + T * u, b = b0 + e;
        cv[u] = e < CT && b < nkc ? cnth[b] : 0;
      }
    };
    auto load_v = [&](int b0) {
#pragma unroll
      for (int u = 0; u < NVT; ++u) {
        const int i = tid + T * u, g = i % (CT / 8), cc = i / (CT / 8);
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          const int b = b0 + 8 * g + r;
          vv[u][r] = b < nkc ? *(const float4*)(cvh + (size_t)b * D + 4 * cc)
                             : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
    };
    auto store_k = [&](int b0) {
#pragma unroll
      for (int u = 0; u < NKT; ++u) {
        const int i = tid + T * u, row = i / (D / 8), c8 = i % (D / 8);
        const float f[8] = {kv[u][0].x, kv[u][0].y, kv[u][0].z, kv[u][0].w,
                            kv[u][1].x, kv[u][1].y, kv[u][1].z, kv[u][1].w};
        *(bf16x8*)&Ks[row * KP + 8 * c8] = pack8(f);
      }
#pragma unroll
      for (int u = 0; u < NBT; ++u) {
        const int e = tid + T * u, b = b0 + e;
        if (e < CT) {
          float bi = -INFINITY;
          if (b < nkc && !((selmask[b >> 5] >> (b & 31)) & 1u) && cv[u] > 0)
            bi = __builtin_amdgcn_logf((float)cv[u]);  // log2 of the size
          bias[e] = bi;
        }
      }
    };
    auto store_v = [&]() {
#pragma unroll
      for (int u = 0; u < NVT; ++u) {
        const int i = tid + T * u, g = i % (CT / 8), cc = i / (CT / 8);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float f[8];
#pragma unroll
          for (int r = 0; r < 8; ++r)
            f[r] = j == 0 ? vv[u][r].x : (j == 1 ? vv[u][r].y : (j == 2 ? vv[u][r].z : vv[u][r].w));
          *(bf16x8*)&Vs[(4 * cc + j) * VP + 8 * g] = pack8(f);
        }
      }
    };
    int b0 = next_live(0);
    if (kPrefetch && b0 < nkc) {
      load_k(b0);
      load_v(b0);
    }
    while (b0 < nkc) {
      __syncthreads();  // the previous tile is fully consumed
      if (!kPrefetch) load_k(b0);
      store_k(b0);
      if (!kPrefetch) load_v(b0);
      store_v();
      __syncthreads();
      const int b1 = next_live(b0 + CT);
      if (kPrefetch && b1 < nkc) {
        load_k(b1);
        load_v(b1);
      }

      f32x16 sacc[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[mt][r] = 0.f;
        const bf16* krow = &Ks[(32 * mt + kswz(l32)) * KP + 8 * h];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          bf16x8 av = *(const bf16x8*)(krow + 16 * ks);
          sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qreg[ks], sacc[mt], 0, 0, 0);
        }
      }
      // logits in log2 units: scale*log2e*q.kbar + log2|b|. The bias of
      // accumulator r of row tile mt is bias[32 mt + (r & 7) + 16 (r >> 3) + 8 h]:
      // two runs of 8 consecutive entries, read as four 16-byte loads.
      float mx = -INFINITY;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        float bv[16];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const float4 b0v = *(const float4*)&bias[32 * mt + 16 * hh + 8 * h];
          const float4 b1v = *(const float4*)&bias[32 * mt + 16 * hh + 8 * h + 4];
          bv[8 * hh + 0] = b0v.x, bv[8 * hh + 1] = b0v.y, bv[8 * hh + 2] = b0v.z, bv[8 * hh + 3] = b0v.w;
          bv[8 * hh + 4] = b1v.x, bv[8 * hh + 5] = b1v.y, bv[8 * hh + 6] = b1v.z, bv[8 * hh + 7] = b1v.w;
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float t = __builtin_fmaf(sacc[mt][r], sl2, bv[r]);
          sacc[mt][r] = t;
          mx = fmaxf(mx, t);
        }
      }
      mx = fmaxf(mx, wave_xor32(mx));
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      float lsum = 0.f;
      bf16x8 pb[MT][2];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          float pv[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) pv[j] = __builtin_amdgcn_exp2f(sacc[mt][8 * s + j] - m_new);
          pb[mt][s] = pack8(pv);
          lsum = sum8(pb[mt][s], lsum);
        }
      l_run = l_run * alpha + lsum;
      m_run = m_new;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
        const bf16* vrow = &Vs[(32 * dt + l32) * VP + 8 * h];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int s = 0; s < 2; ++s) {
            bf16x8 av = *(const bf16x8*)(vrow + 32 * mt + 16 * s);
            oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb[mt][s], oacc[dt], 0, 0, 0);
          }
      }
      b0 = b1;
    }
  }

  // Merge with the sparse part and write to the original position.
  const float l_tot = l_run + wave_xor32(l_run);
  if (prow >= nq) return;
  const float ls = lse_s[qrow];
  float ws = 1.f, wc = 0.f, lse = ls, inv_c = 0.f;
  if (l_tot > 0.f) {
    const float lc = (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2;
    const float mm = fmaxf(ls, lc);
    lse = mm + logf(expf(ls - mm) + expf(lc - mm));
    ws = expf(ls - lse);
    wc = expf(lc - lse);
    inv_c = 1.f / l_tot;
  }
  int orig = perm_q[(size_t)bh * nq + prow];
  orig = orig < 0 ? 0 : (orig >= nq ? nq - 1 : orig);  // memory safety for a bad permutation
  bf16* orow = out + out_row(bh, orig, nq, H, D, layout);
  const bf16* srow = op + qrow * D;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int col = 32 * dt + 8 * g + 4 * h;
      bf16x4 s4 = *(const bf16x4*)(srow + col);
      bf16x4 v4;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        v4[j] = f2bf(ws * bf2f(s4[j]) + wc * (oacc[dt][4 * g + j] * inv_c));
      *(bf16x4*)(orow + col) = v4;
    }
  if (lse_out && h == 0) lse_out[(size_t)bh * nq + orig] = lse;
}

// fp32 path: one thread per query, plain FMA; centroids streamed through LDS.
template <int DP>
__global__ __launch_bounds__(256) void comp_f32_kernel(
    const float* __restrict__ qp, const float* __restrict__ cent_k,
    const float* __restrict__ cent_v, const int32_t* __restrict__ count_k,
    const int32_t* __restrict__ lists, int nq, int H, int nqc, int nkc, int cq, int d, int k,
    float scale, int enable, const float* __restrict__ op, const float* __restrict__ lse_s,
    const int32_t* __restrict__ perm_q, float* __restrict__ out, float* __restrict__ lse_out,
    int layout) {
  constexpr int KC = 32;
  __shared__ float Ksh[KC][DP + 1];
  __shared__ float Vsh[KC][DP + 1];
  __shared__ float bias[KC];
  __shared__ uint32_t selmask[kMaskWords];
  const int a = blockIdx.x, bh = blockIdx.y, i = threadIdx.x;
  const int prow = a * cq + i;
  const bool active = i < cq && prow < nq;
  const size_t qrow = ((size_t)bh * nqc + a) * cq + (i < cq ? i : 0);
  const bool do_comp = enable && k < nkc;
  float q[DP], o[DP];
#pragma unroll
  for (int t = 0; t < DP; ++t) {
    q[t] = (i < cq && t < d) ? qp[qrow * d + t] : 0.f;
    o[t] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  if (do_comp) {
    const int nwords = (nkc + 31) >> 5;
    for (int e = i; e < nwords; e += blockDim.x) selmask[e] = 0u;
    __syncthreads();
    const int32_t* lst = lists + ((size_t)bh * nqc + a) * k;
    for (int e = i; e < k; e += blockDim.x) {
      int b = lst[e];
      if (b >= 0 && b < nkc) atomicOr(&selmask[b >> 5], 1u << (b & 31));
    }
    for (int b0 = 0; b0 < nkc; b0 += KC) {
      const int nb = min(KC, nkc - b0);
      __syncthreads();
      for (int e = i; e < KC * DP; e += blockDim.x) {
        const int r = e / DP, t = e % DP;
        const bool in = r < nb && t < d;
        Ksh[r][t] = in ? cent_k[((size_t)bh * nkc + b0 + r) * d + t] : 0.f;
        Vsh[r][t] = in ? cent_v[((size_t)bh * nkc + b0 + r) * d + t] : 0.f;
      }
      for (int e = i; e < KC; e += blockDim.x) {
        const int b = b0 + e;
        bias[e] = (e < nb && !((selmask[b >> 5] >> (b & 31)) & 1u))
                      ? logf((float)count_k[(size_t)bh * nkc + b])
                      : -INFINITY;
      }
      __syncthreads();
      for (int r = 0; r < nb; ++r) {
        if (bias[r] == -INFINITY) continue;
        float s = 0.f;
#pragma unroll
        for (int t = 0; t < DP; ++t) s = __builtin_fmaf(q[t], Ksh[r][t], s);
        s = s * scale + bias[r];
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
        for (int t = 0; t < DP; ++t) o[t] = __builtin_fmaf(pw, Vsh[r][t], o[t]);
      }
    }
  }
  if (!active) return;
  const float ls = lse_s[qrow];
  float ws = 1.f, wc = 0.f, lse = ls, inv_c = 0.f;
  if (l > 0.f) {
    const float lc = m + logf(l);
    const float mm = fmaxf(ls, lc);
    lse = mm + logf(expf(ls - mm) + expf(lc - mm));
    ws = expf(ls - lse);
    wc = expf(lc - lse);
    inv_c = 1.f / l;
  }
  int orig = perm_q[(size_t)bh * nq + prow];
  orig = orig < 0 ? 0 : (orig >= nq ? nq - 1 : orig);
  float* orow = out + row_off(bh, orig, nq, H, d, layout);
  for (int t = 0; t < d; ++t) orow[t] = ws * op[qrow * d + t] + wc * (o[t] * inv_c);
  if (lse_out) lse_out[(size_t)bh * nq + orig] = lse;
}

template <int D, int CQ>
hipError_t run_bf16(const Prob& P, const void* qp, const float* cent_k, const float* cent_v,
                    const int32_t* count_k, const int32_t* lists, int k, float scale, int enable,
                    const void* op, const float* lse, const int32_t* perm_q, void* out,
                    float* lse_out, hipStream_t st) {
  const int total = P.BH * P.nqc;
  hipLaunchKernelGGL((comp_bf16_kernel<D, CQ>), dim3(total), dim3(CQ * 2), 0, st,
                     (const bf16*)qp, cent_k, cent_v, count_k, lists, P.nq, P.H, P.nqc, P.nkc, k,
                     scale * kLog2e, enable, (const bf16*)op, lse, perm_q, (bf16*)out, lse_out,
                     P.layout, total);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_comp(const Prob& P, const void* qp, const float* cent_k, const float* cent_v,
                       const int32_t* count_k, const int32_t* lists, int k, float scale,
                       int enable, const void* op, const float* lse, const int32_t* perm_q,
                       void* out, float* lse_out, hipStream_t st) {
  if (P.nkc > kMaskWords * 32) return hipErrorInvalidValue;
  if (P.dtype == CA_BF16) {
#define CA_COMP_CASE(D, CQ) \
  if (P.d == D && P.cq == CQ) \
    return run_bf16<D, CQ>(P, qp, cent_k, cent_v, count_k, lists, k, scale, enable, op, lse, \
                           perm_q, out, lse_out, st);
    CA_COMP_CASE(64, 64)
    CA_COMP_CASE(64, 128)
    CA_COMP_CASE(128, 64)
    CA_COMP_CASE(128, 128)
#undef CA_COMP_CASE
    return hipErrorInvalidValue;
  }
  dim3 grid(P.nqc, P.BH);
  const int threads = ((P.cq + 63) / 64) * 64;
#define CA_COMP_F32(DP)                                                                       \
  hipLaunchKernelGGL(comp_f32_kernel<DP>, grid, dim3(threads), 0, st, (const float*)qp,       \
                     cent_k, cent_v, count_k, lists, P.nq, P.H, P.nqc, P.nkc, P.cq, P.d, k,   \
                     scale, enable, (const float*)op, lse, perm_q, (float*)out, lse_out,      \
                     P.layout)
  if (P.d <= 32)
    CA_COMP_F32(32);
  else if (P.d <= 64)
    CA_COMP_F32(64);
  else
    CA_COMP_F32(128);
#undef CA_COMP_F32
  return hipGetLastError();
}

}  // namespace ca
