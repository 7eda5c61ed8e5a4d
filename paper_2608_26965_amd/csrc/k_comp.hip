// Striped mean-compensation (paper: Preliminaries, error in sparse attention;
// App. A) fused with the merge into the block-sparse result and the return to
// the original token order.
//
// Every key cluster b that query cluster a did not select contributes to each
// query of a through its centroid key and value with the logit
// scale*q.kbar_b + ln|b|. These centroid logits form a second softmax whose
// (lse_c, o_c) is merged with the sparse part (lse_s, o_s) in log-sum-exp form.
// bf16: the centroids of a head are first rounded once into bf16 tiles of 128
// (keys row-major, values transposed, plus the log2 cluster sizes) in the
// workspace; every query cluster then streams those tiles into LDS with
// direct-to-LDS copies and contracts them on MFMA exactly like key tiles.
// fp32: one thread per query.
#include <math.h>

#include <type_traits>

#include "attn_tile.h"

namespace ca {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// s_waitcnt immediate (gfx9 encoding) waiting for vmcnt = 0 only.
constexpr int kVmcnt0 = 0x0F70;

__device__ __forceinline__ int xcd_remap(int wg, int total) {
  int per = total >> 3, rem = total & 7;
  int xcd = wg & 7, loc = wg >> 3;
  return xcd < rem ? xcd * (per + 1) + loc : rem * (per + 1) + (xcd - rem) * per + loc;
}



// bf16 centroid tiles (written once per call, read by every query cluster of
// the head): tile t of head bh covers centroids [128 t, 128 t + 128) and holds
//   K   [128][D] bf16   centroid keys, row-major (zero rows past nkc),
//   V^T [D][128] bf16   centroid values transposed (zero columns past nkc),
//   bias[128]    fp32   log2 of the cluster size (-inf: empty or past nkc).
// blockIdx.z = 0 writes K and bias, 1 writes V^T (through an LDS transpose).
template <int D>
__global__ __launch_bounds__(256) void comp_stage_kernel(const float* __restrict__ cent_k,
                                                         const float* __restrict__ cent_v,
                                                         const int32_t* __restrict__ count_k,
                                                         int nkc, int ntile,
                                                         char* __restrict__ tiles) {
  constexpr int CT = kCompTile;
  constexpr int KBYTES = CT * D * 2, VBYTES = D * CT * 2;
  constexpr int TB = KBYTES + VBYTES + CT * 4;
  __shared__ float vs[CT][D + 1];
  const int t = blockIdx.x, bh = blockIdx.y, tid = threadIdx.x;
  const int b0 = t * CT;
  char* tile = tiles + ((size_t)bh * ntile + t) * TB;
  if (blockIdx.z == 0) {
    const float* src = cent_k + (size_t)bh * nkc * D;
    bf16* kt = (bf16*)tile;
    for (int i = tid; i < CT * (D / 8); i += 256) {
      const int row = i / (D / 8), c8 = i % (D / 8), b = b0 + row;
      float4 x = make_float4(0.f, 0.f, 0.f, 0.f), y = x;
      if (b < nkc) {
        x = *(const float4*)(src + (size_t)b * D + 8 * c8);
        y = *(const float4*)(src + (size_t)b * D + 8 * c8 + 4);
      }
      const float f[8] = {x.x, x.y, x.z, x.w, y.x, y.y, y.z, y.w};
      *(bf16x8*)(kt + row * D + 8 * c8) = pack8(f);
    }
    if (tid < CT) {
      const int b = b0 + tid;
      const int c = b < nkc ? count_k[(size_t)bh * nkc + b] : 0;
      ((float*)(tile + KBYTES + VBYTES))[tid] =
          c > 0 ? __builtin_amdgcn_logf((float)c) : -INFINITY;  // log2 of the size
    }
    return;
  }
  const float* src = cent_v + (size_t)bh * nkc * D;
  for (int i = tid; i < CT * (D / 4); i += 256) {
    const int row = i / (D / 4), c4 = i % (D / 4), b = b0 + row;
    float4 x = make_float4(0.f, 0.f, 0.f, 0.f);
    if (b < nkc) x = *(const float4*)(src + (size_t)b * D + 4 * c4);
    vs[row][4 * c4] = x.x;
    vs[row][4 * c4 + 1] = x.y;
    vs[row][4 * c4 + 2] = x.z;
    vs[row][4 * c4 + 3] = x.w;
  }
  __syncthreads();
  bf16* vt = (bf16*)(tile + KBYTES);
  for (int i = tid; i < D * (CT / 8); i += 256) {
    const int dim = i / (CT / 8), g = i % (CT / 8);
    float f[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) f[r] = vs[8 * g + r][dim];
    *(bf16x8*)(vt + dim * CT + 8 * g) = pack8(f);
  }
}

// Centroids per LDS stage: a whole tile of 128 at d = 64; half a tile at
// d = 128, so that two stages and the mask take 74 KB instead of 140 KB and
// two workgroups share a CU.
template <int D>
constexpr int comp_stage_cents() {
  return D == 128 ? kCompTile / 2 : kCompTile;
}

// Waves per SIMD (the second launch bound): as many workgroups as the LDS
// (two stages and the selection mask) allows, capped at two waves per SIMD.
template <int D, int CQ>
constexpr int comp_waves_per_simd() {
  constexpr int lds = 2 * (comp_stage_cents<D>() * (4 * D + 4)) + kMaskWords * 4;
  constexpr int by_lds = (160 * 1024) / lds;
  constexpr int by_waves = 8 / (CQ / 32);
  constexpr int blocks = by_lds < by_waves ? (by_lds < 1 ? 1 : by_lds) : by_waves;
  return blocks * (CQ / 32) / 4 < 1 ? 1 : blocks * (CQ / 32) / 4;
}

template <int D, int CQ>
__global__ __launch_bounds__(CQ * 2, (comp_waves_per_simd<D, CQ>())) void comp_bf16_kernel(
    const bf16* __restrict__ qp, const char* __restrict__ tiles,
    const int32_t* __restrict__ lists, const int32_t* __restrict__ lens, int nq, int H, int nqc,
    int nkc, int ntile, int k, float sl2, int enable, const bf16* __restrict__ op,
    const float* __restrict__ lse_s,
    const int32_t* __restrict__ perm_q, bf16* __restrict__ out, float* __restrict__ lse_out,
    Lay lo, int total) {
  constexpr int NW = CQ / 32;
  constexpr int T = NW * 64;
  constexpr int CT = kCompTile;               // centroids per staged tile
  constexpr int HC = comp_stage_cents<D>();   // centroids per LDS stage
  constexpr int SUB = CT / HC;                // stages per tile
  constexpr int MT = HC / 32;
  constexpr int KS = D / 16;
  constexpr int DT = D / 32;
  constexpr int KROW = 2 * D;   // bytes per centroid key row
  constexpr int VROW = 2 * HC;  // bytes per transposed value row in LDS (2 * CT in the tile)
  constexpr int KBYTES = HC * KROW, VBYTES = D * VROW, BBYTES = HC * 4;
  constexpr int STAGE = KBYTES + VBYTES + BBYTES;
  constexpr int TKB = CT * KROW, TVB = D * 2 * CT;  // a staged tile: K, V^T, bias
  constexpr int TILE = TKB + TVB + CT * 4;
  constexpr int KLD = KBYTES / 1024 / NW;  // direct-to-LDS instructions per wave
  constexpr int VLD = VBYTES / 1024 / NW;
  constexpr int BLANES = BBYTES / 16 / NW;  // lanes of each wave copying the bias row
  constexpr int NL = KLD + VLD + 1;
  static_assert(KLD * 1024 * NW == KBYTES && VLD * 1024 * NW == VBYTES, "tile split");
  static_assert(BLANES * 16 * NW == BBYTES, "bias split");
  // Rescale the running output only when a query's maximum logit grows by more
  // than 2^8 (log2 units): exponentials then stay below 256, exact in fp32.
  constexpr float kLazy = 8.0f;
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];
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

  // Operands of the final merge, loaded up front so that their latency
  // overlaps the set-up instead of ending the kernel.
  const bool row_ok = prow < nq;
  float ls = 0.f;
  int orig = 0;
  bf16x4 s4[DT][4];
  // this query cluster's list length (uniform; clamped for memory safety)
  const int nsel = lens ? min(max(lens[(size_t)bh * nqc + a], 1), k) : k;
  const bool do_comp = enable && nsel < nkc;
  const char* th = tiles + (size_t)bh * ntile * TILE;
  const TileCopy<KROW, KLD, NW> kcopy(w, lane);
  const TileCopy<VROW, VLD, NW, 2 * CT> vcopy(w, lane);
  const uint32_t lds0 = lds_addr(smem);
  const int ng = ntile * SUB;  // stages
  // stage g holds centroids [HC (g % SUB), + HC) of tile g / SUB
  auto issue = [&](int g, int stage) {
    const int s = g % SUB;
    const char* src = th + (size_t)(g / SUB) * TILE;
    const uint32_t dst = lds0 + stage * STAGE;
    kcopy.issue(src + s * KBYTES, dst, w);
    vcopy.issue(src + TKB + s * VROW, dst + KBYTES, w);
    const uint32_t boff = (uint32_t)(w * BLANES * 16);
    const uint32_t bdst = __builtin_amdgcn_readfirstlane(dst + KBYTES + VBYTES + boff);
    if (lane < BLANES) lds_dma16(src + TKB + TVB + s * BBYTES, boff + 16 * lane, bdst);
  };
  bf16x8 qreg[KS];
  if (do_comp) {
    for (int i = tid; i < nwords; i += T) selmask[i] = 0u;
    // The first two tiles are copied before the selection is known (a tile
    // whose centroids are all selected is then skipped, not un-copied).
    issue(0, 0);
    if (ng > 1) issue(1, 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qreg[ks] = *(const bf16x8*)(qp + qrow * D + 16 * ks + 8 * h);
  }
  if (row_ok) {
    ls = lse_s[qrow];
    orig = perm_q[(size_t)bh * nq + prow];
    const bf16* srow = op + qrow * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) s4[dt][g] = *(const bf16x4*)(srow + 32 * dt + 8 * g + 4 * h);
  }
  if (do_comp) {
    wait_lgkm();
    raw_barrier();  // selmask cleared
    const int32_t* lst = lists + ((size_t)bh * nqc + a) * k;
    for (int i = tid; i < nsel; i += T) {
      int b = lst[i];
      if (b >= 0 && b < nkc) atomicOr(&selmask[b >> 5], 1u << (b & 31));
    }
    // Retire every load issued so far, including the first two tile copies
    // (a wait the compiler sees), so that no compiler-inserted vmcnt wait
    // lands inside the loop, where it would also wait for the copy in flight.
    __builtin_amdgcn_s_waitcnt(kVmcnt0);
    wait_lgkm();
    raw_barrier();  // selmask complete

    // A stage is live if it holds at least one unselected centroid.
    auto tile_live = [&](int g) {
      int any = 0;
      const int e0 = g * (HC / 32);
      for (int e = e0; e < e0 + HC / 32 && e < nwords; ++e) {
        const uint32_t wmask = e == nwords - 1 && (nkc & 31) ? (1u << (nkc & 31)) - 1u : ~0u;
        any |= (~selmask[e] & wmask) != 0u;
      }
      return __builtin_amdgcn_readfirstlane(any) != 0;
    };
    int koff[KS];
    {
      const int row = kswz(l32);
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) koff[kk] = swz_off<KROW>(row, 2 * kk + h);
    }
    int voff[MT][2];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) voff[mt][s2] = swz_off<VROW>(l32, 4 * mt + 2 * s2 + h);

    auto body = [&](auto stage_tag, int g) {
      constexpr int S = decltype(stage_tag)::value;
      if (g + 1 < ng)
        wait_vmcnt<NL>();
      else
        wait_vmcnt<0>();
      raw_barrier();
      if (tile_live(g)) {
        const char* ks = smem + S * STAGE;
        const char* vs = ks + KBYTES;
        float* bias = (float*)(smem + S * STAGE + KBYTES + VBYTES);
        // Selected clusters are covered by the sparse part: drop them here.
        if (tid < HC) {
          const int b = g * HC + tid;
          if (b < nkc && ((selmask[b >> 5] >> (b & 31)) & 1u)) bias[tid] = -INFINITY;
        }
        f32x16 sacc[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
          for (int r = 0; r < 16; ++r) sacc[mt][r] = 0.f;
#pragma unroll
          for (int kk = 0; kk < KS; ++kk) {
            const bf16x8 av = *(const bf16x8*)(ks + 32 * mt * KROW + koff[kk]);
            sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qreg[kk], sacc[mt], 0, 0, 0);
          }
        }
        wait_lgkm();
        raw_barrier();  // bias row final
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
            const float x = __builtin_fmaf(sacc[mt][r], sl2, bv[r]);
            sacc[mt][r] = x;
            mx = fmaxf(mx, x);
          }
        }
        mx = fmaxf(mx, wave_xor32(mx));
        if (__builtin_amdgcn_ballot_w64(mx > m_run + kLazy)) {
          const float m_new = fmaxf(m_run, mx);
          const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
          l_run *= alpha;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
          m_run = m_new;
        }
        // A query that has seen no live centroid yet has m_run = -inf and only
        // -inf logits: offset by 0 so that they give 0, not NaN.
        const float m_use = m_run == -INFINITY ? 0.f : m_run;
        float lsum = 0.f;
        bf16x8 pb[MT][2];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int s2 = 0; s2 < 2; ++s2) {
            float pv[8];
#pragma unroll
            for (int j = 0; j < 8; ++j)
              pv[j] = __builtin_amdgcn_exp2f(sacc[mt][8 * s2 + j] - m_use);
            pb[mt][s2] = pack8(pv);
            lsum = sum8(pb[mt][s2], lsum);
          }
        l_run += lsum;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
              const bf16x8 av = *(const bf16x8*)(vs + 32 * dt * VROW + voff[mt][s2]);
              oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb[mt][s2], oacc[dt], 0, 0, 0);
            }
      }
      wait_lgkm();
      raw_barrier();  // every wave is done with this stage
      if (g + 2 < ng) issue(g + 2, S);
    };

    for (int g = 0; g < ng; g += 2) {
      body(std::integral_constant<int, 0>{}, g);
      if (g + 1 < ng) body(std::integral_constant<int, 1>{}, g + 1);
    }
  }

  // Merge with the sparse part and write to the original position.
  const float l_tot = l_run + wave_xor32(l_run);
  if (!row_ok) return;
  float ws = 1.f, wc = 0.f, lse = ls, inv_c = 0.f;
  if (l_tot > 0.f) {
    const float lc = (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2;
    const float mm = fmaxf(ls, lc);
    lse = mm + logf(expf(ls - mm) + expf(lc - mm));
    ws = expf(ls - lse);
    wc = expf(lc - lse);
    inv_c = 1.f / l_tot;
  }
  orig = orig < 0 ? 0 : (orig >= nq ? nq - 1 : orig);  // memory safety for a bad permutation
  bf16* orow = out + row_off(bh, orig, lo);
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 v4;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        v4[j] = f2bf(ws * bf2f(s4[dt][g][j]) + wc * (oacc[dt][4 * g + j] * inv_c));
      *(bf16x4*)(orow + 32 * dt + 8 * g + 4 * h) = v4;
    }
  if (lse_out && h == 0) lse_out[(size_t)bh * nq + orig] = lse;
}

// fp32 path: one thread per query, plain FMA; centroids streamed through LDS.
template <int DP>
__global__ __launch_bounds__(256) void comp_f32_kernel(
    const float* __restrict__ qp, const float* __restrict__ cent_k,
    const float* __restrict__ cent_v, const int32_t* __restrict__ count_k,
    const int32_t* __restrict__ lists, const int32_t* __restrict__ lens, int nq, int H, int nqc,
    int nkc, int cq, int d, int k, float scale, int enable, const float* __restrict__ op,
    const float* __restrict__ lse_s,
    const int32_t* __restrict__ perm_q, float* __restrict__ out, float* __restrict__ lse_out,
    Lay lo) {
  constexpr int KC = 32;
  __shared__ float Ksh[KC][DP + 1];
  __shared__ float Vsh[KC][DP + 1];
  __shared__ float bias[KC];
  __shared__ uint32_t selmask[kMaskWords];
  const int a = blockIdx.x, bh = blockIdx.y, i = threadIdx.x;
  const int prow = a * cq + i;
  const bool active = i < cq && prow < nq;
  const size_t qrow = ((size_t)bh * nqc + a) * cq + (i < cq ? i : 0);
  const int nsel = lens ? min(max(lens[(size_t)bh * nqc + a], 1), k) : k;
  const bool do_comp = enable && nsel < nkc;
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
    for (int e = i; e < nsel; e += blockDim.x) {
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
  float* orow = out + row_off(bh, orig, lo);
  // unrolled over DP with a guard, so that o[] stays in registers
#pragma unroll
  for (int t = 0; t < DP; ++t)
    if (t < d) orow[t] = ws * op[qrow * d + t] + wc * (o[t] * inv_c);
  if (lse_out) lse_out[(size_t)bh * nq + orig] = lse;
}

template <int D, int CQ>
hipError_t run_bf16(const Prob& P, const void* qp, const float* cent_k, const float* cent_v,
                    const int32_t* count_k, const int32_t* lists, const int32_t* lens, int k,
                    float scale, int enable, const void* op, const float* lse,
                    const int32_t* perm_q, void* out, float* lse_out, char* tiles,
                    hipStream_t st) {
  const int total = P.BH * P.nqc;
  const int ntile = (P.nkc + kCompTile - 1) / kCompTile;
  const bool do_comp = enable && (k < P.nkc || lens);
  if (do_comp) {
    if (!tiles) return hipErrorInvalidValue;
    hipLaunchKernelGGL(comp_stage_kernel<D>, dim3(ntile, P.BH, 2), dim3(256), 0, st, cent_k,
                       cent_v, count_k, P.nkc, ntile, tiles);
  }
  hipLaunchKernelGGL((comp_bf16_kernel<D, CQ>), dim3(total), dim3(CQ * 2), 0, st,
                     (const bf16*)qp, (const char*)tiles, lists, lens, P.nq, P.H, P.nqc, P.nkc, ntile, k,
                     scale * kLog2e, enable, (const bf16*)op, lse, perm_q, (bf16*)out, lse_out,
                     P.lo, total);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_comp_stage(const Prob& P, const float* cent_k, const float* cent_v,
                             const int32_t* count_k, char* tiles, hipStream_t st) {
  const int ntile = (P.nkc + kCompTile - 1) / kCompTile;
  if (P.d == 64)
    hipLaunchKernelGGL(comp_stage_kernel<64>, dim3(ntile, P.BH, 2), dim3(256), 0, st, cent_k,
                       cent_v, count_k, P.nkc, ntile, tiles);
  else if (P.d == 128)
    hipLaunchKernelGGL(comp_stage_kernel<128>, dim3(ntile, P.BH, 2), dim3(256), 0, st, cent_k,
                       cent_v, count_k, P.nkc, ntile, tiles);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_comp(const Prob& P, const void* qp, const float* cent_k, const float* cent_v,
                       const int32_t* count_k, const int32_t* lists, const int32_t* lens, int k,
                       float scale,
                       int enable, const void* op, const float* lse, const int32_t* perm_q,
                       void* out, float* lse_out, char* tiles, hipStream_t st) {
  if (enable && (k < P.nkc || lens) && P.nkc > kMaskWords * 32) return hipErrorInvalidValue;
  if (P.dtype == CA_BF16) {
#define CA_COMP_CASE(D, CQ) \
  if (P.d == D && P.cq == CQ) \
    return run_bf16<D, CQ>(P, qp, cent_k, cent_v, count_k, lists, lens, k, scale, enable, op, lse, \
                           perm_q, out, lse_out, tiles, st);
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
                     cent_k, cent_v, count_k, lists, lens, P.nq, P.H, P.nqc, P.nkc, P.cq, P.d, \
                     k,                                                                       \
                     scale, enable, (const float*)op, lse, perm_q, (float*)out, lse_out,      \
                     P.lo)
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
