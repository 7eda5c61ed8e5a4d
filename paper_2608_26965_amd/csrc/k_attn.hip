// Block-sparse attention over selected key clusters (paper: Method, Overview -
// attention over the selected clusters, returning the softmax denominator).
//
// One workgroup per (head, query cluster); the workgroup streams the k
// selected key-cluster tiles through LDS (double-buffered) and runs an online
// softmax. bf16: MFMA 32x32x16 with fp32 accumulation, one wavefront per 32
// queries. fp32: plain FMA, one thread per query.
#include <math.h>

#include <type_traits>

#include "attn_tile.h"

namespace ca {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// s_waitcnt immediate (gfx9 encoding) waiting for vmcnt = 0 only.
constexpr int kVmcnt0 = 0x0F70;

// Workgroup w of a 1-D grid runs on XCD w % 8. The items (head, query
// cluster) are numbered so that each XCD takes a contiguous eighth of a head's
// query clusters (neighbouring query clusters share most selected key tiles,
// which then stay in that XCD's L2), and all eight XCDs work on the same head
// at a time. Slot loc of XCD x holds query cluster x * chunk + loc % chunk of
// head loc / chunk, chunk = ceil(nqc / 8); slots past nqc hold nothing.
__device__ __forceinline__ int head_sync_item(int wg, int nqc, int total) {
  const int x = wg & 7, loc = wg >> 3, chunk = (nqc + 7) >> 3;
  const int bh = loc / chunk, a = x * chunk + loc % chunk;
  return a < nqc && bh * nqc < total ? bh * nqc + a : -1;
}

// Keys per LDS stage: 64, so a key cluster of 128 is two stages. The two
// stages then take 16 KB (d = 64) or 32 KB (d = 128) per buffer pair instead
// of twice that, and the logits of a stage need half the registers: at d = 64
// with query clusters of 128 three workgroups share a CU (three waves per
// SIMD) instead of two, and at d = 128 two instead of one.
template <int D, int CQ, int CK>
constexpr int attn_stage_keys() {
  return CK == 128 ? 64 : CK;
}

// Key halves per stage (SPLIT, query clusters of 64 only). A query cluster of
// 64 is two wavefronts of 32 queries; with d = 128 its double-buffered stages
// (64 KB) let two workgroups share a CU, one wavefront per SIMD with nothing
// to overlap one wave's matrix products with, and with d = 64 LDS allows two
// and a half. Splitting every stage's keys in two gives four wavefronts per
// workgroup in the same LDS: wavefront w takes queries 32 (w % 2) .. + 31
// against the keys of row tile w / 2 of every stage, with a softmax state of
// its own, and the two key halves of a query are merged at the end. The
// launch takes it where a query cluster's selected tiles fit in one XCD's L2
// (4 MiB): beyond that it measured slower than two wavefronts. (For query
// clusters of 128 it measured slower everywhere: eight wavefronts with half
// the work each, and one workgroup per CU.)
template <int D, int CQ, int CK, bool SPLIT>
constexpr int attn_key_split() {
  return CQ == 64 && SPLIT ? 2 : 1;
}
template <int D, int CQ, int CK, bool SPLIT>
constexpr int attn_waves() {
  return CQ / 32 * attn_key_split<D, CQ, CK, SPLIT>();
}
// the key-split kernel for k selected clusters per query cluster
template <int D, int CQ, int CK>
inline bool attn_use_split(int k) {
  return CQ == 64 && (size_t)k * CK * D * 4 <= ((size_t)4 << 20);
}

// Waves per SIMD the bf16 kernel is compiled for (the second launch bound, a
// minimum): as many workgroups as their double-buffered stages fit in LDS,
// capped at two waves per SIMD, so that the MFMA of one wave overlaps the
// softmax of another. Where registers and LDS allow, more workgroups run.
template <int D, int CQ, int CK, bool SPLIT>
constexpr int attn_waves_per_simd() {
  constexpr int nw = attn_waves<D, CQ, CK, SPLIT>();
  constexpr int by_lds = (160 * 1024) / (8 * D * attn_stage_keys<D, CQ, CK>());
  constexpr int by_waves = 8 / nw;
  constexpr int blocks = by_lds < by_waves ? (by_lds < 1 ? 1 : by_lds) : by_waves;
  return blocks * nw / 4 < 1 ? 1 : blocks * nw / 4;
}

// Compensation folded into the attention kernel: the staged centroid tiles of
// the unselected clusters are extra stages of the same online softmax, with
// log2 of the cluster size added to their logits (the merged output of the
// paper's two partial results, formed without writing either of them), and
// the rows go to their original positions.
struct FusedArgs {
  const char* tiles;      // staged centroid tiles [BH][ntile] (NULL: no compensation)
  int ntile;
  const int32_t* perm_q;  // [BH][nq]
  bf16* out;              // strides lo
  float* lse_out;         // [BH][nq] or NULL
  int nq;
  Lay lo;
};

template <int D, int CQ, int CK, bool FUSED, bool SPLIT>
__global__ __launch_bounds__((64 * attn_waves<D, CQ, CK, SPLIT>()),
                             (attn_waves_per_simd<D, CQ, CK, SPLIT>())) void attn_bf16_kernel(
    const bf16* __restrict__ qp, const bf16* __restrict__ kp, const bf16* __restrict__ vp,
    const int32_t* __restrict__ count_k, const int32_t* __restrict__ lists,
    const int32_t* __restrict__ lens, int nqc, int nkc, int k, float sl2, bf16* __restrict__ op,
    float* __restrict__ lse, int total, const int32_t* __restrict__ sched, int cap,
    FusedArgs fa = FusedArgs{}) {
  constexpr int QW = CQ / 32;                       // query tiles
  constexpr int KSPL = attn_key_split<D, CQ, CK, SPLIT>();  // key halves
  constexpr int NW = QW * KSPL;                      // wavefronts
  constexpr int NT = 64 * NW;
  constexpr int HK = attn_stage_keys<D, CQ, CK>();  // keys per stage
  // Where two or more waves share a SIMD, VALU instructions are what the loop
  // is short of: the logits' starting value -m_ref then sits in 16 registers
  // of its own, refreshed only when the reference moves (no per-stage
  // register fill). The key-split kernels (query clusters of 64) keep the
  // fill: the copy would cost them a wave per SIMD (d = 64) or spill (d = 128).
  constexpr bool LEAN = attn_waves_per_simd<D, CQ, CK, SPLIT>() > 1 && KSPL == 1;
  constexpr int SUB = CK / HK;                      // stages per key cluster
  constexpr int MT = HK / 32;   // row tiles of a stage
  constexpr int MW = MT / KSPL;  // row tiles of a stage per wavefront
  static_assert(MW * KSPL == MT, "key split");
  constexpr int KS = D / 16;
  constexpr int DT = D / 32;
  constexpr int KROW = 2 * D;   // bytes per K row
  constexpr int VROW = 2 * HK;  // bytes per V^T row in LDS (2 * CK in HBM)
  constexpr int KBYTES = HK * KROW, VBYTES = D * VROW;
  constexpr int STAGE = KBYTES + VBYTES;
  constexpr int KLD = KBYTES / 1024 / NW;  // direct-to-LDS instructions per wave
  constexpr int VLD = VBYTES / 1024 / NW;
  static_assert(KLD * 1024 * NW == KBYTES && VLD * 1024 * NW == VBYTES, "tile split");
  __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];
  // fused: the query cluster's selection bitmap and the two stages' bias rows
  __shared__ uint32_t selmask[FUSED ? kMaskWords : 1];
  __shared__ int redo;  // some wavefront's fast pass overflowed
  __shared__ __attribute__((aligned(16))) float cbias[2][FUSED ? HK : 4];
  constexpr int SUBC = kCompTile / HK;                     // stages per centroid tile
  constexpr int CTK = kCompTile * KROW, CTV = D * 2 * kCompTile;
  constexpr int CTILE = CTK + CTV + kCompTile * 4;        // bytes of a staged centroid tile
  constexpr int BLANES = FUSED ? HK / 4 / NW : 1;          // lanes per wave copying a bias row
  static_assert(!FUSED || (BLANES >= 1 && BLANES * 16 * NW == HK * 4), "bias split");

  int item;
  if (sched) {
    // scheduled launch: slot loc of XCD x (workgroups run on XCD blockIdx % 8)
    const int x = blockIdx.x & 7, loc = blockIdx.x >> 3;
    if (loc >= sched[x]) return;
    item = sched[8 + x * cap + loc];
  } else {
    item = head_sync_item(blockIdx.x, nqc, total);
    if (item < 0) return;
  }
  const int bh = item / nqc, a = item - bh * nqc;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  // query tile, key half (row tiles kh MW .. + MW - 1)
  const int qw = KSPL > 1 ? w % QW : w, kh = KSPL > 1 ? w / QW : 0;
  const size_t nq_pad = (size_t)nqc * CQ, nk_pad = (size_t)nkc * CK;
  const size_t qrow = (size_t)bh * nq_pad + (size_t)a * CQ + 32 * qw + l32;

  // Queries pre-scaled by sl2 = scale * log2(e) (rounded to bf16 once), so
  // that the logits come out in the exponent's units.
  bf16x8 qreg[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    const bf16x8 q8 = *(const bf16x8*)(qp + qrow * D + 16 * ks + 8 * h);
    float qf[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) qf[i] = (float)q8[i] * sl2;
    qreg[ks] = pack8(qf);
  }
  // Retire the query loads here (a wait the compiler sees), so that no
  // compiler-inserted vmcnt wait lands inside the loop, where it would also
  // wait for the in-flight copy of the next tile.
  __builtin_amdgcn_s_waitcnt(kVmcnt0);

  if (tid == 0) redo = 0;  // ordered before any write by the first stage's barrier
  const int32_t* lst = lists + ((size_t)bh * nqc + a) * k;
  const int32_t* cnth = count_k + (size_t)bh * nkc;
  // this query cluster's list length (uniform; clamped for memory safety)
  const int nt = lens ? min(max(lens[(size_t)bh * nqc + a], 1), k) : k;
  // centroid stages (fused, when some cluster is unselected)
  const int nc = FUSED && fa.tiles && nt < nkc ? fa.ntile * SUBC : 0;
  if (FUSED && nc) {
    const int nwords = (nkc + 31) >> 5;
    for (int i = tid; i < nwords; i += NT) selmask[i] = 0u;
    __syncthreads();
    for (int i = tid; i < nt; i += NT) {
      const int b = lst[i];
      if (b >= 0 && b < nkc) atomicOr(&selmask[b >> 5], 1u << (b & 31));
    }
    // ordered before any read by the first stage's barrier
  }
  auto tile_id = [&](int t) {
    int b = lst[t];
    return b < 0 ? 0 : (b >= nkc ? nkc - 1 : b);
  };
  const TileCopy<KROW, KLD, NW> kcopy(w, lane);
  const TileCopy<VROW, VLD, NW, 2 * CK> vcopy(w, lane);
  // LDS: two key buffers, then two value buffers
  const uint32_t lds0 = lds_addr(smem);
  const uint32_t ldsk = lds0, ldsv = lds0 + 2 * KBYTES;
  // stage g holds keys [HK (g % SUB), HK (g % SUB) + HK) of list entry g / SUB
  auto issue_k = [&](int g, int kb) __attribute__((always_inline)) {
    const int b = tile_id(g / SUB), s = g % SUB;
    kcopy.issue(kp + ((size_t)bh * nk_pad + (size_t)b * CK + (size_t)s * HK) * D,
                ldsk + kb * KBYTES, w);
  };
  auto issue_v = [&](int g, int vb) __attribute__((always_inline)) {
    const int b = tile_id(g / SUB), s = g % SUB;
    vcopy.issue(vp + ((size_t)bh * nkc + b) * (size_t)D * CK + (size_t)s * HK, ldsv + vb * VBYTES,
                w);
  };
  // fused: centroid stage c holds centroids [HK (c % SUBC), + HK) of centroid
  // tile c / SUBC, with their bias row in cbias
  const TileCopy<VROW, VLD, NW, 2 * kCompTile> ccopy(w, lane);
  const char* ctl = FUSED && nc ? fa.tiles + (size_t)bh * fa.ntile * CTILE : nullptr;
  auto issue_c = [&](int c, int kb, int vb, int sb) __attribute__((always_inline)) {
    const int s = c % SUBC;
    const char* src = ctl + (size_t)(c / SUBC) * CTILE;
    kcopy.issue(src + s * KBYTES, ldsk + kb * KBYTES, w);
    ccopy.issue(src + CTK + s * VROW, ldsv + vb * VBYTES, w);
    const uint32_t boff = (uint32_t)(w * BLANES * 16);
    const uint32_t bdst = __builtin_amdgcn_readfirstlane(lds_addr(&cbias[sb][0]) + boff);
    if (lane < BLANES) lds_dma16(src + CTK + CTV + s * HK * 4, boff + 16 * lane, bdst);
  };
  // Loop-invariant LDS read offsets (rows r and r + 32 share the swizzle key).
  int koff[KS];  // with this wavefront's first row tile
  {
    const int row = kswz(l32);
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) koff[kk] = 32 * MW * kh * KROW + swz_off<KROW>(row, 2 * kk + h);
  }
  int voff[MW][2];
#pragma unroll
  for (int mt = 0; mt < MW; ++mt)
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
      voff[mt][s2] = swz_off<VROW>(l32, 4 * (MW * kh + mt) + 2 * s2 + h);

  f32x16 oacc[DT];
  // m_run: running maximum of the scaled logits (log2 units); m_ref: the value
  // the current stage's accumulators start from (-m_ref), so that they hold
  // logit - m_ref and the exponentials need no subtraction.
  float m_run = -INFINITY, m_ref = 0.f;
  f32x16 sinit;  // LEAN: -m_ref in every entry, the first logit product's addend
#pragma unroll
  for (int r = 0; r < 16; ++r) sinit[r] = -m_ref;
  f32x16 sacc[MW];   // logits of this wavefront's keys of the current stage
  bf16x8 pb[MW][2];  // their probabilities (bf16), the value product's operand
  // Row sums on the matrix cores instead of the VALU: a 16x16x32 product of
  // a 0/1 selector R with a probability group (the group's B operand: lane l
  // holds its 8 keys of query l % 32, in k block l / 16) gives in row 0,
  // column n the group's sum for query n (k blocks 0 and 2: lanes n, n + 32)
  // and in row 1 that for query n + 16 (blocks 1 and 3); the other rows are 0.
  // Lane n < 16 thus holds the sums of queries n and n + 16 in entries 0 and 1
  // of the product (lane l holds rows 4 (l / 16) .. + 3 of column l % 16).
  bf16x8 rsel;  // lane l holds R[l % 16][k block l / 16]
  {
    const __bf16 one = (__bf16)((lane & 15) == ((lane >> 4) & 1) ? 1.f : 0.f);
#pragma unroll
    for (int i = 0; i < 8; ++i) rsel[i] = one;
  }
  f32x4 lacc;  // running row sums in that layout
  f32x4 ssum;  // the row sums of a stage that is still to be settled

  // S^T = K Q^T for the stage in key buffer ks
  auto logits = [&](const char* ks) __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < MW; ++mt) {
      if constexpr (!LEAN) {
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[mt][r] = -m_ref;
      }
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        const bf16x8 av = *(const bf16x8*)(ks + 32 * mt * KROW + koff[kk]);
        sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qreg[kk],
                                                           LEAN && kk == 0 ? sinit : sacc[mt], 0, 0, 0);
      }
    }
  };
  // keys of a stage past its cluster's count are padding
  auto mask_pad = [&](int cnt) __attribute__((always_inline)) {
    if (cnt < HK) {
      // only the remainder cluster of a head. Accumulator r of row tile mt
      // holds key 32 mt + 16 (r / 8) + 8 h + r % 8 (acc_key), so the test
      // compares cnt - 8 h with constants and keeps no per-key registers.
      const int ch = cnt - 8 * h - 32 * MW * kh;
#pragma unroll
      for (int mt = 0; mt < MW; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (32 * mt + 16 * (r >> 3) + (r & 7) >= ch) sacc[mt][r] = -INFINITY;
    }
  };
  // probabilities of accumulator group (mt, s2) against m_ref (the
  // accumulators already hold logit - m_ref), or with OFF against m_ref - off,
  // with their row sums added to rs
  auto exp_group = [&](auto off_tag, int mt, int s2, float off, f32x4& rs)
                       __attribute__((always_inline)) {
    float pv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      pv[j] = __builtin_amdgcn_exp2f(decltype(off_tag)::value ? sacc[mt][8 * s2 + j] + off
                                                              : sacc[mt][8 * s2 + j]);
    pb[mt][s2] = pack8(pv);
    rs = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rsel, pb[mt][s2], rs, 0, 0, 0);
  };
  auto exps = [&](auto off_tag, float off, f32x4& rs) __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < MW; ++mt)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) exp_group(off_tag, mt, s2, off, rs);
  };
  // O^T += V^T P^T for the previous stage's probabilities, each group's two
  // (DT) products issued right before that group's probabilities of this
  // stage overwrite them, so the matrix cores run while the exponentials of
  // the next group are formed
  auto pv_exps = [&](const char* vs, f32x4& rs) __attribute__((always_inline)) {
#pragma unroll
    for (int mt = 0; mt < MW; ++mt)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
          const bf16x8 av = *(const bf16x8*)(vs + 32 * dt * VROW + voff[mt][s2]);
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb[mt][s2], oacc[dt], 0, 0, 0);
        }
        exp_group(std::false_type{}, mt, s2, 0.f, rs);
      }
  };
  auto pv = [&](const char* vs) __attribute__((always_inline)) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int mt = 0; mt < MW; ++mt)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const bf16x8 av = *(const bf16x8*)(vs + 32 * dt * VROW + voff[mt][s2]);
          oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb[mt][s2], oacc[dt], 0, 0, 0);
        }
  };
  // Settle a stage whose exponentials were taken against m_ref and whose row
  // sums are in ssum: where this is the first stage (no maximum yet; its
  // accumulators start from 0), or a row sum of the stage exceeds 2^40 (a jump
  // of about 2^34 in a probability), the stage is redone against its own
  // maximum and the output and row sums accumulated so far are rescaled to
  // it. Large exponentials below that cost no accuracy (fp32 and bf16 keep
  // their relative precision at any scale).
  auto settle = [&]() __attribute__((always_inline)) {
    if (__builtin_amdgcn_ballot_w64(!(fmaxf(ssum[0], ssum[1]) <= 0x1p40f) || m_run == -INFINITY)) {
      float mx = -INFINITY;
#pragma unroll
      for (int mt = 0; mt < MW; ++mt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[mt][r]);
      mx = fmaxf(mx, wave_xor32(mx));
      const float m_new = fmaxf(m_run, m_ref + mx);
      // split keys: no maximum yet where every key of the wavefront's half so
      // far was padding (its sums stay 0)
      const float m_use = KSPL > 1 && m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
      // lane n < 16 holds the sums of queries n and n + 16
      lacc[0] *= alpha;
      lacc[1] *= __shfl_xor(alpha, 16, 64);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
      ssum = f32x4{0.f, 0.f, 0.f, 0.f};
      exps(std::true_type{}, m_ref - m_use, ssum);
      m_run = m_new;
      if constexpr (LEAN) {
#pragma unroll
        for (int r = 0; r < 16; ++r) sinit[r] = -m_use;
      }
    }
    lacc[0] += ssum[0];
    lacc[1] += ssum[1];
    m_ref = KSPL > 1 && m_run == -INFINITY ? 0.f : m_run;
  };
  auto sync_stage = [&]() __attribute__((always_inline)) {
    wait_vmcnt<0>();
    wait_lgkm();
    raw_barrier();
  };

  // All stages of the query cluster: the key stages, then (fused) the
  // centroid stages. The first stage sets the reference m_ref (its maximum).
  // In the fast pass (SAFE false) every later stage is taken against that
  // reference as it stands, with no check: probabilities may exceed 1, which
  // costs no accuracy while nothing overflows, and whether anything did is
  // checked once at the end. The safe pass settles every stage as above; it
  // runs only for a query cluster whose fast pass overflowed (a logit jump of
  // about 2^7 or more in log2 units over the first stage's maximum).
  //
  // Key stages, software-pipelined one stage deep. Stage g's keys sit in key
  // buffer g % 2 and its values in value buffer g % 2. At iteration g, after
  // the one barrier (every wavefront is past iteration g-1, so key buffer
  // (g+1) % 2 and value buffer g % 2 are free, and the copies issued at
  // iteration g-1 have landed), the keys of stage g+1 and the values of stage
  // g are copied; the logits of stage g are formed, then the value product of
  // stage g-1 runs interleaved with the exponentials of stage g. The last
  // value product follows the loop.
  const int ng = nt * SUB;
  const char* kbuf0 = smem;
  const char* kbuf1 = smem + KBYTES;
  const char* vbuf0 = smem + 2 * KBYTES;
  const char* vbuf1 = smem + 2 * KBYTES + VBYTES;
  auto run = [&](auto safe_tag) __attribute__((always_inline)) {
    constexpr bool SAFE = decltype(safe_tag)::value;
    m_run = -INFINITY;
    m_ref = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) sinit[r] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[dt][r] = 0.f;
    lacc = f32x4{0.f, 0.f, 0.f, 0.f};
    // a stage's exponentials and their row sums: settled (safe pass) or
    // added to the running sums as they are (fast pass)
    auto stage_exps = [&](auto with_pv, const char* vs) __attribute__((always_inline)) {
      if constexpr (SAFE) ssum = f32x4{0.f, 0.f, 0.f, 0.f};
      f32x4& rs = SAFE ? ssum : lacc;
      if constexpr (decltype(with_pv)::value)
        pv_exps(vs, rs);
      else
        exps(std::false_type{}, 0.f, rs);
      if constexpr (SAFE) settle();
    };
    issue_k(0, 0);
    {
      sync_stage();
      if (1 < ng) issue_k(1, 1);
      issue_v(0, 0);
      logits(kbuf0);
      mask_pad(cnth[tile_id(0)]);
      ssum = f32x4{0.f, 0.f, 0.f, 0.f};
      exps(std::false_type{}, 0.f, ssum);
      settle();
    }
    auto step = [&](auto par_tag, int g) __attribute__((always_inline)) {
      constexpr int P = decltype(par_tag)::value;  // g % 2
      sync_stage();
      if (g + 1 < ng) issue_k(g + 1, P ^ 1);
      issue_v(g, P);
      logits(P ? kbuf1 : kbuf0);
      mask_pad(cnth[tile_id(g / SUB)] - (g % SUB) * HK);
      stage_exps(std::true_type{}, P ? vbuf0 : vbuf1);
    };
    for (int g = 1; g < ng; g += 2) {
      step(std::integral_constant<int, 1>{}, g);
      if (g + 1 < ng) step(std::integral_constant<int, 0>{}, g + 1);
    }
    // the last key stage's value product; the first centroid stage's copies go
    // to the free buffers (both key buffers, value buffer ng % 2) meanwhile
    sync_stage();
    if (FUSED && nc) issue_c(0, 0, ng & 1, 0);
    pv((ng & 1) ? vbuf0 : vbuf1);
    if constexpr (FUSED) {
      // Centroid stages (compensation), after the keys and not pipelined:
      // centroid stage c sits in key buffer c % 2, value buffer (ng + c) % 2
      // and bias row c % 2. The selected clusters are covered by the sparse
      // part: their bias is set to -inf once the row has landed.
      for (int c = 0; c < nc; ++c) {
        const int sb = c & 1, vb = (ng + c) & 1;
        sync_stage();
        if (c + 1 < nc) issue_c(c + 1, sb ^ 1, vb ^ 1, sb ^ 1);
        if (tid < HK) {
          const int b = (c / SUBC) * kCompTile + (c % SUBC) * HK + tid;
          if (b < nkc && ((selmask[b >> 5] >> (b & 31)) & 1u)) cbias[sb][tid] = -INFINITY;
        }
        wait_lgkm();
        raw_barrier();  // bias row final
        logits(sb ? kbuf1 : kbuf0);
        // logit + log2|b|, so that the exponent is sl2 q.kbar + log2|b| - m.
        // The bias of accumulator r of row tile mt is that of key acc_key(mt, r, h):
        // two runs of eight consecutive entries.
#pragma unroll
        for (int mt = 0; mt < MW; ++mt)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const float* brow = &cbias[sb][32 * (MW * kh + mt) + 16 * hh + 8 * h];
            const float4 b0 = *(const float4*)brow;
            const float4 b1 = *(const float4*)(brow + 4);
            const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
            for (int j = 0; j < 8; ++j)
              sacc[mt][8 * hh + j] += bv[j];
          }
        stage_exps(std::false_type{}, nullptr);
        pv(vb ? vbuf1 : vbuf0);
      }
    }
  };
  // the row sum of this lane's query q = lane % 32: lane q % 16, entry q / 16
  auto row_total = [&]() __attribute__((always_inline)) {
    const float l_lo = __shfl(lacc[0], lane & 15, 64), l_hi = __shfl(lacc[1], lane & 15, 64);
    return (lane & 16) ? l_hi : l_lo;
  };
  run(std::false_type{});
  float l_tot = row_total();
  {
    // Did the fast pass overflow? Its row sums are at least 1 (the first
    // stage's maximum) unless something became inf or NaN.
    // A wavefront whose first stage was all padding (a key half past its
    // cluster's count) has no reference yet: the safe pass sets one.
    bool ok = l_tot <= 0x1p126f && (KSPL == 1 || m_run > -INFINITY);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) ok = ok && fabsf(oacc[dt][r]) <= 0x1.fffffep127f;
    if (__builtin_amdgcn_ballot_w64(!ok) && lane == 0) redo = 1;
    __syncthreads();  // also: every wavefront is done with the stage buffers
    if (redo) {
      run(std::true_type{});
      l_tot = row_total();
    }
  }
  // the state's reference: the row sums and outputs are taken against m_ref
  float m_fin = KSPL > 1 ? m_ref : m_run;
  if constexpr (KSPL > 1) {
    // Key half 1 hands its state (reference, row sum, output accumulators) to
    // key half 0 through the stage buffers; the merged state takes the larger
    // reference of the halves that hold any key.
    static_assert(KSPL == 2, "two key halves");
    constexpr int NV = 2 + 16 * DT;  // floats per lane
    // query tiles per round: as many as the stage buffers hold
    constexpr int QR = (2 * STAGE) / (NV * 64 * 4) < QW ? (2 * STAGE) / (NV * 64 * 4) : QW;
    static_assert(QR >= 1, "merge buffer");
    for (int q0 = 0; q0 < QW; q0 += QR) {
      const bool mine = qw >= q0 && qw < q0 + QR;
      float* mb = (float*)smem + (qw - q0) * NV * 64 + lane;  // entry i at mb[64 i] (if mine)
      __syncthreads();  // every wavefront is done with the stage buffers
      if (kh == 1 && mine) {
        mb[0] = m_ref;
        mb[64] = l_tot;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) mb[64 * (2 + 16 * dt + r)] = oacc[dt][r];
      }
      __syncthreads();
      if (kh == 0 && mine) {
        const float lb = mb[64];
        const float ma = l_tot > 0.f ? m_ref : -INFINITY, mbb = lb > 0.f ? mb[0] : -INFINITY;
        const float m = fmaxf(ma, mbb);
        const float mu = m == -INFINITY ? 0.f : m;
        const float sa = __builtin_amdgcn_exp2f(ma - mu), sb = __builtin_amdgcn_exp2f(mbb - mu);
        l_tot = l_tot * sa + lb * sb;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[dt][r] = oacc[dt][r] * sa + mb[64 * (2 + 16 * dt + r)] * sb;
        m_fin = mu;
      }
    }
    if (kh == 1) return;
  }
  const float inv = 1.f / l_tot;
  if constexpr (FUSED) {
    // merged rows to their original positions
    const int prow = a * CQ + 32 * qw + l32;
    if (prow >= fa.nq) return;
    int orig = fa.perm_q[(size_t)bh * fa.nq + prow];
    orig = orig < 0 ? 0 : (orig >= fa.nq ? fa.nq - 1 : orig);  // memory safety for a bad permutation
    bf16* orow = fa.out + row_off(bh, orig, fa.lo);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 v4;
#pragma unroll
        for (int j = 0; j < 4; ++j) v4[j] = f2bf(oacc[dt][4 * g + j] * inv);
        *(bf16x4*)(orow + 32 * dt + 8 * g + 4 * h) = v4;
      }
    if (fa.lse_out && h == 0)
      fa.lse_out[(size_t)bh * fa.nq + orig] = (m_fin + __builtin_amdgcn_logf(l_tot)) * kLn2;
    return;
  }
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
  if (h == 0) lse[qrow] = (m_fin + __builtin_amdgcn_logf(l_tot)) * kLn2;
}

// fp32 path: one thread per query, keys streamed through LDS 32 at a time.
template <int DP>
__global__ __launch_bounds__(256) void attn_f32_kernel(
    const float* __restrict__ qp, const float* __restrict__ kp, const float* __restrict__ vp,
    const int32_t* __restrict__ count_k, const int32_t* __restrict__ lists,
    const int32_t* __restrict__ lens, int nqc, int nkc, int cq, int ck, int d, int k, float scale,
    float* __restrict__ op, float* __restrict__ lse) {
  // 256 threads: query i of the cluster (qpad = cq rounded up to 64) and key
  // part part = tid / qpad of parts = 256 / qpad; part p takes keys p, p +
  // parts, ... of every staged chunk with a softmax state of its own, and the
  // parts are merged at the end (32 queries at a time through LDS).
  constexpr int KC = 32, QB = 32;
  __shared__ float Ksh[KC][DP + 1];
  __shared__ float Vsh[KC][DP + 1];
  __shared__ float mrg[(DP + 2) * QB];  // [field][query of the round]
  const int a = blockIdx.x, bh = blockIdx.y;
  const int qpad = (cq + 63) / 64 * 64, parts = 256 / qpad;
  const int i = threadIdx.x % qpad, part = threadIdx.x / qpad;
  const bool active = i < cq && part < parts;
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
  const int nt = lens ? min(max(lens[(size_t)bh * nqc + a], 1), k) : k;
  for (int tt = 0; tt < nt; ++tt) {
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
      for (int kk = part; kk < nk; kk += parts) {
        // four partial sums: four short dependency chains instead of one
        float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll
        for (int t = 0; t < DP; t += 4) {
          s0 = __builtin_fmaf(q[t], Ksh[kk][t], s0);
          s1 = __builtin_fmaf(q[t + 1], Ksh[kk][t + 1], s1);
          s2 = __builtin_fmaf(q[t + 2], Ksh[kk][t + 2], s2);
          s3 = __builtin_fmaf(q[t + 3], Ksh[kk][t + 3], s3);
        }
        const float s = ((s0 + s1) + (s2 + s3)) * scale;
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
  // merge the key parts into part 0 (a part without keys has l = 0)
  for (int q0 = 0; q0 < qpad; q0 += QB) {
    const bool inq = i >= q0 && i < q0 + QB;
    for (int pp = 1; pp < parts; ++pp) {
      __syncthreads();
      if (active && inq && part == pp) {
        const int j = i - q0;
        mrg[j] = m;
        mrg[QB + j] = l;
#pragma unroll
        for (int t = 0; t < DP; ++t) mrg[(2 + t) * QB + j] = o[t];
      }
      __syncthreads();
      if (active && inq && part == 0) {
        const int j = i - q0;
        const float lb = mrg[QB + j];
        const float ma = l > 0.f ? m : -INFINITY, mb = lb > 0.f ? mrg[j] : -INFINITY;
        const float mm = fmaxf(ma, mb);
        const float mu = mm == -INFINITY ? 0.f : mm;
        const float sa = expf(ma - mu), sb = expf(mb - mu);
        l = l * sa + lb * sb;
#pragma unroll
        for (int t = 0; t < DP; ++t) o[t] = o[t] * sa + mrg[(2 + t) * QB + j] * sb;
        m = mu;
      }
    }
  }
  if (active && part == 0) {
    const float inv = 1.f / l;
    // unrolled over DP with a guard: a loop to d would index o[] at run time
    // and move it to scratch memory
#pragma unroll
    for (int t = 0; t < DP; ++t)
      if (t < d) op[qrow * d + t] = o[t] * inv;
    lse[qrow] = m + logf(l);
  }
}

// Launch order for lists of different lengths. Work of an item (head, query
// cluster) = its list length + 2 (the per-workgroup fixed cost in tiles). The
// items are cut into eight contiguous ranges of about equal work (an item
// goes to XCD floor(8 * work before it / total work)), each range holding at
// most cap items, so neighbouring query clusters (which share key tiles)
// still meet in one L2; block x then lists its range longest first (counting
// sort on the length; the order among equal lengths is not fixed, and does not
// change any result). sched[x] = items of XCD x, sched[8 + x * cap + i] = its
// i-th item.
constexpr int kSchedThreads = 1024;
constexpr int kSchedBins = 4096;

__global__ __launch_bounds__(kSchedThreads) void attn_sched_kernel(const int32_t* __restrict__ lens,
                                                                   int total, int k, int cap,
                                                                   int32_t* __restrict__ sched) {
  __shared__ long long wsum[kSchedThreads / 64];
  __shared__ int bound[9];
  __shared__ int hist[kSchedBins];
  const int x = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  auto work = [&](int i) { return (long long)min(max(lens[i], 1), k) + 2; };
  // 1. exclusive prefix of the work at each thread's contiguous chunk
  const int per = (total + kSchedThreads - 1) / kSchedThreads;
  const int i0 = min(tid * per, total), i1 = min(i0 + per, total);
  long long mine = 0;
  for (int i = i0; i < i1; ++i) mine += work(i);
  long long incl = mine;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const long long y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wsum[wv] = incl;
  if (tid < 9) bound[tid] = tid == 0 ? 0 : total;
  __syncthreads();
  long long before = incl - mine, W = 0;
  for (int i = 0; i < kSchedThreads / 64; ++i) {
    before += i < wv ? wsum[i] : 0;
    W += wsum[i];
  }
  // 2. range boundaries: the first item whose prefix reaches y * W / 8
  {
    long long pre = before;
    for (int i = i0; i < i1; ++i) {
      const long long nxt = pre + work(i);
#pragma unroll
      for (int y = 1; y < 8; ++y) {
        const long long t = (long long)y * W;
        if (8 * pre < t && 8 * nxt >= t) bound[y] = i + 1;
      }
      pre = nxt;
    }
  }
  __syncthreads();
  if (tid == 0) {
    // at most cap items per range, and room for the rest in the ranges after
    int b = 0;
    for (int y = 1; y < 8; ++y) {
      int v = min(bound[y], b + cap);
      v = max(v, total - (8 - y) * cap);
      v = max(v, b);
      bound[y] = v;
      b = v;
    }
  }
  for (int e = tid; e < kSchedBins; e += kSchedThreads) hist[e] = 0;
  __syncthreads();
  const int r0 = bound[x], r1 = bound[x + 1];
  auto key = [&](int i) {
    const int len = min(max(lens[i], 1), k);
    const int bin = k <= kSchedBins ? len - 1 : (int)((long long)(len - 1) * kSchedBins / k);
    return kSchedBins - 1 - bin;  // longest first
  };
  // 3. counting sort of the range
  for (int i = r0 + tid; i < r1; i += kSchedThreads) atomicAdd(&hist[key(i)], 1);
  __syncthreads();
  if (tid < 64) {
    // exclusive scan of the bins, 64 per lane
    int s = 0;
    for (int j = 0; j < kSchedBins / 64; ++j) s += hist[64 * tid + j];
    int inc = s;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(inc, o, 64);
      if (lane >= o) inc += y;
    }
    int run = inc - s;
    for (int j = 0; j < kSchedBins / 64; ++j) {
      const int c = hist[64 * tid + j];
      hist[64 * tid + j] = run;
      run += c;
    }
  }
  __syncthreads();
  int32_t* out = sched + 8 + (size_t)x * cap;
  for (int i = r0 + tid; i < r1; i += kSchedThreads) out[atomicAdd(&hist[key(i)], 1)] = i;
  if (tid == 0) sched[x] = r1 - r0;
}

template <int D, int CQ, int CK, bool FUSED = false>
hipError_t run_bf16(const Prob& P, const void* qp, const void* kp, const void* vp,
                    const int32_t* count_k, const int32_t* lists, const int32_t* lens, int k,
                    float scale, void* op, float* lse, int32_t* sched, hipStream_t st,
                    FusedArgs fa = FusedArgs{}) {
  const int total = P.BH * P.nqc;
  const int cap = attn_sched_cap(total);
  if (sched && lens) {
    hipLaunchKernelGGL(attn_sched_kernel, dim3(8), dim3(kSchedThreads), 0, st, lens, total, k, cap,
                       sched);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  } else {
    sched = nullptr;
  }
  auto launch = [&](auto split_tag) {
    constexpr bool SPLIT = decltype(split_tag)::value;
    hipLaunchKernelGGL((attn_bf16_kernel<D, CQ, CK, FUSED, SPLIT>),
                       dim3(sched ? 8 * cap : 8 * ((P.nqc + 7) / 8) * P.BH),
                       dim3(64 * attn_waves<D, CQ, CK, SPLIT>()), 0, st, (const bf16*)qp,
                       (const bf16*)kp, (const bf16*)vp, count_k, lists, lens, P.nqc, P.nkc, k,
                       scale * kLog2e, (bf16*)op, lse, total, (const int32_t*)sched, cap, fa);
  };
  if constexpr (CQ == 64) {
    if (attn_use_split<D, CQ, CK>(k))
      launch(std::true_type{});
    else
      launch(std::false_type{});
  } else {
    launch(std::false_type{});
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const Prob& P, const void* qp, const void* kp, const void* vp,
                       const int32_t* count_k, const int32_t* lists, const int32_t* lens, int k,
                       float scale, void* op, float* lse, int32_t* sched, hipStream_t st) {
  if (P.dtype == CA_BF16) {
#define CA_ATTN_CASE(D, CQ, CK) \
  if (P.d == D && P.cq == CQ && P.ck == CK) \
    return run_bf16<D, CQ, CK>(P, qp, kp, vp, count_k, lists, lens, k, scale, op, lse, sched, st);
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
  const int threads = 256;  // (cq rounded up to 64) x key parts
  if (P.d <= 32) {
    hipLaunchKernelGGL(attn_f32_kernel<32>, grid, dim3(threads), 0, st, (const float*)qp,
                       (const float*)kp, (const float*)vp, count_k, lists, lens, P.nqc, P.nkc,
                       P.cq, P.ck, P.d, k, scale, (float*)op, lse);
  } else if (P.d <= 64) {
    hipLaunchKernelGGL(attn_f32_kernel<64>, grid, dim3(threads), 0, st, (const float*)qp,
                       (const float*)kp, (const float*)vp, count_k, lists, lens, P.nqc, P.nkc,
                       P.cq, P.ck, P.d, k, scale, (float*)op, lse);
  } else {
    hipLaunchKernelGGL(attn_f32_kernel<128>, grid, dim3(threads), 0, st, (const float*)qp,
                       (const float*)kp, (const float*)vp, count_k, lists, lens, P.nqc, P.nkc,
                       P.cq, P.ck, P.d, k, scale, (float*)op, lse);
  }
  return hipGetLastError();
}

hipError_t launch_attn_fused(const Prob& P, const void* qp, const void* kp, const void* vp,
                             const int32_t* count_k, const int32_t* lists, const int32_t* lens,
                             int k, float scale, const char* tiles, const int32_t* perm_q,
                             void* out, float* lse_out, int32_t* sched, hipStream_t st) {
  if (P.dtype != CA_BF16 || P.nkc > kMaskWords * 32) return hipErrorInvalidValue;
  const FusedArgs fa{tiles, (P.nkc + kCompTile - 1) / kCompTile, perm_q, (bf16*)out, lse_out,
                     P.nq, P.lo};
#define CA_ATTN_CASE(D, CQ, CK) \
  if (P.d == D && P.cq == CQ && P.ck == CK) \
    return run_bf16<D, CQ, CK, true>(P, qp, kp, vp, count_k, lists, lens, k, scale, nullptr, \
                                     nullptr, sched, st, fa);
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

}  // namespace ca
