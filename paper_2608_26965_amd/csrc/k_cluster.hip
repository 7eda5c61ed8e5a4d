// Clustering (paper: Method, Clustering): split spaces (Transforms), the
// diagonalized recursive split, and the permuted copies plus centroids.
//
// Pipeline per head, both sides batched in every launch:
//   moments      X^T X and column sums (fp32 partials, fp64 reduction)
//   eigh         Householder tridiagonal reduction, Sturm bisection and
//                inverse iteration on d x d matrices, one workgroup each
//   transforms   metric roots, the key-side covariance in the query metric,
//                the normalised query representation and its covariance
//   project      Y = X T (queries additionally scaled by 1/|q S_k|)
//   split        levels with nodes larger than the tail size: multi-block
//                radix select (11/11/10-bit digits) + stable partition;
//                remaining levels: one workgroup per node, in LDS
//   gather       permuted Q/K/V, centroids of the original vectors, counts
//
// The split is exact integer work on order-preserving images of the fp32
// coordinates; the only floating-point decision, the highest-variance
// coordinate of a node's subsample, is taken in fp64 with a fixed operation
// order and no contraction, so it is reproducible bit for bit.
#include <math.h>

#include <type_traits>

#include "attn_tile.h"
#include "common.h"

namespace ca {

namespace {

// ---------------------------------------------------------------------------
// Parameters of the two sides (0 = queries, 1 = keys)
// ---------------------------------------------------------------------------

struct Side {
  const void* x;    // input tensor (strides lx)
  Lay lx;
  float* y;         // split coordinates [BH][n][d]
  float* ycol;      // the first kColCopy of them, [BH][kColCopy][n] (or NULL)
  int32_t* perm;    // [BH][n]
  int32_t* cid;     // [BH][n] (may be null)
  int32_t* count;   // [BH][nc]
  float* cent;      // [BH][nc][d]
  void* xp;         // permuted copy [BH][npad][d]
  int n, c, nc, npad, levels, big, tail;
};

struct Ctx {
  Side s[2];
  const void* v;    // values (may be null)
  float* cent_v;
  void* vp;         // value tiles [BH][nkc][d][ck]
  Lay lv;           // strides of the values
  int BH, H, d, dtype, xf, nmax, nblk, mom_rows, proj_rows;
  float* mats;      // [BH][kMats][d][d]
  float* vecs;      // [BH][kVecs][d]
  float* inv_q;     // [BH][nq]
  float* mom_part;  // [2][BH][nblk][d*d + d]
  float* qn_part;   // [BH][nblk][d*d + d]
  bf16* wops;       // [BH][3][2][d][d] transposed hi/lo bf16 operands
  int32_t* idx0;
  int32_t* idx1;
  uint32_t* keys;
  int32_t* node_state;
  uint32_t* hist;
  int32_t* chunk_cnt;
  int max_nodes, hist_slots;
  int split;        // ca_split
  float* dirs;      // [2 levels][2][BH][max_nodes][d] split directions (basic splitting)
};

// Matrix slots
enum { M_A0 = 0, M_CK = 1, M_E0 = 2, M_EK = 3, M_C2 = 4, M_C3 = 5, M_TK = 6, M_TQ = 7 };
// Operand slots (MFMA A operands W^T, split in bf16 hi + lo)
enum { O_FK = 0, O_TK = 1, O_TQ = 2 };
// Vector slots
enum { V_L0 = 0, V_LK = 1, V_MUQ = 2, V_MUK = 3, V_L2 = 4, V_L3 = 5, V_MUR = 6, V_KQ = 7 };

__device__ __forceinline__ float* mat(const Ctx& C, int bh, int slot) {
  return C.mats + ((size_t)bh * kMats + slot) * C.d * C.d;
}
__device__ __forceinline__ bf16* wop(const Ctx& C, int bh, int slot) {
  return C.wops + ((size_t)bh * 3 + slot) * 2 * C.d * C.d;
}
__device__ __forceinline__ float* vec(const Ctx& C, int bh, int slot) {
  return C.vecs + ((size_t)bh * kVecs + slot) * C.d;
}

__device__ __forceinline__ float load_x(const void* x, int bh, int i, const Lay& L, int t,
                                        int dtype) {
  return load_elem(x, row_off(bh, i, L) + t, dtype);
}

// ---------------------------------------------------------------------------
// Second moments: part[pid][blk] = (sum_rows x x^T, sum_rows x) over a row block
// ---------------------------------------------------------------------------

constexpr int kStage = 32;  // rows staged in LDS at a time
constexpr int kDP = kMaxD + 4;

// Accumulates sum_r a_r b_r^T for the rows staged in A/B into per-thread 4x4
// blocks (up to 4 blocks per thread: d <= 128).
__device__ __forceinline__ void acc_outer(float (*A)[kDP], float (*B)[kDP], int rows, int d4,
                                          float acc[4][16]) {
  const int nb = d4 * d4;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int blk = threadIdx.x + 256 * q;
    if (blk >= nb) break;
    const int bi = blk / d4, bj = blk % d4;
    for (int r = 0; r < rows; ++r) {
      const float4 a = *(const float4*)&A[r][4 * bi];
      const float4 b = *(const float4*)&B[r][4 * bj];
      const float av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[q][4 * i + j] = __builtin_fmaf(av[i], bv[j], acc[q][4 * i + j]);
    }
  }
}

__device__ __forceinline__ void write_outer(float* out, int d, int d4, float acc[4][16]) {
  const int nb = d4 * d4;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int blk = threadIdx.x + 256 * q;
    if (blk >= nb) break;
    const int bi = blk / d4, bj = blk % d4;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 4 * bi + i, c = 4 * bj + j;
        if (r < d && c < d) out[r * d + c] = acc[q][4 * i + j];
      }
  }
}

__global__ __launch_bounds__(256) void moments_partial_kernel(Ctx C) {
  __shared__ __attribute__((aligned(16))) float X[kStage][kDP];
  const int pid = blockIdx.y, side = pid / C.BH, bh = pid % C.BH, blk = blockIdx.x;
  const Side& S = C.s[side];
  const int d = C.d, d4 = (d + 3) / 4;
  const int r0 = blk * C.mom_rows, r1 = min(S.n, r0 + C.mom_rows);
  float acc[4][16];
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[q][e] = 0.f;
  float csum = 0.f;
  for (int rs = r0; rs < r1; rs += kStage) {
    const int rows = min(kStage, r1 - rs);
    __syncthreads();
    for (int e = threadIdx.x; e < kStage * 4 * d4; e += 256) {
      const int r = e / (4 * d4), t = e % (4 * d4);
      X[r][t] = (r < rows && t < d)
                    ? load_x(S.x, bh, rs + r, S.lx, t, C.dtype)
                    : 0.f;
    }
    __syncthreads();
    acc_outer(X, X, rows, d4, acc);
    if (threadIdx.x < d)
      for (int r = 0; r < rows; ++r) csum += X[r][threadIdx.x];
  }
  float* out = C.mom_part + ((size_t)pid * C.nblk + blk) * (d * d + d);
  write_outer(out, d, d4, acc);
  if (threadIdx.x < d) out[d * d + threadIdx.x] = csum;
}

// Sum of nb partials p[0], p[stride], ... in fp64: eight independent running
// sums (so the loads overlap), combined in a fixed order (deterministic).
__device__ __forceinline__ double sum_partials(const float* p, size_t stride, int nb) {
  double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  int b = 0;
  for (; b + 8 <= nb; b += 8) {
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[u] += (double)p[(size_t)(b + u) * stride];
  }
  for (; b < nb; ++b) acc[b & 7] += (double)p[(size_t)b * stride];
  return ((acc[0] + acc[1]) + (acc[2] + acc[3])) + ((acc[4] + acc[5]) + (acc[6] + acc[7]));
}

// Reduces the moment partials in fp64, one element per thread, and writes
// the matrices the eigensolver starts from:
//   queries: metric -> Q^T Q / n;  pca -> centred covariance of Q
//   keys:    centred covariance of K (both modes)
// plus the means. Grid: (element blocks, BH, side).
__global__ __launch_bounds__(256) void moments_finish_kernel(Ctx C) {
  const int side = blockIdx.z, bh = blockIdx.y, d = C.d;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= d * d + d) return;
  const int pid = side * C.BH + bh;
  const size_t stride = (size_t)d * d + d;
  const float* part = C.mom_part + (size_t)pid * C.nblk * stride;
  const double n = (double)C.s[side].n;
  if (e >= d * d) {
    const int t = e - d * d;
    vec(C, bh, side == 0 ? V_MUQ : V_MUK)[t] = (float)(sum_partials(part + e, stride, C.nblk) / n);
    return;
  }
  const bool centred = side == 1 || C.xf == CA_XF_PCA;
  const int i = e / d, j = e % d;
  double v = sum_partials(part + e, stride, C.nblk) / n;
  if (centred) {
    const double mi = sum_partials(part + d * d + i, stride, C.nblk) / n;
    const double mj = sum_partials(part + d * d + j, stride, C.nblk) / n;
    v -= mi * mj;
  }
  mat(C, bh, side == 0 ? M_A0 : M_CK)[e] = (float)v;
}

// ---------------------------------------------------------------------------
// Symmetric eigenproblems of the transforms (the algorithm is described at
// eigh_kernel). Output: eigenvalues in descending order and the matching
// eigenvectors as columns.
// ---------------------------------------------------------------------------

// One eigenproblem: A = B, A = B - m m^T, or A = S^T B S (- u u^T with
// u = S^T m); the eigenvectors are oriented so that o . U[:, j] >= 0 with
// o = u (when u is formed) or a given vector, and the split projection
// T = F U (or U) is written in fp32 and, for bf16 inputs, as the transposed
// hi/lo bf16 MFMA operand.
struct EighJob {
  int b, s, m;     // matrix B, factor S (-1: none), vector m (-1: none)
  int rank1;       // subtract u u^T
  int u_out;       // vector slot for u (-1: none)
  int orient;      // orientation vector slot, used when u is not formed
  int vecs, vals;  // oriented eigenvectors (columns, descending) and eigenvalues
  int t_f;         // factor F of the projection T = F U (-1: T = U)
  int t_out, wop_out;
};
struct EighJobs {
  EighJob j[2];
};

// Symmetric eigensolver, one workgroup of kEighM * DM threads per d x d
// problem (d <= DM):
//  1. Householder reduction to a tridiagonal matrix T = Q^T A Q (A fp32 in
//     LDS; column norms and reflector scales in fp64). Every wavefront builds
//     reflector k from column k itself, so the pass over the trailing block,
//     which applies reflector k-1 (the symmetric rank-two update) and forms
//     p = A v_k in the same sweep, needs one barrier a step.
//  2. Off-diagonal entries below 2^-24 of the norm are set to zero, so T
//     splits into unreduced blocks (distinct eigenvalues, eigenvectors with
//     disjoint supports). Eigenvalues by bisection on Sturm counts in fp64:
//     sign changes of the leading minors (division free, rescaled every
//     eight steps), kEighM points per eigenvalue and round.
//  3. Eigenvectors of T by two steps of inverse iteration (an LDL^T
//     factorisation of T - lambda I in fp64) from pseudo-random starts;
//     eigenvalues closer than 1e-8 of the norm form clusters whose vectors
//     are re-orthogonalised (modified Gram-Schmidt) after each step.
//  4. Back-transformation by the reflectors: V = Q Z.
// (Golub and Van Loan, Matrix Computations: the Householder tridiagonal
// reduction, Sturm sequence bisection and inverse iteration.)
constexpr int kEighM = 4;
template <int DM>
constexpr int eigh_threads() {
  return kEighM * DM;
}
// Row stride of the LDS matrices (float4-aligned rows)
__host__ __device__ constexpr int eigh_stride(int dm) { return dm + 4; }
__host__ __device__ constexpr size_t eigh_lds_bytes(int dm) {
  return 2 * (size_t)dm * eigh_stride(dm) * sizeof(float);
}
// Bisection rounds: (kEighM + 1)^-17 of the width 2 is 1.5e-12 of the norm,
// far inside the cluster tolerance, so two inverse-iteration steps converge.
constexpr int kBisectRounds = 17;
constexpr double kDeflate = 0x1p-24;  // relative size of a negligible off-diagonal
constexpr double kClusterTol = 1e-8;  // relative gap below which vectors are re-orthogonalised
constexpr double kPivMin = 0x1p-50;   // smallest pivot magnitude of the LDL^T factorisation
constexpr double kStore = 0x1p-64;    // scale of the intermediate vectors kept in fp32

__device__ __forceinline__ void wave_lds_order() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Cross-lane sums through DPP (no LDS round trip). dpp_add: x + x of lane
// (CTRL); lanes outside the row mask add 0.
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ float dpp_add(float x) {
  return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, ROWS, 0xF, false));
}
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ double dpp_add(double x) {
  const long long b = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)b, CTRL, ROWS, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(b >> 32), CTRL, ROWS, 0xF, false);
  return x + __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}
// Sum over the 4 lanes of a quad (every lane of the quad gets it)
template <typename F>
__device__ __forceinline__ F quad_sum(F x) {
  x = dpp_add<0xB1>(x);  // quad_perm [1, 0, 3, 2]
  return dpp_add<0x4E>(x);  // quad_perm [2, 3, 0, 1]
}
// Sum over the wavefront, returned to every lane (a uniform value)
__device__ __forceinline__ float wave_sum(float x) {
  x = quad_sum(x);
  x = dpp_add<0x141>(x);        // row_half_mirror: 8 lanes
  x = dpp_add<0x140>(x);        // row_mirror: 16 lanes
  x = dpp_add<0x142, 0xA>(x);   // row_bcast15 into rows 1, 3
  x = dpp_add<0x143, 0xC>(x);   // row_bcast31 into rows 2, 3: lane 63 holds the sum
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}
__device__ __forceinline__ double wave_sum(double x) {
  x = quad_sum(x);
  x = dpp_add<0x141>(x);
  x = dpp_add<0x140>(x);
  x = dpp_add<0x142, 0xA>(x);
  x = dpp_add<0x143, 0xC>(x);
  const long long b = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_readlane((int)b, 63), hi = __builtin_amdgcn_readlane((int)(b >> 32), 63);
  return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}
__device__ __forceinline__ float read_lane(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}
// 1 / x in fp64: the hardware reciprocal and two Newton steps
__device__ __forceinline__ double recip64(double x) {
  double r = __builtin_amdgcn_rcp(x);
  double e = fma(-x, r, 1.0);
  r = fma(r, e, r);
  e = fma(-x, r, 1.0);
  return fma(r, e, r);
}

// Number of eigenvalues below x of the block [s, t) of the scaled
// tridiagonal matrix, tq[i] = (diagonal i, squared off-diagonal i - 1): the
// sign changes of the sequence 1, p_s, ..., p_{t-1} of leading minors of
// T - x I (a zero minor counts as a change).
__device__ __forceinline__ int sturm_below(const double2* tq, int s, int t, double x) {
  // A minor that is exactly zero counts as positive: the next one then has
  // the opposite sign of the one before, so the pair adds exactly one change.
  double p2 = 1.0, p1 = tq[s].x - x;
  int cnt = p1 < 0.0;
  int i0 = s + 1;
  for (; i0 + 8 <= t; i0 += 8) {
    double2 q[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) q[u] = tq[i0 + u];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const double p = (q[u].x - x) * p1 - q[u].y * p2;
      cnt += (p < 0.0) != (p1 < 0.0);
      p2 = p1;
      p1 = p;
    }
    int ex;
    (void)frexp(fmax(fabs(p1), fabs(p2)), &ex);
    p1 = ldexp(p1, -ex);
    p2 = ldexp(p2, -ex);
  }
  for (; i0 < t; ++i0) {
    const double2 q = tq[i0];
    const double p = (q.x - x) * p1 - q.y * p2;
    cnt += (p < 0.0) != (p1 < 0.0);
    p2 = p1;
    p1 = p;
  }
  return cnt;
}

// Pseudo-random start of inverse iteration: +-[0.5, 1.5)
__device__ __forceinline__ float start_value(int g, int i) {
  uint32_t h = (uint32_t)(g * 0x9E3779B1u) ^ (uint32_t)(i * 0x85EBCA77u + 0x165667B1u);
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  h ^= h >> 12;
  h *= 0x297A2D39u;
  h ^= h >> 15;
  const float u = 0.5f + (float)(h & 0xFFFFu) * (1.f / 65536.f);
  return (h & 0x10000u) ? -u : u;
}

// 4x4 register blocks of a d x d product (d <= 128, NT threads: at most two
// blocks per thread): acc = op(X) op(Y), op(Z) = Z or Z^T, with X, Y in LDS
// at row stride ld (a multiple of 4, 16-byte aligned rows) and zeros up to a
// multiple of 4; the sum runs over 4 indices per float4 load.
struct MMAcc {
  float v[2][16];
};

template <int NT>
__device__ __forceinline__ void lds_mm(const float* X, bool tX, const float* Y, bool tY, int ld,
                                       int d, MMAcc& acc) {
  const int d4 = (d + 3) >> 2, nb = d4 * d4;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
#pragma unroll
    for (int e = 0; e < 16; ++e) acc.v[u][e] = 0.f;
    const int blk = threadIdx.x + NT * u;
    if (blk >= nb) continue;
    const int i0 = 4 * (blk / d4), j0 = 4 * (blk % d4);
    for (int t = 0; t < d; t += 4) {
      float x[4][4], y[4][4];  // x[a][s] = op(X)[i0 + a][t + s], y[s][b] = op(Y)[t + s][j0 + b]
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float4 xv = *reinterpret_cast<const float4*>(tX ? &X[(t + k) * ld + i0] : &X[(i0 + k) * ld + t]);
        const float4 yv = *reinterpret_cast<const float4*>(tY ? &Y[(j0 + k) * ld + t] : &Y[(t + k) * ld + j0]);
        const float xs[4] = {xv.x, xv.y, xv.z, xv.w}, ys[4] = {yv.x, yv.y, yv.z, yv.w};
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          if (tX) x[m][k] = xs[m]; else x[k][m] = xs[m];
          if (tY) y[m][k] = ys[m]; else y[k][m] = ys[m];
        }
      }
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int b = 0; b < 4; ++b)
            acc.v[u][4 * a + b] = __builtin_fmaf(x[a][s], y[s][b], acc.v[u][4 * a + b]);
    }
  }
}

// Writes acc to an LDS matrix (stride ld); entries outside d x d stay zero.
template <int NT>
__device__ __forceinline__ void lds_mm_store(const MMAcc& acc, float* Z, int ld, int d) {
  const int d4 = (d + 3) >> 2, nb = d4 * d4;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int blk = threadIdx.x + NT * u;
    if (blk >= nb) continue;
    const int i0 = 4 * (blk / d4), j0 = 4 * (blk % d4);
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b)
        Z[(i0 + a) * ld + j0 + b] = i0 + a < d && j0 + b < d ? acc.v[u][4 * a + b] : 0.f;
  }
}

template <int DM>
__global__ __launch_bounds__(eigh_threads<DM>()) void eigh_kernel(Ctx C, EighJobs J) {
  constexpr int NT = eigh_threads<DM>();
  static_assert((DM / 4) * (DM / 4) <= 2 * NT, "two 4x4 product blocks per thread");
  constexpr int EP = eigh_stride(DM);
  constexpr int NW = NT / 64;
  constexpr int CPL = DM / 64;           // rows (or columns) per lane in a wavefront sweep
  constexpr int NQ = DM / (4 * kEighM);  // float4 column groups per thread in a row pass
  constexpr int RW = DM / kEighM;        // rows per thread in the back-transformation
  static_assert(CPL >= 1 && NQ >= 1 && RW % 4 == 0, "matrix size");
  extern __shared__ __attribute__((aligned(16))) float esh[];
  float* A = esh;             // [DM][EP]; row k keeps reflector k once reduced
  float* Vt = esh + DM * EP;  // [DM][EP]: S during the prologue, then Z[g][r] (vector g)
  __shared__ __attribute__((aligned(16))) float vvs[2][NW][DM];  // reflectors, one copy per wave
  __shared__ __attribute__((aligned(16))) float pbuf[2][DM];     // p = A v of the last two steps
  __shared__ float kpart[2][NW];
  __shared__ float trid[2][DM];  // diagonal, off-diagonal of T
  __shared__ double2 tq[DM];     // scaled (diagonal i, squared off-diagonal i - 1)
  __shared__ double es[DM], lam64[DM];
  __shared__ int bs[DM], be[DM], inv[DM];
  __shared__ double sh_tn;
  __shared__ uint64_t sh_link[CPL];
  __shared__ float uvec[DM], ovec[DM], mvec[DM], lam[DM], sgn[DM];
  __shared__ int rnk[DM];
  const int bh = blockIdx.x, d = C.d, tid = threadIdx.x;
  const EighJob& jb = J.j[blockIdx.y];
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  // ---- prologue: the matrix to diagonalize
  {
    const float* Bg = mat(C, bh, jb.b);
    const float* Sg = jb.s >= 0 ? mat(C, bh, jb.s) : nullptr;
    for (int i = wv; i < DM; i += NW)
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int j = lane + 64 * cc;
        const bool in = i < d && j < d;
        A[i * EP + j] = in ? Bg[i * d + j] : 0.f;
        Vt[i * EP + j] = Sg ? (in ? Sg[i * d + j] : 0.f) : 0.f;  // S while it is needed
      }
    if (tid < DM) {
      ovec[tid] = 0.f;
      mvec[tid] = jb.m >= 0 && tid < d ? vec(C, bh, jb.m)[tid] : 0.f;
    }
    __syncthreads();
    if (jb.m >= 0) {
      // u = S^T m (or m)
      if (tid < d) {
        float u;
        if (Sg) {
          float u4[4] = {0.f, 0.f, 0.f, 0.f};
          for (int t = 0; t < d; t += 4)
#pragma unroll
            for (int e = 0; e < 4; ++e)
              u4[e] = __builtin_fmaf(Vt[(t + e) * EP + tid], mvec[t + e], u4[e]);
          u = (u4[0] + u4[1]) + (u4[2] + u4[3]);
        } else {
          u = mvec[tid];
        }
        uvec[tid] = u;
        ovec[tid] = u;
      }
    } else if (tid < d) {
      ovec[tid] = vec(C, bh, jb.orient)[tid];
    }
    if (Sg) {
      // A = S^T (B S)
      MMAcc acc;
      lds_mm<NT>(A, false, Vt, false, EP, d, acc);  // T1 = B S
      __syncthreads();
      lds_mm_store<NT>(acc, A, EP, d);
      __syncthreads();
      lds_mm<NT>(Vt, true, A, false, EP, d, acc);   // S^T T1
      __syncthreads();
      lds_mm_store<NT>(acc, A, EP, d);
    }
    __syncthreads();
    if (jb.rank1)
      for (int i = wv; i < d; i += NW)
#pragma unroll
        for (int cc = 0; cc < CPL; ++cc) {
          const int j = lane + 64 * cc;
          if (j < d) A[i * EP + j] -= uvec[i] * uvec[j];
        }
    if (jb.u_out >= 0 && tid < d) vec(C, bh, jb.u_out)[tid] = uvec[tid];
    __syncthreads();
  }
  // ---- 1. Householder reduction. Step k: reflector H_k = I - v v^T (|v|^2 = 2,
  // support k+1..d-1) from column k after the update by H_{k-1}; the row pass
  // applies H_{k-1} to the block [k+1, d)^2 and accumulates p = A v; with
  // w = p - (v^T p / 2) v, H A H = A - v w^T - w v^T.
  const int nref = d > 2 ? d - 2 : 0;
  {
    // Row pass layout: the 16 lanes of a DPP row share 4 rows (rs, rs + DM/4,
    // rs + DM/2, rs + 3 DM/4; rs = 4 * wave + lane / 16, so the live rows of
    // a step are spread over all wavefronts) and split their float4 column
    // groups (c16, c16 + 16, ...): the vectors are read once per group and
    // used for 4 rows, and the 16 lanes read an A row contiguously.
    constexpr int RPT = 4;               // rows per lane
    constexpr int NG = DM / 64;          // column groups per lane
    const int c16 = lane & 15, rs = 4 * wv + (lane >> 4);
    for (int k = 0; k < nref; ++k) {
      const int cur = k & 1, prv = cur ^ 1;
      float* vcur = vvs[cur][wv];
      const float* vprv = vvs[prv][wv];
      const float* pprv = pbuf[prv];
      float Kp = 0.f, vk = 0.f, wk = 0.f;
      if (k > 0) {
#pragma unroll
        for (int w = 0; w < NW; ++w) Kp += kpart[prv][w];
        Kp *= 0.5f;
        vk = vprv[k];
        wk = pprv[k] - Kp * vk;
      }
      // column k below the diagonal (every wavefront, one or two rows a lane)
      float x[CPL];
      double s2 = 0.0;
#pragma unroll
      for (int h = 0; h < CPL; ++h) {
        const int i = lane + 64 * h;
        float xi = 0.f;
        if (i > k && i < d) {
          xi = A[i * EP + k];
          if (k > 0) {
            const float vi = vprv[i], wi = pprv[i] - Kp * vi;
            xi -= vi * wk + wi * vk;
          }
        }
        x[h] = xi;
        s2 += (double)xi * (double)xi;
      }
      s2 = wave_sum(s2);
      const int i0 = k + 1;
      float x0 = x[0];
#pragma unroll
      for (int h = 1; h < CPL; ++h) x0 = (i0 >> 6) == h ? x[h] : x0;
      x0 = read_lane(x0, i0 & 63);
      // sigma = |x|, alpha = -sign(x0) sigma, scale 1 / sqrt(sigma (sigma + |x0|)):
      // hardware reciprocal square roots with one Newton step each
      double rs2 = __builtin_amdgcn_rsq(s2);
      rs2 = rs2 * fma(-0.5 * s2 * rs2, rs2, 1.5);
      const double sig = s2 > 0.0 ? s2 * rs2 : 0.0;
      const double alpha = x0 >= 0.f ? -sig : sig;
      const double hq = sig * (sig + fabs((double)x0));
      double scl = __builtin_amdgcn_rsq(hq);
      scl = s2 > 0.0 ? scl * fma(-0.5 * hq * scl, scl, 1.5) : 0.0;
#pragma unroll
      for (int h = 0; h < CPL; ++h) {
        const int i = lane + 64 * h;
        float v = 0.f;
        if (i > k && i < d) v = (float)(((double)x[h] - (i == i0 ? alpha : 0.0)) * scl);
        vcur[i] = v;
        if (wv == 0 && i > k && i < d) A[k * EP + i] = v;
      }
      if (wv == 0 && lane == 0) {
        trid[0][k] = A[k * EP + k] - (k > 0 ? 2.f * vk * wk : 0.f);
        trid[1][k] = (float)alpha;
      }
      wave_lds_order();
      // row pass over [k+1, d)^2
      float vr[RPT], wr[RPT], vc[RPT], acc[RPT];
      bool rl[RPT];
#pragma unroll
      for (int r = 0; r < RPT; ++r) {
        const int row = rs + r * (DM / RPT);
        rl[r] = row > k && row < d;
        vc[r] = vcur[row];
        vr[r] = k > 0 ? vprv[row] : 0.f;
        wr[r] = k > 0 ? pprv[row] - Kp * vr[r] : 0.f;
        acc[r] = 0.f;
      }
#pragma unroll
      for (int q = 0; q < NG; ++q) {
        const int j0 = 4 * (c16 + 16 * q);
        if (j0 + 3 <= k) continue;  // every column of the group is dead
        const float4 vn = *reinterpret_cast<const float4*>(&vcur[j0]);
        const float vnv[4] = {vn.x, vn.y, vn.z, vn.w};
        float wpv[4] = {0.f, 0.f, 0.f, 0.f}, vpv[4] = {0.f, 0.f, 0.f, 0.f};
        if (k > 0) {
          const float4 vp = *reinterpret_cast<const float4*>(&vprv[j0]);
          const float4 pp = *reinterpret_cast<const float4*>(&pprv[j0]);
          vpv[0] = vp.x; vpv[1] = vp.y; vpv[2] = vp.z; vpv[3] = vp.w;
          wpv[0] = pp.x - Kp * vp.x; wpv[1] = pp.y - Kp * vp.y;
          wpv[2] = pp.z - Kp * vp.z; wpv[3] = pp.w - Kp * vp.w;
        }
        bool ok[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) ok[e] = j0 + e > k && j0 + e < d;
#pragma unroll
        for (int r = 0; r < RPT; ++r) {
          if (!rl[r]) continue;
          const int row = rs + r * (DM / RPT);
          const float4 a = *reinterpret_cast<const float4*>(&A[row * EP + j0]);
          float av[4] = {a.x, a.y, a.z, a.w};
          if (k > 0) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float upd = av[e] - (vr[r] * wpv[e] + wr[r] * vpv[e]);
              av[e] = ok[e] ? upd : av[e];
            }
            *reinterpret_cast<float4*>(&A[row * EP + j0]) = make_float4(av[0], av[1], av[2], av[3]);
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[r] += ok[e] ? av[e] * vnv[e] : 0.f;
        }
      }
      // row sums over the 16 lanes of the DPP row
      float vp_part = 0.f;
#pragma unroll
      for (int r = 0; r < RPT; ++r) {
        float t = quad_sum(acc[r]);
        t = dpp_add<0x141>(t);  // row_half_mirror
        t = dpp_add<0x140>(t);  // row_mirror
        const int row = rs + r * (DM / RPT);
        if (c16 == 0) {
          pbuf[cur][row] = rl[r] ? t : 0.f;
          vp_part += rl[r] ? vc[r] * t : 0.f;
        }
      }
      vp_part = wave_sum(vp_part);
      if (lane == 0) kpart[cur][wv] = vp_part;
      __syncthreads();
    }
    // the last 2 x 2 block after the last reflector
    if (tid == 0) {
      if (d == 1) {
        trid[0][0] = A[0];
      } else if (d >= 2) {
        const int i = d - 2, j = d - 1;
        float vi = 0.f, wi = 0.f, vj = 0.f, wj = 0.f;
        if (nref > 0) {
          const int l = (nref - 1) & 1;
          float Kp = 0.f;
          for (int w = 0; w < NW; ++w) Kp += kpart[l][w];
          Kp *= 0.5f;
          vi = vvs[l][0][i];
          vj = vvs[l][0][j];
          wi = pbuf[l][i] - Kp * vi;
          wj = pbuf[l][j] - Kp * vj;
        }
        trid[0][i] = A[i * EP + i] - 2.f * vi * wi;
        trid[0][j] = A[j * EP + j] - 2.f * vj * wj;
        trid[1][i] = A[j * EP + i] - (vj * wi + wj * vi);
      }
    }
    __syncthreads();
    // row k < nref holds reflector k in columns k+1..d-1; clear the rest
    for (int idx = tid; idx < DM * DM; idx += NT) {
      const int k = idx / DM, j = idx % DM;
      if (k < nref && j <= k) A[k * EP + j] = 0.f;
    }
    __syncthreads();
  }
  // ---- 2. scaling, deflation, blocks (wavefront 0), then bisection
  if (wv == 0) {
    double tn = 0.0;
    double dv[CPL], ev[CPL];
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      const int i = lane + 64 * h;
      dv[h] = i < d ? (double)trid[0][i] : 0.0;
      ev[h] = i + 1 < d ? (double)trid[1][i] : 0.0;
      const double el = i >= 1 && i < d ? fabs((double)trid[1][i - 1]) : 0.0;
      tn = fmax(tn, fabs(dv[h]) + fabs(ev[h]) + el);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) tn = fmax(tn, __shfl_xor(tn, o, 64));
    const double inv_tn = tn > 0.0 ? 1.0 / tn : 0.0;
    uint64_t brk[CPL];
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      const int i = lane + 64 * h;
      double e = ev[h] * inv_tn;
      if (fabs(e) <= kDeflate) e = 0.0;
      es[i] = e;
      // a block ends after i when i is the last index or T decouples there
      brk[h] = __ballot(i < d && (i == d - 1 || e == 0.0));
    }
    wave_lds_order();
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      const int i = lane + 64 * h;
      const double em = i >= 1 ? es[i - 1] : 0.0;
      tq[i] = make_double2(dv[h] * inv_tn, em * em);
      // start: one past the last break before i; end: one past the first break at or after i
      int st = 0, en = d;
#pragma unroll
      for (int g = CPL - 1; g >= 0; --g) {
        if (g > h) continue;
        const uint64_t m = g == h ? (lane == 0 ? 0ull : (brk[g] & ((~0ull) >> (64 - lane)))) : brk[g];
        if (m && st == 0) st = 64 * g + 63 - __builtin_clzll(m) + 1;
      }
#pragma unroll
      for (int g = 0; g < CPL; ++g) {
        if (g < h) continue;
        const uint64_t m = g == h ? (brk[g] & ((~0ull) << lane)) : brk[g];
        if (m && en == d) en = 64 * g + __builtin_ctzll(m) + 1;
      }
      bs[i] = i < d ? st : 0;
      be[i] = i < d ? en : 1;
    }
    if (lane == 0) sh_tn = tn;
  }
  __syncthreads();
  const double tn = sh_tn;
  {
    const int g = tid / kEighM, q = tid % kEighM;
    const bool live = g < d && tn > 0.0;
    const int s = live ? bs[g] : 0, t = live ? be[g] : 1, j = g - s;
    double lo = -1.0 - 0x1p-40, hi = 1.0 + 0x1p-40;
    for (int round = 0; round < kBisectRounds; ++round) {
      const double step = (hi - lo) / (double)(kEighM + 1);
      const int c = live ? sturm_below(tq, s, t, lo + step * (double)(q + 1)) : 0;
      // counts of the quad's four points (quad_perm broadcasts)
      const int below = (__builtin_amdgcn_update_dpp(0, c, 0x00, 0xF, 0xF, false) <= j) +
                        (__builtin_amdgcn_update_dpp(0, c, 0x55, 0xF, 0xF, false) <= j) +
                        (__builtin_amdgcn_update_dpp(0, c, 0xAA, 0xF, 0xF, false) <= j) +
                        (__builtin_amdgcn_update_dpp(0, c, 0xFF, 0xF, 0xF, false) <= j);
      const double nlo = below > 0 ? lo + step * (double)below : lo;
      const double nhi = below < kEighM ? lo + step * (double)(below + 1) : hi;
      lo = nlo;
      hi = nhi;
    }
    if (q == 0) lam64[g] = live ? 0.5 * (lo + hi) : 0.0;
  }
  __syncthreads();
  // ---- 3. eigenvectors of T: clusters (wavefront 0), start vectors (all)
  if (wv == 0) {
#pragma unroll
    for (int h = 0; h < CPL; ++h) {
      const int g = lane + 64 * h;
      const bool link = g >= 1 && g < d && bs[g] == bs[g - 1] &&
                        lam64[g] - lam64[g - 1] < kClusterTol;
      const uint64_t m = __ballot(link);
      if (lane == 0) sh_link[h] = m;
    }
  }
  for (int idx = tid; idx < DM * DM; idx += NT) {
    const int g = idx / DM, i = idx % DM;
    const bool in = g < d && i >= bs[g] && i < be[g];
    Vt[g * EP + i] = in ? (tn > 0.0 ? start_value(g, i) : (i == g ? 1.f : 0.f)) : 0.f;
  }
  __syncthreads();
  if (tn > 0.0) {
    // vector g on the kEighM lanes of a quad, SEG consecutive entries each.
    // No per-entry masks: the off-diagonal entry at each end of g's block is
    // zero, so both recurrences restart there, and the start vector is zero
    // outside the block, so those entries stay exactly zero.
    constexpr int SEG = DM / kEighM;
    const int g = tid / kEighM, part = tid % kEighM;
    const bool live = g < d;
    const double sigma = live ? lam64[g] : 0.0;
    float* z = Vt + (size_t)(live ? g : 0) * EP + SEG * part;
    const double2* tqs = tq + SEG * part;
    const double* ess = es + SEG * part;
    for (int it = 0; it < 2; ++it) {
      double r[SEG];  // 1 / pivot of this lane's entries
      // forward: T - sigma I = L D L^T, y = L^{-1} b (kept in z, scaled);
      // the quad's lanes take their segments in turn, passing (l, y) on
      double lprev = 0.0, yprev = 0.0;
#pragma unroll
      for (int h = 0; h < kEighM; ++h) {
        if (h > 0) {
          const int src = (lane & ~(kEighM - 1)) + h - 1;
          lprev = __shfl(lprev, src, 64);
          yprev = __shfl(yprev, src, 64);
        }
        if (live && part == h) {
#pragma unroll
          for (int u = 0; u < SEG; ++u) {
            if ((u & 7) == 0) asm volatile("" ::: "memory");
            const double a = tqs[u].x - sigma;
            const double em = u > 0 ? ess[u - 1] : (h > 0 ? es[SEG * h - 1] : 0.0);
            double dl = fma(-lprev, em, a);
            const double y = fma(-lprev, yprev, (double)z[u]);
            dl = fabs(dl) < kPivMin ? (dl < 0.0 ? -kPivMin : kPivMin) : dl;
            r[u] = recip64(dl);
            lprev = ess[u] * r[u];
            yprev = y;
            z[u] = (float)(y * kStore);
          }
        }
      }
      // backward: x = D^{-1} y - L^T x, kept in z (scaled); max |x|
      double xn = 0.0, mx = 0.0;
#pragma unroll
      for (int h = kEighM - 1; h >= 0; --h) {
        if (h < kEighM - 1) xn = __shfl(xn, (lane & ~(kEighM - 1)) + h + 1, 64);
        if (live && part == h) {
#pragma unroll
          for (int u = SEG - 1; u >= 0; --u) {
            if ((u & 7) == 7) asm volatile("" ::: "memory");
            const double xv = r[u] * fma(-ess[u], xn, (double)z[u] * (1.0 / kStore));
            xn = xv;
            mx = fmax(mx, fabs(xv));
            z[u] = (float)(xv * kStore);
          }
        }
      }
      mx = fmax(mx, __shfl_xor(mx, 1, 64));
      mx = fmax(mx, __shfl_xor(mx, 2, 64));
      // normalise
      const double sc = mx > 0.0 ? 1.0 / (mx * kStore) : 0.0;
      double ss = 0.0;
      if (live)
#pragma unroll
        for (int u = 0; u < SEG; ++u) {
          const double v = (double)z[u] * sc;
          ss += v * v;
        }
      ss = quad_sum(ss);
      const double nrm = ss > 0.0 ? sc / sqrt(ss) : 0.0;
      if (live)
#pragma unroll
        for (int u = 0; u < SEG; ++u) z[u] = (float)((double)z[u] * nrm);
      __syncthreads();
      // clusters: modified Gram-Schmidt in slot order (wavefront 0)
      if (wv == 0) {
        for (int h = 0; h < CPL; ++h) {
          uint64_t m = sh_link[h];
          while (m) {
            const int gj = 64 * h + __builtin_ctzll(m);
            m &= m - 1;
            int g0 = gj;
            while (g0 > 0 && ((sh_link[g0 >> 6] >> (g0 & 63)) & 1)) --g0;
            float zj[CPL];
#pragma unroll
            for (int c = 0; c < CPL; ++c) zj[c] = Vt[gj * EP + lane + 64 * c];
            for (int gi = g0; gi < gj; ++gi) {
              float dot = 0.f;
#pragma unroll
              for (int c = 0; c < CPL; ++c) dot += Vt[gi * EP + lane + 64 * c] * zj[c];
              dot = wave_sum(dot);
#pragma unroll
              for (int c = 0; c < CPL; ++c) zj[c] -= dot * Vt[gi * EP + lane + 64 * c];
            }
            float nn = 0.f;
#pragma unroll
            for (int c = 0; c < CPL; ++c) nn += zj[c] * zj[c];
            nn = wave_sum(nn);
            const float rn = nn > 0.f ? 1.f / sqrtf(nn) : 0.f;
#pragma unroll
            for (int c = 0; c < CPL; ++c) Vt[gj * EP + lane + 64 * c] = zj[c] * rn;
            wave_lds_order();
          }
        }
      }
      __syncthreads();
    }
  }
  // ---- 4. back-transformation: vector g (rows split over kEighM threads)
  {
    const int g = tid / kEighM, c = tid % kEighM;
    float zr[RW];
#pragma unroll
    for (int u = 0; u < RW; u += 4) {
      const float4 v4 = *reinterpret_cast<const float4*>(&Vt[g * EP + c * RW + u]);
      zr[u] = v4.x;
      zr[u + 1] = v4.y;
      zr[u + 2] = v4.z;
      zr[u + 3] = v4.w;
    }
    for (int k = nref - 1; k >= 0; --k) {
      float vr[RW];
      float dp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < RW; u += 4) {
        const float4 v4 = *reinterpret_cast<const float4*>(&A[k * EP + c * RW + u]);
        vr[u] = v4.x;
        vr[u + 1] = v4.y;
        vr[u + 2] = v4.z;
        vr[u + 3] = v4.w;
      }
#pragma unroll
      for (int u = 0; u < RW; ++u) dp[u & 3] = __builtin_fmaf(vr[u], zr[u], dp[u & 3]);
      const float dot = quad_sum((dp[0] + dp[1]) + (dp[2] + dp[3]));
#pragma unroll
      for (int u = 0; u < RW; ++u) zr[u] = __builtin_fmaf(-dot, vr[u], zr[u]);
    }
#pragma unroll
    for (int u = 0; u < RW; u += 4)
      *reinterpret_cast<float4*>(&Vt[g * EP + c * RW + u]) =
          make_float4(zr[u], zr[u + 1], zr[u + 2], zr[u + 3]);
  }
  __syncthreads();
  float* Ac = A;
  const float* Vc = Vt;
  // ---- epilogue: eigenvalues, ranks (descending, ties by index), orientation
  if (tid < d) {
    lam[tid] = (float)(lam64[tid] * tn);
    float o4[4] = {0.f, 0.f, 0.f, 0.f};
    for (int t = 0; t < d; t += 4)
#pragma unroll
      for (int e = 0; e < 4; ++e) o4[e] = __builtin_fmaf(ovec[t + e], Vc[tid * EP + t + e], o4[e]);
    const float o = (o4[0] + o4[1]) + (o4[2] + o4[3]);
    sgn[tid] = o < 0.f ? -1.f : 1.f;
  }
  __syncthreads();
  if (tid < d) {
    const float li = lam[tid];
    int r = 0;
    for (int j = 0; j < d; ++j) {
      const float lj = lam[j];
      r += (lj > li) || (lj == li && j < tid);
    }
    rnk[tid] = r;
    inv[r] = tid;
    vec(C, bh, jb.vals)[r] = li;
  }
  __syncthreads();
  float* U = mat(C, bh, jb.vecs);
  float* T = mat(C, bh, jb.t_out);
  bf16* W = jb.wop_out >= 0 ? wop(C, bh, jb.wop_out) : nullptr;
  // Eigenvector g becomes column rnk[g]: U[r][c] = sgn[g] Vc[g][r], g = inv[c]
  // (lanes over c: coalesced rows of U)
  for (int r = wv; r < d; r += NW)
#pragma unroll
    for (int cc = 0; cc < CPL; ++cc) {
      const int c = lane + 64 * cc;
      if (c < d) {
        const int g = inv[c];
        U[r * d + c] = sgn[g] * Vc[g * EP + r];
      }
    }
  // The projection T[r][c] = sgn[g] P[r][g] with P = F V (t_f) or V, and its
  // bf16 operand pair W[c][r] (hi) and W[d * d + c * d + r] (lo).
  const float* P = Vc;  // P[r][g] at Vc[g * EP + r] (V), or at Ac[r * EP + g] (F V)
  const bool fv = jb.t_f >= 0;
  if (fv) {
    // P = F V: F goes into the A region
    const float* Sg = mat(C, bh, jb.t_f);
    for (int i = wv; i < DM; i += NW)
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int j = lane + 64 * cc;
        Ac[i * EP + j] = i < d && j < d ? Sg[i * d + j] : 0.f;
      }
    __syncthreads();
    MMAcc acc;
    lds_mm<NT>(Ac, false, Vc, true, EP, d, acc);
    __syncthreads();
    lds_mm_store<NT>(acc, Ac, EP, d);
    __syncthreads();
    P = Ac;
  }
  for (int r = wv; r < d; r += NW)
#pragma unroll
    for (int cc = 0; cc < CPL; ++cc) {
      const int c = lane + 64 * cc;
      if (c < d) {
        const int g = inv[c];
        T[r * d + c] = sgn[g] * (fv ? P[r * EP + g] : P[g * EP + r]);
      }
    }
  if (W)
    for (int c = wv; c < d; c += NW) {
      const int g = inv[c];
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int r = lane + 64 * cc;
        if (r < d) {
          const float v = sgn[g] * (fv ? P[r * EP + g] : P[g * EP + r]);
          const bf16 hi = (bf16)v;
          W[c * d + r] = hi;
          W[d * d + c * d + r] = (bf16)(v - (float)hi);
        }
      }
    }
}

// ---------------------------------------------------------------------------
// Metric roots: a factor F with F F^T = M. Any such factor gives the same
// split coordinates after the principal-axis step (F = E sqrt(L) R for an
// orthogonal R, which the principal axes absorb), so the root of each metric
// is taken as its Cholesky factor, in fp64; pivots below a relative threshold
// are treated as zero (positive semi-definite metrics; this equals clamping
// the eigenvalues at zero up to rounding).
// ---------------------------------------------------------------------------

constexpr int kCholThreads = 256;
constexpr int kCP = kMaxD + 1;

__global__ __launch_bounds__(kCholThreads) void cholesky_kernel(Ctx C, int in0, int out0, int in1,
                                                                 int out1, int pack1) {
  extern __shared__ __attribute__((aligned(16))) double csh[];  // [d][kCP]
  __shared__ double sh_tol;
  const int bh = blockIdx.x, job = blockIdx.y, d = C.d, tid = threadIdx.x;
  const int tr = tid >> 4, tc = tid & 15;  // 16 x 16 thread grid
  const float* M = mat(C, bh, job == 0 ? in0 : in1);
  float* F = mat(C, bh, job == 0 ? out0 : out1);
  const int pack = job == 1 ? pack1 : -1;
  double* A = csh;
  for (int i = tr; i < d; i += 16)
    for (int k = tc; k < d; k += 16) A[i * kCP + k] = (double)M[i * d + k];
  __syncthreads();
  if (tid < 64) {
    double mx = 0.0;
    for (int i = tid; i < d; i += 64) mx = fmax(mx, A[i * kCP + i]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o, 64));
    if (tid == 0) sh_tol = mx * 1e-12;
  }
  __syncthreads();
  const double tol = sh_tol;
  // Elimination on unscaled columns (the order of an L D L^T factorisation):
  // step j subtracts a_ij a_kj / a_jj from the trailing lower triangle (rows
  // i > j, columns j < k <= i) and leaves column j as it is, so a step reads
  // only column j and needs one barrier. A pivot at or below tol contributes
  // nothing and gives a zero column.
  for (int j = 0; j < d; ++j) {
    const double dj = A[j * kCP + j];  // the same LDS value in every thread
    const double inv = dj > tol ? 1.0 / dj : 0.0;
    for (int i = j + 1 + tr; i < d; i += 16) {
      const double lij = A[i * kCP + j] * inv;
      for (int k = j + 1 + tc; k <= i; k += 16) A[i * kCP + k] -= lij * A[k * kCP + j];
    }
    __syncthreads();
  }
  // Scale: l_jj = sqrt(a_jj), l_ij = a_ij / l_jj.
  __shared__ double piv[kMaxD], ipiv[kMaxD];
  if (tid < d) {
    const double dj = A[tid * kCP + tid];
    const double p = dj > tol ? sqrt(dj) : 0.0;
    piv[tid] = p;
    ipiv[tid] = p > 0.0 ? 1.0 / p : 0.0;
  }
  __syncthreads();
  for (int i = tr; i < d; i += 16)
    for (int k = tc; k <= i; k += 16) A[i * kCP + k] = k == i ? piv[k] : A[i * kCP + k] * ipiv[k];
  __syncthreads();
  for (int i = tr; i < d; i += 16)
    for (int k = tc; k < d; k += 16) F[i * d + k] = k <= i ? (float)A[i * kCP + k] : 0.f;
  if (pack >= 0) {
    // transposed hi/lo bf16 operand of the factor (the MFMA query pass)
    bf16* out = wop(C, bh, pack);
    for (int e = tid; e < d * d; e += kCholThreads) {
      const int i = e / d, k = e % d;  // out row i (output dim), column k (input dim)
      const float w = i <= k ? (float)A[k * kCP + i] : 0.f;
      const bf16 hi = (bf16)w;
      out[e] = hi;
      out[d * d + e] = (bf16)(w - (float)hi);
    }
  }
}

// Metric mode, queries: rho = q S_k, inv = 1/|rho| (0 if rho = 0), r = rho*inv;
// partial sums of r r^T and r per row block; inv is kept for the projection.
__global__ __launch_bounds__(256) void qnorm_partial_kernel(Ctx C) {
  extern __shared__ __attribute__((aligned(16))) float qsh[];
  float* Sk = qsh;                                        // [d][kDP]
  float (*X)[kDP] = (float(*)[kDP])(qsh + kMaxD * kDP);   // [kStage][kDP]
  float (*R)[kDP] = (float(*)[kDP])(qsh + (kMaxD + kStage) * kDP);
  __shared__ float invs[kStage];
  const int bh = blockIdx.y, blk = blockIdx.x, d = C.d, d4 = (d + 3) / 4;
  const Side& S = C.s[0];
  const float* Skg = mat(C, bh, M_EK);
  for (int e = threadIdx.x; e < d * 4 * d4; e += 256) {
    const int t = e / (4 * d4), j = e % (4 * d4);
    Sk[t * kDP + j] = j < d ? Skg[t * d + j] : 0.f;
  }
  const int r0 = blk * C.mom_rows, r1 = min(S.n, r0 + C.mom_rows);
  float acc[4][16];
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[q][e] = 0.f;
  float csum = 0.f;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int rs = r0; rs < r1; rs += kStage) {
    const int rows = min(kStage, r1 - rs);
    __syncthreads();
    for (int e = threadIdx.x; e < kStage * 4 * d4; e += 256) {
      const int r = e / (4 * d4), t = e % (4 * d4);
      X[r][t] = (r < rows && t < d) ? load_x(S.x, bh, rs + r, S.lx, t, C.dtype)
                                    : 0.f;
    }
    __syncthreads();
    // rho for the staged rows
    for (int e = threadIdx.x; e < kStage * d4; e += 256) {
      const int r = e / d4, j4 = e % d4;
      float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
      for (int t = 0; t < d; ++t) {
        const float xv = X[r][t];
        const float4 s4 = *(const float4*)&Sk[t * kDP + 4 * j4];
        a0 = __builtin_fmaf(xv, s4.x, a0);
        a1 = __builtin_fmaf(xv, s4.y, a1);
        a2 = __builtin_fmaf(xv, s4.z, a2);
        a3 = __builtin_fmaf(xv, s4.w, a3);
      }
      *(float4*)&R[r][4 * j4] = make_float4(a0, a1, a2, a3);
    }
    __syncthreads();
    // one wave per row: 1/|rho|
    for (int r = w; r < kStage; r += 4) {
      float s = 0.f;
      for (int t = lane; t < d; t += 64) s = __builtin_fmaf(R[r][t], R[r][t], s);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
      if (lane == 0) {
        const float inv = s > 0.f ? 1.f / sqrtf(s) : 0.f;
        invs[r] = inv;
        if (r < rows) C.inv_q[(size_t)bh * S.n + rs + r] = inv;
      }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < kStage * 4 * d4; e += 256) {
      const int r = e / (4 * d4), t = e % (4 * d4);
      R[r][t] = r < rows ? R[r][t] * invs[r] : 0.f;
    }
    __syncthreads();
    acc_outer(R, R, rows, d4, acc);
    if (threadIdx.x < d)
      for (int r = 0; r < rows; ++r) csum += R[r][threadIdx.x];
  }
  float* out = C.qn_part + ((size_t)bh * C.nblk + blk) * (d * d + d);
  write_outer(out, d, d4, acc);
  if (threadIdx.x < d) out[d * d + threadIdx.x] = csum;
}

// Means of the query-representation partials (fp64 reduction, one element
// per thread): M_C3 <- sum/n of the d x d part, V_MUR <- sum/n of the vector
// part. The partials hold either r r^T and r (then cov(r) = M_C3 - mu mu^T),
// or inv^2 x x^T and inv x (then cov(r) = S_k^T M_C3 S_k - u u^T with
// u = S_k^T V_MUR); the eigensolver's prologue forms cov(r).
__global__ __launch_bounds__(256) void qnorm_finish_kernel(Ctx C) {
  const int bh = blockIdx.y, d = C.d;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= d * d + d) return;
  const size_t stride = (size_t)d * d + d;
  const float* part = C.qn_part + (size_t)bh * C.nblk * stride;
  const double v = sum_partials(part + e, stride, C.nblk) / (double)C.s[0].n;
  if (e < d * d)
    mat(C, bh, M_C3)[e] = (float)v;
  else
    vec(C, bh, V_MUR)[e - d * d] = (float)v;
}

// ---------------------------------------------------------------------------
// Projection Y = X T (fp32), or Y = X for the raw-coordinate mode.
// ---------------------------------------------------------------------------

constexpr int kProjRows = 256;  // rows per projection block (at most)

// Pseudo-random split coordinate in [0, 1) of the random-cluster control:
// output number c (counting from 0) of splitmix64 (S. Vigna's generator,
// started at state 0), top 24 bits, so the value is exact in fp32.
__device__ __forceinline__ float random_coord(int bh, int side, int i, int j) {
  const uint64_t c = ((((uint64_t)bh * 2 + (uint64_t)side) << 22 | (uint64_t)i) << 7) | (uint64_t)j;
  uint64_t z = (c + 1ull) * 0x9e3779b97f4a7c15ull;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  z ^= z >> 31;
  return (float)(uint32_t)(z >> 40) * 0x1p-24f;
}

__global__ __launch_bounds__(256) void project_kernel(Ctx C) {
  extern __shared__ __attribute__((aligned(16))) float psh[];
  float* T = psh;                                        // [d][kDP]
  float (*X)[kDP] = (float(*)[kDP])(psh + kMaxD * kDP);  // [kStage][kDP]
  const int pid = blockIdx.y, side = pid / C.BH, bh = pid % C.BH;
  const Side& S = C.s[side];
  const int d = C.d, d4 = (d + 3) / 4;
  const int r0 = blockIdx.x * C.proj_rows, r1 = min(S.n, r0 + C.proj_rows);
  if (r0 >= r1) return;
  float* Y = S.y + (size_t)bh * S.n * d;
  if (C.xf == CA_XF_NONE) {
    for (int e = threadIdx.x; e < (r1 - r0) * d; e += 256) {
      const int r = r0 + e / d, t = e % d;
      Y[(size_t)r * d + t] = load_x(S.x, bh, r, S.lx, t, C.dtype);
    }
    return;
  }
  if (C.xf == CA_XF_RANDOM) {
    for (int e = threadIdx.x; e < (r1 - r0) * d; e += 256) {
      const int r = r0 + e / d, t = e % d;
      Y[(size_t)r * d + t] = random_coord(bh, side, r, t);
    }
    return;
  }
  const float* Tg = mat(C, bh, side == 0 ? M_TQ : M_TK);
  for (int e = threadIdx.x; e < d * 4 * d4; e += 256) {
    const int t = e / (4 * d4), j = e % (4 * d4);
    T[t * kDP + j] = j < d ? Tg[t * d + j] : 0.f;
  }
  const bool scale = side == 0 && C.xf == CA_XF_METRIC;
  for (int rs = r0; rs < r1; rs += kStage) {
    const int rows = min(kStage, r1 - rs);
    __syncthreads();
    for (int e = threadIdx.x; e < kStage * 4 * d4; e += 256) {
      const int r = e / (4 * d4), t = e % (4 * d4);
      X[r][t] = (r < rows && t < d) ? load_x(S.x, bh, rs + r, S.lx, t, C.dtype)
                                    : 0.f;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < rows * d4; e += 256) {
      const int r = e / d4, j4 = e % d4;
      float a[4] = {0.f, 0.f, 0.f, 0.f};
      for (int t = 0; t < d; ++t) {
        const float xv = X[r][t];
        const float4 t4 = *(const float4*)&T[t * kDP + 4 * j4];
        a[0] = __builtin_fmaf(xv, t4.x, a[0]);
        a[1] = __builtin_fmaf(xv, t4.y, a[1]);
        a[2] = __builtin_fmaf(xv, t4.z, a[2]);
        a[3] = __builtin_fmaf(xv, t4.w, a[3]);
      }
      const float sc = scale ? C.inv_q[(size_t)bh * S.n + rs + r] : 1.f;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (4 * j4 + j < d) Y[(size_t)(rs + r) * d + 4 * j4 + j] = a[j] * sc;
    }
  }
}

// ---------------------------------------------------------------------------
// MFMA versions of the dense passes (bf16 inputs, d in {64, 128}).
//
// A 32-token tile of X is held as MFMA operands: lane l owns token l % 32 and
// features 16 ks + 8 (l / 32) + [0, 8) for k-step ks, loaded with 16-byte
// reads straight from the rows. With X as the B operand and W^T as the A
// operand, (X W)^T comes out with one token per lane (column = token), so
// per-token scalings stay in the lane. For the second moments X^T X the tile
// is first transposed on the matrix core by multiplying with an identity
// operand (exact for bf16 data), which leaves one feature per lane.
// ---------------------------------------------------------------------------

template <int D>
__device__ __forceinline__ void load_xtile(const bf16* __restrict__ x, int bh, int tok0, int lim,
                                           const Lay& L, int l32, int h,
                                           bf16x8 (&xop)[D / 16]) {
  const int tok = tok0 + l32;
  if (tok < lim) {
    const bf16* row = x + row_off(bh, tok, L);
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) xop[ks] = *(const bf16x8*)(row + 16 * ks + 8 * h);
  } else {
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks)
#pragma unroll
      for (int u = 0; u < 8; ++u) xop[ks][u] = (bf16)0.f;
  }
}

// Identity operands: B[k][n] = 1 iff k == n for the two 16-row halves of a
// 32-wide feature tile.
__device__ __forceinline__ void ident_ops(int l32, int h, bf16x8 (&id)[2]) {
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int u = 0; u < 8; ++u) id[s][u] = (bf16)((l32 == 16 * s + 8 * h + u) ? 1.f : 0.f);
}

// xT[ft]: lane l holds feature 32 ft + l % 32 of tokens 8 (r/4) + 4 h + r % 4.
template <int D>
__device__ __forceinline__ void transpose_tile(const bf16x8 (&xop)[D / 16], const bf16x8 (&id)[2],
                                               f32x16 (&xT)[D / 32]) {
#pragma unroll
  for (int ft = 0; ft < D / 32; ++ft) {
#pragma unroll
    for (int r = 0; r < 16; ++r) xT[ft][r] = 0.f;
    xT[ft] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xop[2 * ft], id[0], xT[ft], 0, 0, 0);
    xT[ft] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xop[2 * ft + 1], id[1], xT[ft], 0, 0, 0);
  }
}

__device__ __forceinline__ bf16x8 pack_half(const f32x16& v, int s) {
  float t[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) t[j] = v[8 * s + j];
  return pack8(t);
}

// Stages the hi/lo W^T operands of one head into LDS (row = output dim,
// 2D-byte rows, chunk-swizzled).
template <int D>
__device__ __forceinline__ void stage_wops(const bf16* __restrict__ src, char* lds) {
  constexpr int ROWB = 2 * D, NCH = ROWB / 16;
  for (int c = threadIdx.x; c < 2 * D * NCH; c += 256) {
    const int m = c / (D * NCH), rem = c % (D * NCH);
    const int r = rem / NCH, lc = rem % NCH;
    *(uint4*)(lds + m * D * ROWB + swz_off<ROWB>(r, lc)) =
        *(const uint4*)(src + (size_t)m * D * D + r * D + lc * 8);
  }
}

// acc[ot] = (X W)^T tile ot (output dims 32 ot.., tokens = lanes) with W = hi + lo.
template <int D>
__device__ __forceinline__ void project_tile(const char* wl, const bf16x8 (&xop)[D / 16], int l32,
                                             int h, f32x16 (&acc)[D / 32]) {
  constexpr int ROWB = 2 * D;
#pragma unroll
  for (int ot = 0; ot < D / 32; ++ot) {
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[ot][r] = 0.f;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      const int off = swz_off<ROWB>(32 * ot + l32, 2 * ks + h);
      const bf16x8 ahi = *(const bf16x8*)(wl + off);
      const bf16x8 alo = *(const bf16x8*)(wl + D * ROWB + off);
      acc[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ahi, xop[ks], acc[ot], 0, 0, 0);
      acc[ot] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(alo, xop[ks], acc[ot], 0, 0, 0);
    }
  }
}

// Output tile ot of (X W)^T alone (dims 32 ot.., tokens = lanes).
template <int D>
__device__ __forceinline__ void project_tile1(const char* wl, const bf16x8 (&xop)[D / 16], int l32,
                                              int h, int ot, f32x16& acc) {
  constexpr int ROWB = 2 * D;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    const int off = swz_off<ROWB>(32 * ot + l32, 2 * ks + h);
    const bf16x8 ahi = *(const bf16x8*)(wl + off);
    const bf16x8 alo = *(const bf16x8*)(wl + D * ROWB + off);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ahi, xop[ks], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(alo, xop[ks], acc, 0, 0, 0);
  }
}

// Adds the symmetric Gram tiles (it <= jt) of one wave into red[d][d] (and
// the mirror), waves in a fixed order.
template <int D>
__device__ __forceinline__ void reduce_gram(float* red, const f32x16* g, int w, int l32, int h) {
  constexpr int FT = D / 32;
  for (int wv = 0; wv < 4; ++wv) {
    if (w == wv) {
      int t = 0;
#pragma unroll
      for (int it = 0; it < FT; ++it)
#pragma unroll
        for (int jt = it; jt < FT; ++jt, ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int i = 32 * it + 8 * (r >> 2) + 4 * h + (r & 3), j = 32 * jt + l32;
            const float v = g[t][r];
            red[i * D + j] = wv == 0 ? v : red[i * D + j] + v;
            if (it != jt) red[j * D + i] = wv == 0 ? v : red[j * D + i] + v;
          }
    }
    __syncthreads();
  }
}

template <int D>
__global__ __launch_bounds__(256) void moments_mfma_kernel(Ctx C) {
  constexpr int FT = D / 32, KS = D / 16, NT = FT * (FT + 1) / 2;
  __shared__ float red[D * D];
  __shared__ float csr[4][D];
  const int pid = blockIdx.y, side = pid / C.BH, bh = pid % C.BH, blk = blockIdx.x;
  const Side& S = C.s[side];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const int r0 = blk * C.mom_rows, r1 = min(S.n, r0 + C.mom_rows);
  bf16x8 id[2];
  ident_ops(l32, h, id);
  f32x16 g[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) g[t][r] = 0.f;
  float cs[FT];
#pragma unroll
  for (int ft = 0; ft < FT; ++ft) cs[ft] = 0.f;
  for (int tok0 = r0 + 32 * w; tok0 < r1; tok0 += 128) {
    bf16x8 xop[KS];
    load_xtile<D>((const bf16*)S.x, bh, tok0, r1, S.lx, l32, h, xop);
    f32x16 xT[FT];
    transpose_tile<D>(xop, id, xT);
#pragma unroll
    for (int ft = 0; ft < FT; ++ft)
#pragma unroll
      for (int r = 0; r < 16; ++r) cs[ft] += xT[ft][r];
    int t = 0;
#pragma unroll
    for (int it = 0; it < FT; ++it)
#pragma unroll
      for (int jt = it; jt < FT; ++jt, ++t)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
          g[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pack_half(xT[it], s2),
                                                          pack_half(xT[jt], s2), g[t], 0, 0, 0);
  }
  reduce_gram<D>(red, g, w, l32, h);
#pragma unroll
  for (int ft = 0; ft < FT; ++ft) {
    const float v = cs[ft] + __shfl_xor(cs[ft], 32, 64);
    if (h == 0) csr[w][32 * ft + l32] = v;
  }
  __syncthreads();
  float* out = C.mom_part + ((size_t)pid * C.nblk + blk) * (D * D + D);
  for (int e = tid; e < D * D; e += 256) out[e] = red[e];
  for (int f = tid; f < D; f += 256) out[D * D + f] = ((csr[0][f] + csr[1][f]) + csr[2][f]) + csr[3][f];
}

// Metric mode, queries: rho = q S_k (MFMA, lane = token), inv = 1/|rho| (0 if
// rho = 0) kept for the projection, and per row block the partial sums of
// inv^2 x x^T and inv x (r r^T = S_k^T (inv^2 x x^T) S_k is formed after the
// reduction).
template <int D>
__global__ __launch_bounds__(256) void qnorm_mfma_kernel(Ctx C) {
  constexpr int FT = D / 32, KS = D / 16, NT = FT * (FT + 1) / 2;
  __shared__ __attribute__((aligned(16))) char wl[2 * D * 2 * D];
  __shared__ float red[D * D];
  __shared__ float csr[4][D];
  __shared__ float sinv[4][32];
  const int bh = blockIdx.y, blk = blockIdx.x;
  const Side& S = C.s[0];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  stage_wops<D>(wop(C, bh, O_FK), wl);
  __syncthreads();
  const int r0 = blk * C.mom_rows, r1 = min(S.n, r0 + C.mom_rows);
  bf16x8 id[2];
  ident_ops(l32, h, id);
  f32x16 g[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int r = 0; r < 16; ++r) g[t][r] = 0.f;
  float cs[FT];
#pragma unroll
  for (int ft = 0; ft < FT; ++ft) cs[ft] = 0.f;
  for (int tok0 = r0 + 32 * w; tok0 < r1; tok0 += 128) {
    bf16x8 xop[KS];
    load_xtile<D>((const bf16*)S.x, bh, tok0, r1, S.lx, l32, h, xop);
    f32x16 acc[FT];
    project_tile<D>(wl, xop, l32, h, acc);
    float nrm = 0.f;
#pragma unroll
    for (int ot = 0; ot < FT; ++ot)
#pragma unroll
      for (int r = 0; r < 16; ++r) nrm = __builtin_fmaf(acc[ot][r], acc[ot][r], nrm);
    nrm += __shfl_xor(nrm, 32, 64);
    const float inv = nrm > 0.f ? 1.f / sqrtf(nrm) : 0.f;
    if (h == 0) {
      sinv[w][l32] = inv;
      if (tok0 + l32 < r1) C.inv_q[(size_t)bh * S.n + tok0 + l32] = inv;
    }
    __builtin_amdgcn_wave_barrier();
    f32x16 xT[FT];
    transpose_tile<D>(xop, id, xT);
    float wt[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) wt[r] = sinv[w][8 * (r >> 2) + 4 * h + (r & 3)];
#pragma unroll
    for (int ft = 0; ft < FT; ++ft)
#pragma unroll
      for (int r = 0; r < 16; ++r) cs[ft] = __builtin_fmaf(wt[r], xT[ft][r], cs[ft]);
    int t = 0;
#pragma unroll
    for (int it = 0; it < FT; ++it)
#pragma unroll
      for (int jt = it; jt < FT; ++jt, ++t)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          float bw[8], bl[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float v = wt[8 * s2 + j] * wt[8 * s2 + j] * xT[jt][8 * s2 + j];
            bw[j] = v;
          }
          const bf16x8 bhi = pack8(bw);
#pragma unroll
          for (int j = 0; j < 8; ++j) bl[j] = bw[j] - (float)bhi[j];
          const bf16x8 a = pack_half(xT[it], s2);
          g[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bhi, g[t], 0, 0, 0);
          g[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pack8(bl), g[t], 0, 0, 0);
        }
    __builtin_amdgcn_wave_barrier();
  }
  reduce_gram<D>(red, g, w, l32, h);
#pragma unroll
  for (int ft = 0; ft < FT; ++ft) {
    const float v = cs[ft] + __shfl_xor(cs[ft], 32, 64);
    if (h == 0) csr[w][32 * ft + l32] = v;
  }
  __syncthreads();
  float* out = C.qn_part + ((size_t)bh * C.nblk + blk) * (D * D + D);
  for (int e = tid; e < D * D; e += 256) out[e] = red[e];
  for (int f = tid; f < D; f += 256) out[D * D + f] = ((csr[0][f] + csr[1][f]) + csr[2][f]) + csr[3][f];
}

// Y = X T (keys) or inv * (X W_Q) (metric queries), lane = token, fp32 rows.
template <int D>
__global__ __launch_bounds__(256, 2) void project_mfma_kernel(Ctx C) {
  constexpr int FT = D / 32, KS = D / 16;
  __shared__ __attribute__((aligned(16))) char wl[2 * D * 2 * D];
  const int pid = blockIdx.y, side = pid / C.BH, bh = pid % C.BH;
  const Side& S = C.s[side];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, h = lane >> 5, l32 = lane & 31;
  const int r0 = blockIdx.x * C.proj_rows, r1 = min(S.n, r0 + C.proj_rows);
  if (r0 >= r1) return;
  stage_wops<D>(wop(C, bh, side == 0 ? O_TQ : O_TK), wl);
  __syncthreads();
  const bool scale = side == 0 && C.xf == CA_XF_METRIC;
  float* Y = S.y + (size_t)bh * S.n * D;
  for (int tok0 = r0 + 32 * w; tok0 < r1; tok0 += 128) {
    bf16x8 xop[KS];
    load_xtile<D>((const bf16*)S.x, bh, tok0, r1, S.lx, l32, h, xop);
    const int tok = tok0 + l32;
    const float sc = scale && tok < r1 ? C.inv_q[(size_t)bh * S.n + tok] : 1.f;
    float* yrow = Y + (size_t)tok * D;
    // one 32-column output tile at a time: a single accumulator stays live
    // (not unrolled, so the operand reads of later tiles are not hoisted)
#pragma unroll 1
    for (int ot = 0; ot < FT; ++ot) {
      f32x16 acc;
      project_tile1<D>(wl, xop, l32, h, ot, acc);
      if (tok < r1) {
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int col = 32 * ot + 8 * g4 + 4 * h;
          *(float4*)(yrow + col) = make_float4(acc[4 * g4] * sc, acc[4 * g4 + 1] * sc,
                                               acc[4 * g4 + 2] * sc, acc[4 * g4 + 3] * sc);
        }
        // the same values of coordinates 0 .. 15, coordinate-major: each
        // store is 32 consecutive tokens of one coordinate per half-wave
        if (ot == 0 && S.ycol) {
          static_assert(kColCopy == 16, "coordinates of g4 = 0, 1 of the first tile");
#pragma unroll
          for (int g4 = 0; g4 < 2; ++g4)
#pragma unroll
            for (int e = 0; e < 4; ++e)
              S.ycol[((size_t)bh * kColCopy + 8 * g4 + 4 * h + e) * S.n + tok] =
                  acc[4 * g4 + e] * sc;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Recursive split
// ---------------------------------------------------------------------------

// Highest-variance coordinate of the node's subsample, computed by one
// wavefront: lane t owns coordinates t and t + 64. fp64, two passes over the
// rows in order, mean = sum/m, variance = sum((y - mean)^2)/m, no contraction;
// ties go to the lowest coordinate. The sample rows are located first (lane j
// holds the row of sample j and j + 64), then read in batches of B
// independent loads; with at most B samples both passes use the one batch, so
// the whole choice costs two memory round trips (B = 64 where registers allow).
template <int B>
__device__ int choose_coordinate(const float* __restrict__ Y, int d, const int32_t* idx,
                                 bool identity, int start, int size, int lane,
                                 double* mean_out = nullptr, double* var_out = nullptr) {
#pragma clang fp contract(off)
  const int m = size < d ? size : d;
  int row[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int j = lane + 64 * h;
    int r = 0;
    if (j < m) {
      const int p = start + (int)(((int64_t)(2 * j + 1) * size) / (2 * m));
      r = identity ? p : idx[p];
    }
    row[h] = r;
  }
  double best = -1.0, bmean = 0.0;
  int bt = 0x7fffffff;
  for (int half = 0; half * 64 < d; ++half) {
    const int t = lane + 64 * half;
    const bool tv = t < d;
    const float* Yt = Y + (tv ? t : 0);
    double acc = 0.0;
    float v[B];
    auto load = [&](int j0) {
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const int j = j0 + u;
        const int r = __builtin_amdgcn_readlane(j < 64 ? row[0] : row[1], j & 63);
        v[u] = Yt[(size_t)r * d];
      }
    };
    for (int j0 = 0; j0 < m; j0 += B) {
      load(j0);
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (j0 + u < m) acc = acc + (double)v[u];
    }
    const double mean = acc / (double)m;
    double acc2 = 0.0;
    for (int j0 = 0; j0 < m; j0 += B) {
      if (B < 64 || m > B) load(j0);  // (a single batch of 64 is still in registers)
#pragma unroll
      for (int u = 0; u < B; ++u)
        if (j0 + u < m) {
          const double dv = (double)v[u] - mean;
          const double sq = dv * dv;
          acc2 = acc2 + sq;
        }
    }
    const double var = acc2 / (double)m;
    if (tv && (var > best || (var == best && t < bt))) {
      best = var;
      bmean = mean;
      bt = t;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const double ob = __shfl_xor(best, o, 64);
    const double om = __shfl_xor(bmean, o, 64);
    const int ot = __shfl_xor(bt, o, 64);
    if (ob > best || (ob == best && ot < bt)) {
      best = ob;
      bmean = om;
      bt = ot;
    }
  }
  if (mean_out) *mean_out = bmean;
  if (var_out) *var_out = best;
  return bt;
}

// Multi-block levels. A node's split threshold is its m_L-th smallest key,
// found exactly in two steps:
//   keys:   every chunk block gathers its keys and counts them into kBins
//           linear bins over [mean - 4 sd, mean + 4 sd] of the node's sample
//           (the clamped linear map is monotone, so each bin is a contiguous
//           key range); the chunk's histogram goes to its own slot.
//   select: one workgroup per node sums the chunk histograms, finds the bin
//           holding the wanted rank, collects that bin's keys (typically a
//           few hundred) and selects exactly among them with an 8-bit radix
//           select; it also turns the per-chunk counts below / equal to the
//           threshold into exclusive prefixes for the stable scatter.
// Kernel boundaries order the steps: no grid-wide fences or arrival counters.
//
// Node state (int32): 0 j* (-1: leaf), 1 threshold key, 2 rank among keys
// equal to the threshold, 3 left size, 4 start, 5 size, 6 bin origin (float),
// 7 number of chunks, 8 bin scale (float), 9 rank of the threshold.
__device__ __forceinline__ int32_t* node_ptr(const Ctx& C, int pid, int node) {
  return C.node_state + ((size_t)pid * C.max_nodes + node) * kNodeInts;
}

__device__ __forceinline__ float key_value(uint32_t key) {
  return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

// Bin of a key: floor((v - lo) * scale) clamped to [0, kBins); infinities and
// NaNs go to the end bin their key order puts them in.
__device__ __forceinline__ int lin_bin(uint32_t key, float lo, float scale) {
  if (key >= 0xFF800000u) return kBins - 1;  // +inf, positive NaNs
  if (key <= 0x007FFFFFu) return 0;          // -inf, negative NaNs
  float t = (key_value(key) - lo) * scale;
  t = fminf(fmaxf(t, 0.f), (float)(kBins - 1));
  return (int)t;
}

constexpr int kPer = kChunk / 256;  // positions per thread in a 256-thread chunk block

struct LevelArgs {
  int level;
  int first;  // input permutation is the identity
  int cpn;    // chunk slots per node at this level
  const int32_t* idx_in;
  int32_t* idx_out;
};

__global__ __launch_bounds__(64) void split_choose_kernel(Ctx C, LevelArgs L) {
  const int pid = blockIdx.y, side = pid / C.BH, bh = pid % C.BH, node = blockIdx.x;
  const Side& S = C.s[side];
  if (L.level >= S.big) return;
  int start, size;
  node_range(S.n, S.c, L.level, node, &start, &size);
  int32_t* ns = node_ptr(C, pid, node);
  const int lane = threadIdx.x;
  if (size <= S.c) {
    if (lane == 0) ns[0] = -1;
    return;
  }
  const int32_t* idx = L.idx_in + (size_t)pid * C.nmax;
  double mean, var;
  const int js = choose_coordinate<64>(S.y + (size_t)bh * S.n * C.d, C.d, idx, L.first, start, size,
                                   lane, &mean, &var);
  if (lane == 0) {
    const double sd = sqrt(var);
    float lo = (float)(mean - 4.0 * sd), scale = (float)((double)kBins / (8.0 * sd));
    if (!(sd > 0.0) || !isfinite(lo) || !isfinite(scale)) {
      lo = 0.f;
      scale = 0.f;  // one bin: the select step falls back to streaming
    }
    const int mL = left_size(size, S.c);
    ns[0] = js;
    ns[10] = 0;
    ns[1] = 0;
    ns[2] = 0;
    ns[3] = mL;
    ns[4] = start;
    ns[5] = size;
    ns[6] = __float_as_int(lo);
    ns[7] = (size + kChunk - 1) / kChunk;
    ns[8] = __float_as_int(scale);
    ns[9] = mL - 1;
  }
}

// ---------------------------------------------------------------------------
// Basic splitting (Method: recursive splitting, basic; a variation of
// principal direction divisive partitioning): the direction of each node at
// one level, by power iteration on its strided subsample. Every reduction
// runs in a fixed order with separately rounded products and sums (no fused
// multiply-add), so the directions, and the splits made on them, are
// reproducible bit for bit.
// ---------------------------------------------------------------------------

// Separately rounded fp32 operations: a product is never fused into the sum
// that follows it, and the quotient and square root are the correctly rounded
// ones (the default contraction would otherwise turn a + x * y into an FMA,
// and the HIP __f*_rn intrinsics are plain operators here).
__device__ __forceinline__ float add_rn(float a, float b) {
#pragma clang fp contract(off)
  return a + b;
}
__device__ __forceinline__ float sub_rn(float a, float b) {
#pragma clang fp contract(off)
  return a - b;
}
__device__ __forceinline__ float mul_rn(float a, float b) {
#pragma clang fp contract(off)
  return a * b;
}
__device__ __forceinline__ float div_rn(float a, float b) { return a / b; }
__device__ __forceinline__ float sqrt_rn(float a) { return __builtin_sqrtf(a); }

constexpr int kBasicThreads = 128;
constexpr int kBasicIters = 8;

__device__ __forceinline__ float* dir_ptr(const Ctx& C, int level, int pid, int node) {
  return C.dirs + ((((size_t)(level & 1) * 2 * C.BH) + pid) * C.max_nodes + node) * C.d;
}

// Output number c (counting from 0) of splitmix64 started at state 0
// (S. Vigna's generator).
__device__ __forceinline__ uint64_t splitmix64_at(uint64_t c) {
  uint64_t z = (c + 1ull) * 0x9e3779b97f4a7c15ull;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

// Approximately standard normal: the sum of 12 uniforms minus 6 (Irwin-Hall),
// uniform u the top 24 bits of output 16 c + u, summed as integers.
__device__ __forceinline__ float irwin_hall(uint64_t c) {
  long long sum = 0;
#pragma unroll
  for (int u = 0; u < 12; ++u) sum += (long long)(splitmix64_at(c * 16ull + (uint64_t)u) >> 40);
  return (float)((double)sum * 0x1p-24 - 6.0);
}

// One block per node of the level. Dynamic LDS: the subsample, m x (d + 1).
// D is the feature count when it is a compile-time constant (64, 128), so the
// in-order chains unroll and their LDS reads are issued ahead; D = 0 reads d
// from the problem. Norms are computed by every thread from the same LDS
// values (identical results), which saves a barrier per iteration.
template <int D>
__global__ __launch_bounds__(kBasicThreads) void basic_choose_kernel(Ctx C, LevelArgs L) {
  extern __shared__ __attribute__((aligned(16))) float bsub[];
  __shared__ float mu[kMaxD], v[kMaxD], t[kMaxD], w[kMaxD];
  const int pid = blockIdx.y, side = pid / C.BH, bh = pid % C.BH, node = blockIdx.x;
  const Side& S = C.s[side];
  if (L.level >= S.big) return;
  int start, size;
  node_range(S.n, S.c, L.level, node, &start, &size);
  int32_t* ns = node_ptr(C, pid, node);
  const int tid = threadIdx.x, d = D ? D : C.d, DP = d + 1;
  if (size <= S.c) {
    if (tid == 0) ns[0] = -1;
    return;
  }
  const int m = d < size ? d : size;
  const int32_t* idx = L.idx_in + (size_t)pid * C.nmax;
  const float* Y = S.y + (size_t)bh * S.n * d;
  if (D != 0 && D % 4 == 0) {
    // float4 reads of the sample rows
    const int d4 = d / 4;
    for (int e = tid; e < m * d4; e += kBasicThreads) {
      const int j = e / d4, k4 = e % d4;
      const int p = (int)(((long long)(2 * j + 1) * size) / (2 * m));
      const int row = L.first ? start + p : idx[start + p];
      const float4 x = *(const float4*)(Y + (size_t)row * d + 4 * k4);
      float* dst = bsub + j * DP + 4 * k4;
      dst[0] = x.x;
      dst[1] = x.y;
      dst[2] = x.z;
      dst[3] = x.w;
    }
  } else {
    for (int e = tid; e < m * d; e += kBasicThreads) {
      const int j = e / d, k = e % d;
      const int p = (int)(((long long)(2 * j + 1) * size) / (2 * m));
      const int row = L.first ? start + p : idx[start + p];
      bsub[j * DP + k] = Y[(size_t)row * d + k];
    }
  }
  // warm start noise of this node
  if (tid < d) {
    const uint64_t base = ((((uint64_t)(2 * bh + side) << 5 | (uint64_t)L.level) << 20 |
                            (uint64_t)node) << 7);
    t[tid] = irwin_hall(base | (uint64_t)tid);
  }
  __syncthreads();
  if (tid < d) {
    float a = 0.f;
    for (int j = 0; j < m; ++j) a = add_rn(a, bsub[j * DP + tid]);
    mu[tid] = div_rn(a, (float)m);
  }
  __syncthreads();
  for (int e = tid; e < m * d; e += kBasicThreads) {
    const int j = e / d, k = e % d;
    bsub[j * DP + k] = sub_rn(bsub[j * DP + k], mu[k]);
  }
  // the parent's direction one level up, mixed with the noise
  const float* vp = L.level > 0 ? dir_ptr(C, L.level - 1, pid, node >> 1) : nullptr;
  if (tid < d) {
    float vk = t[tid];
    if (vp) {
      float nv = 0.f, nr = 0.f;
#pragma unroll 16
      for (int k = 0; k < d; ++k) {
        const float pk = vp[k];
        nv = add_rn(nv, mul_rn(pk, pk));
        nr = add_rn(nr, mul_rn(t[k], t[k]));
      }
      const float sc = div_rn(sqrt_rn(nv), sqrt_rn(nr));
      vk = mul_rn(add_rn(vp[tid], mul_rn(vk, sc)), 0.5f);
    }
    v[tid] = vk;
  }
  for (int it = 0; it < kBasicIters; ++it) {
    __syncthreads();
    if (tid < m) {
      float a = 0.f;
#pragma unroll 16
      for (int k = 0; k < d; ++k) a = add_rn(a, mul_rn(bsub[tid * DP + k], v[k]));
      t[tid] = a;
    }
    __syncthreads();
    if (tid < d) {
      float a = 0.f;
#pragma unroll 16
      for (int j = 0; j < m; ++j) a = add_rn(a, mul_rn(t[j], bsub[j * DP + tid]));
      w[tid] = a;
    }
    __syncthreads();
    if (tid < d) {
      float nn = 0.f;
#pragma unroll 16
      for (int k = 0; k < d; ++k) nn = add_rn(nn, mul_rn(w[k], w[k]));
      if (nn > 0.f) v[tid] = div_rn(w[tid], sqrt_rn(nn));
    }
  }
  __syncthreads();
  float* vo = dir_ptr(C, L.level, pid, node);
  if (tid < d) vo[tid] = v[tid];
  // spread of the subsample's projections, for the linear bins of the select
  if (tid < m) {
    float a = 0.f;
#pragma unroll 16
    for (int k = 0; k < d; ++k) a = add_rn(a, mul_rn(bsub[tid * DP + k], v[k]));
    t[tid] = a;
  }
  __syncthreads();
  if (tid == 0) {
    double mp = 0.0, vv = 0.0;
    for (int k = 0; k < d; ++k) mp += (double)mu[k] * (double)v[k];
    for (int j = 0; j < m; ++j) vv += (double)t[j] * (double)t[j];
    const double sd = sqrt(vv / m);
    float lo = (float)(mp - 4.0 * sd), scale = (float)((double)kBins / (8.0 * sd));
    if (!(sd > 0.0) || !isfinite(lo) || !isfinite(scale)) {
      lo = 0.f;
      scale = 0.f;  // one bin: the select step falls back to streaming
    }
    const int mL = left_size(size, S.c);
    ns[0] = 0;
    ns[1] = 0;
    ns[2] = 0;
    ns[3] = mL;
    ns[10] = 0;
    ns[4] = start;
    ns[5] = size;
    ns[6] = __float_as_int(lo);
    ns[7] = (size + kChunk - 1) / kChunk;
    ns[8] = __float_as_int(scale);
    ns[9] = mL - 1;
  }
}

// d = 64: one wavefront per node. Lane j holds sample row j and lane k holds
// coordinate k of every sample row (the sample column), both read straight
// from HBM, so each in-order chain runs on registers and 16-byte broadcast
// reads of one LDS vector (v, t or w). Same operations, in the same order, as
// basic_choose_kernel.
__global__ __launch_bounds__(64) void basic_choose64_kernel(Ctx C, LevelArgs L) {
  constexpr int D = 64;
  __shared__ __attribute__((aligned(16))) float mu[D], v[D], t[D], w[D];
  const int pid = blockIdx.y, side = pid / C.BH, bh = pid % C.BH, node = blockIdx.x;
  const Side& S = C.s[side];
  if (L.level >= S.big) return;
  int start, size;
  node_range(S.n, S.c, L.level, node, &start, &size);
  int32_t* ns = node_ptr(C, pid, node);
  const int lane = threadIdx.x;
  if (size <= S.c) {
    if (lane == 0) ns[0] = -1;
    return;
  }
  const int m = D < size ? D : size;
  const int32_t* idx = L.idx_in + (size_t)pid * C.nmax;
  const float* Y = S.y + (size_t)bh * S.n * D;
  int myrow = L.first ? start : idx[start];
  if (lane < m) {
    const int p = (int)(((long long)(2 * lane + 1) * size) / (2 * m));
    myrow = L.first ? start + p : idx[start + p];
  }
  float row[D], col[D];
  {
    const float4* src = (const float4*)(Y + (size_t)myrow * D);
#pragma unroll
    for (int k4 = 0; k4 < D / 4; ++k4) {
      const float4 x = src[k4];
      row[4 * k4] = x.x;
      row[4 * k4 + 1] = x.y;
      row[4 * k4 + 2] = x.z;
      row[4 * k4 + 3] = x.w;
    }
  }
  // Entries past the m sample rows are held at exactly zero, so every chain
  // can run over all D terms without branches: a sum that starts at +0 never
  // becomes -0 in round-to-nearest, so adding a zero product leaves it as is.
  uint32_t keep[D / 32];
#pragma unroll
  for (int h = 0; h < D / 32; ++h)
    keep[h] = m >= 32 * (h + 1) ? 0xFFFFFFFFu : (m <= 32 * h ? 0u : (1u << (m - 32 * h)) - 1u);
  auto kept = [&](float x, int j) {
    return __uint_as_float(__float_as_uint(x) & (0u - ((keep[j >> 5] >> (j & 31)) & 1u)));
  };
#pragma unroll
  for (int j = 0; j < D; ++j) {
    const int rj = __builtin_amdgcn_readlane(myrow, j);
    col[j] = kept(Y[(size_t)rj * D + lane], j);
  }
  float a = 0.f;
#pragma unroll
  for (int j = 0; j < D; ++j) a = add_rn(a, col[j]);
  const float muk = div_rn(a, (float)m);
  mu[lane] = muk;
#pragma unroll
  for (int j = 0; j < D; ++j) col[j] = kept(sub_rn(col[j], muk), j);
  const uint64_t base = ((((uint64_t)(2 * bh + side) << 5 | (uint64_t)L.level) << 20 |
                          (uint64_t)node) << 7);
  const float noise = irwin_hall(base | (uint64_t)lane);
  t[lane] = noise;
  __syncthreads();
#pragma unroll
  for (int k4 = 0; k4 < D / 4; ++k4) {
    const float4 u = *(const float4*)(mu + 4 * k4);
    row[4 * k4] = sub_rn(row[4 * k4], u.x);
    row[4 * k4 + 1] = sub_rn(row[4 * k4 + 1], u.y);
    row[4 * k4 + 2] = sub_rn(row[4 * k4 + 2], u.z);
    row[4 * k4 + 3] = sub_rn(row[4 * k4 + 3], u.w);
  }
  // warm start: the parent's direction one level up, mixed with the noise
  float vk = noise;
  if (L.level > 0) {
    const float* vp = dir_ptr(C, L.level - 1, pid, node >> 1);
    float nv = 0.f, nr = 0.f;
#pragma unroll
    for (int k4 = 0; k4 < D / 4; ++k4) {
      const float4 pv = *(const float4*)(vp + 4 * k4);
      const float4 r4 = *(const float4*)(t + 4 * k4);
      nv = add_rn(nv, mul_rn(pv.x, pv.x));
      nr = add_rn(nr, mul_rn(r4.x, r4.x));
      nv = add_rn(nv, mul_rn(pv.y, pv.y));
      nr = add_rn(nr, mul_rn(r4.y, r4.y));
      nv = add_rn(nv, mul_rn(pv.z, pv.z));
      nr = add_rn(nr, mul_rn(r4.z, r4.z));
      nv = add_rn(nv, mul_rn(pv.w, pv.w));
      nr = add_rn(nr, mul_rn(r4.w, r4.w));
    }
    const float sc = div_rn(sqrt_rn(nv), sqrt_rn(nr));
    vk = mul_rn(add_rn(vp[lane], mul_rn(noise, sc)), 0.5f);
  }
  __syncthreads();
  v[lane] = vk;
  for (int it = 0; it < kBasicIters; ++it) {
    __syncthreads();
    float ta = 0.f;
#pragma unroll
    for (int k4 = 0; k4 < D / 4; ++k4) {
      const float4 q = *(const float4*)(v + 4 * k4);
      ta = add_rn(ta, mul_rn(row[4 * k4], q.x));
      ta = add_rn(ta, mul_rn(row[4 * k4 + 1], q.y));
      ta = add_rn(ta, mul_rn(row[4 * k4 + 2], q.z));
      ta = add_rn(ta, mul_rn(row[4 * k4 + 3], q.w));
    }
    t[lane] = lane < m ? ta : 0.f;
    __syncthreads();
    float wa = 0.f;
#pragma unroll
    for (int j4 = 0; j4 < D / 4; ++j4) {
      const float4 q = *(const float4*)(t + 4 * j4);
      wa = add_rn(wa, mul_rn(q.x, col[4 * j4]));
      wa = add_rn(wa, mul_rn(q.y, col[4 * j4 + 1]));
      wa = add_rn(wa, mul_rn(q.z, col[4 * j4 + 2]));
      wa = add_rn(wa, mul_rn(q.w, col[4 * j4 + 3]));
    }
    w[lane] = wa;
    __syncthreads();
    float nn = 0.f;
#pragma unroll
    for (int k4 = 0; k4 < D / 4; ++k4) {
      const float4 q = *(const float4*)(w + 4 * k4);
      nn = add_rn(nn, mul_rn(q.x, q.x));
      nn = add_rn(nn, mul_rn(q.y, q.y));
      nn = add_rn(nn, mul_rn(q.z, q.z));
      nn = add_rn(nn, mul_rn(q.w, q.w));
    }
    if (nn > 0.f) v[lane] = div_rn(wa, sqrt_rn(nn));
  }
  __syncthreads();
  dir_ptr(C, L.level, pid, node)[lane] = v[lane];
  // spread of the subsample's projections, for the linear bins of the select
  float ta = 0.f;
#pragma unroll
  for (int k4 = 0; k4 < D / 4; ++k4) {
    const float4 q = *(const float4*)(v + 4 * k4);
    ta = add_rn(ta, mul_rn(row[4 * k4], q.x));
    ta = add_rn(ta, mul_rn(row[4 * k4 + 1], q.y));
    ta = add_rn(ta, mul_rn(row[4 * k4 + 2], q.z));
    ta = add_rn(ta, mul_rn(row[4 * k4 + 3], q.w));
  }
  t[lane] = ta;
  __syncthreads();
  if (lane == 0) {
    double mp = 0.0, vv = 0.0;
    for (int k = 0; k < D; ++k) mp += (double)mu[k] * (double)v[k];
    for (int j = 0; j < m; ++j) vv += (double)t[j] * (double)t[j];
    const double sd = sqrt(vv / m);
    float lo = (float)(mp - 4.0 * sd), scale = (float)((double)kBins / (8.0 * sd));
    if (!(sd > 0.0) || !isfinite(lo) || !isfinite(scale)) {
      lo = 0.f;
      scale = 0.f;  // one bin: the select step falls back to streaming
    }
    const int mL = left_size(size, S.c);
    ns[0] = 0;
    ns[1] = 0;
    ns[2] = 0;
    ns[3] = mL;
    ns[4] = start;
    ns[5] = size;
    ns[6] = __float_as_int(lo);
    ns[7] = (size + kChunk - 1) / kChunk;
    ns[8] = __float_as_int(scale);
    ns[9] = mL - 1;
    ns[10] = 0;
  }
}

// The order after the last split level, copied to perm (basic splitting runs
// every level with the multi-block kernels, so no tail pass is needed).
__global__ __launch_bounds__(256) void copy_order_kernel(Ctx C, int parity0, int parity1) {
  const int pid = blockIdx.y, side = pid / C.BH, bh = pid % C.BH;
  const Side& S = C.s[side];
  const int32_t* src = ((side == 0 ? parity0 : parity1) ? C.idx1 : C.idx0) + (size_t)pid * C.nmax;
  int32_t* perm = S.perm + (size_t)bh * S.n;
  const bool identity = S.big == 0;
  for (int o = blockIdx.x * 256 + threadIdx.x; o < S.n; o += gridDim.x * 256)
    perm[o] = identity ? o : src[o];
}

// T_K = F_q and T_Q = F_k (basic splitting in the metric root space), and
// for the MFMA projection their transposed hi/lo bf16 operands: W_Q^T is the
// operand the Cholesky pass already packed for F_k, W_K^T is packed here.
__global__ __launch_bounds__(256) void copy_roots_kernel(Ctx C, int pack) {
  const int bh = blockIdx.x, d = C.d, dd = d * d;
  const float* Fq = mat(C, bh, M_E0);
  for (int e = threadIdx.x; e < dd; e += 256) {
    mat(C, bh, M_TK)[e] = Fq[e];
    mat(C, bh, M_TQ)[e] = mat(C, bh, M_EK)[e];
  }
  if (!pack) return;
  bf16* tk = wop(C, bh, O_TK);
  bf16* tq = wop(C, bh, O_TQ);
  const bf16* fk = wop(C, bh, O_FK);
  for (int e = threadIdx.x; e < dd; e += 256) {
    const int i = e / d, k = e % d;  // row i = output dim, column k = input dim
    const float w = Fq[k * d + i];
    const bf16 hi = (bf16)w;
    tk[e] = hi;
    tk[dd + e] = (bf16)(w - (float)hi);
    tq[e] = fk[e];
    tq[dd + e] = fk[dd + e];
  }
}

// Block-wide exclusive scan (NT threads).
template <int NT>
__device__ __forceinline__ int block_scan(int x, int* wsum, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int v = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(v, o, 64);
    if (lane >= o) v += y;
  }
  if (lane == 63) wsum[w] = v;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) {
    const int ws = wsum[i];
    base += i < w ? ws : 0;
    tot += ws;
  }
  __syncthreads();
  *total = tot;
  return base + v - x;
}

__device__ __forceinline__ int scan256(int x, int* wsum, int* total) {
  return block_scan<256>(x, wsum, total);
}

// Keys of one chunk and its linear-bin histogram.
// Projection keys of a thread's kPer rows on the direction dv (LDS): each row
// is read whole with 16-byte loads, R rows at a time (two at d = 64, one at
// d = 128 to bound registers), and its coordinates are summed in order with
// separately rounded products.
template <int D>
__device__ __forceinline__ void basic_keys(const float* __restrict__ Y, const int (&rows)[kPer],
                                           const float* dv, int nu, uint32_t (&kv)[kPer]) {
  constexpr int D4 = D / 4, R = D <= 64 ? 2 : 1;
#pragma unroll
  for (int u = 0; u < kPer; u += R) {
    if (u >= nu) break;  // block-uniform: no position of the chunk is left
    float4 x[R][D4];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const float4* src = (const float4*)(Y + (size_t)rows[u + r] * D);
#pragma unroll
      for (int k = 0; k < D4; ++k) x[r][k] = src[k];
    }
    float a[R];
#pragma unroll
    for (int r = 0; r < R; ++r) a[r] = 0.f;
#pragma unroll
    for (int k = 0; k < D4; ++k) {
      const float4 w = *(const float4*)(dv + 4 * k);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        a[r] = add_rn(a[r], mul_rn(x[r][k].x, w.x));
        a[r] = add_rn(a[r], mul_rn(x[r][k].y, w.y));
        a[r] = add_rn(a[r], mul_rn(x[r][k].z, w.z));
        a[r] = add_rn(a[r], mul_rn(x[r][k].w, w.w));
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) kv[u + r] = ordered_bits(a[r]);
  }
}

// BD < 0: keys are the chosen coordinate (diagonalized splitting); BD >= 0:
// projections on the node's direction (basic splitting), BD = d when it is
// 64 or 128, else 0.
template <int BD>
__global__ __launch_bounds__(256) void split_keys_kernel(Ctx C, LevelArgs L) {
  __shared__ int lh[kBins];
  const int pid = blockIdx.z, side = pid / C.BH, bh = pid % C.BH, node = blockIdx.y;
  const Side& S = C.s[side];
  if (L.level >= S.big) return;
  int32_t* ns = node_ptr(C, pid, node);
  const int js = ns[0];
  if (js < 0) return;
  const int start = ns[4], size = ns[5];
  const float lo = __int_as_float(ns[6]), scale = __int_as_float(ns[8]);
  const int c0 = blockIdx.x * kChunk;
  if (c0 >= size) return;
  const int c1 = min(size, c0 + kChunk);
  for (int b = threadIdx.x; b < kBins; b += 256) lh[b] = 0;
  const float* Y = S.y + (size_t)bh * S.n * C.d;
  const int32_t* idx = L.idx_in + (size_t)pid * C.nmax;
  uint32_t* keys = C.keys + (size_t)pid * C.nmax;
  // All of a thread's loads are issued before any is used.
  int rows[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int o = c0 + threadIdx.x + 256 * u;
    rows[u] = o < c1 ? (L.first ? start + o : idx[start + o]) : 0;
  }
  uint32_t kv[kPer];
  if constexpr (BD >= 0) {
    // projection on the node's direction, coordinates summed in order
    __shared__ __attribute__((aligned(16))) float dv[kMaxD];
    const float* dir = dir_ptr(C, L.level, pid, node);
    for (int k = threadIdx.x; k < C.d; k += 256) dv[k] = dir[k];
    __syncthreads();
    if constexpr (BD > 0)
      basic_keys<BD>(Y, rows, dv, (c1 - c0 + 255) / 256, kv);
    else
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const float* yr = Y + (size_t)rows[u] * C.d;
        float a = 0.f;
        for (int k = 0; k < C.d; ++k) a = add_rn(a, mul_rn(yr[k], dv[k]));
        kv[u] = ordered_bits(a);
      }
  } else if (S.ycol && js < kColCopy) {
    // the node's coordinate from its contiguous column: the nodes of a level
    // share few columns, so the lines they read are mostly used in full
    const float* col = S.ycol + ((size_t)bh * kColCopy + js) * S.n;
#pragma unroll
    for (int u = 0; u < kPer; ++u) kv[u] = ordered_bits(col[rows[u]]);
  } else {
#pragma unroll
    for (int u = 0; u < kPer; ++u) kv[u] = ordered_bits(Y[(size_t)rows[u] * C.d + js]);
  }
  {
    if (size <= kChunk) {
      // The whole node is in this block: exact select of the rank-th key here
      // (four 8-bit digits, high first), and no histogram for the select pass.
      __shared__ int rh[256];
      __shared__ int sh_digit, sh_rank;
      const int tid = threadIdx.x, lane = tid & 63;
      uint32_t thr = 0u;
      int r = ns[9];
      for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        rh[tid] = 0;
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
          const int o = tid + 256 * u;
          if (o < c1 && (pass == 0 || (kv[u] >> (shift + 8)) == (thr >> (shift + 8))))
            atomicAdd(&rh[(kv[u] >> shift) & 255u], 1);
        }
        __syncthreads();
        if (tid < 64) {
          int cnt[4], sum = 0;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            cnt[i] = rh[4 * tid + i];
            sum += cnt[i];
          }
          int incl = sum;
#pragma unroll
          for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(incl, o, 64);
            if (lane >= o) incl += y;
          }
          int acc = incl - sum;
          if (r >= acc && r < incl) {
            for (int i = 0; i < 4; ++i) {
              if (r < acc + cnt[i]) {
                sh_digit = 4 * tid + i;
                sh_rank = r - acc;
                break;
              }
              acc += cnt[i];
            }
          }
        }
        __syncthreads();
        thr |= (uint32_t)sh_digit << shift;
        r = sh_rank;
      }
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int o = tid + 256 * u;
        if (o < c1) keys[start + o] = kv[u];
      }
      if (tid == 0) {
        int32_t* cc = C.chunk_cnt + ((size_t)pid * C.hist_slots + (size_t)node * L.cpn) * 2;
        cc[0] = 0;
        cc[1] = 0;
        ns[1] = (int)thr;
        ns[2] = r;
        ns[10] = 1;  // selected
      }
      return;
    }
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int o = c0 + threadIdx.x + 256 * u;
    if (o < c1) {
      keys[start + o] = kv[u];
      atomicAdd(&lh[lin_bin(kv[u], lo, scale)], 1);
    }
  }
  __syncthreads();
  uint4* gh = reinterpret_cast<uint4*>(
      C.hist + ((size_t)pid * C.hist_slots + (size_t)node * L.cpn + blockIdx.x) * kBins);
  for (int b = threadIdx.x; b < kBins / 4; b += 256)
    gh[b] = make_uint4((uint32_t)lh[4 * b], (uint32_t)lh[4 * b + 1], (uint32_t)lh[4 * b + 2],
                       (uint32_t)lh[4 * b + 3]);
}

constexpr int kSelThreads = 1024;
constexpr int kCand = 8192;         // candidates held in LDS
constexpr int kMaxNodeChunks = 1024;  // chunks of one node (4M positions)
static_assert(kBins == 4 * kSelThreads, "one uint4 of bins per select thread");

__global__ __launch_bounds__(kSelThreads) void split_select_kernel(Ctx C, LevelArgs L) {
  __shared__ uint32_t ckey[kCand];
  __shared__ uint16_t cchunk[kCand];
  __shared__ int below_ch[kMaxNodeChunks], less_ch[kMaxNodeChunks], eq_ch[kMaxNodeChunks];
  __shared__ int rh[256];
  __shared__ int wsum[kSelThreads / 64];
  __shared__ int sh_bin, sh_below, sh_ncand, sh_digit, sh_rank;
  const int pid = blockIdx.y, node = blockIdx.x, side = pid / C.BH;
  const Side& S = C.s[side];
  if (L.level >= S.big) return;
  int32_t* ns = node_ptr(C, pid, node);
  if (ns[0] < 0 || ns[10]) return;  // a leaf, or selected with its keys
  const int start = ns[4], size = ns[5], nch = ns[7];
  const float lo = __int_as_float(ns[6]), scale = __int_as_float(ns[8]);
  const int tid = threadIdx.x, lane = tid & 63;
  const uint4* H = reinterpret_cast<const uint4*>(
      C.hist + ((size_t)pid * C.hist_slots + (size_t)node * L.cpn) * kBins);
  const uint32_t* keys = C.keys + (size_t)pid * C.nmax + start;
  for (int ch = tid; ch < nch; ch += kSelThreads) {
    below_ch[ch] = 0;
    less_ch[ch] = 0;
    eq_ch[ch] = 0;
  }
  if (tid == 0) sh_ncand = 0;
  // 1. node histogram: thread t owns bins 4t .. 4t+3
  uint32_t nb[4] = {0u, 0u, 0u, 0u};
  for (int ch0 = 0; ch0 < nch; ch0 += 8) {
    uint4 hv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      hv[u] = ch0 + u < nch ? H[(size_t)(ch0 + u) * (kBins / 4) + tid] : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      nb[0] += hv[u].x;
      nb[1] += hv[u].y;
      nb[2] += hv[u].z;
      nb[3] += hv[u].w;
    }
  }
  const int rank = ns[9];
  int tot;
  const int before = block_scan<kSelThreads>((int)(nb[0] + nb[1] + nb[2] + nb[3]), wsum, &tot);
  {
    int acc = before;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (rank >= acc && rank < acc + (int)nb[i]) {
        sh_bin = 4 * tid + i;
        sh_below = acc;
      }
      acc += (int)nb[i];
    }
  }
  __syncthreads();
  const int bstar = sh_bin, below = sh_below;
  // 2. per-chunk counts of keys in bins below b*
  for (int ch0 = 0; ch0 < nch; ch0 += 8) {
    uint4 hv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      hv[u] = ch0 + u < nch && 4 * tid < bstar ? H[(size_t)(ch0 + u) * (kBins / 4) + tid]
                                                : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      int part = (int)hv[u].x + (4 * tid + 1 < bstar ? (int)hv[u].y : 0) +
                 (4 * tid + 2 < bstar ? (int)hv[u].z : 0) +
                 (4 * tid + 3 < bstar ? (int)hv[u].w : 0);
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o, 64);
      if (lane == 0 && part) atomicAdd(&below_ch[ch0 + u], part);
    }
  }
  // 3. collect the keys of bin b*
  constexpr int B = 16;
  for (int o0 = 0; o0 < size; o0 += B * kSelThreads) {
    uint32_t kv[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int o = o0 + tid + kSelThreads * u;
      kv[u] = o < size ? keys[o] : 0u;
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int o = o0 + tid + kSelThreads * u;
      const bool hit = o < size && lin_bin(kv[u], lo, scale) == bstar;
      const uint64_t m = __ballot(hit);
      if (m == 0) continue;
      int base = 0;
      if (lane == 0) base = atomicAdd(&sh_ncand, __popcll(m));
      base = __shfl(base, 0, 64);
      if (hit) {
        const int slot = base + (int)__popcll(m & ((1ull << lane) - 1ull));
        if (slot < kCand) {
          ckey[slot] = kv[u];
          cchunk[slot] = (uint16_t)(o / kChunk);
        }
      }
    }
  }
  __syncthreads();
  const int ncand = sh_ncand;
  const bool in_lds = ncand <= kCand;
  // 4. exact select among the candidates: four 8-bit digits, high first
  uint32_t thr = 0u;
  int r = rank - below;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (tid < 256) rh[tid] = 0;
    __syncthreads();
    auto count = [&](uint32_t key) {
      if (pass == 0 || (key >> (shift + 8)) == (thr >> (shift + 8)))
        atomicAdd(&rh[(key >> shift) & 255u], 1);
    };
    if (in_lds) {
      for (int i = tid; i < ncand; i += kSelThreads) count(ckey[i]);
    } else {
      for (int o = tid; o < size; o += kSelThreads) {
        const uint32_t key = keys[o];
        if (lin_bin(key, lo, scale) == bstar) count(key);
      }
    }
    __syncthreads();
    if (tid < 64) {
      int cnt[4], sum = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        cnt[i] = rh[4 * tid + i];
        sum += cnt[i];
      }
      int incl = sum;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
      }
      int acc = incl - sum;
      if (r >= acc && r < incl) {
        for (int i = 0; i < 4; ++i) {
          if (r < acc + cnt[i]) {
            sh_digit = 4 * tid + i;
            sh_rank = r - acc;
            break;
          }
          acc += cnt[i];
        }
      }
    }
    __syncthreads();
    thr |= (uint32_t)sh_digit << shift;
    r = sh_rank;
    __syncthreads();
  }
  // 5. per-chunk counts of candidates below / equal to the threshold
  auto tally = [&](uint32_t key, int ch) {
    if (key < thr) atomicAdd(&less_ch[ch], 1);
    else if (key == thr) atomicAdd(&eq_ch[ch], 1);
  };
  if (in_lds) {
    for (int i = tid; i < ncand; i += kSelThreads) tally(ckey[i], cchunk[i]);
  } else {
    for (int o = tid; o < size; o += kSelThreads) {
      const uint32_t key = keys[o];
      if (lin_bin(key, lo, scale) == bstar) tally(key, o / kChunk);
    }
  }
  __syncthreads();
  // 6. exclusive prefixes over the node's chunks
  int32_t* cc = C.chunk_cnt + ((size_t)pid * C.hist_slots + (size_t)node * L.cpn) * 2;
  int base_l = 0, base_e = 0;
  for (int g = 0; g < nch; g += kSelThreads) {
    const int ch = g + tid;
    const int l = ch < nch ? below_ch[ch] + less_ch[ch] : 0, e = ch < nch ? eq_ch[ch] : 0;
    int sl, se;
    const int xl = block_scan<kSelThreads>(l, wsum, &sl);
    const int xe = block_scan<kSelThreads>(e, wsum, &se);
    if (ch < nch) {
      cc[2 * ch] = base_l + xl;
      cc[2 * ch + 1] = base_e + xe;
    }
    base_l += sl;
    base_e += se;
  }
  if (tid == 0) {
    ns[1] = (int)thr;
    ns[2] = r;
  }
}

// Stable partition of every node: the m_L smallest (key, position) pairs go
// left in node order, the rest right in node order. Nodes that are already
// leaves are copied.
// LDS slot of position i of a chunk: one pad word per 16, so that the
// 16-position runs of consecutive threads start on different banks.
__device__ __forceinline__ int scat_slot(int i) { return i + (i >> 4); }

__global__ __launch_bounds__(256) void split_scatter_kernel(Ctx C, LevelArgs L) {
  __shared__ int wsum[4];
  __shared__ uint32_t skey[kChunk + kChunk / 16];
  __shared__ int32_t srow[kChunk + kChunk / 16];
  __shared__ int32_t sout[kChunk];
  const int pid = blockIdx.z, side = pid / C.BH, node = blockIdx.y;
  const Side& S = C.s[side];
  if (L.level >= S.big) return;
  int start, size;
  node_range(S.n, S.c, L.level, node, &start, &size);
  const int c0 = blockIdx.x * kChunk;
  if (c0 >= size) return;
  const int c1 = min(size, c0 + kChunk), nc = c1 - c0;
  const int32_t* idx_in = L.idx_in + (size_t)pid * C.nmax;
  int32_t* idx_out = L.idx_out + (size_t)pid * C.nmax;
  const int32_t* ns = node_ptr(C, pid, node);
  const int t = threadIdx.x;
  if (size <= S.c) {
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int o = c0 + t + 256 * u;
      if (o < c1) idx_out[start + o] = L.first ? start + o : idx_in[start + o];
    }
    return;
  }
  const uint32_t thr = (uint32_t)ns[1];
  const int need_eq = ns[2] + 1, mL = ns[3];
  const int32_t* cc =
      C.chunk_cnt + ((size_t)pid * C.hist_slots + (size_t)node * L.cpn + blockIdx.x) * 2;
  const int less0 = cc[0], eq0 = cc[1];
  const uint32_t* keys = C.keys + (size_t)pid * C.nmax;
  // coalesced loads of the chunk's keys and rows into LDS
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = t + 256 * u;
    if (i < nc) {
      skey[scat_slot(i)] = keys[start + c0 + i];
      srow[scat_slot(i)] = L.first ? start + c0 + i : idx_in[start + c0 + i];
    }
  }
  __syncthreads();
  // Each thread owns kPer consecutive positions (the scan order).
  const int i0 = t * kPer;
  uint32_t kv[kPer];
  int less = 0, eq = 0;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = i0 + u;
    kv[u] = i < nc ? skey[scat_slot(i)] : 0xFFFFFFFFu;
    less += i < nc && kv[u] < thr;
    eq += i < nc && kv[u] == thr;
  }
  int tot;
  const int packed = scan256((less << 16) | eq, wsum, &tot);
  // The chunk's left-goers land in one contiguous range of the node starting
  // at lmin, its right-goers in one starting at rmin: stage both in order,
  // left part first, then write them out coalesced.
  const int lmin = less0 + min(eq0, need_eq);
  const int rmin = mL + (c0 - lmin);
  const int tot_less = tot >> 16, tot_eq = tot & 0xFFFF;
  const int nleft = tot_less + min(eq0 + tot_eq, need_eq) - min(eq0, need_eq);
  int lb = less0 + (packed >> 16), eb = eq0 + (packed & 0xFFFF);
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = i0 + u;
    if (i >= nc) break;
    const uint32_t key = kv[u];
    const int Lo = lb + min(eb, need_eq);
    const bool left = key < thr || (key == thr && eb < need_eq);
    const int loc = left ? Lo - lmin : nleft + (c0 + i - Lo) - (c0 - lmin);
    if (loc >= 0 && loc < nc) sout[loc] = srow[scat_slot(i)];
    lb += key < thr;
    eb += key == thr;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int i = t + 256 * u;
    if (i < nc) {
      const int dst = i < nleft ? lmin + i : rmin + (i - nleft);
      if (dst >= 0 && dst < size) idx_out[start + dst] = sout[i];
    }
  }
}

// Remaining levels of one node (at most the side's tail size) in one
// workgroup: per level every active sub-node picks its coordinate (one
// wavefront each), keys are gathered, a four-pass 8-bit radix select runs on
// per-sub-node LDS histograms, and a block-wide scan partitions stably.
constexpr int kTailThreads = 512;
constexpr int kMaxSub = 32;

__device__ __forceinline__ int scan_tail(int x, int* wsum) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int v = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(v, o, 64);
    if (lane >= o) v += y;
  }
  if (lane == 63) wsum[w] = v;
  __syncthreads();
  int base = 0;
#pragma unroll
  for (int i = 0; i < kTailThreads / 64; ++i)
    if (i < w) base += wsum[i];
  __syncthreads();
  return base + v - x;
}

__global__ __launch_bounds__(kTailThreads, 4) void split_tail_kernel(Ctx C, int parity0, int parity1) {
  __shared__ int32_t ia[kTail], ib[kTail];
  __shared__ uint32_t keys[kTail];
  __shared__ int scan[kTail + 1];
  __shared__ int hist[kMaxSub][256];
  __shared__ int sub_start[2 * kMaxSub + 2], sub_size[2 * kMaxSub + 2];
  __shared__ int sub_js[2 * kMaxSub + 2], sub_thr[2 * kMaxSub + 2], sub_rank[2 * kMaxSub + 2];
  __shared__ int act_list[kMaxSub], act_of[2 * kMaxSub + 2];
  __shared__ int wsum[kTailThreads / 64];
  __shared__ int sh_nact;
  const int pid = blockIdx.y, side = pid / C.BH, bh = pid % C.BH, node = blockIdx.x;
  const Side& S = C.s[side];
  if (node >= (1 << S.big)) return;
  int start, size;
  node_range(S.n, S.c, S.big, node, &start, &size);
  const int par = side == 0 ? parity0 : parity1;
  const bool identity = S.big == 0;
  const int32_t* src = (par ? C.idx1 : C.idx0) + (size_t)pid * C.nmax;
  for (int o = threadIdx.x; o < size; o += kTailThreads) ia[o] = identity ? start + o : src[start + o];
  const float* Y = S.y + (size_t)bh * S.n * C.d;
  const int d = C.d, c = S.c;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int32_t* cur = ia;
  int32_t* nxt = ib;
  const int nsub_levels = S.levels - S.big;
  for (int r = 0; r < nsub_levels; ++r) {
    const int nslots = 1 << r;
    __syncthreads();
    if (threadIdx.x < 64) {
      // Sub-node ranges at this level (relative to the node), one lane per
      // slot (at most tail / c <= 64 slots), and the active list.
      const int sl = threadIdx.x;
      int st = 0, s = size;
      if (sl < nslots) {
        for (int b = r - 1; b >= 0; --b) {
          const int bit = (sl >> b) & 1;
          const int mL = s > c ? left_size(s, c) : s;
          if (bit) {
            st += mL;
            s -= mL;
          } else {
            s = mL;
          }
        }
      }
      const bool act = sl < nslots && s > c;
      const uint64_t am = __ballot(act);
      if (sl < nslots) {
        const int rank = (int)__popcll(am & ((1ull << sl) - 1ull));
        sub_start[sl] = st;
        sub_size[sl] = s;
        act_of[sl] = act ? rank : -1;
        if (act) act_list[rank] = sl;
      }
      if (sl == 0) {
        sub_start[nslots] = size;
        sh_nact = (int)__popcll(am);
      }
    }
    __syncthreads();
    const int nact = sh_nact;
    if (nact == 0) break;
    // coordinate choice: one wavefront per active sub-node
    for (int a = w; a < nact; a += kTailThreads / 64) {
      const int sl = act_list[a];
      const int js = choose_coordinate<64>(Y, d, cur, false, sub_start[sl], sub_size[sl], lane);
      if (lane == 0) {
        sub_js[sl] = js;
        sub_thr[sl] = 0;
        sub_rank[sl] = left_size(sub_size[sl], c) - 1;
      }
    }
    __syncthreads();
    // keys; slot of position o by binary search over the sub-node starts
    {
      constexpr int PT = kTail / kTailThreads;
      int gsl[PT], grow[PT];
#pragma unroll
      for (int u = 0; u < PT; ++u) {
        const int o = threadIdx.x + kTailThreads * u;
        // The last slot starting at or before o is the non-empty slot holding
        // o: empty slots start where the next non-empty slot starts.
        int lo = 0, hi = nslots - 1;
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (sub_start[mid] <= o)
            lo = mid;
          else
            hi = mid - 1;
        }
        gsl[u] = lo;
        grow[u] = o < size && act_of[lo] >= 0 ? cur[o] : -1;
      }
      // the chosen coordinate, from the coordinate-major copy when it holds
      // it (the nodes of a head run together, so they share its lines)
      float gv[PT];
#pragma unroll
      for (int u = 0; u < PT; ++u) {
        gv[u] = 0.f;
        if (grow[u] >= 0) {
          const int js = sub_js[gsl[u]];
          gv[u] = S.ycol && js < kColCopy ? S.ycol[((size_t)bh * kColCopy + js) * S.n + grow[u]]
                                          : Y[(size_t)grow[u] * d + js];
        }
      }
#pragma unroll
      for (int u = 0; u < PT; ++u) {
        const int o = threadIdx.x + kTailThreads * u;
        if (o < size) {
          scan[o] = gsl[u];  // slot id (temporarily)
          keys[o] = grow[u] >= 0 ? ordered_bits(gv[u]) : 0u;
        }
      }
    }
    // four 8-bit digit passes
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      const int mshift = shift + 8;
      __syncthreads();
      for (int e = threadIdx.x; e < nact * 256; e += kTailThreads) hist[e / 256][e % 256] = 0;
      __syncthreads();
      for (int o = threadIdx.x; o < size; o += kTailThreads) {
        const int sl = scan[o], a = act_of[sl];
        if (a < 0) continue;
        const uint32_t key = keys[o];
        const uint32_t pre = (uint32_t)sub_thr[sl];
        if (mshift == 32 || (key >> mshift) == (pre >> mshift))
          atomicAdd(&hist[a][(key >> shift) & 255], 1);
      }
      __syncthreads();
      for (int a = w; a < nact; a += kTailThreads / 64) {
        const int sl = act_list[a];
        const int rank = sub_rank[sl];
        int cnt[4], sum = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          cnt[i] = hist[a][4 * lane + i];
          sum += cnt[i];
        }
        int incl = sum;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_up(incl, o, 64);
          if (lane >= o) incl += y;
        }
        const int before = incl - sum;
        if (rank >= before && rank < incl) {
          int acc = before;
          for (int i = 0; i < 4; ++i) {
            if (rank < acc + cnt[i]) {
              sub_thr[sl] = (int)((uint32_t)sub_thr[sl] | ((uint32_t)(4 * lane + i) << shift));
              sub_rank[sl] = rank - acc;
              break;
            }
            acc += cnt[i];
          }
        }
      }
    }
    __syncthreads();
    // stable partition: scan of packed (less, equal) counts in position order
    constexpr int per = kTail / kTailThreads;
    const int o0 = threadIdx.x * per;
    int less = 0, eq = 0;
    for (int o = o0; o < o0 + per && o < size; ++o) {
      const int sl = scan[o];
      if (act_of[sl] < 0) continue;
      const uint32_t thr = (uint32_t)sub_thr[sl];
      less += keys[o] < thr;
      eq += keys[o] == thr;
    }
    const int packed0 = scan_tail((less << 16) | eq, wsum);
    // exclusive prefix at every position (packed), then per-sub-node offsets
    int run = packed0;
    int slots_local[per];
    for (int u = 0; u < per; ++u) {
      const int o = o0 + u;
      if (o >= size) break;
      const int sl = scan[o];
      slots_local[u] = sl;
      const uint32_t thr = (uint32_t)sub_thr[sl];
      const bool act = act_of[sl] >= 0;
      const int inc = act ? (((keys[o] < thr) ? 1 : 0) << 16) | ((keys[o] == thr) ? 1 : 0) : 0;
      scan[o] = run;  // overwrite slot id by the exclusive prefix
      run += inc;
    }
    __syncthreads();
    int newpos[per];
    for (int u = 0; u < per; ++u) {
      const int o = o0 + u;
      if (o >= size) break;
      const int sl = slots_local[u];
      const int st = sub_start[sl];
      if (act_of[sl] < 0) {
        newpos[u] = o;
        continue;
      }
      const int base = scan[st];
      const int rel = scan[o] - base;
      const int lb = rel >> 16, eb = rel & 0xFFFF;
      const uint32_t thr = (uint32_t)sub_thr[sl];
      const int need_eq = sub_rank[sl] + 1;
      const int mL = left_size(sub_size[sl], c);
      const int Lo = lb + min(eb, need_eq);
      const bool left = keys[o] < thr || (keys[o] == thr && eb < need_eq);
      const int rel_dst = left ? Lo : mL + (o - st - Lo);
      newpos[u] = (rel_dst >= 0 && rel_dst < sub_size[sl]) ? st + rel_dst : -1;
    }
    __syncthreads();
    for (int u = 0; u < per; ++u) {
      const int o = o0 + u;
      if (o >= size) break;
      if (newpos[u] >= 0) nxt[newpos[u]] = cur[o];
    }
    int32_t* t = cur;
    cur = nxt;
    nxt = t;
  }
  __syncthreads();
  int32_t* perm = S.perm + (size_t)bh * S.n;
  for (int o = threadIdx.x; o < size; o += kTailThreads) perm[start + o] = cur[o];
}

// ---------------------------------------------------------------------------
// Gather: permuted copies (pad rows zero), centroids of the original vectors,
// counts, cluster ids. Values follow the key permutation and are stored per
// key cluster as a d x c tile (dimension-major), which is the operand layout
// of the value product in the attention kernels.
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(128) void gather_kernel(Ctx C) {
  extern __shared__ __attribute__((aligned(16))) float gsh[];  // value tile staging [c][d]
  const int pid = blockIdx.y, side = pid / C.BH, bh = pid % C.BH, a = blockIdx.x;
  const Side& S = C.s[side];
  if (a >= S.nc) return;
  const int d = C.d, c = S.c, t = threadIdx.x;
  const int cnt = min(c, S.n - a * c);
  const int32_t* perm = S.perm + (size_t)bh * S.n + (size_t)a * c;
  if (t == 0) S.count[(size_t)bh * S.nc + a] = cnt;
  if (S.cid)
    for (int r = t; r < cnt; r += 128) S.cid[(size_t)bh * S.n + perm[r]] = a;
  const size_t xrow0 = ((size_t)bh * S.npad + (size_t)a * c) * d;
  const bool vals = side == 1 && C.v != nullptr;
  for (int tt = t; tt < d; tt += 128) {
    float s = 0.f, sv = 0.f;
    for (int r = 0; r < c; ++r) {
      float x = 0.f, xv = 0.f;
      if (r < cnt) {
        const int i = perm[r];
        x = load_x(S.x, bh, i, S.lx, tt, C.dtype);
        s += x;
        if (vals) {
          xv = load_x(C.v, bh, i, C.lv, tt, C.dtype);
          sv += xv;
        }
      }
      store_elem(S.xp, xrow0 + (size_t)r * d + tt, C.dtype, x);
      if (vals) gsh[r * d + tt] = xv;
    }
    S.cent[((size_t)bh * S.nc + a) * d + tt] = s / (float)cnt;
    if (vals) C.cent_v[((size_t)bh * S.nc + a) * d + tt] = sv / (float)cnt;
  }
  if (vals) {
    __syncthreads();
    const size_t vt0 = ((size_t)bh * S.nc + a) * (size_t)d * c;
    for (int e = t; e < d * c; e += 128) {
      const int dd = e / c, r = e % c;
      store_elem(C.vp, vt0 + e, C.dtype, gsh[r * d + dd]);
    }
  }
}

// Fast gather for rows that are a whole number of 16-byte chunks: one
// workgroup per cluster copies the cluster's rows chunk by chunk (coalesced
// on both sides), sums the centroids in registers and then across the
// workgroup in a fixed order (deterministic), and transposes the value rows
// through LDS so that the value tiles are written 16 bytes at a time.
template <typename T>
__global__ __launch_bounds__(256) void gather_fast_kernel(Ctx C) {
  extern __shared__ __attribute__((aligned(16))) float gfs[];
  constexpr int EPC = 16 / sizeof(T);  // elements per 16-byte chunk
  const int pid = blockIdx.y, side = pid / C.BH, bh = pid % C.BH, a = blockIdx.x;
  const Side& S = C.s[side];
  if (a >= S.nc) return;
  const int d = C.d, c = S.c, tid = threadIdx.x;
  const int cpr = d / EPC;        // chunks per row (divides 256: d <= 128)
  const int rstep = 256 / cpr;    // row stride of one thread
  const int col = tid % cpr, r0 = tid / cpr;
  const int cnt = min(c, S.n - a * c);
  const int32_t* perm = S.perm + (size_t)bh * S.n + (size_t)a * c;
  const bool vals = side == 1 && C.v != nullptr;
  float* part = gfs;                            // [rstep][d] partial sums of x
  float* partv = gfs + rstep * d;               // [rstep][d] partial sums of v
  T* vstage = (T*)(gfs + 2 * rstep * d);        // [c][d] value rows
  if (tid == 0) S.count[(size_t)bh * S.nc + a] = cnt;
  if (S.cid)
    for (int r = tid; r < cnt; r += 256) S.cid[(size_t)bh * S.n + perm[r]] = a;
  float acc[EPC], accv[EPC];
#pragma unroll
  for (int u = 0; u < EPC; ++u) acc[u] = accv[u] = 0.f;
  T* dst = (T*)S.xp + ((size_t)bh * S.npad + (size_t)a * c) * d;
  // A thread's rows r0, r0 + rstep, ... (at most kGatherRows of them): all
  // loads are issued before the first is used.
  constexpr int kGatherRows = 8;
  for (int rb = r0; rb < c; rb += kGatherRows * rstep) {
    uint4 chunk[kGatherRows], vchunk[kGatherRows];
#pragma unroll
    for (int u = 0; u < kGatherRows; ++u) {
      const int r = rb + u * rstep;
      chunk[u] = vchunk[u] = make_uint4(0u, 0u, 0u, 0u);
      if (r < cnt) {
        const int i = perm[r];
        chunk[u] = *(const uint4*)((const T*)S.x + row_off(bh, i, S.lx) + col * EPC);
        if (vals)
          vchunk[u] =
              *(const uint4*)((const T*)C.v + row_off(bh, i, C.lv) + col * EPC);
      }
    }
#pragma unroll
    for (int u = 0; u < kGatherRows; ++u) {
      const int r = rb + u * rstep;
      if (r >= c) break;
      *(uint4*)(dst + (size_t)r * d + col * EPC) = chunk[u];
      union {
        uint4 v;
        T e[EPC];
      } cx, cv;
      cx.v = chunk[u];
#pragma unroll
      for (int e = 0; e < EPC; ++e) acc[e] += (float)cx.e[e];
      if (vals) {
        *(uint4*)(vstage + r * d + col * EPC) = vchunk[u];
        cv.v = vchunk[u];
#pragma unroll
        for (int e = 0; e < EPC; ++e) accv[e] += (float)cv.e[e];
      }
    }
  }
#pragma unroll
  for (int u = 0; u < EPC; ++u) {
    part[r0 * d + col * EPC + u] = acc[u];
    if (vals) partv[r0 * d + col * EPC + u] = accv[u];
  }
  __syncthreads();
  for (int f = tid; f < d; f += 256) {
    float sx = 0.f, sv = 0.f;
    for (int g = 0; g < rstep; ++g) {
      sx += part[g * d + f];
      if (vals) sv += partv[g * d + f];
    }
    S.cent[((size_t)bh * S.nc + a) * d + f] = sx / (float)cnt;
    if (vals) C.cent_v[((size_t)bh * S.nc + a) * d + f] = sv / (float)cnt;
  }
  if (vals) {
    // value tile [d][c]: chunk = EPC consecutive rows of one dimension
    T* vt = (T*)C.vp + ((size_t)bh * S.nc + a) * (size_t)d * c;
    const int cpc = c / EPC;  // chunks per tile row (c >= EPC)
    for (int e = tid; e < d * cpc; e += 256) {
      const int f = e / cpc, rr = (e % cpc) * EPC;
      union {
        uint4 v;
        T e[EPC];
      } tmp;
#pragma unroll
      for (int u = 0; u < EPC; ++u) tmp.e[u] = vstage[(rr + u) * d + f];
      *(uint4*)(vt + (size_t)f * c + rr) = tmp.v;
    }
  }
}

int tail_size(int c) { return c * 64 < kTail ? c * 64 : kTail; }

}  // namespace

int split_level_cpn(const Prob& P, int big_q, int big_k, int l) {
  int maxs = 0;
  for (int side = 0; side < 2; ++side) {
    const int n = side == 0 ? P.nq : P.nk, c = side == 0 ? P.cq : P.ck;
    if (l >= (side == 0 ? big_q : big_k)) continue;
    for (int node = 0; node < (1 << l); ++node) {
      int st, s;
      node_range(n, c, l, node, &st, &s);
      if (s > maxs) maxs = s;
    }
  }
  return (maxs + kChunk - 1) / kChunk;
}

int split_hist_slots(const Prob& P, int big_q, int big_k) {
  const int big = big_q > big_k ? big_q : big_k;
  int slots = 1;
  for (int l = 0; l < big; ++l) {
    const int s = (1 << l) * split_level_cpn(P, big_q, big_k, l);
    if (s > slots) slots = s;
  }
  return slots;
}

int split_big_levels(int n, int c, int L) {
  const int tail = tail_size(c);
  int l = 0;
  while (l < L) {
    int maxs = 0;
    for (int node = 0; node < (1 << l); ++node) {
      int st, s;
      node_range(n, c, l, node, &st, &s);
      if (s > maxs) maxs = s;
    }
    if (maxs <= tail) break;
    ++l;
  }
  return l;
}

namespace {
// Kernels that use more than 64 KiB of dynamic LDS declare their size once. A
// refusal is not fatal here: the launch itself reports a real limit.
constexpr size_t kEighLds = eigh_lds_bytes(kMaxD);
constexpr size_t kCholLds = (size_t)kMaxD * kCP * sizeof(double);
constexpr size_t kQnormLds = (size_t)(kMaxD + 2 * kStage) * kDP * sizeof(float);
constexpr size_t kProjLds = (size_t)(kMaxD + kStage) * kDP * sizeof(float);
constexpr size_t kGatherLds = (size_t)kMaxC * kMaxD * sizeof(float);
hipError_t set_lds_limits() {
  static bool done = [] {
    (void)hipFuncSetAttribute((const void*)eigh_kernel<128>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)kEighLds);
    (void)hipFuncSetAttribute((const void*)eigh_kernel<64>,
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)eigh_lds_bytes(64));
    (void)hipFuncSetAttribute((const void*)cholesky_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                        (int)kCholLds);
    (void)hipFuncSetAttribute((const void*)qnorm_partial_kernel,
                        hipFuncAttributeMaxDynamicSharedMemorySize, (int)kQnormLds);
    (void)hipFuncSetAttribute((const void*)project_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                        (int)kProjLds);
    (void)hipFuncSetAttribute((const void*)gather_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                        (int)kGatherLds);
    for (const void* f : {(const void*)basic_choose_kernel<0>, (const void*)basic_choose_kernel<128>})
      (void)hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)((size_t)kMaxD * (kMaxD + 1) * sizeof(float)));
    (void)hipFuncSetAttribute((const void*)gather_fast_kernel<bf16>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    (void)hipFuncSetAttribute((const void*)gather_fast_kernel<float>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    (void)hipGetLastError();
    return true;
  }();
  (void)done;
  return hipSuccess;
}
}  // namespace

hipError_t launch_cluster(const Prob& P, const void* q, const void* k, const void* v,
                          const ca_cluster_out* out, char* ws, const Workspace& W,
                          hipStream_t st) {
  {
    hipError_t le = set_lds_limits();
    if (le != hipSuccess) return le;
  }
  Ctx C = {};
  const int d = P.d;
  C.BH = P.BH;
  C.H = P.H;
  C.d = d;
  C.dtype = P.dtype;
  C.lv = P.lv;
  C.xf = P.xf;
  C.nmax = P.nq > P.nk ? P.nq : P.nk;
  C.nblk = W.nblk_mom;
  C.mom_rows = W.mom_rows;
  C.proj_rows = kProjRows;  // set for the projection launch below
  C.v = v;
  C.cent_v = out->cent_v;
  C.vp = out->vp;
  C.mats = (float*)(ws + W.mats);
  C.vecs = (float*)(ws + W.vecs);
  C.inv_q = (float*)(ws + W.inv_q);
  C.mom_part = (float*)(ws + W.mom_part);
  C.qn_part = (float*)(ws + W.qn_part);
  C.wops = (bf16*)(ws + W.wops);
  C.idx0 = (int32_t*)(ws + W.idx0);
  C.idx1 = (int32_t*)(ws + W.idx1);
  C.keys = (uint32_t*)(ws + W.keys);
  C.node_state = (int32_t*)(ws + W.node_state);
  C.hist = (uint32_t*)(ws + W.hist);
  C.chunk_cnt = (int32_t*)(ws + W.chunk_cnt);
  C.max_nodes = W.max_big_nodes;
  C.hist_slots = W.hist_slots;
  C.split = P.split;
  C.dirs = (float*)(ws + W.dirs);
  const bool basic = P.split == CA_SPLIT_BASIC;
  Side& Sq = C.s[0];
  Side& Sk = C.s[1];
  Sq.x = q;
  Sk.x = k;
  Sq.lx = P.lq;
  Sk.lx = P.lk;
  if (P.lq.H < 1 || P.lk.H < 1 || P.lv.H < 1) return hipErrorInvalidValue;
  Sq.y = out->yq_dbg ? out->yq_dbg : (float*)(ws + W.y_q);
  Sk.y = out->yk_dbg ? out->yk_dbg : (float*)(ws + W.y_k);
  // coordinate-major leading coordinates, where a multi-block level reads them
  const bool cols = col_copy_used(P);
  Sq.ycol = cols && W.big_q > 0 ? (float*)(ws + W.ycol_q) : nullptr;
  Sk.ycol = cols && W.big_k > 0 ? (float*)(ws + W.ycol_k) : nullptr;
  Sq.perm = out->perm_q;
  Sk.perm = out->perm_k;
  Sq.cid = out->cid_q;
  Sk.cid = out->cid_k;
  Sq.count = out->count_q;
  Sk.count = out->count_k;
  Sq.cent = out->cent_q;
  Sk.cent = out->cent_k;
  Sq.xp = out->qp;
  Sk.xp = out->kp;
  Sq.n = P.nq;
  Sk.n = P.nk;
  Sq.c = P.cq;
  Sk.c = P.ck;
  Sq.nc = P.nqc;
  Sk.nc = P.nkc;
  Sq.npad = P.nq_pad;
  Sk.npad = P.nk_pad;
  Sq.levels = W.levels_q;
  Sk.levels = W.levels_k;
  Sq.big = W.big_q;
  Sk.big = W.big_k;
  Sq.tail = tail_size(P.cq);
  Sk.tail = tail_size(P.ck);
  const int BH = P.BH;
  hipError_t e;
#define CA_CHECK()                          \
  do {                                      \
    e = hipGetLastError();                  \
    if (e != hipSuccess) return e;          \
  } while (0)

  const bool mfma = P.dtype == CA_BF16 && (d == 64 || d == 128);
  const bool transformed = P.xf != CA_XF_NONE && P.xf != CA_XF_RANDOM;
  if (transformed) {
    if (mfma && d == 64)
      hipLaunchKernelGGL(moments_mfma_kernel<64>, dim3(C.nblk, 2 * BH), dim3(256), 0, st, C);
    else if (mfma)
      hipLaunchKernelGGL(moments_mfma_kernel<128>, dim3(C.nblk, 2 * BH), dim3(256), 0, st, C);
    else
      hipLaunchKernelGGL(moments_partial_kernel, dim3(C.nblk, 2 * BH), dim3(256), 0, st, C);
    CA_CHECK();
    const dim3 fgrid((d * d + d + 255) / 256, BH, 2);
    hipLaunchKernelGGL(moments_finish_kernel, fgrid, dim3(256), 0, st, C);
    CA_CHECK();
    const int wq = P.dtype == CA_BF16 ? (int)O_TQ : -1, wk = P.dtype == CA_BF16 ? (int)O_TK : -1;
    EighJobs J;
    if (P.xf == CA_XF_PCA) {
      // principal axes of the centred queries and keys, oriented by the means
      J.j[0] = {M_A0, -1, -1, 0, -1, V_MUQ, M_E0, V_L0, -1, M_TQ, wq};
      J.j[1] = {M_CK, -1, -1, 0, -1, V_MUK, M_EK, V_LK, -1, M_TK, wk};
    } else {
      hipLaunchKernelGGL(cholesky_kernel, dim3(BH, 2), dim3(kCholThreads), kCholLds, st, C,
                         (int)M_A0, (int)M_E0, (int)M_CK, (int)M_EK,
                         P.dtype == CA_BF16 ? (int)O_FK : -1);
      CA_CHECK();
      if (P.xf == CA_XF_METRIC) {
        const size_t qlds = kQnormLds;
        if (mfma && d == 64)
          hipLaunchKernelGGL(qnorm_mfma_kernel<64>, dim3(C.nblk, BH), dim3(256), 0, st, C);
        else if (mfma)
          hipLaunchKernelGGL(qnorm_mfma_kernel<128>, dim3(C.nblk, BH), dim3(256), 0, st, C);
        else
          hipLaunchKernelGGL(qnorm_partial_kernel, dim3(C.nblk, BH), dim3(256), qlds, st, C);
        CA_CHECK();
        hipLaunchKernelGGL(qnorm_finish_kernel, dim3((d * d + d + 255) / 256, BH), dim3(256), 0,
                           st, C);
        CA_CHECK();
      }
      // keys: C2 = S_q^T C_K S_q, oriented by S_q^T mu_K, T_K = S_q U2
      J.j[0] = {M_CK, M_E0, V_MUK, 0, V_KQ, -1, M_C2, V_L2, M_E0, M_TK, wk};
      if (P.xf == CA_XF_ADAPTIVE)
        // queries: cov(q S_k) = S_k^T (Q^T Q / n - mu_Q mu_Q^T) S_k, oriented by
        // S_k^T mu_Q (the mean of q S_k), W_Q = S_k U3; no normalisation
        J.j[1] = {M_A0, M_EK, V_MUQ, 1, -1, -1, M_C3, V_L3, M_EK, M_TQ, wq};
      else if (mfma)
        // queries: cov(r(q)), oriented by mu_r, W_Q = S_k U3
        J.j[1] = {M_C3, M_EK, V_MUR, 1, V_MUR, -1, M_C3, V_L3, M_EK, M_TQ, wq};
      else
        J.j[1] = {M_C3, -1, V_MUR, 1, -1, -1, M_C3, V_L3, M_EK, M_TQ, wq};
    }
    if (basic)  // the metric root space: the Cholesky factors are the projections
      hipLaunchKernelGGL(copy_roots_kernel, dim3(BH), dim3(256), 0, st, C, (int)mfma);
    else if (d <= 64)
      hipLaunchKernelGGL(eigh_kernel<64>, dim3(BH, 2), dim3(eigh_threads<64>()), eigh_lds_bytes(64), st, C, J);
    else
      hipLaunchKernelGGL(eigh_kernel<128>, dim3(BH, 2), dim3(eigh_threads<128>()), kEighLds, st, C, J);
    CA_CHECK();
  }
  {
    const int nmax = C.nmax;
    const size_t plds = kProjLds;
    // the MFMA pass takes 128 rows per step, the fp32 one 32
    C.proj_rows = rows_per_block(nmax, mfma && transformed ? 128 : 32, kProjRows, 2 * BH);
    const dim3 pgrid((nmax + C.proj_rows - 1) / C.proj_rows, 2 * BH);
    if (mfma && transformed && d == 64)
      hipLaunchKernelGGL(project_mfma_kernel<64>, pgrid, dim3(256), 0, st, C);
    else if (mfma && transformed)
      hipLaunchKernelGGL(project_mfma_kernel<128>, pgrid, dim3(256), 0, st, C);
    else
      hipLaunchKernelGGL(project_kernel, pgrid, dim3(256), plds, st, C);
    CA_CHECK();
  }
  const int big = W.big_q > W.big_k ? W.big_q : W.big_k;
  for (int l = 0; l < big; ++l) {
    LevelArgs L;
    L.level = l;
    L.first = l == 0;
    L.idx_in = (l & 1) ? C.idx1 : C.idx0;
    L.idx_out = (l & 1) ? C.idx0 : C.idx1;
    const int cpn = split_level_cpn(P, W.big_q, W.big_k, l);
    L.cpn = cpn;
    if (basic) {
      const size_t blds = (size_t)d * (d + 1) * sizeof(float);
      if (d == 64)
        hipLaunchKernelGGL(basic_choose64_kernel, dim3(1 << l, 2 * BH), dim3(64), 0, st, C, L);
      else if (d == 128)
        hipLaunchKernelGGL(basic_choose_kernel<128>, dim3(1 << l, 2 * BH), dim3(kBasicThreads),
                           blds, st, C, L);
      else
        hipLaunchKernelGGL(basic_choose_kernel<0>, dim3(1 << l, 2 * BH), dim3(kBasicThreads),
                           blds, st, C, L);
    }
    else
      hipLaunchKernelGGL(split_choose_kernel, dim3(1 << l, 2 * BH), dim3(64), 0, st, C, L);
    CA_CHECK();
    const dim3 kgrid(cpn, 1 << l, 2 * BH);
    if (!basic)
      hipLaunchKernelGGL(split_keys_kernel<-1>, kgrid, dim3(256), 0, st, C, L);
    else if (d == 64)
      hipLaunchKernelGGL(split_keys_kernel<64>, kgrid, dim3(256), 0, st, C, L);
    else if (d == 128)
      hipLaunchKernelGGL(split_keys_kernel<128>, kgrid, dim3(256), 0, st, C, L);
    else
      hipLaunchKernelGGL(split_keys_kernel<0>, kgrid, dim3(256), 0, st, C, L);
    CA_CHECK();
    hipLaunchKernelGGL(split_select_kernel, dim3(1 << l, 2 * BH), dim3(kSelThreads), 0, st, C, L);
    CA_CHECK();
    hipLaunchKernelGGL(split_scatter_kernel, dim3(cpn, 1 << l, 2 * BH), dim3(256), 0, st, C, L);
    CA_CHECK();
  }
  {
    // After its last multi-block level, side s holds its order in idx[(big_s) & 1].
    const int nodes = 1 << big;
    if (basic)
      hipLaunchKernelGGL(copy_order_kernel, dim3((C.nmax + 255) / 256 < 1024 ? (C.nmax + 255) / 256 : 1024, 2 * BH),
                         dim3(256), 0, st, C, W.big_q & 1, W.big_k & 1);
    else
      hipLaunchKernelGGL(split_tail_kernel, dim3(nodes, 2 * BH), dim3(kTailThreads), 0, st, C,
                         W.big_q & 1, W.big_k & 1);
    CA_CHECK();
  }
  {
    const int maxc = P.nqc > P.nkc ? P.nqc : P.nkc;
    const int epc = 16 / (int)P.esize;
    const bool fast = (d % epc == 0) && (P.ck % epc == 0) && ((256 / (d / epc)) * (d / epc) == 256);
    if (fast) {
      const int rstep = 256 / (d / epc);
      const size_t glds = (size_t)2 * rstep * d * sizeof(float) + (v ? (size_t)P.ck * d * P.esize : 0);
      if (P.dtype == CA_BF16)
        hipLaunchKernelGGL(gather_fast_kernel<bf16>, dim3(maxc, 2 * BH), dim3(256), glds, st, C);
      else
        hipLaunchKernelGGL(gather_fast_kernel<float>, dim3(maxc, 2 * BH), dim3(256), glds, st, C);
    } else {
      const size_t glds = v ? (size_t)P.ck * d * sizeof(float) : 0;
      hipLaunchKernelGGL(gather_kernel, dim3(maxc, 2 * BH), dim3(128), glds, st, C);
    }
    CA_CHECK();
  }
#undef CA_CHECK
  return hipSuccess;
}

// ---------------------------------------------------------------------------
// Checked mode: flag bits of the tensors holding a NaN or an infinity
// ---------------------------------------------------------------------------

namespace {

__global__ void flags_clear_kernel(int32_t* flags) { flags[0] = 0; }

// One block of 256 threads per 64 rows of one tensor (blockIdx.y: 0 q, 1 k,
// 2 v); a value is non-finite when its exponent bits are all ones.
__global__ __launch_bounds__(256) void check_finite_kernel(const void* q, const void* k,
                                                           const void* v, Lay lq, Lay lk, Lay lv,
                                                           int nq, int nk, int BH, int d,
                                                           int dtype, int32_t* flags) {
  const int t = blockIdx.y;
  const void* x = t == 0 ? q : (t == 1 ? k : v);
  const Lay& L = t == 0 ? lq : (t == 1 ? lk : lv);
  const int n = t == 0 ? nq : nk;
  const long long rows = (long long)BH * n;
  const long long r0 = (long long)blockIdx.x * 64;
  int bad = 0;
  if (x != nullptr) {
    for (int e = threadIdx.x; e < 64 * d; e += 256) {
      const long long r = r0 + e / d;
      if (r >= rows) break;
      const int bh = (int)(r / n), i = (int)(r % n), c = e % d;
      const size_t off = row_off(bh, i, L) + c;
      if (dtype == CA_BF16) {
        const uint16_t u = ((const uint16_t*)x)[off];
        bad |= (u & 0x7F80u) == 0x7F80u;
      } else {
        const uint32_t u = ((const uint32_t*)x)[off];
        bad |= (u & 0x7F800000u) == 0x7F800000u;
      }
    }
  }
  if (__syncthreads_or(bad) && threadIdx.x == 0) atomicOr(flags, 1 << t);
}

}  // namespace

hipError_t launch_check_finite(const Prob& P, const void* q, const void* k, const void* v,
                               int32_t* flags, hipStream_t st) {
  hipLaunchKernelGGL(flags_clear_kernel, dim3(1), dim3(1), 0, st, flags);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const long long rows = (long long)P.BH * (P.nq > P.nk ? P.nq : P.nk);
  const unsigned blocks = (unsigned)((rows + 63) / 64);
  hipLaunchKernelGGL(check_finite_kernel, dim3(blocks, v ? 3 : 2), dim3(256), 0, st, q, k, v,
                     P.lq, P.lk, P.lv, P.nq, P.nk, P.BH, P.d, P.dtype, flags);
  return hipGetLastError();
}

}  // namespace ca
