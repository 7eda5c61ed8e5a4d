// Internal declarations shared by the HIP translation units of libclusterattn.
// Not part of the public ABI (see include/clusterattn.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/clusterattn.h"

namespace ca {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;

constexpr int kMaxD = 128;
constexpr int kMaxC = 256;

// ---- scalar conversions -------------------------------------------------

__device__ __forceinline__ float bf2f(bf16 x) {
  return __uint_as_float(((uint32_t)__builtin_bit_cast(uint16_t, x)) << 16);
}
// Round to nearest even (the hardware conversion, v_cvt_pk_bf16_f32).
__device__ __forceinline__ bf16 f2bf(float f) { return (bf16)f; }
__device__ __forceinline__ float load_elem(const void* base, size_t idx, int dtype) {
  return dtype == CA_BF16 ? bf2f(((const bf16*)base)[idx]) : ((const float*)base)[idx];
}
__device__ __forceinline__ void store_elem(void* base, size_t idx, int dtype, float v) {
  if (dtype == CA_BF16)
    ((bf16*)base)[idx] = f2bf(v);
  else
    ((float*)base)[idx] = v;
}

// Order-preserving map of a float to uint32 (ascending float -> ascending
// unsigned); -0.0 is first turned into +0.0 so that the two compare equal.
__device__ __forceinline__ uint32_t ordered_bits(float f) {
  uint32_t u = __float_as_uint(f + 0.0f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// ---- problem description ---------------------------------------------------

// Element strides of a [B][H][N][d] tensor whose last dimension is
// contiguous: (batch b, head h, token i, dim 0) sits at b sb + h sh + i sn.
struct Lay {
  int64_t sb, sh, sn;
  int H;
};

// Element offset of (bh = b H + h, token i, dim 0).
__host__ __device__ __forceinline__ size_t row_off(int bh, int i, const Lay& L) {
  const int b = bh / L.H, h = bh - b * L.H;
  return (size_t)((int64_t)b * L.sb + (int64_t)h * L.sh + (int64_t)i * L.sn);
}

struct Prob {
  int B, H, BH, nq, nk, d, cq, ck, dtype, xf, layout, split;
  int nqc, nkc, nq_pad, nk_pad;
  size_t esize;
  Lay lq, lk, lv, lo;  // q, k, v and the output
};

// ---- the split tree -----------------------------------------------------------
// Node sizes depend only on (n, c): a node of s > c tokens sends
// c*floor(ceil(s/c)/2) tokens left and the rest right. A node of s <= c is a
// leaf and is carried down a level as (left = itself, right = empty), so level
// l has 2^l slots. Every node starts at a multiple of c.

__host__ __device__ __forceinline__ int left_size(int s, int c) {
  return c * (((s + c - 1) / c) / 2);
}
// Range [start, start+size) of slot `node` at level `lvl` of a tree over n tokens.
__host__ __device__ __forceinline__ void node_range(int n, int c, int lvl, int node, int* start,
                                                     int* size) {
  int st = 0, s = n;
  for (int b = lvl - 1; b >= 0; --b) {
    int bit = (node >> b) & 1;
    int mL = s > c ? left_size(s, c) : s;
    if (bit) {
      st += mL;
      s -= mL;
    } else {
      s = mL;
    }
  }
  *start = st;
  *size = s;
}
inline int num_levels(int n, int c) {
  int nc = (n + c - 1) / c, L = 0;
  while ((1 << L) < nc) ++L;
  return L;
}

// ---- workspace layout ---------------------------------------------------------

struct Workspace {
  // clustering
  size_t y_q, y_k;          // fp32 [BH][n][d] split coordinates (unless exported)
  size_t ycol_q, ycol_k;    // fp32 [BH][kColCopy][n] their first coordinates, coordinate-major
  size_t idx0, idx1, keys;  // int32 / uint32 [2][BH][nmax]
  size_t mom_part;          // fp32 [2][BH][nblk][d*d + d]
  size_t mats;              // fp32 [BH][kMats][d][d]
  size_t vecs;              // fp32 [BH][kVecs][d]
  size_t inv_q;             // fp32 [BH][nq]
  size_t qn_part;           // fp32 [BH][nblk_q][d*d + d]
  size_t wops;              // bf16 [BH][3][2][d][d] MFMA operands (transposed hi/lo)
  size_t node_state;        // int32 [2][BH][max_big_nodes][kNodeInts]
  size_t hist;              // uint32 [2][BH][hist_slots][kBins] chunk histograms
  size_t chunk_cnt;         // int32 [2][BH][hist_slots][2] chunk prefixes (less, equal)
  size_t dirs;              // fp32 [2 levels][2][BH][max_big_nodes][d] split directions (basic)
  // selection
  size_t scores;            // fp32 [BH][nqc][nkc]
  // attention schedule of lists with lengths
  size_t sched;             // int32 [8 + 8 * attn_sched_cap(BH * nqc)]
  // compensation
  size_t comp_tiles;        // bf16 centroid tiles [BH][ceil(nkc/kCompTile)][comp_tile_bytes]
  size_t total;
  // derived split parameters
  int nblk_mom;             // row blocks per tensor for moment partials
  int mom_rows;             // rows per moment-partial block
  int levels_q, levels_k;   // split levels per side
  int big_q, big_k;         // levels done by the multi-block kernels
  int max_big_nodes;        // nodes at the deepest multi-block level
  int hist_slots;           // chunk slots of the busiest multi-block level
};

// Leading split coordinates also kept coordinate-major (one contiguous column
// per coordinate), from which the multi-block keys pass reads a node's chosen
// coordinate: the upper levels choose among the leading principal coordinates.
constexpr int kColCopy = 16;
// The column copy exists for bf16 problems with d = 64 or 128 in a transformed
// space (the MFMA projection writes it) and diagonalized splitting.
inline bool col_copy_used(const Prob& P) {
  return P.dtype == CA_BF16 && (P.d == 64 || P.d == 128) && P.xf != CA_XF_NONE &&
         P.xf != CA_XF_RANDOM && P.split == CA_SPLIT_DIAG;
}
constexpr int kMats = 8;
constexpr int kVecs = 8;
constexpr int kNodeInts = 16;
constexpr int kBins = 4096;       // linear bins of the multi-block split select
constexpr int kChunk = 4096;      // tokens per block in the multi-block split passes
constexpr int kTail = 2048;       // nodes of at most this size finish in one workgroup
constexpr int kMomRows = 4096;    // rows per moment-partial block (at most)
constexpr int kCompTile = 128;    // centroids per tile of the bf16 compensation kernel
constexpr int kMaskWords = 2048;  // selection bitmap words in LDS: up to 65536 key clusters

// Rows per block of a pass over the rows of `tensors` tensors of n rows, one
// workgroup per block: cap, or fewer (in multiples of gran, the rows the pass
// takes per step) where the launch would otherwise have fewer than 512
// workgroups, two per CU. Each block is one workgroup's serial loop over its
// rows, so a short sequence in a few blocks is latency-bound, while more
// blocks than that only add per-block work (the moment passes' partials).
inline int rows_per_block(int n, int gran, int cap, int tensors) {
  const int want = (512 + tensors - 1) / tensors;  // blocks per tensor
  int r = (n + want - 1) / want;
  r = (r + gran - 1) / gran * gran;
  return r < cap ? r : cap;
}
// moment partials: 128 rows per step for the MFMA passes, 32 for the fp32 ones
inline int moment_rows(int nmax, int dtype, int tensors) {
  return rows_per_block(nmax, dtype == CA_BF16 ? 128 : 32, kMomRows, tensors);
}

// Bytes of one bf16 compensation tile: kCompTile centroid key rows [kCompTile][d]
// bf16, the centroid values transposed [d][kCompTile] bf16, and kCompTile fp32
// biases (log2 of the cluster size).
inline size_t comp_tile_bytes(int d) { return (size_t)kCompTile * (4 * d + 4); }

void plan_workspace(const Prob& P, Workspace* W);
// Number of split levels done by the multi-block kernels (nodes above the tail size).
int split_big_levels(int n, int c, int levels);
// Chunk blocks per node at multi-block level l (largest node of either side
// still split by the multi-block kernels there), and the most chunk slots any
// multi-block level needs.
int split_level_cpn(const Prob& P, int big_q, int big_k, int l);
int split_hist_slots(const Prob& P, int big_q, int big_k);

// ---- launchers (return hipError_t of the last launch) ----------------------

// Checked mode: flags[0] = bit 0 (q), 1 (k), 2 (v, if given) for a tensor
// holding a NaN or an infinity; cleared first on the stream.
hipError_t launch_check_finite(const Prob& P, const void* q, const void* k, const void* v,
                               int32_t* flags, hipStream_t st);
hipError_t launch_cluster(const Prob& P, const void* q, const void* k, const void* v,
                          const ca_cluster_out* out, char* ws, const Workspace& W,
                          hipStream_t st);
hipError_t launch_select(const Prob& P, const float* cq, const float* ck, const float* scores_in,
                         float* scores, int k, int32_t* lists, hipStream_t st);
hipError_t launch_select_hist(const Prob& P, const float* cq, const float* ck,
                              const int32_t* count_k, const float* scores_in, float* scores,
                              int min_count, float recall, float scale, int32_t* lists,
                              int32_t* lens, hipStream_t st);
// lens (optional): per query cluster list lengths, clamped to [1, k] on the device.
// Items per XCD of the attention schedule: about 1.25 times the mean, so a
// range of short lists can take more items than one of long lists.
inline int attn_sched_cap(int items) { return (5 * items + 31) / 32 + 1; }
// sched: workspace region of the schedule (bf16 with lens; else may be NULL).
hipError_t launch_attn(const Prob& P, const void* qp, const void* kp, const void* vp,
                       const int32_t* count_k, const int32_t* lists, const int32_t* lens, int k,
                       float scale, void* op, float* lse, int32_t* sched, hipStream_t st);
// tiles: workspace region of the bf16 centroid tiles (bf16 with compensation
// only; ignored otherwise).
hipError_t launch_comp(const Prob& P, const void* qp, const float* cent_k, const float* cent_v,
                       const int32_t* count_k, const int32_t* lists, const int32_t* lens, int k,
                       float scale,
                       int enable, const void* op, const float* lse, const int32_t* perm_q,
                       void* out, float* lse_out, char* tiles, hipStream_t st);

// Writes the bf16 centroid tiles (keys, transposed values, log2 sizes) of
// every head into tiles (bf16 problems).
hipError_t launch_comp_stage(const Prob& P, const float* cent_k, const float* cent_v,
                             const int32_t* count_k, char* tiles, hipStream_t st);
// Block-sparse attention with the striped mean compensation folded in (bf16):
// after its selected key clusters each query cluster continues the same
// online softmax over the unselected centroids (tiles: staged centroid tiles,
// or NULL for no compensation) and writes the merged rows to their original
// positions (out, problem layout) and lse_out (optional).
hipError_t launch_attn_fused(const Prob& P, const void* qp, const void* kp, const void* vp,
                             const int32_t* count_k, const int32_t* lists, const int32_t* lens,
                             int k, float scale, const char* tiles, const int32_t* perm_q,
                             void* out, float* lse_out, int32_t* sched, hipStream_t st);

}  // namespace ca
