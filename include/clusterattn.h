/*
 * clusterattn.h - C ABI of the ClusterAttention hot path on MI355X (gfx950).
 *
 * ClusterAttention replaces bidirectional softmax attention, per head, by four
 * steps (paper: Method, Overview; Preliminaries, motivation for sparse
 * attention):
 *   1. ca_cluster            split queries and keys into clusters of a fixed
 *                            power-of-two size (Method: Clustering), and form
 *                            the permuted Q/K/V and the cluster centroids;
 *   2. ca_select             score every query cluster against every key
 *                            cluster by centroid dot products and keep the top-k
 *                            key clusters (Method: Cluster assignment);
 *   3. ca_block_sparse_attn  softmax attention of each query cluster onto the
 *                            keys of its selected clusters, returning the output
 *                            and the softmax denominator (Method: Overview);
 *   4. ca_compensate         striped mean-compensation: every skipped key
 *                            cluster enters through its centroid key and value
 *                            weighted by its size, merged with step 3, and the
 *                            rows restored to the original token order
 *                            (Preliminaries: error in sparse attention; App. A).
 * ca_attn_compensated computes steps 3 and 4 in one pass (bf16): the same
 * result without the intermediate op/lse arrays.
 *
 * Conventions shared by every call
 * --------------------------------
 * - All data pointers are DEVICE pointers (hipMalloc'd or equivalent) on the
 *   current HIP device. The caller owns every buffer; the library never
 *   allocates, frees or synchronises. Work is enqueued on `stream` (a
 *   hipStream_t; NULL = the default stream) and buffers must stay alive until
 *   the stream has passed it.
 * - Q/K/V and the final output use the problem's layout (ca_layout) with the
 *   last dimension contiguous. Every other array is dense, row-major, with the
 *   shape given in its comment; BH = batch * heads, heads vary fastest.
 * - Derived sizes: nqc = ceil(nq/cq), nkc = ceil(nk/ck), nq_pad = nqc*cq,
 *   nk_pad = nkc*ck. Clusters hold exactly cq (ck) tokens except the last one,
 *   which holds the remainder; its missing rows are zero-filled padding that
 *   never influences a result.
 * - Every call validates its arguments before touching the GPU. On any status
 *   other than CA_OK nothing has been enqueued. CA_E_DEVICE means a HIP launch
 *   error after validation; ca_last_error() then gives the HIP error text.
 *   No C++ exception crosses this interface.
 * - Every output element is written (including padding rows). Outputs must not
 *   alias inputs. Results are deterministic: two identical calls give
 *   bit-identical outputs.
 * - Non-finite inputs (NaN/Inf) are not checked by the steps: the calls stay
 *   memory-safe but the results are unspecified. Checked mode is the separate
 *   call ca_check_finite, which flags them on the device.
 * - Calls on different streams may run concurrently if their outputs and
 *   workspaces do not overlap.
 */
#ifndef CLUSTERATTN_H_
#define CLUSTERATTN_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CA_ABI_VERSION 8

#if defined(__GNUC__) || defined(__clang__)
#define CA_API __attribute__((visibility("default")))
#else
#define CA_API
#endif

typedef enum {
  CA_OK = 0,
  CA_E_INVALID = 1,     /* bad argument: null pointer, size out of range, c not a power of two, k not in [1, nkc] */
  CA_E_UNSUPPORTED = 2, /* valid but not built: e.g. bf16 attention with d not in {64, 128} */
  CA_E_WORKSPACE = 3,   /* workspace smaller than ca_workspace_size() */
  CA_E_DEVICE = 4,      /* HIP reported an error while enqueueing */
  CA_E_NONFINITE = 5    /* checked mode: an input holds NaN or Inf (reported by the caller's
                           read of ca_check_finite's flags; no call returns it itself, since
                           the library never synchronises) */
} ca_status;

typedef enum { CA_F32 = 0, CA_BF16 = 1 } ca_dtype;

/* Space in which the recursive split is done (Method: Transforms).
 *   CA_XF_NONE:   the raw coordinates.
 *   CA_XF_PCA:    principal coordinates of the raw vectors (diagonalized
 *                 splitting without the attention-aware metrics).
 *   CA_XF_METRIC: keys in the query-induced metric Q^T Q / n, queries through
 *                 r(q) = q S_k / |q S_k| with S_k S_k^T = the key covariance
 *                 (top-k representation, App. B.2), each side then on its own
 *                 principal coordinates. This is the evaluated method.
 *   CA_XF_ADAPTIVE: keys as CA_XF_METRIC; queries through the unnormalised
 *                 r(q) = q S_k (the metric K_c^T K_c / n of the centred keys,
 *                 Method: query clustering for adaptive assignment; App. B.1),
 *                 on its principal coordinates. For use with the adaptive
 *                 (attention-mass) selection of ca_select_hist.
 *   CA_XF_RANDOM: the random-cluster control (Experiments: baselines, random
 *                 clusters routed by centroid scores): tokens are split on
 *                 pseudo-random coordinates y[i][j] = (splitmix64 output
 *                 number c, top 24 bits) / 2^24 with c = (((2 bh + side) <<
 *                 22 | i) << 7) | j (bh = b * heads + h, side 0 queries / 1
 *                 keys; splitmix64 as published by S. Vigna, started at state
 *                 0), which partitions them into clusters at random. */
typedef enum {
  CA_XF_NONE = 0,
  CA_XF_PCA = 1,
  CA_XF_METRIC = 2,
  CA_XF_ADAPTIVE = 3,
  CA_XF_RANDOM = 4
} ca_transform;

/* Recursive split algorithm (Method: Recursive splitting).
 *   CA_SPLIT_DIAG:  diagonalized splitting (the evaluated method): at each node
 *                   the global principal coordinate of highest variance on a
 *                   subsample (see ca_cluster).
 *   CA_SPLIT_BASIC: basic splitting, a variation of principal direction
 *                   divisive partitioning: at each node the first principal
 *                   direction of the subsample's centred covariance by 8
 *                   power iterations, warm-started from the mean of the
 *                   parent's direction and random normal noise rescaled to its
 *                   norm; every member is projected on it and the split is
 *                   made on the projections. Supported with CA_XF_NONE and
 *                   CA_XF_METRIC (the metric root space without principal
 *                   axes: keys k S_q, queries q S_k / |q S_k|, no
 *                   eigendecomposition). Arithmetic (fp32, fixed order, no
 *                   fused multiply-add): mean mu = (sum of the m subsample
 *                   rows in order) / m; rows centred; per iteration t_j =
 *                   sum_k (x_jk - mu_k) v_k, w_k = sum_j t_j (x_jk - mu_k),
 *                   v = w / sqrt(sum_k w_k^2) (a zero w keeps v); start v0 =
 *                   noise at the root, else (v_p + r sqrt(|v_p|^2) /
 *                   sqrt(|r|^2)) / 2; projections sum_k y_ik v_k. Noise of
 *                   the node at slot s of level l of head bh, side (0 queries,
 *                   1 keys), coordinate k: (sum over u < 12 of the top 24 bits
 *                   of splitmix64 output 16 c + u) / 2^24 - 6 (fp64, rounded
 *                   once to fp32), c = ((((2 bh + side) << 5 | l) << 20 | s)
 *                   << 7) | k. */
typedef enum { CA_SPLIT_DIAG = 0, CA_SPLIT_BASIC = 1 } ca_split;

/* Layout of Q, K, V and the final output: BHND = [B][H][N][d],
 * BNHD = [B][N][H][d] (the usual activation layout of a transformer), both
 * dense; STRIDED = any element strides given in the problem (for instance
 * views of a fused QKV projection, [B][N][3][H][d], with the output in a
 * tensor of its own). In every layout the last dimension is contiguous. */
typedef enum { CA_LAYOUT_BHND = 0, CA_LAYOUT_BNHD = 1, CA_LAYOUT_STRIDED = 2 } ca_layout;

typedef struct {
  int32_t batch, heads;  /* >= 1 */
  int32_t nq, nk;        /* real query / key tokens per head, >= 1 */
  int32_t d;             /* head dimension, 1..128 (attention: see below) */
  int32_t cq, ck;        /* cluster sizes, powers of two in [1, 256] */
  int32_t dtype;         /* ca_dtype of Q/K/V, permuted copies and output */
  int32_t transform;     /* ca_transform (ca_cluster only) */
  int32_t layout;        /* ca_layout of Q/K/V/out */
  int32_t split;         /* ca_split (ca_cluster only) */
  /* CA_LAYOUT_STRIDED only (ignored by the dense layouts): element strides
   * {batch, head, token} of q, k, v and the output; element (b, h, i, t) of
   * q sits at q + b q_stride[0] + h q_stride[1] + i q_stride[2] + t. Each
   * stride is >= 0 and a multiple of 16 bytes' worth of elements (8 for
   * bf16, 4 for fp32), and the tensors' base pointers are 16-byte aligned,
   * so that rows can be read and written in 16-byte pieces. The output's
   * rows must not overlap one another or any input (not checked). */
  int64_t q_stride[3], k_stride[3], v_stride[3], out_stride[3];
} ca_problem;

/* Outputs of ca_cluster. Required unless marked optional. */
typedef struct {
  int32_t* perm_q;   /* [BH][nq]  original query index at each cluster-ordered position */
  int32_t* perm_k;   /* [BH][nk]  same for keys */
  int32_t* cid_q;    /* [BH][nq]  cluster of original query i (optional, may be NULL) */
  int32_t* cid_k;    /* [BH][nk]  cluster of original key i (optional, may be NULL) */
  int32_t* count_q;  /* [BH][nqc] real members per query cluster */
  int32_t* count_k;  /* [BH][nkc] real members per key cluster */
  float* cent_q;     /* [BH][nqc][d] fp32 mean of the ORIGINAL query vectors of each cluster */
  float* cent_k;     /* [BH][nkc][d] same for keys */
  float* cent_v;     /* [BH][nkc][d] same for values (values follow the key clusters);
                        optional: NULL (with v == NULL) skips values */
  void* qp;          /* [BH][nq_pad][d] dtype: queries in cluster order, pad rows zero */
  void* kp;          /* [BH][nk_pad][d] dtype: keys in cluster order, pad rows zero */
  void* vp;          /* [BH][nkc][d][ck] dtype: value tiles. For every key cluster the ck value
                        rows in cluster order, stored transposed (dimension-major, ck
                        contiguous), pad columns zero. This is the operand layout of the
                        value product in the attention calls. Optional: NULL with v. */
  float* yq_dbg;     /* [BH][nq][d] optional: the query split coordinates (original order) */
  float* yk_dbg;     /* [BH][nk][d] optional: the key split coordinates (original order) */
} ca_cluster_out;

/* ABI version compiled into the library (CA_ABI_VERSION). */
CA_API int ca_abi_version(void);

/* Static text for a status code. */
CA_API const char* ca_status_str(int status);

/* Detail of the last non-OK status returned on the calling thread ("" if none). */
CA_API const char* ca_last_error(void);

/* Bytes of workspace ca_cluster, ca_select and ca_compensate need for this
 * problem with k kept key clusters (k is only used for validation; the size
 * does not depend on it). Host-only; enqueues nothing. Workspace must be
 * 256-byte aligned. */
CA_API int ca_workspace_size(const ca_problem* p, int32_t k, size_t* bytes);

/* Step 1: clustering (Method: Clustering, Recursive splitting - diagonalized
 * variant; Transforms).
 *
 * Per head, queries and keys are each mapped to their split space (transform)
 * and recursively split: at a node of s > c tokens, a subsample of
 * m = min(d, s) members at positions floor((2j+1)s/(2m)) of the node (in
 * ascending original-index order) picks the coordinate of highest fp64
 * population variance (two-pass, sequential, ties to the lower coordinate);
 * the node's c*floor(ceil(s/c)/2) members with the smallest (coordinate value,
 * original index) go left, the rest right, both keeping index order; leaves
 * are numbered left to right. This is deterministic: given the split
 * coordinates (exported through yq_dbg / yk_dbg) the permutation is exact.
 *
 * q, k: [B,H,nq|nk,d] in the problem layout and dtype. v: same shape as k, or
 * NULL to skip the value outputs. ws: device workspace of ws_bytes >=
 * ca_workspace_size(). */
CA_API int ca_cluster(const ca_problem* p, const void* q, const void* k, const void* v,
               const ca_cluster_out* out, void* ws, size_t ws_bytes, void* stream);

/* Step 2: assignment (Method: Cluster assignment - scoring and top-k
 * selection). scores[a][b] = cent_q[a] . cent_k[b] (fp32, the mean pairwise
 * logit up to the 1/sqrt(d) factor; for bf16 problems with d = 64 or 128 and
 * 16-byte aligned centroids they are formed on the matrix cores from a
 * three-term bf16 split of the fp32 centroids, about 2^-16 relative per
 * product); lists[a] = the k key clusters with the largest scores, ties to
 * the lower index, in ascending order.
 *
 * cent_q: [BH][nqc][d], cent_k: [BH][nkc][d] fp32. scores_in: optional
 * [BH][nqc][nkc] fp32 scores to rank instead of computing them (NULL:
 * compute). scores_out: optional [BH][nqc][nkc] export of the ranked scores.
 * lists: [BH][nqc][k] int32 output. 1 <= k <= nkc. */
CA_API int ca_select(const ca_problem* p, const float* cent_q, const float* cent_k,
              const float* scores_in, float* scores_out, int32_t k, int32_t* lists,
              void* ws, size_t ws_bytes, void* stream);

/* Step 2, histogram variant (Method: Cluster assignment - selection, the
 * two-pass histogram). For query cluster a, with S = the centroid scores of
 * its row: a 16384-step grid over [min S, max S] (coarse bins of 128 steps,
 * each refined into 128), g_b = min(16383, floor((S_b - min S) * (16384 /
 * (max S - min S)))) in fp32; the estimated attention mass of key cluster b,
 * count_k[b] * exp(scale * (S_b - max S)), in fixed point (2^-32 units, fp64
 * arithmetic, exact integer sums); need = ceil(mass_recall * total mass).
 * The coarse histogram finds the highest coarse bin whose lower edge keeps
 * at least min_count clusters and at least `need` mass; its 128 fine bins
 * find the highest such edge G inside it; every b with g_b >= G is selected.
 * If all scores are equal, or min_count >= nkc, every cluster is selected.
 *   top-k through the histogram: min_count = k, mass_recall = 0 (at least k
 *   clusters: the ties inside the edge's fine bin are kept);
 *   adaptive assignment: min_count = 16, mass_recall in (0, 1].
 *
 * cent_q, cent_k, scores_in, scores_out: as ca_select. count_k: [BH][nkc].
 * min_count >= 1; mass_recall in [0, 1]; scale <= 0 selects 1/sqrt(d).
 * lists: [BH][nqc][nkc] int32 output, lens[a] ascending cluster indices in
 * row a (the rest of the row is not written); lens: [BH][nqc] int32 output,
 * each in [1, nkc]. Pass lists with list stride k = nkc and lens to the
 * attention and compensation calls. ws: as ca_select. */
CA_API int ca_select_hist(const ca_problem* p, const float* cent_q, const float* cent_k,
                   const int32_t* count_k, const float* scores_in, float* scores_out,
                   int32_t min_count, float mass_recall, float scale, int32_t* lists,
                   int32_t* lens, void* ws, size_t ws_bytes, void* stream);

/* Step 3: block-sparse attention (Method: Overview - attention over the
 * selected clusters, returning the softmax denominator).
 *
 * For query row p of cluster a (permuted order), over the real keys j of the
 * clusters in lists[a]:  s_j = scale * qp[p] . kp[j],
 *   op[p]  = sum_j e^{s_j - m} vp[j] / sum_j e^{s_j - m},
 *   lse[p] = m + ln sum_j e^{s_j - m}   (natural log; m = max_j s_j).
 * Key rows past count_k[b] in a cluster are padding and are excluded.
 *
 * qp: [BH][nq_pad][d], kp: [BH][nk_pad][d], vp: [BH][nkc][d][ck] value tiles
 * as written by ca_cluster (all dtype), count_k: [BH][nkc], each in [1, ck],
 * lists: [BH][nqc][k] with entries in [0, nkc) (not checked on the device;
 * out-of-range entries are clamped), lens: optional [BH][nqc] list lengths
 * (NULL: every list has k entries; otherwise row a uses its first lens[a]
 * entries, clamped to [1, k] on the device), op: [BH][nq_pad][d] dtype, lse:
 * [BH][nq_pad] fp32. scale <= 0 selects 1/sqrt(d). Padding query rows get
 * defined values that callers ignore. bf16: d in {64, 128}, cq and ck in
 * {64, 128}; fp32: d % 4 == 0, any cq, ck.
 *
 * ws: optional device workspace of ws_bytes >= ca_workspace_size(). With
 * lens given (lists of different lengths) the bf16 path uses it to schedule
 * the query clusters: they are cut into eight contiguous ranges of about
 * equal work, one per XCD, and each range runs longest list first. With ws
 * NULL (ws_bytes 0) the query clusters run in index order. The results are
 * the same either way: only the order in which workgroups start changes. */
CA_API int ca_block_sparse_attn(const ca_problem* p, const void* qp, const void* kp, const void* vp,
                         const int32_t* count_k, const int32_t* lists, const int32_t* lens,
                         int32_t k, float scale, void* op, float* lse, void* ws,
                         size_t ws_bytes, void* stream);

/* Step 4: striped mean-compensation and un-permutation (Preliminaries: error
 * in sparse attention; App. A).
 *
 * For query row p of cluster a: every key cluster b NOT in lists[a] adds the
 * logit t_b = scale * qp[p] . cent_k[b] + ln count_k[b] with value cent_v[b];
 *   lse_c = ln sum_b e^{t_b},  o_c = sum_b e^{t_b - lse_c} cent_v[b],
 *   lse   = ln(e^{lse[p]} + e^{lse_c}),
 *   out   = e^{lse[p] - lse} op[p] + e^{lse_c - lse} o_c,
 * written to out[perm_q[p]] (original token order, problem layout). With
 * enable == 0, or when every cluster is selected, out = op[p], lse = lse[p].
 *
 * qp, op: [BH][nq_pad][d] dtype; cent_k, cent_v: [BH][nkc][d] fp32; count_k:
 * [BH][nkc]; lists: [BH][nqc][k], lens: optional list lengths as in
 * ca_block_sparse_attn; lse: [BH][nq_pad] fp32; perm_q: [BH][nq];
 * out: [B,H,nq,d] in the problem layout and dtype; lse_out: optional
 * [BH][nq] fp32 in original order. ws: device workspace of ws_bytes >=
 * ca_workspace_size(), where the bf16 path stages the centroids as bf16
 * tiles; required only for bf16 with enable != 0 and either k < nkc or lens
 * given (otherwise it may be NULL with ws_bytes 0). Compensation keeps a
 * selection bitmap of the key clusters per query cluster: with enable != 0
 * and either k < nkc or lens given, more than 65536 key clusters return
 * CA_E_UNSUPPORTED (enable == 0, or every cluster kept, has no such limit). */
CA_API int ca_compensate(const ca_problem* p, const void* qp, const float* cent_k, const float* cent_v,
                  const int32_t* count_k, const int32_t* lists, const int32_t* lens, int32_t k,
                  float scale,
                  int32_t enable, const void* op, const float* lse, const int32_t* perm_q,
                  void* out, float* lse_out, void* ws, size_t ws_bytes, void* stream);

/* Steps 3 and 4 in one pass (bf16 problems; Method: Overview; Preliminaries:
 * error in sparse attention; App. A).
 *
 * The result of ca_block_sparse_attn followed by ca_compensate on the same
 * arguments, up to rounding: each query cluster runs one online softmax over
 * the keys of its selected clusters and then over the centroid keys of the
 * unselected clusters, the logit of centroid b being
 * scale * qp[p] . cent_k[b] + ln count_k[b]. Combining the two parts inside
 * one softmax gives the merged output and lse directly (ln of the sum of both
 * parts' exponentials), so op and lse are never formed or rounded, and the
 * rows go straight to out[perm_q[p]].
 *
 * Arguments as in ca_block_sparse_attn (qp, kp, vp, count_k, lists, lens, k,
 * scale) and ca_compensate (cent_k, cent_v, enable, perm_q, out, lse_out).
 * ws: device workspace of ws_bytes >= ca_workspace_size(); required when
 * enable != 0 and either k < nkc or lens is given (the centroids are staged
 * there as bf16 tiles) and used for the launch schedule when lens is given;
 * otherwise it may be NULL with ws_bytes 0. Returns CA_E_UNSUPPORTED for fp32
 * problems and for more than 65536 key clusters. */
CA_API int ca_attn_compensated(const ca_problem* p, const void* qp, const void* kp, const void* vp,
                               const float* cent_k, const float* cent_v, const int32_t* count_k,
                               const int32_t* lists, const int32_t* lens, int32_t k, float scale,
                               int32_t enable, const int32_t* perm_q, void* out, float* lse_out,
                               void* ws, size_t ws_bytes, void* stream);

/* Checked mode (the method is defined for finite query, key and value
 * vectors; Method: Overview). Scans q, k and v (v may be NULL) in the
 * problem's layout and writes flags[0] on the stream: bit 0 if q holds a NaN
 * or an infinity, bit 1 for k, bit 2 for v; 0 when all are finite. flags: one
 * device int32, cleared by this call before the scan (no memset is
 * recorded); read it once the stream has passed the call, and treat a
 * non-zero value as CA_E_NONFINITE. Reads each input once (an HBM pass over
 * q, k and v). */
CA_API int ca_check_finite(const ca_problem* p, const void* q, const void* k, const void* v,
                           int32_t* flags, void* stream);

/* ca_attn_compensated without a workspace, for callers that cannot allocate
 * device memory: code under HIP graph capture, serving loops and harnesses
 * that forbid allocation. Same arguments and result as ca_attn_compensated
 * (bit for bit; the same kernels run), minus ws and ws_bytes.
 *
 * The centroid tiles (compensation with unselected clusters:
 * BH * ceil(nkc/128) * 128 * (4 d + 4) bytes, rounded up to 256) and the
 * launch schedule (lens given: (16 + 8 * floor((5 * BH * nqc + 31) / 32)) * 4
 * bytes) go to a scratch array that the library holds on every device it
 * runs on: 32 MiB (33554432 bytes), part of the library's code object, kept
 * until the process ends. Returns CA_E_WORKSPACE, with nothing enqueued,
 * when a problem needs more; ca_attn_compensated with a workspace has no
 * such limit. This call allocates nothing: no hipMalloc and no allocating
 * library routine (the array's device address is looked up once per device,
 * on the first call with that device current).
 *
 * All calls on one device share that device's array, which keeps the last
 * call's contents. Calls that overlap in time on one device (on different
 * streams, or from host threads without ordering between them) race and give
 * wrong results; calls ordered on one stream are safe. */
CA_API int ca_attn_compensated_noalloc(const ca_problem* p, const void* qp, const void* kp,
                                       const void* vp, const float* cent_k, const float* cent_v,
                                       const int32_t* count_k, const int32_t* lists,
                                       const int32_t* lens, int32_t k, float scale,
                                       int32_t enable, const int32_t* perm_q, void* out,
                                       float* lse_out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CLUSTERATTN_H_ */
