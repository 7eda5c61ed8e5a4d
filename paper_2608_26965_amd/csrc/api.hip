// C ABI of libclusterattn: argument validation, workspace planning and dispatch.
// Every entry point validates completely before the first HIP call, so a
// non-OK status means nothing was enqueued.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "common.h"

// Device memory of ca_attn_compensated_noalloc: the staged centroid tiles and
// the launch schedule. Every device the library runs on holds its own copy,
// from the code object's load until the process ends. Host code never uses
// this name as an address: each device's address comes from
// hipGetSymbolAddress (scratch_on_current_device below).
static constexpr size_t kScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

thread_local char g_err[512] = "";

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return status;
}

int ok() {
  g_err[0] = '\0';
  return CA_OK;
}

int device_status(hipError_t e, const char* where) {
  if (e == hipSuccess) return ok();
  return fail(CA_E_DEVICE, "%s: %s", where, hipGetErrorString(e));
}

bool pow2(int x) { return x >= 1 && (x & (x - 1)) == 0; }

// Validates the problem descriptor and fills the derived sizes.
int check_problem(const ca_problem* p, ca::Prob* P) {
  if (!p) return fail(CA_E_INVALID, "problem is NULL");
  if (p->batch < 1 || p->heads < 1) return fail(CA_E_INVALID, "batch and heads must be >= 1");
  if (p->nq < 1 || p->nk < 1) return fail(CA_E_INVALID, "nq and nk must be >= 1");
  if ((int64_t)p->batch * p->heads > (1 << 20)) return fail(CA_E_INVALID, "batch*heads too large");
  if (p->nq > (1 << 22) || p->nk > (1 << 22)) return fail(CA_E_INVALID, "nq/nk above 2^22");
  if (p->d < 1 || p->d > ca::kMaxD) return fail(CA_E_INVALID, "d must be in [1, %d]", ca::kMaxD);
  if (!pow2(p->cq) || !pow2(p->ck) || p->cq > ca::kMaxC || p->ck > ca::kMaxC)
    return fail(CA_E_INVALID, "cluster sizes must be powers of two in [1, %d]", ca::kMaxC);
  if (p->dtype != CA_F32 && p->dtype != CA_BF16) return fail(CA_E_INVALID, "unknown dtype");
  if (p->transform < CA_XF_NONE || p->transform > CA_XF_RANDOM)
    return fail(CA_E_INVALID, "unknown transform");
  if (p->layout != CA_LAYOUT_BHND && p->layout != CA_LAYOUT_BNHD &&
      p->layout != CA_LAYOUT_STRIDED)
    return fail(CA_E_INVALID, "unknown layout");
  if (p->split != CA_SPLIT_DIAG && p->split != CA_SPLIT_BASIC)
    return fail(CA_E_INVALID, "unknown split");
  if (p->split == CA_SPLIT_BASIC && p->transform != CA_XF_NONE && p->transform != CA_XF_METRIC)
    return fail(CA_E_UNSUPPORTED, "basic splitting runs with CA_XF_NONE or CA_XF_METRIC");
  P->B = p->batch;
  P->H = p->heads;
  P->BH = p->batch * p->heads;
  P->nq = p->nq;
  P->nk = p->nk;
  P->d = p->d;
  P->cq = p->cq;
  P->ck = p->ck;
  P->dtype = p->dtype;
  P->xf = p->transform;
  P->layout = p->layout;
  P->split = p->split;
  P->nqc = (p->nq + p->cq - 1) / p->cq;
  P->nkc = (p->nk + p->ck - 1) / p->ck;
  P->nq_pad = P->nqc * p->cq;
  P->nk_pad = P->nkc * p->ck;
  P->esize = p->dtype == CA_BF16 ? 2 : 4;
  // element strides of q, k, v and the output
  auto dense = [&](int n) {
    ca::Lay L;
    L.H = p->heads;
    if (p->layout == CA_LAYOUT_BHND) {
      L.sn = p->d;
      L.sh = (int64_t)n * p->d;
      L.sb = (int64_t)p->heads * n * p->d;
    } else {
      L.sh = p->d;
      L.sn = (int64_t)p->heads * p->d;
      L.sb = (int64_t)n * p->heads * p->d;
    }
    return L;
  };
  if (p->layout == CA_LAYOUT_STRIDED) {
    const int64_t unit = 16 / (int64_t)P->esize;
    const int64_t* st[4] = {p->q_stride, p->k_stride, p->v_stride, p->out_stride};
    const char* nm[4] = {"q", "k", "v", "out"};
    ca::Lay* dst[4] = {&P->lq, &P->lk, &P->lv, &P->lo};
    for (int t = 0; t < 4; ++t) {
      for (int j = 0; j < 3; ++j)
        if (st[t][j] < 0 || st[t][j] % unit != 0)
          return fail(CA_E_INVALID,
                      "%s_stride[%d] = %lld: strides must be >= 0 and multiples of %lld elements",
                      nm[t], j, (long long)st[t][j], (long long)unit);
      dst[t]->sb = st[t][0];
      dst[t]->sh = st[t][1];
      dst[t]->sn = st[t][2];
      dst[t]->H = p->heads;
    }
  } else {
    P->lq = P->lo = dense(p->nq);
    P->lk = P->lv = dense(p->nk);
  }
  return CA_OK;
}

// The 16-byte alignment strided tensors need (the dense layouts keep their
// own row alignment).
int check_aligned(const ca::Prob& P, const void* x, const char* what) {
  if (P.layout == CA_LAYOUT_STRIDED && ((uintptr_t)x & 15u) != 0)
    return fail(CA_E_INVALID, "%s must be 16-byte aligned with CA_LAYOUT_STRIDED", what);
  return CA_OK;
}

int check_k(const ca::Prob& P, int32_t k) {
  if (k < 1 || k > P.nkc) return fail(CA_E_INVALID, "k=%d not in [1, nkc=%d]", k, P.nkc);
  return CA_OK;
}

int check_ws(const ca::Workspace& W, const void* ws, size_t ws_bytes) {
  if (ws_bytes < W.total)
    return fail(CA_E_WORKSPACE, "workspace of %zu bytes, need %zu", ws_bytes, W.total);
  if (W.total > 0 && !ws) return fail(CA_E_INVALID, "workspace is NULL");
  if (((uintptr_t)ws & 255u) != 0) return fail(CA_E_INVALID, "workspace must be 256-byte aligned");
  return CA_OK;
}

// The scratch array's address on the current device, looked up once per
// device with that device current and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

int scratch_on_current_device(char** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return device_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(CA_E_UNSUPPORTED, "device %d: scratch is kept for devices 0..%d", dev,
                kMaxDevices - 1);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return device_status(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(CA_E_DEVICE, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = (char*)p;
  }
  *out = g_scratch_ptr[dev];
  return CA_OK;
}

int check_attn_shape(const ca::Prob& P) {
  if (P.dtype == CA_BF16) {
    if (P.d != 64 && P.d != 128)
      return fail(CA_E_UNSUPPORTED, "bf16 attention needs d in {64, 128}, got %d", P.d);
    if ((P.cq != 64 && P.cq != 128) || (P.ck != 64 && P.ck != 128))
      return fail(CA_E_UNSUPPORTED, "bf16 attention needs cq, ck in {64, 128}");
  } else if (P.d % 4 != 0) {
    return fail(CA_E_UNSUPPORTED, "fp32 attention needs d %% 4 == 0, got %d", P.d);
  }
  return CA_OK;
}

}  // namespace

namespace ca {

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

void plan_workspace(const Prob& P, Workspace* W) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += align256(bytes);
    return o;
  };
  const size_t BH = P.BH, d = P.d;
  const int nmax = P.nq > P.nk ? P.nq : P.nk;
  W->mom_rows = moment_rows(nmax, P.dtype, 2 * P.BH);
  W->nblk_mom = (nmax + W->mom_rows - 1) / W->mom_rows;
  W->levels_q = num_levels(P.nq, P.cq);
  W->levels_k = num_levels(P.nk, P.ck);
  // Basic splitting runs every level with the multi-block kernels.
  const bool basic = P.split == CA_SPLIT_BASIC;
  W->big_q = basic ? W->levels_q : split_big_levels(P.nq, P.cq, W->levels_q);
  W->big_k = basic ? W->levels_k : split_big_levels(P.nk, P.ck, W->levels_k);
  int bigmax = W->big_q > W->big_k ? W->big_q : W->big_k;
  W->max_big_nodes = bigmax > 0 ? (1 << (bigmax - 1)) : 1;
  W->hist_slots = split_hist_slots(P, W->big_q, W->big_k);

  W->y_q = take(BH * P.nq * d * 4);
  W->y_k = take(BH * P.nk * d * 4);
  const bool cols = col_copy_used(P);
  W->ycol_q = take(cols ? BH * kColCopy * P.nq * 4 : 0);
  W->ycol_k = take(cols ? BH * kColCopy * P.nk * 4 : 0);
  W->idx0 = take(2 * BH * nmax * 4);
  W->idx1 = take(2 * BH * nmax * 4);
  W->keys = take(2 * BH * nmax * 4);
  W->mom_part = take(2 * BH * W->nblk_mom * (d * d + d) * 4);
  W->mats = take(BH * kMats * d * d * 4);
  W->vecs = take(BH * kVecs * d * 4);
  W->inv_q = take(BH * P.nq * 4);
  W->qn_part = take(BH * W->nblk_mom * (d * d + d) * 4);
  W->wops = take(BH * 3 * 2 * d * d * 2);
  W->node_state = take(2 * BH * W->max_big_nodes * kNodeInts * 4);
  W->hist = take(2 * BH * W->hist_slots * kBins * 4);
  W->chunk_cnt = take(2 * BH * W->hist_slots * 2 * 4);
  W->dirs = take(basic ? 2 * 2 * BH * W->max_big_nodes * d * 4 : 0);
  W->scores = take(BH * P.nqc * P.nkc * 4);
  W->sched = take(((size_t)8 + 8 * (size_t)attn_sched_cap((int)(BH * P.nqc))) * 4);
  const size_t ntile = (P.nkc + kCompTile - 1) / kCompTile;
  W->comp_tiles = take(P.dtype == CA_BF16 ? BH * ntile * comp_tile_bytes(P.d) : 0);
  W->total = off;
}

}  // namespace ca

extern "C" {

int ca_abi_version(void) { return CA_ABI_VERSION; }

const char* ca_status_str(int status) {
  switch (status) {
    case CA_OK: return "CA_OK";
    case CA_E_INVALID: return "CA_E_INVALID: invalid argument";
    case CA_E_UNSUPPORTED: return "CA_E_UNSUPPORTED: combination not built";
    case CA_E_WORKSPACE: return "CA_E_WORKSPACE: workspace too small";
    case CA_E_DEVICE: return "CA_E_DEVICE: HIP error";
    case CA_E_NONFINITE: return "CA_E_NONFINITE: an input holds NaN or Inf";
    default: return "unknown status";
  }
}

const char* ca_last_error(void) { return g_err; }

int ca_workspace_size(const ca_problem* p, int32_t k, size_t* bytes) {
  ca::Prob P;
  int s = check_problem(p, &P);
  if (s) return s;
  if ((s = check_k(P, k))) return s;
  if (!bytes) return fail(CA_E_INVALID, "bytes is NULL");
  ca::Workspace W;
  ca::plan_workspace(P, &W);
  *bytes = W.total;
  return ok();
}

int ca_cluster(const ca_problem* p, const void* q, const void* k, const void* v,
               const ca_cluster_out* out, void* ws, size_t ws_bytes, void* stream) {
  ca::Prob P;
  int s = check_problem(p, &P);
  if (s) return s;
  if (!q || !k) return fail(CA_E_INVALID, "q and k are required");
  if (!out) return fail(CA_E_INVALID, "out is NULL");
  if (!out->perm_q || !out->perm_k || !out->count_q || !out->count_k || !out->cent_q ||
      !out->cent_k || !out->qp || !out->kp)
    return fail(CA_E_INVALID, "a required output of ca_cluster is NULL");
  bool want_v = v != nullptr;
  if (want_v && (!out->cent_v || !out->vp))
    return fail(CA_E_INVALID, "v given but cent_v or vp is NULL");
  if ((s = check_aligned(P, q, "q")) || (s = check_aligned(P, k, "k")) ||
      (want_v && (s = check_aligned(P, v, "v"))))
    return s;
  ca::Workspace W;
  ca::plan_workspace(P, &W);
  if ((s = check_ws(W, ws, ws_bytes))) return s;
  return device_status(
      ca::launch_cluster(P, q, k, v, out, (char*)ws, W, (hipStream_t)stream), "ca_cluster");
}

int ca_select(const ca_problem* p, const float* cent_q, const float* cent_k,
              const float* scores_in, float* scores_out, int32_t k, int32_t* lists, void* ws,
              size_t ws_bytes, void* stream) {
  ca::Prob P;
  int s = check_problem(p, &P);
  if (s) return s;
  if ((s = check_k(P, k))) return s;
  if (!lists) return fail(CA_E_INVALID, "lists is NULL");
  if (!scores_in && (!cent_q || !cent_k))
    return fail(CA_E_INVALID, "cent_q and cent_k are required when scores_in is NULL");
  float* scores = scores_out;
  if (!scores_in && !scores) {
    ca::Workspace W;
    ca::plan_workspace(P, &W);
    if ((s = check_ws(W, ws, ws_bytes))) return s;
    scores = (float*)((char*)ws + W.scores);
  }
  return device_status(ca::launch_select(P, cent_q, cent_k, scores_in, scores, k, lists,
                                         (hipStream_t)stream),
                       "ca_select");
}

int ca_select_hist(const ca_problem* p, const float* cent_q, const float* cent_k,
                   const int32_t* count_k, const float* scores_in, float* scores_out,
                   int32_t min_count, float mass_recall, float scale, int32_t* lists,
                   int32_t* lens, void* ws, size_t ws_bytes, void* stream) {
  ca::Prob P;
  int s = check_problem(p, &P);
  if (s) return s;
  if (!lists || !lens || !count_k) return fail(CA_E_INVALID, "lists, lens and count_k are required");
  if (!scores_in && (!cent_q || !cent_k))
    return fail(CA_E_INVALID, "cent_q and cent_k are required when scores_in is NULL");
  if (min_count < 1) return fail(CA_E_INVALID, "min_count=%d must be >= 1", min_count);
  if (!(mass_recall >= 0.0f && mass_recall <= 1.0f))
    return fail(CA_E_INVALID, "mass_recall must be in [0, 1]");
  float* scores = scores_out;
  if (!scores_in && !scores) {
    ca::Workspace W;
    ca::plan_workspace(P, &W);
    if ((s = check_ws(W, ws, ws_bytes))) return s;
    scores = (float*)((char*)ws + W.scores);
  }
  if (!(scale > 0.0f)) scale = 1.0f / sqrtf((float)P.d);
  return device_status(ca::launch_select_hist(P, cent_q, cent_k, count_k, scores_in, scores,
                                              min_count, mass_recall, scale, lists, lens,
                                              (hipStream_t)stream),
                       "ca_select_hist");
}

int ca_block_sparse_attn(const ca_problem* p, const void* qp, const void* kp, const void* vp,
                         const int32_t* count_k, const int32_t* lists, const int32_t* lens,
                         int32_t k, float scale, void* op, float* lse, void* ws, size_t ws_bytes,
                         void* stream) {
  ca::Prob P;
  int s = check_problem(p, &P);
  if (s) return s;
  if ((s = check_k(P, k))) return s;
  if (!qp || !kp || !vp || !count_k || !lists || !op || !lse)
    return fail(CA_E_INVALID, "a required pointer of ca_block_sparse_attn is NULL");
  if ((s = check_attn_shape(P))) return s;
  int32_t* sched = nullptr;
  if (ws && lens && P.dtype == CA_BF16) {
    ca::Workspace W;
    ca::plan_workspace(P, &W);
    if ((s = check_ws(W, ws, ws_bytes))) return s;
    sched = (int32_t*)((char*)ws + W.sched);
  }
  if (!(scale > 0.0f)) scale = 1.0f / sqrtf((float)P.d);
  return device_status(ca::launch_attn(P, qp, kp, vp, count_k, lists, lens, k, scale, op, lse,
                                       sched, (hipStream_t)stream),
                       "ca_block_sparse_attn");
}

int ca_compensate(const ca_problem* p, const void* qp, const float* cent_k, const float* cent_v,
                  const int32_t* count_k, const int32_t* lists, const int32_t* lens, int32_t k,
                  float scale,
                  int32_t enable, const void* op, const float* lse, const int32_t* perm_q,
                  void* out, float* lse_out, void* ws, size_t ws_bytes, void* stream) {
  ca::Prob P;
  int s = check_problem(p, &P);
  if (s) return s;
  if ((s = check_k(P, k))) return s;
  if (!op || !lse || !perm_q || !out)
    return fail(CA_E_INVALID, "a required pointer of ca_compensate is NULL");
  if ((s = check_aligned(P, out, "out"))) return s;
  if (enable && (!qp || !cent_k || !cent_v || !count_k || !lists))
    return fail(CA_E_INVALID, "compensation needs qp, cent_k, cent_v, count_k and lists");
  if ((s = check_attn_shape(P))) return s;
  // the selection bitmap of a query cluster (in LDS) exists only when some
  // cluster can be unselected and compensation runs
  if (enable && (k < P.nkc || lens) && P.nkc > ca::kMaskWords * 32)
    return fail(CA_E_UNSUPPORTED,
                "ca_compensate: compensation supports at most %d key clusters (got %d; "
                "enable = 0 has no such limit)", ca::kMaskWords * 32, P.nkc);
  char* tiles = nullptr;
  if (P.dtype == CA_BF16 && enable && (k < P.nkc || lens)) {
    ca::Workspace W;
    ca::plan_workspace(P, &W);
    if ((s = check_ws(W, ws, ws_bytes))) return s;
    tiles = (char*)ws + W.comp_tiles;
  }
  if (!(scale > 0.0f)) scale = 1.0f / sqrtf((float)P.d);
  return device_status(ca::launch_comp(P, qp, cent_k, cent_v, count_k, lists, lens, k, scale,
                                       enable, op, lse, perm_q, out, lse_out, tiles,
                                       (hipStream_t)stream),
                       "ca_compensate");
}

int ca_attn_compensated(const ca_problem* p, const void* qp, const void* kp, const void* vp,
                        const float* cent_k, const float* cent_v, const int32_t* count_k,
                        const int32_t* lists, const int32_t* lens, int32_t k, float scale,
                        int32_t enable, const int32_t* perm_q, void* out, float* lse_out,
                        void* ws, size_t ws_bytes, void* stream) {
  ca::Prob P;
  int s = check_problem(p, &P);
  if (s) return s;
  if ((s = check_k(P, k))) return s;
  if (P.dtype != CA_BF16) return fail(CA_E_UNSUPPORTED, "ca_attn_compensated needs bf16 inputs");
  if (!qp || !kp || !vp || !count_k || !lists || !perm_q || !out)
    return fail(CA_E_INVALID, "a required pointer of ca_attn_compensated is NULL");
  if ((s = check_aligned(P, out, "out"))) return s;
  if (enable && (!cent_k || !cent_v))
    return fail(CA_E_INVALID, "compensation needs cent_k and cent_v");
  if ((s = check_attn_shape(P))) return s;
  if (P.nkc > ca::kMaskWords * 32)
    return fail(CA_E_UNSUPPORTED, "ca_attn_compensated supports at most 65536 key clusters");
  const bool comp = enable && (k < P.nkc || lens);
  char* tiles = nullptr;
  int32_t* sched = nullptr;
  if (comp || (ws && lens)) {
    ca::Workspace W;
    ca::plan_workspace(P, &W);
    if ((s = check_ws(W, ws, ws_bytes))) return s;
    if (comp) tiles = (char*)ws + W.comp_tiles;
    if (lens) sched = (int32_t*)((char*)ws + W.sched);
  }
  if (!(scale > 0.0f)) scale = 1.0f / sqrtf((float)P.d);
  hipStream_t st = (hipStream_t)stream;
  if (tiles) {
    s = device_status(ca::launch_comp_stage(P, cent_k, cent_v, count_k, tiles, st),
                      "ca_attn_compensated");
    if (s) return s;
  }
  return device_status(ca::launch_attn_fused(P, qp, kp, vp, count_k, lists, lens, k, scale, tiles,
                                             perm_q, out, lse_out, sched, st),
                       "ca_attn_compensated");
}

int ca_attn_compensated_noalloc(const ca_problem* p, const void* qp, const void* kp,
                                const void* vp, const float* cent_k, const float* cent_v,
                                const int32_t* count_k, const int32_t* lists,
                                const int32_t* lens, int32_t k, float scale, int32_t enable,
                                const int32_t* perm_q, void* out, float* lse_out,
                                void* stream) {
  ca::Prob P;
  int s = check_problem(p, &P);
  if (s) return s;
  if ((s = check_k(P, k))) return s;
  if (P.dtype != CA_BF16)
    return fail(CA_E_UNSUPPORTED, "ca_attn_compensated_noalloc needs bf16 inputs");
  if (!qp || !kp || !vp || !count_k || !lists || !perm_q || !out)
    return fail(CA_E_INVALID, "a required pointer of ca_attn_compensated_noalloc is NULL");
  if ((s = check_aligned(P, out, "out"))) return s;
  if (enable && (!cent_k || !cent_v))
    return fail(CA_E_INVALID, "compensation needs cent_k and cent_v");
  if ((s = check_attn_shape(P))) return s;
  if (P.nkc > ca::kMaskWords * 32)
    return fail(CA_E_UNSUPPORTED,
                "ca_attn_compensated_noalloc supports at most 65536 key clusters");
  // the same regions as the workspace of ca_attn_compensated: centroid
  // tiles (compensation with unselected clusters), then the schedule (lens)
  const bool comp = enable && (k < P.nkc || lens);
  const size_t ntile = (size_t)(P.nkc + ca::kCompTile - 1) / ca::kCompTile;
  const size_t tile_bytes =
      comp ? ca::align256((size_t)P.BH * ntile * ca::comp_tile_bytes(P.d)) : 0;
  const size_t sched_bytes =
      lens ? ((size_t)8 + 8 * (size_t)ca::attn_sched_cap((int)((size_t)P.BH * P.nqc))) * 4 : 0;
  if (tile_bytes + sched_bytes > kScratchBytes)
    return fail(CA_E_WORKSPACE,
                "ca_attn_compensated_noalloc: this problem needs %zu bytes of scratch, the "
                "library holds %zu per device (use ca_attn_compensated with a workspace)",
                tile_bytes + sched_bytes, kScratchBytes);
  char* base = nullptr;
  if (tile_bytes + sched_bytes > 0 && (s = scratch_on_current_device(&base))) return s;
  char* tiles = comp ? base : nullptr;
  int32_t* sched = lens ? (int32_t*)(base + tile_bytes) : nullptr;
  if (!(scale > 0.0f)) scale = 1.0f / sqrtf((float)P.d);
  hipStream_t st = (hipStream_t)stream;
  if (tiles) {
    s = device_status(ca::launch_comp_stage(P, cent_k, cent_v, count_k, tiles, st),
                      "ca_attn_compensated_noalloc");
    if (s) return s;
  }
  return device_status(ca::launch_attn_fused(P, qp, kp, vp, count_k, lists, lens, k, scale, tiles,
                                             perm_q, out, lse_out, sched, st),
                       "ca_attn_compensated_noalloc");
}

int ca_check_finite(const ca_problem* p, const void* q, const void* k, const void* v,
                    int32_t* flags, void* stream) {
  ca::Prob P;
  int s = check_problem(p, &P);
  if (s) return s;
  if (!q || !k || !flags) return fail(CA_E_INVALID, "q, k and flags are required");
  if ((s = check_aligned(P, q, "q")) || (s = check_aligned(P, k, "k")) ||
      (v && (s = check_aligned(P, v, "v"))))
    return s;
  return device_status(ca::launch_check_finite(P, q, k, v, flags, (hipStream_t)stream),
                       "ca_check_finite");
}

}  // extern "C"
