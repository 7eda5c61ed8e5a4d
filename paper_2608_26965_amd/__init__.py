"""ClusterAttention on MI355X: Python binding of libclusterattn (HIP, gfx950).

Every step runs in the HIP library; this module only allocates tensors with
torch and passes their device pointers and the current stream to the four
C-ABI calls (see include/clusterattn.h):

    cluster -> select -> block_sparse_attn -> compensate

``forward`` chains them for one attention layer. There is no CPU fallback: if
the library is not built, importing the calls raises.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import torch

from . import _lib
from ._lib import (CA_BF16, CA_F32, CA_LAYOUT_BHND, CA_LAYOUT_BNHD, CA_LAYOUT_STRIDED,
                   CA_SPLIT_BASIC, CA_SPLIT_DIAG, CA_XF_ADAPTIVE, CA_XF_METRIC, CA_XF_NONE,
                   CA_XF_PCA, CA_XF_RANDOM, CAError)

__all__ = ["Problem", "bhnd_strides", "workspace_size", "cluster", "select", "select_hist", "block_sparse_attn",
           "compensate", "attn_compensated", "attn_compensated_noalloc", "check_finite",
           "forward", "CAError", "abi_version"]

_XF = {"none": CA_XF_NONE, "pca": CA_XF_PCA, "metric": CA_XF_METRIC, "adaptive": CA_XF_ADAPTIVE,
       "random": CA_XF_RANDOM}
_LAYOUT = {"bhnd": CA_LAYOUT_BHND, "bnhd": CA_LAYOUT_BNHD, "strided": CA_LAYOUT_STRIDED}
_SPLIT = {"diag": CA_SPLIT_DIAG, "basic": CA_SPLIT_BASIC}
_DT = {torch.float32: CA_F32, torch.bfloat16: CA_BF16}


def abi_version() -> int:
    return _lib.load().ca_abi_version()


@dataclass(frozen=True)
class Problem:
    batch: int
    heads: int
    nq: int
    nk: int
    d: int
    cq: int
    ck: int
    dtype: torch.dtype = torch.bfloat16
    transform: str = "metric"
    layout: str = "bhnd"
    split: str = "diag"
    # layout "strided": element strides (batch, head, token) of q, k, v, out
    q_stride: tuple = (0, 0, 0)
    k_stride: tuple = (0, 0, 0)
    v_stride: tuple = (0, 0, 0)
    out_stride: tuple = (0, 0, 0)

    @property
    def bh(self):
        return self.batch * self.heads

    @property
    def nqc(self):
        return -(-self.nq // self.cq)

    @property
    def nkc(self):
        return -(-self.nk // self.ck)

    @property
    def nq_pad(self):
        return self.nqc * self.cq

    @property
    def nk_pad(self):
        return self.nkc * self.ck

    def c(self) -> _lib.CaProblem:
        st = [(__import__("ctypes").c_int64 * 3)(*t) for t in
              (self.q_stride, self.k_stride, self.v_stride, self.out_stride)]
        return _lib.CaProblem(self.batch, self.heads, self.nq, self.nk, self.d, self.cq, self.ck,
                              _DT[self.dtype], _XF[self.transform], _LAYOUT[self.layout],
                              _SPLIT[self.split], *st)

    def shape(self, n):
        """Shape of a dense output tensor: [B,H,n,d] for "bhnd" and "strided"
        (whose out_stride must then describe it; see bhnd_strides), else
        [B,n,H,d]."""
        if self.layout in ("bhnd", "strided"):
            return (self.batch, self.heads, n, self.d)
        return (self.batch, n, self.heads, self.d)


def bhnd_strides(t) -> tuple:
    """(batch, head, token) element strides of a tensor viewed as [B,H,N,d]
    with its last dimension contiguous (any permutation or slice of a larger
    tensor, e.g. one third of a fused [B,N,3,H,d] projection)."""
    if t.dim() != 4 or t.stride(3) != 1:
        raise ValueError("expected a [B,H,N,d] view whose last dimension is contiguous")
    return (t.stride(0), t.stride(1), t.stride(2))


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(device):
    return torch.cuda.current_stream(device).cuda_stream


def workspace_size(p: Problem, k: int = 1) -> int:
    n = __import__("ctypes").c_size_t(0)
    _lib.check(_lib.load().ca_workspace_size(p.c(), k, n), "ca_workspace_size")
    return n.value


def workspace(p: Problem, device, k: int = 1) -> torch.Tensor:
    return torch.empty(max(workspace_size(p, k), 256), dtype=torch.uint8, device=device)


def cluster(p: Problem, q, k, v=None, *, export_y=False, ws=None):
    """Step 1. Returns a dict of device tensors: perm_q/perm_k [BH,n],
    cid_q/cid_k [BH,n], count_q/count_k [BH,nc], cent_q/cent_k/cent_v [BH,nc,d],
    qp/kp [BH,n_pad,d], vp [BH,nkc,d,ck] (value tiles), and yq/yk [BH,n,d] if
    export_y."""
    dev = q.device
    i32 = dict(dtype=torch.int32, device=dev)
    f32 = dict(dtype=torch.float32, device=dev)
    BH, d = p.bh, p.d
    r = dict(
        perm_q=torch.empty(BH, p.nq, **i32), perm_k=torch.empty(BH, p.nk, **i32),
        cid_q=torch.empty(BH, p.nq, **i32), cid_k=torch.empty(BH, p.nk, **i32),
        count_q=torch.empty(BH, p.nqc, **i32), count_k=torch.empty(BH, p.nkc, **i32),
        cent_q=torch.empty(BH, p.nqc, d, **f32), cent_k=torch.empty(BH, p.nkc, d, **f32),
        qp=torch.empty(BH, p.nq_pad, d, dtype=p.dtype, device=dev),
        kp=torch.empty(BH, p.nk_pad, d, dtype=p.dtype, device=dev),
    )
    if v is not None:
        r["cent_v"] = torch.empty(BH, p.nkc, d, **f32)
        r["vp"] = torch.empty(BH, p.nkc, d, p.ck, dtype=p.dtype, device=dev)
    if export_y:
        r["yq"] = torch.empty(BH, p.nq, d, **f32)
        r["yk"] = torch.empty(BH, p.nk, d, **f32)
    out = _lib.CaClusterOut(*(_ptr(r.get(n)) for n in (
        "perm_q", "perm_k", "cid_q", "cid_k", "count_q", "count_k", "cent_q", "cent_k", "cent_v",
        "qp", "kp", "vp", "yq", "yk")))
    if ws is None:
        ws = workspace(p, dev)
    st = _lib.load().ca_cluster(p.c(), _ptr(q), _ptr(k), _ptr(v), out, _ptr(ws), ws.numel(),
                                _stream(dev))
    _lib.check(st, "ca_cluster")
    return r


def select(p: Problem, cent_q, cent_k, keep_k: int, *, scores_in=None, export_scores=False,
           ws=None):
    """Step 2. Returns (lists [BH,nqc,k] int32 ascending, scores or None)."""
    dev = (cent_q if cent_q is not None else scores_in).device
    lists = torch.empty(p.bh, p.nqc, keep_k, dtype=torch.int32, device=dev)
    scores = None
    if export_scores:
        scores = torch.empty(p.bh, p.nqc, p.nkc, dtype=torch.float32, device=dev)
    if ws is None and scores_in is None and scores is None:
        ws = workspace(p, dev, keep_k)
    st = _lib.load().ca_select(p.c(), _ptr(cent_q), _ptr(cent_k), _ptr(scores_in), _ptr(scores),
                               keep_k, _ptr(lists), _ptr(ws), 0 if ws is None else ws.numel(),
                               _stream(dev))
    _lib.check(st, "ca_select")
    return lists, scores


# `forward` takes a `select=` mode argument; this name reaches the top-k call from there.
select_topk = select


def select_hist(p: Problem, cent_q, cent_k, count_k, min_count: int, mass_recall: float = 0.0,
                scale: float = 0.0, *, scores_in=None, export_scores=False, ws=None):
    """Step 2, the two-pass histogram selection. min_count = k with
    mass_recall = 0 is top-k through the histogram (at least k clusters);
    min_count = 16 with mass_recall in (0, 1] is adaptive assignment.
    Returns (lists [BH,nqc,nkc] int32, lens [BH,nqc] int32, scores or None);
    row a of lists holds lens[a] ascending cluster indices."""
    dev = (cent_q if cent_q is not None else scores_in).device
    lists = torch.empty(p.bh, p.nqc, p.nkc, dtype=torch.int32, device=dev)
    lens = torch.empty(p.bh, p.nqc, dtype=torch.int32, device=dev)
    scores = None
    if export_scores:
        scores = torch.empty(p.bh, p.nqc, p.nkc, dtype=torch.float32, device=dev)
    if ws is None and scores_in is None and scores is None:
        ws = workspace(p, dev)
    st = _lib.load().ca_select_hist(p.c(), _ptr(cent_q), _ptr(cent_k), _ptr(count_k),
                                    _ptr(scores_in), _ptr(scores), int(min_count),
                                    float(mass_recall), float(scale), _ptr(lists), _ptr(lens),
                                    _ptr(ws), 0 if ws is None else ws.numel(), _stream(dev))
    _lib.check(st, "ca_select_hist")
    return lists, lens, scores


def block_sparse_attn(p: Problem, qp, kp, vp, count_k, lists, keep_k: int, scale: float = 0.0,
                      lens=None, ws=None):
    """Step 3. Returns (op [BH,nq_pad,d] dtype, lse [BH,nq_pad] fp32). keep_k is
    the list stride; lens (optional) the per-cluster list lengths; ws
    (optional) the workspace, with which lists of different lengths are
    scheduled longest first per XCD."""
    dev = qp.device
    op = torch.empty(p.bh, p.nq_pad, p.d, dtype=p.dtype, device=dev)
    lse = torch.empty(p.bh, p.nq_pad, dtype=torch.float32, device=dev)
    st = _lib.load().ca_block_sparse_attn(p.c(), _ptr(qp), _ptr(kp), _ptr(vp), _ptr(count_k),
                                          _ptr(lists), _ptr(lens), keep_k, float(scale), _ptr(op),
                                          _ptr(lse), _ptr(ws), ws.numel() if ws is not None else 0,
                                          _stream(dev))
    _lib.check(st, "ca_block_sparse_attn")
    return op, lse


def compensate(p: Problem, qp, cent_k, cent_v, count_k, lists, keep_k: int, op, lse, perm_q,
               scale: float = 0.0, enable: bool = True, want_lse: bool = False, out=None,
               ws=None, lens=None):
    """Step 4. Returns (out in the problem layout, lse [BH,nq] or None)."""
    dev = op.device
    if out is None:
        out = torch.empty(p.shape(p.nq), dtype=p.dtype, device=dev)
    lse_out = torch.empty(p.bh, p.nq, dtype=torch.float32, device=dev) if want_lse else None
    if (ws is None and enable and p.dtype == torch.bfloat16
            and (keep_k < p.nkc or lens is not None)):
        ws = workspace(p, dev, keep_k)
    st = _lib.load().ca_compensate(p.c(), _ptr(qp), _ptr(cent_k), _ptr(cent_v), _ptr(count_k),
                                   _ptr(lists), _ptr(lens), keep_k, float(scale),
                                   int(bool(enable)), _ptr(op),
                                   _ptr(lse), _ptr(perm_q), _ptr(out), _ptr(lse_out), _ptr(ws),
                                   0 if ws is None else ws.numel(), _stream(dev))
    _lib.check(st, "ca_compensate")
    return out, lse_out


def attn_compensated(p: Problem, qp, kp, vp, cent_k, cent_v, count_k, lists, keep_k: int,
                     perm_q, scale: float = 0.0, enable: bool = True, want_lse: bool = False,
                     out=None, ws=None, lens=None):
    """Steps 3 and 4 in one pass (bf16). Returns (out in the problem layout,
    lse [BH,nq] or None), as block_sparse_attn followed by compensate."""
    dev = qp.device
    if out is None:
        out = torch.empty(p.shape(p.nq), dtype=p.dtype, device=dev)
    lse_out = torch.empty(p.bh, p.nq, dtype=torch.float32, device=dev) if want_lse else None
    if ws is None and ((enable and keep_k < p.nkc) or lens is not None):
        ws = workspace(p, dev, keep_k)
    st = _lib.load().ca_attn_compensated(p.c(), _ptr(qp), _ptr(kp), _ptr(vp), _ptr(cent_k),
                                         _ptr(cent_v), _ptr(count_k), _ptr(lists), _ptr(lens),
                                         keep_k, float(scale), int(bool(enable)), _ptr(perm_q),
                                         _ptr(out), _ptr(lse_out), _ptr(ws),
                                         0 if ws is None else ws.numel(), _stream(dev))
    _lib.check(st, "ca_attn_compensated")
    return out, lse_out


def attn_compensated_noalloc(p: Problem, qp, kp, vp, cent_k, cent_v, count_k, lists,
                             keep_k: int, perm_q, scale: float = 0.0, enable: bool = True,
                             want_lse: bool = False, out=None, lens=None):
    """attn_compensated without a workspace: the library's per-device scratch
    holds the centroid tiles and the schedule (see the header for its size
    and for calls that overlap on one device). Allocates nothing when out
    (and lse, with want_lse) are supplied by the caller: pass out= and, for
    the lse, call the C function directly."""
    dev = qp.device
    if out is None:
        out = torch.empty(p.shape(p.nq), dtype=p.dtype, device=dev)
    lse_out = torch.empty(p.bh, p.nq, dtype=torch.float32, device=dev) if want_lse else None
    st = _lib.load().ca_attn_compensated_noalloc(p.c(), _ptr(qp), _ptr(kp), _ptr(vp),
                                                 _ptr(cent_k), _ptr(cent_v), _ptr(count_k),
                                                 _ptr(lists), _ptr(lens), keep_k, float(scale),
                                                 int(bool(enable)), _ptr(perm_q), _ptr(out),
                                                 _ptr(lse_out), _stream(dev))
    _lib.check(st, "ca_attn_compensated_noalloc")
    return out, lse_out


def check_finite(p: Problem, q, k, v=None, *, raise_error=True) -> int:
    """Checked mode: ca_check_finite on the current stream, then a
    synchronisation to read its flags (bit 0 q, 1 k, 2 v hold a NaN or an
    infinity). Raises CAError with CA_E_NONFINITE when raise_error and any bit
    is set; returns the flags."""
    flags = torch.empty(1, dtype=torch.int32, device=q.device)
    st = _lib.load().ca_check_finite(p.c(), _ptr(q), _ptr(k), _ptr(v), _ptr(flags),
                                     _stream(q.device))
    _lib.check(st, "ca_check_finite")
    f = int(flags.item())
    if f and raise_error:
        which = ", ".join(n for b, n in ((1, "q"), (2, "k"), (4, "v")) if f & b)
        raise CAError(_lib.CA_E_NONFINITE, "ca_check_finite", f"non-finite values in {which}")
    return f


def keep_to_k(keep: float, n_kc: int) -> int:
    """Kept key clusters for a keep fraction: ceil(keep * n_kc), in [1, n_kc]."""
    return max(1, min(n_kc, int(math.ceil(keep * n_kc - 1e-9))))


def forward(q, k, v, cq=128, ck=None, keep=None, keep_k=None, transform="metric",
            compensation=True, scale=None, layout="bhnd", return_parts=False, select="topk",
            mass_recall=0.9, min_count=16, one_pass=True, checked=False):
    """ClusterAttention for one layer. q, k, v: [B,H,N,d] ("bhnd") or [B,N,H,d]
    ("bnhd"), bf16 or fp32, on one GPU; with layout="strided", any [B,H,N,d]
    views whose last dimension is contiguous (for instance slices of a fused
    [B,N,3,H,d] projection), read in place; the output is then a new dense
    [B,H,N,d] tensor.

    select="topk": exact top-k of either a fraction (``keep``) or a count
    (``keep_k``) of key clusters per query cluster; select="hist": the
    two-pass histogram top-k (at least that many clusters); select="adaptive":
    attention-mass recall ``mass_recall`` with at least ``min_count`` clusters
    (use it with transform="adaptive"). bf16 layers run steps 3 and 4 in one
    pass (attn_compensated) unless one_pass is False or return_parts asks for
    the sparse part's output and lse. checked=True first runs the checked
    mode (check_finite), which synchronises and raises CAError with
    CA_E_NONFINITE on NaN or Inf inputs."""
    ck = cq if ck is None else ck
    if layout in ("bhnd", "strided"):
        B, H, nq, d = q.shape
        nk = k.shape[2]
    else:
        B, nq, H, d = q.shape
        nk = k.shape[1]
    if layout == "strided":
        dense_out = (H * nq * d, nq * d, d)
        p = Problem(B, H, nq, nk, d, cq, ck, q.dtype, transform, layout,
                    q_stride=bhnd_strides(q), k_stride=bhnd_strides(k), v_stride=bhnd_strides(v),
                    out_stride=dense_out)
    else:
        p = Problem(B, H, nq, nk, d, cq, ck, q.dtype, transform, layout)
    if checked:
        check_finite(p, q, k, v)
    if keep_k is None:
        keep_k = keep_to_k(1.0 / 8 if keep is None else keep, p.nkc)
    sc = 0.0 if scale is None else float(scale)
    ws = workspace(p, q.device, keep_k)
    c = cluster(p, q, k, v, ws=ws)
    lens = None
    stride = keep_k
    if select == "topk":
        lists, _ = select_topk(p, c["cent_q"], c["cent_k"], keep_k, ws=ws)
    elif select in ("hist", "adaptive"):
        floor, recall = (keep_k, 0.0) if select == "hist" else (min_count, mass_recall)
        lists, lens, _ = select_hist(p, c["cent_q"], c["cent_k"], c["count_k"], floor, recall,
                                     sc, ws=ws)
        stride = p.nkc
    else:
        raise ValueError(select)
    if one_pass and not return_parts and p.dtype == torch.bfloat16:
        out, _ = attn_compensated(p, c["qp"], c["kp"], c["vp"], c["cent_k"], c["cent_v"],
                                  c["count_k"], lists, stride, c["perm_q"], sc, compensation,
                                  ws=ws, lens=lens)
        return out
    op, lse = block_sparse_attn(p, c["qp"], c["kp"], c["vp"], c["count_k"], lists, stride, sc,
                                lens=lens, ws=ws)
    out, lse_out = compensate(p, c["qp"], c["cent_k"], c["cent_v"], c["count_k"], lists, stride,
                              op, lse, c["perm_q"], sc, compensation, want_lse=return_parts, ws=ws,
                              lens=lens)
    if return_parts:
        return out, dict(c, lists=lists, lens=lens, op=op, lse_s=lse, lse=lse_out, problem=p)
    return out

