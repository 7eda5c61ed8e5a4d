"""ctypes view of libclusterattn.so (include/clusterattn.h). Marshalling only."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libclusterattn.so")

CA_OK, CA_E_INVALID, CA_E_UNSUPPORTED, CA_E_WORKSPACE, CA_E_DEVICE, CA_E_NONFINITE = range(6)
CA_F32, CA_BF16 = 0, 1
CA_XF_NONE, CA_XF_PCA, CA_XF_METRIC, CA_XF_ADAPTIVE, CA_XF_RANDOM = 0, 1, 2, 3, 4
CA_LAYOUT_BHND, CA_LAYOUT_BNHD, CA_LAYOUT_STRIDED = 0, 1, 2
CA_SPLIT_DIAG, CA_SPLIT_BASIC = 0, 1

EXPORTS = (
    "ca_abi_version",
    "ca_status_str",
    "ca_last_error",
    "ca_workspace_size",
    "ca_cluster",
    "ca_select",
    "ca_select_hist",
    "ca_block_sparse_attn",
    "ca_compensate",
    "ca_attn_compensated",
    "ca_attn_compensated_noalloc",
    "ca_check_finite",
)

_i32 = ctypes.c_int32
_vp = ctypes.c_void_p


class CaProblem(ctypes.Structure):
    _fields_ = ([(n, _i32) for n in ("batch", "heads", "nq", "nk", "d", "cq", "ck", "dtype",
                                     "transform", "layout", "split")]
                + [(n, ctypes.c_int64 * 3) for n in ("q_stride", "k_stride", "v_stride",
                                                     "out_stride")])


class CaClusterOut(ctypes.Structure):
    _fields_ = [(n, _vp) for n in ("perm_q", "perm_k", "cid_q", "cid_k", "count_q", "count_k",
                                   "cent_q", "cent_k", "cent_v", "qp", "kp", "vp", "yq_dbg",
                                   "yk_dbg")]


class CAError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: {detail or status_str(status)} (status {status})")
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    """Load the HIP library; raises if it has not been built (there is no
    fallback implementation)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2608_26965_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER(CaProblem)
    lib.ca_abi_version.restype = ctypes.c_int
    lib.ca_abi_version.argtypes = []
    lib.ca_status_str.restype = ctypes.c_char_p
    lib.ca_status_str.argtypes = [ctypes.c_int]
    lib.ca_last_error.restype = ctypes.c_char_p
    lib.ca_last_error.argtypes = []
    lib.ca_workspace_size.restype = ctypes.c_int
    lib.ca_workspace_size.argtypes = [P, _i32, ctypes.POINTER(ctypes.c_size_t)]
    lib.ca_cluster.restype = ctypes.c_int
    lib.ca_cluster.argtypes = [P, _vp, _vp, _vp, ctypes.POINTER(CaClusterOut), _vp,
                               ctypes.c_size_t, _vp]
    lib.ca_select.restype = ctypes.c_int
    lib.ca_select.argtypes = [P, _vp, _vp, _vp, _vp, _i32, _vp, _vp, ctypes.c_size_t, _vp]
    lib.ca_block_sparse_attn.restype = ctypes.c_int
    lib.ca_block_sparse_attn.argtypes = [P, _vp, _vp, _vp, _vp, _vp, _vp, _i32, ctypes.c_float,
                                         _vp, _vp, _vp, ctypes.c_size_t, _vp]
    lib.ca_select_hist.restype = ctypes.c_int
    lib.ca_select_hist.argtypes = [P, _vp, _vp, _vp, _vp, _vp, _i32, ctypes.c_float,
                                   ctypes.c_float, _vp, _vp, _vp, ctypes.c_size_t, _vp]
    lib.ca_compensate.restype = ctypes.c_int
    lib.ca_compensate.argtypes = [P, _vp, _vp, _vp, _vp, _vp, _vp, _i32, ctypes.c_float, _i32,
                                  _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
    lib.ca_attn_compensated.restype = ctypes.c_int
    lib.ca_attn_compensated.argtypes = [P, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32,
                                        ctypes.c_float, _i32, _vp, _vp, _vp, _vp, ctypes.c_size_t,
                                        _vp]
    lib.ca_attn_compensated_noalloc.restype = ctypes.c_int
    lib.ca_attn_compensated_noalloc.argtypes = [P, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i32,
                                                ctypes.c_float, _i32, _vp, _vp, _vp, _vp]
    lib.ca_check_finite.restype = ctypes.c_int
    lib.ca_check_finite.argtypes = [P, _vp, _vp, _vp, _vp, _vp]
    _lib = lib
    return lib


def status_str(status: int) -> str:
    return load().ca_status_str(status).decode()


def last_error() -> str:
    return load().ca_last_error().decode()


def check(status: int, where: str) -> None:
    if status != CA_OK:
        raise CAError(status, where, last_error())
