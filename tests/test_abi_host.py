"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every symbol the header declares, and rejects invalid arguments before
touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib():
    from paper_2608_26965_amd import _lib as L
    try:
        return L, L.load()
    except ImportError as e:  # pragma: no cover
        pytest.skip(str(e))


def test_header_symbols_exported():
    L, lib = _lib()
    hdr = open(os.path.join(ROOT, "include", "clusterattn.h")).read()
    declared = set(re.findall(r"CA_API\s+[\w\s\*]+?\b(ca_\w+)\s*\(", hdr))
    assert declared == set(L.EXPORTS)
    for name in declared:
        assert hasattr(lib, name)
    assert lib.ca_abi_version() == 8


def _prob(**kw):
    from paper_2608_26965_amd import _lib as L
    base = dict(batch=1, heads=2, nq=1000, nk=1000, d=64, cq=64, ck=64, dtype=L.CA_BF16,
                transform=L.CA_XF_METRIC, layout=L.CA_LAYOUT_BHND, split=L.CA_SPLIT_DIAG)
    base.update(kw)
    return L.CaProblem(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(cq=48), 1), (dict(ck=512), 1), (dict(d=0), 1), (dict(d=129), 1), (dict(nq=0), 1),
    (dict(dtype=7), 1), (dict(transform=5), 1), (dict(split=2), 1),
    (dict(split=1, transform=1), 2), (dict(split=1, transform=3), 2), (dict(layout=3), 1), (dict(heads=0), 1),
])
def test_invalid_problem(kw, status):
    L, lib = _lib()
    n = ctypes.c_size_t(0)
    assert lib.ca_workspace_size(_prob(**kw), 1, n) == status
    assert L.last_error() != ""


def test_workspace_and_k_validation():
    L, lib = _lib()
    n = ctypes.c_size_t(0)
    assert lib.ca_workspace_size(_prob(), 16, n) == 0 and n.value > 0
    assert lib.ca_workspace_size(_prob(), 17, n) == L.CA_E_INVALID  # nkc = 16
    assert lib.ca_workspace_size(_prob(), 0, n) == L.CA_E_INVALID
    assert "k=0" in L.last_error()


def test_calls_reject_before_enqueue():
    L, lib = _lib()
    p = _prob()
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    out = L.CaClusterOut()
    assert lib.ca_cluster(p, None, fake, None, out, None, 0, None) == L.CA_E_INVALID
    assert lib.ca_cluster(p, fake, fake, None, out, None, 0, None) == L.CA_E_INVALID
    full = L.CaClusterOut(*([0x1000] * 14))
    assert lib.ca_cluster(p, fake, fake, None, full, fake, 16, None) == L.CA_E_WORKSPACE
    assert lib.ca_select(p, None, None, None, None, 4, fake, None, 0, None) == L.CA_E_INVALID
    assert lib.ca_select(p, fake, fake, None, None, 4, fake, None, 0, None) == L.CA_E_WORKSPACE
    args = [fake] * 5 + [None]  # qp, kp, vp, count_k, lists; lens omitted
    assert lib.ca_block_sparse_attn(p, *args, 0, 0.0, fake, fake, None, 0, None) == L.CA_E_INVALID
    assert lib.ca_block_sparse_attn(p, *args, 99, 0.0, fake, fake, None, 0, None) == L.CA_E_INVALID
    assert lib.ca_block_sparse_attn(_prob(d=48), *args, 2, 0.0, fake, fake, None, 0, None) == \
        L.CA_E_UNSUPPORTED
    assert lib.ca_block_sparse_attn(_prob(cq=32), *args, 2, 0.0, fake, fake, None, 0, None) == \
        L.CA_E_UNSUPPORTED
    # with list lengths, a workspace (for the schedule) is checked for its size
    largs = [fake] * 6  # ... and lens given
    assert lib.ca_block_sparse_attn(p, *largs, 2, 0.0, fake, fake, fake, 16, None) == \
        L.CA_E_WORKSPACE
    assert lib.ca_compensate(p, fake, fake, fake, fake, fake, None, 2, 0.0, 1, None, fake, fake,
                             fake, None, None, 0, None) == L.CA_E_INVALID
    assert lib.ca_compensate(p, None, None, None, None, None, None, 2, 0.0, 1, fake, fake, fake,
                             fake, None, None, 0, None) == L.CA_E_INVALID
    # bf16 with compensation stages the centroids in the workspace
    assert lib.ca_compensate(p, fake, fake, fake, fake, fake, None, 2, 0.0, 1, fake, fake, fake,
                             fake, None, fake, 16, None) == L.CA_E_WORKSPACE
    # ... also when every list may be full length but lengths are given
    assert lib.ca_compensate(p, fake, fake, fake, fake, fake, fake, 16, 0.0, 1, fake, fake, fake,
                             fake, None, fake, 16, None) == L.CA_E_WORKSPACE
    # steps 3 and 4 in one pass: (qp, kp, vp, cent_k, cent_v, count_k, lists, lens), k, scale,
    # enable, perm_q, out, lse_out, ws, ws_bytes, stream
    fa = [fake] * 7 + [None]
    assert lib.ca_attn_compensated(p, *fa, 2, 0.0, 1, None, fake, None, None, 0, None) == \
        L.CA_E_INVALID
    fb = [fake] * 3 + [None, None] + [fake] * 2 + [None]  # centroids missing
    assert lib.ca_attn_compensated(p, *fb, 2, 0.0, 1, fake, fake, None, None, 0, None) == \
        L.CA_E_INVALID
    assert lib.ca_attn_compensated(_prob(dtype=L.CA_F32), *fa, 2, 0.0, 1, fake, fake, None, None,
                                   0, None) == L.CA_E_UNSUPPORTED
    assert lib.ca_attn_compensated(p, *fa, 99, 0.0, 1, fake, fake, None, None, 0, None) == \
        L.CA_E_INVALID
    # the largest problem (2^22 keys in clusters of 64) has 65536 key clusters, what
    # the selection bitmap holds: accepted up to the workspace check; one key more
    # is not a valid problem
    big = _prob(nq=64, nk=1 << 22)
    assert lib.ca_attn_compensated(big, *fa, 2, 0.0, 1, fake, fake, None, fake, 16, None) == \
        L.CA_E_WORKSPACE
    assert lib.ca_attn_compensated(_prob(nq=64, nk=(1 << 22) + 1), *fa, 2, 0.0, 1, fake, fake,
                                   None, fake, 16, None) == L.CA_E_INVALID
    # compensation needs the workspace for the centroid tiles
    assert lib.ca_attn_compensated(p, *fa, 2, 0.0, 1, fake, fake, None, fake, 16, None) == \
        L.CA_E_WORKSPACE
    assert lib.ca_attn_compensated(p, *fa, 2, 0.0, 1, fake, fake, None, None, 0, None) == \
        L.CA_E_WORKSPACE
    # histogram selection: lists, lens and count_k are required; thresholds in range
    sh = [fake, fake, fake, None, None]  # cent_q, cent_k, count_k, scores_in, scores_out
    assert lib.ca_select_hist(p, *sh, 16, 0.5, 0.0, fake, None, None, 0, None) == L.CA_E_INVALID
    assert lib.ca_select_hist(p, *sh, 0, 0.5, 0.0, fake, fake, None, 0, None) == L.CA_E_INVALID
    assert lib.ca_select_hist(p, *sh, 4, 1.5, 0.0, fake, fake, None, 0, None) == L.CA_E_INVALID
    assert lib.ca_select_hist(p, *sh, 4, float("nan"), 0.0, fake, fake, None, 0, None) == \
        L.CA_E_INVALID
    assert lib.ca_select_hist(p, *sh, 4, 0.5, 0.0, fake, fake, fake, 16, None) == L.CA_E_WORKSPACE
    ws_misaligned = ctypes.c_void_p(0x1001)
    need = ctypes.c_size_t(0)
    lib.ca_workspace_size(p, 1, need)
    assert lib.ca_cluster(p, fake, fake, None, full, ws_misaligned, need.value, None) == \
        L.CA_E_INVALID
    assert "aligned" in L.last_error()


def test_status_strings():
    L, lib = _lib()
    for s in range(5):
        assert lib.ca_status_str(s).decode().startswith("CA_")


def test_noalloc_rejects_oversize_before_enqueue():
    """ca_attn_compensated_noalloc refuses a problem whose centroid tiles
    exceed the library's scratch array (CA_E_WORKSPACE, naming both sizes)
    before any HIP call, and validates like ca_attn_compensated."""
    L, lib = _lib()
    fake = 256
    big = _prob(heads=64, nq=4096, nk=1024 * 128, d=128, cq=128, ck=128)
    st = lib.ca_attn_compensated_noalloc(big, fake, fake, fake, fake, fake, fake, fake, None, 2,
                                         0.0, 1, fake, fake, None, None)
    assert st == L.CA_E_WORKSPACE
    assert "33554432" in L.last_error()
    # compensation off needs no scratch, so the same problem passes validation
    # up to the launch, which is not attempted here; a NULL output is refused
    assert lib.ca_attn_compensated_noalloc(big, fake, fake, fake, fake, fake, fake, fake, None, 2,
                                           0.0, 0, fake, None, None, None) == L.CA_E_INVALID
    assert lib.ca_attn_compensated_noalloc(_prob(dtype=L.CA_F32), fake, fake, fake, fake, fake,
                                           fake, fake, None, 2, 0.0, 1, fake, fake, None,
                                           None) == L.CA_E_UNSUPPORTED


def test_compensate_cluster_limit_only_when_compensating():
    """The compensation's per-query-cluster selection bitmap holds 65536 key
    clusters: more are refused (CA_E_UNSUPPORTED, with the count) when
    compensation runs, before anything is enqueued."""
    L, lib = _lib()
    fake = 256
    p = _prob(dtype=L.CA_F32, nq=64, nk=(1 << 21), cq=16, ck=16)  # 131072 key clusters
    st = lib.ca_compensate(p, fake, fake, fake, fake, fake, None, 2, 0.0, 1, fake, fake, fake,
                           fake, None, None, 0, None)
    assert st == L.CA_E_UNSUPPORTED
    assert "131072" in L.last_error()


def test_strided_layout_validation():
    """CA_LAYOUT_STRIDED: strides must be non-negative multiples of 16 bytes'
    worth of elements; strided tensors must be 16-byte aligned."""
    L, lib = _lib()
    fake = 256
    ok = dict(layout=L.CA_LAYOUT_STRIDED)
    P = L.CaProblem
    good = _prob(**ok)
    for name in ("q_stride", "k_stride", "v_stride", "out_stride"):
        getattr(good, name)[:] = [2 * 1000 * 64 * 3, 64, 3 * 2 * 64]
    n = ctypes.c_size_t(0)
    assert lib.ca_workspace_size(good, 2, n) == L.CA_OK
    bad = _prob(**ok)
    for name in ("q_stride", "k_stride", "v_stride", "out_stride"):
        getattr(bad, name)[:] = [2 * 1000 * 64 * 3, 64, 3 * 2 * 64]
    bad.k_stride[2] = 100  # not a multiple of 8 bf16 elements
    assert lib.ca_workspace_size(bad, 2, n) == L.CA_E_INVALID
    assert "k_stride[2]" in L.last_error()
    bad.k_stride[2] = -8
    assert lib.ca_workspace_size(bad, 2, n) == L.CA_E_INVALID
    # misaligned q is refused before anything is enqueued
    out = L.CaClusterOut(*([fake] * 12 + [None, None]))
    assert lib.ca_cluster(good, fake + 2, fake, fake, out, fake, 1 << 40, None) == L.CA_E_INVALID
    assert "16-byte aligned" in L.last_error()
    assert lib.ca_abi_version() == 8


def test_check_finite_validation():
    """ca_check_finite validates before enqueueing: q, k and flags required."""
    L, lib = _lib()
    fake = 256
    p = _prob()
    assert lib.ca_check_finite(p, fake, None, None, fake, None) == L.CA_E_INVALID
    assert lib.ca_check_finite(p, fake, fake, None, None, None) == L.CA_E_INVALID
    assert lib.ca_check_finite(_prob(d=0), fake, fake, None, fake, None) == L.CA_E_INVALID
    assert "NaN" in lib.ca_status_str(L.CA_E_NONFINITE).decode()
