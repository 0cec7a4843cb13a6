"""Host-only checks of the C ABI: the library loads, exports every declared entry point, its
pure host functions agree with the oracle, and every argument check returns its status before
anything is launched (these calls pass dummy, never-dereferenced pointers)."""

import ctypes
import os
import re

import pytest

from oracle import fenwick

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "libloglinear.h")

ll = pytest.importorskip("paper_2506_04761_amd", reason="libloglinear.so not built")
lib = ll.lib

FAKE = ctypes.c_void_p(4096)  # non-null, 256-aligned, never dereferenced by a failing check


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ll_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert {"ll_mamba2_fwd", "ll_gdn_fwd", "ll_num_levels", "ll_workspace_size",
            "ll_debug_level_map", "ll_status_string", "ll_supported"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_num_levels_matches_oracle():
    for T in list(range(1, 700)) + [2048, 8192, 65536]:
        assert ll.ll_num_levels(T) == fenwick.num_levels(T)
    assert ll.ll_num_levels(2 ** 20) == 21
    assert ll.ll_num_levels(0) == -1


def test_supported_shapes_cover_the_workloads():
    assert ll.ll_supported(ll.LL_MAMBA2, ll.LL_F32, 16, 16, 16)
    assert ll.ll_supported(ll.LL_MAMBA2, ll.LL_BF16, 64, 64, 64)
    assert ll.ll_supported(ll.LL_MAMBA2, ll.LL_BF16, 64, 128, 64)
    assert ll.ll_supported(ll.LL_MAMBA2, ll.LL_BF16, 64, 128, 128)
    assert not ll.ll_supported(ll.LL_MAMBA2, ll.LL_BF16, 64, 96, 128)
    assert not ll.ll_supported(ll.LL_MAMBA2, 7, 64, 128, 128)


def test_workspace_size():
    ws = ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, 1, 65536, 16, 128, 128, 64, 1)
    assert ws > 0 and ws % 256 == 0
    assert ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, 1, 65536, 16, 128, 128, 64, 0) > 0
    assert ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, 1, 100, 16, 128, 128, 64, 1) == 0  # T % C
    assert ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, 1, 192, 16, 128, 128, 48, 1) == 0  # C not 2^k
    assert ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, 0, 64, 1, 128, 128, 64, 1) == 0
    assert ll.ll_workspace_size(ll.LL_MAMBA2, 9, 1, 64, 1, 128, 128, 64, 1) == 0


def _m2(q=FAKE, k=FAKE, v=FAKE, la=FAKE, lam=FAKE, o=FAKE, B=1, T=128, H=2, dk=64, dv=64, C=64,
        dtype=1, ws=FAKE, wsb=1 << 40):
    return lib.ll_mamba2_fwd(q, k, v, la, lam, o, B, T, H, dk, dv, C, dtype, ws, wsb, None)


def _m2g(H=4, Hqk=2, q=FAKE, T=128, dk=64, dv=64, C=64):
    return lib.ll_mamba2_fwd_grouped(q, FAKE, FAKE, FAKE, FAKE, FAKE, 1, T, H, Hqk, dk, dv, C, 1, FAKE, 1 << 40, None)


def _m2n(q=FAKE, la=FAKE, lam=FAKE, o=FAKE, B=1, T=128, H=2, dk=64, dv=64, C=64, dtype=1):
    return lib.ll_mamba2_fwd_noalloc(q, FAKE, FAKE, la, lam, o, B, T, H, dk, dv, C, dtype, None)


def test_noalloc_checks_and_scratch_limit_return_before_launch():
    """The allocation-free forward runs the checks of ll_mamba2_fwd, then rejects arguments whose
    workspace exceeds its static scratch, all before touching a device."""
    assert _m2n(q=None) == ll._lib.LL_ERR_NULL_ARG
    assert _m2n(o=None) == ll._lib.LL_ERR_NULL_ARG
    assert _m2n(T=100) == ll._lib.LL_ERR_BAD_SHAPE
    assert _m2n(dk=96) == ll._lib.LL_ERR_UNSUPPORTED
    cap = ll.LL_NOALLOC_SCRATCH_BYTES
    # bf16, C = 64, d = 128 with lambda: the single-pass workspace, about 256 bytes per token and head
    for lam, T in ((FAKE, 16384), (None, 65536)):
        need = ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, 1, T, 16, 128, 128, 64, lam is not None)
        assert need > cap
        assert _m2n(lam=lam, T=T, H=16, dk=128, dv=128) == ll._lib.LL_ERR_SCRATCH
    assert ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, 1, 8192, 16, 128, 128, 64, 1) <= cap
    assert ll.ll_status_string(ll._lib.LL_ERR_SCRATCH).startswith("LL_ERR_SCRATCH")


def test_mamba2_grouped_argument_checks_return_before_launch():
    assert _m2g(q=None) == ll._lib.LL_ERR_NULL_ARG
    assert _m2g(Hqk=0) == ll._lib.LL_ERR_BAD_SHAPE
    assert _m2g(Hqk=3) == ll._lib.LL_ERR_BAD_SHAPE   # 4 heads do not split into groups of 3
    assert _m2g(Hqk=8) == ll._lib.LL_ERR_BAD_SHAPE   # more query/key heads than heads
    assert _m2g(T=100) == ll._lib.LL_ERR_BAD_SHAPE
    assert _m2g(dk=96) == ll._lib.LL_ERR_UNSUPPORTED


def test_decode_state_bytes():
    n = ll.ll_decode_state_bytes(2, 3, 64, 64, 10)
    assert n > 0 and n % 256 == 0 and n >= 2 * 3 * 10 * 64 * 64 * 4
    assert ll.ll_decode_state_bytes(0, 3, 64, 64, 10) == 0
    assert ll.ll_decode_state_bytes(2, 3, 64, 64, 0) == 0


def _dec(q=FAKE, state=FAKE, t=5, B=2, H=3, dk=64, dv=64, L=10, dtype=1, sb=1 << 40):
    return lib.ll_mamba2_decode_step(q, FAKE, FAKE, FAKE, FAKE, FAKE, state, sb, t, B, H, dk, dv, L, dtype, None)


def test_decode_argument_checks_return_before_launch():
    assert _dec(q=None) == ll._lib.LL_ERR_NULL_ARG
    assert _dec(state=None) == ll._lib.LL_ERR_NULL_ARG
    assert _dec(B=0) == ll._lib.LL_ERR_BAD_SHAPE
    assert _dec(t=-1) == ll._lib.LL_ERR_BAD_SHAPE
    assert _dec(t=512, L=10) == ll._lib.LL_ERR_BAD_SHAPE     # 10 levels hold tokens t < 2^9
    assert _dec(dk=96) == ll._lib.LL_ERR_UNSUPPORTED
    assert _dec(dtype=4) == ll._lib.LL_ERR_UNSUPPORTED
    assert _dec(L=33) == ll._lib.LL_ERR_UNSUPPORTED
    assert _dec(sb=1000) == ll._lib.LL_ERR_WORKSPACE
    assert _dec(state=ctypes.c_void_p(4096 + 16)) == ll._lib.LL_ERR_WORKSPACE
    assert lib.ll_mamba2_decode_init(None, 1 << 40, 2, 3, 64, 64, 10, 1, None) == ll._lib.LL_ERR_NULL_ARG
    assert lib.ll_mamba2_decode_init(FAKE, 1000, 2, 3, 64, 64, 10, 1, None) == ll._lib.LL_ERR_WORKSPACE


def test_gdn_decode_argument_checks_return_before_launch():
    def d(beta=FAKE, t=5, L=10, dk=64, sb=1 << 40):
        return lib.ll_gdn_decode_step(FAKE, FAKE, FAKE, FAKE, beta, FAKE, FAKE, FAKE, sb, t, 2, 3, dk, 64, L, 1, None)
    assert d(beta=None) == ll._lib.LL_ERR_NULL_ARG
    assert d(t=512) == ll._lib.LL_ERR_BAD_SHAPE
    assert d(dk=96) == ll._lib.LL_ERR_UNSUPPORTED
    assert d(sb=1000) == ll._lib.LL_ERR_WORKSPACE
    assert lib.ll_gdn_decode_init(None, 1 << 40, 2, 3, 64, 64, 10, 1, None) == ll._lib.LL_ERR_NULL_ARG


def test_mamba2_argument_checks_return_before_launch():
    assert _m2(q=None) == ll._lib.LL_ERR_NULL_ARG
    assert _m2(la=None) == ll._lib.LL_ERR_NULL_ARG
    assert _m2(o=None) == ll._lib.LL_ERR_NULL_ARG
    assert _m2(ws=None) == ll._lib.LL_ERR_NULL_ARG
    assert _m2(T=100) == ll._lib.LL_ERR_BAD_SHAPE
    assert _m2(C=48, T=96) == ll._lib.LL_ERR_BAD_SHAPE
    assert _m2(B=0) == ll._lib.LL_ERR_BAD_SHAPE
    assert _m2(H=0) == ll._lib.LL_ERR_BAD_SHAPE
    assert _m2(dk=96) == ll._lib.LL_ERR_UNSUPPORTED
    assert _m2(dtype=5) == ll._lib.LL_ERR_UNSUPPORTED
    assert _m2(C=32, T=128) == ll._lib.LL_ERR_UNSUPPORTED
    assert _m2(wsb=1000) == ll._lib.LL_ERR_WORKSPACE
    assert _m2(ws=ctypes.c_void_p(4096 + 8)) == ll._lib.LL_ERR_WORKSPACE


def _bwd(lam=FAKE, do=FAKE, dla=FAKE, T=128, dk=64, dv=64, C=64, dtype=1, ws=FAKE, wsb=1 << 40, staged=False, ev=None,
         Hqk=None):
    ptrs = [FAKE, FAKE, FAKE, FAKE, lam, do, FAKE, FAKE, FAKE, dla, FAKE]
    tail = [dk, dv, C, dtype, ws, wsb, None]
    if staged:
        return lib.ll_mamba2_bwd_staged(*ptrs, 1, T, 2, 2 if Hqk is None else Hqk, *tail, ev)
    if Hqk is not None:
        return lib.ll_mamba2_bwd_grouped(*ptrs, 1, T, 2, Hqk, *tail)
    return lib.ll_mamba2_bwd(*ptrs, 1, T, 2, *tail)


def test_mamba2_bwd_argument_checks_return_before_launch():
    assert _bwd(lam=None) == ll._lib.LL_ERR_NULL_ARG     # lambda is required by the backward
    assert _bwd(do=None) == ll._lib.LL_ERR_NULL_ARG
    assert _bwd(dla=None) == ll._lib.LL_ERR_NULL_ARG
    assert _bwd(ws=None) == ll._lib.LL_ERR_NULL_ARG
    assert _bwd(T=100) == ll._lib.LL_ERR_BAD_SHAPE
    assert _bwd(dk=96) == ll._lib.LL_ERR_UNSUPPORTED
    assert _bwd(dtype=3) == ll._lib.LL_ERR_UNSUPPORTED
    assert _bwd(wsb=1000) == ll._lib.LL_ERR_WORKSPACE
    assert _bwd(ws=ctypes.c_void_p(4096 + 64)) == ll._lib.LL_ERR_WORKSPACE
    assert _bwd(staged=True, ev=None) == ll._lib.LL_ERR_NULL_ARG
    assert _bwd(staged=True, ev=(ctypes.c_void_p * 5)(4096, 4096, None, 4096, 4096)) == ll._lib.LL_ERR_NULL_ARG
    assert _bwd(Hqk=0) == ll._lib.LL_ERR_BAD_SHAPE
    assert _bwd(Hqk=3) == ll._lib.LL_ERR_BAD_SHAPE   # more query/key heads than heads
    assert _bwd(Hqk=1, lam=None) == ll._lib.LL_ERR_NULL_ARG
    assert _bwd(Hqk=1, wsb=1000) == ll._lib.LL_ERR_WORKSPACE


def test_mamba2_bwd_after_fwd_argument_checks():
    def c(lam=FAKE, ws=FAKE, wsb=1 << 40, T=128):
        return lib.ll_mamba2_bwd_after_fwd(FAKE, FAKE, FAKE, FAKE, lam, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, T, 2,
                                           2, 64, 64, 64, 1, ws, wsb, None)
    assert c(lam=None) == ll._lib.LL_ERR_NULL_ARG
    assert c(ws=None) == ll._lib.LL_ERR_NULL_ARG
    assert c(T=100) == ll._lib.LL_ERR_BAD_SHAPE
    assert c(wsb=1000) == ll._lib.LL_ERR_WORKSPACE


def test_mamba2_bwd_workspace_and_support():
    for shape in ((ll.LL_F32, 16, 16, 16), (ll.LL_BF16, 64, 128, 128), (ll.LL_BF16, 64, 128, 64)):
        assert ll.ll_supported(ll.LL_MAMBA2_BWD, *shape)
    assert not ll.ll_supported(ll.LL_MAMBA2_BWD, ll.LL_BF16, 64, 96, 64)
    fwd = ll.ll_workspace_size(ll.LL_MAMBA2, ll.LL_BF16, 1, 65536, 16, 128, 128, 64, 1)
    bwd = ll.ll_workspace_size(ll.LL_MAMBA2_BWD, ll.LL_BF16, 1, 65536, 16, 128, 128, 64, 1)
    assert bwd > fwd and bwd % 256 == 0
    assert ll.ll_workspace_size(ll.LL_MAMBA2_BWD, ll.LL_BF16, 1, 65536, 16, 128, 128, 64, 0) == 0
    assert ll.ll_workspace_size(ll.LL_MAMBA2_BWD, ll.LL_BF16, 1, 64, 1, 128, 128, 64, 1) > 0
    ws = lib.ll_mamba2_bwd_workspace_size
    assert ws(ll.LL_BF16, 2, 16384, 48, 48, 128, 64, 64) == \
        ll.ll_workspace_size(ll.LL_MAMBA2_BWD, ll.LL_BF16, 2, 16384, 48, 128, 64, 64, 1)
    # shared heads add per-head dq and dk scratch (2 x B T H d_k bf16)
    assert ws(ll.LL_BF16, 2, 16384, 48, 1, 128, 64, 64) >= ws(ll.LL_BF16, 2, 16384, 48, 48, 128, 64, 64) + \
        2 * 2 * 16384 * 48 * 128 * 2
    assert ws(ll.LL_BF16, 2, 16384, 48, 5, 128, 64, 64) == 0


def test_size_limits_return_before_launch():
    # B * H beyond the second grid dimension; more tiles than a sequence may have
    assert _m2(B=300, H=300) == ll._lib.LL_ERR_UNSUPPORTED
    assert _m2(T=128 * 8193) == ll._lib.LL_ERR_UNSUPPORTED
    assert lib.ll_mamba2_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 300, 128, 300, 64, 64, 64, 1,
                             FAKE, 1 << 40, None) == ll._lib.LL_ERR_UNSUPPORTED


def test_gdn_argument_checks_return_before_launch():
    def g(beta=FAKE, T=128, ws=FAKE, wsb=1 << 40, dk=128, dv=128):
        return lib.ll_gdn_fwd(FAKE, FAKE, FAKE, FAKE, beta, FAKE, FAKE, 1, T, 2, dk, dv, 64, 1, ws, wsb, None)
    assert g(beta=None) == ll._lib.LL_ERR_NULL_ARG
    assert g(T=100) == ll._lib.LL_ERR_BAD_SHAPE
    assert g(dk=96) == ll._lib.LL_ERR_UNSUPPORTED
    assert ll.ll_supported(ll.LL_GDN, ll.LL_BF16, 64, 128, 128)
    assert not ll.ll_supported(ll.LL_GDN, ll.LL_F32, 64, 128, 128)


def test_debug_level_map_checks():
    assert lib.ll_debug_level_map(64, 16, None, None) == ll._lib.LL_ERR_NULL_ARG
    assert lib.ll_debug_level_map(60, 16, FAKE, None) == ll._lib.LL_ERR_BAD_SHAPE
    assert lib.ll_debug_level_map(1 << 15, 16, FAKE, None) == ll._lib.LL_ERR_UNSUPPORTED


def test_status_strings():
    for s in range(7):
        assert ll.ll_status_string(s).startswith("LL_")


def _ml(lam=FAKE, form=0, T=128, dk=64, dv=64, C=64, dtype=1, ws=FAKE, wsb=1 << 40, staged=False, ev=None, B=1, H=2):
    args = [FAKE, FAKE, FAKE, FAKE, lam, form, FAKE, B, T, H, dk, dv, C, dtype, ws, wsb, None]
    if staged:
        return lib.ll_mamba2_fwd_matrix_lambda_staged(*args, ev)
    return lib.ll_mamba2_fwd_matrix_lambda(*args)


def test_matrix_lambda_argument_checks_return_before_launch():
    assert _ml(lam=None) == ll._lib.LL_ERR_NULL_ARG
    assert _ml(ws=None) == ll._lib.LL_ERR_NULL_ARG
    assert _ml(form=2) == ll._lib.LL_ERR_BAD_SHAPE
    assert _ml(lam=ctypes.c_void_p(4096 + 4)) == ll._lib.LL_ERR_BAD_SHAPE   # Lambda must be 16-byte aligned
    assert _ml(T=100) == ll._lib.LL_ERR_BAD_SHAPE
    assert _ml(dk=96) == ll._lib.LL_ERR_UNSUPPORTED
    assert _ml(dtype=7) == ll._lib.LL_ERR_UNSUPPORTED
    assert _ml(B=300, H=300) == ll._lib.LL_ERR_UNSUPPORTED
    assert _ml(wsb=1000) == ll._lib.LL_ERR_WORKSPACE
    assert _ml(ws=ctypes.c_void_p(4096 + 8)) == ll._lib.LL_ERR_WORKSPACE
    assert _ml(staged=True, ev=None) == ll._lib.LL_ERR_NULL_ARG
    five_nulls = (ctypes.c_void_p * 5)()
    assert _ml(staged=True, ev=five_nulls) == ll._lib.LL_ERR_NULL_ARG


def test_matrix_lambda_workspace_size():
    ws = lib.ll_mamba2_matrix_lambda_workspace_size
    for dtype, esize, C, dk, dv in ((ll.LL_F32, 4, 16, 16, 16), (ll.LL_BF16, 2, 64, 128, 128)):
        B, T, H = 2, 4096, 3
        L = ll.ll_num_levels(T)
        # diagonal weights: the three-kernel forward's summaries only; full matrices: those (rounded
        # up to 256 bytes), then the level queries
        diag = ws(ll.LL_LAMBDA_DIAG, dtype, B, T, H, dk, dv, C)
        assert diag > 0
        assert ws(ll.LL_LAMBDA_FULL, dtype, B, T, H, dk, dv, C) == (diag + 255) // 256 * 256 + B * T * H * L * dk * esize
        if dtype == ll.LL_F32:  # the scalar-weight forward of this shape uses the same summaries
            assert diag == ll.ll_workspace_size(ll.LL_MAMBA2, dtype, B, T, H, dk, dv, C, 1)
    assert ws(ll.LL_LAMBDA_FULL, ll.LL_BF16, 1, 100, 1, 64, 64, 64) == 0
    assert ws(ll.LL_LAMBDA_FULL, 9, 1, 128, 1, 64, 64, 64) == 0
    assert ws(2, ll.LL_BF16, 1, 128, 1, 64, 64, 64) == 0
