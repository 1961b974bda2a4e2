"""The C ABI library loads, exports every entry point include/ress.h declares, and
validates arguments on the host (CPU only: every call here fails validation or
has no work, so nothing reaches the GPU)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ress.h")


def declared_entry_points():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ress_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def ress():
    import paper_2609_35593_amd as r

    return r


def test_header_declares_the_boundary():
    assert declared_entry_points() == ["ress_block_drift_sq", "ress_dense_attn", "ress_out_proj_residual",
                                       "ress_out_proj_residual_f32",
                                       "ress_qkv_proj_pool", "ress_select", "ress_select_noalloc",
                                       "ress_select_workspace_size", "ress_sparse_attn", "ress_sparse_attn_out_f32",
                                       "ress_status_string"]


def test_library_exports_every_declared_symbol(ress):
    raw = C.CDLL(ress.LIB_PATH)
    for name in declared_entry_points():
        assert hasattr(raw, name), name


def test_status_strings(ress):
    for st in (0, -1, -2, -3, -4):
        assert ress.status_string(st).startswith("RESS_")
    assert "unknown" in ress.status_string(7)


def _ws(ress, **kw):
    base = dict(H=16, N=43968, bq=128, bk=128, n_special_tail=160)
    base.update(kw)
    H, N = base.pop("H"), base.pop("N")
    shape = ress.make_shape(H, N, **base)
    n = C.c_size_t(0)
    return ress.lib.ress_select_workspace_size(C.byref(shape), C.byref(n)), n.value


def test_workspace_size(ress):
    st, n = _ws(ress)
    assert st == 0
    align = lambda x: (x + 255) // 256 * 256
    # qbar, kbar, vbar (float64 [16][344][64]) and the per-block quadratic term [16][344]
    assert n == 3 * align(16 * 344 * 64 * 8) + align(16 * 344 * 8)
    assert _ws(ress, N=0, n_special_tail=0) == (0, 0)
    assert _ws(ress, H=0) == (0, 0)
    assert _ws(ress, N=4096 * 128, H=1, n_special_tail=0)[0] == 0
    assert _ws(ress, N=4096 * 128 + 1, H=1, n_special_tail=0)[0] == ress.RESS_E_UNSUPPORTED
    assert _ws(ress, bq=96)[0] == ress.RESS_E_UNSUPPORTED
    assert _ws(ress, H=257)[0] == ress.RESS_E_UNSUPPORTED
    assert _ws(ress, N=-1)[0] == ress.RESS_E_INVALID_ARG
    assert _ws(ress, N=(1 << 24) + 1, H=1, n_special_tail=0)[0] == ress.RESS_E_UNSUPPORTED
    assert _ws(ress, n_special_tail=43969)[0] == ress.RESS_E_INVALID_ARG
    shape = ress.make_shape(16, 100, bq=64, bk=64, D=32)
    assert ress.lib.ress_select_workspace_size(C.byref(shape), C.byref(C.c_size_t())) == ress.RESS_E_UNSUPPORTED


def _select_status(ress, shape, params, budgets, ws_bytes=1 << 30, ws_ptr=1 << 40, ptr=1 << 41, gram_ptr=None):
    arr = (C.c_int32 * len(budgets))(*budgets)
    p = C.c_void_p(ptr)
    gram = p if gram_ptr is None else C.c_void_p(gram_ptr)
    return ress.lib.ress_select(C.byref(shape), C.byref(params) if params is not None else None, p, p, p, gram,
                                C.cast(arr, C.c_void_p), p, p, None, None, None, C.c_void_p(ws_ptr), ws_bytes,
                                None)


def test_select_rejects_before_launch(ress):
    """Each invalid call returns its code from host validation (the fake device
    pointers are never dereferenced)."""
    shape = ress.make_shape(2, 1230, bq=64, bk=64, n_special_tail=30)  # 20 blocks, 2 forced
    good = ress.ress_select_params(5, 0.5, 1e-4, 1, 1)
    bad_rounds = ress.ress_select_params(33, 0.5, 1e-4, 1, 1)
    bad_eps = ress.ress_select_params(5, 0.5, 0.0, 1, 1)
    bad_rho = ress.ress_select_params(5, float("nan"), 1e-4, 1, 1)
    assert _select_status(ress, shape, bad_rounds, [6, 6]) == ress.RESS_E_INVALID_ARG
    assert _select_status(ress, shape, bad_eps, [6, 6]) == ress.RESS_E_INVALID_ARG
    assert _select_status(ress, shape, bad_rho, [6, 6]) == ress.RESS_E_INVALID_ARG
    assert _select_status(ress, shape, None, [6, 6]) == ress.RESS_E_INVALID_ARG
    for crit, tau in ((4, 0.0), (-1, 0.0), (1, 1.5), (1, -0.1), (1, float("nan")), (0, 0.5), (3, 0.2)):
        bad = ress.ress_select_params(5, 0.5, 1e-4, 1, 1, crit, tau)
        assert _select_status(ress, shape, bad, [6, 6]) == ress.RESS_E_INVALID_ARG, (crit, tau)
    assert _select_status(ress, shape, good, [19, 6]) == ress.RESS_E_INVALID_ARG  # > 18 candidates
    assert _select_status(ress, shape, good, [6, -1]) == ress.RESS_E_INVALID_ARG
    # two forced blocks already meet the two-block floor: c_h = 0 is allowed, the
    # workspace check comes next
    assert _select_status(ress, shape, good, [0, 6], ws_bytes=16) == ress.RESS_E_WORKSPACE
    assert _select_status(ress, shape, good, [6, 6], ws_ptr=(1 << 40) + 8) == ress.RESS_E_WORKSPACE
    one_forced = ress.make_shape(2, 1230, bq=64, bk=64, n_special_tail=10)  # only block 19 forced
    assert _select_status(ress, one_forced, good, [0, 6]) == ress.RESS_E_INVALID_ARG
    assert _select_status(ress, shape, good, [6, 6], ptr=0) == ress.RESS_E_INVALID_ARG
    assert _select_status(ress, shape, good, [6, 6], ptr=(1 << 41) + 8) == ress.RESS_E_INVALID_ARG  # q/k/v not 16-byte aligned
    assert _select_status(ress, shape, good, [6, 6], gram_ptr=(1 << 42) + 4) == ress.RESS_E_INVALID_ARG  # gram
    empty = ress.make_shape(0, 1230, bq=64, bk=64)
    assert _select_status(ress, empty, good, [], ptr=0, ws_ptr=0, ws_bytes=0) == ress.RESS_OK


def test_attention_rejects_before_launch(ress):
    shape = ress.make_shape(2, 1230, bq=64, bk=64)
    p = C.c_void_p(1 << 41)
    o = C.c_void_p(1 << 42)
    assert ress.lib.ress_dense_attn(C.byref(shape), p, C.c_void_p(1 << 43), C.c_void_p(1 << 44), 0.0, o,
                                    None) == ress.RESS_E_INVALID_ARG
    assert ress.lib.ress_dense_attn(C.byref(shape), p, C.c_void_p(1 << 43), C.c_void_p(1 << 44),
                                    float("inf"), o, None) == ress.RESS_E_INVALID_ARG
    assert ress.lib.ress_dense_attn(C.byref(shape), p, C.c_void_p(1 << 43), C.c_void_p(1 << 44), 0.125, p,
                                    None) == ress.RESS_E_INVALID_ARG  # o aliases q
    assert ress.lib.ress_sparse_attn(C.byref(shape), p, C.c_void_p(1 << 43), C.c_void_p(1 << 44), None, p,
                                     0.125, o, None) == ress.RESS_E_INVALID_ARG
    for fn in (ress.lib.ress_sparse_attn, ress.lib.ress_sparse_attn_out_f32):
        assert fn(C.byref(shape), p, C.c_void_p(1 << 43), C.c_void_p(1 << 44), p, p, 0.125, p,
                  None) == ress.RESS_E_INVALID_ARG  # o aliases q
        assert fn(C.byref(shape), p, C.c_void_p(1 << 43), C.c_void_p(1 << 44), p, p, 0.125,
                  C.c_void_p((1 << 42) + 4), None) == ress.RESS_E_INVALID_ARG  # o not 16-byte aligned
    for misaligned in ((p, C.c_void_p((1 << 43) + 2), C.c_void_p(1 << 44), o),
                       (p, C.c_void_p(1 << 43), C.c_void_p(1 << 44), C.c_void_p((1 << 42) + 8))):
        assert ress.lib.ress_dense_attn(C.byref(shape), misaligned[0], misaligned[1], misaligned[2], 0.125,
                                        misaligned[3], None) == ress.RESS_E_INVALID_ARG
    huge = ress.make_shape(1, (1 << 24) + 1, bq=128, bk=128)
    assert ress.lib.ress_dense_attn(C.byref(huge), p, p, p, 0.125, o, None) == ress.RESS_E_UNSUPPORTED
    bad = ress.make_shape(2, 1230, bq=32, bk=64)
    assert ress.lib.ress_dense_attn(C.byref(bad), p, p, p, 0.125, o, None) == ress.RESS_E_UNSUPPORTED
    empty = ress.make_shape(2, 0, bq=64, bk=64)
    assert ress.lib.ress_dense_attn(C.byref(empty), None, None, None, 0.125, None, None) == ress.RESS_OK


def test_projections_reject_before_launch(ress):
    """Validation of the fused projections (nothing is launched on these paths)."""
    p = [C.c_void_p((1 << 41) + (n << 30)) for n in range(6)]
    ws = C.c_void_p(1 << 40)
    shape = ress.make_shape(8, 1000, bq=128, bk=128)
    need = ress.ress_select_workspace_size(shape)
    qkv = ress.lib.ress_qkv_proj_pool
    assert qkv(C.byref(ress.make_shape(6, 1000, bq=128, bk=128)), p[0], p[1], p[2], p[3], p[4], p[5], ws, need,
               None) == ress.RESS_E_UNSUPPORTED  # H not a multiple of 4
    assert qkv(C.byref(shape), p[0], p[1], p[2], p[3], p[4], p[5], ws, need - 1, None) == ress.RESS_E_WORKSPACE
    assert qkv(C.byref(shape), p[0], p[1], p[2], p[3], p[4], p[5], C.c_void_p((1 << 40) + 64), need,
               None) == ress.RESS_E_WORKSPACE  # not 256-byte aligned
    assert qkv(C.byref(shape), p[0], p[1], p[0], p[3], p[4], p[5], ws, need, None) == ress.RESS_E_INVALID_ARG
    assert qkv(C.byref(shape), p[0], p[1], p[2], p[2], p[4], p[5], ws, need, None) == ress.RESS_E_INVALID_ARG
    assert qkv(C.byref(shape), p[0], None, p[2], p[3], p[4], p[5], ws, need, None) == ress.RESS_E_INVALID_ARG
    assert qkv(C.byref(shape), C.c_void_p((1 << 41) + 8), p[1], p[2], p[3], p[4], p[5], ws, need,
               None) == ress.RESS_E_INVALID_ARG  # x not 16-byte aligned
    assert qkv(C.byref(shape), p[0], p[1], p[2], p[3], p[4], C.c_void_p((1 << 41) + (5 << 30) + 4), ws, need,
               None) == ress.RESS_E_INVALID_ARG  # gram not 16-byte aligned
    empty = ress.make_shape(8, 0, bq=128, bk=128)
    assert qkv(C.byref(empty), None, None, None, None, None, None, None, 0, None) == ress.RESS_OK
    out = ress.lib.ress_out_proj_residual
    assert out(C.byref(ress.make_shape(2, 1000, bq=128, bk=128)), p[0], p[1], p[2], p[3],
               None) == ress.RESS_E_UNSUPPORTED
    assert out(C.byref(shape), p[0], p[1], p[2], p[0], None) == ress.RESS_E_INVALID_ARG  # resid_out aliases o
    assert out(C.byref(shape), p[0], p[1], p[2], None, None) == ress.RESS_E_INVALID_ARG
    assert out(C.byref(empty), None, None, None, None, None) == ress.RESS_OK
    out32 = ress.lib.ress_out_proj_residual_f32
    assert out32(C.byref(ress.make_shape(2, 1000, bq=128, bk=128)), p[0], p[1], p[2], p[3],
                 None) == ress.RESS_E_UNSUPPORTED
    assert out32(C.byref(shape), p[0], p[1], p[2], p[0], None) == ress.RESS_E_INVALID_ARG  # resid_out aliases o
    assert out32(C.byref(shape), p[0], p[1], p[2], p[1], None) == ress.RESS_E_INVALID_ARG  # resid_out aliases w_o
    assert out32(C.byref(shape), p[0], p[1], None, p[3], None) == ress.RESS_E_INVALID_ARG
    assert out32(C.byref(shape), p[0], p[1], C.c_void_p((1 << 41) + 4), p[3], None) == ress.RESS_E_INVALID_ARG
    assert out32(C.byref(empty), None, None, None, None, None) == ress.RESS_OK


def test_select_with_pooled_state_needs_no_qkv(ress):
    """pooled_in_workspace: q, k, v may be NULL; everything else is still checked."""
    shape = ress.make_shape(2, 1230, bq=64, bk=64)
    params = ress.ress_select_params(5, 0.5, 1e-4, 1, 1, 0, 0.0, 1)
    budget = np.array([6, 6], np.int32)
    need = ress.ress_select_workspace_size(shape)
    p = C.c_void_p(1 << 41)
    st = ress.lib.ress_select(C.byref(shape), C.byref(params), None, None, None, p, budget.ctypes.data, p, p, None,
                              None, None, C.c_void_p(1 << 40), need - 1, None)
    assert st == ress.RESS_E_WORKSPACE  # reached the workspace check: q, k, v were not required
    params.pooled_in_workspace = 0
    st = ress.lib.ress_select(C.byref(shape), C.byref(params), None, None, None, p, budget.ctypes.data, p, p, None,
                              None, None, C.c_void_p(1 << 40), need, None)
    assert st == ress.RESS_E_INVALID_ARG


def test_block_drift_sq_checks(ress):
    """ress_block_drift_sq rejects null, misaligned and aliasing arguments on the
    host (nothing reaches the GPU) and does nothing without work."""
    f = ress.lib.ress_block_drift_sq
    sh = ress.make_shape(4, 1000, bq=128, bk=128)
    p = [C.c_void_p((1 << 41) + (n << 30)) for n in range(4)]
    assert f(C.byref(sh), None, p[1], p[2], p[3], None) == ress.RESS_E_INVALID_ARG
    assert f(C.byref(sh), p[0], p[1], p[2], None, None) == ress.RESS_E_INVALID_ARG
    assert f(C.byref(sh), C.c_void_p((1 << 41) + 4), p[1], p[2], p[3], None) == ress.RESS_E_INVALID_ARG
    assert f(C.byref(sh), p[0], p[1], p[2], p[0], None) == ress.RESS_E_INVALID_ARG  # out aliases a
    assert f(C.byref(ress.make_shape(4, 1000, bq=96, bk=128)), p[0], p[1], p[2], p[3], None) == ress.RESS_E_UNSUPPORTED
    assert f(C.byref(ress.make_shape(4, 0, bq=128, bk=128)), None, None, None, None, None) == ress.RESS_OK
