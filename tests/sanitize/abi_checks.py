"""Host-side argument checks of the C ABI, run in a child process against a
build of the ABI layer with AddressSanitizer and UndefinedBehaviorSanitizer on
its host code (no GPU, no torch): every call fails validation or has no work.
Usage: python abi_checks.py <library>"""
import ctypes as C
import sys

import numpy as np

lib = C.CDLL(sys.argv[1])


class Shape(C.Structure):
    _fields_ = [("H", C.c_int), ("N", C.c_int), ("D", C.c_int), ("bq", C.c_int), ("bk", C.c_int),
                ("n_special_tail", C.c_int)]


class Params(C.Structure):
    _fields_ = [("rounds", C.c_int), ("rho", C.c_double), ("eps", C.c_double), ("swap_floor", C.c_int),
                ("dense_special_queries", C.c_int), ("criterion", C.c_int), ("cdf_tau", C.c_double),
                ("pooled_in_workspace", C.c_int)]


INVALID, UNSUPPORTED, WORKSPACE = -1, -2, -3
vp, sz = C.c_void_p, C.c_size_t
lib.ress_select_workspace_size.argtypes = [C.POINTER(Shape), C.POINTER(sz)]
lib.ress_select.argtypes = [C.POINTER(Shape), C.POINTER(Params)] + [vp] * 11 + [sz, vp]
lib.ress_select_noalloc.argtypes = [C.POINTER(Shape), C.POINTER(Params)] + [vp] * 11
lib.ress_sparse_attn.argtypes = [C.POINTER(Shape), vp, vp, vp, vp, vp, C.c_float, vp, vp]
lib.ress_dense_attn.argtypes = [C.POINTER(Shape), vp, vp, vp, C.c_float, vp, vp]
lib.ress_qkv_proj_pool.argtypes = [C.POINTER(Shape)] + [vp] * 7 + [sz, vp]
lib.ress_out_proj_residual.argtypes = [C.POINTER(Shape)] + [vp] * 5
lib.ress_out_proj_residual_f32.argtypes = [C.POINTER(Shape)] + [vp] * 5
lib.ress_block_drift_sq.argtypes = [C.POINTER(Shape)] + [vp] * 5
lib.ress_status_string.restype = C.c_char_p

checks = 0


def expect(got, want, what):
    global checks
    checks += 1
    assert got == want, (what, got, want)


for st in range(-6, 3):
    assert lib.ress_status_string(st)
p = [vp((1 << 41) + (n << 30)) for n in range(8)]
good = Shape(16, 43968, 64, 128, 128, 160)
n = sz(0)
expect(lib.ress_select_workspace_size(C.byref(good), C.byref(n)), 0, "workspace size")
need = n.value
for bad, want in ((Shape(16, 43968, 32, 128, 128, 160), UNSUPPORTED), (Shape(16, 43968, 64, 96, 128, 160), UNSUPPORTED),
                  (Shape(-1, 100, 64, 64, 64, 0), INVALID), (Shape(2, 100, 64, 64, 64, 101), INVALID),
                  (Shape(300, 100, 64, 64, 64, 0), UNSUPPORTED), (Shape(1, 64 * 4097, 64, 64, 64, 0), UNSUPPORTED)):
    expect(lib.ress_select_workspace_size(C.byref(bad), C.byref(n)), want, "bad shape")
expect(lib.ress_select_workspace_size(None, C.byref(n)), INVALID, "null shape")
expect(lib.ress_select_workspace_size(C.byref(good), None), INVALID, "null out")
budget = np.full(16, 84, np.int32)
prm = Params(5, 0.5, 1e-4, 1, 1, 0, 0.0, 0)
args = lambda ws, wsb: [p[0], p[1], p[2], p[3], budget.ctypes.data, p[4], p[5], None, None, None, ws, wsb, None]
expect(lib.ress_select(C.byref(good), C.byref(prm), *args(None, need)), WORKSPACE, "no workspace")
expect(lib.ress_select(C.byref(good), C.byref(prm), *args(p[6], need - 1)), WORKSPACE, "small workspace")
expect(lib.ress_select(C.byref(good), None, *args(p[6], need)), INVALID, "null params")
for field, value in (("rounds", -1), ("rounds", 33), ("rho", -0.5), ("eps", 0.0), ("criterion", 4), ("cdf_tau", 0.5),
                     ("swap_floor", -1)):
    bad = Params(5, 0.5, 1e-4, 1, 1, 0, 0.0, 0)
    setattr(bad, field, value)
    expect(lib.ress_select(C.byref(good), C.byref(bad), *args(p[6], need)), INVALID, field)
for b in (343, -1):
    bb = budget.copy()
    bb[3] = b
    expect(lib.ress_select(C.byref(good), C.byref(prm), p[0], p[1], p[2], p[3], bb.ctypes.data, p[4], p[5], None, None,
                           None, p[6], need, None), INVALID, "budget")
expect(lib.ress_select(C.byref(Shape(0, 100, 64, 64, 64, 0)), C.byref(prm), *args(None, 0)), 0, "empty")
expect(lib.ress_select_noalloc(C.byref(Shape(64, 137400, 64, 128, 128, 500)), C.byref(prm), p[0], p[1], p[2], p[3],
                               np.full(64, 100, np.int32).ctypes.data, p[4], p[5], None, None, None, None),
       UNSUPPORTED, "noalloc over its scratch")
for sh in (Shape(16, 43968, 64, 128, 128, 160), Shape(4, 1000, 64, 64, 128, 5)):
    expect(lib.ress_sparse_attn(C.byref(sh), p[0], p[1], p[2], None, p[4], 0.125, p[5], None), INVALID, "no lists")
    expect(lib.ress_sparse_attn(C.byref(sh), p[0], p[1], p[2], p[3], p[4], -1.0, p[5], None), INVALID, "scale")
    expect(lib.ress_dense_attn(C.byref(sh), p[0], p[1], p[2], 0.125, p[0], None), INVALID, "o aliases q")
    expect(lib.ress_dense_attn(C.byref(sh), vp((1 << 41) + 8), p[1], p[2], 0.125, p[5], None), INVALID, "alignment")
sh4 = Shape(4, 1000, 64, 128, 128, 0)
expect(lib.ress_qkv_proj_pool(C.byref(Shape(2, 1000, 64, 128, 128, 0)), *p[:7], sz(1 << 30), None), UNSUPPORTED, "H % 4")
expect(lib.ress_qkv_proj_pool(C.byref(sh4), p[0], p[1], p[0], p[3], p[4], p[5], p[6], sz(1 << 30), None), INVALID,
       "q aliases x")
expect(lib.ress_out_proj_residual(C.byref(sh4), p[0], p[1], p[2], p[0], None), INVALID, "resid_out aliases o")
expect(lib.ress_out_proj_residual_f32(C.byref(sh4), p[0], p[1], None, p[3], None), INVALID, "no resid_in")
expect(lib.ress_block_drift_sq(C.byref(sh4), None, p[1], p[2], p[3], None), INVALID, "drift sq null")
expect(lib.ress_block_drift_sq(C.byref(sh4), p[0], p[1], p[2], p[0], None), INVALID, "drift sq aliasing")
print(f"abi checks ok: {checks}", flush=True)
