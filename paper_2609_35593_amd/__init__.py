"""Python binding of libress, the MI355X (gfx950) hot path of ReSS.

Thin ctypes marshalling over the C ABI in include/ress.h; the functions carry
the C entry points' names. Every step of the path runs in the HIP kernels of
libress.so: this module only checks tensor metadata, allocates outputs with
torch when the caller passes none, and passes pointers and the current stream.
There is no fallback: if libress.so is missing the import fails.
"""
from __future__ import annotations

import ctypes as C
import math
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libress.so")

RESS_OK = 0
RESS_E_INVALID_ARG = -1
RESS_E_UNSUPPORTED = -2
RESS_E_WORKSPACE = -3
RESS_E_HIP = -4
MAX_KEY_BLOCKS = 4096
NOALLOC_SCRATCH_BYTES = 48 << 20


class ress_shape(C.Structure):
    _fields_ = [("H", C.c_int), ("N", C.c_int), ("D", C.c_int), ("bq", C.c_int), ("bk", C.c_int),
                ("n_special_tail", C.c_int)]


class ress_select_params(C.Structure):
    _fields_ = [("rounds", C.c_int), ("rho", C.c_double), ("eps", C.c_double), ("swap_floor", C.c_int),
                ("dense_special_queries", C.c_int), ("criterion", C.c_int), ("cdf_tau", C.c_double),
                ("pooled_in_workspace", C.c_int)]


# Selection criteria (include/ress.h).
CRITERION_DRIFT, CRITERION_PROBABILITY, CRITERION_DRIFT_MAX_SWAP, CRITERION_DRIFT_MAX_FULL = 0, 1, 2, 3


class RessError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_string(status)} ({status})")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; g.build()'` "
                          "or `python paper_2609_35593_amd/build.py`")
    L = C.CDLL(LIB_PATH)
    vp, i, f, sz = C.c_void_p, C.c_int, C.c_float, C.c_size_t
    L.ress_status_string.argtypes = [i]
    L.ress_status_string.restype = C.c_char_p
    L.ress_select_workspace_size.argtypes = [C.POINTER(ress_shape), C.POINTER(sz)]
    L.ress_select_workspace_size.restype = i
    L.ress_select.argtypes = [C.POINTER(ress_shape), C.POINTER(ress_select_params), vp, vp, vp, vp, vp, vp, vp,
                              vp, vp, vp, vp, sz, vp]
    L.ress_select.restype = i
    L.ress_select_noalloc.argtypes = [C.POINTER(ress_shape), C.POINTER(ress_select_params), vp, vp, vp, vp, vp, vp,
                                      vp, vp, vp, vp, vp]
    L.ress_select_noalloc.restype = i
    L.ress_block_drift_sq.argtypes = [C.POINTER(ress_shape), vp, vp, vp, vp, vp]
    L.ress_block_drift_sq.restype = i
    L.ress_sparse_attn.argtypes = [C.POINTER(ress_shape), vp, vp, vp, vp, vp, f, vp, vp]
    L.ress_sparse_attn.restype = i
    L.ress_sparse_attn_out_f32.argtypes = [C.POINTER(ress_shape), vp, vp, vp, vp, vp, f, vp, vp]
    L.ress_sparse_attn_out_f32.restype = i
    L.ress_dense_attn.argtypes = [C.POINTER(ress_shape), vp, vp, vp, f, vp, vp]
    L.ress_qkv_proj_pool.argtypes = [C.POINTER(ress_shape), vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.ress_qkv_proj_pool.restype = i
    L.ress_out_proj_residual.argtypes = [C.POINTER(ress_shape), vp, vp, vp, vp, vp]
    L.ress_out_proj_residual.restype = i
    L.ress_out_proj_residual_f32.argtypes = [C.POINTER(ress_shape), vp, vp, vp, vp, vp]
    L.ress_out_proj_residual_f32.restype = i
    L.ress_dense_attn.restype = i
    return L


lib = _load()


def status_string(status: int) -> str:
    return lib.ress_status_string(int(status)).decode()


ress_status_string = status_string


def make_shape(H: int, N: int, *, bq: int, bk: int, n_special_tail: int = 0, D: int = 64) -> ress_shape:
    return ress_shape(int(H), int(N), int(D), int(bq), int(bk), int(n_special_tail))


def _ptr(t) -> int | None:
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream, device) -> int:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _check_qkv(q, k, v):
    for name, t in (("q", q), ("k", k), ("v", v)):
        if not (t.is_cuda and t.dtype == torch.bfloat16 and t.is_contiguous() and t.dim() == 3):
            raise ValueError(f"{name} must be a contiguous CUDA bfloat16 tensor [H][N][D]")
    if not (q.shape == k.shape == v.shape) or q.device != k.device or q.device != v.device:
        raise ValueError("q, k, v must share shape and device")


def _check_out(name, t, dtype, shape, device):
    """A caller-provided output (or workspace) tensor must match what the kernels write."""
    if not (t.is_cuda and t.device == device and t.dtype == dtype and t.is_contiguous()
            and tuple(t.shape) == tuple(shape)):
        raise ValueError(f"{name} must be a contiguous {dtype} tensor of shape {tuple(shape)} on {device}")


def _workspace_bytes(workspace, device):
    """Size in bytes of a caller's workspace tensor (the library checks it is enough)."""
    if not (workspace.is_cuda and workspace.device == device and workspace.is_contiguous()):
        raise ValueError(f"workspace must be a contiguous tensor on {device}")
    return workspace.numel() * workspace.element_size()


def ress_select_workspace_size(shape: ress_shape) -> int:
    n = C.c_size_t(0)
    st = lib.ress_select_workspace_size(C.byref(shape), C.byref(n))
    if st != RESS_OK:
        raise RessError(st, "ress_select_workspace_size")
    return n.value


def ress_select(q, k, v, gram, keep_budget, *, bq: int, bk: int, n_special_tail: int = 0,
                rounds: int = 5, rho: float = 0.5, eps: float = 1e-4, swap_floor: int = 1,
                dense_special_queries: bool = True, criterion: int = CRITERION_DRIFT, cdf_tau: float = 0.0,
                kept_count=None, kept_idx=None, drift=None, key_out=None, prob_out=None,
                want_drift: bool = True, want_debug: bool = False, workspace=None,
                pooled_in_workspace: bool = False, stream=None) -> dict:
    """Drift-based block selection for one layer (see include/ress.h).
    keep_budget: host int32 [H]. With pooled_in_workspace, `workspace` holds the
    pooled state written by ress_qkv_proj_pool (q, k, v give the shape only).
    Returns the output tensors in a dict."""
    _check_qkv(q, k, v)
    H, N, D = q.shape
    shape = make_shape(H, N, bq=bq, bk=bk, n_special_tail=n_special_tail, D=D)
    n_qb, n_kb = (N + bq - 1) // bq, (N + bk - 1) // bk
    dev = q.device
    _check_out("gram", gram, torch.float32, (H, D, D), dev)
    budget = np.ascontiguousarray(np.asarray(keep_budget, dtype=np.int32).reshape(-1))
    if budget.shape[0] != H:
        raise ValueError("keep_budget must hold one int per head")
    if kept_count is None:
        kept_count = torch.empty((H, n_qb), dtype=torch.int32, device=dev)
    if kept_idx is None:
        kept_idx = torch.empty((H, n_qb, n_kb), dtype=torch.int32, device=dev)
    if drift is None and want_drift:
        drift = torch.empty((H, n_qb, 2), dtype=torch.float64, device=dev)
    if want_debug:
        if key_out is None:
            key_out = torch.empty((H, n_qb, n_kb), dtype=torch.float64, device=dev)
        if prob_out is None:
            prob_out = torch.empty((H, n_qb, n_kb), dtype=torch.float64, device=dev)
    _check_out("kept_count", kept_count, torch.int32, (H, n_qb), dev)
    _check_out("kept_idx", kept_idx, torch.int32, (H, n_qb, n_kb), dev)
    for name, t, shp in (("drift", drift, (H, n_qb, 2)), ("key_out", key_out, (H, n_qb, n_kb)),
                         ("prob_out", prob_out, (H, n_qb, n_kb))):
        if t is not None:
            _check_out(name, t, torch.float64, shp, dev)
    need = ress_select_workspace_size(shape)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    ws_bytes = _workspace_bytes(workspace, dev)
    params = ress_select_params(int(rounds), float(rho), float(eps), int(swap_floor), int(bool(dense_special_queries)),
                                int(criterion), float(cdf_tau), int(bool(pooled_in_workspace)))
    st = lib.ress_select(C.byref(shape), C.byref(params), _ptr(q), _ptr(k), _ptr(v), _ptr(gram),
                         budget.ctypes.data, _ptr(kept_count), _ptr(kept_idx), _ptr(drift), _ptr(key_out),
                         _ptr(prob_out), _ptr(workspace), ws_bytes, _stream(stream, dev))
    if st != RESS_OK:
        raise RessError(st, "ress_select")
    return dict(kept_count=kept_count, kept_idx=kept_idx, drift=drift, key=key_out, prob=prob_out)


def ress_select_noalloc(q, k, v, gram, keep_budget, *, bq: int, bk: int, kept_count, kept_idx,
                        n_special_tail: int = 0, rounds: int = 5, rho: float = 0.5, eps: float = 1e-4,
                        swap_floor: int = 1, dense_special_queries: bool = True, criterion: int = CRITERION_DRIFT,
                        cdf_tau: float = 0.0, drift=None, key_out=None, prob_out=None, stream=None) -> dict:
    """ress_select with the library's fixed per-GPU scratch instead of a workspace
    (see include/ress.h): neither this binding nor the library allocates; every
    output is the caller's."""
    _check_qkv(q, k, v)
    H, N, D = q.shape
    shape = make_shape(H, N, bq=bq, bk=bk, n_special_tail=n_special_tail, D=D)
    n_qb, n_kb = (N + bq - 1) // bq, (N + bk - 1) // bk
    dev = q.device
    _check_out("gram", gram, torch.float32, (H, D, D), dev)
    budget = np.ascontiguousarray(np.asarray(keep_budget, dtype=np.int32).reshape(-1))
    if budget.shape[0] != H:
        raise ValueError("keep_budget must hold one int per head")
    _check_out("kept_count", kept_count, torch.int32, (H, n_qb), dev)
    _check_out("kept_idx", kept_idx, torch.int32, (H, n_qb, n_kb), dev)
    for name, t, shp in (("drift", drift, (H, n_qb, 2)), ("key_out", key_out, (H, n_qb, n_kb)),
                         ("prob_out", prob_out, (H, n_qb, n_kb))):
        if t is not None:
            _check_out(name, t, torch.float64, shp, dev)
    params = ress_select_params(int(rounds), float(rho), float(eps), int(swap_floor), int(bool(dense_special_queries)),
                                int(criterion), float(cdf_tau), 0)
    st = lib.ress_select_noalloc(C.byref(shape), C.byref(params), _ptr(q), _ptr(k), _ptr(v), _ptr(gram),
                                 budget.ctypes.data, _ptr(kept_count), _ptr(kept_idx), _ptr(drift), _ptr(key_out),
                                 _ptr(prob_out), _stream(stream, dev))
    if st != RESS_OK:
        raise RessError(st, "ress_select_noalloc")
    return dict(kept_count=kept_count, kept_idx=kept_idx, drift=drift, key=key_out, prob=prob_out)


def _sparse_call(fn, name, q, k, v, kept_count, kept_idx, bq, bk, n_special_tail, scale, out, out_dtype, stream):
    _check_qkv(q, k, v)
    H, N, D = q.shape
    shape = make_shape(H, N, bq=bq, bk=bk, n_special_tail=n_special_tail, D=D)
    n_qb, n_kb = (N + bq - 1) // bq, (N + bk - 1) // bk
    for name, t in (("kept_count", kept_count), ("kept_idx", kept_idx)):
        if not (t.is_cuda and t.device == q.device and t.dtype == torch.int32 and t.is_contiguous()):
            raise ValueError(f"{name} must be a contiguous int32 tensor on {q.device}")
    if kept_count.numel() != H * n_qb or kept_idx.numel() != H * n_qb * n_kb:
        raise ValueError("kept_count must be [H][n_qb] and kept_idx [H][n_qb][n_kb]")
    if out is None:
        out = torch.empty(q.shape, dtype=out_dtype, device=q.device)
    _check_out("out", out, out_dtype, q.shape, q.device)
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    st = fn(C.byref(shape), _ptr(q), _ptr(k), _ptr(v), _ptr(kept_count), _ptr(kept_idx), float(scale), _ptr(out),
            _stream(stream, q.device))
    if st != RESS_OK:
        raise RessError(st, name)
    return out


def ress_sparse_attn(q, k, v, kept_count, kept_idx, *, bq: int, bk: int, n_special_tail: int = 0,
                     scale: float | None = None, out=None, stream=None):
    """Block-sparse attention over the kept key blocks (see include/ress.h)."""
    return _sparse_call(lib.ress_sparse_attn, "ress_sparse_attn", q, k, v, kept_count, kept_idx, bq, bk,
                        n_special_tail, scale, out, torch.bfloat16, stream)


def ress_sparse_attn_out_f32(q, k, v, kept_count, kept_idx, *, bq: int, bk: int, n_special_tail: int = 0,
                             scale: float | None = None, out=None, stream=None):
    """ress_sparse_attn with a float32 output (see include/ress.h)."""
    return _sparse_call(lib.ress_sparse_attn_out_f32, "ress_sparse_attn_out_f32", q, k, v, kept_count, kept_idx,
                        bq, bk, n_special_tail, scale, out, torch.float32, stream)


def ress_dense_attn(q, k, v, *, bq: int, bk: int, n_special_tail: int = 0, scale: float | None = None,
                    out=None, stream=None):
    """Dense attention over every key block (see include/ress.h)."""
    _check_qkv(q, k, v)
    H, N, D = q.shape
    shape = make_shape(H, N, bq=bq, bk=bk, n_special_tail=n_special_tail, D=D)
    if out is None:
        out = torch.empty_like(q)
    _check_out("out", out, torch.bfloat16, q.shape, q.device)
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    st = lib.ress_dense_attn(C.byref(shape), _ptr(q), _ptr(k), _ptr(v), float(scale), _ptr(out),
                             _stream(stream, q.device))
    if st != RESS_OK:
        raise RessError(st, "ress_dense_attn")
    return out


def _check_bf16(name, t, shape):
    if not (t.is_cuda and t.dtype == torch.bfloat16 and t.is_contiguous() and tuple(t.shape) == tuple(shape)):
        raise ValueError(f"{name} must be a contiguous CUDA bfloat16 tensor of shape {tuple(shape)}")


def ress_qkv_proj_pool(x, w_qkv, gram, *, bq: int, bk: int, n_special_tail: int = 0, q=None, k=None, v=None,
                       workspace=None, stream=None) -> dict:
    """QKV projection with block pooling in its epilogue (see include/ress.h).
    x: bf16 [N][H*64]; w_qkv: bf16 [3*H*64][H*64]. Returns q, k, v (bf16
    [H][N][64]) and the workspace holding the pooled state, for ress_select(...,
    workspace=..., pooled_in_workspace=True)."""
    N, dm = x.shape
    H, D = dm // 64, 64
    _check_bf16("x", x, (N, dm))
    _check_bf16("w_qkv", w_qkv, (3 * dm, dm))
    dev = x.device
    if w_qkv.device != dev:
        raise ValueError("x and w_qkv must share a device")
    _check_out("gram", gram, torch.float32, (H, D, D), dev)
    shape = make_shape(H, N, bq=bq, bk=bk, n_special_tail=n_special_tail, D=D)
    q = torch.empty((H, N, D), dtype=torch.bfloat16, device=dev) if q is None else q
    k = torch.empty((H, N, D), dtype=torch.bfloat16, device=dev) if k is None else k
    v = torch.empty((H, N, D), dtype=torch.bfloat16, device=dev) if v is None else v
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check_out(name, t, torch.bfloat16, (H, N, D), dev)
    need = ress_select_workspace_size(shape)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    ws_bytes = _workspace_bytes(workspace, dev)
    st = lib.ress_qkv_proj_pool(C.byref(shape), _ptr(x), _ptr(w_qkv), _ptr(q), _ptr(k), _ptr(v), _ptr(gram),
                                _ptr(workspace), ws_bytes, _stream(stream, dev))
    if st != RESS_OK:
        raise RessError(st, "ress_qkv_proj_pool")
    return dict(q=q, k=k, v=v, workspace=workspace)


def ress_out_proj_residual(o, w_o, resid_in, *, resid_out=None, stream=None):
    """resid_out = resid_in + concat_h(o[h]) w_o^T (see include/ress.h).
    o: bf16 [H][N][64]; w_o: bf16 [H*64][H*64]; resid_in/out: bf16 [N][H*64]."""
    H, N, D = o.shape
    _check_bf16("o", o, (H, N, D))
    _check_bf16("w_o", w_o, (H * D, H * D))
    _check_bf16("resid_in", resid_in, (N, H * D))
    resid_out = torch.empty_like(resid_in) if resid_out is None else resid_out
    _check_bf16("resid_out", resid_out, (N, H * D))
    if not (w_o.device == resid_in.device == resid_out.device == o.device):
        raise ValueError("o, w_o, resid_in and resid_out must share a device")
    shape = make_shape(H, N, bq=128, bk=128, D=D)
    st = lib.ress_out_proj_residual(C.byref(shape), _ptr(o), _ptr(w_o), _ptr(resid_in), _ptr(resid_out),
                                    _stream(stream, o.device))
    if st != RESS_OK:
        raise RessError(st, "ress_out_proj_residual")
    return resid_out


def ress_out_proj_residual_f32(o, w_o, resid_in, *, resid_out=None, stream=None):
    """resid_out = resid_in + concat_h(o[h]) w_o^T with a float32 stream (see
    include/ress.h). o: bf16 [H][N][64]; w_o: bf16 [H*64][H*64]; resid_in/out:
    float32 [N][H*64] (resid_out may be resid_in)."""
    H, N, D = o.shape
    _check_bf16("o", o, (H, N, D))
    _check_bf16("w_o", w_o, (H * D, H * D))
    dev = o.device
    _check_out("resid_in", resid_in, torch.float32, (N, H * D), dev)
    resid_out = torch.empty_like(resid_in) if resid_out is None else resid_out
    _check_out("resid_out", resid_out, torch.float32, (N, H * D), dev)
    if w_o.device != dev:
        raise ValueError("o and w_o must share a device")
    shape = make_shape(H, N, bq=128, bk=128, D=D)
    st = lib.ress_out_proj_residual_f32(C.byref(shape), _ptr(o), _ptr(w_o), _ptr(resid_in), _ptr(resid_out),
                                        _stream(stream, dev))
    if st != RESS_OK:
        raise RessError(st, "ress_out_proj_residual_f32")
    return resid_out


def ress_block_drift_sq(a, b, gram, *, bq: int, out=None, stream=None):
    """Per query block sum over its tokens of (a_t - b_t)^T M_h (a_t - b_t) (see
    include/ress.h). a, b: float32 [H][N][64]; gram: float32 [H][64][64].
    Returns float64 [H][n_qb]."""
    H, N, D = a.shape
    dev = a.device
    for name, t in (("a", a), ("b", b)):
        _check_out(name, t, torch.float32, (H, N, D), dev)
    _check_out("gram", gram, torch.float32, (H, D, D), dev)
    n_qb = (N + bq - 1) // bq
    out = torch.empty((H, n_qb), dtype=torch.float64, device=dev) if out is None else out
    _check_out("out", out, torch.float64, (H, n_qb), dev)
    shape = make_shape(H, N, bq=bq, bk=bq, D=D)
    st = lib.ress_block_drift_sq(C.byref(shape), _ptr(a), _ptr(b), _ptr(gram), _ptr(out), _stream(stream, dev))
    if st != RESS_OK:
        raise RessError(st, "ress_block_drift_sq")
    return out


def bf16_from_bits(bits: np.ndarray, device) -> torch.Tensor:
    """Device bf16 tensor holding the given uint16 bit patterns."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).to(device)
