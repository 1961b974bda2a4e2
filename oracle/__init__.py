"""ctypes wrapper around the float64 CPU oracle (oracle/ress_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
benchmark's CPU-baseline leg. The GPU product path never imports it, and it never
imports the product package.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libress_oracle.so")
_libs = {}

_dp = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")
_fp = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_u16 = np.ctypeslib.ndpointer(dtype=np.uint16, flags="C_CONTIGUOUS")
_u8 = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")
_i32 = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")


def _opt(ptr_type):
    """ndpointer that also accepts None."""

    class _Opt(ptr_type):
        @classmethod
        def from_param(cls, obj):
            if obj is None:
                return C.c_void_p(None)
            return ptr_type.from_param(obj)

    return _Opt


def lib(path: str | None = None):
    """The loaded oracle library (the one built from oracle/ress_oracle.c unless
    `path` names another build of the same source)."""
    path = _LIB_PATH if path is None else path
    if path not in _libs:
        if path == _LIB_PATH and not os.path.exists(path):
            from . import build as _b

            _b.build()
        L = C.CDLL(path)
        i, d = C.c_int, C.c_double
        L.ro_max_threads.restype = i
        L.ro_set_threads.argtypes = [i]
        L.ro_pool.argtypes = [i, i, i, i, _u16, _dp]
        L.ro_forced_blocks.argtypes = [i, i, i, _u8]
        L.ro_pooled_row.argtypes = [i, i, _dp, _dp, _dp, _dp, _dp]
        L.ro_scores_row.argtypes = [i, i, _dp, _dp, _dp, _dp, d, _dp, _dp]
        L.ro_objective.argtypes = [i, i, _dp, _dp, _dp, _dp, _u8, d, _opt(_dp), C.POINTER(d), C.POINTER(d)]
        L.ro_objective.restype = d
        L.ro_deltas.argtypes = [i, i, _dp, _dp, _dp, _dp, _dp, _u8, _u8, d, _dp]
        L.ro_swaps.argtypes = [i, d, i, i]
        L.ro_swaps.restype = i
        L.ro_select_row.argtypes = [i, i, _dp, _dp, _dp, _dp, _u8, i, i, d, d, i, i, i, d, _u8, _dp, _dp,
                                    C.POINTER(d), C.POINTER(d), C.POINTER(d), _opt(_dp), _opt(_u8),
                                    C.POINTER(i)]
        L.ro_select.argtypes = [i, i, i, i, i, i, _u16, _u16, _u16, _fp, _i32, i, d, d, i, i, i, d, i,
                                _opt(_i32), _i32, _i32, _opt(_dp), _opt(_dp), _opt(_dp), _opt(_dp)]
        L.ro_select.restype = i
        L.ro_attn_tokens.argtypes = [i, i, i, i, i, _u16, _u16, _u16, d, _opt(_i32), _opt(_i32), i,
                                     _i32, _i32, _dp]
        _libs[path] = L
    return _libs[path]


_active = [None]


class use_library:
    """Context manager: route the wrappers below to another build of the oracle
    source (the mutation tests use it to show that the pins catch planted errors)."""

    def __init__(self, path: str):
        self.path = path

    def __enter__(self):
        self.prev = _active[0]
        _active[0] = self.path
        return self

    def __exit__(self, *exc):
        _active[0] = self.prev
        return False


def _L():
    return lib(_active[0])


def max_threads() -> int:
    return _L().ro_max_threads()


def set_threads(n: int) -> None:
    _L().ro_set_threads(int(n))


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def pool(x: np.ndarray, b: int) -> np.ndarray:
    """Block means of bf16 bits x [H][N][D] -> float64 [H][n_blocks][D]."""
    x = _c(x, np.uint16)
    H, N, D = x.shape
    out = np.zeros((H, (N + b - 1) // b, D), dtype=np.float64)
    _L().ro_pool(H, N, D, b, x, out)
    return out


def forced_blocks(N: int, bk: int, n_special: int) -> np.ndarray:
    out = np.zeros((N + bk - 1) // bk, dtype=np.uint8)
    _L().ro_forced_blocks(N, bk, n_special, out)
    return out.astype(bool)


def pooled_row(qbar_i, kbar, vbar):
    """Eq. 1 for one row: returns (P [n_kb], vbar_i [D])."""
    kbar, vbar = _c(kbar, np.float64), _c(vbar, np.float64)
    nkb, D = kbar.shape
    P = np.zeros(nkb)
    vb = np.zeros(D)
    _L().ro_pooled_row(D, nkb, _c(qbar_i, np.float64), kbar, vbar, P, vb)
    return P, vb


def scores_row(P, vbar_i, vbar, M, eps=1e-4):
    """Eqs. 4-7: returns (s, key) for every key block."""
    vbar = _c(vbar, np.float64)
    nkb, D = vbar.shape
    s = np.zeros(nkb)
    key = np.zeros(nkb)
    _L().ro_scores_row(D, nkb, _c(P, np.float64), _c(vbar_i, np.float64), vbar,
                        _c(M, np.float64), float(eps), s, key)
    return s, key


def objective(P, vbar_i, vbar, M, inD, eps=1e-4):
    """Eqs. 10-12: returns (J, g, K, G) of the drop set inD."""
    vbar = _c(vbar, np.float64)
    nkb, D = vbar.shape
    g = np.zeros(D)
    K = C.c_double()
    G = C.c_double()
    J = _L().ro_objective(D, nkb, _c(P, np.float64), _c(vbar_i, np.float64), vbar,
                           _c(M, np.float64), _c(inD, np.uint8), float(eps), g, C.byref(K),
                           C.byref(G))
    return J, g, K.value, G.value


def deltas(P, s, vbar_i, vbar, M, inD, cand, eps=1e-4):
    """Eqs. 13-16: exact single-swap decrease dJ for each candidate."""
    vbar = _c(vbar, np.float64)
    nkb, D = vbar.shape
    dJ = np.full(nkb, np.nan)
    _L().ro_deltas(D, nkb, _c(P, np.float64), _c(s, np.float64), _c(vbar_i, np.float64), vbar,
                    _c(M, np.float64), _c(inD, np.uint8), _c(cand, np.uint8), float(eps), dJ)
    return dJ


def swaps(c: int, rho: float, r: int, swap_floor: int = 1) -> int:
    return _L().ro_swaps(int(c), float(rho), int(r), int(swap_floor))


# Selection criteria (the paper's comparisons, Table 2 and Fig. 8 (Sec. 6.1); see the list
# at the top of ress_oracle.c).
DRIFT, PROBABILITY, DRIFT_MAX_SWAP, DRIFT_MAX_FULL = 0, 1, 2, 3


def select_row(qbar_i, kbar, vbar, M, forced, c, rounds=5, rho=0.5, eps=1e-4, swap_floor=1,
               dense_row=False, criterion=DRIFT, cdf_tau=0.0):
    """Secs. 4.2-4.3 for one row, with the trajectory of drop sets."""
    kbar, vbar = _c(kbar, np.float64), _c(vbar, np.float64)
    nkb, D = kbar.shape
    kept = np.zeros(nkb, np.uint8)
    P = np.zeros(nkb)
    key = np.zeros(nkb)
    J0, Jb, mg = C.c_double(), C.c_double(), C.c_double()
    tJ = np.zeros(rounds + 1)
    tD = np.zeros((rounds + 1, nkb), np.uint8)
    ns = C.c_int()
    _L().ro_select_row(D, nkb, _c(qbar_i, np.float64), kbar, vbar, _c(M, np.float64),
                        _c(forced, np.uint8), int(c), int(rounds), float(rho), float(eps),
                        int(swap_floor), int(bool(dense_row)), int(criterion), float(cdf_tau), kept, P, key,
                        C.byref(J0),
                        C.byref(Jb), C.byref(mg), tJ, tD, C.byref(ns))
    n = ns.value
    return dict(kept=kept.astype(bool), P=P, key=key, J_init=J0.value, J_best=Jb.value,
                margin=mg.value, trace_J=tJ[:n], trace_D=tD[:n].astype(bool))


def select(q, k, v, gram, budgets, *, N, bq, bk, n_special, rounds=5, rho=0.5, eps=1e-4,
           swap_floor=1, dense_special_queries=True, rows=None, want_key=True, criterion=DRIFT,
           cdf_tau=0.0):
    """Selection for every row (rows=None) or for the flat rows h * n_qb + i given.
    Returns kept_count [R], kept_idx [R][n_kb], drift [R][2], key/prob [R][n_kb], margin [R]."""
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    H, _, D = q.shape
    nqb, nkb = (N + bq - 1) // bq, (N + bk - 1) // bk
    rws = None if rows is None else _c(rows, np.int32)
    R = H * nqb if rows is None else len(rws)
    kc = np.zeros(R, np.int32)
    ki = np.zeros((R, nkb), np.int32)
    drift = np.zeros((R, 2))
    key = np.zeros((R, nkb)) if want_key else None
    prob = np.zeros((R, nkb)) if want_key else None
    margin = np.zeros(R)
    _L().ro_select(H, N, D, bq, bk, n_special, q, k, v, _c(gram, np.float32),
                    _c(budgets, np.int32), int(rounds), float(rho), float(eps), int(swap_floor),
                    int(bool(dense_special_queries)), int(criterion), float(cdf_tau), R, rws, kc, ki, drift,
                    key, prob, margin)
    return dict(kept_count=kc, kept_idx=ki, drift=drift, key=key, prob=prob, margin=margin)


def attn_tokens(q, k, v, *, N, bq, bk, scale, sel_h, sel_t, kept_count=None, kept_idx=None):
    """Exact attention of the selected (head, token) queries; dense when kept_idx is None."""
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    H, _, D = q.shape
    sh, st = _c(sel_h, np.int32), _c(sel_t, np.int32)
    out = np.zeros((len(sh), D))
    kc = None if kept_idx is None else _c(kept_count, np.int32).reshape(-1)
    ki = None if kept_idx is None else _c(kept_idx, np.int32).reshape(-1)
    _L().ro_attn_tokens(H, N, D, bq, bk, q, k, v, float(scale), kc, ki, len(sh), sh, st, out)
    return out


def block_masking_change(q, k, v, gram, *, N, bq, bk, scale, h, i, blocks):
    """The reference measurement of Sec. 3 (Fig. 2) for query block i of head h:
    for each key block j in `blocks`, mask only block j and take the change in what
    attention writes into the residual stream, the Euclidean norm over the query
    block's tokens of W_O^h (O_t(B minus j) - O_t(B)), with ||W_O^h x||^2 = x^T M_h x.
    Returns float64 [len(blocks)]."""
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    H, _, D = q.shape
    n_qb, n_kb = (N + bq - 1) // bq, (N + bk - 1) // bk
    toks = np.arange(i * bq, min((i + 1) * bq, N), dtype=np.int32)
    heads = np.full(len(toks), h, np.int32)
    dense = attn_tokens(q, k, v, N=N, bq=bq, bk=bk, scale=scale, sel_h=heads, sel_t=toks)
    M = np.asarray(gram[h], dtype=np.float64)
    out = np.empty(len(blocks))
    for n, j in enumerate(blocks):
        keep = [b for b in range(n_kb) if b != j]
        kc = np.zeros((H, n_qb), np.int32)
        ki = np.full((H, n_qb, n_kb), -1, np.int32)
        kc[h, i] = len(keep)
        ki[h, i, :len(keep)] = keep
        d = attn_tokens(q, k, v, N=N, bq=bq, bk=bk, scale=scale, sel_h=heads, sel_t=toks, kept_count=kc,
                        kept_idx=ki) - dense
        out[n] = np.sqrt(max(float(np.einsum("td,de,te->", d, M, d)), 0.0))
    return out


def spearman(a, b) -> float:
    """Spearman rank correlation: the Pearson correlation of the two rankings,
    tied values sharing their average rank (nan if either ranking is constant)."""
    def ranks(x):
        x = np.asarray(x, dtype=np.float64)
        order = np.argsort(x, kind="mergesort")
        sx = x[order]
        r = np.empty(len(x))
        s = 0
        while s < len(x):
            e = s
            while e + 1 < len(x) and sx[e + 1] == sx[s]:
                e += 1
            r[order[s:e + 1]] = 0.5 * (s + e)
            s = e + 1
        return r
    ra, rb = ranks(a), ranks(b)
    ra -= ra.mean()
    rb -= rb.mean()
    den = np.sqrt(np.dot(ra, ra) * np.dot(rb, rb))
    return float(np.dot(ra, rb) / den) if den > 0 else float("nan")


def bf16_bits_nearest(x) -> np.ndarray:
    """float64 values rounded once to the nearest bf16 (ties to even), as uint16
    bit patterns (finite values in the normal range)."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                       # x = m 2^e, 0.5 <= |m| < 1
    r = np.ldexp(np.round(np.ldexp(m, 8)), e - 8)  # 8 significant bits, np.round: half to even
    return (r.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _f64(bits) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def qkv_projection(x, w_qkv, H: int):
    """The layer's QKV projection, [Q K V]_t = W_qkv x_t, from bf16 bits x [N][64H]
    and w_qkv [3*64H][64H], in float64, each output rounded once to bf16; returns
    the bits of q, k, v [H][N][64] (rows 64h .. 64h+63 of each third are head h)."""
    y = _f64(x) @ _f64(w_qkv).T              # [N][3*64H]
    N = y.shape[0]
    parts = y.reshape(N, 3, H, 64).transpose(1, 2, 0, 3)  # [3][H][N][64]
    b = bf16_bits_nearest(parts)
    return b[0], b[1], b[2]


def out_projection_residual(o, w_o, resid):
    """resid_t + W_O concat_h(O[h][t]) in float64 from bf16 bits o [H][N][64],
    w_o [64H][64H], resid [N][64H], rounded once to bf16 (bits [N][64H])."""
    H, N, D = np.asarray(o).shape
    flat = _f64(o).transpose(1, 0, 2).reshape(N, H * D)
    return bf16_bits_nearest(_f64(resid) + flat @ _f64(w_o).T)


def out_projection_f64(o_rows, w_o, resid=None):
    """What the attention sublayer adds to the residual stream, W_O concat_h(o_h)
    (Sec. 3, "The Right Objective"), plus resid if given, in float64 without any
    rounding. o_rows: float64 [n][64H] attention outputs of n tokens, channel
    64h + d for head h; w_o: bf16 bits [64H][64H] (out features x in features);
    resid: float [n][64H] or None. Returns float64 [n][64H]."""
    y = np.asarray(o_rows, dtype=np.float64) @ _f64(w_o).T
    return y if resid is None else y + np.asarray(resid, dtype=np.float64)


def head_major_rows(o, tokens=None):
    """Attention outputs o [H][N][64] (bf16 bits or float values) of the given
    tokens as float64 rows [n][64H] in the residual stream's channel order 64h + d."""
    o = np.asarray(o)
    x = _f64(o) if o.dtype == np.uint16 else o.astype(np.float64)
    if tokens is not None:
        x = x[:, np.asarray(tokens)]
    H, n, D = x.shape
    return x.transpose(1, 0, 2).reshape(n, H * D)


def block_drift_sq(a, b, gram, *, bq: int):
    """Per query block i of head h, the sum over its tokens t of
    (a_t - b_t)^T M_h (a_t - b_t) = ||W_O^h (a_t - b_t)||^2 (the masking
    measurement of Sec. 3), in float64; a, b float [H][N][D], gram [H][D][D].
    Returns float64 [H][n_qb]."""
    x = np.asarray(a, dtype=np.float64) - np.asarray(b, dtype=np.float64)
    M = np.asarray(gram, dtype=np.float64)
    H, N, _ = x.shape
    n_qb = (N + bq - 1) // bq
    out = np.zeros((H, n_qb))
    for h in range(H):
        q = np.einsum("td,de,te->t", x[h], M[h], x[h])
        for i in range(n_qb):
            out[h, i] = q[i * bq:min((i + 1) * bq, N)].sum()
    return out

