"""CPU fp64 oracle of the WaveFilter filter+attend path -- TEST INFRASTRUCTURE.

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this module.  The product path never does.  It wraps the plain C
implementation in ``wf_oracle.c`` (see that file for the paper passages each
step follows) with numpy in / numpy out helpers; all arithmetic is in float64.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wf_oracle.c")
_LIB = os.path.join(_HERE, "libwf_oracle.so")

HAAR, DB2 = 0, 1
SYMMETRIC, PERIODIC = 0, 1

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2 -fopenmp); returns the library path."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-std=c99", "-Wall", "-Wextra", "-o", tmp, _SRC,
                               "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    dp = ctypes.POINTER(ctypes.c_double)
    lp = ctypes.POINTER(ctypes.c_long)
    i, l, d = ctypes.c_int, ctypes.c_long, ctypes.c_double
    lib.wf_ref_dwt.argtypes = [dp, i, i, i, i, i, dp, dp]
    lib.wf_ref_skim.argtypes = [dp, dp, i, i, i, d, dp]
    lib.wf_ref_topk.argtypes = [dp, l, l, lp]
    lib.wf_ref_scan.argtypes = [dp, dp, i, i, i, i, lp, i, l, d, dp, lp]
    lib.wf_ref_attn.argtypes = [dp, dp, dp, lp, l, dp, dp, l, i, i, d, dp]
    lib.wf_ref_filter_attend_unit.argtypes = [
        dp, dp, dp, dp, dp, i, i, i, i, i, i, i, i, l, d, dp, dp, dp, lp, dp, lp]
    lib.wf_ref_filter_attend.argtypes = [
        dp, dp, dp, dp, dp, i, i, i, i, i, i, i, i, i, l, d, dp, lp]
    lib.wf_ref_max_threads.argtypes = []
    lib.wf_ref_recursion_count.argtypes = [d, l]
    lib.wf_ref_recursion_count.restype = ctypes.c_long
    lib.wf_ref_recursive_select.argtypes = [dp, dp, i, i, i, i, i, i, dp, d,
                                            lp, lp, lp]
    lib.wf_ref_filter_attend_recursive.argtypes = [
        dp, dp, dp, dp, dp, i, i, i, i, i, i, i, i, dp, d, dp, lp, lp]
    for name in ("wf_ref_dwt", "wf_ref_skim", "wf_ref_topk", "wf_ref_scan",
                 "wf_ref_attn", "wf_ref_filter_attend_unit",
                 "wf_ref_filter_attend", "wf_ref_max_threads",
                 "wf_ref_recursive_select", "wf_ref_filter_attend_recursive"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _f64(x) -> np.ndarray:
    if hasattr(x, "detach"):  # torch tensor: exact upcast of bf16 / fp32
        import torch
        x = x.detach().to("cpu", torch.float64).numpy()
    return np.ascontiguousarray(x, dtype=np.float64)


def _i64(x) -> np.ndarray:
    if hasattr(x, "detach"):
        x = x.detach().cpu().numpy()
    return np.ascontiguousarray(x, dtype=np.int64)


def _dp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _lp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_long))


def _null_d():
    return ctypes.POINTER(ctypes.c_double)()


def _null_l():
    return ctypes.POINTER(ctypes.c_long)()


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments")


def wavelet_code(name: str) -> int:
    return {"haar": HAAR, "db2": DB2}[name]


def boundary_code(name: str) -> int:
    return {"symmetric": SYMMETRIC, "periodic": PERIODIC}[name]


def default_scale(d: int) -> float:
    return 1.0 / np.sqrt(d)


def dwt(x, levels: int, wavelet: str = "haar", boundary: str = "symmetric",
        details: bool = False):
    """O1.  x [L, d] -> A_J [L>>J, d] (and [D_1, ..., D_J] if details)."""
    x = _f64(x)
    if x.ndim == 1:
        x = x[:, None]
    L, d = x.shape
    A = np.empty((L >> levels, d))
    nd = sum(L >> j for j in range(1, levels + 1))
    D = np.empty((nd, d)) if details else None
    _check(_load().wf_ref_dwt(_dp(x), L, d, levels, wavelet_code(wavelet),
                              boundary_code(boundary), _dp(A),
                              _dp(D) if details else _null_d()), "dwt")
    if not details:
        return A
    out, row = [], 0
    for j in range(1, levels + 1):
        out.append(D[row:row + (L >> j)])
        row += L >> j
    return A, out


def skim(Q, A, scale: float | None = None) -> np.ndarray:
    """O2.  Q [B, d], A [n, d] -> W [n]."""
    Q, A = _f64(Q), _f64(A)
    B, d = Q.shape
    n = A.shape[0]
    scale = default_scale(d) if scale is None else scale
    W = np.empty(n)
    _check(_load().wf_ref_skim(_dp(Q), _dp(A), B, n, d, scale, _dp(W)), "skim")
    return W


def topk(score, k: int) -> np.ndarray:
    """O3/O6.  The k best positions (ties to the lower index), ascending."""
    s = _f64(score).ravel()
    out = np.empty(k, dtype=np.int64)
    _check(_load().wf_ref_topk(_dp(s), s.size, k, _lp(out)), "topk")
    return out


def scan(Q, K, seg, levels: int, budget: int, scale: float | None = None):
    """O4-O6.  Returns (W' over the pool [S 2^J], tok [k_eff] ascending)."""
    Q, K, seg = _f64(Q), _f64(K), _i64(seg)
    B, d = Q.shape
    L = K.shape[0]
    S = seg.size
    P = S << levels
    keff = min(budget, P)
    scale = default_scale(d) if scale is None else scale
    Wp = np.empty(P)
    tok = np.empty(keff, dtype=np.int64)
    _check(_load().wf_ref_scan(_dp(Q), _dp(K), B, L, d, levels, _lp(seg), S,
                               budget, scale, _dp(Wp), _lp(tok)), "scan")
    return Wp, tok


def attend(Q, K, V, tok, Kg=None, Vg=None, scale: float | None = None):
    """O7-O8.  Attention of Q over [K[tok]; Kg] / [V[tok]; Vg]."""
    Q, K, V, tok = _f64(Q), _f64(K), _f64(V), _i64(tok)
    B, d = Q.shape
    G = 0 if Kg is None else int(Kg.shape[0])
    kg = _f64(Kg) if G else None
    vg = _f64(Vg) if G else None
    scale = default_scale(d) if scale is None else scale
    O = np.empty((B, d))
    _check(_load().wf_ref_attn(_dp(Q), _dp(K), _dp(V), _lp(tok), tok.size,
                               _dp(kg) if G else _null_d(),
                               _dp(vg) if G else _null_d(), G, B, d, scale,
                               _dp(O)), "attn")
    return O


def filter_attend_unit(Q, K, V, levels: int, segments: int, budget: int,
                       wavelet: str = "haar", boundary: str = "symmetric",
                       Kg=None, Vg=None, scale: float | None = None) -> dict:
    """O1-O8 for one unit; returns every intermediate as a dict."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    B, d = Q.shape
    L = K.shape[0]
    G = 0 if Kg is None else int(Kg.shape[0])
    kg = _f64(Kg) if G else None
    vg = _f64(Vg) if G else None
    n = L >> levels
    P = segments << levels
    keff = min(budget, P)
    scale = default_scale(d) if scale is None else scale
    out = dict(O=np.empty((B, d)), approx=np.empty((n, d)), W=np.empty(n),
               seg=np.empty(segments, dtype=np.int64), Wp=np.empty(P),
               tok=np.empty(keff, dtype=np.int64))
    _check(_load().wf_ref_filter_attend_unit(
        _dp(Q), _dp(K), _dp(V), _dp(kg) if G else _null_d(),
        _dp(vg) if G else _null_d(), L, d, B, G, levels,
        wavelet_code(wavelet), boundary_code(boundary), segments, budget,
        scale, _dp(out["O"]), _dp(out["approx"]), _dp(out["W"]),
        _lp(out["seg"]), _dp(out["Wp"]), _lp(out["tok"])), "filter_attend")
    return out


def filter_attend(Q, K, V, levels: int, segments: int, budget: int,
                  wavelet: str = "haar", boundary: str = "symmetric",
                  Kg=None, Vg=None, scale: float | None = None):
    """O1-O8 over many units in parallel (OpenMP).  Q [U, B, d], K/V [U, L, d].
    Returns (O [U, B, d], tok [U, k_eff])."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    U, B, d = Q.shape
    L = K.shape[1]
    G = 0 if Kg is None else int(Kg.shape[1])
    kg = _f64(Kg) if G else None
    vg = _f64(Vg) if G else None
    keff = min(budget, segments << levels)
    scale = default_scale(d) if scale is None else scale
    O = np.empty((U, B, d))
    tok = np.empty((U, keff), dtype=np.int64)
    _check(_load().wf_ref_filter_attend(
        _dp(Q), _dp(K), _dp(V), _dp(kg) if G else _null_d(),
        _dp(vg) if G else _null_d(), U, L, d, B, G, levels,
        wavelet_code(wavelet), boundary_code(boundary), segments, budget,
        scale, _dp(O), _lp(tok)), "filter_attend")
    return O, tok


def recursion_count(m: float, n: int) -> int:
    """c = max(1, ceil(m n)) capped at n, m taken as given (double)."""
    return int(_load().wf_ref_recursion_count(float(m), int(n)))


def recursive_select(Q, K, levels: int, proportions, wavelet: str = "haar",
                     boundary: str = "symmetric",
                     scale: float | None = None):
    """R1 for one unit.  proportions[b - 1] = m_b, b = 1..levels.
    Returns (tok = mu^0 ascending, counts [levels] with c_b at b - 1)."""
    Q, K = _f64(Q), _f64(K)
    B, d = Q.shape
    L = K.shape[0]
    prop = _f64(np.asarray(proportions, dtype=np.float64))
    if prop.size != levels:
        raise ValueError("one proportion per scale")
    scale = default_scale(d) if scale is None else scale
    counts = np.empty(levels, dtype=np.int64)
    tok = np.empty(L, dtype=np.int64)
    n_tok = np.zeros(1, dtype=np.int64)
    _check(_load().wf_ref_recursive_select(
        _dp(Q), _dp(K), B, L, d, levels, wavelet_code(wavelet),
        boundary_code(boundary), _dp(prop), scale, _lp(counts), _lp(tok),
        _lp(n_tok)), "recursive_select")
    return tok[:int(n_tok[0])].copy(), counts


def filter_attend_recursive(Q, K, V, levels: int, proportions,
                            wavelet: str = "haar",
                            boundary: str = "symmetric", Kg=None, Vg=None,
                            scale: float | None = None):
    """R1 + O7-O8 over many units (OpenMP).  Q [U, B, d], K/V [U, L, d].
    Returns (O [U, B, d], tok list of per-unit mu^0 arrays)."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    U, B, d = Q.shape
    L = K.shape[1]
    G = 0 if Kg is None else int(Kg.shape[1])
    kg = _f64(Kg) if G else None
    vg = _f64(Vg) if G else None
    prop = _f64(np.asarray(proportions, dtype=np.float64))
    if prop.size != levels:
        raise ValueError("one proportion per scale")
    scale = default_scale(d) if scale is None else scale
    O = np.empty((U, B, d))
    tok = np.empty((U, L), dtype=np.int64)
    n_tok = np.empty(U, dtype=np.int64)
    _check(_load().wf_ref_filter_attend_recursive(
        _dp(Q), _dp(K), _dp(V), _dp(kg) if G else _null_d(),
        _dp(vg) if G else _null_d(), U, L, d, B, G, levels,
        wavelet_code(wavelet), boundary_code(boundary), _dp(prop), scale,
        _dp(O), _lp(tok), _lp(n_tok)), "filter_attend_recursive")
    return O, [tok[u, :n_tok[u]].copy() for u in range(U)]


def filter_attend_shared(Q, K, V, levels: int, segments: int, budget: int,
                         wavelet: str = "haar", boundary: str = "symmetric",
                         Kg=None, Vg=None, scale: float | None = None) -> dict:
    """One selection shared by the H heads of a sequence (the layer-shared
    variant of the per-head selection).  Q [H, B, d], K/V [H, L, d], Kg/Vg
    [H, G, d].  eqs. 7-8 per head over its own keys, the column sums W
    added over the heads; eq. 9 on that sum gives the regions; eq. 10 the
    pool; the scan's W' (eqs. 7-8 over the pool, per head) added over the
    heads; its top k_eff the tokens; then every head attends over its own
    K/V rows at those tokens, the L mod 2^J remainder rows and its tail
    (eq. 3 form).  Returns dict(W, seg, Wp, tok, O [H, B, d]).
    """
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    H, B, d = Q.shape
    L = K.shape[1]
    Lf = (L >> levels) << levels
    G = 0 if Kg is None else int(Kg.shape[1])
    n = Lf >> levels
    W = np.zeros(n)
    for h in range(H):
        W += skim(Q[h], dwt(K[h, :Lf], levels, wavelet, boundary), scale)
    seg = topk(W, segments)
    keff = min(budget, segments << levels)
    pool = (seg[:, None] * (1 << levels) + np.arange(1 << levels)[None, :]).ravel()
    Wp = np.zeros(pool.size)
    for h in range(H):
        Wp += scan(Q[h], K[h], seg, levels, budget, scale)[0]
    tok = pool[topk(Wp, keff)]
    keep = np.concatenate([tok, np.arange(Lf, L)])
    O = np.empty((H, B, d))
    for h in range(H):
        O[h] = attend(Q[h], K[h], V[h], keep, Kg[h] if G else None,
                      Vg[h] if G else None, scale)
    return dict(W=W, seg=seg, Wp=Wp, tok=tok, O=O)


def max_threads() -> int:
    return int(_load().wf_ref_max_threads())
