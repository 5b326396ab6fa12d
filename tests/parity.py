"""Stage-wise comparison of the GPU path with the CPU oracle.

Rules (tolerances from the task's stated bar, applied per stage so that one
near-tie cannot cascade):
  * DWT coefficients: |gpu - ref| <= 1e-3 |ref| + 1e-3 rms(ref) per unit and
    level (a mixed bound, so near-zero coefficients do not divide by ~0).
  * index sets: equal to the oracle's selection, except for positions whose
    oracle score lies within 1e-3 (relative) of the k-th largest score.
    Sizes, order (ascending) and uniqueness are exact.
  * token selection is checked conditionally: the oracle's scan runs on the
    GPU's own coarse regions; attention is checked on the GPU's own tokens.
  * attention output: max |gpu - ref| <= 2e-2 for bf16 inputs, 1e-4 for fp32.
  * scores (W, W'): relative 1e-3 -- the band the selection rule allows.
"""
from __future__ import annotations

import os
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

import oracle

O_TOL = {"bf16": 2e-2, "f32": 1e-4}
SEL_REL = 1e-3
COEF_REL = 1e-3


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def f64(t) -> np.ndarray:
    if isinstance(t, torch.Tensor):
        return t.detach().to("cpu", torch.float64).numpy()
    return np.asarray(t, dtype=np.float64)


def i64(t) -> np.ndarray:
    if isinstance(t, torch.Tensor):
        return t.detach().cpu().numpy().astype(np.int64)
    return np.asarray(t, dtype=np.int64)


def check_coefficients(gpu, ref, what: str) -> None:
    gpu, ref = f64(gpu), f64(ref)
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    rms = np.sqrt(np.mean(ref ** 2))
    bound = COEF_REL * np.abs(ref) + COEF_REL * rms
    err = np.abs(gpu - ref)
    bad = err > bound
    assert not bad.any(), (f"{what}: {bad.sum()} coefficients outside "
                           f"tolerance, worst err {err.max():.3e} (rms {rms:.3e})")


def check_scores(gpu, ref, what: str, rel: float = SEL_REL) -> None:
    gpu, ref = f64(gpu), f64(ref)
    assert gpu.shape == ref.shape
    tiny = 1e-30
    bad = np.abs(gpu - ref) > rel * np.abs(ref) + tiny
    assert not bad.any(), (f"{what}: {bad.sum()} scores off by more than "
                           f"{rel} relative; worst {np.max(np.abs(gpu-ref)/np.maximum(np.abs(ref), tiny)):.3e}")


def oracle_selection(scores: np.ndarray, k: int) -> np.ndarray:
    n = scores.size
    order = np.lexsort((np.arange(n), -scores))
    return np.sort(order[:k])


def check_selection(sel, scores, k: int, what: str) -> int:
    """sel: GPU-chosen positions into `scores` (oracle scores, fp64).
    Returns the number of (allowed) disagreements with the oracle."""
    sel = i64(sel).ravel()
    scores = f64(scores).ravel()
    n = scores.size
    assert sel.size == k, (what, sel.size, k)
    assert sel.min() >= 0 and sel.max() < n, what
    assert np.all(np.diff(sel) > 0), f"{what}: not strictly ascending"
    order = np.lexsort((np.arange(n), -scores))
    ref = np.sort(order[:k])
    thr = scores[order[k - 1]]
    band = np.abs(scores - thr) <= SEL_REL * abs(thr)
    diff = np.setxor1d(sel, ref)
    outside = diff[~band[diff]]
    assert outside.size == 0, (f"{what}: {outside.size} picks differ outside "
                               f"the tie band (e.g. {outside[:5]})")
    return int(diff.size)


def pool_tokens(seg, levels: int) -> np.ndarray:
    seg = i64(seg)
    run = 1 << levels
    return (seg[:, None] * run + np.arange(run)[None, :]).ravel()


def check_unit(*, Q, K, V, levels, segments, budget, wavelet, boundary,
               dtype, seg_gpu, tok_gpu, O_gpu, Kg=None, Vg=None, W_gpu=None,
               Wp_gpu=None, what=""):
    """Full conditional check of one unit's GPU outputs.  A length that is
    not a multiple of 2^J is filtered on its first Lf positions; the rest is
    always attended, after the selected positions."""
    L = K.shape[0]
    Lf = (L >> levels) << levels
    A_ref = oracle.dwt(K[:Lf], levels, wavelet, boundary)
    W_ref = oracle.skim(Q, A_ref)
    if W_gpu is not None:
        check_scores(W_gpu, W_ref, f"{what} W")
    n_seg_diff = check_selection(seg_gpu, W_ref, segments, f"{what} seg")
    Wp_ref, tok_ref = oracle.scan(Q, K, seg_gpu, levels, budget)
    if Wp_gpu is not None:
        check_scores(Wp_gpu, Wp_ref, f"{what} W'")
    pool = pool_tokens(seg_gpu, levels)
    tok = i64(tok_gpu)
    keff = min(budget, pool.size)
    pos = np.searchsorted(pool, tok)
    assert np.all(pos < pool.size) and np.all(pool[np.minimum(pos, pool.size - 1)] == tok), \
        f"{what}: tokens outside the pool of the GPU's regions"
    n_tok_diff = check_selection(pos, Wp_ref, keff, f"{what} tok")
    O_ref = oracle.attend(Q, K, V, np.concatenate([tok, np.arange(Lf, L)]), Kg, Vg)
    err = np.max(np.abs(f64(O_gpu) - O_ref))
    assert err <= O_TOL[dtype], f"{what}: O max abs err {err:.3e} > {O_TOL[dtype]}"
    return dict(seg_diff=n_seg_diff, tok_diff=n_tok_diff, o_err=float(err))


def oracle_workers() -> int:
    """Threads for per-unit oracle checks: the host's cores, at most 16
    (the oracle's C entry points release the GIL while they run)."""
    return max(1, min(16, os.cpu_count() or 1))


def check_units(w, *, Q, K, V, seg, tok, O, Kg=None, Vg=None, units=None,
                what: str = "") -> list[dict]:
    """check_unit on every unit of a launch (or on `units`), in a thread
    pool.  Q/K/V/O [batch, heads, ...] as the GPU saw them, seg/tok the GPU's
    index outputs.  Returns the per-unit summaries in unit order."""
    U = w.units

    def flat(t):
        return None if t is None else t.reshape(U, *t.shape[2:])

    q, k, v, kg, vg = (flat(t) for t in (Q, K, V, Kg, Vg))
    sg, tk, o = flat(seg), flat(tok), flat(O)
    todo = list(range(U)) if units is None else list(units)

    def one(u):
        return check_unit(
            Q=q[u], K=k[u], V=v[u], Kg=None if kg is None else kg[u],
            Vg=None if vg is None else vg[u], levels=w.levels,
            segments=w.segments, budget=w.budget, wavelet=w.wavelet,
            boundary=w.boundary, dtype=w.dtype, seg_gpu=sg[u], tok_gpu=tk[u],
            O_gpu=o[u], what=f"{what} unit {u}")

    with ThreadPoolExecutor(max_workers=oracle_workers()) as ex:
        return list(ex.map(one, todo))


def summary(stats: list[dict]) -> str:
    """One line over many unit checks: units, allowed index differences
    inside the tie band, worst output error."""
    return (f"{len(stats)} units, seg diffs {sum(s['seg_diff'] for s in stats)}, "
            f"tok diffs {sum(s['tok_diff'] for s in stats)}, "
            f"max O err {max(s['o_err'] for s in stats):.2e}")


def check_shared_sequence(*, Q, K, V, levels, segments, budget, wavelet,
                          boundary, dtype, seg_gpu, tok_gpu, O_gpu, Kg=None,
                          Vg=None, what=""):
    """Conditional check of one sequence's shared selection: Q/K/V [H, ...]
    of its heads, seg_gpu [S] and tok_gpu [k_eff] shared, O_gpu [H, B, d].
    W is the heads' eq. 8 column sums added; W' the heads' scan weights over
    the GPU's own pool added; each head's output is checked on the GPU's own
    tokens."""
    H = Q.shape[0]
    L = K.shape[1]
    Lf = (L >> levels) << levels
    W_ref = sum(oracle.skim(Q[h], oracle.dwt(K[h, :Lf], levels, wavelet, boundary))
                for h in range(H))
    n_seg_diff = check_selection(seg_gpu, W_ref, segments, f"{what} seg")
    Wp_ref = sum(oracle.scan(Q[h], K[h], seg_gpu, levels, budget)[0] for h in range(H))
    pool = pool_tokens(seg_gpu, levels)
    tok = i64(tok_gpu)
    keff = min(budget, pool.size)
    pos = np.searchsorted(pool, tok)
    assert np.all(pos < pool.size) and np.all(pool[np.minimum(pos, pool.size - 1)] == tok), \
        f"{what}: tokens outside the pool of the GPU's regions"
    n_tok_diff = check_selection(pos, Wp_ref, keff, f"{what} tok")
    keep = np.concatenate([tok, np.arange(Lf, L)])
    err = 0.0
    for h in range(H):
        O_ref = oracle.attend(Q[h], K[h], V[h], keep, None if Kg is None else Kg[h],
                              None if Vg is None else Vg[h])
        err = max(err, float(np.max(np.abs(f64(O_gpu[h]) - O_ref))))
    assert err <= O_TOL[dtype], f"{what}: O max abs err {err:.3e} > {O_TOL[dtype]}"
    return dict(seg_diff=n_seg_diff, tok_diff=n_tok_diff, o_err=err)
