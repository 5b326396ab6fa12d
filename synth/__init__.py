"""Seeded synthetic inputs for the WaveFilter filter+attend path.

This module only draws random tensors and describes workload shapes.  It holds
none of the method's arithmetic (no transform, scoring, selection or
attention), so the CPU oracle and the GPU path can both consume its output
without sharing any computation.

Workloads stand in for the paper's long-context evaluations (LongBench and
RULER, Section 4 "Implementation Details"), whose data and model weights are
not available: the keys are an AR(1) process along the sequence plus white
noise, with a few 16-token "needle" spans that carry a per-head direction u,
and the queries lean towards u, which mimics needle-retrieval structure only.

Recipe for one (layer, batch, head) unit, all in float64:
  * sequence generator  Generator(PCG64(SeedSequence([seed, layer, batch, 1_000_003])))
      - needle starts: integers(0, L - 16 + 1), redrawn until no two spans
        overlap (spans are shared by every head of one sequence)
  * unit generator      Generator(PCG64(SeedSequence([seed, layer, batch, head])))
      draws, in this order:
      - u   : d standard normals, normalised to unit length
      - eps : [L, d] standard normals
      - eta : [L, d] standard normals
      - z   : [B, d] standard normals
      - v   : [L, d] standard normals (the values)
  * keys:    k_0 = eps_0,  k_t = rho k_{t-1} + sqrt(1 - rho^2) eps_t
             (stationary unit-variance AR(1) along the sequence)
             K = k + 0.3 eta;  K[s:s+16] += 3 u for every needle start s
  * queries: Q = z / sqrt(d) + 2 u
  * values:  V = v
  * rounding: once, on the host: float64 -> float32 (round to nearest even),
    then for bf16 workloads float32 -> bfloat16 (round to nearest even on
    the dropped 16 bits, the same rule as torch's conversion).
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace

import numpy as np
from scipy.signal import lfilter

NEEDLE_LEN = 16
_SEQ_TAG = 1_000_003


@dataclass(frozen=True)
class Workload:
    """Shape and selection sizes of one synthetic workload."""

    name: str
    batch: int
    heads: int
    ctx_len: int          # L, prompt positions that are filtered
    head_dim: int         # d
    q_len: int            # B, query positions of the current block
    dtype: str            # "bf16" or "f32"
    rho: float            # AR(1) coefficient of the keys
    needles: int          # needle spans per sequence
    wavelet: str          # "haar" or "db2"
    boundary: str         # "symmetric" or "periodic" (db2 only)
    levels: int           # J, DWT levels
    segments: int         # S, coarse segments kept by the skim
    budget: int           # k, tokens kept by the scan
    seed: int
    layers: int = 1
    gen_len: int = 0      # G, always-kept generation tail (K_g, V_g)
    # multi-scale recursion: m_b at index b - 1 (empty: the two-stage path)
    proportions: tuple = ()
    # the prompt's A_J is computed once and reused by every step
    cached: bool = False
    # one selection per sequence, shared by its heads
    shared: bool = False
    description: str = field(default="", compare=False)

    @property
    def units(self) -> int:
        return self.batch * self.heads


def _pool_segments(ctx_len: int, levels: int, budget: int) -> int:
    """Coarse segments kept when only a token budget is given: a candidate
    pool of twice the budget, capped by the number of coarse coefficients."""
    n_coarse = ctx_len >> levels
    return min(n_coarse, -(-2 * budget // (1 << levels)))


WORKLOADS: dict[str, Workload] = {}


def _add(w: Workload) -> None:
    WORKLOADS[w.name] = w


_add(Workload("tiny", batch=1, heads=2, ctx_len=1024, head_dim=64, q_len=32,
              dtype="f32", rho=0.95, needles=1, wavelet="haar",
              boundary="symmetric", levels=3, segments=8, budget=128, seed=0,
              description="tiny CPU-seconds instance: 2 heads, d=64, L=1024, "
                          "B=32, fp32, Haar J=3, 8 segments, budget 128"))
_add(Workload("tiny_scan", batch=1, heads=2, ctx_len=1024, head_dim=64,
              q_len=32, dtype="f32", rho=0.95, needles=1, wavelet="haar",
              boundary="symmetric", levels=3, segments=32, budget=128, seed=0,
              description="tiny instance with a pool (256) larger than the "
                          "budget (128)"))
_add(Workload("layer8b", batch=1, heads=32, ctx_len=4096, head_dim=128,
              q_len=32, dtype="bf16", rho=0.95, needles=4, wavelet="haar",
              boundary="symmetric", levels=3,
              segments=_pool_segments(4096, 3, 512), budget=512, seed=1,
              description="8B-DLM single layer: 32 heads, d=128, L=4096, "
                          "B=32, bf16, Haar J=3, budget 512"))
_add(Workload("long16k", batch=1, heads=32, ctx_len=16384, head_dim=128,
              q_len=32, dtype="bf16", rho=0.98, needles=8, wavelet="haar",
              boundary="symmetric", levels=4,
              segments=_pool_segments(16384, 4, 1024), budget=1024, seed=2,
              layers=32,
              description="long context: 32 heads, d=128, L=16384, B=32, "
                          "bf16, Haar J=4, budget 1024, 32 layers"))
_add(Workload("headline32k", batch=4, heads=32, ctx_len=32768, head_dim=128,
              q_len=64, dtype="bf16", rho=0.98, needles=8, wavelet="haar",
              boundary="symmetric", levels=5,
              segments=_pool_segments(32768, 5, 2048), budget=2048, seed=3,
              description="32K context: batch 4, 32 heads, d=128, L=32768, "
                          "B=64, bf16, Haar J=5, budget 2048"))
_add(Workload("stress128k", batch=1, heads=32, ctx_len=131072, head_dim=128,
              q_len=32, dtype="bf16", rho=0.99, needles=16, wavelet="db2",
              boundary="symmetric", levels=6,
              segments=_pool_segments(131072, 6, 4096), budget=4096, seed=4,
              description="128K stress: 32 heads, d=128, L=131072, B=32, "
                          "bf16, Daubechies-2 J=6 symmetric, budget 4096"))


# The paper's own schedule (scales B..1, proportions m_b) on the inputs of
# two of the workloads above (same seeds, hence the same tensors).
_add(Workload("recursion8b", batch=1, heads=32, ctx_len=4096, head_dim=128,
              q_len=32, dtype="bf16", rho=0.95, needles=4, wavelet="haar",
              boundary="symmetric", levels=3,
              segments=_pool_segments(4096, 3, 512), budget=512, seed=1,
              proportions=(0.5, 0.5, 0.25),
              description="8B-DLM layer with the multi-scale recursion: 32 "
                          "heads, d=128, L=4096, B=32, bf16, Haar, scales "
                          "3..1, m = (0.25, 0.5, 0.5) from the top"))
_add(Workload("recursion32k", batch=4, heads=32, ctx_len=32768, head_dim=128,
              q_len=64, dtype="bf16", rho=0.98, needles=8, wavelet="haar",
              boundary="symmetric", levels=2,
              segments=_pool_segments(32768, 2, 2048), budget=2048, seed=3,
              proportions=(0.5, 0.25),
              description="32K context with the multi-scale recursion at the "
                          "paper's scale B=2: batch 4, 32 heads, d=128, "
                          "L=32768, B=64, bf16, Haar, m_2=0.25, m_1=0.5 "
                          "(4096 positions kept)"))


_add(Workload("tail32k", batch=4, heads=32, ctx_len=32768 + 20, head_dim=128,
              q_len=64, dtype="bf16", rho=0.98, needles=8, wavelet="haar",
              boundary="symmetric", levels=5,
              segments=_pool_segments(32768, 5, 2048), budget=2048, seed=5,
              gen_len=64,
              description="32K context that is not a multiple of 2^J, with a "
                          "generation tail: batch 4, 32 heads, d=128, "
                          "L=32788 (20 positions always kept), G=64, B=64, "
                          "bf16, Haar J=5, budget 2048"))
_add(Workload("shared32k", batch=4, heads=32, ctx_len=32768, head_dim=128,
              q_len=64, dtype="bf16", rho=0.98, needles=8, wavelet="haar",
              boundary="symmetric", levels=5,
              segments=_pool_segments(32768, 5, 2048), budget=2048, seed=3,
              shared=True,
              description="32K context with one selection per sequence shared "
                          "by its 32 heads: batch 4, d=128, L=32768, B=64, "
                          "bf16, Haar J=5, budget 2048"))
_add(Workload("cached32k", batch=4, heads=32, ctx_len=32768, head_dim=128,
              q_len=64, dtype="bf16", rho=0.98, needles=8, wavelet="haar",
              boundary="symmetric", levels=5,
              segments=_pool_segments(32768, 5, 2048), budget=2048, seed=3,
              cached=True,
              description="32K context, one step with the prompt's A_J "
                          "cached from an earlier step: batch 4, 32 heads, "
                          "d=128, L=32768, B=64, bf16, Haar J=5, budget 2048"))


def needle_starts(w: Workload, layer: int, batch: int) -> np.ndarray:
    """Sorted, non-overlapping needle starts of one sequence."""
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([w.seed, layer, batch, _SEQ_TAG])))
    starts: list[int] = []
    while len(starts) < w.needles:
        s = int(rng.integers(0, w.ctx_len - NEEDLE_LEN + 1))
        if all(abs(s - t) >= NEEDLE_LEN for t in starts):
            starts.append(s)
    return np.array(sorted(starts), dtype=np.int64)


def unit_f64(w: Workload, layer: int, batch: int, head: int):
    """Draw one unit in float64: returns (Q [B,d], K [L,d], V [L,d])."""
    L = w.ctx_len
    d, B = w.head_dim, w.q_len
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([w.seed, layer, batch, head])))
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    eps = rng.standard_normal((L, d))
    eta = rng.standard_normal((L, d))
    z = rng.standard_normal((B, d))
    v = rng.standard_normal((L, d))
    drive = math.sqrt(1.0 - w.rho * w.rho) * eps
    drive[0] = eps[0]
    k = lfilter([1.0], [1.0, -w.rho], drive, axis=0)
    K = k + 0.3 * eta
    for s in needle_starts(w, layer, batch):
        K[s:s + NEEDLE_LEN] += 3.0 * u
    Q = z / math.sqrt(d) + 2.0 * u
    return Q, K, v


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    """float64 -> float32 (round to nearest even) -> bfloat16 bits (round to
    nearest even on the 16 dropped bits); inputs are finite."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    u = u.astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def _rounded(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return _bf16_bits(x)
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


def _to_torch(a: np.ndarray, dtype: str):
    import torch
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    return torch.from_numpy(a)


def round_host(x: np.ndarray, dtype: str):
    """Round a float64 array once to the workload dtype; returns a torch
    tensor (float32 or bfloat16) on the CPU."""
    return _to_torch(_rounded(x, dtype), dtype)


def _unit_rounded(args):
    # numpy only: runs in worker threads
    w, layer, b, h = args
    Q, K, V = unit_f64(w, layer, b, h)
    return b, h, [_rounded(x, w.dtype) for x in (Q, K, V)]


def make_inputs(w: Workload, layer: int = 0, workers: int | None = None):
    """All units of one layer, rounded once to the workload dtype.

    Returns torch CPU tensors Q [batch, heads, B, d], K and V
    [batch, heads, L, d] in the workload dtype (bfloat16 or float32).
    Units are drawn in worker threads (numpy's generators and scipy's filter
    release the GIL); no process is forked, since a fork would inherit the
    parent's OpenMP state and can deadlock.
    """
    import torch
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    Q = torch.empty((w.batch, w.heads, w.q_len, w.head_dim), dtype=tdt)
    K = torch.empty((w.batch, w.heads, w.ctx_len, w.head_dim), dtype=tdt)
    V = torch.empty_like(K)
    jobs = [(w, layer, b, h) for b in range(w.batch) for h in range(w.heads)]
    if workers is None:
        workers = min(16, os.cpu_count() or 1, len(jobs))

    def put(b, h, arrs):
        q, k, v = (_to_torch(a, w.dtype) for a in arrs)
        Q[b, h] = q
        K[b, h] = k
        V[b, h] = v

    if workers <= 1 or len(jobs) == 1:
        for job in jobs:
            put(*_unit_rounded(job))
    else:
        with ThreadPoolExecutor(max_workers=workers) as ex:
            for b, h, arrs in ex.map(_unit_rounded, jobs):
                put(b, h, arrs)
    return Q, K, V


def make_tail(w: Workload, gen_len: int, layer: int = 0):
    """Generation-position keys/values K_g, V_g [batch, heads, G, d], drawn
    with the same key/value model from their own seeds (tag 2_000_003)."""
    import torch
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    Kg = torch.empty((w.batch, w.heads, gen_len, w.head_dim), dtype=tdt)
    Vg = torch.empty_like(Kg)
    for b in range(w.batch):
        for h in range(w.heads):
            rng = np.random.Generator(np.random.PCG64(
                np.random.SeedSequence([w.seed, layer, b, h, 2_000_003])))
            kg = rng.standard_normal((gen_len, w.head_dim))
            vg = rng.standard_normal((gen_len, w.head_dim))
            Kg[b, h] = round_host(kg, w.dtype)
            Vg[b, h] = round_host(vg, w.dtype)
    return Kg, Vg


def small_variant(w: Workload, **changes) -> Workload:
    """A copy of a workload with some fields changed (for tests)."""
    return replace(w, **changes)
