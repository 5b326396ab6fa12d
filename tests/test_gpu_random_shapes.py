"""GPU parity on seeded random shapes: the fused, cached and shared calls
against the oracle, on every unit, for shapes drawn across element types,
head sizes, wavelets and extensions, 1..7 levels, lengths with and without
a remainder, 1..100 query rows, any S and k, and generation tails; shapes
drawn onto the coefficient-tile sequence whose selections run in their
consumers (W over all CUs, the top-S in the scan's statistics pass, the
top-k in the attention); and the multi-scale recursion (eqs. 9-11) with
1..6 scales and random proportions, every scale checked on the GPU's own
kept blocks.  The draws are fixed (seeds 2026, 2028 and 2027), so a failure
names a reproducible case."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import synth
from parity import check_shared_sequence, check_units, f64, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def wf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2606_00724_amd as wf
    return wf


def _cases(n=96, seed=2026):
    rng = np.random.default_rng(seed)
    base = synth.WORKLOADS["tiny"]
    out = []
    while len(out) < n:
        # every other case on the token-level path (bf16, Haar 3..5 levels or
        # db2 at 6, at most 64 query rows)
        token = len(out) % 2 == 0
        J = int(rng.integers(3, 6)) if token else int(rng.integers(1, 8))
        nJ = int(rng.integers(2, 160))
        rem = int(rng.integers(1, 1 << J)) if J > 0 and rng.random() < 0.4 else 0
        S = int(rng.integers(1, nJ + 1))
        w = synth.small_variant(
            base, name=f"rand{len(out)}",
            batch=int(rng.integers(1, 3)), heads=int(rng.integers(1, 4)),
            ctx_len=(nJ << J) + rem, head_dim=int(rng.choice([64, 128])),
            q_len=int(rng.choice([1, 7, 16, 17, 32, 33, 48, 64] if token
                                 else [1, 7, 16, 17, 32, 33, 48, 64, 65, 100])),
            dtype="bf16" if token else str(rng.choice(["bf16", "bf16", "f32"])),
            wavelet="haar" if token else str(rng.choice(["haar", "haar", "db2"])),
            boundary=str(rng.choice(["symmetric", "periodic"])),
            levels=J, segments=S, budget=int(rng.integers(1, (S << J) + 40)),
            gen_len=int(rng.choice([0, 0, 8, 17])), needles=1,
            seed=100 + len(out))
        if w.ctx_len < synth.NEEDLE_LEN:
            continue
        out.append(w)
    return out


CASES = _cases()


def _inputs(w):
    Q, K, V = synth.make_inputs(w)
    Kg = Vg = None
    if w.gen_len:
        Kg, Vg = synth.make_tail(w, w.gen_len)
    return Q, K, V, Kg, Vg


def _dev(x):
    return None if x is None else x.cuda()


def _consumer_select_cases(n=24, seed=2028):
    """bf16, at most 64 query rows and a multiple of 4 coefficients, off the
    token-level path: Haar at 1, 2, 6 or 7 levels, db2 at 1..5 or 7."""
    rng = np.random.default_rng(seed)
    base = synth.WORKLOADS["tiny"]
    out = []
    while len(out) < n:
        wavelet = str(rng.choice(["haar", "db2"]))
        J = int(rng.choice([1, 2, 6, 7] if wavelet == "haar" else [1, 2, 3, 4, 5, 7]))
        nJ = 4 * int(rng.integers(1, 40))
        rem = int(rng.integers(1, 1 << J)) if rng.random() < 0.4 else 0
        S = int(rng.integers(1, nJ + 1))
        w = synth.small_variant(
            base, name=f"crand{len(out)}",
            batch=int(rng.integers(1, 3)), heads=int(rng.integers(1, 4)),
            ctx_len=(nJ << J) + rem, head_dim=int(rng.choice([64, 128])),
            q_len=int(rng.choice([1, 7, 16, 17, 32, 33, 48, 64])), dtype="bf16",
            wavelet=wavelet, boundary=str(rng.choice(["symmetric", "periodic"])),
            levels=J, segments=S, budget=int(rng.integers(1, (S << J) + 40)),
            gen_len=int(rng.choice([0, 0, 8, 17])), needles=1,
            seed=300 + len(out))
        if w.ctx_len < synth.NEEDLE_LEN:
            continue
        out.append(w)
    return out


CONSUMER_CASES = _consumer_select_cases()


def _check_case(wf, w, i, what, cached):
    p = wf.params_for(w)
    if wf.workspace_bytes(p, wf.OP_FUSED) == 0:
        pytest.skip(f"{w} is outside the parameter limits")
    say(f"[case] {what} {i}: {w.batch}x{w.heads} L={w.ctx_len} d={w.head_dim} "
        f"B={w.q_len} {w.dtype} {w.wavelet}/{w.boundary} J={w.levels} "
        f"S={w.segments} k={w.budget} G={w.gen_len}; {wf.fused_kernel_names(p)}")
    Q, K, V, Kg, Vg = _inputs(w)
    O, tok, seg = wf.filter_attend(p, Q.cuda(), K.cuda(), V.cuda(), _dev(Kg),
                                   _dev(Vg), want_indices=True)
    torch.cuda.synchronize()
    check_units(w, Q=Q, K=K, V=V, Kg=Kg, Vg=Vg, seg=seg.cpu(), tok=tok.cpu(),
                O=O.cpu(), what=f"{what} {i} fused")
    if cached:
        Kd = K.cuda()
        approx = wf.dwt_approx(p, Kd)
        O, tok, seg = wf.filter_attend_cached(p, Q.cuda(), approx, Kd, V.cuda(),
                                              _dev(Kg), _dev(Vg),
                                              want_indices=True)
        torch.cuda.synchronize()
        check_units(w, Q=Q, K=K, V=V, Kg=Kg, Vg=Vg, seg=seg.cpu(),
                    tok=tok.cpu(), O=O.cpu(), what=f"{what} {i} cached")
    O, tok, seg = wf.filter_attend_shared(p, Q.cuda(), K.cuda(), V.cuda(),
                                          _dev(Kg), _dev(Vg), want_indices=True)
    torch.cuda.synchronize()
    O, tok, seg = O.cpu(), tok.cpu(), seg.cpu()
    for b in range(w.batch):
        check_shared_sequence(
            Q=f64(Q[b]), K=f64(K[b]), V=f64(V[b]),
            Kg=None if Kg is None else f64(Kg[b]),
            Vg=None if Vg is None else f64(Vg[b]), levels=w.levels,
            segments=w.segments, budget=w.budget, wavelet=w.wavelet,
            boundary=w.boundary, dtype=w.dtype, seg_gpu=seg[b],
            tok_gpu=tok[b], O_gpu=O[b], what=f"{what} {i} shared {b}")


@pytest.mark.parametrize("i", range(len(CASES)))
def test_random_shape(wf, i):
    _check_case(wf, CASES[i], i, "random", cached=i % 3 == 0)


@pytest.mark.parametrize("i", range(len(CONSUMER_CASES)))
def test_random_consumer_selects(wf, i):
    """Every case takes the sequence with W over all CUs and the selections
    in their consumers, through the fused, cached and shared calls."""
    w = CONSUMER_CASES[i]
    names = wf.fused_kernel_names(wf.params_for(w))
    assert names[1] == "skim_weights", names
    _check_case(wf, w, i, "consumer", cached=True)


def _rec_cases(n=32, seed=2027):
    rng = np.random.default_rng(seed)
    base = synth.WORKLOADS["tiny"]
    out = []
    while len(out) < n:
        B = int(rng.integers(1, 7))
        nB = int(rng.integers(2, 120))
        rem = int(rng.integers(1, 1 << B)) if rng.random() < 0.4 else 0
        w = synth.small_variant(
            base, name=f"rrand{len(out)}",
            batch=int(rng.integers(1, 3)), heads=int(rng.integers(1, 3)),
            ctx_len=(nB << B) + rem, head_dim=int(rng.choice([64, 128])),
            q_len=int(rng.choice([1, 16, 17, 32, 64, 65])),
            dtype=str(rng.choice(["bf16", "bf16", "f32"])),
            wavelet=str(rng.choice(["haar", "haar", "db2"])),
            boundary=str(rng.choice(["symmetric", "periodic"])),
            levels=B, proportions=tuple(float(x) for x in rng.uniform(0.1, 1.0, B)),
            gen_len=int(rng.choice([0, 0, 8])), needles=1, seed=500 + len(out))
        if w.ctx_len < synth.NEEDLE_LEN:
            continue
        out.append(w)
    return out


REC_CASES = _rec_cases()


@pytest.mark.parametrize("i", range(len(REC_CASES)))
def test_random_recursion(wf, i):
    import test_gpu_recursion as rec
    w = REC_CASES[i]
    p = wf.params_for(w)
    if wf.recursive_workspace_bytes(p, w.proportions) == 0:
        pytest.skip("outside the parameter limits")
    say(f"[case] rec {i}: {w.batch}x{w.heads} L={w.ctx_len} d={w.head_dim} "
        f"B={w.q_len} {w.dtype} {w.wavelet}/{w.boundary} scales={w.levels} "
        f"m={[round(m, 3) for m in w.proportions]} G={w.gen_len}")
    rec.check(wf, w)
