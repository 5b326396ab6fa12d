"""GPU parity of the multi-scale recursion (wf_filter_attend_recursive)
against the oracle's R1 (scales B..1, eqs. 9-11) and O7-O8, for Haar and
Daubechies-2.

The kept positions mu^0 must equal the oracle's exactly (these seeds put no
weight within rounding of a selection threshold at any scale; a failure
reports the sizes and the first differing position).  O is checked on the
GPU's own positions against the oracle's attention, to the tolerance of the
two-stage path.  Proportions reach the oracle as the float32 values the
library receives.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import synth
from parity import O_TOL, f64, i64, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def wf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2606_00724_amd as wf
    return wf


_TINY = synth.WORKLOADS["tiny"]


def V_(name, **kw):
    return synth.small_variant(_TINY, name=name, **kw)


CASES = {
    "rec_f32_b3": V_("rf3", levels=3, proportions=(0.5, 0.5, 0.25)),
    "rec_bf16_b1_b17": V_("rb1", ctx_len=2048, levels=1, q_len=17,
                          dtype="bf16", proportions=(0.3,)),
    "rec_bf16_b2_tail": V_("rb2", ctx_len=2048, head_dim=128, q_len=48,
                           levels=2, dtype="bf16", gen_len=32,
                           proportions=(0.5, 0.3)),
    "rec_bf16_b5_b64": V_("rb5", ctx_len=4096, head_dim=128, q_len=64,
                          levels=5, dtype="bf16",
                          proportions=(0.9, 0.7, 0.5, 0.5, 0.125)),
    "rec_bf16_b6_narrow": V_("rb6", ctx_len=512, levels=6, dtype="bf16",
                             proportions=(0.5, 0.5, 0.5, 0.5, 0.5, 0.25)),
    "rec_f32_keep_all": V_("rka", ctx_len=256, levels=3, q_len=16,
                           proportions=(1.0, 1.0, 1.0)),
    # a length that is not a multiple of 2^B: the remainder follows mu^0
    "rec_bf16_b3_rem": V_("rrm", ctx_len=1024 + 6, levels=3, dtype="bf16",
                          gen_len=8, proportions=(0.5, 0.5, 0.25)),
    # Daubechies-2: every scale's transform of the gathered blocks reads
    # across their joins (banded filter from J = 2 at d = 128 bf16, the
    # cascade below), symmetric or periodic at the gathered sequence's end
    "rec_db2_sym_b2": V_("rd2s", ctx_len=2048, head_dim=128, levels=2,
                         dtype="bf16", wavelet="db2", proportions=(0.5, 0.3)),
    "rec_db2_per_b3_f32": V_("rd2p", ctx_len=1024, levels=3, wavelet="db2",
                             boundary="periodic", proportions=(0.5, 0.5, 0.25)),
    "rec_db2_sym_b4_rem": V_("rd2r", ctx_len=4096 + 9, head_dim=128, levels=4,
                             dtype="bf16", wavelet="db2", gen_len=16,
                             proportions=(0.6, 0.5, 0.5, 0.25)),
    "rec_db2_per_b2_tail": V_("rd2t", ctx_len=2048, head_dim=128, levels=2,
                              dtype="bf16", wavelet="db2", boundary="periodic",
                              gen_len=24, proportions=(0.5, 0.4)),
    # more than 64 query rows: coefficient tiles at every scale
    "rec_bf16_b3_q100": V_("rq1", ctx_len=2048, levels=3, q_len=100,
                           dtype="bf16", proportions=(0.5, 0.5, 0.25)),
}

_cache: dict = {}


def inputs(w):
    if w not in _cache:
        say(f"[inputs] generating {w.name}")
        Q, K, V = synth.make_inputs(w)
        Kg = Vg = None
        if w.gen_len:
            Kg, Vg = synth.make_tail(w, w.gen_len)
        if len(_cache) > 2:
            _cache.clear()
        _cache[w] = (Q, K, V, Kg, Vg)
    return _cache[w]


def props32(w):
    return [float(np.float32(m)) for m in w.proportions]


def run(wf, w, Q, K, V, Kg, Vg):
    p = wf.params_for(w)
    dev = "cuda"
    say(f"[gpu] {w.name}: wf_filter_attend_recursive")
    O, tok = wf.filter_attend_recursive(
        p, w.proportions, Q.to(dev), K.to(dev), V.to(dev),
        Kg.to(dev) if Kg is not None else None,
        Vg.to(dev) if Vg is not None else None)
    torch.cuda.synchronize()
    say(f"[gpu] {w.name}: done")
    return O.cpu(), tok.cpu()


def unit(t, w, u):
    if t is None:
        return None
    return t.reshape(w.units, *t.shape[2:])[u]


def sample_units(w, n):
    if w.units <= n:
        return list(range(w.units))
    rng = np.random.default_rng(4321)
    return sorted({0, w.units - 1, *rng.choice(w.units, n - 2, replace=False).tolist()})


def check(wf, w, n_units=8):
    Q, K, V, Kg, Vg = inputs(w)
    O, tok = run(wf, w, Q, K, V, Kg, Vg)
    counts = wf.recursion_counts(wf.params_for(w), w.proportions)
    assert tok.shape[-1] == 2 * counts[0]
    Lf = (w.ctx_len >> w.levels) << w.levels
    errs = []
    for u in sample_units(w, n_units):
        q, k, v = unit(Q, w, u), unit(K, w, u), unit(V, w, u)
        kg, vg = unit(Kg, w, u), unit(Vg, w, u)
        want, want_counts = oracle.recursive_select(q, k, w.levels, props32(w),
                                                    w.wavelet, w.boundary)
        assert list(want_counts) == counts, f"{w.name} unit {u}: counts"
        got = np.concatenate([i64(unit(tok, w, u)), np.arange(Lf, w.ctx_len)])
        if not np.array_equal(got, want):
            bad = int(np.argmax(got != want)) if got.size == want.size else -1
            raise AssertionError(
                f"{w.name} unit {u}: mu^0 differs (sizes {got.size}/{want.size}, "
                f"first difference at {bad})")
        ref = oracle.attend(q, k, v, got, kg, vg)
        err = float(np.abs(f64(unit(O, w, u)) - ref).max())
        assert err <= O_TOL[w.dtype], f"{w.name} unit {u}: O err {err:.3e}"
        errs.append(err)
    say(f"[parity] {w.name}: {len(errs)} units, |mu^0| = {2 * counts[0]} "
        f"(+{w.ctx_len - Lf} kept), "
        f"max O err {max(errs):.1e}")


@pytest.mark.parametrize("name", list(CASES))
def test_recursion_edge_shapes(wf, name):
    check(wf, CASES[name])


def test_recursion_keep_all_is_dense(wf):
    w = CASES["rec_f32_keep_all"]
    Q, K, V, _, _ = inputs(w)
    O, tok = run(wf, w, Q, K, V, None, None)
    for u in range(w.units):
        assert torch.equal(unit(tok, w, u), torch.arange(w.ctx_len, dtype=torch.int32))
        q, k, v = (f64(unit(x, w, u)) for x in (Q, K, V))
        s = q @ k.T / np.sqrt(w.head_dim)
        pr = np.exp(s - s.max(1, keepdims=True))
        dense = (pr / pr.sum(1, keepdims=True)) @ v
        assert np.abs(f64(unit(O, w, u)) - dense).max() <= O_TOL[w.dtype]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_recursion_constant_keys_keep_the_first_positions(wf, dtype):
    w = V_("rconst", ctx_len=512, levels=3, dtype=dtype,
           proportions=(0.5, 0.25, 0.5))
    Q, K, V, _, _ = inputs(w)
    K = torch.full_like(K, 0.375)
    O, tok = run(wf, w, Q, K, V, None, None)
    n = 2 * wf.recursion_counts(wf.params_for(w), w.proportions)[0]
    for u in range(w.units):
        assert unit(tok, w, u).tolist() == list(range(n))


@pytest.mark.parametrize("name", ["recursion8b", "recursion32k"])
def test_recursion_workloads(wf, name):
    w = synth.WORKLOADS[name]
    check(wf, w, n_units=8 if name == "recursion8b" else 4)


def test_recursion_is_deterministic(wf):
    w = CASES["rec_bf16_b5_b64"]
    Q, K, V, _, _ = inputs(w)
    a = run(wf, w, Q, K, V, None, None)
    b = run(wf, w, Q, K, V, None, None)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
