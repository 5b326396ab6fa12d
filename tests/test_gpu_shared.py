"""GPU parity of wf_filter_attend_shared (one selection per sequence,
shared by its heads), on the token-level and the general path, against the
oracle's filter_attend_shared: the
regions against the heads' summed W (tie band), the tokens conditionally on
the GPU's regions against the heads' summed W', every head's output on the
GPU's tokens; every sequence of every case."""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor

import pytest
import torch

import synth
from parity import check_shared_sequence, f64, oracle_workers, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def wf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2606_00724_amd as wf
    return wf


_TINY = synth.WORKLOADS["tiny"]
_BF = dict(dtype="bf16")


def V_(name, **kw):
    return synth.small_variant(_TINY, name=name, **kw)


CASES = {
    "sh_j4_h4": V_("sh4", heads=4, ctx_len=2048, head_dim=128, levels=4,
                   segments=20, budget=150, q_len=24, **_BF),
    # two sequences of three heads, a remainder and a generation tail, d 64
    "sh_j3_rem_tail": V_("shr", batch=2, heads=3, ctx_len=1024 + 5, levels=3,
                         segments=30, budget=100, q_len=17, gen_len=16, **_BF),
    "sh_j5_b64": V_("sh5", batch=2, heads=5, ctx_len=32 * 70, head_dim=128,
                    levels=5, segments=12, budget=300, q_len=64, **_BF),
    "sh_db2_j6": V_("shd", heads=4, ctx_len=64 * 40, head_dim=128, levels=6,
                    segments=6, budget=200, q_len=32, wavelet="db2", **_BF),
    # every region and token kept; one head
    "sh_keep_all": V_("sha", heads=2, ctx_len=512, head_dim=128, levels=3,
                      segments=64, budget=512, q_len=16, **_BF),
    "sh_one_head": V_("sh1", heads=1, ctx_len=2048, head_dim=128, levels=4,
                      segments=16, budget=100, q_len=32, **_BF),
    # the general path: fp32 keys, J outside 3..5, more than 64 query rows,
    # db2 on coefficient tiles, a remainder and a tail
    "shg_f32": V_("sg1", batch=2, heads=3, ctx_len=1024, levels=3, segments=12,
                  budget=60, q_len=17),
    "shg_j2_b100": V_("sg2", heads=3, ctx_len=1024 + 3, head_dim=128, levels=2,
                      segments=40, budget=90, q_len=100, gen_len=8, **_BF),
    "shg_db2_j3": V_("sg3", heads=4, ctx_len=2048, head_dim=128, levels=3,
                     segments=16, budget=64, wavelet="db2", **_BF),
    "shg_j7_wide": V_("sg4", heads=2, ctx_len=128 * 40, levels=7, segments=5,
                      budget=300, q_len=24, **_BF),
    # 4096 coarse blocks: the per-unit W from its own wide kernel
    "shg_f32_4096": V_("sg5", heads=2, ctx_len=8 * 4096, levels=3, segments=64,
                       budget=300, q_len=16),
}

_cache: dict = {}


def inputs(w):
    if w not in _cache:
        say(f"[inputs] generating {w.name}")
        Q, K, V = synth.make_inputs(w)
        Kg = Vg = None
        if w.gen_len:
            Kg, Vg = synth.make_tail(w, w.gen_len)
        _cache.clear()
        _cache[w] = (Q, K, V, Kg, Vg)
    return _cache[w]


def run(wf, w, Q, K, V, Kg, Vg):
    p = wf.params_for(w)
    say(f"[gpu] {w.name}: wf_filter_attend_shared")
    O, tok, seg = wf.filter_attend_shared(
        p, Q.cuda(), K.cuda(), V.cuda(),
        Kg.cuda() if Kg is not None else None,
        Vg.cuda() if Vg is not None else None, want_indices=True)
    torch.cuda.synchronize()
    say(f"[gpu] {w.name}: done")
    return O.cpu(), tok.cpu(), seg.cpu()


def check(wf, w):
    Q, K, V, Kg, Vg = inputs(w)
    O, tok, seg = run(wf, w, Q, K, V, Kg, Vg)

    def one(b):
        return check_shared_sequence(
            Q=f64(Q[b]), K=f64(K[b]), V=f64(V[b]),
            Kg=None if Kg is None else f64(Kg[b]),
            Vg=None if Vg is None else f64(Vg[b]), levels=w.levels,
            segments=w.segments, budget=w.budget, wavelet=w.wavelet,
            boundary=w.boundary, dtype=w.dtype, seg_gpu=seg[b], tok_gpu=tok[b],
            O_gpu=O[b], what=f"{w.name} sequence {b}")

    with ThreadPoolExecutor(max_workers=min(oracle_workers(), w.batch)) as ex:
        res = list(ex.map(one, range(w.batch)))
    say(f"[parity] {w.name} shared: {w.batch} sequences x {w.heads} heads, "
        f"seg diffs {sum(r['seg_diff'] for r in res)}, tok diffs "
        f"{sum(r['tok_diff'] for r in res)}, max O err {max(r['o_err'] for r in res):.2e}")


@pytest.mark.parametrize("name", list(CASES))
def test_shared_edge_shapes(wf, name):
    check(wf, CASES[name])


@pytest.mark.parametrize("name", ["layer8b", "headline32k"])
def test_shared_workloads(wf, name):
    check(wf, synth.WORKLOADS[name])


def test_shared_is_deterministic(wf):
    w = CASES["sh_j4_h4"]
    Q, K, V, _, _ = inputs(w)
    first = run(wf, w, Q, K, V, None, None)
    for r in range(9):
        again = run(wf, w, Q, K, V, None, None)
        for x, y in zip(first, again):
            assert torch.equal(x, y), f"run {r + 2} differs from run 1"


def test_shared_timed_matches_plain(wf):
    """The timed call queues the same kernels, with events between them."""
    w = CASES["sh_j3_rem_tail"]
    Q, K, V, Kg, Vg = inputs(w)
    p = wf.params_for(w)
    names = wf.shared_kernel_names(p)
    O0, tok0, seg0 = run(wf, w, Q, K, V, Kg, Vg)
    Qd, Kd, Vd, Kgd, Vgd = (x.cuda() for x in (Q, K, V, Kg, Vg))
    O = torch.empty_like(Qd)
    tok = torch.empty_like(tok0, device="cuda")
    seg = torch.empty_like(seg0, device="cuda")
    ws = wf.alloc_workspace(p, wf.OP_SHARED, Qd.device)
    import bench
    ev = bench.HipEvents(len(names) + 1)
    handles = ev.ev
    wf.wf_filter_attend_shared_timed(p, Qd, Kd, Vd, Kgd, Vgd, O, tok, seg, ws, handles)
    torch.cuda.synchronize()
    assert torch.equal(O.cpu(), O0) and torch.equal(tok.cpu(), tok0)
    assert torch.equal(seg.cpu(), seg0)
    assert all(ev.elapsed_ms(i, i + 1) >= 0 for i in range(len(names)))
    ev.close()
