"""wf_filter_attend_noalloc: the fused call on the library's own per-device
scratch (no workspace argument, nothing allocated) gives exactly what
wf_filter_attend with a workspace gives, on two calls in a row, the second
one smaller (the scratch keeps the first call's contents), and rejects
parameters whose workspace exceeds the scratch before queueing anything."""
from __future__ import annotations

import ctypes

import pytest
import torch

import synth
from parity import check_units, say, summary

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def wf():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2606_00724_amd as wf
    return wf


def _both(wf, w):
    say(f"[inputs] generating {w.name}")
    Q, K, V = synth.make_inputs(w)
    Kg = Vg = None
    if w.gen_len:
        Kg, Vg = synth.make_tail(w, w.gen_len)
    p = wf.params_for(w)
    assert wf.workspace_bytes(p, wf.OP_FUSED) <= wf.NOALLOC_SCRATCH_BYTES
    dev = torch.device("cuda")
    args = [x.to(dev) if x is not None else None for x in (Q, K, V, Kg, Vg)]
    keff = wf.effective_budget(p)
    outs = []
    for noalloc in (False, True):
        O = torch.empty_like(args[0])
        tok = torch.empty((p.batch, p.heads, keff), dtype=torch.int32, device=dev)
        seg = torch.empty((p.batch, p.heads, p.segments), dtype=torch.int32,
                          device=dev)
        say(f"[gpu] {w.name}: {'wf_filter_attend_noalloc' if noalloc else 'wf_filter_attend'}")
        if noalloc:
            wf.wf_filter_attend_noalloc(p, *args, O, tok, seg)
        else:
            ws = wf.alloc_workspace(p, wf.OP_FUSED, dev)
            wf.wf_filter_attend(p, *args, O, tok, seg, ws)
        torch.cuda.synchronize()
        outs.append((O.cpu(), tok.cpu(), seg.cpu()))
    return (Q, K, V, Kg, Vg), outs


def test_noalloc_equals_the_workspace_call(wf):
    big = synth.WORKLOADS["layer8b"]
    small = synth.small_variant(big, name="layer8b_small", heads=8,
                                ctx_len=2048 + 44, segments=40, budget=200,
                                gen_len=16)
    for w in (big, small):  # the second call is smaller than the first
        (Q, K, V, Kg, Vg), (ref, got) = _both(wf, w)
        for x, y, name in zip(ref, got, ("O", "tok", "seg")):
            assert torch.equal(x, y), f"{w.name}: {name} differs"
        stats = check_units(w, Q=Q, K=K, V=V, Kg=Kg, Vg=Vg, seg=got[2],
                            tok=got[1], O=got[0], what=f"{w.name} noalloc")
        say(f"[parity] {w.name} noalloc: {summary(stats)}")


def test_noalloc_rejects_oversized_parameters(wf):
    w = synth.WORKLOADS["headline32k"]
    p = wf.params_for(w)
    assert wf.workspace_bytes(p, wf.OP_FUSED) > wf.NOALLOC_SCRATCH_BYTES
    fake = ctypes.c_void_p(0x10000)
    lib = wf.library()
    rc = lib.wf_filter_attend_noalloc(ctypes.byref(p), fake, fake, fake, None,
                                      None, fake, None, None, None)
    assert rc == 3 and b"scratch" in lib.wf_last_error()
