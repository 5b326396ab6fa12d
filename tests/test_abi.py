"""C-ABI checks that need no GPU: the library loads, exports every function
include/wavefilter.h declares, and rejects bad arguments on the host with the
documented status codes before anything is queued."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wavefilter.h")


@pytest.fixture(scope="module")
def wfpkg():
    lib = os.path.join(ROOT, "paper_2606_00724_amd", "libwavefilter.so")
    if not os.path.exists(lib):
        # the build script does not import the package (no library needed)
        import importlib.util
        spec = importlib.util.spec_from_file_location(
            "wf_build", os.path.join(ROOT, "paper_2606_00724_amd", "build.py"))
        mod = importlib.util.module_from_spec(spec)
        spec.loader.exec_module(mod)
        mod.build()
    import paper_2606_00724_amd as wf
    return wf


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wf_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("wf_dwt_keys", "wf_skim_score", "wf_scan_select",
                     "wf_gather_kv", "wf_sparse_attn", "wf_filter_attend"):
        assert required in names


def test_every_declared_symbol_is_exported(wfpkg):
    lib = ctypes.CDLL(wfpkg.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing
    assert set(declared_functions()) == set(wfpkg.EXPORTED)


def test_status_strings(wfpkg):
    lib = wfpkg.library()
    for code, name in wfpkg._STATUS.items():
        assert lib.wf_status_str(code).decode() == name


def _params(wfpkg, **kw):
    base = dict(batch=1, heads=2, ctx_len=1024, head_dim=64, q_len=32,
                levels=3, segments=8, budget=128, dtype="f32")
    base.update(kw)
    return wfpkg.make_params(**base)


@pytest.mark.parametrize("change,code", [
    (dict(head_dim=96), 2),
    (dict(q_len=0), 1),
    (dict(q_len=257), 2),
    (dict(levels=0), 1),
    (dict(levels=11), 2),
    (dict(ctx_len=4, levels=3), 1),
    (dict(segments=0), 1),
    (dict(segments=129), 1),
    (dict(budget=0), 1),
    (dict(gen_len=-1), 1),
    (dict(batch=0), 1),
    (dict(wavelet=7), 1),
    (dict(boundary=5), 1),
    (dict(dtype=9), 1),
    (dict(scale=float("inf")), 1),
])
def test_invalid_params_are_rejected_on_the_host(wfpkg, change, code):
    p = _params(wfpkg, **change)
    lib = wfpkg.library()
    fake = ctypes.c_void_p(0x10000)
    rc = lib.wf_filter_attend(ctypes.byref(p), fake, fake, fake, None, None,
                              fake, None, None, fake, 1 << 40, None)
    assert rc == code, lib.wf_last_error()
    assert lib.wf_last_error().decode()
    assert wfpkg.workspace_bytes(p, wfpkg.OP_FUSED) == 0
    assert wfpkg.effective_budget(p) == -1


def test_pointer_and_workspace_checks(wfpkg):
    p = _params(wfpkg)
    lib = wfpkg.library()
    good = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10008)
    need = wfpkg.workspace_bytes(p, wfpkg.OP_FUSED)
    assert need > 0
    call = lambda Q, K, V, O, ws, nb, Kg=None, Vg=None: lib.wf_filter_attend(
        ctypes.byref(p), Q, K, V, Kg, Vg, O, None, None, ws, nb, None)
    assert call(None, good, good, good, good, need) == 1
    assert call(good, odd, good, good, good, need) == 1
    assert call(good, good, good, good, None, need) == 3
    assert call(good, good, good, good, good, need - 1) == 3
    assert call(good, good, good, good, ctypes.c_void_p(0x10010), need) == 3
    pg = _params(wfpkg, gen_len=4)
    rc = lib.wf_filter_attend(ctypes.byref(pg), good, good, good, None, None,
                              good, None, None, good, 1 << 40, None)
    assert rc == 1 and b"Kg" in lib.wf_last_error()
    assert lib.wf_sparse_attn(ctypes.byref(p), good, good, good, 0, good,
                              good, 1 << 40, None) == 1


def test_budget_and_workspace_arithmetic(wfpkg):
    p = _params(wfpkg)                       # S 2^J = 64 < k = 128
    assert wfpkg.effective_budget(p) == 64
    p2 = _params(wfpkg, segments=32)         # pool 256 > k
    assert wfpkg.effective_budget(p2) == 128
    a = wfpkg.workspace_bytes(p, wfpkg.OP_FUSED)
    b = wfpkg.workspace_bytes(_params(wfpkg, batch=4), wfpkg.OP_FUSED)
    assert b > a > 0
    for op in (wfpkg.OP_SKIM, wfpkg.OP_SCAN, wfpkg.OP_ATTN):
        assert 0 < wfpkg.workspace_bytes(p, op) <= a
    assert wfpkg.workspace_bytes(p, 17) == 0
    assert wfpkg.fused_kernel_names(p)[0] == "skim_tile"


@pytest.mark.parametrize("change,path", [
    (dict(), "general"),                                   # fp32 keys
    (dict(dtype="bf16"), "token"),
    (dict(dtype="bf16", levels=5), "token"),
    (dict(dtype="bf16", levels=2), "wide"),                # blocks < 8 tokens
    (dict(dtype="bf16", levels=6), "wide"),                # blocks > 32 tokens
    (dict(dtype="bf16", q_len=65), "general"),             # > 64 query rows
    (dict(dtype="bf16", wavelet="db2"), "wide"),
    (dict(dtype="bf16", wavelet="db2", levels=6, segments=4), "token"),   # db2 band over token logits
    (dict(dtype="bf16", wavelet="db2", levels=6, segments=2, ctx_len=192), "general"),  # 3 coefficients
    (dict(dtype="bf16", wavelet="db2", levels=7, segments=2), "wide"),
])
def test_fused_kernel_sequence_follows_the_path(wfpkg, change, path):
    """Token-level path for bf16 Haar at 3..5 levels (db2 at 6); otherwise
    coefficient tiles, and with bf16 keys, at most 64 query rows and a
    multiple of 4 coefficients W over all CUs with the top-S in the
    statistics pass and the top-k in the attention."""
    p = _params(wfpkg, **change)
    names = wfpkg.fused_kernel_names(p)
    if path == "token":
        assert names == ["token_skim", "block_weights", "scan_weights",
                         "sparse_attn", "attn_combine"]
    elif path == "wide":
        assert names == ["skim_tile", "skim_weights", "scan_stats",
                         "scan_weights", "sparse_attn", "attn_combine"]
    else:
        assert names == ["skim_tile", "skim_select", "scan_stats",
                         "scan_weights", "scan_select", "sparse_attn",
                         "attn_combine"]
    # the token path's workspace holds block statistics, not scan slices
    assert wfpkg.workspace_bytes(p, wfpkg.OP_FUSED) > 0


@pytest.mark.parametrize("change,selects,wide", [
    (dict(), False, False),                   # fp32 keys: the select kernels
    (dict(dtype="bf16"), True, True),
    (dict(dtype="bf16", q_len=256), True, False),   # past 64 query rows
    (dict(dtype="bf16", wavelet="db2"), True, True),
    (dict(dtype="bf16", ctx_len=1048), True, False),  # 131 coefficients
])
def test_cached_step_attention_selects_with_bf16_keys(wfpkg, change, selects,
                                                      wide):
    """With bf16 keys the attention takes the top-k itself; with at most 64
    query rows and a multiple of 4 coefficients W is formed over all CUs and
    the statistics pass takes the top-S."""
    p = _params(wfpkg, **change)
    names = wfpkg.cached_kernel_names(p)
    head = ["skim_tile", "skim_weights" if wide else "skim_select",
            "scan_stats", "scan_weights"]
    tail = ["sparse_attn", "attn_combine"]
    assert names == head + ([] if selects else ["scan_select"]) + tail


def test_shared_selection_kernel_sequences(wfpkg):
    p = _params(wfpkg, dtype="bf16", heads=4)
    assert wfpkg.shared_kernel_names(p) == [
        "token_skim", "block_weights", "head_sum_w", "scan_weights",
        "head_sum_wpool", "sparse_attn", "attn_combine"]
    # the fused regions plus the heads' sums and the shared regions
    assert (wfpkg.workspace_bytes(p, wfpkg.OP_SHARED)
            > wfpkg.workspace_bytes(p, wfpkg.OP_FUSED))
    pf = _params(wfpkg, heads=4)               # fp32: the general path
    assert wfpkg.shared_kernel_names(pf) == [
        "skim_tile", "skim_weights", "head_sum_w", "select_regions",
        "scan_stats", "scan_weights", "head_sum_wpool", "scan_select",
        "sparse_attn", "attn_combine"]
    # 131 coefficients: W comes from the per-unit skim select
    po = _params(wfpkg, heads=4, ctx_len=1048)
    assert wfpkg.shared_kernel_names(po)[1] == "skim_select"
    assert (wfpkg.workspace_bytes(pf, wfpkg.OP_SHARED)
            > wfpkg.workspace_bytes(pf, wfpkg.OP_FUSED))
    lib = wfpkg.library()
    good = ctypes.c_void_p(0x10000)
    # pointers and workspace are checked before anything is queued
    rc = lib.wf_filter_attend_shared(ctypes.byref(p), good, good, good, None,
                                     None, None, None, None, good, 1 << 40,
                                     None)
    assert rc == 1 and b"O" in lib.wf_last_error()
    need = wfpkg.workspace_bytes(p, wfpkg.OP_SHARED)
    rc = lib.wf_filter_attend_shared(ctypes.byref(p), good, good, good, None,
                                     None, good, None, None, good, need - 1,
                                     None)
    assert rc == 3


def test_binding_rejects_host_tensors(wfpkg):
    import torch
    p = _params(wfpkg)
    x = torch.zeros(4)
    with pytest.raises(ValueError):
        wfpkg.wf_dwt_keys(p, x, x)


def test_product_path_does_not_use_the_oracle():
    """The GPU path never imports, links or loads the CPU oracle."""
    pkg = os.path.join(ROOT, "paper_2606_00724_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read().lower()
                assert "oracle" not in text, f
    assert "oracle" not in open(HEADER).read().lower()


# ------------------------------------------------------------ recursion

@pytest.mark.parametrize("levels,props", [
    (1, [0.25]), (2, [0.5, 0.25]), (3, [0.3, 0.55, 0.01]),
    (5, [0.9, 0.7, 0.5, 0.5, 0.125])])
def test_recursion_counts_match_the_oracle(wfpkg, ref, levels, props):
    """The library's count arithmetic equals the oracle's on the same
    (float32) proportions: c_b = max(1, ceil(m_b n_b)), n_b = 2 c_{b+1}."""
    import numpy as np
    p = _params(wfpkg, ctx_len=2048, levels=levels, dtype="bf16")
    got = wfpkg.recursion_counts(p, props)
    n = 2048 >> levels
    want = [0] * levels
    for b in range(levels, 0, -1):
        want[b - 1] = ref.recursion_count(float(np.float32(props[b - 1])), n)
        n = 2 * want[b - 1]
    assert got == want
    assert wfpkg.recursive_workspace_bytes(p, props) > 0


@pytest.mark.parametrize("props", [[0.0, 0.5], [1.5, 0.5], [float("nan"), 1.0],
                                   [0.5, -0.1]])
def test_recursion_rejects_bad_proportions(wfpkg, props):
    lib = wfpkg.library()
    p = _params(wfpkg, levels=2, dtype="bf16")
    arr = (ctypes.c_float * 2)(*props)
    out = (ctypes.c_int32 * 2)()
    assert lib.wf_recursion_counts(ctypes.byref(p), arr, out) == 1
    assert lib.wf_recursive_workspace_bytes(ctypes.byref(p), arr) == 0
    assert lib.wf_recursion_counts(ctypes.byref(p), None, out) == 1


def test_recursion_db2_kernel_sequence(wfpkg):
    """The db2 recursion runs coefficient tiles at every scale (the token
    path is Haar's), two kernels a scale, then the attention."""
    p = _params(wfpkg, levels=2, dtype="bf16", wavelet="db2")
    assert wfpkg.recursive_kernel_names(p) == [
        "rec_tiles_b2", "rec_select_b2", "rec_tiles_b1", "rec_select_b1",
        "sparse_attn", "attn_combine"]
    assert wfpkg.recursive_workspace_bytes(p, [0.5, 0.5]) > 0


def test_recursion_kernel_sequence(wfpkg):
    p = _params(wfpkg, levels=3, dtype="bf16")
    assert wfpkg.recursive_kernel_names(p) == [
        "rec_tiles_b3", "rec_select_b3", "rec_tiles_b2", "rec_select_b2",
        "rec_tiles_b1", "rec_select_b1", "sparse_attn", "attn_combine"]


# ------------------------------------------------------------ binding checks

def _fused_tensors(wfpkg, p):
    import torch
    dt = wfpkg.torch_dtype(p)
    U, d = p.batch * p.heads, p.head_dim
    return dict(
        Q=torch.zeros((p.batch, p.heads, p.q_len, d), dtype=dt),
        K=torch.zeros((p.batch, p.heads, p.ctx_len, d), dtype=dt),
        V=torch.zeros((p.batch, p.heads, p.ctx_len, d), dtype=dt),
        O=torch.zeros((p.batch, p.heads, p.q_len, d), dtype=dt),
        tok=torch.zeros(U * wfpkg.effective_budget(p), dtype=torch.int32),
        seg=torch.zeros(U * p.segments, dtype=torch.int32))


@pytest.mark.parametrize("field,bad,err,needle", [
    ("K", lambda t: t.to(__import__("torch").bfloat16), TypeError, "K: dtype"),
    ("V", lambda t: t[:, :, :-1].contiguous(), ValueError, "V:"),
    ("Q", lambda t: t.double(), TypeError, "Q: dtype"),
    ("O", lambda t: t[:, :1].contiguous(), ValueError, "O:"),
    ("tok", lambda t: t[:-1].contiguous(), ValueError, "tok_idx:"),
    ("seg", lambda t: t.long(), TypeError, "seg_idx: dtype"),
])
def test_binding_checks_types_and_sizes(wfpkg, field, bad, err, needle):
    """The wrappers compare every tensor's element type and count with the
    parameters before anything reaches the library (the kernels index the
    buffers by the parameters alone)."""
    p = _params(wfpkg)
    t = _fused_tensors(wfpkg, p)
    t[field] = bad(t[field])
    with pytest.raises(err, match=needle):
        wfpkg.wf_filter_attend(p, t["Q"], t["K"], t["V"], None, None, t["O"],
                               t["tok"], t["seg"], None)


def test_binding_checks_the_tail_and_approximation(wfpkg):
    import torch
    pg = _params(wfpkg, gen_len=4)
    t = _fused_tensors(wfpkg, pg)
    with pytest.raises(ValueError, match="Kg is required"):
        wfpkg.wf_filter_attend(pg, t["Q"], t["K"], t["V"], None, None, t["O"],
                               None, None, None)
    p = _params(wfpkg)
    t = _fused_tensors(wfpkg, p)
    A = torch.zeros((p.batch, p.heads, (p.ctx_len >> p.levels) - 1, p.head_dim))
    with pytest.raises(ValueError, match="approx:"):
        wfpkg.wf_filter_attend_cached(p, t["Q"], A, t["K"], t["V"], None, None,
                                      t["O"], None, None, None)
    K16 = t["K"].to(torch.bfloat16)
    with pytest.raises(TypeError, match="K: dtype"):
        wfpkg.wf_dwt_keys(p, K16, A)


def test_binding_checks_shared_outputs(wfpkg):
    """The shared call's index outputs hold one list per sequence."""
    import torch
    p = _params(wfpkg, dtype="bf16", heads=4)
    t = _fused_tensors(wfpkg, p)
    per_unit = torch.zeros(p.batch * p.heads * wfpkg.effective_budget(p),
                           dtype=torch.int32)
    with pytest.raises(ValueError, match="tok_idx:"):
        wfpkg.wf_filter_attend_shared(p, t["Q"], t["K"], t["V"], None, None,
                                      t["O"], per_unit, None, None)
    seg = torch.zeros(p.batch * p.segments + 1, dtype=torch.int32)
    with pytest.raises(ValueError, match="seg_idx:"):
        wfpkg.wf_filter_attend_shared(p, t["Q"], t["K"], t["V"], None, None,
                                      t["O"], None, seg, None)


def test_binding_checks_recursion_outputs(wfpkg):
    import torch
    p = _params(wfpkg, levels=3, dtype="bf16")
    props = [0.5, 0.5, 0.25]
    counts = wfpkg.recursion_counts(p, props)
    t = _fused_tensors(wfpkg, p)
    U = p.batch * p.heads
    assert wfpkg.kept_elements(p, props) == U * (counts[1] + counts[2])
    kept = torch.zeros(wfpkg.kept_elements(p, props) + 1, dtype=torch.int32)
    tok = torch.zeros(U * 2 * counts[0], dtype=torch.int32)
    with pytest.raises(ValueError, match="kept_idx:"):
        wfpkg.wf_filter_attend_recursive(p, props, t["Q"], t["K"], t["V"],
                                         None, None, t["O"], tok, None,
                                         kept_idx=kept)
    with pytest.raises(ValueError, match="tok_idx:"):
        wfpkg.wf_filter_attend_recursive(p, props, t["Q"], t["K"], t["V"],
                                         None, None, t["O"], tok[1:], None)


def test_noalloc_rejects_oversized_parameters_on_the_host(wfpkg):
    """The allocation-free entry point refuses parameters whose workspace is
    larger than its scratch, before touching the device."""
    p = _params(wfpkg, batch=4, heads=32, ctx_len=32768, head_dim=128,
                q_len=64, levels=5, segments=128, budget=2048, dtype="bf16")
    assert wfpkg.workspace_bytes(p, wfpkg.OP_FUSED) > wfpkg.NOALLOC_SCRATCH_BYTES
    lib = wfpkg.library()
    fake = ctypes.c_void_p(0x10000)
    rc = lib.wf_filter_attend_noalloc(ctypes.byref(p), fake, fake, fake, None,
                                      None, fake, None, None, None)
    assert rc == 3 and b"scratch" in lib.wf_last_error()
    bad = _params(wfpkg, head_dim=96)
    assert lib.wf_filter_attend_noalloc(ctypes.byref(bad), fake, fake, fake,
                                        None, None, fake, None, None,
                                        None) == 2
