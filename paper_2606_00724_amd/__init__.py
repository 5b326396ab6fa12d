"""Python binding of libwavefilter.so, the gfx950 WaveFilter filter+attend path.

Argument marshalling only: every ``wf_*`` function here forwards torch device
tensors (pointers) and a HIP stream to the C entry point of the same name
declared in include/wavefilter.h, and raises :class:`WfError` on a non-OK
status.  Torch supplies device memory and streams; all arithmetic runs in the
library's HIP kernels.  There is no fallback: importing this package fails if
the library has not been built (``python -m paper_2606_00724_amd.build``).
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwavefilter.so")

HAAR, DB2 = 0, 1
EXT_SYMMETRIC, EXT_PERIODIC = 0, 1
BF16, F32 = 0, 1
OP_SKIM, OP_SCAN, OP_ATTN, OP_FUSED, OP_CACHED, OP_SHARED = 0, 1, 2, 3, 4, 5
MAX_LEVELS, MAX_Q_LEN = 10, 256
NOALLOC_SCRATCH_BYTES = 32 << 20

_STATUS = {0: "WF_OK", 1: "WF_ERR_INVALID_ARG", 2: "WF_ERR_UNSUPPORTED",
           3: "WF_ERR_WORKSPACE", 4: "WF_ERR_HIP"}

EXPORTED = ("wf_workspace_bytes", "wf_effective_budget", "wf_dwt_keys",
            "wf_skim_score", "wf_scan_select", "wf_gather_kv",
            "wf_sparse_attn", "wf_filter_attend", "wf_filter_attend_timed",
            "wf_filter_attend_noalloc",
            "wf_filter_attend_kernels", "wf_filter_attend_kernel_name",
            "wf_filter_attend_cached", "wf_filter_attend_cached_timed",
            "wf_filter_attend_cached_kernels",
            "wf_filter_attend_cached_kernel_name",
            "wf_filter_attend_shared", "wf_filter_attend_shared_timed",
            "wf_filter_attend_shared_kernels",
            "wf_filter_attend_shared_kernel_name",
            "wf_recursion_counts", "wf_recursive_workspace_bytes",
            "wf_filter_attend_recursive", "wf_filter_attend_recursive_timed",
            "wf_filter_attend_recursive_kernels",
            "wf_filter_attend_recursive_kernel_name",
            "wf_init", "wf_status_str", "wf_last_error")


class WfParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "batch", "heads", "ctx_len", "head_dim", "q_len", "gen_len", "levels",
        "wavelet", "boundary", "dtype", "segments", "budget")] + [
        ("scale", ctypes.c_float)]

    def as_dict(self) -> dict:
        return {n: getattr(self, n) for n, _ in self._fields_}


class WfError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        self.status_name = _STATUS.get(status, str(status))
        super().__init__(f"{self.status_name}: {message}")


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with "
            "`python -m paper_2606_00724_amd.build` (hipcc, gfx950)")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER(WfParams)
    vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32
    fp, ip = ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_int32)
    sig = {
        "wf_workspace_bytes": (sz, [P, i32]),
        "wf_effective_budget": (i32, [P]),
        "wf_dwt_keys": (ctypes.c_int, [P, vp, vp, vp, vp]),
        "wf_skim_score": (ctypes.c_int, [P, vp, vp, vp, vp, vp, sz, vp]),
        "wf_scan_select": (ctypes.c_int, [P, vp, vp, vp, vp, vp, vp, sz, vp]),
        "wf_gather_kv": (ctypes.c_int, [P, vp, vp, vp, vp, vp, vp, vp, vp]),
        "wf_sparse_attn": (ctypes.c_int, [P, vp, vp, vp, i32, vp, vp, sz, vp]),
        "wf_filter_attend": (ctypes.c_int,
                             [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "wf_filter_attend_timed": (ctypes.c_int,
                                   [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                    vp, ctypes.POINTER(vp), i32]),
        "wf_filter_attend_noalloc": (ctypes.c_int,
                                     [P, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
        "wf_filter_attend_shared": (ctypes.c_int,
                                    [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                     vp]),
        "wf_filter_attend_shared_timed": (ctypes.c_int,
                                          [P, vp, vp, vp, vp, vp, vp, vp, vp,
                                           vp, sz, vp, ctypes.POINTER(vp),
                                           i32]),
        "wf_filter_attend_shared_kernels": (i32, [P]),
        "wf_filter_attend_shared_kernel_name": (ctypes.c_char_p, [P, i32]),
        "wf_filter_attend_kernels": (i32, [P]),
        "wf_filter_attend_kernel_name": (ctypes.c_char_p, [P, i32]),
        "wf_filter_attend_cached": (ctypes.c_int,
                                    [P, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                     vp, sz, vp]),
        "wf_filter_attend_cached_timed": (ctypes.c_int,
                                          [P, vp, vp, vp, vp, vp, vp, vp, vp,
                                           vp, vp, sz, vp, ctypes.POINTER(vp),
                                           i32]),
        "wf_filter_attend_cached_kernels": (i32, [P]),
        "wf_filter_attend_cached_kernel_name": (ctypes.c_char_p, [P, i32]),
        "wf_recursion_counts": (ctypes.c_int, [P, fp, ip]),
        "wf_recursive_workspace_bytes": (sz, [P, fp]),
        "wf_filter_attend_recursive": (ctypes.c_int,
                                       [P, fp, vp, vp, vp, vp, vp, vp, vp, vp,
                                        vp, sz, vp]),
        "wf_filter_attend_recursive_timed": (ctypes.c_int,
                                             [P, fp, vp, vp, vp, vp, vp, vp,
                                              vp, vp, vp, sz, vp,
                                              ctypes.POINTER(vp), i32]),
        "wf_filter_attend_recursive_kernels": (i32, [P]),
        "wf_filter_attend_recursive_kernel_name": (ctypes.c_char_p, [P, i32]),
        "wf_init": (ctypes.c_int, []),
        "wf_status_str": (ctypes.c_char_p, [ctypes.c_int]),
        "wf_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def library() -> ctypes.CDLL:
    return _lib


# ------------------------------------------------------------ parameters

def make_params(*, batch: int, heads: int, ctx_len: int, head_dim: int,
                q_len: int, levels: int, segments: int, budget: int,
                gen_len: int = 0, wavelet: str | int = "haar",
                boundary: str | int = "symmetric", dtype: str | int = "bf16",
                scale: float = 0.0) -> WfParams:
    w = {"haar": HAAR, "db2": DB2}.get(wavelet, wavelet)
    b = {"symmetric": EXT_SYMMETRIC, "periodic": EXT_PERIODIC}.get(boundary,
                                                                   boundary)
    dt = {"bf16": BF16, "f32": F32, torch.bfloat16: BF16,
          torch.float32: F32}.get(dtype, dtype)
    return WfParams(batch, heads, ctx_len, head_dim, q_len, gen_len, levels,
                    w, b, dt, segments, budget, scale)


def params_for(w, gen_len: int | None = None) -> WfParams:
    """Parameters of a workload description (any object with the fields of
    ``synth.Workload``)."""
    return make_params(batch=w.batch, heads=w.heads, ctx_len=w.ctx_len,
                       head_dim=w.head_dim, q_len=w.q_len, levels=w.levels,
                       segments=w.segments, budget=w.budget,
                       gen_len=w.gen_len if gen_len is None else gen_len,
                       wavelet=w.wavelet, boundary=w.boundary, dtype=w.dtype)


def torch_dtype(p: WfParams) -> torch.dtype:
    return torch.bfloat16 if p.dtype == BF16 else torch.float32


def workspace_bytes(p: WfParams, op: int) -> int:
    return int(_lib.wf_workspace_bytes(ctypes.byref(p), op))


def effective_budget(p: WfParams) -> int:
    return int(_lib.wf_effective_budget(ctypes.byref(p)))


def fused_kernel_names(p: WfParams) -> list[str]:
    n = _lib.wf_filter_attend_kernels(ctypes.byref(p))
    return [_lib.wf_filter_attend_kernel_name(ctypes.byref(p), i).decode()
            for i in range(n)]


# ------------------------------------------------------------ marshalling

def _ptr(t) -> int | None:
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"expected a torch tensor, got {type(t).__name__}")
    if t.device.type != "cuda":
        raise ValueError("tensors passed to the WaveFilter library must be on "
                         "a GPU")
    if not t.is_contiguous():
        raise ValueError("tensors passed to the WaveFilter library must be "
                         "contiguous")
    return t.data_ptr()


def _expect(t, name: str, dtype: torch.dtype, numel: int,
            nullable: bool = False) -> None:
    """The element type and count a tensor must have for these parameters
    (the kernels index it by the parameters alone)."""
    if t is None:
        if nullable:
            return
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor, got {type(t).__name__}")
    if t.dtype != dtype:
        raise TypeError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if t.numel() != numel:
        raise ValueError(f"{name}: {t.numel()} elements, expected {numel} "
                         f"for these parameters")


def _units(p) -> int:
    return p.batch * p.heads


def _remainder(p) -> int:
    return p.ctx_len - ((p.ctx_len >> p.levels) << p.levels)


def _expect_qkv(p, Q=None, K=None, V=None, Kg=None, Vg=None, O=None,
                tail: bool = False) -> None:
    """Q/O, K/V (when given) and, for calls that read the generation tail,
    Kg/Vg (required iff gen_len > 0)."""
    dt, U, d = torch_dtype(p), _units(p), p.head_dim
    for name, t in (("Q", Q), ("O", O)):
        if t is not None:
            _expect(t, name, dt, U * p.q_len * d)
    for name, t in (("K", K), ("V", V)):
        if t is not None:
            _expect(t, name, dt, U * p.ctx_len * d)
    if tail:
        for name, t in (("Kg", Kg), ("Vg", Vg)):
            _expect(t, name, dt, U * p.gen_len * d, nullable=p.gen_len == 0)


def _ws(t) -> tuple[int | None, int]:
    if t is None:
        return None, 0
    return _ptr(t), t.numel() * t.element_size()


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _torch_stream(stream) -> torch.cuda.Stream:
    """The stream the library will queue on, as a torch stream, so that the
    buffers a wrapper allocates belong to it (the caching allocator then
    reuses them only after the kernels queued there)."""
    if stream is None:
        return torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream))


def _check(status: int) -> None:
    if status != 0:
        raise WfError(status, _lib.wf_last_error().decode())


def wf_init():
    """Loads the library's kernels onto the current device (optional: the
    first call on a device otherwise does it, stalling that call)."""
    _check(_lib.wf_init())


def wf_dwt_keys(p, K, approx, details=None, stream=None):
    U, d = _units(p), p.head_dim
    Lf = (p.ctx_len >> p.levels) << p.levels
    _expect_qkv(p, K=K)
    _expect(approx, "approx", torch.float32, U * (p.ctx_len >> p.levels) * d)
    _expect(details, "details", torch.float32,
            U * sum(Lf >> j for j in range(1, p.levels + 1)) * d, nullable=True)
    _check(_lib.wf_dwt_keys(ctypes.byref(p), _ptr(K), _ptr(approx),
                            _ptr(details), _stream(stream)))


def wf_skim_score(p, Q, approx, seg_score, seg_idx, workspace, stream=None):
    U, nJ = _units(p), p.ctx_len >> p.levels
    _expect_qkv(p, Q=Q)
    _expect(approx, "approx", torch.float32, U * nJ * p.head_dim)
    _expect(seg_score, "seg_score", torch.float32, U * nJ)
    _expect(seg_idx, "seg_idx", torch.int32, U * p.segments)
    ws, nb = _ws(workspace)
    _check(_lib.wf_skim_score(ctypes.byref(p), _ptr(Q), _ptr(approx),
                              _ptr(seg_score), _ptr(seg_idx), ws, nb,
                              _stream(stream)))


def wf_scan_select(p, Q, K, seg_idx, tok_score, tok_idx, workspace,
                   stream=None):
    U = _units(p)
    _expect_qkv(p, Q=Q, K=K)
    _expect(seg_idx, "seg_idx", torch.int32, U * p.segments)
    _expect(tok_score, "tok_score", torch.float32,
            U * (p.segments << p.levels), nullable=True)
    _expect(tok_idx, "tok_idx", torch.int32, U * effective_budget(p))
    ws, nb = _ws(workspace)
    _check(_lib.wf_scan_select(ctypes.byref(p), _ptr(Q), _ptr(K),
                               _ptr(seg_idx), _ptr(tok_score), _ptr(tok_idx),
                               ws, nb, _stream(stream)))


def wf_gather_kv(p, K, V, tok_idx, Kg, Vg, Ks, Vs, stream=None):
    U, keff = _units(p), effective_budget(p)
    _expect_qkv(p, K=K, V=V, Kg=Kg, Vg=Vg, tail=True)
    _expect(tok_idx, "tok_idx", torch.int32, U * keff)
    rows = keff + _remainder(p) + p.gen_len
    for name, t in (("Ks", Ks), ("Vs", Vs)):
        _expect(t, name, torch_dtype(p), U * rows * p.head_dim)
    _check(_lib.wf_gather_kv(ctypes.byref(p), _ptr(K), _ptr(V), _ptr(tok_idx),
                             _ptr(Kg), _ptr(Vg), _ptr(Ks), _ptr(Vs),
                             _stream(stream)))


def wf_sparse_attn(p, Q, Ks, Vs, n_kv, O, workspace, stream=None):
    _expect_qkv(p, Q=Q, O=O)
    for name, t in (("Ks", Ks), ("Vs", Vs)):
        _expect(t, name, torch_dtype(p), _units(p) * int(n_kv) * p.head_dim)
    ws, nb = _ws(workspace)
    _check(_lib.wf_sparse_attn(ctypes.byref(p), _ptr(Q), _ptr(Ks), _ptr(Vs),
                               int(n_kv), _ptr(O), ws, nb, _stream(stream)))


def _expect_fused(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx) -> None:
    _expect_qkv(p, Q=Q, K=K, V=V, Kg=Kg, Vg=Vg, O=O, tail=True)
    _expect(tok_idx, "tok_idx", torch.int32, _units(p) * effective_budget(p),
            nullable=True)
    _expect(seg_idx, "seg_idx", torch.int32, _units(p) * p.segments,
            nullable=True)


def wf_filter_attend(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx, workspace,
                     stream=None):
    _expect_fused(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx)
    ws, nb = _ws(workspace)
    _check(_lib.wf_filter_attend(ctypes.byref(p), _ptr(Q), _ptr(K), _ptr(V),
                                 _ptr(Kg), _ptr(Vg), _ptr(O), _ptr(tok_idx),
                                 _ptr(seg_idx), ws, nb, _stream(stream)))


def wf_filter_attend_noalloc(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx,
                             stream=None):
    """wf_filter_attend on the library's own per-device scratch: no
    workspace, nothing allocated (calls that overlap on one GPU race)."""
    _expect_fused(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx)
    _check(_lib.wf_filter_attend_noalloc(ctypes.byref(p), _ptr(Q), _ptr(K),
                                         _ptr(V), _ptr(Kg), _ptr(Vg), _ptr(O),
                                         _ptr(tok_idx), _ptr(seg_idx),
                                         _stream(stream)))


def wf_filter_attend_timed(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx,
                           workspace, events, stream=None):
    """``events``: sequence of raw hipEvent_t handles (ints)."""
    _expect_fused(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx)
    ws, nb = _ws(workspace)
    arr = (ctypes.c_void_p * len(events))(*events)
    _check(_lib.wf_filter_attend_timed(ctypes.byref(p), _ptr(Q), _ptr(K),
                                       _ptr(V), _ptr(Kg), _ptr(Vg), _ptr(O),
                                       _ptr(tok_idx), _ptr(seg_idx), ws, nb,
                                       _stream(stream), arr, len(events)))


# ------------------------------------------------------------ grouped heads
# Grouped-query attention: g query heads share one KV head.  Their selection
# is one selection per KV head with W summed over the g heads' query rows;
# since W is a column sum of row-wise softmaxes, that is the selection of the
# stacked block of g * B rows, and attention is row-wise, so the stacked call
# also returns every head's own output.  Heads of a group are adjacent
# (query head h uses KV head h // g), which makes the stacking a view.

def grouped_view(Q: torch.Tensor, group: int) -> torch.Tensor:
    """[batch, heads_q, B, d] -> [batch, heads_q // group, group * B, d]."""
    b, hq, B, d = Q.shape
    if hq % group:
        raise ValueError(f"{hq} query heads are not groups of {group}")
    return Q.reshape(b, hq // group, group * B, d)


def filter_attend_grouped(p_kv: WfParams, group: int, Q, K, V, Kg=None,
                          Vg=None, want_indices: bool = False, stream=None):
    """One selection per KV head for its `group` query heads.  p_kv: the
    parameters with heads = KV heads and q_len = group * B.  Returns O
    [batch, heads_q, B, d] (and the per-KV-head tok, seg)."""
    Qs = grouped_view(Q, group)
    if p_kv.heads != Qs.shape[1] or p_kv.q_len != Qs.shape[2]:
        raise ValueError("p_kv must describe the stacked query blocks")
    out = filter_attend(p_kv, Qs, K, V, Kg, Vg, want_indices=want_indices,
                        stream=stream)
    if want_indices:
        O, tok, seg = out
        return O.reshape(Q.shape), tok, seg
    return out.reshape(Q.shape)


# ------------------------------------------------------------ shared selection
# One selection per sequence, shared by its heads (W and W' summed over the
# heads before each top-k); every head attends over the shared tokens.

def shared_kernel_names(p: WfParams) -> list[str]:
    n = _lib.wf_filter_attend_shared_kernels(ctypes.byref(p))
    return [_lib.wf_filter_attend_shared_kernel_name(ctypes.byref(p),
                                                     i).decode()
            for i in range(max(n, 0))]


def _expect_shared(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx) -> None:
    _expect_qkv(p, Q=Q, K=K, V=V, Kg=Kg, Vg=Vg, O=O, tail=True)
    _expect(tok_idx, "tok_idx", torch.int32, p.batch * effective_budget(p),
            nullable=True)
    _expect(seg_idx, "seg_idx", torch.int32, p.batch * p.segments,
            nullable=True)


def wf_filter_attend_shared(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx,
                            workspace, stream=None):
    _expect_shared(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx)
    ws, nb = _ws(workspace)
    _check(_lib.wf_filter_attend_shared(
        ctypes.byref(p), _ptr(Q), _ptr(K), _ptr(V), _ptr(Kg), _ptr(Vg),
        _ptr(O), _ptr(tok_idx), _ptr(seg_idx), ws, nb, _stream(stream)))


def wf_filter_attend_shared_timed(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx,
                                  workspace, events, stream=None):
    _expect_shared(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx)
    ws, nb = _ws(workspace)
    arr = (ctypes.c_void_p * len(events))(*events)
    _check(_lib.wf_filter_attend_shared_timed(
        ctypes.byref(p), _ptr(Q), _ptr(K), _ptr(V), _ptr(Kg), _ptr(Vg),
        _ptr(O), _ptr(tok_idx), _ptr(seg_idx), ws, nb, _stream(stream), arr,
        len(events)))


def filter_attend_shared(p: WfParams, Q, K, V, Kg=None, Vg=None,
                         workspace=None, want_indices: bool = False,
                         stream=None):
    """Allocates O (and the per-sequence index outputs tok [batch, k_eff],
    seg [batch, S]) and runs wf_filter_attend_shared.  Returns O, or (O,
    tok, seg) when want_indices."""
    with torch.cuda.stream(_torch_stream(stream)):
        O = torch.empty_like(Q)
        tok = seg = None
        if want_indices:
            tok = torch.empty((p.batch, effective_budget(p)),
                              dtype=torch.int32, device=Q.device)
            seg = torch.empty((p.batch, p.segments), dtype=torch.int32,
                              device=Q.device)
        if workspace is None:
            workspace = alloc_workspace(p, OP_SHARED, Q.device)
    wf_filter_attend_shared(p, Q, K, V, Kg, Vg, O, tok, seg, workspace,
                            stream)
    return (O, tok, seg) if want_indices else O


# ------------------------------------------------------------ cached A_J
# A_J of the prompt keys (wf_dwt_keys) reused by every later step.

def cached_kernel_names(p: WfParams) -> list[str]:
    n = _lib.wf_filter_attend_cached_kernels(ctypes.byref(p))
    return [_lib.wf_filter_attend_cached_kernel_name(ctypes.byref(p),
                                                     i).decode()
            for i in range(n)]


def _expect_approx(p, approx) -> None:
    _expect(approx, "approx", torch.float32,
            _units(p) * (p.ctx_len >> p.levels) * p.head_dim)


def wf_filter_attend_cached(p, Q, approx, K, V, Kg, Vg, O, tok_idx, seg_idx,
                            workspace, stream=None):
    _expect_fused(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx)
    _expect_approx(p, approx)
    ws, nb = _ws(workspace)
    _check(_lib.wf_filter_attend_cached(
        ctypes.byref(p), _ptr(Q), _ptr(approx), _ptr(K), _ptr(V), _ptr(Kg),
        _ptr(Vg), _ptr(O), _ptr(tok_idx), _ptr(seg_idx), ws, nb,
        _stream(stream)))


def wf_filter_attend_cached_timed(p, Q, approx, K, V, Kg, Vg, O, tok_idx,
                                  seg_idx, workspace, events, stream=None):
    _expect_fused(p, Q, K, V, Kg, Vg, O, tok_idx, seg_idx)
    _expect_approx(p, approx)
    ws, nb = _ws(workspace)
    arr = (ctypes.c_void_p * len(events))(*events)
    _check(_lib.wf_filter_attend_cached_timed(
        ctypes.byref(p), _ptr(Q), _ptr(approx), _ptr(K), _ptr(V), _ptr(Kg),
        _ptr(Vg), _ptr(O), _ptr(tok_idx), _ptr(seg_idx), ws, nb,
        _stream(stream), arr, len(events)))


def dwt_approx(p: WfParams, K, stream=None) -> torch.Tensor:
    """A_J of K (fp32 [batch, heads, ctx_len >> levels, d])."""
    with torch.cuda.stream(_torch_stream(stream)):
        approx = torch.empty((p.batch, p.heads, p.ctx_len >> p.levels,
                              p.head_dim), dtype=torch.float32,
                             device=K.device)
    wf_dwt_keys(p, K, approx, None, stream)
    return approx


def filter_attend_cached(p: WfParams, Q, approx, K, V, Kg=None, Vg=None,
                         workspace=None, want_indices: bool = False,
                         stream=None):
    """Allocates O (and the index outputs) and runs wf_filter_attend_cached.
    Returns O, or (O, tok_idx, seg_idx) when want_indices.  What it
    allocates belongs to the stream the kernels run on."""
    with torch.cuda.stream(_torch_stream(stream)):
        O = torch.empty_like(Q)
        tok = seg = None
        if want_indices:
            tok = torch.empty((p.batch, p.heads, effective_budget(p)),
                              dtype=torch.int32, device=Q.device)
            seg = torch.empty((p.batch, p.heads, p.segments),
                              dtype=torch.int32, device=Q.device)
        if workspace is None:
            workspace = alloc_workspace(p, OP_CACHED, Q.device)
    wf_filter_attend_cached(p, Q, approx, K, V, Kg, Vg, O, tok, seg,
                            workspace, stream)
    return (O, tok, seg) if want_indices else O


# ------------------------------------------------------------ recursion
# proportions: one float per scale, m_b at index b - 1 (host values).

def _props(p: WfParams, proportions):
    vals = [float(m) for m in proportions]
    if len(vals) != p.levels:
        raise ValueError(f"{p.levels} proportions needed, got {len(vals)}")
    return (ctypes.c_float * len(vals))(*vals)


def recursion_counts(p: WfParams, proportions) -> list[int]:
    """c_b per scale (index b - 1); mu^0 has 2 c_1 positions."""
    out = (ctypes.c_int32 * p.levels)()
    _check(_lib.wf_recursion_counts(ctypes.byref(p), _props(p, proportions),
                                    out))
    return list(out)


def recursive_workspace_bytes(p: WfParams, proportions) -> int:
    return int(_lib.wf_recursive_workspace_bytes(ctypes.byref(p),
                                                 _props(p, proportions)))


def recursive_kernel_names(p: WfParams) -> list[str]:
    n = _lib.wf_filter_attend_recursive_kernels(ctypes.byref(p))
    return [_lib.wf_filter_attend_recursive_kernel_name(ctypes.byref(p),
                                                        i).decode()
            for i in range(n)]


def kept_elements(p: WfParams, proportions) -> int:
    """Elements of the kept_idx output: batch * heads * (c_B + ... + c_2)."""
    return _units(p) * sum(recursion_counts(p, proportions)[1:])


def _expect_recursive(p, proportions, Q, K, V, Kg, Vg, O, tok_idx,
                      kept_idx) -> None:
    _expect_qkv(p, Q=Q, K=K, V=V, Kg=Kg, Vg=Vg, O=O, tail=True)
    counts = recursion_counts(p, proportions)
    _expect(tok_idx, "tok_idx", torch.int32, _units(p) * 2 * counts[0],
            nullable=True)
    _expect(kept_idx, "kept_idx", torch.int32, _units(p) * sum(counts[1:]),
            nullable=True)


def wf_filter_attend_recursive(p, proportions, Q, K, V, Kg, Vg, O, tok_idx,
                               workspace, stream=None, kept_idx=None):
    _expect_recursive(p, proportions, Q, K, V, Kg, Vg, O, tok_idx, kept_idx)
    ws, nb = _ws(workspace)
    _check(_lib.wf_filter_attend_recursive(
        ctypes.byref(p), _props(p, proportions), _ptr(Q), _ptr(K), _ptr(V),
        _ptr(Kg), _ptr(Vg), _ptr(O), _ptr(tok_idx), _ptr(kept_idx), ws, nb,
        _stream(stream)))


def wf_filter_attend_recursive_timed(p, proportions, Q, K, V, Kg, Vg, O,
                                     tok_idx, workspace, events, stream=None,
                                     kept_idx=None):
    _expect_recursive(p, proportions, Q, K, V, Kg, Vg, O, tok_idx, kept_idx)
    ws, nb = _ws(workspace)
    arr = (ctypes.c_void_p * len(events))(*events)
    _check(_lib.wf_filter_attend_recursive_timed(
        ctypes.byref(p), _props(p, proportions), _ptr(Q), _ptr(K), _ptr(V),
        _ptr(Kg), _ptr(Vg), _ptr(O), _ptr(tok_idx), _ptr(kept_idx), ws, nb,
        _stream(stream), arr, len(events)))


def filter_attend_recursive(p: WfParams, proportions, Q, K, V, Kg=None,
                            Vg=None, workspace=None, stream=None,
                            want_kept: bool = False):
    """Allocates O, mu^0 and the workspace (on the stream the kernels run
    on); returns (O, tok_idx), or (O, tok_idx, kept_idx) when want_kept."""
    counts = recursion_counts(p, proportions)
    with torch.cuda.stream(_torch_stream(stream)):
        O = torch.empty_like(Q)
        tok = torch.empty((p.batch, p.heads, 2 * counts[0]),
                          dtype=torch.int32, device=Q.device)
        kept = None
        if want_kept:
            kept = torch.empty(max(1, _units(p) * sum(counts[1:])),
                               dtype=torch.int32, device=Q.device)
            kept = kept[:_units(p) * sum(counts[1:])]
        if workspace is None:
            nb = recursive_workspace_bytes(p, proportions)
            workspace = torch.empty(nb, dtype=torch.uint8, device=Q.device)
    wf_filter_attend_recursive(p, proportions, Q, K, V, Kg, Vg, O, tok,
                               workspace, stream, kept_idx=kept)
    return (O, tok, kept) if want_kept else (O, tok)


# ------------------------------------------------------------ allocation
# Torch allocates the buffers; the library only reads and writes them.

def alloc_workspace(p: WfParams, op: int, device) -> torch.Tensor | None:
    nb = workspace_bytes(p, op)
    if nb == 0:
        return None
    # torch's caching allocator returns 256-byte aligned blocks
    return torch.empty(nb, dtype=torch.uint8, device=device)


def filter_attend(p: WfParams, Q, K, V, Kg=None, Vg=None, workspace=None,
                  want_indices: bool = False, stream=None):
    """Allocates O (and the index outputs) and runs wf_filter_attend.
    Returns O, or (O, tok_idx, seg_idx) when want_indices.  What it
    allocates belongs to the stream the kernels run on."""
    with torch.cuda.stream(_torch_stream(stream)):
        O = torch.empty_like(Q)
        tok = seg = None
        if want_indices:
            tok = torch.empty((p.batch, p.heads, effective_budget(p)),
                              dtype=torch.int32, device=Q.device)
            seg = torch.empty((p.batch, p.heads, p.segments),
                              dtype=torch.int32, device=Q.device)
        if workspace is None:
            workspace = alloc_workspace(p, OP_FUSED, Q.device)
    wf_filter_attend(p, Q, K, V, Kg, Vg, O, tok, seg, workspace, stream)
    return (O, tok, seg) if want_indices else O
