"""MI355X (gfx950) chunkwise Gated Delta Rule-2 operator -- Python binding.

A thin ctypes layer over the C ABI in include/gdr2.h (libgdr2.so, built by
``python -m paper_2605_22791_amd.build``).  It only marshals arguments:
shapes and dtypes are read from the torch tensors, outputs and workspace are
allocated with torch when the caller does not pass them, and every step of the
operator runs in the HIP kernels of the library on the current torch stream.

If the library is missing the functions raise; there is no fallback.
"""

import ctypes
import os

__all__ = [
    "GDR2_OK", "GDR2_EINVAL", "GDR2_EUNSUPPORTED", "GDR2_EWORKSPACE", "GDR2_EHIP",
    "GDR2_BF16", "GDR2_FP32", "Gdr2Problem", "Gdr2Error", "lib", "lib_path",
    "gdr2_chunk_workspace_bytes", "gdr2_chunk_fwd", "gdr2_chunk_bwd", "gdr2_chunk_fwd_save",
    "gdr2_chunk_bwd_saved", "gdr2_varlen_workspace_bytes", "gdr2_chunk_fwd_varlen", "gdr2_chunk_bwd_varlen",
    "gdr2_recurrent_varlen",
    "gdr2_recurrent_step", "gdr2_status_str", "CHUNK", "KERNEL_NAMES",
    "gdr2_profile_enable", "gdr2_profile_collect", "Gdr2Stage", "gdr2_fused_workspace_bytes",
    "gdr2_fused_fwd", "gdr2_fused_bwd", "gdr2_fused_recurrent", "gdr2_chunk_fwd_noalloc",
    "NOALLOC_SCRATCH_BYTES",
]

GDR2_OK, GDR2_EINVAL, GDR2_EUNSUPPORTED, GDR2_EWORKSPACE, GDR2_EHIP = 0, 1, 2, 3, 4
GDR2_BF16, GDR2_FP32 = 0, 1
CHUNK = 64
NOALLOC_SCRATCH_BYTES = 64 << 20   # GDR2_NOALLOC_SCRATCH_BYTES in include/gdr2.h
# kernel ids of the measurement support (gdr2_kernel_id in include/gdr2.h)
KERNEL_NAMES = ["fwd_intra", "fwd_state", "bwd_recompute_intra", "bwd_recompute_state",
                "bwd_state", "bwd_wy", "bwd_intra", "recurrent", "stage_bwd", "stage_fwd"]

_HERE = os.path.dirname(os.path.abspath(__file__))


def lib_path():
    return os.path.join(_HERE, "libgdr2.so")


class Gdr2Problem(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("H", ctypes.c_int32),
                ("Dk", ctypes.c_int32), ("Dv", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("scale", ctypes.c_float), ("dtype", ctypes.c_int32), ("Hv", ctypes.c_int32)]


class Gdr2Stage(ctypes.Structure):
    _fields_ = [("a_log", ctypes.c_void_p), ("delta", ctypes.c_void_p), ("eps", ctypes.c_float)]


class Gdr2Error(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {gdr2_status_str(status)} ({status})")


_LIB = None


def lib():
    """The loaded libgdr2.so (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        path = lib_path()
        if not os.path.exists(path):
            raise ImportError(f"GDR-2 HIP library not built: {path} is missing "
                              "(run python -m paper_2605_22791_amd.build)")
        L = ctypes.CDLL(path)
        P = ctypes.POINTER(Gdr2Problem)
        vp = ctypes.c_void_p
        L.gdr2_chunk_workspace_bytes.argtypes = [P, ctypes.c_int, ctypes.POINTER(ctypes.c_size_t)]
        L.gdr2_chunk_workspace_bytes.restype = ctypes.c_int
        L.gdr2_chunk_fwd.argtypes = [P] + [vp] * 10 + [ctypes.c_size_t, vp]
        L.gdr2_chunk_fwd.restype = ctypes.c_int
        L.gdr2_chunk_bwd.argtypes = [P] + [vp] * 17 + [ctypes.c_size_t, vp]
        L.gdr2_chunk_bwd.restype = ctypes.c_int
        L.gdr2_chunk_fwd_noalloc.argtypes = [P] + [vp] * 10
        L.gdr2_chunk_fwd_noalloc.restype = ctypes.c_int
        L.gdr2_chunk_fwd_save.argtypes = L.gdr2_chunk_fwd.argtypes
        L.gdr2_chunk_fwd_save.restype = ctypes.c_int
        L.gdr2_chunk_bwd_saved.argtypes = L.gdr2_chunk_bwd.argtypes
        L.gdr2_chunk_bwd_saved.restype = ctypes.c_int
        L.gdr2_recurrent_step.argtypes = [P] + [vp] * 8 + [vp]
        L.gdr2_recurrent_step.restype = ctypes.c_int
        i32 = ctypes.c_int32
        L.gdr2_varlen_workspace_bytes.argtypes = [P, i32, ctypes.c_int, ctypes.POINTER(ctypes.c_size_t)]
        L.gdr2_varlen_workspace_bytes.restype = ctypes.c_int
        L.gdr2_chunk_fwd_varlen.argtypes = [P, vp, i32] + [vp] * 10 + [ctypes.c_size_t, ctypes.c_int, vp]
        L.gdr2_chunk_fwd_varlen.restype = ctypes.c_int
        L.gdr2_chunk_bwd_varlen.argtypes = [P, vp, i32] + [vp] * 17 + [ctypes.c_size_t, ctypes.c_int, vp]
        L.gdr2_chunk_bwd_varlen.restype = ctypes.c_int
        L.gdr2_recurrent_varlen.argtypes = [P, vp, i32] + [vp] * 8 + [vp]
        L.gdr2_recurrent_varlen.restype = ctypes.c_int
        S = ctypes.POINTER(Gdr2Stage)
        L.gdr2_fused_workspace_bytes.restype = ctypes.c_int
        L.gdr2_fused_workspace_bytes.argtypes = [P, i32, ctypes.c_int, ctypes.POINTER(ctypes.c_size_t)]
        L.gdr2_fused_fwd.restype = ctypes.c_int
        L.gdr2_fused_fwd.argtypes = [P, S, vp, i32] + [vp] * 10 + [ctypes.c_size_t, ctypes.c_int, vp]
        L.gdr2_fused_bwd.restype = ctypes.c_int
        L.gdr2_fused_bwd.argtypes = [P, S, vp, i32] + [vp] * 19 + [ctypes.c_size_t, ctypes.c_int, vp]
        L.gdr2_fused_recurrent.restype = ctypes.c_int
        L.gdr2_fused_recurrent.argtypes = [P, S, vp, i32] + [vp] * 8 + [vp]
        L.gdr2_profile_enable.argtypes = [ctypes.c_int]
        L.gdr2_profile_enable.restype = ctypes.c_int
        L.gdr2_profile_collect.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_longlong),
                                           ctypes.c_int]
        L.gdr2_profile_collect.restype = ctypes.c_int
        L.gdr2_status_str.argtypes = [ctypes.c_int]
        L.gdr2_status_str.restype = ctypes.c_char_p
        _LIB = L
    return _LIB


def gdr2_status_str(status):
    return lib().gdr2_status_str(int(status)).decode()


def _check(status, where):
    if status != GDR2_OK:
        raise Gdr2Error(status, where)


# --------------------------------------------------------------------------- torch helpers
def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return GDR2_BF16
    if t.dtype == torch.float32:
        return GDR2_FP32
    raise TypeError(f"unsupported dtype {t.dtype} (bfloat16 or float32)")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(_torch().cuda.current_stream().cuda_stream)


def _problem(q, v, scale, chunk=CHUNK):
    B, T, H, Dk = q.shape
    Hv, Dv = v.shape[2], v.shape[-1]
    if scale is None:
        scale = Dk ** -0.5
    return Gdr2Problem(B, T, H, Dk, Dv, chunk, float(scale), _dtype_code(q), Hv)


def _require(name, t, shape, dtype, device=None):
    """t is None or a contiguous device tensor of this shape and dtype (on
    `device` when given: every buffer of a call lives on its inputs' GPU)."""
    if t is None:
        return
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype or not t.is_contiguous() or not t.is_cuda:
        raise ValueError(f"{name}: expected contiguous {dtype} device tensor of shape {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)} (contiguous={t.is_contiguous()}, cuda={t.is_cuda})")
    if device is not None and t.device != device:
        raise ValueError(f"{name}: on {t.device}, the call's inputs are on {device}")


def _require_ws(ws, need, device):
    """The workspace: a contiguous uint8 tensor on the inputs' GPU (its numel is
    the byte count handed to the library, which rejects one below `need`)."""
    torch = _torch()
    _require("ws", ws, (ws.numel(),), torch.uint8, device)
    if ws.numel() < need:
        raise ValueError(f"ws: {ws.numel()} bytes, the call needs {need}")


def _require_grads(g, shapes, device):
    """Caller-supplied gradient buffers: each of the shape and dtype the
    library writes (shapes: name -> (shape, dtype))."""
    for n, (shape, dtype) in shapes.items():
        _require(n, g.get(n), shape, dtype, device)


def _on(t):
    """Context that makes t's GPU current for the library call (its stream is
    that device's current stream)."""
    return _torch().cuda.device(t.device)


def _validate(q, k, v, log_alpha, b, w):
    """Shapes: q, k, b, log_alpha (B, T, H, Dk); v, w (B, T, Hv, Dv) with Hv a
    multiple of H (grouped value heads when Hv > H).  Returns B, T, Hv, Dk, Dv:
    outputs and states live on the value heads."""
    torch = _torch()
    B, T, H, Dk = q.shape
    Hv, Dv = v.shape[2], v.shape[-1]
    if Hv % H != 0:
        raise ValueError(f"value heads ({Hv}) must be a multiple of key heads ({H})")
    dev = q.device
    for n, t in (("q", q), ("k", k), ("b", b)):
        _require(n, t, (B, T, H, Dk), q.dtype, dev)
    for n, t in (("v", v), ("w", w)):
        _require(n, t, (B, T, Hv, Dv), q.dtype, dev)
    _require("log_alpha", log_alpha, (B, T, H, Dk), torch.float32, dev)
    return B, T, Hv, Dk, Dv


# --------------------------------------------------------------------------- public calls
def gdr2_chunk_workspace_bytes(problem, for_backward):
    """Bytes of workspace for a Gdr2Problem (for_backward: 0 forward, 1 backward)."""
    n = ctypes.c_size_t(0)
    _check(lib().gdr2_chunk_workspace_bytes(ctypes.byref(problem), int(for_backward), ctypes.byref(n)),
           "gdr2_chunk_workspace_bytes")
    return n.value


def gdr2_chunk_fwd(q, k, v, log_alpha, b, w, S0=None, *, scale=None, o=None, S_T=None,
                   want_state=True, ws=None, save=False):
    """Chunkwise GDR-2 forward.  Returns (o, S_T) (S_T None unless wanted).

    save=True calls gdr2_chunk_fwd_save: ws (backward-sized, required) then
    holds the intermediates that gdr2_chunk_bwd(..., saved=True) reads."""
    torch = _torch()
    B, T, H, Dk, Dv = _validate(q, k, v, log_alpha, b, w)
    _require("S0", S0, (B, H, Dk, Dv), torch.float32, q.device)
    prob = _problem(q, v, scale)
    if o is None:
        o = torch.empty((B, T, H, Dv), dtype=q.dtype, device=q.device)
    _require("o", o, (B, T, H, Dv), q.dtype, q.device)
    if S_T is None and want_state:
        S_T = torch.empty((B, H, Dk, Dv), dtype=torch.float32, device=q.device)
    _require("S_T", S_T, (B, H, Dk, Dv), torch.float32, q.device)
    need = gdr2_chunk_workspace_bytes(prob, 1 if save else 0)
    if ws is None:
        if save:
            raise ValueError("save=True needs the workspace that the backward will read")
        ws = torch.empty(need, dtype=torch.uint8, device=q.device)
    _require_ws(ws, need, q.device)
    fn = lib().gdr2_chunk_fwd_save if save else lib().gdr2_chunk_fwd
    with _on(q):
        st = fn(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(b),
                                  _ptr(w), _ptr(S0), _ptr(o), _ptr(S_T), _ptr(ws), ws.numel(), _stream())
    _check(st, "gdr2_chunk_fwd_save" if save else "gdr2_chunk_fwd")
    return o, S_T


def gdr2_chunk_fwd_noalloc(q, k, v, log_alpha, b, w, S0=None, *, scale=None, o=None, S_T=None,
                           want_state=True):
    """Chunkwise GDR-2 forward without a workspace argument (gdr2_chunk_fwd_noalloc:
    the library's fixed per-GPU array, NOALLOC_SCRATCH_BYTES).  Returns (o, S_T).
    Pass o (and S_T) to keep the call free of allocations; the C call itself
    allocates nothing."""
    torch = _torch()
    B, T, H, Dk, Dv = _validate(q, k, v, log_alpha, b, w)
    _require("S0", S0, (B, H, Dk, Dv), torch.float32, q.device)
    prob = _problem(q, v, scale)
    if o is None:
        o = torch.empty((B, T, H, Dv), dtype=q.dtype, device=q.device)
    _require("o", o, (B, T, H, Dv), q.dtype, q.device)
    if S_T is None and want_state:
        S_T = torch.empty((B, H, Dk, Dv), dtype=torch.float32, device=q.device)
    _require("S_T", S_T, (B, H, Dk, Dv), torch.float32, q.device)
    with _on(q):
        st = lib().gdr2_chunk_fwd_noalloc(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha),
                                          _ptr(b), _ptr(w), _ptr(S0), _ptr(o), _ptr(S_T), _stream())
    _check(st, "gdr2_chunk_fwd_noalloc")
    return o, S_T


def gdr2_chunk_bwd(q, k, v, log_alpha, b, w, S0, dout, dS_T=None, *, scale=None, grads=None,
                   want_dS0=True, ws=None, saved=False):
    """Gate-aware chunkwise backward.  Returns dict dq, dk, dv, dlog_alpha, db, dw, dS0.

    saved=True calls gdr2_chunk_bwd_saved on the ws a save=True forward filled."""
    torch = _torch()
    B, T, H, Dk, Dv = _validate(q, k, v, log_alpha, b, w)
    _require("S0", S0, (B, H, Dk, Dv), torch.float32, q.device)
    _require("dout", dout, (B, T, H, Dv), q.dtype, q.device)
    _require("dS_T", dS_T, (B, H, Dk, Dv), torch.float32, q.device)
    prob = _problem(q, v, scale)
    g = dict(grads or {})
    dev = q.device
    g.setdefault("dq", torch.empty_like(q))
    g.setdefault("dk", torch.empty_like(k))
    g.setdefault("dv", torch.empty_like(v))
    g.setdefault("dlog_alpha", torch.empty_like(log_alpha))
    g.setdefault("db", torch.empty_like(b))
    g.setdefault("dw", torch.empty_like(w))
    if want_dS0:
        g.setdefault("dS0", torch.empty((B, H, Dk, Dv), dtype=torch.float32, device=dev))
    else:
        g.setdefault("dS0", None)
    need = gdr2_chunk_workspace_bytes(prob, 1)
    if ws is None:
        if saved:
            raise ValueError("saved=True needs the workspace of the saving forward")
        ws = torch.empty(need, dtype=torch.uint8, device=dev)
    _require_ws(ws, need, dev)
    _require_grads(g, {"dq": (q.shape, q.dtype), "dk": (k.shape, q.dtype), "dv": (v.shape, q.dtype),
                       "dlog_alpha": (log_alpha.shape, torch.float32), "db": (b.shape, q.dtype),
                       "dw": (w.shape, q.dtype), "dS0": ((B, H, Dk, Dv), torch.float32)}, dev)
    fn = lib().gdr2_chunk_bwd_saved if saved else lib().gdr2_chunk_bwd
    with _on(q):
        st = fn(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha), _ptr(b),
                                  _ptr(w), _ptr(S0), _ptr(dout), _ptr(dS_T), _ptr(g["dq"]), _ptr(g["dk"]),
                                  _ptr(g["dv"]), _ptr(g["dlog_alpha"]), _ptr(g["db"]), _ptr(g["dw"]),
                                  _ptr(g["dS0"]), _ptr(ws), ws.numel(), _stream())
    _check(st, "gdr2_chunk_bwd_saved" if saved else "gdr2_chunk_bwd")
    return g


def gdr2_recurrent_step(q, k, v, log_alpha, b, w, S, *, scale=None, o=None):
    """Token-by-token forward over q.shape[1] tokens; S (fp32) updated in place.  Returns o."""
    torch = _torch()
    B, T, H, Dk, Dv = _validate(q, k, v, log_alpha, b, w)
    _require("S", S, (B, H, Dk, Dv), torch.float32, q.device)
    prob = _problem(q, v, scale)
    if o is None:
        o = torch.empty((B, T, H, Dv), dtype=q.dtype, device=q.device)
    _require("o", o, (B, T, H, Dv), q.dtype, q.device)
    with _on(q):
        st = lib().gdr2_recurrent_step(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v), _ptr(log_alpha),
                                       _ptr(b), _ptr(w), _ptr(S), _ptr(o), _stream())
    _check(st, "gdr2_recurrent_step")
    return o


# --------------------------------------------------------------------------- packed sequences
def _cu(cu_seqlens, T, device=None):
    torch = _torch()
    if cu_seqlens.dim() != 1 or cu_seqlens.numel() < 2:
        raise ValueError("cu_seqlens: expected a 1-D tensor of n_seqs + 1 offsets")
    _require("cu_seqlens", cu_seqlens, (cu_seqlens.numel(),), torch.int32, device)
    return cu_seqlens.numel() - 1


def gdr2_varlen_workspace_bytes(problem, n_seqs, for_backward):
    """Bytes of workspace of a packed call of n_seqs sequences."""
    n = ctypes.c_size_t(0)
    _check(lib().gdr2_varlen_workspace_bytes(ctypes.byref(problem), int(n_seqs), int(for_backward),
                                             ctypes.byref(n)), "gdr2_varlen_workspace_bytes")
    return n.value


def gdr2_chunk_fwd_varlen(q, k, v, log_alpha, b, w, cu_seqlens, S0=None, *, scale=None, o=None, S_T=None,
                          want_state=True, ws=None, save=False):
    """Chunk forward of a packed batch: q.. of shape (1, T, H, D), sequence s owns
    tokens cu_seqlens[s] .. cu_seqlens[s+1) (int32 device tensor).  States are
    (n_seqs, H, Dk, Dv).  Returns (o, S_T); save=True as in gdr2_chunk_fwd."""
    torch = _torch()
    B, T, H, Dk, Dv = _validate(q, k, v, log_alpha, b, w)
    N = _cu(cu_seqlens, T, q.device)
    _require("S0", S0, (N, H, Dk, Dv), torch.float32, q.device)
    prob = _problem(q, v, scale)
    if o is None:
        o = torch.empty((B, T, H, Dv), dtype=q.dtype, device=q.device)
    _require("o", o, (B, T, H, Dv), q.dtype, q.device)
    if S_T is None and want_state:
        S_T = torch.empty((N, H, Dk, Dv), dtype=torch.float32, device=q.device)
    _require("S_T", S_T, (N, H, Dk, Dv), torch.float32, q.device)
    need = gdr2_varlen_workspace_bytes(prob, N, 1 if save else 0)
    if ws is None:
        if save:
            raise ValueError("save=True needs the workspace that the backward will read")
        ws = torch.empty(need, dtype=torch.uint8, device=q.device)
    _require_ws(ws, need, q.device)
    with _on(q):
        st = lib().gdr2_chunk_fwd_varlen(ctypes.byref(prob), _ptr(cu_seqlens), N, _ptr(q), _ptr(k), _ptr(v),
                                         _ptr(log_alpha), _ptr(b), _ptr(w), _ptr(S0), _ptr(o), _ptr(S_T), _ptr(ws),
                                         ws.numel(), 1 if save else 0, _stream())
    _check(st, "gdr2_chunk_fwd_varlen")
    return o, S_T


def gdr2_chunk_bwd_varlen(q, k, v, log_alpha, b, w, cu_seqlens, S0, dout, dS_T=None, *, scale=None,
                          grads=None, want_dS0=True, ws=None, saved=False):
    """Backward of a packed batch; returns dict dq, dk, dv, dlog_alpha, db, dw, dS0."""
    torch = _torch()
    B, T, H, Dk, Dv = _validate(q, k, v, log_alpha, b, w)
    N = _cu(cu_seqlens, T, q.device)
    _require("S0", S0, (N, H, Dk, Dv), torch.float32, q.device)
    _require("dout", dout, (B, T, H, Dv), q.dtype, q.device)
    _require("dS_T", dS_T, (N, H, Dk, Dv), torch.float32, q.device)
    prob = _problem(q, v, scale)
    g = dict(grads or {})
    for n, like in (("dq", q), ("dk", k), ("dv", v), ("dlog_alpha", log_alpha), ("db", b), ("dw", w)):
        g.setdefault(n, torch.empty_like(like))
    if want_dS0:
        g.setdefault("dS0", torch.empty((N, H, Dk, Dv), dtype=torch.float32, device=q.device))
    else:
        g.setdefault("dS0", None)
    need = gdr2_varlen_workspace_bytes(prob, N, 1)
    if ws is None:
        if saved:
            raise ValueError("saved=True needs the workspace of the saving forward")
        ws = torch.empty(need, dtype=torch.uint8, device=q.device)
    _require_ws(ws, need, q.device)
    _require_grads(g, {"dq": (q.shape, q.dtype), "dk": (k.shape, q.dtype), "dv": (v.shape, q.dtype),
                       "dlog_alpha": (log_alpha.shape, torch.float32), "db": (b.shape, q.dtype),
                       "dw": (w.shape, q.dtype), "dS0": ((N, H, Dk, Dv), torch.float32)}, q.device)
    with _on(q):
        st = lib().gdr2_chunk_bwd_varlen(ctypes.byref(prob), _ptr(cu_seqlens), N, _ptr(q), _ptr(k), _ptr(v),
                                         _ptr(log_alpha), _ptr(b), _ptr(w), _ptr(S0), _ptr(dout), _ptr(dS_T),
                                         _ptr(g["dq"]), _ptr(g["dk"]), _ptr(g["dv"]), _ptr(g["dlog_alpha"]),
                                         _ptr(g["db"]), _ptr(g["dw"]), _ptr(g["dS0"]), _ptr(ws), ws.numel(),
                                         1 if saved else 0, _stream())
    _check(st, "gdr2_chunk_bwd_varlen")
    return g


def gdr2_recurrent_varlen(q, k, v, log_alpha, b, w, cu_seqlens, S, *, scale=None, o=None):
    """Token-by-token forward of a packed batch; S (n_seqs, H, Dk, Dv) updated in place.  Returns o."""
    torch = _torch()
    B, T, H, Dk, Dv = _validate(q, k, v, log_alpha, b, w)
    N = _cu(cu_seqlens, T, q.device)
    _require("S", S, (N, H, Dk, Dv), torch.float32, q.device)
    prob = _problem(q, v, scale)
    if o is None:
        o = torch.empty((B, T, H, Dv), dtype=q.dtype, device=q.device)
    _require("o", o, (B, T, H, Dv), q.dtype, q.device)
    with _on(q):
        st = lib().gdr2_recurrent_varlen(ctypes.byref(prob), _ptr(cu_seqlens), N, _ptr(q), _ptr(k), _ptr(v),
                                         _ptr(log_alpha), _ptr(b), _ptr(w), _ptr(S), _ptr(o), _stream())
    _check(st, "gdr2_recurrent_varlen")
    return o


def gdr2_profile_enable(on=True):
    """Enable / disable per-kernel hipEvent timing for the calling thread."""
    _check(lib().gdr2_profile_enable(1 if on else 0), "gdr2_profile_enable")


def gdr2_profile_collect():
    """Wait for timed launches; return {kernel: (total_ms, launches)} and reset."""
    n = len(KERNEL_NAMES)
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_longlong * n)()
    _check(lib().gdr2_profile_collect(ms, cnt, n), "gdr2_profile_collect")
    return {KERNEL_NAMES[i]: (ms[i], cnt[i]) for i in range(n)}


# --------------------------------------------------------------------------- fused input stage
def _stage(a_log, delta, H, Dk, eps, device):
    torch = _torch()
    _require("a_log", a_log, (H,), torch.float32, device)
    _require("delta", delta, (H, Dk), torch.float32, device)
    return Gdr2Stage(a_log.data_ptr(), delta.data_ptr(), float(eps))


def gdr2_fused_workspace_bytes(problem, n_seqs, for_backward):
    """Bytes of workspace of a fused chunk call (n_seqs = 0: fixed length)."""
    n = ctypes.c_size_t(0)
    _check(lib().gdr2_fused_workspace_bytes(ctypes.byref(problem), int(n_seqs), int(for_backward),
                                            ctypes.byref(n)), "gdr2_fused_workspace_bytes")
    return n.value


def _fused_shapes(q, k, v, f, b, w, cu_seqlens):
    B, T, H, Dk, Dv = _validate(q, k, v, f, b, w)
    N = _cu(cu_seqlens, T, q.device) if cu_seqlens is not None else 0
    return B, T, H, Dk, Dv, N


def gdr2_fused_fwd(q, k, v, f, a_log, delta, b, w, S0=None, *, cu_seqlens=None, scale=None, eps=1e-6, o=None,
                   S_T=None, want_state=True, ws=None, save=False):
    """Forward from the raw projections: q, k (not normalised), f the decay
    projection (fp32, (B, T, H, Dk)), a_log (H,), delta (H, Dk).  Returns (o, S_T)."""
    torch = _torch()
    B, T, Hv, Dk, Dv, N = _fused_shapes(q, k, v, f, b, w, cu_seqlens)
    NS = N if N > 0 else B
    stg = _stage(a_log, delta, q.shape[2], Dk, eps, q.device)
    _require("S0", S0, (NS, Hv, Dk, Dv), torch.float32, q.device)
    prob = _problem(q, v, scale)
    if o is None:
        o = torch.empty((B, T, Hv, Dv), dtype=q.dtype, device=q.device)
    _require("o", o, (B, T, Hv, Dv), q.dtype, q.device)
    if S_T is None and want_state:
        S_T = torch.empty((NS, Hv, Dk, Dv), dtype=torch.float32, device=q.device)
    _require("S_T", S_T, (NS, Hv, Dk, Dv), torch.float32, q.device)
    if ws is None:
        if save:
            raise ValueError("save=True needs the workspace that the backward will read")
        ws = torch.empty(gdr2_fused_workspace_bytes(prob, N, 0), dtype=torch.uint8, device=q.device)
    _require_ws(ws, gdr2_fused_workspace_bytes(prob, N, 1 if save else 0), q.device)
    with _on(q):
        st = lib().gdr2_fused_fwd(ctypes.byref(prob), ctypes.byref(stg), _ptr(cu_seqlens), N, _ptr(q), _ptr(k),
                                  _ptr(v), _ptr(f), _ptr(b), _ptr(w), _ptr(S0), _ptr(o), _ptr(S_T), _ptr(ws),
                                  ws.numel(), 1 if save else 0, _stream())
    _check(st, "gdr2_fused_fwd")
    return o, S_T


def gdr2_fused_bwd(q, k, v, f, a_log, delta, b, w, S0, dout, dS_T=None, *, cu_seqlens=None, scale=None,
                   eps=1e-6, grads=None, want_dS0=True, ws=None, saved=False):
    """Backward from the raw projections; returns dict dq, dk (raw q, k), dv,
    df, da, ddelta, db, dw, dS0."""
    torch = _torch()
    B, T, Hv, Dk, Dv, N = _fused_shapes(q, k, v, f, b, w, cu_seqlens)
    NS = N if N > 0 else B
    H = q.shape[2]
    stg = _stage(a_log, delta, H, Dk, eps, q.device)
    _require("S0", S0, (NS, Hv, Dk, Dv), torch.float32, q.device)
    _require("dout", dout, (B, T, Hv, Dv), q.dtype, q.device)
    _require("dS_T", dS_T, (NS, Hv, Dk, Dv), torch.float32, q.device)
    prob = _problem(q, v, scale)
    g = dict(grads or {})
    for n, like in (("dq", q), ("dk", k), ("dv", v), ("df", f), ("db", b), ("dw", w), ("da", a_log),
                    ("ddelta", delta)):
        g.setdefault(n, torch.empty_like(like))
    if want_dS0:
        g.setdefault("dS0", torch.empty((NS, Hv, Dk, Dv), dtype=torch.float32, device=q.device))
    else:
        g.setdefault("dS0", None)
    if ws is None:
        if saved:
            raise ValueError("saved=True needs the workspace of the saving forward")
        ws = torch.empty(gdr2_fused_workspace_bytes(prob, N, 1), dtype=torch.uint8, device=q.device)
    _require_ws(ws, gdr2_fused_workspace_bytes(prob, N, 1), q.device)
    _require_grads(g, {"dq": (q.shape, q.dtype), "dk": (k.shape, q.dtype), "dv": (v.shape, q.dtype),
                       "df": (f.shape, torch.float32), "db": (b.shape, q.dtype), "dw": (w.shape, q.dtype),
                       "da": (a_log.shape, torch.float32), "ddelta": (delta.shape, torch.float32),
                       "dS0": ((NS, Hv, Dk, Dv), torch.float32)}, q.device)
    with _on(q):
        st = lib().gdr2_fused_bwd(ctypes.byref(prob), ctypes.byref(stg), _ptr(cu_seqlens), N, _ptr(q), _ptr(k),
                                  _ptr(v), _ptr(f), _ptr(b), _ptr(w), _ptr(S0), _ptr(dout), _ptr(dS_T), _ptr(g["dq"]),
                                  _ptr(g["dk"]), _ptr(g["dv"]), _ptr(g["df"]), _ptr(g["da"]), _ptr(g["ddelta"]),
                                  _ptr(g["db"]), _ptr(g["dw"]), _ptr(g["dS0"]), _ptr(ws), ws.numel(),
                                  1 if saved else 0, _stream())
    _check(st, "gdr2_fused_bwd")
    return g


def gdr2_fused_recurrent(q, k, v, f, a_log, delta, b, w, S, *, cu_seqlens=None, scale=None, eps=1e-6, o=None):
    """Token-by-token forward from the raw projections; S updated in place.  Returns o."""
    torch = _torch()
    B, T, Hv, Dk, Dv, N = _fused_shapes(q, k, v, f, b, w, cu_seqlens)
    NS = N if N > 0 else B
    stg = _stage(a_log, delta, q.shape[2], Dk, eps, q.device)
    _require("S", S, (NS, Hv, Dk, Dv), torch.float32, q.device)
    prob = _problem(q, v, scale)
    if o is None:
        o = torch.empty((B, T, Hv, Dv), dtype=q.dtype, device=q.device)
    _require("o", o, (B, T, Hv, Dv), q.dtype, q.device)
    with _on(q):
        st = lib().gdr2_fused_recurrent(ctypes.byref(prob), ctypes.byref(stg), _ptr(cu_seqlens), N, _ptr(q), _ptr(k),
                                        _ptr(v), _ptr(f), _ptr(b), _ptr(w), _ptr(S), _ptr(o), _stream())
    _check(st, "gdr2_fused_recurrent")
    return o
