"""C-ABI checks that need no GPU: exports, argument validation, workspace sizes.

Every call here is rejected by validation, which the library performs before
any HIP call, so the (fake, never dereferenced) pointers are safe.
"""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2605_22791_amd as g2
from paper_2605_22791_amd.inputs import bf16_round, CONFIGS, config

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gdr2.h")

pytestmark = pytest.mark.skipif(not os.path.exists(g2.lib_path()),
                                reason="libgdr2.so not built (python -m paper_2605_22791_amd.build)")

FAKE = 0x10000  # 16-byte aligned, never dereferenced


def _declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:gdr2_status|const char\*)\s+(gdr2_\w+)\s*\(", text, re.M)))


def test_header_declares_the_entry_points():
    assert _declared_symbols() == sorted(["gdr2_chunk_workspace_bytes", "gdr2_chunk_fwd",
                                          "gdr2_chunk_bwd", "gdr2_chunk_fwd_save",
                                          "gdr2_chunk_bwd_saved", "gdr2_recurrent_step",
                                          "gdr2_varlen_workspace_bytes", "gdr2_chunk_fwd_varlen",
                                          "gdr2_chunk_bwd_varlen", "gdr2_recurrent_varlen",
                                          "gdr2_status_str", "gdr2_profile_enable",
                                          "gdr2_profile_collect", "gdr2_fused_workspace_bytes",
                                          "gdr2_fused_fwd", "gdr2_fused_bwd", "gdr2_fused_recurrent",
                                          "gdr2_chunk_fwd_noalloc"])


def test_library_exports_every_declared_symbol():
    L = g2.lib()
    for name in _declared_symbols():
        assert hasattr(L, name), name


def test_status_strings():
    for code in range(5):
        s = g2.gdr2_status_str(code)
        assert s.startswith("GDR2_")
    assert g2.gdr2_status_str(99) == "GDR2_UNKNOWN"


def test_profile_collect_without_launches():
    L = g2.lib()
    k = len(g2.KERNEL_NAMES)
    ms = (ctypes.c_double * k)()
    n = (ctypes.c_longlong * k)()
    assert L.gdr2_profile_collect(ms, n, k - 1) == g2.GDR2_EINVAL
    assert L.gdr2_profile_enable(1) == g2.GDR2_OK
    assert L.gdr2_profile_collect(ms, n, k) == g2.GDR2_OK
    assert L.gdr2_profile_enable(0) == g2.GDR2_OK
    assert list(n) == [0] * k and list(ms) == [0.0] * k


def _prob(**kw):
    d = dict(B=2, T=128, H=4, Dk=128, Dv=128, chunk=64, scale=128 ** -0.5, dtype=g2.GDR2_BF16)
    d.update(kw)
    return g2.Gdr2Problem(**d)


def _fwd(prob, q=FAKE, ws_bytes=None, S0=None, ptrs=None):
    L = g2.lib()
    p = [q, FAKE, FAKE, FAKE, FAKE, FAKE, S0, FAKE, None, FAKE]
    if ptrs:
        for i, val in ptrs.items():
            p[i] = val
    n = ws_bytes if ws_bytes is not None else (1 << 40)
    pp = ctypes.byref(prob) if prob is not None else None
    return L.gdr2_chunk_fwd(pp, *[ctypes.c_void_p(x) if x else None for x in p], n, None)


def _bwd(prob, ws_bytes=None, ptrs=None):
    L = g2.lib()
    p = [FAKE] * 6 + [None, FAKE, None] + [FAKE] * 6 + [None, FAKE]
    if ptrs:
        for i, val in ptrs.items():
            p[i] = val
    n = ws_bytes if ws_bytes is not None else (1 << 40)
    return L.gdr2_chunk_bwd(ctypes.byref(prob), *[ctypes.c_void_p(x) if x else None for x in p], n, None)


def _rec(prob, ptrs=None):
    L = g2.lib()
    p = [FAKE] * 8
    if ptrs:
        for i, val in ptrs.items():
            p[i] = val
    return L.gdr2_recurrent_step(ctypes.byref(prob), *[ctypes.c_void_p(x) if x else None for x in p], None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), g2.GDR2_EINVAL), (dict(T=-64), g2.GDR2_EINVAL), (dict(H=0), g2.GDR2_EINVAL),
    (dict(Dk=0), g2.GDR2_EINVAL), (dict(scale=float("nan")), g2.GDR2_EINVAL),
    (dict(scale=float("inf")), g2.GDR2_EINVAL), (dict(dtype=7), g2.GDR2_EINVAL),
    (dict(Dk=96), g2.GDR2_EUNSUPPORTED), (dict(Dv=256), g2.GDR2_EUNSUPPORTED),
    (dict(chunk=32), g2.GDR2_EUNSUPPORTED),
    (dict(B=1 << 20, T=1 << 16), g2.GDR2_EUNSUPPORTED),
])
def test_problem_validation(kw, code):
    assert _fwd(_prob(**kw)) == code
    assert _bwd(_prob(**kw)) == code
    n = ctypes.c_size_t(0)
    assert g2.lib().gdr2_chunk_workspace_bytes(ctypes.byref(_prob(**kw)), 0, ctypes.byref(n)) == code


def test_null_problem_and_null_out_size():
    assert _fwd(None) == g2.GDR2_EINVAL
    assert g2.lib().gdr2_chunk_workspace_bytes(ctypes.byref(_prob()), 0, None) == g2.GDR2_EINVAL


@pytest.mark.parametrize("idx", range(10))
def test_forward_pointer_checks(idx):
    # required pointers: q k v log_alpha b w (0-5), o (7), ws (9); S0 (6) and S_T (8) optional
    if idx in (6, 8):
        assert _fwd(_prob(), ptrs={idx: FAKE + 4}) == g2.GDR2_EINVAL   # misaligned optional
        return
    assert _fwd(_prob(), ptrs={idx: None}) == g2.GDR2_EINVAL
    assert _fwd(_prob(), ptrs={idx: FAKE + 8}) == g2.GDR2_EINVAL


def test_backward_pointer_checks():
    required = [0, 1, 2, 3, 4, 5, 7, 9, 10, 11, 12, 13, 14, 16]
    for idx in required:
        assert _bwd(_prob(), ptrs={idx: None}) == g2.GDR2_EINVAL, idx
    for idx in (6, 8, 15):
        assert _bwd(_prob(), ptrs={idx: FAKE + 4}) == g2.GDR2_EINVAL, idx


def test_recurrent_validation():
    assert _rec(_prob(B=0)) == g2.GDR2_EINVAL
    assert _rec(_prob(Dk=32)) == g2.GDR2_EUNSUPPORTED
    for idx in range(8):
        assert _rec(_prob(T=1), ptrs={idx: None}) == g2.GDR2_EINVAL


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_workspace_size_and_check(dtype):
    p = _prob(B=2, T=256, H=4, Dk=128, Dv=64)
    p.dtype = g2.GDR2_FP32 if dtype == "fp32" else g2.GDR2_BF16
    fwd = g2.gdr2_chunk_workspace_bytes(p, 0)
    bwd = g2.gdr2_chunk_workspace_bytes(p, 1)
    NC = 2 * 4 * (256 // 64)
    r = lambda n: (n * 4 + 255) // 256 * 256      # fp32 tiles, 256-byte aligned regions
    rb = lambda n: (n + 255) // 256 * 256         # byte regions
    fwd32 = r(NC * 64 * 128) + r(NC * 64 * 64) + 2 * r(NC * 64 * 128) + r(NC * 64 * 64) + r(NC * 128)
    extras = 2 * r(NC * 128 * 64) + 2 * r(NC * 64 * 64) + 2 * r(NC * 64 * 64) + r(NC * 64 * 128)
    if dtype == "fp32":
        exp_fwd = fwd32
    else:
        # fragment-ordered bf16 tiles: Y, Qg (hi/lo), A_qk (hi/lo), Ktail^T (hi/lo), U (fp32), gamma_C
        exp_fwd = (rb(NC * 4 * 4 * 1024) + rb(NC * 4 * 4 * 2048) + rb(NC * 8 * 2048) + rb(NC * 8 * 2 * 2048)
                   + rb(NC * 4 * 4 * 1024) + rb(NC * 512))
    if dtype == "fp32":
        exp_bwd = exp_fwd + extras
    else:
        # chunk states and their gradients in fp16 with one fp32 scale per 16 x 32 block,
        # R in fp16 fragment blocks; dR as split bf16 16 x 16 blocks, A as fp16 16 x 16
        # blocks with one fp32 scale each
        states = rb(NC * 128 * 64 * 2) + rb(NC * (128 // 16) * (64 // 32) * 4)
        rfrag = rb(NC * 4 * (64 // 32) * 1024) + rb(NC * 4 * (64 // 32) * 4)     # R: fp16 blocks + scales
        dr = rb(NC * (64 // 16) * 4 * 1024)                                       # dR
        am = rb(NC * 16 * 512) + rb(NC * 16 * 4)                                  # A
        exp_bwd = exp_fwd + 2 * states + rfrag + dr + am
    assert fwd == exp_fwd and bwd == exp_bwd
    assert _fwd(p, ws_bytes=fwd - 1) == g2.GDR2_EWORKSPACE
    assert _bwd(p, ws_bytes=bwd - 1) == g2.GDR2_EWORKSPACE
    if bwd > fwd:
        assert _bwd(p, ws_bytes=fwd) == g2.GDR2_EWORKSPACE


def test_bf16_round_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 3.14159], dtype=np.float32)
    y = bf16_round(x)
    assert y[0] == 1.0
    assert y[1] == 1.0                  # tie -> even (mantissa 0)
    assert y[2] == 1.0 + 4 * 2 ** -8    # tie -> even (rounds up)
    assert y[3] == 1.0
    assert y[4] == -2.5
    assert abs(y[5] - 3.140625) < 1e-7
    assert np.all((y.view(np.uint32) & 0xFFFF) == 0)


def test_input_recipes():
    d0 = config(0)
    assert d0["q"].shape == (1, 256, 2, 64) and d0["dtype"] == "fp32" and d0["S0"] is None
    assert np.allclose(np.linalg.norm(d0["k"], axis=-1), 1.0, atol=1e-6)
    assert np.all(d0["log_alpha"] <= 0) and np.all((d0["b"] > 0) & (d0["b"] < 1))
    d1 = config(1, decay="scalar", T=128)
    assert np.all(d1["b"] == d1["b"][..., :1]) and np.all(d1["w"][..., :1] == d1["b"][..., :1])
    assert np.all(d1["log_alpha"] == d1["log_alpha"][..., :1])
    assert np.all((d1["q"].view(np.uint32) & 0xFFFF) == 0)
    assert set(CONFIGS) == {0, 1, 2, 3, 4}


def test_saved_training_path_validation():
    """gdr2_chunk_fwd_save needs the backward-sized workspace; both saved-path calls
    validate like their plain counterparts before any launch."""
    L = g2.lib()
    p = _prob(B=2, T=256, H=4, Dk=128, Dv=64)
    fwd = g2.gdr2_chunk_workspace_bytes(p, 0)
    bwd = g2.gdr2_chunk_workspace_bytes(p, 1)
    assert bwd > fwd
    vp = lambda xs: [ctypes.c_void_p(x) if x else None for x in xs]
    fargs = [FAKE] * 6 + [None, FAKE, None, FAKE]
    assert L.gdr2_chunk_fwd_save(ctypes.byref(p), *vp(fargs), fwd, None) == g2.GDR2_EWORKSPACE
    assert L.gdr2_chunk_fwd_save(ctypes.byref(p), *vp(fargs), bwd - 1, None) == g2.GDR2_EWORKSPACE
    bad = list(fargs)
    bad[0] = None
    assert L.gdr2_chunk_fwd_save(ctypes.byref(p), *vp(bad), bwd, None) == g2.GDR2_EINVAL
    bargs = [FAKE] * 6 + [None, FAKE, None] + [FAKE] * 6 + [None, FAKE]
    assert L.gdr2_chunk_bwd_saved(ctypes.byref(p), *vp(bargs), bwd - 1, None) == g2.GDR2_EWORKSPACE
    bad = list(bargs)
    bad[7] = None                      # dout
    assert L.gdr2_chunk_bwd_saved(ctypes.byref(p), *vp(bad), bwd, None) == g2.GDR2_EINVAL
    q = _prob(Dk=96)
    assert L.gdr2_chunk_bwd_saved(ctypes.byref(q), *vp(bargs), 1 << 40, None) == g2.GDR2_EUNSUPPORTED


def test_workspace_segment_buffers():
    """bf16 problems with few scans and long sequences get the segment maps of
    the sequence-parallel scans appended to the workspace; others do not."""
    from tests.gpu_common import ws_layout_bf16, seg_buffer_bytes, scan_segments
    assert scan_segments(1, 65536, 16, 128) == (8, 128)
    assert scan_segments(8, 4096, 16, 128) == (1, 64)
    assert scan_segments(1, 640, 2, 128) == (1, 10)
    assert scan_segments(1, 3200, 2, 64) == (4, 13)
    for (B, T, H, Dk, Dv) in [(1, 3200, 2, 128, 64), (1, 4096, 4, 64, 128), (2, 1024, 4, 128, 128),
                              (8, 4096, 16, 128, 128), (1, 640, 2, 64, 64)]:
        p = _prob(B=B, T=T, H=H, Dk=Dk, Dv=Dv)
        p.dtype = g2.GDR2_BF16
        extra = seg_buffer_bytes(B, T, H, Dk, Dv)
        for bwd in (0, 1):
            _, base, _ = ws_layout_bf16(B, T, H, Dk, Dv, bwd=bool(bwd))
            assert g2.gdr2_chunk_workspace_bytes(p, bwd) == base + extra, (B, T, H, Dk, Dv, bwd)
        p.dtype = g2.GDR2_FP32
        assert seg_buffer_bytes(B, T, H, Dk, Dv, "fp32") == 0


def test_partial_last_chunk_workspace():
    """T need not be a multiple of 64: a sequence of T tokens takes ceil(T/64)
    chunks (the last one partial), so the workspace equals that of the next multiple."""
    for dtype in (g2.GDR2_BF16, g2.GDR2_FP32):
        for bwd in (0, 1):
            a = _prob(B=2, T=100, dtype=dtype)
            b = _prob(B=2, T=128, dtype=dtype)
            assert g2.gdr2_chunk_workspace_bytes(a, bwd) == g2.gdr2_chunk_workspace_bytes(b, bwd)
            assert g2.gdr2_chunk_workspace_bytes(_prob(T=65, dtype=dtype), bwd) == \
                g2.gdr2_chunk_workspace_bytes(_prob(T=128, dtype=dtype), bwd)


def _vfwd(prob, cu=FAKE, n=3, ws_bytes=1 << 40, save=0):
    L = g2.lib()
    p = [FAKE] * 6 + [None, FAKE, None, FAKE]
    return L.gdr2_chunk_fwd_varlen(ctypes.byref(prob), ctypes.c_void_p(cu) if cu else None, n,
                                   *[ctypes.c_void_p(x) if x else None for x in p], ws_bytes, save, None)


def _vbwd(prob, cu=FAKE, n=3, ws_bytes=1 << 40, saved=0):
    L = g2.lib()
    p = [FAKE] * 6 + [None, FAKE, None] + [FAKE] * 6 + [None, FAKE]
    return L.gdr2_chunk_bwd_varlen(ctypes.byref(prob), ctypes.c_void_p(cu) if cu else None, n,
                                   *[ctypes.c_void_p(x) if x else None for x in p], ws_bytes, saved, None)


def test_varlen_validation():
    """Packed calls: B must be 1, n_seqs >= 1 (at most 2^24), cu_seqlens non-null and
    4-byte aligned, and the workspace large enough -- all checked before any launch."""
    L = g2.lib()
    p1 = _prob(B=1, T=1000)
    n = ctypes.c_size_t(0)
    assert L.gdr2_varlen_workspace_bytes(ctypes.byref(p1), 0, 0, ctypes.byref(n)) == g2.GDR2_EINVAL
    assert L.gdr2_varlen_workspace_bytes(ctypes.byref(_prob(B=2)), 3, 0, ctypes.byref(n)) == g2.GDR2_EINVAL
    assert L.gdr2_varlen_workspace_bytes(ctypes.byref(p1), (1 << 24) + 1, 0, ctypes.byref(n)) == \
        g2.GDR2_EUNSUPPORTED
    assert L.gdr2_varlen_workspace_bytes(ctypes.byref(p1), 3, 0, None) == g2.GDR2_EINVAL
    for call in (_vfwd, _vbwd):
        assert call(_prob(B=2, T=1000)) == g2.GDR2_EINVAL
        assert call(p1, cu=None) == g2.GDR2_EINVAL
        assert call(p1, cu=FAKE + 2) == g2.GDR2_EINVAL
        assert call(p1, n=0) == g2.GDR2_EINVAL
        assert call(_prob(B=1, T=1000, Dk=96)) == g2.GDR2_EUNSUPPORTED
    fwd = g2.gdr2_varlen_workspace_bytes(p1, 3, 0)
    bwd = g2.gdr2_varlen_workspace_bytes(p1, 3, 1)
    assert _vfwd(p1, ws_bytes=fwd - 1) == g2.GDR2_EWORKSPACE
    assert _vfwd(p1, ws_bytes=fwd, save=1) == g2.GDR2_EWORKSPACE
    assert _vbwd(p1, ws_bytes=bwd - 1) == g2.GDR2_EWORKSPACE
    vp = lambda xs: [ctypes.c_void_p(x) if x else None for x in xs]
    assert L.gdr2_recurrent_varlen(ctypes.byref(p1), None, 3, *vp([FAKE] * 8), None) == g2.GDR2_EINVAL
    assert L.gdr2_recurrent_varlen(ctypes.byref(p1), ctypes.c_void_p(FAKE), 0, *vp([FAKE] * 8), None) == \
        g2.GDR2_EINVAL


def test_varlen_workspace_size():
    """A packed call of N sequences and T tokens reserves floor(T/64) + N chunk
    slots per head (an upper bound of sum ceil(L_s/64)) plus the chunk table."""
    from tests.gpu_common import ws_layout_bf16
    for (T, N, H, Dk, Dv) in [(1000, 3, 4, 128, 64), (64, 1, 2, 64, 64), (4096, 37, 16, 128, 128)]:
        p = _prob(B=1, T=T, H=H, Dk=Dk, Dv=Dv)
        for bwd in (0, 1):
            _, total, NC = ws_layout_bf16(1, T, H, Dk, Dv, bwd=bool(bwd), nseq=N)
            assert NC == H * (T // 64 + N)
            assert g2.gdr2_varlen_workspace_bytes(p, N, bwd) == total, (T, N, bwd)


def test_grouped_value_heads_validation_and_workspace():
    """Hv must be a multiple of H (0 means Hv = H).  A grouped problem keeps the
    key-side tiles once per key head and U (and the backward's per-value-head
    regions) per value head; its backward adds four fp32 (B, T, H, Dk) regions in
    which the key-side gradients of a group's value heads add up."""
    from tests.gpu_common import ws_layout_bf16, seg_buffer_bytes
    assert _fwd(_prob(H=4, Hv=6)) == g2.GDR2_EINVAL
    assert _bwd(_prob(H=4, Hv=-4)) == g2.GDR2_EINVAL
    n = ctypes.c_size_t(0)
    assert g2.lib().gdr2_chunk_workspace_bytes(ctypes.byref(_prob(H=4, Hv=10)), 1, ctypes.byref(n)) == \
        g2.GDR2_EINVAL
    r = lambda x: (x * 4 + 255) // 256 * 256
    for (B, T, H, Hv, Dk, Dv) in [(2, 256, 4, 8, 128, 64), (1, 100, 2, 8, 64, 128), (2, 128, 4, 4, 128, 128)]:
        p = _prob(B=B, T=T, H=H, Hv=Hv, Dk=Dk, Dv=Dv)
        G = Hv // H
        _, fwd, _ = ws_layout_bf16(B, T, Hv, Dk, Dv, bwd=False, G=G)
        assert g2.gdr2_chunk_workspace_bytes(p, 0) == fwd + seg_buffer_bytes(B, T, Hv, Dk, Dv)
        _, base, _ = ws_layout_bf16(B, T, Hv, Dk, Dv, bwd=True, G=G)
        part = 4 * r(B * T * H * Dk) if Hv > H else 0  # fp32 group sums on the key-head axis
        assert g2.gdr2_chunk_workspace_bytes(p, 1) == base + part + seg_buffer_bytes(B, T, Hv, Dk, Dv)


# --------------------------------------------------------------------------- fused input stage
def _stg(a=FAKE, d=FAKE, eps=1e-6):
    return g2.Gdr2Stage(a, d, eps)


def _ffwd(prob, stage, cu=None, n=0, ws_bytes=1 << 40, save=0):
    L = g2.lib()
    p = [FAKE] * 6 + [None, FAKE, None, FAKE]
    return L.gdr2_fused_fwd(ctypes.byref(prob), ctypes.byref(stage) if stage is not None else None,
                            ctypes.c_void_p(cu) if cu else None, n,
                            *[ctypes.c_void_p(x) if x else None for x in p], ws_bytes, save, None)


def _fbwd(prob, stage, da=FAKE, ddelta=FAKE, ws_bytes=1 << 40, saved=0):
    L = g2.lib()
    p = [FAKE] * 6 + [None, FAKE, None] + [FAKE] * 4 + [da, ddelta] + [FAKE, FAKE, None, FAKE]
    return L.gdr2_fused_bwd(ctypes.byref(prob), ctypes.byref(stage) if stage is not None else None, None, 0,
                            *[ctypes.c_void_p(x) if x else None for x in p], ws_bytes, saved, None)


def test_fused_stage_validation():
    """The stage needs a_log (4-byte aligned), delta (16-byte aligned) and a finite
    eps >= 0; the backward needs da and an aligned ddelta -- all rejected before
    any launch."""
    L = g2.lib()
    p = _prob()
    for call in (_ffwd, _fbwd):
        assert call(p, None) == g2.GDR2_EINVAL
        assert call(p, _stg(a=0)) == g2.GDR2_EINVAL
        assert call(p, _stg(d=0)) == g2.GDR2_EINVAL
        assert call(p, _stg(a=FAKE + 2)) == g2.GDR2_EINVAL
        assert call(p, _stg(d=FAKE + 4)) == g2.GDR2_EINVAL
        assert call(p, _stg(eps=-1e-6)) == g2.GDR2_EINVAL
        assert call(p, _stg(eps=float("nan"))) == g2.GDR2_EINVAL
        assert call(_prob(Dk=96), _stg()) == g2.GDR2_EUNSUPPORTED
    assert _fbwd(p, _stg(), da=0) == g2.GDR2_EINVAL
    assert _fbwd(p, _stg(), ddelta=FAKE + 4) == g2.GDR2_EINVAL
    n = ctypes.c_size_t(0)
    assert L.gdr2_fused_workspace_bytes(ctypes.byref(p), -1, 0, ctypes.byref(n)) == g2.GDR2_EINVAL
    fwd = g2.gdr2_fused_workspace_bytes(p, 0, 0)
    bwd = g2.gdr2_fused_workspace_bytes(p, 0, 1)
    assert _ffwd(p, _stg(), ws_bytes=fwd - 1) == g2.GDR2_EWORKSPACE
    assert _ffwd(p, _stg(), ws_bytes=fwd, save=1) == g2.GDR2_EWORKSPACE
    assert _fbwd(p, _stg(), ws_bytes=bwd - 1) == g2.GDR2_EWORKSPACE
    # packed: B must be 1, cu_seqlens needed when n_seqs > 0
    assert _ffwd(_prob(B=2), _stg(), cu=FAKE, n=3) == g2.GDR2_EINVAL
    assert _ffwd(_prob(B=1), _stg(), cu=None, n=3) == g2.GDR2_EINVAL
    vp = lambda xs: [ctypes.c_void_p(x) if x else None for x in xs]
    st = _stg(d=FAKE + 4)
    assert L.gdr2_fused_recurrent(ctypes.byref(p), ctypes.byref(st), None, 0, *vp([FAKE] * 8), None) == \
        g2.GDR2_EINVAL
    assert L.gdr2_fused_recurrent(ctypes.byref(p), None, None, 0, *vp([FAKE] * 8), None) == g2.GDR2_EINVAL


def test_fused_workspace_size():
    """The fused forward needs what the plain one needs; a saving forward and the
    backward add the inverse norms of q and k ((B T, H) fp32 each), the per-
    workgroup decay-parameter partials (slots x Hv x 4 waves x (Dk + 1)), the
    64-range sums (64 x H x (Dk + 1)) and, for Hv = H, fp32 gradients of the
    normalised q and k ((B T, Hv, Dk) each)."""
    r = lambda x: (x * 4 + 255) // 256 * 256
    for (B, T, H, Hv, Dk, Dv, N) in [(2, 256, 4, 4, 128, 64, 0), (1, 100, 2, 8, 64, 128, 0),
                                     (1, 1000, 4, 4, 128, 128, 3)]:
        p = _prob(B=B, T=T, H=H, Hv=Hv, Dk=Dk, Dv=Dv)
        plain = (lambda bwd: g2.gdr2_varlen_workspace_bytes(p, N, bwd)) if N else \
            (lambda bwd: g2.gdr2_chunk_workspace_bytes(p, bwd))
        assert g2.gdr2_fused_workspace_bytes(p, N, 0) == plain(0)
        slots = T // 64 + N if N else B * (-(-T // 64))
        extra = 2 * r(B * T * H) + r(slots * Hv * 4 * Dk) + r(slots * Hv * 4) + r(64 * H * (Dk + 1))
        if Hv == H:   # fp32 dq, dk of the normalised tensors (grouped calls have them already)
            extra += 2 * r(B * T * Hv * Dk)
        assert g2.gdr2_fused_workspace_bytes(p, N, 1) == plain(1) + extra, (B, T, H, Hv, N)


def test_fused_workspace_size_fp32():
    """fp32 problems run the stage as passes of their own: the workspace is the
    fp32 operator's, then the normalised q, k and g ((B T, H, Dk) fp32 each) and
    the inverse norms; the backward adds the gradients of those three, the
    per-row partials of da and the 64-range sums."""
    r = lambda x: (x * 4 + 255) // 256 * 256
    for (B, T, H, Hv, Dk, Dv) in [(2, 256, 4, 4, 128, 64), (1, 100, 2, 4, 64, 128)]:
        p = _prob(B=B, T=T, H=H, Hv=Hv, Dk=Dk, Dv=Dv, dtype=g2.GDR2_FP32)
        n = B * T * H
        fwd = 3 * r(n * Dk) + 2 * r(n)
        assert g2.gdr2_fused_workspace_bytes(p, 0, 0) == g2.gdr2_chunk_workspace_bytes(p, 0) + fwd
        bwd = fwd + 3 * r(n * Dk) + r(n) + r(64 * H * (Dk + 1))
        assert g2.gdr2_fused_workspace_bytes(p, 0, 1) == g2.gdr2_chunk_workspace_bytes(p, 1) + bwd


def _noalloc(prob, ptrs=None):
    L = g2.lib()
    p = [FAKE] * 6 + [None, FAKE, None]
    if ptrs:
        for i, val in ptrs.items():
            p[i] = val
    pp = ctypes.byref(prob) if prob is not None else None
    return L.gdr2_chunk_fwd_noalloc(pp, *[ctypes.c_void_p(x) if x else None for x in p], None)


def test_noalloc_forward_validation():
    """gdr2_chunk_fwd_noalloc checks everything before its first HIP call: the
    problem, every pointer, and that the forward's workspace fits its fixed
    array (the training shape's 1.08 GB does not: GDR2_EWORKSPACE)."""
    assert _noalloc(None) == g2.GDR2_EINVAL
    assert _noalloc(_prob(B=0)) == g2.GDR2_EINVAL
    assert _noalloc(_prob(Dk=96)) == g2.GDR2_EUNSUPPORTED
    for idx in (0, 1, 2, 3, 4, 5, 7):
        assert _noalloc(_prob(), ptrs={idx: None}) == g2.GDR2_EINVAL, idx
        assert _noalloc(_prob(), ptrs={idx: FAKE + 8}) == g2.GDR2_EINVAL, idx
    for idx in (6, 8):
        assert _noalloc(_prob(), ptrs={idx: FAKE + 4}) == g2.GDR2_EINVAL, idx
    big = _prob(B=8, T=4096, H=16)
    assert g2.gdr2_chunk_workspace_bytes(big, 0) > g2.NOALLOC_SCRATCH_BYTES
    assert _noalloc(big) == g2.GDR2_EWORKSPACE
    # the largest fixed-length problem of this head size that fits, and one chunk more
    per = g2.gdr2_chunk_workspace_bytes(_prob(B=1, H=1, T=64), 0)
    n = g2.NOALLOC_SCRATCH_BYTES // per
    while g2.gdr2_chunk_workspace_bytes(_prob(B=1, H=1, T=64 * n), 0) > g2.NOALLOC_SCRATCH_BYTES:
        n -= 1
    assert _noalloc(_prob(B=1, H=1, T=64 * (n + 1))) == g2.GDR2_EWORKSPACE


def test_noalloc_scratch_size_matches_header():
    m = re.search(r"#define\s+GDR2_NOALLOC_SCRATCH_BYTES\s+\(\(size_t\)(\d+)\s*<<\s*(\d+)\)", open(HEADER).read())
    assert m is not None
    assert int(m.group(1)) << int(m.group(2)) == g2.NOALLOC_SCRATCH_BYTES
