"""GPU parity of the gate-aware chunkwise backward against the fp64 adjoint.

All seven gradients (dq, dk, dv, dlog_alpha, db, dw, dS0) are compared per
tensor by rel-L2: 1e-5 in fp32 mode, 2e-3 for bf16 problems (dlog_alpha and
dS0 are fp32 tensors but belong to a bf16 call and share its bound).
"""

import numpy as np
import pytest

from oracle import gdr2_recurrent_bwd, gdr2_chunk_bwd_ref
from paper_2605_22791_amd.inputs import config, make_inputs
from tests.helpers import rel_l2
from tests.gpu_common import dev_inputs, host, heads, pick, ws_layout, ws_view, CH

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-5, "bf16": 2e-3}
NAMES = [("dq", "dq"), ("dk", "dk"), ("dv", "dv"), ("dlog_alpha", "dg"), ("db", "db"), ("dw", "dw")]


def _case(msg):
    print(f"\n[gpu case] {msg}", flush=True)


def _run_bwd(d, ws=None):
    import paper_2605_22791_amd as g2
    x = dev_inputs(d)
    g = g2.gdr2_chunk_bwd(x["q"], x["k"], x["v"], x["log_alpha"], x["b"], x["w"], x["S0"], x["do"],
                          x["dST"], scale=d["scale"], ws=ws)
    return {n: host(t) for n, t in g.items()}


def _adjoint(d):
    return gdr2_recurrent_bwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"], d["do"],
                              d["dST"], d["scale"])


def _compare(got, ref, tol, pairs=None):
    worst = {}
    for gn, rn in NAMES:
        x = got[gn] if pairs is None else pick(got[gn], pairs)
        worst[gn] = rel_l2(x, ref[rn])
    x = got["dS0"] if pairs is None else pick(got["dS0"], pairs, state=True)
    worst["dS0"] = rel_l2(x, ref["dS0"])
    print({k: f"{v:.2e}" for k, v in worst.items()})
    for k, v in worst.items():
        assert v < tol, (k, v)


@pytest.mark.parametrize("Dk,Dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
def test_fp32_backward_small(Dk, Dv):
    d = make_inputs(1, 256, 2, Dk, Dv, seed=60 + Dk + Dv, dtype="fp32", s0_std=0.05, with_dST=True)
    _case(f"fp32 bwd B1 H2 T256 Dk{Dk} Dv{Dv} with S0 and dS_T")
    got = _run_bwd(d)
    _compare(got, _adjoint(d), TOL["fp32"])


def test_fp32_backward_workspace_intermediates():
    """dA_qk, dT and the chunk states against App. B's chunk equations (scaled dO)."""
    import torch
    d = make_inputs(1, 192, 1, 64, 64, seed=61, dtype="fp32", s0_std=0.1, with_dST=True)
    B, T, H, Dk, Dv = 1, 192, 1, 64, 64
    lay, total = ws_layout(B, T, H, Dk, Dv, True)
    ws = torch.full((total,), 0xFF, dtype=torch.uint8, device="cuda")
    _case("fp32 bwd workspace intermediates")
    _run_bwd(d, ws=ws)
    torch.cuda.synchronize()
    NT = T // CH
    from oracle.chunkwise import gdr2_chunk_fwd_ref
    _, _, it = gdr2_chunk_fwd_ref(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"],
                                  d["scale"], C=CH, keep=True)
    Hs = host(ws_view(ws, lay, "Hs", (B, H, NT, Dk, Dv)))
    Rs = host(ws_view(ws, lay, "Rs", (B, H, NT, CH, Dv)))
    assert rel_l2(Hs, it["h"]) < TOL["fp32"] and rel_l2(Rs, it["R"]) < TOL["fp32"]
    dAqk = host(ws_view(ws, lay, "DAqk", (B, H, NT, CH, CH)))
    dO = d["scale"] * d["do"].astype(np.float64)
    for n in range(NT):
        ref = np.tril(dO[0, n * CH:(n + 1) * CH, 0] @ it["R"][0, 0, n].T)
        assert rel_l2(dAqk[0, 0, n], ref) < TOL["fp32"]


@pytest.mark.parametrize("decay", ["channel", "scalar"])
def test_config1_bf16_backward_kda_gdn_limits(decay):
    d = config(1, decay=decay)
    _case(f"config1 bf16 bwd, tied gates, {decay} decay")
    got = _run_bwd(d)
    ref = _adjoint(d)
    _compare(got, ref, TOL["bf16"])
    # tied-gate identity on the GPU result: sum_c db + sum_c dw = dL/dbeta of the adjoint
    dbeta = got["db"].sum(-1) + got["dw"].sum(-1)
    dbeta_ref = ref["db"].sum(-1) + ref["dw"].sum(-1)
    assert rel_l2(dbeta, dbeta_ref) < TOL["bf16"]


def test_backward_determinism_and_poisoned_outputs():
    import torch
    import paper_2605_22791_amd as g2
    d = make_inputs(2, 256, 2, 128, 128, seed=62, dtype="bf16", s0_std=0.02, with_dST=True)
    _case("bwd determinism / poisoned outputs")
    x = dev_inputs(d)
    res = []
    for _ in range(2):
        grads = {n: torch.full_like(x[src], float("nan")) for n, src in
                 [("dq", "q"), ("dk", "k"), ("dv", "v"), ("dlog_alpha", "log_alpha"), ("db", "b"), ("dw", "w")]}
        grads["dS0"] = torch.full_like(x["S0"], float("nan"))
        g = g2.gdr2_chunk_bwd(x["q"], x["k"], x["v"], x["log_alpha"], x["b"], x["w"], x["S0"], x["do"],
                              x["dST"], scale=d["scale"], grads=grads)
        res.append({n: t.clone() for n, t in g.items()})
    for n in res[0]:
        assert torch.isfinite(res[0][n].float()).all(), n
        assert torch.equal(res[0][n], res[1][n]), n


def test_extreme_decay_backward():
    d = make_inputs(1, 128, 2, 64, 64, seed=63, dtype="fp32", s0_std=0.1, with_dST=True)
    la = d["log_alpha"].copy()
    la[0, 20, 0, :8] = -90.0
    la[0, 70, 1, 5:40] = -200.0
    d["log_alpha"] = la
    _case("bwd extreme decay spike")
    got = _run_bwd(d)
    _compare(got, _adjoint(d), TOL["fp32"])


def test_config2_full_size_backward_sampled_heads():
    d = config(2)
    pairs = [(0, 0), (5, 11)]
    _case("config2 bwd full size; adjoint on 2 heads")
    got = _run_bwd(d)
    for n, t in got.items():
        assert np.all(np.isfinite(t)), n
    sub = heads(d, pairs)
    ref = gdr2_recurrent_bwd(sub["q"], sub["k"], sub["v"], sub["log_alpha"], sub["b"], sub["w"], None,
                             sub["do"], None, d["scale"])
    _compare(got, ref, TOL["bf16"], pairs=pairs)


@pytest.mark.parametrize("Dk,Dv", [(64, 64), (64, 128), (128, 64), (128, 128)])
def test_bf16_backward_head_dims(Dk, Dv):
    # B*H = 6 chunk-heads of 5 chunks, with S0 and dS_T
    d = make_inputs(2, 320, 3, Dk, Dv, seed=64 + Dk + Dv, dtype="bf16", s0_std=0.05, with_dST=True)
    _case(f"bf16 bwd B2 H3 T320 Dk{Dk} Dv{Dv} with S0 and dS_T")
    _compare(_run_bwd(d), _adjoint(d), TOL["bf16"])


@pytest.mark.parametrize("Dk,Dv", [(64, 128), (128, 128)])
def test_bf16_long_memory_decay(Dk, Dv):
    """Slow decay (log_alpha = -softplus(N(0,1) - 5), about -0.01 per token): the
    state remembers hundreds of tokens, so the intra-chunk products' rounding
    reaches the state instead of fading within a few tokens.  With T in one bf16
    pass and A a bf16 operand of Y and U this regime took db past 2e-3 at Dk = 64."""
    d = make_inputs(2, 512, 2, Dk, Dv, seed=67 + Dk, dtype="bf16", decay_shift=-5.0, s0_std=0.05,
                    with_dST=True)
    _case(f"bf16 fwd+bwd long memory B2 H2 T512 Dk{Dk} Dv{Dv}")
    import paper_2605_22791_amd as g2
    from oracle import gdr2_recurrent_fwd
    x = dev_inputs(d)
    o, ST = g2.gdr2_chunk_fwd(x["q"], x["k"], x["v"], x["log_alpha"], x["b"], x["w"], x["S0"], scale=d["scale"])
    o_ref, S_ref = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"], d["scale"])
    e_o, e_s = rel_l2(host(o), o_ref), rel_l2(host(ST), S_ref)
    print("o", e_o, "S_T", e_s)
    assert e_o < TOL["bf16"] and e_s < TOL["bf16"]
    _compare(_run_bwd(d), _adjoint(d), TOL["bf16"])


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("case", ["no_erase_no_write", "no_erase", "no_decay"])
def test_degenerate_gates(dtype, case):
    """Gates at the ends of their range (Sec. 3.1): b = 0 erases nothing, w = 0
    writes nothing, log_alpha = 0 keeps the state.  With b = w = 0 the state
    only decays, so Ebar, Z, U, R and the Gram T vanish and A = I; with b = 0,
    w = 1 the rule is a decayed linear-attention write; with no decay every
    gamma is 1.  Forward and backward against the fp64 recurrence; a gradient
    whose exact value is zero (dv = dZ * w with w = 0) must come out exactly
    zero."""
    b_val, w_val = {"no_erase_no_write": (0.0, 0.0), "no_erase": (0.0, 1.0), "no_decay": (None, None)}[case]
    from oracle import gdr2_recurrent_fwd
    import paper_2605_22791_amd as g2
    d = make_inputs(2, 160, 2, 128, 64, seed=71, dtype=dtype, s0_std=0.05, with_dST=True)
    if case == "no_decay":
        d["log_alpha"] = np.zeros_like(d["log_alpha"])
    else:
        d["b"] = np.full_like(d["b"], b_val)
        d["w"] = np.full_like(d["w"], w_val)
        # a weak decay: with nothing written, S_T is S0 times the decay of all
        # 160 tokens, which at the usual decay (about e^-112) is below fp32's range
        d["log_alpha"] = (0.05 * d["log_alpha"]).astype(np.float32)
    _case(f"{dtype} degenerate gates: {case}")
    x = dev_inputs(d)
    o, ST = g2.gdr2_chunk_fwd(x["q"], x["k"], x["v"], x["log_alpha"], x["b"], x["w"], x["S0"], scale=d["scale"])
    o_ref, S_ref = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"], d["scale"])
    e_o, e_s = rel_l2(host(o), o_ref), rel_l2(host(ST), S_ref)
    print("o", e_o, "S_T", e_s)
    assert e_o < TOL[dtype] and e_s < TOL[dtype]
    got, ref = _run_bwd(d), _adjoint(d)
    for gn, rn in NAMES + [("dS0", "dS0")]:
        if not np.any(ref[rn]):
            assert not np.any(got[gn]), gn
            continue
        err = rel_l2(got[gn], ref[rn])
        print(gn, f"{err:.2e}")
        assert err < TOL[dtype], (gn, err)
    if w_val == 0.0:
        assert not np.any(ref["dv"])


def test_binding_refuses_bad_buffers():
    """Buffers that would send a kernel out of bounds are refused by the binding
    before any launch: a gradient buffer of the wrong shape or dtype, a
    workspace on the host, of the wrong dtype or too small, an output of the
    wrong shape."""
    import torch
    import paper_2605_22791_amd as g2
    d = make_inputs(1, 64, 2, 64, 64, seed=72, dtype="bf16")
    x = dev_inputs(d)
    args = [x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")]
    _case("binding: bad buffers refused")
    bad_grads = ({"dq": torch.empty(1, 64, 2, 32, dtype=torch.bfloat16, device="cuda")},
                 {"dlog_alpha": torch.empty(1, 64, 2, 64, dtype=torch.bfloat16, device="cuda")},
                 {"dS0": torch.empty(1, 2, 64, 32, dtype=torch.float32, device="cuda")})
    for g in bad_grads:
        with pytest.raises(ValueError):
            g2.gdr2_chunk_bwd(*args, None, x["do"], scale=d["scale"], grads=g)
    prob = g2._problem(x["q"], x["v"], d["scale"])
    need = g2.gdr2_chunk_workspace_bytes(prob, 0)
    for ws in (torch.empty(need, dtype=torch.uint8),
               torch.empty(need, dtype=torch.float32, device="cuda"),
               torch.empty(need - 1, dtype=torch.uint8, device="cuda")):
        with pytest.raises(ValueError):
            g2.gdr2_chunk_fwd(*args, scale=d["scale"], ws=ws)
    S = torch.zeros(1, 2, 64, 64, dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError):
        g2.gdr2_recurrent_step(*args, S, scale=d["scale"], o=torch.empty(1, 64, 2, 32, dtype=torch.bfloat16,
                                                                          device="cuda"))
    # the same call with correct buffers runs
    o, _ = g2.gdr2_chunk_fwd(*args, scale=d["scale"], ws=torch.empty(need, dtype=torch.uint8, device="cuda"))
    assert torch.isfinite(o.float()).all()


def test_bf16_backward_single_chunk_no_state():
    d = make_inputs(1, 64, 2, 128, 128, seed=65, dtype="bf16")
    _case("bf16 bwd one chunk, S0 = 0, dS_T = 0")
    _compare(_run_bwd(d), _adjoint(d), TOL["bf16"])


@pytest.mark.parametrize("T", [64, 100, 128, 192, 256])
@pytest.mark.parametrize("Dk,Dv", [(128, 128), (64, 64)])
def test_bf16_saved_path_few_chunks(T, Dk, Dv):
    """The saved training path on sequences of one to four chunks (T = 100: a
    full chunk and a partial one): the reverse scan walks two chunks per trip
    with the next two chunks' operands in flight, and the first and last trips
    load chunks they do not use, so an odd or even chunk count, one chunk and
    two chunks are its edge cases.  The workspace is NaN-poisoned, so a read of
    a region no kernel wrote (the causal zero blocks of A_qk and A are not
    stored) would show in the outputs.  These tensors are small (8 K elements
    at one chunk and d = 64), and the bf16 rounding of the exact result alone
    then ranges over 1.5e-3 .. 2.1e-3 rel-L2 by seed: a bf16-typed output is
    held to max(2e-3, 1.1 x that floor), computed here from the oracle."""
    import torch
    import paper_2605_22791_amd as g2
    from oracle import gdr2_recurrent_fwd
    d = make_inputs(1, T, 2, Dk, Dv, seed=80 + T + Dk, dtype="bf16", s0_std=0.05, with_dST=True)
    _case(f"bf16 saved path B1 H2 T{T} Dk{Dk} Dv{Dv}")
    x = dev_inputs(d)
    args = [x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")]
    prob = g2._problem(x["q"], x["v"], d["scale"])
    ws = torch.full((g2.gdr2_chunk_workspace_bytes(prob, 1),), 0xFF, dtype=torch.uint8, device="cuda")
    o, ST = g2.gdr2_chunk_fwd(*args, x["S0"], scale=d["scale"], ws=ws, save=True)
    g = g2.gdr2_chunk_bwd(*args, x["S0"], x["do"], x["dST"], scale=d["scale"], ws=ws, saved=True)
    torch.cuda.synchronize()
    o_ref, S_ref = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"],
                                      d["scale"])
    ref = _adjoint(d)

    def bound(x, bf16_typed):
        if not bf16_typed:
            return TOL["bf16"]
        xb = torch.tensor(x, dtype=torch.float64).to(torch.bfloat16).to(torch.float64).numpy()
        return max(TOL["bf16"], 1.1 * rel_l2(xb, x))

    got = {n: host(t) for n, t in g.items()}
    checks = [("o", host(o), o_ref, True), ("S_T", host(ST), S_ref, False), ("dS0", got["dS0"], ref["dS0"], False)]
    checks += [(gn, got[gn], ref[rn], gn != "dlog_alpha") for gn, rn in NAMES]
    for name, x, r, bf in checks:
        err, lim = rel_l2(x, r), bound(r, bf)
        print(f"{name}: {err:.2e} (bound {lim:.2e})")
        assert err < lim, (name, err, lim)


def test_bf16_extreme_decay_backward():
    """Decay spikes push a block's internal decay past e^60: the diagonal blocks
    of the decay products are then formed element by element."""
    d = make_inputs(1, 192, 2, 128, 128, seed=66, dtype="bf16", s0_std=0.1, with_dST=True)
    la = d["log_alpha"].copy()
    la[0, 20, 0, :8] = -90.0
    la[0, 70, 1, 5:40] = -200.0
    la[0, 75, 1, 30:] = -70.0
    la[0, 140:150, 0, :] = -9.0
    d["log_alpha"] = la
    _case("bf16 bwd extreme decay spikes")
    _compare(_run_bwd(d), _adjoint(d), TOL["bf16"])


@pytest.mark.parametrize("Dk,Dv", [(64, 128), (128, 64)])
def test_bf16_backward_workspace_intermediates(Dk, Dv):
    """A (fp16 16 x 16 blocks with block scales) and dR (split bf16 16 x 16
    blocks) in the backward workspace against the chunk algebra: A = (I + T)^{-1}
    (App. A.2) and the reverse recursion of App. B.1, dR = scale A_qk^T dO +
    Ktail dS_C."""
    import torch
    from oracle.chunkwise import gdr2_chunk_fwd_ref
    from tests.gpu_common import ws_layout_bf16, decode_tiles_f16, decode_tiles_split, round_tiles_f16
    B, T, H = 1, 192, 2
    d = make_inputs(B, T, H, Dk, Dv, seed=67, dtype="bf16", s0_std=0.05, with_dST=True)
    lay, total, NC = ws_layout_bf16(B, T, H, Dk, Dv, bwd=True)
    ws = torch.full((total,), 0xFF, dtype=torch.uint8, device="cuda")
    _case(f"bf16 bwd workspace intermediates Dk{Dk} Dv{Dv}")
    _run_bwd(d, ws=ws)
    torch.cuda.synchronize()
    raw = ws.cpu().numpy()
    _, _, it = gdr2_chunk_fwd_ref(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"],
                                  d["scale"], C=CH, keep=True)
    NT = T // CH
    worst = {"A": 0.0, "A_rounded": 0.0, "dR": 0.0}
    for bi in range(B):
        for hi in range(H):
            dS = d["dST"][bi, hi].astype(np.float64)
            for n in range(NT - 1, -1, -1):
                ch = (bi * H + hi) * NT + n
                dO = d["scale"] * d["do"][bi, n * CH:(n + 1) * CH, hi].astype(np.float64)
                dR = it["Aqk"][bi, hi, n].T @ dO + it["Ktail"][bi, hi, n] @ dS
                dS = it["gC"][bi, hi, n][:, None] * dS + it["Qg"][bi, hi, n].T @ dO - it["Y"][bi, hi, n].T @ dR

                def region(name):
                    off, per = lay[name]
                    return raw[off + ch * per: off + (ch + 1) * per]

                # A[r][s]: blocks [s][r];  dR[r][v]: blocks [v][r]
                A = decode_tiles_f16(region("Am"), region("Amsc"), 4, 4)
                # the tiles above the diagonal are zero and not stored
                for rb_ in range(4):
                    for sb_ in range(rb_ + 1, 4):
                        A[16 * rb_:16 * rb_ + 16, 16 * sb_:16 * sb_ + 16] = 0.0
                dRg = decode_tiles_split(region("DR"), Dv // 16, 4)
                Aref = it["A"][bi, hi, n]
                worst["A"] = max(worst["A"], rel_l2(A, Aref))
                worst["A_rounded"] = max(worst["A_rounded"], rel_l2(A, round_tiles_f16(Aref)))
                worst["dR"] = max(worst["dR"], rel_l2(dRg, dR))
    print({k_: f"{v_:.2e}" for k_, v_ in worst.items()})
    # A's copy is fp16 under a power-of-two block scale: every element within
    # half an fp16 ulp (relative 2^-11) of the fp32 value, so within 4.9e-4 of
    # the exact one in rel-L2.  A itself comes from a Gram matrix whose products
    # are fp32-accurate (split hi/lo) and an fp32 solve (about 2e-7), so its copy
    # matches the exact A rounded the same way but for rounding ties (a one-pass
    # bf16 Gram would put it near 1e-3).  dR is kept split (fp32-accurate):
    # dR = scale A_qk^T dO + Ktail dS_C takes dS_C from the reverse scan, whose
    # Y^T dR product uses the bf16 Y (about 1e-5).
    assert worst["A_rounded"] < 3e-5 and worst["A"] < 4.9e-4 and worst["dR"] < 1e-4, worst


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_saved_training_path_matches_recompute(dtype):
    """gdr2_chunk_fwd_save / gdr2_chunk_bwd_saved run the same kernels on the same
    inputs as the recomputing backward, so o, S_T and every gradient must be
    bit-identical to it (and therefore within the bound of the adjoint)."""
    import torch
    import paper_2605_22791_amd as g2
    d = make_inputs(2, 256, 3, 128, 64, seed=68, dtype=dtype, s0_std=0.05, with_dST=True)
    _case(f"{dtype} saved training path B2 H3 T256 Dk128 Dv64")
    x = dev_inputs(d)
    args = [x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")]
    prob = g2._problem(x["q"], x["v"], d["scale"])
    ws = torch.full((g2.gdr2_chunk_workspace_bytes(prob, 1),), 0xFF, dtype=torch.uint8, device="cuda")
    o_s, S_s = g2.gdr2_chunk_fwd(*args, x["S0"], scale=d["scale"], ws=ws, save=True)
    g_s = g2.gdr2_chunk_bwd(*args, x["S0"], x["do"], x["dST"], scale=d["scale"], ws=ws, saved=True)
    o_r, S_r = g2.gdr2_chunk_fwd(*args, x["S0"], scale=d["scale"])
    g_r = g2.gdr2_chunk_bwd(*args, x["S0"], x["do"], x["dST"], scale=d["scale"])
    torch.cuda.synchronize()
    assert torch.equal(o_s, o_r) and torch.equal(S_s, S_r)
    for n in g_r:
        assert torch.equal(g_s[n], g_r[n]), n
    _compare({n: host(t) for n, t in g_s.items()}, _adjoint(d), TOL[dtype])


def test_config3_long_context_backward_sampled_head():
    """B=1 H=16 T=65536 (1024 chunks per head, slow-forgetting decay, S0 != 0):
    the reverse scan carries dS across every chunk; adjoint on one head."""
    d = config(3)
    d["dST"] = None
    pairs = [(0, 11)]
    _case("config3 bwd B1 H16 T65536 d128 bf16; adjoint on 1 head")
    import paper_2605_22791_amd as g2
    x = dev_inputs(d)
    g = g2.gdr2_chunk_bwd(x["q"], x["k"], x["v"], x["log_alpha"], x["b"], x["w"], x["S0"], x["do"], None,
                          scale=d["scale"])
    got = {n: host(t) for n, t in g.items()}
    for n, t in got.items():
        assert np.all(np.isfinite(t)), n
    sub = heads(d, pairs)
    ref = gdr2_recurrent_bwd(sub["q"], sub["k"], sub["v"], sub["log_alpha"], sub["b"], sub["w"], sub["S0"],
                             sub["do"], None, d["scale"])
    _compare(got, ref, TOL["bf16"], pairs=pairs)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_negative_eigenvalue_backward(dtype):
    """b in [0, 2] (negative-eigenvalue variant, Sec. 3.1; NEXT-4): the same
    operator on a wider erase range, forward and every gradient against the
    adjoint, with a partial last chunk (T = 300)."""
    d = make_inputs(1, 300, 2, 128, 128, seed=69, dtype=dtype, s0_std=0.05, with_dST=True)
    d["b"] = 2.0 * d["b"]   # exact in bf16
    _case(f"{dtype} bwd, erase gate in [0, 2], T300")
    _compare(_run_bwd(d), _adjoint(d), TOL[dtype])


def test_negative_eigenvalue_reflections_keep_the_state_norm():
    """b = 2 with unit keys, no decay and no write: 4096 Householder reflections
    per head; the bf16 path's fp32 state keeps its Frobenius norm to 2e-4 (the
    drift is the rounding of the one bf16 product on the state path, Y S with
    the bf16 part of S; 6.7e-5 measured).  The keys are +-1/2 on four random
    channels, unit vectors exactly in bf16."""
    import paper_2605_22791_amd as g2
    d = make_inputs(1, 4096, 2, 128, 128, seed=70, dtype="bf16", s0_std=0.05)
    rng = np.random.default_rng(70)
    k = np.zeros_like(d["k"])
    for t in range(k.shape[1]):
        for h in range(k.shape[2]):
            k[0, t, h, rng.choice(128, 4, replace=False)] = rng.choice([-0.5, 0.5], 4)
    d["k"] = k
    d["b"] = np.full_like(d["b"], 2.0)
    d["log_alpha"] = np.zeros_like(d["log_alpha"])
    d["w"] = np.zeros_like(d["w"])
    _case("bf16 fwd, 4096 reflections")
    x = dev_inputs(d)
    _, ST = g2.gdr2_chunk_fwd(*[x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")], x["S0"], scale=d["scale"])
    n0 = np.linalg.norm(d["S0"].astype(np.float64), axis=(-2, -1))
    n1 = np.linalg.norm(host(ST), axis=(-2, -1))
    print("norm ratio", n1 / n0)
    assert np.allclose(n1, n0, rtol=2e-4)


def test_config2_stored_path_sampled_heads():
    """The path bench.py times: gdr2_chunk_fwd_save + gdr2_chunk_bwd_saved at the
    1.3B-layer training shape (B8 H16 T4096 d128 bf16, App. D.3 with stored
    chunk states), where B*H = 128 puts the two value slices of each head on
    one XCD.  o, S_T and all seven gradients against the fp64 recurrence and
    its adjoint on three (batch, head) pairs, the first, a middle and the last."""
    import torch
    import paper_2605_22791_amd as g2
    from oracle import gdr2_recurrent_fwd
    d = config(2)
    pairs = [(0, 0), (5, 11), (7, 15)]
    _case("config2 stored training path B8 H16 T4096 d128 bf16; oracle on 3 heads")
    x = dev_inputs(d)
    args = [x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")]
    prob = g2._problem(x["q"], x["v"], d["scale"])
    ws = torch.empty(g2.gdr2_chunk_workspace_bytes(prob, 1), dtype=torch.uint8, device="cuda")
    o, ST = g2.gdr2_chunk_fwd(*args, None, scale=d["scale"], ws=ws, save=True)
    g = g2.gdr2_chunk_bwd(*args, None, x["do"], None, scale=d["scale"], ws=ws, saved=True)
    torch.cuda.synchronize()
    got = {n: host(t) for n, t in g.items()}
    o, ST = host(o), host(ST)
    del ws, x, g
    for n, t in list(got.items()) + [("o", o), ("S_T", ST)]:
        assert np.all(np.isfinite(t)), n
    sub = heads(d, pairs)
    o_ref, S_ref = gdr2_recurrent_fwd(sub["q"], sub["k"], sub["v"], sub["log_alpha"], sub["b"], sub["w"], None,
                                      d["scale"])
    ro, rs = rel_l2(pick(o, pairs), o_ref), rel_l2(pick(ST, pairs, state=True), S_ref)
    print(f"rel o {ro:.2e} S_T {rs:.2e}")
    assert ro < TOL["bf16"] and rs < TOL["bf16"]
    ref = gdr2_recurrent_bwd(sub["q"], sub["k"], sub["v"], sub["log_alpha"], sub["b"], sub["w"], None,
                             sub["do"], None, d["scale"])
    _compare(got, ref, TOL["bf16"], pairs=pairs)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("mode", ["scalar_erase", "scalar_write"])
def test_scalarized_gate_modes(mode, dtype):
    """Table 5's gate-structure modes: one of the two gates averaged over its
    channels and broadcast, the other channel-wise.  scalar_erase: b = mean_c(b) 1
    with a channel-wise w; scalar_write: a channel-wise b with w = mean_c(w) 1.
    The operator is unchanged; forward and every gradient against the fp64
    recurrence and adjoint (T = 300: five chunks, the last one with 44 rows), and the
    gradient of the scalar gate itself (the channel sum of the broadcast gate's
    gradient) against the adjoint's."""
    from oracle import gdr2_recurrent_fwd
    from paper_2605_22791_amd.inputs import bf16_round
    import paper_2605_22791_amd as g2
    d = make_inputs(2, 300, 2, 128, 128, seed=73, dtype=dtype, s0_std=0.05, with_dST=True)
    rnd = bf16_round if dtype == "bf16" else (lambda y: y.astype(np.float32))
    name = "b" if mode == "scalar_erase" else "w"
    d[name] = np.ascontiguousarray(np.broadcast_to(rnd(d[name].mean(axis=-1, keepdims=True)), d[name].shape))
    _case(f"{dtype} gate mode {mode}, B2 H2 T300 d128")
    x = dev_inputs(d)
    o, ST = g2.gdr2_chunk_fwd(*[x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")], x["S0"], scale=d["scale"])
    o_ref, S_ref = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"], d["scale"])
    e_o, e_s = rel_l2(host(o), o_ref), rel_l2(host(ST), S_ref)
    print(f"o {e_o:.2e} S_T {e_s:.2e}")
    assert e_o < TOL[dtype] and e_s < TOL[dtype]
    got, ref = _run_bwd(d), _adjoint(d)
    _compare(got, ref, TOL[dtype])
    # the scalar gate's gradient is the channel sum of the broadcast gate's, which
    # the caller forms from the dtype-typed output: its error floor is that of
    # the same sum over the rounded exact gradient (the rounding errors of Dk or
    # Dv terms add up while the sum partly cancels), plus the kernel's own error
    gn = "db" if name == "b" else "dw"
    e_g = rel_l2(got[gn].sum(-1), ref[gn].sum(-1))
    floor = rel_l2(rnd(ref[gn].astype(np.float32)).sum(-1), ref[gn].sum(-1)) if dtype == "bf16" else 0.0
    print(f"scalar-gate gradient {e_g:.2e} (rounding floor {floor:.2e})")
    assert e_g < np.hypot(floor, TOL[dtype] if dtype == "fp32" else 1.2e-3), (e_g, floor)
