"""GPU parity of the chunkwise forward against the fp64 oracle.

Tolerances (rel-L2 per output tensor, oracle on the identical inputs): 1e-5 in
fp32 mode, 2e-3 for bf16 problems.  Large workloads run whole on the GPU and
are compared on sampled (batch, head) pairs, which the oracle computes exactly.
"""

import numpy as np
import pytest

from oracle import gdr2_recurrent_fwd, gdr2_chunk_fwd_ref
from paper_2605_22791_amd.inputs import config, make_inputs
from tests.helpers import rel_l2
from tests.gpu_common import dev_inputs, host, heads, pick, ws_layout, ws_view, CH

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-5, "bf16": 2e-3}


def _run_fwd(d, S0=True, ws=None):
    import paper_2605_22791_amd as g2
    x = dev_inputs(d)
    o, ST = g2.gdr2_chunk_fwd(x["q"], x["k"], x["v"], x["log_alpha"], x["b"], x["w"],
                              x["S0"] if S0 else None, scale=d["scale"], ws=ws)
    return host(o), host(ST), x


def _oracle(d):
    return gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"], d["scale"])


def _case(msg):
    print(f"\n[gpu case] {msg}", flush=True)


def test_config0_fp32_forward():
    d = config(0)
    _case("config0 fp32 B1 H2 T256 d64")
    o, ST, _ = _run_fwd(d)
    o_ref, S_ref = _oracle(d)
    print("rel o", rel_l2(o, o_ref), "S_T", rel_l2(ST, S_ref))
    assert rel_l2(o, o_ref) < TOL["fp32"]
    assert rel_l2(ST, S_ref) < TOL["fp32"]


def test_config0_workspace_intermediates():
    """Per-kernel parity: Y, U, Ktail, Qg, A_qk, gamma_C against App. A's chunk algebra."""
    import torch
    import paper_2605_22791_amd as g2
    d = config(0, s0_std=0.1)
    B, T, H, Dk, Dv = d["B"], d["T"], d["H"], d["Dk"], d["Dv"]
    lay, total = ws_layout(B, T, H, Dk, Dv, False)
    ws = torch.full((total,), 0xFF, dtype=torch.uint8, device="cuda")   # NaN-poisoned
    _case("config0 workspace intermediates")
    _run_fwd(d, ws=ws)
    torch.cuda.synchronize()
    _, _, it = gdr2_chunk_fwd_ref(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"],
                                  d["scale"], C=CH, keep=True)
    NT = T // CH
    got = {n: host(ws_view(ws, lay, n, shape)) for n, shape in
           [("Y", (B, H, NT, CH, Dk)), ("U", (B, H, NT, CH, Dv)), ("Kt", (B, H, NT, CH, Dk)),
            ("Qg", (B, H, NT, CH, Dk)), ("Aqk", (B, H, NT, CH, CH)), ("GC", (B, H, NT, Dk))]}
    ref = {"Y": it["Y"], "U": it["U"], "Kt": it["Ktail"], "Qg": it["Qg"], "Aqk": it["Aqk"], "GC": it["gC"]}
    for n in ref:
        assert np.all(np.isfinite(got[n])), n
        assert rel_l2(got[n], ref[n]) < TOL["fp32"], (n, rel_l2(got[n], ref[n]))


@pytest.mark.parametrize("decay", ["channel", "scalar"])
def test_config1_bf16_forward_kda_gdn_limits(decay):
    d = config(1, decay=decay)
    _case(f"config1 bf16 tied gates, {decay} decay")
    o, ST, _ = _run_fwd(d)
    o_ref, S_ref = _oracle(d)
    print("rel o", rel_l2(o, o_ref), "S_T", rel_l2(ST, S_ref))
    assert rel_l2(o, o_ref) < TOL["bf16"]
    assert rel_l2(ST, S_ref) < TOL["bf16"]


@pytest.mark.parametrize("Dk,Dv,dtype", [(64, 128, "fp32"), (128, 64, "fp32"), (128, 128, "fp32"),
                                         (64, 64, "bf16")])
def test_head_dims(Dk, Dv, dtype):
    d = make_inputs(2, 192, 3, Dk, Dv, seed=40 + Dk + Dv, dtype=dtype, s0_std=0.05)
    _case(f"head dims Dk{Dk} Dv{Dv} {dtype}")
    o, ST, _ = _run_fwd(d)
    o_ref, S_ref = _oracle(d)
    assert rel_l2(o, o_ref) < TOL[dtype]
    assert rel_l2(ST, S_ref) < TOL[dtype]


def test_state_passing_split_equals_one_call():
    import paper_2605_22791_amd as g2
    d = make_inputs(1, 320, 2, 128, 128, seed=50, dtype="fp32", s0_std=0.05)
    _case("state passing 320 = 128 + 192")
    x = dev_inputs(d)
    o_all, S_all = g2.gdr2_chunk_fwd(x["q"], x["k"], x["v"], x["log_alpha"], x["b"], x["w"], x["S0"], scale=d["scale"])
    sl = lambda t, a, b_: t[:, a:b_].contiguous()
    args1 = [sl(x[n], 0, 128) for n in ("q", "k", "v", "log_alpha", "b", "w")]
    args2 = [sl(x[n], 128, 320) for n in ("q", "k", "v", "log_alpha", "b", "w")]
    o1, S1 = g2.gdr2_chunk_fwd(*args1, x["S0"], scale=d["scale"])
    o2, S2 = g2.gdr2_chunk_fwd(*args2, S1, scale=d["scale"])
    assert rel_l2(np.concatenate([host(o1), host(o2)], axis=1), host(o_all)) < 1e-6
    assert rel_l2(host(S2), host(S_all)) < 1e-6


def test_determinism_and_every_output_written():
    import torch
    import paper_2605_22791_amd as g2
    d = make_inputs(2, 256, 2, 128, 128, seed=51, dtype="bf16", s0_std=0.02)
    _case("determinism / poisoned outputs")
    x = dev_inputs(d)
    outs = []
    for _ in range(2):
        o = torch.full_like(x["v"], float("nan"))
        ST = torch.full((2, 2, 128, 128), float("nan"), device="cuda")
        g2.gdr2_chunk_fwd(x["q"], x["k"], x["v"], x["log_alpha"], x["b"], x["w"], x["S0"],
                          scale=d["scale"], o=o, S_T=ST)
        outs.append((o.clone(), ST.clone()))
    assert torch.isfinite(outs[0][0].float()).all() and torch.isfinite(outs[0][1]).all()
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


def test_extreme_decay_uses_exact_diagonal_blocks():
    """A decay spike (g = -90 on some channels) makes a block's internal decay
    exceed fp32's exp range; the diagonal tiles then take the element-wise path."""
    d = make_inputs(1, 128, 2, 64, 64, seed=52, dtype="fp32", s0_std=0.1)
    la = d["log_alpha"].copy()
    la[0, 20, 0, :8] = -90.0
    la[0, 70, 1, 5:40] = -200.0
    la[0, 75, 1, 30:] = -70.0
    d["log_alpha"] = la
    _case("extreme decay spike")
    o, ST, _ = _run_fwd(d)
    o_ref, S_ref = _oracle(d)
    print("rel o", rel_l2(o, o_ref), "S_T", rel_l2(ST, S_ref))
    assert rel_l2(o, o_ref) < TOL["fp32"]
    assert rel_l2(ST, S_ref) < TOL["fp32"]


def test_negative_eigenvalue_erase_range():
    """b in [0, 2] (negative-eigenvalue variant, Sec. 3.1): same operator, wider input range."""
    d = make_inputs(2, 256, 2, 128, 128, seed=53, dtype="fp32", s0_std=0.05)
    d["b"] = 2.0 * d["b"]
    _case("erase gate in [0,2]")
    o, ST, _ = _run_fwd(d)
    o_ref, S_ref = _oracle(d)
    assert rel_l2(o, o_ref) < TOL["fp32"]
    assert rel_l2(ST, S_ref) < TOL["fp32"]


def test_config2_full_size_sampled_heads():
    d = config(2)
    pairs = [(0, 0), (7, 15), (3, 9)]
    _case("config2 full size B8 H16 T4096 d128 bf16; oracle on 3 heads")
    o, ST, _ = _run_fwd(d)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(ST))
    sub = heads(d, pairs)
    o_ref, S_ref = gdr2_recurrent_fwd(sub["q"], sub["k"], sub["v"], sub["log_alpha"], sub["b"], sub["w"],
                                      None, d["scale"])
    ro, rs = rel_l2(pick(o, pairs), o_ref), rel_l2(pick(ST, pairs, state=True), S_ref)
    print("rel o", ro, "S_T", rs)
    assert ro < TOL["bf16"] and rs < TOL["bf16"]


def test_config3_long_context_sampled_head():
    d = config(3)
    pairs = [(0, 5)]
    _case("config3 B1 H16 T65536 d128 bf16; oracle on 1 head")
    o, ST, _ = _run_fwd(d)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(ST))
    sub = heads(d, pairs)
    o_ref, S_ref = gdr2_recurrent_fwd(sub["q"], sub["k"], sub["v"], sub["log_alpha"], sub["b"], sub["w"],
                                      sub["S0"], d["scale"])
    ro, rs = rel_l2(pick(o, pairs), o_ref), rel_l2(pick(ST, pairs, state=True), S_ref)
    print("rel o", ro, "S_T", rs)
    assert ro < TOL["bf16"] and rs < TOL["bf16"]
