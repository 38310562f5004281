"""GPU parity of the fused input stage (App. C.1, App. D.1 - D.2).

The fused calls take the raw projections: q and k are L2-normalised inside the
kernels (y = x (sum x^2 + eps)^(-1/2), rounded to bf16 as the operand of the
bf16 path) and the log-decay is formed in fp32 from the decay projection f as
g = -exp(a) softplus(f + delta).  The backward returns the gradients of the
raw inputs (dq, dk through the normalisation VJP; df, da, ddelta through the
activation).  The oracle is oracle.layer: the same stage in fp64 (normalised
q, k rounded to bf16 for a bf16 operator), then the fp64 token recurrence and
its adjoint.  Tolerances as elsewhere: rel-L2 2e-3 (bf16), 1e-5 (fp32).
"""

import numpy as np
import pytest

from oracle.layer import gdr2_fused_bwd, gdr2_fused_fwd
from paper_2605_22791_amd.inputs import make_fused
from tests.helpers import rel_l2
from tests.gpu_common import host

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-5, "bf16": 2e-3}
OUTS = ("o", "S_T", "dq", "dk", "dv", "df", "da", "ddelta", "db", "dw", "dS0")
ARGS = ("q", "k", "v", "f", "a", "delta", "b", "w")


def _case(msg):
    print(f"\n[gpu case] {msg}", flush=True)


def _dev(d):
    import torch
    io = torch.bfloat16 if d["dtype"] == "bf16" else torch.float32
    x = {}
    for n in ("q", "k", "v", "b", "w", "do"):
        x[n] = torch.from_numpy(np.ascontiguousarray(d[n])).cuda().to(io).contiguous()
    for n in ("f", "a", "delta", "S0", "dST"):
        x[n] = None if d.get(n) is None else torch.from_numpy(np.ascontiguousarray(d[n])).cuda().contiguous()
    x["cu"] = torch.from_numpy(d["cu_seqlens"]).cuda() if "cu_seqlens" in d else None
    return x


def _run(d, save=False, backward=True):
    import torch
    import paper_2605_22791_amd as g2
    x = _dev(d)
    args = [x[n] for n in ARGS]
    kw = dict(cu_seqlens=x["cu"], scale=d["scale"], eps=d["eps"])
    ws = None
    if save:
        prob = g2._problem(x["q"], x["v"], d["scale"])
        n = 0 if x["cu"] is None else x["cu"].numel() - 1
        ws = torch.empty(g2.gdr2_fused_workspace_bytes(prob, n, 1), dtype=torch.uint8, device="cuda")
    o, ST = g2.gdr2_fused_fwd(*args, x["S0"], ws=ws, save=save, **kw)
    out = {"o": host(o), "S_T": host(ST)}
    if backward:
        g = g2.gdr2_fused_bwd(*args, x["S0"], x["do"], x["dST"], ws=ws, saved=save, **kw)
        out.update({n: host(t) for n, t in g.items()})
    return out


def _oracle(d, backward=True):
    args = [d[n] for n in ARGS]
    kw = dict(scale=d["scale"], eps=d["eps"], cu_seqlens=d.get("cu_seqlens"), dtype=d["dtype"])
    o, ST = gdr2_fused_fwd(*args, d["S0"], **kw)
    r = {"o": o, "S_T": ST}
    if backward:
        r.update(gdr2_fused_bwd(*args, d["S0"], d["do"], d["dST"], **kw))
    return r


def _check(got, ref, tol, names=OUTS):
    err = {n: rel_l2(got[n], ref[n]) for n in names}
    print({k: f"{v:.2e}" for k, v in err.items()})
    for k, v in err.items():
        assert v < tol, (k, v)


@pytest.mark.parametrize("Dk,Dv", [(128, 128), (64, 128), (128, 64)])
def test_fused_matches_oracle(Dk, Dv):
    """B = 2, T = 200 (a ragged last chunk), H = 2: forward and every gradient."""
    d = make_fused(2, 200, 2, Dk, Dv, seed=300 + Dk + Dv, s0_std=0.05, with_dST=True)
    _case(f"fused bf16 B2 T200 H2 Dk{Dk} Dv{Dv}")
    _check(_run(d), _oracle(d), TOL["bf16"])


def test_fused_saved_path_equals_recompute():
    d = make_fused(1, 320, 3, 128, 128, seed=310, s0_std=0.05, with_dST=True)
    _case("fused bf16 B1 T320 H3: saving forward + saved backward vs recompute")
    got_s = _run(d, save=True)
    got_r = _run(d)
    for n in OUTS:
        assert np.array_equal(got_s[n], got_r[n]), n
    _check(got_r, _oracle(d), TOL["bf16"])


def test_fused_strong_decay_diagonal_blocks():
    """f shifted so that the log-decay reaches tens per token: the diagonal
    blocks whose decay exceeds e^60 are formed element by element, with the
    normalised q read from the kernel's inverse norms."""
    d = make_fused(1, 192, 2, 128, 128, seed=311, s0_std=0.05, with_dST=True)
    d["f"] = (d["f"] + 7.0).astype(np.float32)
    _case("fused bf16 B1 T192 H2, strong decay")
    _check(_run(d), _oracle(d), TOL["bf16"])


def test_fused_grouped_value_heads():
    d = make_fused(2, 130, 2, 128, 128, seed=312, Hv=4, s0_std=0.05, with_dST=True)
    _case("fused bf16 grouped H2 Hv4 B2 T130")
    _check(_run(d), _oracle(d), TOL["bf16"])


@pytest.mark.parametrize("Hv", [2, 4])
def test_fused_packed_batch(Hv):
    lengths = [100, 0, 64, 1, 130, 63]
    d = make_fused(0, 0, 2, 128, 64, seed=313 + Hv, Hv=Hv, lengths=lengths, s0_std=0.05, with_dST=True)
    _case(f"fused bf16 packed {lengths} H2 Hv{Hv}")
    _check(_run(d), _oracle(d), TOL["bf16"])
    got_s = _run(d, save=True)
    got_r = _run(d)
    for n in OUTS:
        assert np.array_equal(got_s[n], got_r[n]), n


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_fused_recurrent(dtype):
    import paper_2605_22791_amd as g2
    for lengths in (None, [5, 0, 1, 17]):
        if lengths is None:
            d = make_fused(2, 9, 2, 128, 64, seed=314, dtype=dtype, Hv=4, s0_std=0.05)
        else:
            d = make_fused(0, 0, 2, 64, 128, seed=315, dtype=dtype, lengths=lengths, s0_std=0.05)
        _case(f"fused recurrent {dtype} lengths {lengths}")
        x = _dev(d)
        S = x["S0"].clone()
        o = g2.gdr2_fused_recurrent(*[x[n] for n in ARGS], S, cu_seqlens=x["cu"], scale=d["scale"], eps=d["eps"])
        ref = _oracle(d, backward=False)
        e_o, e_s = rel_l2(host(o), ref["o"]), rel_l2(host(S), ref["S_T"])
        print("o", e_o, "S", e_s)
        assert e_o < TOL[dtype] and e_s < (1e-5 if dtype == "fp32" else 1e-4)


def test_fused_full_size_sampled_heads():
    """The training shape (B = 8, H = 16, T = 4096, d = 128) in one fused forward
    and backward; two (batch, head) pairs against the oracle run on their slice
    alone (ddelta and da sum over every pair: checked as the sums of df and of
    the pairs' own terms in the small cases), and ddelta against the sum of the
    returned df (its definition)."""
    import torch
    d = make_fused(8, 4096, 16, 128, 128, seed=2, s0_std=0.0, with_dST=False)
    _case("fused bf16 B8 T4096 H16 d128 (full size)")
    got = _run(d)
    torch.cuda.synchronize()
    dd = got["df"].sum(axis=(0, 1))
    assert rel_l2(got["ddelta"], dd) < 1e-5
    for (b, h) in ((0, 0), (5, 11)):
        sub = {n: d[n] for n in ("scale", "eps", "dtype")}
        for n in ("q", "k", "v", "f", "b", "w", "do"):
            sub[n] = d[n][b:b + 1, :, h:h + 1]
        sub["a"], sub["delta"] = d["a"][h:h + 1], d["delta"][h:h + 1]
        sub["S0"], sub["dST"] = None, None
        ref = _oracle(sub)
        part = {n: got[n][b:b + 1, :, h:h + 1] for n in ("o", "dq", "dk", "dv", "df", "db", "dw")}
        part["S_T"] = got["S_T"][b:b + 1, h:h + 1]
        _check(part, ref, TOL["bf16"], names=tuple(part))


def test_fused_decay_activation_over_its_domain():
    """fp32 decoding with f + delta spread over [-40, 40]: both tails of softplus
    (e^x for very negative x, x for large x) and the middle, against the fp64
    activation; the state after 24 tokens carries every token's decay."""
    import paper_2605_22791_amd as g2
    d = make_fused(1, 24, 2, 64, 64, seed=316, dtype="fp32", s0_std=0.5)
    rng = np.random.default_rng(17)
    d["f"] = (rng.uniform(-40.0, 40.0, d["f"].shape) - d["delta"][None, None]).astype(np.float32)
    d["a"] = np.array([-3.0, 0.5], dtype=np.float32)  # small magnitudes keep the large-x tokens' decay finite-sized
    _case("fused recurrent fp32, f + delta over [-40, 40]")
    x = _dev(d)
    S = x["S0"].clone()
    o = g2.gdr2_fused_recurrent(*[x[n] for n in ARGS], S, scale=d["scale"], eps=d["eps"])
    ref = _oracle(d, backward=False)
    e_o, e_s = rel_l2(host(o), ref["o"]), rel_l2(host(S), ref["S_T"])
    print("o", e_o, "S", e_s)
    assert e_o < 1e-5 and e_s < 1e-5


@pytest.mark.parametrize("case", ["plain", "grouped", "packed"])
def test_fused_fp32_chunk(case):
    """fp32 problems (the 1e-5 parity mode) run the stage as passes of their own
    around the fp32 operator: forward and every gradient at 1e-5, stored path
    bit-identical to the recomputing one."""
    if case == "plain":
        d = make_fused(2, 200, 2, 64, 128, seed=320, dtype="fp32", s0_std=0.05, with_dST=True)
    elif case == "grouped":
        d = make_fused(1, 130, 2, 128, 64, seed=321, dtype="fp32", Hv=4, s0_std=0.05, with_dST=True)
    else:
        d = make_fused(0, 0, 2, 128, 128, seed=322, dtype="fp32", lengths=[70, 0, 1, 130], s0_std=0.05,
                       with_dST=True)
    _case(f"fused fp32 chunk, {case}")
    got = _run(d)
    _check(got, _oracle(d), TOL["fp32"])
    got_s = _run(d, save=True)
    for n in OUTS:
        assert np.array_equal(got_s[n], got[n]), n
