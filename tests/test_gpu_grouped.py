"""GPU parity of grouped value heads (Sec. 3.5, App. C.1; NEXT-2).

Hv = G * H value heads share the H key heads: value head j reads q, k, the
log-decay and b of key head j // G, while v, w, o, dout and the states live on
the value heads; dq, dk, db and dlog_alpha sum over each group.  The oracle is
the fp64 recurrence with the key side repeated over the groups (and its adjoint
summed back).  Tolerances as elsewhere (rel-L2 2e-3 bf16, 1e-5 fp32).
"""

import numpy as np
import pytest

from oracle import gdr2_grouped_bwd, gdr2_grouped_fwd, gdr2_packed_bwd, gdr2_packed_fwd
from paper_2605_22791_amd.inputs import make_grouped
from tests.helpers import rel_l2
from tests.gpu_common import dev_inputs, host

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-5, "bf16": 2e-3}
GRADS = ("dq", "dk", "dv", "dlog_alpha", "db", "dw", "dS0")
REF = {"dlog_alpha": "dg"}
ARGS = ("q", "k", "v", "log_alpha", "b", "w")


def _case(msg):
    print(f"\n[gpu case] {msg}", flush=True)


def _check(got, ref, tol):
    err = {n: rel_l2(got[n], ref[REF.get(n, n)]) for n in ("o", "S_T") + GRADS}
    print({k: f"{v:.2e}" for k, v in err.items()})
    for k, v in err.items():
        assert v < tol, (k, v)


def _run(d, save=False):
    import torch
    import paper_2605_22791_amd as g2
    x = dev_inputs(d)
    args = [x[n] for n in ARGS]
    ws = None
    if save:
        prob = g2._problem(x["q"], x["v"], d["scale"])
        ws = torch.empty(g2.gdr2_chunk_workspace_bytes(prob, 1), dtype=torch.uint8, device="cuda")
    o, ST = g2.gdr2_chunk_fwd(*args, x["S0"], scale=d["scale"], ws=ws, save=save)
    g = g2.gdr2_chunk_bwd(*args, x["S0"], x["do"], x["dST"], scale=d["scale"], ws=ws, saved=save)
    out = {"o": host(o), "S_T": host(ST)}
    out.update({n: host(t) for n, t in g.items()})
    return out


def _oracle(d):
    args = [d[n] for n in ARGS]
    o, ST = gdr2_grouped_fwd(*args, d["S0"], d["scale"])
    r = gdr2_grouped_bwd(*args, d["S0"], d["do"], d["dST"], d["scale"])
    r.update(o=o, S_T=ST)
    return r


@pytest.mark.parametrize("dtype,G", [("bf16", 2), ("bf16", 4), ("fp32", 2), ("fp32", 4)])
def test_grouped_value_heads_match_oracle(dtype, G):
    d = make_grouped(2, 200, 2, 2 * G, 128, 128, seed=140 + G, dtype=dtype, s0_std=0.05, with_dST=True)
    _case(f"grouped {dtype} B2 T200 H2 Hv{2 * G}")
    _check(_run(d), _oracle(d), TOL[dtype])


def test_grouped_saved_path_and_head_dims():
    """Dk = 64, Dv = 128, G = 2: stored training path bit-identical to the recomputing one."""
    d = make_grouped(1, 320, 2, 4, 64, 128, seed=146, dtype="bf16", s0_std=0.05, with_dST=True)
    _case("grouped bf16 B1 T320 H2 Hv4 Dk64 Dv128, saved vs recompute")
    got_s = _run(d, save=True)
    got_r = _run(d)
    for n in got_r:
        assert np.array_equal(got_s[n], got_r[n]), n
    _check(got_r, _oracle(d), TOL["bf16"])


@pytest.mark.parametrize("B,H,Hv,Dv", [(2, 4, 8, 128), (4, 2, 4, 64), (4, 2, 8, 128)])
def test_grouped_scans_grouped_on_xcds(B, H, Hv, Dv):
    """Enough (batch, key head) pairs (a multiple of 8) for the scans to place the
    value slices of one key head's value heads on one XCD (the grouped block
    order); G = 2 and 4, one and two value slices per head."""
    d = make_grouped(B, 192, H, Hv, 128, Dv, seed=150 + B + Hv + Dv, dtype="bf16", s0_std=0.05, with_dST=True)
    assert (B * H) % 8 == 0
    _case(f"grouped bf16 B{B} T192 H{H} Hv{Hv} Dv{Dv}: XCD-grouped scan order")
    _check(_run(d), _oracle(d), TOL["bf16"])


def test_grouped_segmented_scans_grouped_on_xcds():
    """B1 H2 Hv4 T4096: four segments per sequence and a multiple of 8 (key head,
    segment) units, so the sequence-parallel scans take the XCD-grouped order."""
    from tests.gpu_common import scan_segments
    nseg = scan_segments(1, 4096, 4, 128)[0]
    assert nseg > 1 and (2 * nseg) % 8 == 0
    d = make_grouped(1, 4096, 2, 4, 128, 128, seed=149, dtype="bf16", decay_shift=-2.0, s0_std=0.05,
                     with_dST=True)
    _case(f"grouped bf16 B1 T4096 H2 Hv4, {nseg} segments, XCD-grouped order")
    _check(_run(d), _oracle(d), TOL["bf16"])


def test_grouped_long_sequence_parallel_scans():
    """B1 H1 Hv2 T2048: few scans and long sequences switch the sequence-parallel scans on."""
    from tests.gpu_common import scan_segments
    assert scan_segments(1, 2048, 2, 128)[0] > 1
    d = make_grouped(1, 2048, 1, 2, 128, 128, seed=147, dtype="bf16", decay_shift=-2.0, s0_std=0.05,
                     with_dST=True)
    _case("grouped bf16 B1 T2048 H1 Hv2, segmented scans")
    _check(_run(d), _oracle(d), TOL["bf16"])


def test_grouped_packed_batch():
    import torch
    import paper_2605_22791_amd as g2
    lengths = [70, 0, 130, 5]
    cu_np = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    d = make_grouped(1, int(cu_np[-1]), 2, 4, 128, 64, seed=148, dtype="bf16")
    rng = np.random.default_rng(148)
    N = len(lengths)
    d["S0"] = (0.05 * rng.standard_normal((N, 4, 128, 64))).astype(np.float32)
    d["dST"] = rng.standard_normal((N, 4, 128, 64)).astype(np.float32)
    _case(f"grouped packed bf16 lengths {lengths} H2 Hv4")
    x = dev_inputs(d)
    cu = torch.from_numpy(cu_np).cuda()
    args = [x[n] for n in ARGS]
    o, ST = g2.gdr2_chunk_fwd_varlen(*args, cu, x["S0"], scale=d["scale"])
    g = g2.gdr2_chunk_bwd_varlen(*args, cu, x["S0"], x["do"], x["dST"], scale=d["scale"])
    got = {"o": host(o), "S_T": host(ST)}
    got.update({n: host(t) for n, t in g.items()})
    # oracle: packed (per sequence) over the key side repeated across the groups
    G = 2
    rep = {n: np.repeat(d[n].astype(np.float64), G, axis=2) for n in ("q", "k", "log_alpha", "b")}
    eargs = [rep["q"], rep["k"], d["v"], rep["log_alpha"], rep["b"], d["w"]]
    o_r, S_r = gdr2_packed_fwd(*eargs, cu_np, d["S0"], d["scale"])
    r = gdr2_packed_bwd(*eargs, cu_np, d["S0"], d["do"], d["dST"], d["scale"])
    for n in ("dq", "dk", "dg", "db"):
        r[n] = r[n].reshape(1, -1, 2, G, 128).sum(axis=3)
    r.update(o=o_r, S_T=S_r)
    _check(got, r, TOL["bf16"])


def test_grouped_recurrent_decode():
    import paper_2605_22791_amd as g2
    d = make_grouped(3, 1, 2, 8, 128, 128, seed=149, dtype="bf16", s0_std=0.05)
    _case("grouped recurrent B3 T1 H2 Hv8")
    x = dev_inputs(d)
    S = x["S0"].clone()
    o = g2.gdr2_recurrent_step(*[x[n] for n in ARGS], S, scale=d["scale"])
    o_r, S_r = gdr2_grouped_fwd(*[d[n] for n in ARGS], d["S0"], d["scale"])
    e_o, e_s = rel_l2(host(o), o_r), rel_l2(host(S), S_r)
    print("o", e_o, "S", e_s)
    assert e_o < TOL["bf16"] and e_s < 1e-5
