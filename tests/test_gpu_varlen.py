"""GPU parity of packed variable-length batches and of partial last chunks (App. C.6).

A packed batch lays its sequences end to end along T; the operator chunks each
sequence on its own, so the state restarts at every boundary and the result
for sequence s is the recurrence (Sec. 3.1) over its tokens alone, from its own
S0.  The oracle is exactly that: the fp64 token recurrence and its adjoint run
per sequence.  Lengths mix empty sequences, single tokens, exact multiples of
the chunk and ragged tails.  Tolerances as elsewhere (rel-L2 2e-3 bf16, 1e-5 fp32).
"""

import numpy as np
import pytest

from oracle import gdr2_packed_bwd, gdr2_packed_fwd, gdr2_recurrent_bwd, gdr2_recurrent_fwd
from paper_2605_22791_amd.inputs import make_inputs, make_packed
from tests.helpers import rel_l2
from tests.gpu_common import dev_inputs, host, ws_layout_bf16

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-5, "bf16": 2e-3}
GRADS = ("dq", "dk", "dv", "dlog_alpha", "db", "dw")
REF = {"dlog_alpha": "dg"}


def _case(msg):
    print(f"\n[gpu case] {msg}", flush=True)


def oracle_packed(d, backward=True):
    """The oracle's packed batch (App. C.6): the fp64 recurrence and adjoint per sequence."""
    args = [d[n] for n in ("q", "k", "v", "log_alpha", "b", "w")]
    o, ST = gdr2_packed_fwd(*args, d["cu_seqlens"], d["S0"], d["scale"])
    out = {"o": o, "S_T": ST}
    if backward:
        g = gdr2_packed_bwd(*args, d["cu_seqlens"], d["S0"], d["do"], d.get("dST"), d["scale"])
        out.update({n: g[REF.get(n, n)] for n in GRADS})
        out["dS0"] = g["dS0"]
    return out


def _run_packed(d, save=False):
    import torch
    import paper_2605_22791_amd as g2
    x = dev_inputs(d)
    cu = torch.from_numpy(d["cu_seqlens"]).cuda()
    args = [x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")]
    ws = None
    if save:
        prob = g2._problem(x["q"], x["v"], d["scale"])
        ws = torch.empty(g2.gdr2_varlen_workspace_bytes(prob, len(d["lengths"]), 1), dtype=torch.uint8,
                         device="cuda")
    o, ST = g2.gdr2_chunk_fwd_varlen(*args, cu, x["S0"], scale=d["scale"], ws=ws, save=save)
    g = g2.gdr2_chunk_bwd_varlen(*args, cu, x["S0"], x["do"], x["dST"], scale=d["scale"], ws=ws, saved=save)
    out = {"o": host(o), "S_T": host(ST)}
    out.update({n: host(t) for n, t in g.items()})
    return out


def _compare(got, ref, tol):
    err = {n: rel_l2(got[n], ref[n]) for n in ("o", "S_T", "dS0") + GRADS}
    print({k: f"{v:.2e}" for k, v in err.items()})
    for k, v in err.items():
        assert v < tol, (k, v)


LENGTHS = [100, 64, 1, 0, 257, 130, 63, 65]


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("Dk,Dv", [(128, 128), (64, 128), (128, 64)])
def test_packed_batch_matches_per_sequence_oracle(dtype, Dk, Dv):
    d = make_packed(LENGTHS, 2, Dk, Dv, seed=120 + Dk + Dv, dtype=dtype, decay_shift=-1.0, s0_std=0.05,
                    with_dST=True)
    _case(f"packed {dtype} lengths {LENGTHS} H2 Dk{Dk} Dv{Dv}")
    _compare(_run_packed(d), oracle_packed(d), TOL[dtype])


def test_packed_saved_path_and_many_sequences():
    """40 sequences of 0..300 tokens, H = 4: the stored training path returns
    the same as the recomputing one, and both match the oracle."""
    rng = np.random.default_rng(7)
    lengths = [int(x) for x in rng.integers(0, 301, size=40)]
    d = make_packed(lengths, 4, 128, 128, seed=125, dtype="bf16", decay_shift=-2.0, s0_std=0.05, with_dST=True)
    _case(f"packed bf16, 40 sequences, T = {sum(lengths)}, H4, saved vs recompute")
    got_s = _run_packed(d, save=True)
    got_r = _run_packed(d)
    for n in got_r:
        assert np.array_equal(got_s[n], got_r[n]), n
    _compare(got_r, oracle_packed(d), TOL["bf16"])


def test_packed_equals_separate_calls():
    """Each sequence of a packed batch gives exactly what a fixed-length call on
    its tokens alone gives (same chunking from the sequence start)."""
    import torch
    import paper_2605_22791_amd as g2
    lengths = [130, 64, 7, 200]
    d = make_packed(lengths, 2, 128, 128, seed=126, dtype="bf16", s0_std=0.05, with_dST=True)
    _case(f"packed vs separate fixed-length calls, lengths {lengths}")
    got = _run_packed(d)
    cu = d["cu_seqlens"]
    for s in range(len(lengths)):
        a, b = int(cu[s]), int(cu[s + 1])
        ds = {n: (d[n][:, a:b] if d[n] is not None else None) for n in ("q", "k", "v", "log_alpha", "b", "w", "do")}
        ds.update(S0=d["S0"][s:s + 1], dST=d["dST"][s:s + 1], dtype="bf16", scale=d["scale"])
        x = dev_inputs(ds)
        args = [x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")]
        o, ST = g2.gdr2_chunk_fwd(*args, x["S0"], scale=d["scale"])
        g = g2.gdr2_chunk_bwd(*args, x["S0"], x["do"], x["dST"], scale=d["scale"])
        torch.cuda.synchronize()
        assert np.array_equal(host(o), got["o"][:, a:b]), s
        assert np.array_equal(host(ST)[0], got["S_T"][s]), s
        assert np.array_equal(host(g["dS0"])[0], got["dS0"][s]), s
        for n in GRADS:
            assert np.array_equal(host(g[n]), got[n][:, a:b]), (s, n)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_fixed_length_partial_last_chunk(dtype):
    """T = 100 and T = 65: the last chunk of every sequence is partial."""
    import paper_2605_22791_amd as g2
    for T in (100, 65):
        d = make_inputs(2, T, 2, 128, 128, seed=127 + T, dtype=dtype, s0_std=0.05, with_dST=True)
        _case(f"fixed-length {dtype} B2 T{T} H2")
        x = dev_inputs(d)
        args = [x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")]
        o, ST = g2.gdr2_chunk_fwd(*args, x["S0"], scale=d["scale"])
        g = g2.gdr2_chunk_bwd(*args, x["S0"], x["do"], x["dST"], scale=d["scale"])
        o_ref, S_ref = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"],
                                          d["scale"])
        ref = gdr2_recurrent_bwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"], d["do"],
                                 d["dST"], d["scale"])
        err = {"o": rel_l2(host(o), o_ref), "S_T": rel_l2(host(ST), S_ref), "dS0": rel_l2(host(g["dS0"]), ref["dS0"])}
        for n in GRADS:
            err[n] = rel_l2(host(g[n]), ref[REF.get(n, n)])
        print({k: f"{v:.2e}" for k, v in err.items()})
        for k, v in err.items():
            assert v < TOL[dtype], (T, k, v)


def test_recurrent_varlen_matches_oracle():
    import torch
    import paper_2605_22791_amd as g2
    lengths = [5, 0, 1, 17]
    d = make_packed(lengths, 3, 64, 128, seed=128, dtype="bf16", s0_std=0.05)
    _case(f"recurrent packed lengths {lengths}")
    x = dev_inputs(d)
    cu = torch.from_numpy(d["cu_seqlens"]).cuda()
    S = x["S0"].clone()
    o = g2.gdr2_recurrent_varlen(*[x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")], cu, S,
                                 scale=d["scale"])
    ref = oracle_packed(d, backward=False)
    e_o, e_s = rel_l2(host(o), ref["o"]), rel_l2(host(S), ref["S_T"])
    print("o", e_o, "S", e_s)
    assert e_o < TOL["bf16"] and e_s < 1e-5


def test_chunk_table_in_workspace():
    """The device chunk table: every sequence cut into ceil(L/64) chunks from its
    own first token, the last one holding the remainder; empty sequences none;
    the scans take the sequences longest first."""
    import torch
    import paper_2605_22791_amd as g2
    lengths = [100, 0, 64, 1, 129]
    d = make_packed(lengths, 2, 64, 64, seed=129, dtype="bf16")
    x = dev_inputs(d)
    cu = torch.from_numpy(d["cu_seqlens"]).cuda()
    prob = g2._problem(x["q"], x["v"], d["scale"])
    T, N = sum(lengths), len(lengths)
    lay, total, _ = ws_layout_bf16(1, T, 2, 64, 64, bwd=False, nseq=N)
    assert total == g2.gdr2_varlen_workspace_bytes(prob, N, 0)
    ws = torch.zeros(total, dtype=torch.uint8, device="cuda")
    _case("varlen chunk table")
    g2.gdr2_chunk_fwd_varlen(*[x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")], cu, None, scale=d["scale"],
                             ws=ws)
    torch.cuda.synchronize()
    raw = ws.cpu().numpy()
    region = lambda n: raw[lay[n][0]: lay[n][0] + lay[n][1]].view(np.int32)
    coff, ct0, clen = region("coff"), region("ct0"), region("clen")
    exp_off, exp_t0, exp_len = [0], [], []
    for s, L in enumerate(lengths):
        for j in range(-(-L // 64)):
            exp_t0.append(int(d["cu_seqlens"][s]) + 64 * j)
            exp_len.append(min(64, L - 64 * j))
        exp_off.append(len(exp_t0))
    assert list(coff) == exp_off
    assert list(ct0[:len(exp_t0)]) == exp_t0 and list(clen[:len(exp_len)]) == exp_len
    # scan order: a permutation of the sequences by non-increasing chunk count
    order = list(region("sorder"))
    counts = [exp_off[s + 1] - exp_off[s] for s in range(N)]
    assert sorted(order) == list(range(N))
    assert all(counts[order[i]] >= counts[order[i + 1]] for i in range(N - 1))
