"""GPU parity of the recurrent (decode) kernel and the chunk -> decode hand-off."""

import numpy as np
import pytest

from oracle import gdr2_recurrent_fwd
from paper_2605_22791_amd.inputs import make_inputs, decode_inputs
from tests.helpers import rel_l2
from tests.gpu_common import dev_inputs, host, heads, pick

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-5, "bf16": 2e-3}


def _case(msg):
    print(f"\n[gpu case] {msg}", flush=True)


@pytest.mark.parametrize("Dk,Dv,dtype,T", [(128, 128, "fp32", 50), (64, 128, "bf16", 33),
                                           (128, 64, "fp32", 7), (64, 64, "bf16", 1)])
def test_recurrent_multi_token(Dk, Dv, dtype, T):
    import paper_2605_22791_amd as g2
    d = make_inputs(3, T, 2, Dk, Dv, seed=70 + T, dtype=dtype, s0_std=0.05)
    _case(f"recurrent T={T} Dk{Dk} Dv{Dv} {dtype}")
    x = dev_inputs(d)
    S = x["S0"].clone()
    o = g2.gdr2_recurrent_step(x["q"], x["k"], x["v"], x["log_alpha"], x["b"], x["w"], S, scale=d["scale"])
    o_ref, S_ref = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"], d["scale"])
    assert rel_l2(host(o), o_ref) < TOL[dtype]
    assert rel_l2(host(S), S_ref) < TOL[dtype] / 4


def test_decode_steps_config4_shape_sampled():
    """B=256, H=16, d=128, one token per call, 32 consecutive calls; oracle on 4 heads."""
    import torch
    import paper_2605_22791_amd as g2
    steps = 32
    dd = decode_inputs(steps)
    full = dd["full"]
    _case("decode B256 H16 d128, 32 steps")
    S = torch.zeros((256, 16, 128, 128), dtype=torch.float32, device="cuda")
    outs = []
    xs = {n: torch.from_numpy(dd[n]).cuda().to(torch.bfloat16 if n != "log_alpha" else torch.float32)
          for n in ("q", "k", "v", "log_alpha", "b", "w")}
    for t in range(steps):
        o = g2.gdr2_recurrent_step(*[xs[n][t] for n in ("q", "k", "v", "log_alpha", "b", "w")], S,
                                   scale=dd["scale"])
        outs.append(host(o))
    o_all = np.concatenate(outs, axis=1)          # (B, steps, H, D)
    pairs = [(0, 0), (255, 15), (100, 7), (31, 3)]
    sub = heads(full, pairs)
    o_ref, S_ref = gdr2_recurrent_fwd(sub["q"], sub["k"], sub["v"], sub["log_alpha"], sub["b"], sub["w"],
                                      None, dd["scale"])
    ro = rel_l2(pick(o_all, pairs), o_ref)
    rs = rel_l2(pick(host(S), pairs, state=True), S_ref)
    print("rel o", ro, "S", rs)
    assert ro < TOL["bf16"] and rs < TOL["bf16"]


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_chunk_then_decode_handoff(dtype):
    """chunk_fwd over a 256-token prompt, then 8 recurrent steps == oracle over 264 tokens."""
    import paper_2605_22791_amd as g2
    d = make_inputs(2, 264, 2, 128, 128, seed=80, dtype=dtype, s0_std=0.05)
    _case(f"chunk->decode hand-off {dtype}")
    x = dev_inputs(d)
    pre = [x[n][:, :256].contiguous() for n in ("q", "k", "v", "log_alpha", "b", "w")]
    o1, S = g2.gdr2_chunk_fwd(*pre, x["S0"], scale=d["scale"])
    outs = [host(o1)]
    for t in range(256, 264):
        step = [x[n][:, t:t + 1].contiguous() for n in ("q", "k", "v", "log_alpha", "b", "w")]
        outs.append(host(g2.gdr2_recurrent_step(*step, S, scale=d["scale"])))
    o_ref, S_ref = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"], d["scale"])
    assert rel_l2(np.concatenate(outs, axis=1), o_ref) < TOL[dtype]
    assert rel_l2(host(S), S_ref) < TOL[dtype]
