"""GPU check of the allocation-free forward (gdr2_chunk_fwd_noalloc) through
the C ABI: two calls in a row on the library's fixed per-GPU array, the second
on a smaller problem, each against gdr2_chunk_fwd with a workspace of its own.
Both run the same kernels on the same workspace layout, so o and S_T must be
bit-identical; they are also held to the oracle's bound (rel-L2 2e-3, bf16).
The first call is long and narrow enough to take the sequence-parallel scan
(its segment maps live in the array too) and ends in a partial chunk."""

import numpy as np
import pytest

from oracle import gdr2_recurrent_fwd
from paper_2605_22791_amd.inputs import make_inputs
from tests.helpers import rel_l2
from tests.gpu_common import dev_inputs, host, scan_segments

pytestmark = pytest.mark.gpu

TOL = 2e-3


def _one(B, T, H, Dk, Dv, seed):
    import torch
    import paper_2605_22791_amd as g2
    print(f"\n[gpu case] noalloc forward B{B} T{T} H{H} Dk{Dk} Dv{Dv}", flush=True)
    d = make_inputs(B, T, H, Dk, Dv, seed=seed, dtype="bf16", s0_std=0.05)
    x = dev_inputs(d)
    args = [x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")]
    prob = g2._problem(x["q"], x["v"], d["scale"])
    assert g2.gdr2_chunk_workspace_bytes(prob, 0) <= g2.NOALLOC_SCRATCH_BYTES
    o = torch.full_like(x["v"], float("nan"))
    ST = torch.full((B, H, Dk, Dv), float("nan"), dtype=torch.float32, device="cuda")
    g2.gdr2_chunk_fwd_noalloc(*args, x["S0"], scale=d["scale"], o=o, S_T=ST)
    o_ref, S_ref = g2.gdr2_chunk_fwd(*args, x["S0"], scale=d["scale"])
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref) and torch.equal(ST, S_ref)
    oo, So = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"], d["scale"])
    e_o, e_s = rel_l2(host(o), oo), rel_l2(host(ST), So)
    print(f"rel o {e_o:.2e} S_T {e_s:.2e}", flush=True)
    assert e_o < TOL and e_s < TOL


def test_noalloc_forward_two_calls_second_smaller():
    assert scan_segments(1, 2100, 4, 128)[0] > 1
    _one(1, 2100, 4, 128, 128, seed=91)
    _one(2, 300, 2, 64, 64, seed=92)


def test_noalloc_rejects_a_problem_beyond_its_array():
    import torch
    import paper_2605_22791_amd as g2
    print("\n[gpu case] noalloc forward: workspace beyond the fixed array", flush=True)
    B, T, H, D = 1, 64 * 512, 1, 128
    x = {n: torch.zeros((B, T, H, D), dtype=torch.bfloat16, device="cuda") for n in ("q", "k", "v", "b", "w")}
    la = torch.zeros((B, T, H, D), dtype=torch.float32, device="cuda")
    with pytest.raises(g2.Gdr2Error) as err:
        g2.gdr2_chunk_fwd_noalloc(x["q"], x["k"], x["v"], la, x["b"], x["w"])
    assert err.value.status == g2.GDR2_EWORKSPACE
