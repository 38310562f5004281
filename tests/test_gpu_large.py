"""GPU parity at sizes past 32-bit offsets: B = 8, H = 16, T = 65536, d = 128
bf16 (8.6 M tokens per head row).  Every input and output tensor is larger
than 2 GB and the chunk-state regions of the workspace (h and dh: one
Dk x Dv state per chunk-head, 131072 chunk-heads) hold 2^31 floats each, so an
index computed in 32 bits anywhere on the path would land in the wrong place.
Inputs are drawn on the device (inputs.make_inputs_device); the last
(batch, head) pair, which has the highest offsets in every tensor, and one in
the middle are compared with the fp64 oracle run on their slice alone.
Tolerance as elsewhere: rel-L2 2e-3.
"""

import numpy as np
import pytest

from oracle import gdr2_recurrent_bwd, gdr2_recurrent_fwd
from paper_2605_22791_amd.inputs import make_inputs_device
from tests.helpers import rel_l2

pytestmark = pytest.mark.gpu

TOL = 2e-3


def test_past_32bit_offsets_sampled_heads():
    import torch
    import paper_2605_22791_amd as g2
    B, T, H, D = 8, 65536, 16, 128
    print(f"\n[gpu case] bf16 B{B} H{H} T{T} d{D}: 64-bit offsets", flush=True)
    x = make_inputs_device(B, T, H, D, D, seed=81, decay_shift=-2.0)
    args = [x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")]
    o, ST = g2.gdr2_chunk_fwd(*args, None, scale=x["scale"])
    grads = g2.gdr2_chunk_bwd(*args, None, x["do"], None, scale=x["scale"])
    torch.cuda.synchronize()
    for (bi, hi) in ((B - 1, H - 1), (3, 6)):
        def sl(t):
            return t[bi:bi + 1, :, hi:hi + 1].float().cpu().numpy().astype(np.float32)
        d = {n: sl(x[n]) for n in ("q", "k", "v", "log_alpha", "b", "w", "do")}
        o_ref, S_ref = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], None, x["scale"])
        ref = gdr2_recurrent_bwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], None, d["do"], None,
                                 x["scale"])
        err = {"o": rel_l2(sl(o), o_ref),
               "S_T": rel_l2(ST[bi:bi + 1, hi:hi + 1].cpu().numpy(), S_ref)}
        for gn, rn in (("dq", "dq"), ("dk", "dk"), ("dv", "dv"), ("dlog_alpha", "dg"), ("db", "db"), ("dw", "dw")):
            err[gn] = rel_l2(sl(grads[gn]), ref[rn])
        print((bi, hi), {k: f"{v:.2e}" for k, v in err.items()}, flush=True)
        for k, v in err.items():
            assert v < TOL, ((bi, hi), k, v)
