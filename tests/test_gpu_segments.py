"""GPU parity of the sequence-parallel state scans (bf16 path).

When a problem has few (sequence, value-slice) scans and long sequences, the
library cuts every sequence into segments: per-segment maps S_end = M S_start + N
(identity start with no input gives M, zero start gives N), a chain over the
segments, and a rescan of every segment from its true start state; the reverse
scan of the backward does the same from the segment ends.  These cases pick
shapes that switch the mode on (with a ragged last segment) and compare the
outputs, the final state, every gradient and the chunk states left in the
workspace with the fp64 oracle (rel-L2 2e-3, the bf16 bound).
"""

import numpy as np
import pytest

from oracle import gdr2_recurrent_bwd, gdr2_recurrent_fwd
from oracle.chunkwise import gdr2_chunk_fwd_ref
from paper_2605_22791_amd.inputs import make_inputs
from tests.helpers import rel_l2
from tests.gpu_common import dev_inputs, host, scan_segments, seg_buffer_bytes, ws_layout_bf16, CH, \
    decode_states_f16

pytestmark = pytest.mark.gpu

TOL = 2e-3
GRADS = ("dq", "dk", "dv", "dlog_alpha", "db", "dw", "dS0")
REF = {"dlog_alpha": "dg"}


def _case(msg):
    print(f"\n[gpu case] {msg}", flush=True)


def _fwd_bwd(d, ws=None, save=False):
    import paper_2605_22791_amd as g2
    x = dev_inputs(d)
    args = [x[n] for n in ("q", "k", "v", "log_alpha", "b", "w")]
    o, ST = g2.gdr2_chunk_fwd(*args, x["S0"], scale=d["scale"], ws=ws, save=save)
    g = g2.gdr2_chunk_bwd(*args, x["S0"], x["do"], x["dST"], scale=d["scale"], ws=ws, saved=save)
    return host(o), host(ST), {n: host(t) for n, t in g.items()}


def _check(d, o, ST, g):
    o_ref, S_ref = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"],
                                      d["scale"])
    ref = gdr2_recurrent_bwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"], d["do"],
                             d["dST"], d["scale"])
    err = {"o": rel_l2(o, o_ref), "S_T": rel_l2(ST, S_ref)}
    for n in GRADS:
        err[n] = rel_l2(g[n], ref[REF.get(n, n)])
    print({k: f"{v:.2e}" for k, v in err.items()})
    for k, v in err.items():
        assert v < TOL, (k, v)


@pytest.mark.parametrize("Dk,Dv", [(128, 128), (64, 128), (128, 64), (64, 64)])
def test_segmented_scans_match_oracle(Dk, Dv):
    # 50 chunks per head: 4 segments of 13, 13, 13 and 11 chunks
    B, T, H = 1, 3200, 2
    nseg, seg_len = scan_segments(B, T, H, Dv)
    assert (nseg, seg_len) == (4, 13)
    with_state = Dk != 64 or Dv != 64   # the (64, 64) case starts and ends at zero
    d = make_inputs(B, T, H, Dk, Dv, seed=90 + Dk + Dv, dtype="bf16", decay_shift=-2.0,
                    s0_std=0.05 if with_state else 0.0, with_dST=with_state)
    _case(f"segmented scans B{B} H{H} T{T} Dk{Dk} Dv{Dv} nseg {nseg}")
    _check(d, *_fwd_bwd(d))


def test_segmented_saved_path_and_chunk_states():
    """Saving forward + saved backward under segmentation: bit-identical to the
    recomputing backward, and the chunk-start states it leaves in the workspace
    (the rescan's states across segment boundaries) match the oracle's."""
    import torch
    import paper_2605_22791_amd as g2
    B, T, H, Dk, Dv = 1, 2048, 2, 128, 128
    nseg, seg_len = scan_segments(B, T, H, Dv)
    assert nseg == 4 and seg_len == 8
    d = make_inputs(B, T, H, Dk, Dv, seed=95, dtype="bf16", decay_shift=-3.0, s0_std=0.05, with_dST=True)
    x = dev_inputs(d)
    prob = g2._problem(x["q"], x["v"], d["scale"])
    lay, total, NC = ws_layout_bf16(B, T, H, Dk, Dv, bwd=True)
    nbytes = g2.gdr2_chunk_workspace_bytes(prob, 1)
    assert nbytes == total + seg_buffer_bytes(B, T, H, Dk, Dv)
    ws = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")
    _case(f"segmented saved path B{B} H{H} T{T} nseg {nseg}")
    o_s, S_s, g_s = _fwd_bwd(d, ws=ws, save=True)
    torch.cuda.synchronize()
    off, per = lay["Hs"]
    soff, sper = lay["Hsc"]
    NT = T // CH
    raw = ws.cpu().numpy()
    Hs = decode_states_f16(raw[off:off + NC * per], raw[soff:soff + NC * sper], NC, Dk, Dv).reshape(B, H, NT, Dk, Dv)
    _, _, it = gdr2_chunk_fwd_ref(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"],
                                  d["scale"], C=CH, keep=True)
    err_h = rel_l2(Hs, it["h"])
    print("chunk states rel", f"{err_h:.2e}")
    # the copies are fp16 with one power-of-two scale per 16 x 32 block that puts
    # the block's largest value in [2^14, 2^15): 11 significant bits each, about
    # 1.5e-4 rel-L2 over the states; a scale off by 2^k would show as 2^k times that
    assert err_h < 4e-4
    o_r, S_r, g_r = _fwd_bwd(d)
    assert np.array_equal(o_s, o_r) and np.array_equal(S_s, S_r)
    for n in GRADS:
        assert np.array_equal(g_s[n], g_r[n]), n
    _check(d, o_s, S_s, g_s)
