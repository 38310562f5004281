"""Small numeric helpers shared by the tests (no operator arithmetic)."""

import numpy as np


def rel_l2(x, ref):
    """||x - ref||_2 / ||ref||_2 in float64 (0 when both are zero)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref.ravel())
    num = np.linalg.norm((x - ref).ravel())
    if den == 0.0:
        return num
    return num / den


def small_problem(B, T, H, Dk, Dv, seed, s0=True, dST=False, gates="channel",
                  decay="channel", decay_shift=0.0):
    """fp64-friendly random problem for oracle pins (float32 draws, no rounding)."""
    from paper_2605_22791_amd.inputs import make_inputs
    d = make_inputs(B, T, H, Dk, Dv, seed=seed, dtype="fp32", decay_shift=decay_shift,
                    s0_std=0.5 if s0 else 0.0, gates=gates, decay=decay, with_dST=dST)
    return d
