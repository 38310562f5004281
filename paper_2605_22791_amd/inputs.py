"""Seeded synthetic inputs for the GDR-2 operator (no operator arithmetic here).

This module only draws random numbers and shapes them the way the paper's layer
produces them; it computes nothing of the recurrence.  The tests, the bench and
the CPU oracle all consume what it returns, so both sides see identical values.

Recipe (one numpy PCG64 generator per call, ``default_rng(seed)``):
  * draws are float32 normals, in the fixed order q, k, v, log_alpha, the
    gates (b then w, or one tied beta), S0, do;
  * q and k are L2-normalised per (batch, token, head) in float32, as the layer
    does before the recurrence (App. D.2);
  * log_alpha = -softplus(N(0,1) + shift) in float32: the paper's
    -exp(a) * softplus(x + delta) with a = 0 (eq. eq_gdn2_decay_param);
  * gates = sigmoid(N(0,1)) (eq. eq_gdn2_gate_param); tied mode draws one
    beta per (batch, token, head) and broadcasts it to every channel;
  * for bf16 problems q, k, v, b, w and do are rounded to the nearest bfloat16
    (round-to-nearest-even) and kept as float32 carriers of those exact values;
    log_alpha and the states stay float32.
"""

import numpy as np

__all__ = ["bf16_round", "make_inputs", "config", "CONFIGS", "decode_inputs"]


def bf16_round(x):
    """Round float32 values to the nearest bfloat16 (ties to even); float32 out."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def _softplus(x):
    return np.logaddexp(np.float32(0), x).astype(np.float32)


def _sigmoid(x):
    return (1.0 / (1.0 + np.exp(-x))).astype(np.float32)


def _l2n(x):
    n = np.sqrt(np.sum(x * x, axis=-1, keepdims=True, dtype=np.float32))
    return (x / n).astype(np.float32)


def make_inputs(B, T, H, Dk, Dv, seed, dtype="bf16", decay_shift=0.0,
                decay="channel", gates="channel", s0_std=0.0, with_do=True,
                with_dST=False):
    """Draw one problem.  Returns a dict of float32 numpy arrays plus metadata.

    decay: "channel" (per key channel) or "scalar" (one value per token-head,
           broadcast over Dk);  gates: "channel" or "tied".
    """
    rng = np.random.default_rng(seed)
    f32 = np.float32
    q = _l2n(rng.standard_normal((B, T, H, Dk), dtype=f32))
    k = _l2n(rng.standard_normal((B, T, H, Dk), dtype=f32))
    v = rng.standard_normal((B, T, H, Dv), dtype=f32)
    if decay == "channel":
        la = -_softplus(rng.standard_normal((B, T, H, Dk), dtype=f32) + f32(decay_shift))
    elif decay == "scalar":
        la1 = -_softplus(rng.standard_normal((B, T, H, 1), dtype=f32) + f32(decay_shift))
        la = np.ascontiguousarray(np.broadcast_to(la1, (B, T, H, Dk)))
    else:
        raise ValueError(decay)
    if gates == "channel":
        b = _sigmoid(rng.standard_normal((B, T, H, Dk), dtype=f32))
        w = _sigmoid(rng.standard_normal((B, T, H, Dv), dtype=f32))
        beta = None
    elif gates == "tied":
        beta = _sigmoid(rng.standard_normal((B, T, H, 1), dtype=f32))
        if dtype == "bf16":
            beta = bf16_round(beta)
        b = np.ascontiguousarray(np.broadcast_to(beta, (B, T, H, Dk)))
        w = np.ascontiguousarray(np.broadcast_to(beta, (B, T, H, Dv)))
        beta = beta[..., 0]
    else:
        raise ValueError(gates)
    S0 = (s0_std * rng.standard_normal((B, H, Dk, Dv), dtype=f32)).astype(f32) if s0_std > 0 else None
    do = rng.standard_normal((B, T, H, Dv), dtype=f32) if with_do else None
    dST = rng.standard_normal((B, H, Dk, Dv), dtype=f32) if with_dST else None
    if dtype == "bf16":
        q, k, v, b, w = (bf16_round(x) for x in (q, k, v, b, w))
        if do is not None:
            do = bf16_round(do)
    out = dict(q=q, k=k, v=v, log_alpha=la.astype(f32), b=b, w=w, S0=S0, do=do, dST=dST,
               beta=beta, scale=float(1.0 / np.sqrt(Dk)), dtype=dtype,
               B=B, T=T, H=H, Dk=Dk, Dv=Dv)
    if decay == "scalar":
        out["log_alpha_scalar"] = out["log_alpha"][..., 0].copy()
    return out


# The five workloads (shape, precision, distributions).  Seeds: config i uses seed i.
CONFIGS = {
    0: dict(B=1, H=2, T=256, Dk=64, Dv=64, dtype="fp32", decay_shift=0.0, s0_std=0.0,
            desc="tiny fp32 forward"),
    1: dict(B=2, H=4, T=1024, Dk=128, Dv=128, dtype="bf16", decay_shift=0.0, s0_std=0.02,
            gates="tied", desc="gate-collapse check (KDA / Gated DeltaNet limits)"),
    2: dict(B=8, H=16, T=4096, Dk=128, Dv=128, dtype="bf16", decay_shift=-2.0, s0_std=0.0,
            desc="1.3B-layer training shape"),
    3: dict(B=1, H=16, T=65536, Dk=128, Dv=128, dtype="bf16", decay_shift=-4.0, s0_std=0.02,
            desc="long context"),
    4: dict(B=256, H=16, T=1, Dk=128, Dv=128, dtype="bf16", decay_shift=-2.0, s0_std=0.0,
            desc="decode, one token per call"),
}


def config(idx, decay="channel", **overrides):
    """Inputs of workload ``idx`` (config 1 takes decay="channel" or "scalar")."""
    c = dict(CONFIGS[idx])
    c.pop("desc")
    c.update(overrides)
    gates = c.pop("gates", "channel")
    return make_inputs(c.pop("B"), c.pop("T"), c.pop("H"), c.pop("Dk"), c.pop("Dv"),
                       seed=c.pop("seed", idx), gates=gates, decay=decay, **c)


def decode_inputs(steps, B=256, H=16, D=128, seed=4, decay_shift=-2.0):
    """``steps`` consecutive one-token inputs, stacked on a leading axis:
    q, k, b, log_alpha (steps, B, 1, H, D); v, w likewise (bf16-rounded)."""
    d = make_inputs(B, steps, H, D, D, seed=seed, dtype="bf16", decay_shift=decay_shift,
                    with_do=False)
    out = {}
    for n in ("q", "k", "v", "log_alpha", "b", "w"):
        x = d[n]                                   # (B, steps, H, D)
        out[n] = np.ascontiguousarray(np.moveaxis(x, 1, 0)[:, :, None])
    out["scale"] = d["scale"]
    out["full"] = d
    return out
