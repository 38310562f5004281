"""Seeded synthetic inputs for the GDR-2 operator (no operator arithmetic here).

This module only draws random numbers and shapes them the way the paper's layer
produces them; it computes nothing of the recurrence.  The tests, the bench and
the CPU oracle all consume what it returns, so both sides see identical values.

Recipe (numpy PCG64 streams from ``SeedSequence(seed)``):
  * draws are float32 normals, in the fixed order q, k, v, log_alpha, the
    gates (b then w, or one tied beta), S0, do, dS_T; draw i uses child i of
    the seed's SeedSequence, and a draw of n values is cut into fixed pieces of
    2^21 values (whole rows), piece j drawn from child j of the draw's
    sequence, so the values do not depend on how many threads fill them;
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

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

__all__ = ["bf16_round", "make_inputs", "config", "CONFIGS", "decode_inputs", "make_fused"]


def bf16_round(x):
    """Round float32 values to the nearest bfloat16 (ties to even); float32 out.
    (Finite inputs: the 32-bit sum cannot overflow below the NaN range.)"""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


_PIECE = 1 << 21
_WORKERS = max(1, min(16, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else 4))


def _draw(ss, shape, post=None):
    """float32 normals of `shape` from SeedSequence `ss`, in fixed pieces of
    _PIECE values (whole rows of the last axis), each piece from its own child
    stream; `post` maps a piece (rows x last axis) to its final values."""
    n = int(np.prod(shape))
    last = shape[-1]
    piece = max(last, (_PIECE // last) * last)
    nb = -(-n // piece)
    kids = ss.spawn(nb)
    out = np.empty(n, dtype=np.float32)

    def work(j):
        lo, hi = j * piece, min(n, (j + 1) * piece)
        x = np.random.default_rng(kids[j]).standard_normal(hi - lo, dtype=np.float32)
        if post is not None:
            x = post(x.reshape(-1, last)).reshape(-1)
        out[lo:hi] = x

    if nb == 1:
        work(0)
    else:
        with ThreadPoolExecutor(min(_WORKERS, nb)) as ex:
            list(ex.map(work, range(nb)))
    return out.reshape(shape)


def _softplus(x):
    return np.logaddexp(np.float32(0), x).astype(np.float32)


def _sigmoid(x):
    return (1.0 / (1.0 + np.exp(-x))).astype(np.float32)


def _l2n(x):
    n = np.sqrt(np.einsum("...d,...d->...", x, x, dtype=np.float32))[..., None]
    return (x / n).astype(np.float32)


def make_inputs(B, T, H, Dk, Dv, seed, dtype="bf16", decay_shift=0.0,
                decay="channel", gates="channel", s0_std=0.0, with_do=True,
                with_dST=False):
    """Draw one problem.  Returns a dict of float32 numpy arrays plus metadata.

    decay: "channel" (per key channel) or "scalar" (one value per token-head,
           broadcast over Dk);  gates: "channel" or "tied".
    """
    f32 = np.float32
    kids = np.random.SeedSequence(seed).spawn(9)
    rnd = (lambda x: bf16_round(x)) if dtype == "bf16" else (lambda x: x)
    shift = f32(decay_shift)
    q = _draw(kids[0], (B, T, H, Dk), lambda x: rnd(_l2n(x)))
    k = _draw(kids[1], (B, T, H, Dk), lambda x: rnd(_l2n(x)))
    v = _draw(kids[2], (B, T, H, Dv), rnd)
    if decay == "channel":
        la = _draw(kids[3], (B, T, H, Dk), lambda x: -_softplus(x + shift))
    elif decay == "scalar":
        la1 = _draw(kids[3], (B, T, H, 1), lambda x: -_softplus(x + shift))
        la = np.ascontiguousarray(np.broadcast_to(la1, (B, T, H, Dk)))
    else:
        raise ValueError(decay)
    if gates == "channel":
        b = _draw(kids[4], (B, T, H, Dk), lambda x: rnd(_sigmoid(x)))
        w = _draw(kids[5], (B, T, H, Dv), lambda x: rnd(_sigmoid(x)))
        beta = None
    elif gates == "tied":
        beta = _draw(kids[4], (B, T, H, 1), lambda x: rnd(_sigmoid(x)))
        b = np.ascontiguousarray(np.broadcast_to(beta, (B, T, H, Dk)))
        w = np.ascontiguousarray(np.broadcast_to(beta, (B, T, H, Dv)))
        beta = beta[..., 0]
    else:
        raise ValueError(gates)
    S0 = _draw(kids[6], (B, H, Dk, Dv), lambda x: (s0_std * x).astype(f32)) if s0_std > 0 else None
    do = _draw(kids[7], (B, T, H, Dv), rnd) if with_do else None
    dST = _draw(kids[8], (B, H, Dk, Dv)) if with_dST else None
    out = dict(q=q, k=k, v=v, log_alpha=la.astype(f32), b=b, w=w, S0=S0, do=do, dST=dST,
               beta=beta, scale=float(1.0 / np.sqrt(Dk)), dtype=dtype,
               B=B, T=T, H=H, Dk=Dk, Dv=Dv)
    if decay == "scalar":
        out["log_alpha_scalar"] = out["log_alpha"][..., 0].copy()
    return out


def make_inputs_device(B, T, H, Dk, Dv, seed, decay_shift=0.0, device="cuda"):
    """make_inputs' bf16 channel-gate recipe drawn on the device with torch's
    generator, for shapes whose host copies would take tens of GB: q, k unit
    rows, v, b = sigmoid, w = sigmoid and do in bf16, log_alpha =
    -softplus(N(0,1) + decay_shift) in fp32, no S0.  Returns a dict of device
    tensors (the same distributions as make_inputs, not the same values)."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    bf = torch.bfloat16

    def normal(*shape):
        return torch.randn(shape, generator=gen, device=device, dtype=torch.float32)

    def unit_rows(x):
        return (x / torch.sqrt((x * x).sum(dim=-1, keepdim=True))).to(bf)

    out = dict(q=unit_rows(normal(B, T, H, Dk)), k=unit_rows(normal(B, T, H, Dk)),
               v=normal(B, T, H, Dv).to(bf))
    out["log_alpha"] = -torch.nn.functional.softplus(normal(B, T, H, Dk) + decay_shift)
    out["b"] = torch.sigmoid(normal(B, T, H, Dk)).to(bf)
    out["w"] = torch.sigmoid(normal(B, T, H, Dv)).to(bf)
    out["do"] = normal(B, T, H, Dv).to(bf)
    out["scale"] = float(1.0 / np.sqrt(Dk))
    return out


def make_decode_device(steps, B=256, H=16, D=128, seed=4, decay_shift=-2.0, device="cuda"):
    """Decode inputs for `steps` consecutive one-token calls, drawn on the device
    with torch's generator (make_inputs' bf16 channel-gate recipe, as in
    make_inputs_device): q, k, v, b, w bf16 and log_alpha fp32, each of shape
    (steps, B, 1, H, D), so call t takes x[t].  At B = 256 and 1024 steps every
    tensor holds 537 M values, which is why they are not drawn on the host."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    bf = torch.bfloat16
    shape = (steps, B, 1, H, D)

    def normal():
        return torch.randn(shape, generator=gen, device=device, dtype=torch.float32)

    def unit_rows(x):
        return (x / torch.sqrt((x * x).sum(dim=-1, keepdim=True))).to(bf)

    out = dict(q=unit_rows(normal()), k=unit_rows(normal()), v=normal().to(bf))
    out["log_alpha"] = -torch.nn.functional.softplus(normal() + decay_shift)
    out["b"] = torch.sigmoid(normal()).to(bf)
    out["w"] = torch.sigmoid(normal()).to(bf)
    out["scale"] = float(1.0 / np.sqrt(D))
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


def make_packed(lengths, H, Dk, Dv, seed, dtype="bf16", decay_shift=0.0, s0_std=0.0, with_dST=False):
    """A packed variable-length batch (App. C.6): sequences of the given lengths
    laid end to end along T (B = 1), drawn like make_inputs, with their offsets
    ``cu_seqlens`` (int32, len(lengths) + 1) and per-sequence start states /
    final-state gradients of shape (n_seqs, H, Dk, Dv)."""
    lengths = [int(x) for x in lengths]
    T = sum(lengths)
    if T <= 0:
        raise ValueError("a packed batch needs at least one token")
    d = make_inputs(1, T, H, Dk, Dv, seed, dtype=dtype, decay_shift=decay_shift)
    N = len(lengths)
    rng = np.random.default_rng(np.random.SeedSequence([seed, 0x9ac4ed]))
    f32 = np.float32
    d["S0"] = (s0_std * rng.standard_normal((N, H, Dk, Dv))).astype(f32) if s0_std > 0 else None
    d["dST"] = rng.standard_normal((N, H, Dk, Dv)).astype(f32) if with_dST else None
    d["cu_seqlens"] = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    d["lengths"] = lengths
    return d


def make_grouped(B, T, H, Hv, Dk, Dv, seed, dtype="bf16", decay_shift=0.0, s0_std=0.0, with_dST=False):
    """Grouped value heads (Hv = G * H): the key side (q, k, log_alpha, b) is
    drawn with H heads and the value side (v, w, do and the states) with Hv
    heads, each exactly as make_inputs draws it."""
    kd = make_inputs(B, T, H, Dk, Dv, seed, dtype=dtype, decay_shift=decay_shift)
    vd = make_inputs(B, T, Hv, Dk, Dv, seed + 7919, dtype=dtype, s0_std=s0_std, with_dST=with_dST)
    d = dict(kd)
    for n in ("v", "w", "do", "S0", "dST"):
        d[n] = vd[n]
    d["H"], d["Hv"] = H, Hv
    return d


def make_fused(B, T, H, Dk, Dv, seed, dtype="bf16", Hv=None, lengths=None, s0_std=0.0, with_dST=False):
    """Raw projections for the fused input stage (normalisation and decay
    activation in the operator): q and k as the projections leave them
    (normal, not normalised), the decay projection output f, one decay
    magnitude a per key head and one bias delta per key channel.

    Recipe (children of SeedSequence(seed), one per draw, in this order):
      q, k ~ N(0, 1)                              (B, T, H, Dk), bf16-rounded for bf16
      v ~ N(0, 1), w = sigmoid(N(0, 1))           (B, T, Hv, Dv), bf16-rounded
      f ~ N(0, 1)                                 (B, T, H, Dk), float32
      b = sigmoid(N(0, 1))                        (B, T, H, Dk), bf16-rounded
      a = log(U[1, 16])                           (H,), float32
      delta ~ U[-6.9, -2.25]                      (H, Dk), float32 (the usual range of the
                                                  decay-bias initialisation: softplus(delta) in
                                                  about [1e-3, 1e-1])
      S0 = s0_std N(0, 1), do ~ N(0, 1), dS_T ~ N(0, 1) on the value heads.
    lengths: a packed batch (B = 1, T = sum) with cu_seqlens and per-sequence
    states (n_seqs, Hv, Dk, Dv)."""
    f32 = np.float32
    Hv = H if Hv is None else Hv
    if lengths is not None:
        lengths = [int(x) for x in lengths]
        B, T = 1, sum(lengths)
        if T <= 0:
            raise ValueError("a packed batch needs at least one token")
    NS = len(lengths) if lengths is not None else B
    kids = np.random.SeedSequence(seed).spawn(11)
    rnd = (lambda x: bf16_round(x)) if dtype == "bf16" else (lambda x: x)
    q = _draw(kids[0], (B, T, H, Dk), rnd)
    k = _draw(kids[1], (B, T, H, Dk), rnd)
    v = _draw(kids[2], (B, T, Hv, Dv), rnd)
    f = _draw(kids[3], (B, T, H, Dk))
    b = _draw(kids[4], (B, T, H, Dk), lambda x: rnd(_sigmoid(x)))
    w = _draw(kids[5], (B, T, Hv, Dv), lambda x: rnd(_sigmoid(x)))
    a = np.log(np.random.default_rng(kids[6]).uniform(1.0, 16.0, size=H)).astype(f32)
    delta = np.random.default_rng(kids[7]).uniform(-6.9, -2.25, size=(H, Dk)).astype(f32)
    S0 = _draw(kids[8], (NS, Hv, Dk, Dv), lambda x: (s0_std * x).astype(f32)) if s0_std > 0 else None
    do = _draw(kids[9], (B, T, Hv, Dv), rnd)
    dST = _draw(kids[10], (NS, Hv, Dk, Dv)) if with_dST else None
    out = dict(q=q, k=k, v=v, f=f, a=a, delta=delta, b=b, w=w, S0=S0, do=do, dST=dST,
               scale=float(1.0 / np.sqrt(Dk)), dtype=dtype, B=B, T=T, H=H, Hv=Hv, Dk=Dk, Dv=Dv, eps=1e-6)
    if lengths is not None:
        out["cu_seqlens"] = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
        out["lengths"] = lengths
    return out


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
