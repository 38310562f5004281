"""The layer-side input stage around the operator, and its adjoint (fp64 numpy).

TEST INFRASTRUCTURE ONLY -- see oracle/__init__.py.

Two steps sit between the projections and the recurrence:

  * Query/key normalisation (App. D.2, Sec. 4.1 block design): q and k are
    L2-normalised per (token, head) before the update.  The paper gives no
    epsilon; this build reads the normalisation as
        y = x * (sum_c x_c^2 + eps)^(-1/2)
    with a small eps (1e-6 by default), which is the plain x / ||x|| for eps = 0.
    Its vector-Jacobian product (the usual one of an L2 normalisation) is, with
    r = (sum x^2 + eps)^(-1/2) and y = r x,
        dx = r * (dy - y <y, dy>),
    exact for every eps (d r / d x = -r^3 x).

  * Log-decay activation (eq. eq_gdn2_decay_param; App. C.1, eq.
    eq_app_layer_decay), formed in fp32 before the recurrence (App. D.1):
        g[b, t, h, c] = -exp(a[h]) * softplus(f[b, t, h, c] + delta[h, c])
    with f the decay projection's output, a one value per key head broadcast
    over the Dk channels, delta one bias per key channel.  Its adjoint, with
    x = f + delta and sigma the logistic function:
        df     = dg * (-exp(a) * sigma(x))
        ddelta = sum over (b, t) of df
        da[h]  = sum over (b, t, c) of dg * g

The fused operator is the recurrence of oracle/recurrent.py run on
(l2norm(q), l2norm(k), v, g, b, w); its backward is that recurrence's adjoint
followed by the two VJPs above.  The kernels take q and k in the model dtype
(App. D.3: only the state and the accumulators are fp32), so for a bf16
operator the normalised q and k are rounded to bf16 (nearest, ties to even)
before the recurrence, as the cast between an unfused normalisation and the
operator would; the rounding passes gradients through unchanged, so the VJP is
taken at the unrounded y.  Grouped value heads (Sec. 3.5) and packed
batches (App. C.6) compose the same way: the normalisation and the activation
act on the key heads, before any repetition over a group.
"""

import numpy as np

from .recurrent import (gdr2_grouped_bwd, gdr2_grouped_fwd, gdr2_packed_bwd, gdr2_packed_fwd,
                        gdr2_recurrent_bwd, gdr2_recurrent_fwd)

__all__ = ["l2norm", "l2norm_vjp", "softplus", "decay_activation", "decay_activation_vjp",
           "round_bf16", "gdr2_fused_fwd", "gdr2_fused_bwd"]


def round_bf16(x):
    """Nearest bfloat16 value of each element (ties to the even significand),
    as float64.  A bfloat16 keeps 8 significant bits: with x = m 2^e, m in
    [1, 2), the spacing is 2^(e - 7); values are rounded on that grid.  Zero,
    infinities and NaN pass through; values beyond the largest bfloat16 are
    rounded on the top binade's grid (overflow to infinity is not modelled)."""
    x = np.asarray(x, dtype=np.float64)
    out = np.array(x, dtype=np.float64)
    fin = np.isfinite(x) & (x != 0)
    e = np.floor(np.log2(np.abs(x[fin])))
    e = np.maximum(e, -126.0)  # subnormal bfloat16 share the smallest normal spacing
    step = np.exp2(e - 7.0)
    out[fin] = np.round(x[fin] / step) * step  # np.round: half to even
    return out


def l2norm(x, eps=1e-6):
    """y = x (sum x^2 + eps)^(-1/2) over the last axis (App. D.2)."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps)


def l2norm_vjp(x, dy, eps=1e-6):
    """dx = r (dy - y <y, dy>) with r = (sum x^2 + eps)^(-1/2), y = r x."""
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    r = 1.0 / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps)
    y = r * x
    return r * (dy - y * np.sum(y * dy, axis=-1, keepdims=True))


def softplus(x):
    """log(1 + e^x), written as max(x, 0) + log1p(e^-|x|) so that it neither
    overflows for large x nor loses the tiny values of very negative x."""
    x = np.asarray(x, dtype=np.float64)
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


def _sigmoid(x):
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def decay_activation(f, a, delta):
    """g = -exp(a) * softplus(f + delta): f (B, T, H, Dk), a (H,), delta (H, Dk)."""
    f = np.asarray(f, dtype=np.float64)
    A = np.exp(np.asarray(a, dtype=np.float64))[:, None]
    return -A * softplus(f + np.asarray(delta, dtype=np.float64))


def decay_activation_vjp(f, a, delta, dg):
    """(df, da, ddelta) of L = <g, dg> for g = decay_activation(f, a, delta)."""
    f = np.asarray(f, dtype=np.float64)
    dg = np.asarray(dg, dtype=np.float64)
    A = np.exp(np.asarray(a, dtype=np.float64))[:, None]
    x = f + np.asarray(delta, dtype=np.float64)
    df = dg * (-A * _sigmoid(x))
    g = -A * softplus(x)
    da = np.sum(dg * g, axis=(0, 1, 3))
    ddelta = np.sum(df, axis=(0, 1))
    return df, da, ddelta


def _stage(q, k, f, a, delta, eps, dtype):
    qn, kn = l2norm(q, eps), l2norm(k, eps)
    if dtype == "bf16":
        qn, kn = round_bf16(qn), round_bf16(kn)
    return qn, kn, decay_activation(f, a, delta)


def gdr2_fused_fwd(q, k, v, f, a, delta, b, w, S0=None, scale=1.0, eps=1e-6, cu_seqlens=None, dtype="fp64"):
    """Forward from the raw projections: (o, S_T).  q, k, f, b on H key heads;
    v, w on Hv = G H value heads; cu_seqlens (packed batch, B = 1) or None;
    dtype: the operator's q / k dtype ("bf16" rounds the normalised q, k)."""
    qn, kn, g = _stage(q, k, f, a, delta, eps, dtype)
    G = np.shape(v)[2] // np.shape(q)[2]
    if cu_seqlens is not None:
        if G > 1:
            qn, kn, g, b = [np.repeat(np.asarray(x, dtype=np.float64), G, axis=2) for x in (qn, kn, g, b)]
        return gdr2_packed_fwd(qn, kn, v, g, b, w, cu_seqlens, S0, scale)
    if G > 1:
        return gdr2_grouped_fwd(qn, kn, v, g, b, w, S0, scale)
    return gdr2_recurrent_fwd(qn, kn, v, g, b, w, S0, scale)


def gdr2_fused_bwd(q, k, v, f, a, delta, b, w, S0, do, dS_T=None, scale=1.0, eps=1e-6, cu_seqlens=None,
                   dtype="fp64"):
    """Adjoint of gdr2_fused_fwd: dict dq, dk (raw q, k), df, da, ddelta, db,
    dv, dw, dS0."""
    qn, kn, g = _stage(q, k, f, a, delta, eps, dtype)
    H, Hv = np.shape(q)[2], np.shape(v)[2]
    G = Hv // H
    if cu_seqlens is not None:
        if G > 1:
            qe, ke, ge, be = [np.repeat(np.asarray(x, dtype=np.float64), G, axis=2) for x in (qn, kn, g, b)]
            r = gdr2_packed_bwd(qe, ke, v, ge, be, w, cu_seqlens, S0, do, dS_T, scale)
            for n in ("dq", "dk", "dg", "db"):
                x = r[n]
                r[n] = x.reshape(x.shape[0], x.shape[1], H, G, x.shape[3]).sum(axis=3)
        else:
            r = gdr2_packed_bwd(qn, kn, v, g, b, w, cu_seqlens, S0, do, dS_T, scale)
    elif G > 1:
        r = gdr2_grouped_bwd(qn, kn, v, g, b, w, S0, do, dS_T, scale)
    else:
        r = gdr2_recurrent_bwd(qn, kn, v, g, b, w, S0, do, dS_T, scale)
    out = {"dq": l2norm_vjp(q, r["dq"], eps), "dk": l2norm_vjp(k, r["dk"], eps)}
    out["df"], out["da"], out["ddelta"] = decay_activation_vjp(f, a, delta, r["dg"])
    for n in ("db", "dv", "dw", "dS0"):
        out[n] = r[n]
    return out
