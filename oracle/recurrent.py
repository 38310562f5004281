"""Token-by-token GDR-2 recurrence and its reverse-time adjoint (fp64 numpy).

TEST INFRASTRUCTURE ONLY -- see oracle/__init__.py.

Forward (Sec. 3.1, eqs. eq_gdn2_e_z / eq_gdn2_residual / eq_gdn2_recurrence;
restated per token in App. A, eq. eq_app_gdn2_step).  For every (batch, head)
independently, starting from S = S0 (zeros when absent):

    a_t   = exp(g_t)                    decay, g_t the log-decay (key channels)
    Sbar  = Diag(a_t) S_{t-1}           decay first
    e_t   = b_t * k_t                   erase factor (key side)
    z_t   = w_t * v_t                   write factor (value side)
    r_t   = Sbar^T e_t                  read along the gated erase direction
    S_t   = Sbar + k_t (z_t - r_t)^T    edit
    o_t   = scale * S_t^T q_t           read-out with the post-update state

``scale`` is an explicit output scale (callers use 1/sqrt(d_k)); the paper's
o_t = S_t^T q_t is scale = 1.  It multiplies the output only.

Backward: the adjoint of the loop above for the scalar loss
    L = sum_t <o_t, do_t> + <S_T, dS_T>
derived by reversing each assignment (chain rule, one line per forward line).
It reproduces the gradient the method defines (App. B reaches the same values
in chunk form; the oracle pins compare the two and check both against central
finite differences).

Layouts follow the operator: q, k, b, g are (B, T, H, Dk); v, w, o are
(B, T, H, Dv); states are (B, H, Dk, Dv).
"""

import numpy as np

__all__ = ["gdr2_recurrent_fwd", "gdr2_recurrent_bwd", "gdr2_step_states", "gdr2_packed_fwd",
           "gdr2_packed_bwd", "gdr2_grouped_fwd", "gdr2_grouped_bwd"]


def _f64(*xs):
    return [np.asarray(x, dtype=np.float64) for x in xs]


def _shapes(k, v):
    B, T, H, Dk = k.shape
    Dv = v.shape[-1]
    return B, T, H, Dk, Dv


def _step(S, q_t, k_t, v_t, g_t, b_t, w_t):
    """One token of eq. eq_gdn2_residual for all (b, h) at once.

    Returns (S_t, Sbar, r) with S of shape (B, H, Dk, Dv).
    """
    a = np.exp(g_t)                                   # (B,H,Dk)
    Sbar = a[..., :, None] * S                        # Diag(a) S
    e = b_t * k_t                                     # (B,H,Dk)
    z = w_t * v_t                                     # (B,H,Dv)
    r = np.einsum("bhkv,bhk->bhv", Sbar, e)           # Sbar^T e
    S_new = Sbar + k_t[..., :, None] * (z - r)[..., None, :]
    return S_new, Sbar, r


def gdr2_recurrent_fwd(q, k, v, g, b, w, S0=None, scale=1.0):
    """Forward of the token recurrence.  Returns (o, S_T) in float64."""
    q, k, v, g, b, w = _f64(q, k, v, g, b, w)
    B, T, H, Dk, Dv = _shapes(k, v)
    S = np.zeros((B, H, Dk, Dv)) if S0 is None else np.array(S0, dtype=np.float64)
    o = np.empty((B, T, H, Dv))
    for t in range(T):
        S, _, _ = _step(S, q[:, t], k[:, t], v[:, t], g[:, t], b[:, t], w[:, t])
        o[:, t] = scale * np.einsum("bhkv,bhk->bhv", S, q[:, t])
    return o, S


def gdr2_step_states(q, k, v, g, b, w, S0=None):
    """All states S_0..S_T and decayed states Sbar_1..Sbar_T (small T only).

    Returns (S_all, Sbar_all) with shapes (T+1, B, H, Dk, Dv) and
    (T, B, H, Dk, Dv).  Used by the pins that inspect intermediate states.
    """
    q, k, v, g, b, w = _f64(q, k, v, g, b, w)
    B, T, H, Dk, Dv = _shapes(k, v)
    S = np.zeros((B, H, Dk, Dv)) if S0 is None else np.array(S0, dtype=np.float64)
    S_all = [S]
    Sbar_all = []
    for t in range(T):
        S, Sbar, _ = _step(S, q[:, t], k[:, t], v[:, t], g[:, t], b[:, t], w[:, t])
        S_all.append(S)
        Sbar_all.append(Sbar)
    return np.stack(S_all), np.stack(Sbar_all)


def gdr2_recurrent_bwd(q, k, v, g, b, w, S0, do, dS_T=None, scale=1.0, ckpt=64):
    """Reverse-time adjoint of ``gdr2_recurrent_fwd``.

    Returns a dict with dq, dk, dv, dg (gradient of the log-decay), db, dw and
    dS0, all float64, for L = sum_t <o_t, do_t> + <S_T, dS_T>.

    The forward states are recomputed segment by segment from checkpoints
    stored every ``ckpt`` tokens, so memory stays O(ckpt * B*H*Dk*Dv).
    """
    q, k, v, g, b, w, do = _f64(q, k, v, g, b, w, do)
    B, T, H, Dk, Dv = _shapes(k, v)
    S = np.zeros((B, H, Dk, Dv)) if S0 is None else np.array(S0, dtype=np.float64)

    # forward sweep keeping a checkpoint at the start of every segment
    starts = list(range(0, T, ckpt))
    ckpts = {}
    for t in range(T):
        if t in starts:
            ckpts[t] = S
        S, _, _ = _step(S, q[:, t], k[:, t], v[:, t], g[:, t], b[:, t], w[:, t])

    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    dg = np.zeros_like(g)
    db = np.zeros_like(b)
    dw = np.zeros_like(w)
    dS = np.zeros((B, H, Dk, Dv)) if dS_T is None else np.array(dS_T, dtype=np.float64)

    for t0 in reversed(starts):
        t1 = min(t0 + ckpt, T)
        # recompute S_{t0-1+1..t1} inside the segment; seg[i] = state before token t0+i
        seg = [ckpts[t0]]
        for t in range(t0, t1):
            Sn, _, _ = _step(seg[-1], q[:, t], k[:, t], v[:, t], g[:, t], b[:, t], w[:, t])
            seg.append(Sn)
        for t in range(t1 - 1, t0 - 1, -1):
            S_prev = seg[t - t0]
            S_t = seg[t - t0 + 1]
            q_t, k_t, v_t, g_t, b_t, w_t = q[:, t], k[:, t], v[:, t], g[:, t], b[:, t], w[:, t]
            a = np.exp(g_t)
            Sbar = a[..., :, None] * S_prev
            e = b_t * k_t
            z = w_t * v_t
            r = np.einsum("bhkv,bhk->bhv", Sbar, e)
            # o_t = scale * S_t^T q_t
            dq[:, t] = scale * np.einsum("bhkv,bhv->bhk", S_t, do[:, t])
            dS = dS + scale * q_t[..., :, None] * do[:, t][..., None, :]
            # S_t = Sbar + k (z - r)^T
            u = np.einsum("bhkv,bhk->bhv", dS, k_t)        # d(z - r)
            dk_t = np.einsum("bhkv,bhv->bhk", dS, z - r)
            dz = u
            dr = -u
            dSbar = dS.copy()
            # r = Sbar^T e
            dSbar += e[..., :, None] * dr[..., None, :]
            de = np.einsum("bhkv,bhv->bhk", Sbar, dr)
            # z = w * v ; e = b * k
            dw[:, t] = dz * v_t
            dv[:, t] = dz * w_t
            db[:, t] = de * k_t
            dk[:, t] = dk_t + de * b_t
            # Sbar = Diag(exp(g)) S_prev
            dg[:, t] = a * np.einsum("bhkv,bhkv->bhk", dSbar, S_prev)
            dS = a[..., :, None] * dSbar
    return dict(dq=dq, dk=dk, dv=dv, dg=dg, db=db, dw=dw, dS0=dS)


# ---------------------------------------------------------------------------
# Packed variable-length batches (App. C.6): B = 1 and sequence s owns tokens
# cu[s] .. cu[s+1) of the (1, T, H, D) tensors.  The state restarts at every
# boundary, so a packed batch is nothing but its sequences run one by one from
# their own start states (S0 / dS_T of shape (n_seqs, H, Dk, Dv)).

def gdr2_packed_fwd(q, k, v, g, b, w, cu_seqlens, S0=None, scale=1.0):
    """Forward of a packed batch.  Returns (o (1, T, H, Dv), S_T (n_seqs, H, Dk, Dv))."""
    q, k, v, g, b, w = _f64(q, k, v, g, b, w)
    _, T, H, Dk, Dv = _shapes(k, v)
    cu = [int(x) for x in cu_seqlens]
    N = len(cu) - 1
    S0 = np.zeros((N, H, Dk, Dv)) if S0 is None else np.asarray(S0, dtype=np.float64)
    o = np.zeros((1, T, H, Dv))
    ST = np.array(S0, dtype=np.float64)
    for s in range(N):
        a, e = cu[s], cu[s + 1]
        if e > a:
            sl = [x[:, a:e] for x in (q, k, v, g, b, w)]
            o[:, a:e], S = gdr2_recurrent_fwd(*sl, S0[s:s + 1], scale)
            ST[s] = S[0]
    return o, ST


def gdr2_packed_bwd(q, k, v, g, b, w, cu_seqlens, S0, do, dS_T=None, scale=1.0):
    """Adjoint of gdr2_packed_fwd: dict dq, dk, dv, dg, db, dw (1, T, H, .) and dS0 (n_seqs, H, Dk, Dv)."""
    q, k, v, g, b, w, do = _f64(q, k, v, g, b, w, do)
    _, T, H, Dk, Dv = _shapes(k, v)
    cu = [int(x) for x in cu_seqlens]
    N = len(cu) - 1
    S0 = np.zeros((N, H, Dk, Dv)) if S0 is None else np.asarray(S0, dtype=np.float64)
    dS_T = np.zeros((N, H, Dk, Dv)) if dS_T is None else np.asarray(dS_T, dtype=np.float64)
    out = {n: np.zeros_like(x) for n, x in (("dq", q), ("dk", k), ("dv", v), ("dg", g), ("db", b), ("dw", w))}
    out["dS0"] = np.array(dS_T, dtype=np.float64)
    for s in range(N):
        a, e = cu[s], cu[s + 1]
        if e > a:
            sl = [x[:, a:e] for x in (q, k, v, g, b, w)]
            r = gdr2_recurrent_bwd(*sl, S0[s:s + 1], do[:, a:e], dS_T[s:s + 1], scale)
            for n in ("dq", "dk", "dv", "dg", "db", "dw"):
                out[n][:, a:e] = r[n]
            out["dS0"][s] = r["dS0"][0]
    return out


# ---------------------------------------------------------------------------
# Grouped value heads (Sec. 3.5, App. C.1): with Hv = G * H value heads, q, k,
# the log-decay and b (H heads) are repeated across each group of G
# consecutive value heads (value head j uses key head j // G), while v, w, the
# outputs and the states live on the value heads.  The key-side gradients are
# therefore the sums over the group (the adjoint of the repetition).

def _repeat_keys(G, *xs):
    return [np.repeat(np.asarray(x, dtype=np.float64), G, axis=2) for x in xs]


def gdr2_grouped_fwd(q, k, v, g, b, w, S0=None, scale=1.0):
    """Forward with Hv = v.shape[2] value heads over H = q.shape[2] key heads."""
    G = np.shape(v)[2] // np.shape(q)[2]
    qe, ke, ge, be = _repeat_keys(G, q, k, g, b)
    return gdr2_recurrent_fwd(qe, ke, v, ge, be, w, S0, scale)


def gdr2_grouped_bwd(q, k, v, g, b, w, S0, do, dS_T=None, scale=1.0):
    """Adjoint of gdr2_grouped_fwd: dq, dk, dg, db on the key heads (group sums),
    dv, dw and dS0 on the value heads."""
    H, Hv = np.shape(q)[2], np.shape(v)[2]
    G = Hv // H
    qe, ke, ge, be = _repeat_keys(G, q, k, g, b)
    r = gdr2_recurrent_bwd(qe, ke, v, ge, be, w, S0, do, dS_T, scale)
    for n in ("dq", "dk", "dg", "db"):
        x = r[n]
        r[n] = x.reshape(x.shape[0], x.shape[1], H, G, x.shape[3]).sum(axis=3)
    return r
