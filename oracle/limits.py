"""Independent textbook recurrences that GDR-2 reduces to (fp64 numpy).

TEST INFRASTRUCTURE ONLY -- see oracle/__init__.py.

Each function is written from its own equation in Sec. 2 of the paper, as a
matrix product per token (not by calling the GDR-2 recurrence), so that the
tied-gate reductions of Sec. 3.1 / App. A.5 are checked against code that does
not share a line with ``oracle.recurrent``.

Shapes: q, k (B, T, H, Dk); v (B, T, H, Dv); per-token scalars (B, T, H);
channel-wise decays (B, T, H, Dk); states (B, H, Dk, Dv).
"""

import numpy as np

__all__ = ["kda_fwd", "gdn_fwd", "linear_attention_parallel", "mamba2_parallel",
           "pure_decay_readout"]


def kda_fwd(q, k, v, log_alpha, beta, S0=None, scale=1.0):
    """KDA (eq. eq_kda_recurrence): S_t = (I - beta_t k_t k_t^T) Diag(alpha_t) S_{t-1}
    + beta_t k_t v_t^T, o_t = scale * S_t^T q_t.  log_alpha (B,T,H,Dk), beta (B,T,H)."""
    q, k, v, log_alpha, beta = [np.asarray(x, dtype=np.float64) for x in (q, k, v, log_alpha, beta)]
    B, T, H, Dk = k.shape
    Dv = v.shape[-1]
    o = np.zeros((B, T, H, Dv))
    S_T = np.zeros((B, H, Dk, Dv))
    I = np.eye(Dk)
    for bi in range(B):
        for hi in range(H):
            S = np.zeros((Dk, Dv)) if S0 is None else np.array(S0[bi, hi], dtype=np.float64)
            for t in range(T):
                kt = k[bi, t, hi][:, None]
                D = np.diag(np.exp(log_alpha[bi, t, hi]))
                bt = beta[bi, t, hi]
                S = (I - bt * (kt @ kt.T)) @ D @ S + bt * kt @ v[bi, t, hi][None, :]
                o[bi, t, hi] = scale * (S.T @ q[bi, t, hi])
            S_T[bi, hi] = S
    return o, S_T


def gdn_fwd(q, k, v, log_alpha, beta, S0=None, scale=1.0):
    """Gated DeltaNet (eq. eq_gdn_recurrence): S_t = alpha_t (I - beta_t k_t k_t^T) S_{t-1}
    + beta_t k_t v_t^T with a scalar alpha_t = exp(log_alpha_t); log_alpha, beta (B,T,H)."""
    q, k, v, log_alpha, beta = [np.asarray(x, dtype=np.float64) for x in (q, k, v, log_alpha, beta)]
    B, T, H, Dk = k.shape
    Dv = v.shape[-1]
    o = np.zeros((B, T, H, Dv))
    S_T = np.zeros((B, H, Dk, Dv))
    I = np.eye(Dk)
    for bi in range(B):
        for hi in range(H):
            S = np.zeros((Dk, Dv)) if S0 is None else np.array(S0[bi, hi], dtype=np.float64)
            for t in range(T):
                kt = k[bi, t, hi][:, None]
                at = np.exp(log_alpha[bi, t, hi])
                bt = beta[bi, t, hi]
                S = at * (I - bt * (kt @ kt.T)) @ S + bt * kt @ v[bi, t, hi][None, :]
                o[bi, t, hi] = scale * (S.T @ q[bi, t, hi])
            S_T[bi, hi] = S
    return o, S_T


def linear_attention_parallel(q, k, v, S0=None, scale=1.0):
    """Causal parallel form (eq. eq_linear_attention_parallel), plus the start
    state read by every query: O = scale * ((Q K^T (.) M) V + Q S0)."""
    q, k, v = [np.asarray(x, dtype=np.float64) for x in (q, k, v)]
    B, T, H, Dk = k.shape
    Dv = v.shape[-1]
    M = np.tril(np.ones((T, T)))
    o = np.zeros((B, T, H, Dv))
    for bi in range(B):
        for hi in range(H):
            Q, K, V = q[bi, :, hi], k[bi, :, hi], v[bi, :, hi]
            O = (Q @ K.T * M) @ V
            if S0 is not None:
                O = O + Q @ S0[bi, hi]
            o[bi, :, hi] = scale * O
    return o


def mamba2_parallel(q, k, v, log_alpha, S0=None, scale=1.0):
    """Mamba-2 scalar decay (eq. eq_mamba2_recurrence) in closed form: the write
    at step s is read at step t >= s with factor gamma_t / gamma_s, and the start
    state with factor gamma_t, gamma_t = prod_{i<=t} alpha_i.  log_alpha (B,T,H)."""
    q, k, v, log_alpha = [np.asarray(x, dtype=np.float64) for x in (q, k, v, log_alpha)]
    B, T, H, Dk = k.shape
    Dv = v.shape[-1]
    o = np.zeros((B, T, H, Dv))
    for bi in range(B):
        for hi in range(H):
            Gc = np.cumsum(log_alpha[bi, :, hi])
            decay = np.exp(Gc[:, None] - Gc[None, :]) * np.tril(np.ones((T, T)))
            Q, K, V = q[bi, :, hi], k[bi, :, hi], v[bi, :, hi]
            O = ((Q @ K.T) * decay) @ V
            if S0 is not None:
                O = O + np.exp(Gc)[:, None] * (Q @ S0[bi, hi])
            o[bi, :, hi] = scale * O
    return o


def pure_decay_readout(q, log_alpha, S0, scale=1.0):
    """No erase, no write: S_t = Diag(gamma_t) S0, so o_t = scale * (gamma_t * q_t)^T S0."""
    q, log_alpha, S0 = [np.asarray(x, dtype=np.float64) for x in (q, log_alpha, S0)]
    gam = np.exp(np.cumsum(log_alpha, axis=1))            # (B,T,H,Dk)
    return scale * np.einsum("bthk,bhkv->bthv", gam * q, S0)
