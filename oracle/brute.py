"""Brute-force GDR-2 through explicit per-token transition matrices (fp64).

TEST INFRASTRUCTURE ONLY -- see oracle/__init__.py.

Eq. eq_gdn2_recurrence written as an affine map S_t = M_t S_{t-1} + k_t z_t^T
with the dense d_k x d_k transition M_t = (I - k_t (b_t*k_t)^T) Diag(alpha_t).
Unrolling gives, for every t,
    S_t = (M_t ... M_1) S_0 + sum_{s<=t} (M_t ... M_{s+1}) k_s z_s^T ,
and o_t = scale * S_t^T q_t.  The products are formed explicitly (O(T^2 d^3)),
so this is for tiny shapes only (d <= 8, T <= 32).
"""

import numpy as np

__all__ = ["gdr2_brute_fwd"]


def gdr2_brute_fwd(q, k, v, g, b, w, S0=None, scale=1.0):
    q, k, v, g, b, w = [np.asarray(x, dtype=np.float64) for x in (q, k, v, g, b, w)]
    B, T, H, Dk = k.shape
    Dv = v.shape[-1]
    o = np.zeros((B, T, H, Dv))
    S_T = np.zeros((B, H, Dk, Dv))
    I = np.eye(Dk)
    for bi in range(B):
        for hi in range(H):
            S0h = np.zeros((Dk, Dv)) if S0 is None else np.array(S0[bi, hi], dtype=np.float64)
            M = []
            W = []
            for t in range(T):
                kt = k[bi, t, hi][:, None]
                et = (b[bi, t, hi] * k[bi, t, hi])[:, None]
                M.append((I - kt @ et.T) @ np.diag(np.exp(g[bi, t, hi])))
                W.append(kt @ (w[bi, t, hi] * v[bi, t, hi])[None, :])
            for t in range(T):
                # P(t, s) = M_t M_{t-1} ... M_{s+1}; P(t, t) = I
                St = np.zeros((Dk, Dv))
                for s in range(-1, t + 1):
                    P = I.copy()
                    for j in range(t, s, -1):
                        P = P @ M[j]
                    St = St + (P @ S0h if s == -1 else P @ W[s])
                o[bi, t, hi] = scale * (St.T @ q[bi, t, hi])
                if t == T - 1:
                    S_T[bi, hi] = St
    return o, S_T
