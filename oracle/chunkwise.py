"""Chunkwise WY form of GDR-2 (App. A) and its backward (App. B), fp64 numpy.

TEST INFRASTRUCTURE ONLY -- see oracle/__init__.py.

This is the paper's chunk algebra written out plainly, one (batch, head, chunk)
at a time, with no blocking, fusion or reordering beyond what the equations
state.  It exists for two reasons: the pins check that it equals the token
recurrence (so the chunk equations are read correctly), and the GPU tests
compare per-kernel intermediates (A, Y, U, A_qk, chunk states ...) with it.

Forward, per chunk with start state S0 (App. A):
    G_r   = sum_{i<=r} g_i,  gamma_r = exp(G_r)               eq_app_gamma
    Kbar  = K / gamma,  Ebar = gamma * (B * K),  Z = W * V     eq_app_gate_matrices
    T     = tril(Ebar Kbar^T, -1),  A = (I + T)^{-1}           eq_app_wy_definitions
    Y     = A Ebar,  U = A Z                                   eq_app_wy_definitions
    R     = U - Y S0                                           eq_app_residual_matrix
    S_C   = Diag(gamma_C) S0 + Ktail^T R,
            Ktail_r = (gamma_C / gamma_r) * k_r                eq_app_chunk_state / eq_app_ktail
    O     = Qg S0 + Aqk R,  Qg_r = gamma_r * q_r,
            Aqk_rs = 1[r>=s] q_r^T Diag(gamma_r/gamma_s) k_s   eq_app_chunk_output / eq_app_aqk
The output is multiplied by ``scale`` (1 in the paper's notation).

Backward, per chunk in reverse chunk order (App. B, Sec. B.1-B.5), with the
upstream dO (already multiplied by ``scale``) and dS_C (gradient of the chunk's
end state; dS_T for the last chunk, the next chunk's dS0 otherwise).  One
reading is added where the paper is silent: the accumulated d gamma_C is added
to row C of d gamma before dG = d gamma * gamma (gamma_C *is* that row).
"""

import numpy as np
from scipy.linalg import solve_triangular

__all__ = ["gdr2_chunk_fwd_ref", "gdr2_chunk_bwd_ref"]


def _chunk_bounds(T, C):
    return [(s, min(s + C, T)) for s in range(0, T, C)]


def _chunk_prep(Q, K, V, Gl, Bg, W):
    """Per-chunk quantities of App. A (all float64, rows = tokens of the chunk)."""
    G = np.cumsum(Gl, axis=0)                          # eq_app_gamma
    gam = np.exp(G)
    Kbar = K / gam                                     # eq_app_gate_matrices
    Ebar = gam * (Bg * K)
    Z = W * V
    L = Ebar.shape[0]
    T = np.tril(Ebar @ Kbar.T, -1)                     # eq_app_wy_definitions
    A = solve_triangular(np.eye(L) + T, np.eye(L), lower=True, unit_diagonal=True)
    Y = A @ Ebar
    U = A @ Z
    Qg = gam * Q                                       # eq_app_chunk_output
    Ktail = (gam[-1] / gam) * K                        # eq_app_ktail
    Aqk = np.tril(Qg @ Kbar.T)                         # eq_app_aqk (diagonal included)
    return dict(G=G, gam=gam, Kbar=Kbar, Ebar=Ebar, Z=Z, T=T, A=A, Y=Y, U=U,
                Qg=Qg, Ktail=Ktail, Aqk=Aqk)


def gdr2_chunk_fwd_ref(q, k, v, g, b, w, S0=None, scale=1.0, C=64, keep=False):
    """Chunkwise forward.  Returns (o, S_T) or (o, S_T, inter) with ``keep``.

    ``inter`` maps names to arrays of shape (B, H, NT, ...): G, T, A, Y, U, Qg,
    Ktail, Aqk, gC (= gamma_C), h (state at the start of each chunk), R.
    A ragged last chunk (T % C != 0) is handled with its true length; with
    ``keep`` T must be a multiple of C so the arrays stack.
    """
    q, k, v, g, b, w = [np.asarray(x, dtype=np.float64) for x in (q, k, v, g, b, w)]
    B, T, H, Dk = k.shape
    Dv = v.shape[-1]
    o = np.zeros((B, T, H, Dv))
    S_T = np.zeros((B, H, Dk, Dv))
    names = ["G", "T", "A", "Y", "U", "Qg", "Ktail", "Aqk", "gC", "h", "R"]
    inter = {n: [[None] * H for _ in range(B)] for n in names} if keep else None
    for bi in range(B):
        for hi in range(H):
            S = np.zeros((Dk, Dv)) if S0 is None else np.array(S0[bi, hi], dtype=np.float64)
            rec = {n: [] for n in names} if keep else None
            for (t0, t1) in _chunk_bounds(T, C):
                sl = slice(t0, t1)
                c = _chunk_prep(q[bi, sl, hi], k[bi, sl, hi], v[bi, sl, hi],
                                g[bi, sl, hi], b[bi, sl, hi], w[bi, sl, hi])
                R = c["U"] - c["Y"] @ S                               # eq_app_residual_matrix
                o[bi, sl, hi] = scale * (c["Qg"] @ S + c["Aqk"] @ R)  # eq_app_chunk_output
                if keep:
                    for n in ["G", "T", "A", "Y", "U", "Qg", "Ktail", "Aqk"]:
                        rec[n].append(c[n])
                    rec["gC"].append(c["gam"][-1])
                    rec["h"].append(S)
                    rec["R"].append(R)
                S = c["gam"][-1][:, None] * S + c["Ktail"].T @ R      # eq_app_chunk_state
            S_T[bi, hi] = S
            if keep:
                for n in names:
                    inter[n][bi][hi] = np.stack(rec[n])
    if keep:
        inter = {n: np.stack([np.stack(inter[n][bi]) for bi in range(B)]) for n in names}
        return o, S_T, inter
    return o, S_T


def gdr2_chunk_bwd_ref(q, k, v, g, b, w, S0, do, dS_T=None, scale=1.0, C=64,
                       mutation=None):
    """Chunkwise backward of App. B.  Returns the same dict as the adjoint.

    ``mutation="scalar_post_scale"`` deliberately plants the shortcut that App.
    B.6 shows to be invalid for untied gates: dA is accumulated against the
    ungated V and gamma*K and then post-multiplied by one scalar per column
    (the channel mean of w_s, resp. b_s).  It is only used to prove that the
    finite-difference pin has the power to catch that mistake.
    """
    q, k, v, g, b, w, do = [np.asarray(x, dtype=np.float64) for x in (q, k, v, g, b, w, do)]
    B, T, H, Dk = k.shape
    Dv = v.shape[-1]
    out = {n: np.zeros_like(x) for n, x in
           [("dq", q), ("dk", k), ("dv", v), ("dg", g), ("db", b), ("dw", w)]}
    dS0_all = np.zeros((B, H, Dk, Dv))
    bounds = _chunk_bounds(T, C)
    for bi in range(B):
        for hi in range(H):
            # forward sweep: chunk start states
            S = np.zeros((Dk, Dv)) if S0 is None else np.array(S0[bi, hi], dtype=np.float64)
            starts = []
            preps = []
            for (t0, t1) in bounds:
                sl = slice(t0, t1)
                c = _chunk_prep(q[bi, sl, hi], k[bi, sl, hi], v[bi, sl, hi],
                                g[bi, sl, hi], b[bi, sl, hi], w[bi, sl, hi])
                starts.append(S)
                preps.append(c)
                R = c["U"] - c["Y"] @ S
                S = c["gam"][-1][:, None] * S + c["Ktail"].T @ R
            dSC = np.zeros((Dk, Dv)) if dS_T is None else np.array(dS_T[bi, hi], dtype=np.float64)
            for ci in range(len(bounds) - 1, -1, -1):
                t0, t1 = bounds[ci]
                sl = slice(t0, t1)
                c = preps[ci]
                Sst = starts[ci]
                Kc, Vc, Qc = k[bi, sl, hi], v[bi, sl, hi], q[bi, sl, hi]
                Bc, Wc = b[bi, sl, hi], w[bi, sl, hi]
                dO = scale * do[bi, sl, hi]
                gam, gC = c["gam"], c["gam"][-1]
                A, Z, Ebar, Kbar = c["A"], c["Z"], c["Ebar"], c["Kbar"]
                Qg, Ktail, Aqk, Y, U = c["Qg"], c["Ktail"], c["Aqk"], c["Y"], c["U"]
                R = U - Y @ Sst                                 # eq_app_bwd_R
                # B.1 output path
                dAqk = np.tril(dO @ R.T)                        # eq_app_daqk_from_output (causal mask)
                dR = Aqk.T @ dO                                 # eq_app_dR_from_output
                dQg = dO @ Sst.T                                # eq_app_dQg_from_output
                dS0 = Qg.T @ dO                                 # eq_app_dS_from_output
                # B.1 state path
                dR += Ktail @ dSC                               # eq_app_dR_from_state
                dKtail = R @ dSC.T                              # eq_app_dKtail_from_state
                dS0 += gC[:, None] * dSC                        # eq_app_dS_from_state
                dgC = np.sum(dSC * Sst, axis=1)                 # eq_app_dgammaC_from_state
                # B.1 residual
                dU = dR                                         # eq_app_dU_from_R
                dY = -dR @ Sst.T                                # eq_app_dY_from_R
                dS0 += -Y.T @ dR                                # eq_app_dS_from_R
                # B.2 gate-aware WY inverse path
                if mutation == "scalar_post_scale":
                    wbar = Wc.mean(axis=1)
                    bbar = Bc.mean(axis=1)
                    dA = (dU @ Vc.T) * wbar[None, :] + (dY @ (gam * Kc).T) * bbar[None, :]
                else:
                    dA = dU @ Z.T + dY @ Ebar.T                 # eq_app_bwd_U / eq_app_bwd_Y
                dZ = A.T @ dU
                dEbar = A.T @ dY
                dT = -np.tril(A.T @ dA @ A.T, -1)               # eq_app_dT
                dEbar += dT @ Kbar                              # eq_app_dE_from_T
                dKbar = dT.T @ Ebar                             # eq_app_dKbar_from_T
                # B.3 scores and tail keys
                dQg += dAqk @ Kbar                              # eq_app_dQg_from_scores
                dKbar += dAqk.T @ Qg                            # eq_app_dKbar_from_scores
                dKbar += dKtail * gC[None, :]                   # eq_app_dKbar_from_tail
                dgC += np.sum(dKtail * Kbar, axis=0)            # eq_app_dgammaC_from_tail
                # B.4 elementwise gates and cumulative decay
                out["dw"][bi, sl, hi] = dZ * Vc                 # eq_app_dW_dV
                out["dv"][bi, sl, hi] = dZ * Wc
                out["db"][bi, sl, hi] = dEbar * gam * Kc        # eq_app_dB_from_E
                dK = dEbar * gam * Bc                           # eq_app_dK_from_E
                dgam = dEbar * Bc * Kc                          # eq_app_dgamma_from_E
                dK += dKbar / gam                               # eq_app_dK_from_Kbar
                dgam += -dKbar * Kc / gam ** 2                  # eq_app_dgamma_from_Kbar
                out["dq"][bi, sl, hi] = dQg * gam               # eq_app_dQ_from_Qg
                dgam += dQg * Qc                                # eq_app_dgamma_from_Qg
                out["dk"][bi, sl, hi] = dK
                dgam[-1] += dgC                                 # gamma_C is row C of gamma
                dG = dgam * gam                                 # eq_app_dg_reverse_cumsum
                out["dg"][bi, sl, hi] = np.cumsum(dG[::-1], axis=0)[::-1]
                dSC = dS0
            dS0_all[bi, hi] = dSC
    out["dS0"] = dS0_all
    return out
