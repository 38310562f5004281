"""Pins of the forward oracle against what the paper and mathematics fix.

Every check compares the oracle with something other than itself: closed
forms, independent textbook recurrences, brute-force transition products or
structural identities.  CPU only.
"""

import numpy as np
import pytest

from oracle import gdr2_recurrent_fwd, gdr2_chunk_fwd_ref, gdr2_step_states, limits, brute
from tests.helpers import rel_l2, small_problem


def _fwd(d, **kw):
    return gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"],
                              d["S0"], d["scale"], **kw)


@pytest.mark.parametrize("C,T", [(16, 64), (32, 96), (64, 128), (16, 50), (64, 100)])
def test_P1_chunk_equals_token(C, T):
    """App. A chunk form (WY) == token recurrence, incl. a ragged last chunk."""
    d = small_problem(2, T, 2, 16, 12, seed=10 + C + T)
    o_ref, S_ref = _fwd(d)
    o, S = gdr2_chunk_fwd_ref(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"],
                              d["S0"], d["scale"], C=C)
    assert rel_l2(o, o_ref) < 1e-12
    assert rel_l2(S, S_ref) < 1e-12


def test_P1_chunk_size_is_free():
    """C is a free parameter of the chunk algebra: C in {8,16,32,64} agree."""
    d = small_problem(1, 128, 2, 8, 8, seed=3)
    outs = [gdr2_chunk_fwd_ref(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"],
                               d["S0"], d["scale"], C=C)[0] for C in (8, 16, 32, 64)]
    for o in outs[1:]:
        assert rel_l2(o, outs[0]) < 1e-12


def test_P2_brute_force_transition_products():
    """Dense products of M_t = (I - k e^T) Diag(alpha) on tiny inputs."""
    d = small_problem(1, 12, 2, 4, 3, seed=5)
    o_ref, S_ref = _fwd(d)
    o, S = brute.gdr2_brute_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"],
                                d["S0"], d["scale"])
    assert rel_l2(o, o_ref) < 1e-12
    assert rel_l2(S, S_ref) < 1e-12


def test_P3_tied_gates_reduce_to_KDA():
    """b = beta*1, w = beta*1 gives KDA (Sec. 3.1; App. A.5)."""
    d = small_problem(1, 40, 2, 8, 6, seed=7, gates="tied")
    o, S = _fwd(d)
    o_k, S_k = limits.kda_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["beta"], d["S0"], d["scale"])
    assert rel_l2(o, o_k) < 1e-12
    assert rel_l2(S, S_k) < 1e-12


def test_P3_tied_gates_and_scalar_decay_reduce_to_GDN():
    """Tying the decay to a scalar as well gives Gated DeltaNet."""
    d = small_problem(1, 40, 2, 8, 6, seed=8, gates="tied", decay="scalar")
    o, S = _fwd(d)
    o_g, S_g = limits.gdn_fwd(d["q"], d["k"], d["v"], d["log_alpha_scalar"], d["beta"],
                              d["S0"], d["scale"])
    assert rel_l2(o, o_g) < 1e-12
    assert rel_l2(S, S_g) < 1e-12


def test_P3_untied_gates_differ_from_KDA():
    """Control: with untied channel gates the KDA recurrence is NOT reproduced."""
    d = small_problem(1, 40, 2, 8, 6, seed=9)
    o, _ = _fwd(d)
    beta = d["b"].mean(axis=-1)
    o_k, _ = limits.kda_fwd(d["q"], d["k"], d["v"], d["log_alpha"], beta, d["S0"], d["scale"])
    assert rel_l2(o, o_k) > 1e-3


def test_P4_no_edit_no_decay_is_linear_attention():
    """b=0, w=1, g=0: O = scale*((Q K^T . M) V + Q S0) (eq. eq_linear_attention_parallel)."""
    d = small_problem(2, 30, 2, 6, 5, seed=11)
    z = np.zeros_like(d["b"])
    o, _ = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], np.zeros_like(d["log_alpha"]), z,
                              np.ones_like(d["w"]), d["S0"], d["scale"])
    o_ref = limits.linear_attention_parallel(d["q"], d["k"], d["v"], d["S0"], d["scale"])
    assert rel_l2(o, o_ref) < 1e-12


def test_P5_no_edit_scalar_decay_is_mamba2():
    """b=0, w=1, scalar g: read factor gamma_t/gamma_s (eq. eq_mamba2_recurrence)."""
    d = small_problem(1, 30, 2, 6, 5, seed=12, decay="scalar")
    o, _ = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], np.zeros_like(d["b"]),
                              np.ones_like(d["w"]), d["S0"], d["scale"])
    o_ref = limits.mamba2_parallel(d["q"], d["k"], d["v"], d["log_alpha_scalar"], d["S0"], d["scale"])
    assert rel_l2(o, o_ref) < 1e-12


def test_P6_pure_decay():
    """b=0, w=0: o_t = scale * (gamma_t * q_t)^T S0 with channel-wise gamma."""
    d = small_problem(1, 25, 2, 6, 5, seed=13)
    o, _ = gdr2_recurrent_fwd(d["q"], d["k"], d["v"], d["log_alpha"], np.zeros_like(d["b"]),
                              np.zeros_like(d["w"]), d["S0"], d["scale"])
    o_ref = limits.pure_decay_readout(d["q"], d["log_alpha"], d["S0"], d["scale"])
    assert rel_l2(o, o_ref) < 1e-12


def test_P7_unit_key_read_after_write():
    """||k||=1: S_t^T k_t = Sbar^T((1-b)*k) + w*v; b=w=1 overwrites: S_t^T k_t = v_t."""
    d = small_problem(1, 20, 1, 8, 5, seed=14)
    k64 = d["k"].astype(np.float64)
    d["k"] = k64 / np.linalg.norm(k64, axis=-1, keepdims=True)   # exactly unit in fp64
    S_all, Sbar_all = gdr2_step_states(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"])
    for t in range(20):
        kt, bt, wt, vt = (np.asarray(d[n][0, t, 0], dtype=np.float64) for n in ("k", "b", "w", "v"))
        lhs = S_all[t + 1][0, 0].T @ kt
        rhs = Sbar_all[t][0, 0].T @ ((1 - bt) * kt) + wt * vt
        assert rel_l2(lhs, rhs) < 1e-12
    ones_b, ones_w = np.ones_like(d["b"]), np.ones_like(d["w"])
    S_all, _ = gdr2_step_states(d["q"], d["k"], d["v"], d["log_alpha"], ones_b, ones_w, d["S0"])
    for t in range(20):
        assert rel_l2(S_all[t + 1][0, 0].T @ d["k"][0, t, 0], d["v"][0, t, 0]) < 1e-12


def test_P8_state_minimises_online_objective():
    """S_t is the minimiser of ||S - Sbar||^2 - 2 <S^T k, z - Sbar^T e>
    (eq. eq_gdn2_online_objective): the objective is quadratic with Hessian 2I,
    so L(S_t + eps*D) - L(S_t) = eps^2 ||D||^2 for every D."""
    d = small_problem(1, 10, 1, 6, 4, seed=15)
    S_all, Sbar_all = gdr2_step_states(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"])
    rng = np.random.default_rng(0)
    for t in range(10):
        kt = d["k"][0, t, 0].astype(np.float64)
        e = d["b"][0, t, 0].astype(np.float64) * kt
        z = d["w"][0, t, 0].astype(np.float64) * d["v"][0, t, 0]
        Sb = Sbar_all[t][0, 0]
        St = S_all[t + 1][0, 0]

        def L(S):
            return np.sum((S - Sb) ** 2) - 2 * np.dot(S.T @ kt, z - Sb.T @ e)

        for eps in (1e-1, 1.0):
            D = rng.standard_normal(St.shape)
            assert abs(L(St + eps * D) - L(St) - eps ** 2 * np.sum(D * D)) < 1e-10 * (1 + eps ** 2 * np.sum(D * D))


def test_P9_state_passing():
    """Splitting the sequence and passing S_T as the next S0 equals one call."""
    d = small_problem(1, 96, 2, 8, 8, seed=16)
    o, S = _fwd(d)
    sl1 = {n: d[n][:, :40] for n in ("q", "k", "v", "log_alpha", "b", "w")}
    sl2 = {n: d[n][:, 40:] for n in ("q", "k", "v", "log_alpha", "b", "w")}
    o1, S1 = gdr2_recurrent_fwd(sl1["q"], sl1["k"], sl1["v"], sl1["log_alpha"], sl1["b"], sl1["w"], d["S0"], d["scale"])
    o2, S2 = gdr2_chunk_fwd_ref(sl2["q"], sl2["k"], sl2["v"], sl2["log_alpha"], sl2["b"], sl2["w"], S1, d["scale"], C=16)
    assert rel_l2(np.concatenate([o1, o2], axis=1), o) < 1e-12
    assert rel_l2(S2, S) < 1e-12


def test_P10_joint_linearity_in_S0_and_v():
    """o and S_T are linear in (S0, v) jointly: additive and homogeneous."""
    d1 = small_problem(1, 30, 2, 6, 5, seed=17)
    d2 = small_problem(1, 30, 2, 6, 5, seed=18)
    for dd in (d1, d2):
        dd["v"] = dd["v"].astype(np.float64)
        dd["S0"] = dd["S0"].astype(np.float64)
    args = lambda v, S0: (d1["q"], d1["k"], v, d1["log_alpha"], d1["b"], d1["w"], S0, d1["scale"])
    oa, Sa = gdr2_recurrent_fwd(*args(d1["v"], d1["S0"]))
    ob, Sb = gdr2_recurrent_fwd(*args(d2["v"], d2["S0"]))
    oab, Sab = gdr2_recurrent_fwd(*args(d1["v"] + 3.0 * d2["v"], d1["S0"] + 3.0 * d2["S0"]))
    assert rel_l2(oab, oa + 3.0 * ob) < 1e-12
    assert rel_l2(Sab, Sa + 3.0 * Sb) < 1e-12


def test_chunk_internals_wy_identities():
    """A (I+T) = I; the row recurrences of App. A.4 for Y and U; and the
    prefix-state lemma of App. A.2 against the normalised token states."""
    d = small_problem(1, 32, 1, 8, 6, seed=19)
    C = 32
    o, S, it = gdr2_chunk_fwd_ref(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"],
                                  d["S0"], d["scale"], C=C, keep=True)
    A, T, Y, U, G = it["A"][0, 0, 0], it["T"][0, 0, 0], it["Y"][0, 0, 0], it["U"][0, 0, 0], it["G"][0, 0, 0]
    assert np.abs(A @ (np.eye(C) + T) - np.eye(C)).max() < 1e-12
    gam = np.exp(G)
    K = d["k"][0, :, 0].astype(np.float64)
    Ebar = gam * d["b"][0, :, 0] * K
    Kbar = K / gam
    Z = d["w"][0, :, 0].astype(np.float64) * d["v"][0, :, 0]
    for r in range(C):   # eq. eq_app_y_row / eq_app_u_row
        yr = Ebar[r] - sum(np.dot(Ebar[r], Kbar[s]) * Y[s] for s in range(r))
        ur = Z[r] - sum(np.dot(Ebar[r], Kbar[s]) * U[s] for s in range(r))
        assert rel_l2(Y[r], yr) < 1e-12 and rel_l2(U[r], ur) < 1e-12
    R = it["R"][0, 0, 0]
    S0 = d["S0"][0, 0].astype(np.float64)
    S_all, _ = gdr2_step_states(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"])
    for r in range(1, C + 1):  # eq. eq_app_prefix_state: Shat_r = S0 + Kbar_{<=r}^T R_{<=r}
        Shat = S0 + Kbar[:r].T @ R[:r]
        assert rel_l2(gam[r - 1][:, None] * Shat, S_all[r][0, 0]) < 1e-11


def test_P11_packed_batch_restarts_at_boundaries():
    """App. C.6: a packed batch resets the state at every sequence boundary.
    Each sequence's outputs equal the dense transition-product form run on its
    tokens alone (brute force, an independent path), changing one sequence's
    tokens leaves the others untouched, and an empty sequence passes S0 through."""
    from oracle import gdr2_packed_fwd
    lengths = [7, 0, 12, 1]
    cu = np.concatenate([[0], np.cumsum(lengths)])
    d = small_problem(1, int(cu[-1]), 2, 5, 4, seed=19)
    rng = np.random.default_rng(3)
    S0 = rng.standard_normal((len(lengths), 2, 5, 4))
    args = lambda dd: (dd["q"], dd["k"], dd["v"], dd["log_alpha"], dd["b"], dd["w"])
    o, ST = gdr2_packed_fwd(*args(d), cu, S0, d["scale"])
    for s, L in enumerate(lengths):
        a, e = int(cu[s]), int(cu[s + 1])
        if L == 0:
            assert np.array_equal(ST[s], S0[s])
            continue
        sl = [x[:, a:e] for x in args(d)]
        ob, Sb = brute.gdr2_brute_fwd(*sl, S0[s:s + 1], d["scale"])
        assert rel_l2(o[:, a:e], ob) < 1e-12 and rel_l2(ST[s], Sb[0]) < 1e-12
    d2 = {n: np.array(x, copy=True) for n, x in d.items() if isinstance(x, np.ndarray)}
    d2.update(scale=d["scale"])
    for n in ("q", "k", "v", "log_alpha", "b", "w"):
        d2[n][:, :7] = rng.standard_normal(d2[n][:, :7].shape) * 0.3 - (0.5 if n == "log_alpha" else 0.0)
    o2, ST2 = gdr2_packed_fwd(*args(d2), cu, S0, d["scale"])
    assert not np.allclose(o2[:, :7], o[:, :7])
    assert np.array_equal(o2[:, 7:], o[:, 7:]) and np.array_equal(ST2[1:], ST[1:])


def test_P12_negative_eigenvalue_reflection_preserves_the_state_norm():
    """Sec. 3.1, negative-eigenvalue range b in [0, 2]: with b = 2, unit keys, no
    decay (g = 0) and no write (w = 0) every step applies I - 2 k k^T, a Householder
    reflection, so the Frobenius norm of the state is preserved exactly and two
    equal consecutive keys undo each other."""
    d = small_problem(1, 40, 2, 6, 5, seed=29)
    k = d["k"].astype(np.float64)
    d["k"] = k / np.linalg.norm(k, axis=-1, keepdims=True)   # unit in fp64
    d["b"] = np.full_like(d["b"], 2.0)
    d["log_alpha"] = np.zeros_like(d["log_alpha"])
    d["w"] = np.zeros_like(d["w"])
    S0 = d["S0"].astype(np.float64)
    _, S = _fwd(d)
    assert np.allclose(np.linalg.norm(S, axis=(-2, -1)), np.linalg.norm(S0, axis=(-2, -1)), rtol=1e-12)
    d["k"][:, 1] = d["k"][:, 0]
    d2 = {n: (x[:, :2] if isinstance(x, np.ndarray) and x.ndim == 4 and x.shape[1] == 40 else x) for n, x in d.items()}
    _, S2 = _fwd(d2)
    assert rel_l2(S2, S0) < 1e-12


def test_P13_scalar_erase_gate_is_KDA_with_rescaled_values():
    """Table 5's scalar-erase mode, b = beta 1 with a channel-wise w: the update
    (I - beta k k^T) D S + k (w . v)^T is KDA's (I - beta k k^T) D S + beta k v'^T
    with v' = (w . v) / beta, so the oracle must equal the independent KDA
    recurrence run on v'."""
    d = small_problem(2, 40, 2, 8, 6, seed=12)
    beta = d["b"].mean(axis=-1)
    d["b"] = np.ascontiguousarray(np.broadcast_to(beta[..., None], d["b"].shape))
    o, S = _fwd(d)
    v_kda = d["w"].astype(np.float64) * d["v"] / beta[..., None]
    o_k, S_k = limits.kda_fwd(d["q"], d["k"], v_kda, d["log_alpha"], beta, d["S0"], d["scale"])
    assert rel_l2(o, o_k) < 1e-12
    assert rel_l2(S, S_k) < 1e-12


def test_P13_scalar_write_gate_against_brute_force():
    """Table 5's scalar-write mode, a channel-wise b with w = omega 1: the oracle
    against explicit transition products (the write becomes omega k v^T)."""
    d = small_problem(1, 12, 2, 4, 3, seed=13)
    omega = d["w"].mean(axis=-1)
    d["w"] = np.ascontiguousarray(np.broadcast_to(omega[..., None], d["w"].shape))
    o, S = _fwd(d)
    o_b, S_b = brute.gdr2_brute_fwd(d["q"], d["k"], d["v"], d["log_alpha"], d["b"], d["w"], d["S0"], d["scale"])
    assert rel_l2(o, o_b) < 1e-12
    assert rel_l2(S, S_b) < 1e-12
