"""Central finite differences of the GDR-2 loss (fp64).

TEST INFRASTRUCTURE ONLY -- see oracle/__init__.py.

The loss is the one the adjoint differentiates,
    L(inputs) = sum_t <o_t, do_t> + <S_T, dS_T>,
evaluated with a forward function supplied by the caller (the token recurrence,
or an independent reduction for the tied-gate pins).  ``fd_grad`` perturbs
every element (tiny shapes); ``fd_directional`` returns the derivative along
one direction per input (any size).
"""

import numpy as np

__all__ = ["loss", "fd_grad", "fd_directional"]


def loss(fwd, inputs, do, dS_T=None):
    o, S_T = fwd(**inputs)
    val = float(np.sum(np.asarray(o, dtype=np.float64) * do))
    if dS_T is not None:
        val += float(np.sum(S_T * dS_T))
    return val


def fd_grad(fwd, inputs, name, do, dS_T=None, h=1e-6):
    """Full central-difference gradient of L w.r.t. ``inputs[name]``."""
    base = {kk: np.array(vv, dtype=np.float64) if vv is not None else None for kk, vv in inputs.items()}
    x = base[name]
    grad = np.zeros_like(x)
    flat = x.reshape(-1)
    gflat = grad.reshape(-1)
    for i in range(flat.size):
        old = flat[i]
        flat[i] = old + h
        lp = loss(fwd, base, do, dS_T)
        flat[i] = old - h
        lm = loss(fwd, base, do, dS_T)
        flat[i] = old
        gflat[i] = (lp - lm) / (2 * h)
    return grad


def fd_directional(fwd, inputs, direction, do, dS_T=None, h=1e-5):
    """(L(x + h d) - L(x - h d)) / 2h for a dict ``direction`` of perturbations."""
    plus = {}
    minus = {}
    for kk, vv in inputs.items():
        if vv is None:
            plus[kk] = minus[kk] = None
            continue
        x = np.asarray(vv, dtype=np.float64)
        d = direction.get(kk)
        plus[kk] = x if d is None else x + h * d
        minus[kk] = x if d is None else x - h * d
    return (loss(fwd, plus, do, dS_T) - loss(fwd, minus, do, dS_T)) / (2 * h)
