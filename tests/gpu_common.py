"""Helpers for the GPU parity tests (device transfer, workspace views, oracle on head subsets)."""

import numpy as np

CH = 64


def torch_mod():
    import torch
    return torch


def dev_inputs(d, device="cuda"):
    """Copy a generated problem to the device in the operator's dtypes."""
    torch = torch_mod()
    io = torch.bfloat16 if d["dtype"] == "bf16" else torch.float32
    out = {}
    for n in ("q", "k", "v", "b", "w", "do"):
        if d.get(n) is not None:
            out[n] = torch.from_numpy(np.ascontiguousarray(d[n])).to(device).to(io).contiguous()
    out["log_alpha"] = torch.from_numpy(np.ascontiguousarray(d["log_alpha"])).to(device).contiguous()
    for n in ("S0", "dST"):
        out[n] = None if d.get(n) is None else torch.from_numpy(np.ascontiguousarray(d[n])).to(device).contiguous()
    return out


def host(t):
    return None if t is None else t.detach().float().cpu().numpy().astype(np.float64)


def heads(d, pairs):
    """Restrict a problem to the listed (b, h) pairs, stacked on the batch axis."""
    sub = dict(d)
    for n in ("q", "k", "v", "log_alpha", "b", "w", "do"):
        if d.get(n) is not None:
            sub[n] = np.stack([d[n][b, :, h:h + 1] for (b, h) in pairs])
    for n in ("S0", "dST"):
        if d.get(n) is not None:
            sub[n] = np.stack([d[n][b, h:h + 1] for (b, h) in pairs])
    sub["B"], sub["H"] = len(pairs), 1
    return sub


def pick(x, pairs, state=False):
    """Same selection on a (B,T,H,D) or (B,H,Dk,Dv) result array."""
    if state:
        return np.stack([x[b, h:h + 1] for (b, h) in pairs])
    return np.stack([x[b, :, h:h + 1] for (b, h) in pairs])


def ws_layout(B, T, H, Dk, Dv, bwd):
    """Byte offsets of the workspace regions (mirrors the library's layout)."""
    NC = B * H * (T // CH)
    r = lambda nfl: (nfl * 4 + 255) // 256 * 256
    names = [("Y", NC * CH * Dk), ("U", NC * CH * Dv), ("Kt", NC * CH * Dk), ("Qg", NC * CH * Dk),
             ("Aqk", NC * CH * CH), ("GC", NC * Dk)]
    if bwd:
        names += [("Hs", NC * Dk * Dv), ("Rs", NC * CH * Dv), ("DH", NC * Dk * Dv), ("DR", NC * CH * Dv),
                  ("DAqk", NC * CH * CH), ("DT", NC * CH * CH), ("DEg", NC * CH * Dk)]
    off = 0
    out = {}
    for n, nf in names:
        out[n] = (off, nf)
        off += r(nf)
    return out, off


def ws_view(ws, lay, name, shape):
    torch = torch_mod()
    off, nf = lay[name]
    return ws[off:off + nf * 4].view(torch.float32).view(*shape)
