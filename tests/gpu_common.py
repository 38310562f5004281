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


# --------------------------------------------------------------------------- bf16 path workspace
def bf16_bits_to_f32(u16):
    """uint16 bfloat16 bit patterns -> float32 (exact)."""
    return (u16.astype(np.uint32) << 16).view(np.float32)


def ws_layout_bf16(B, T, H, Dk, Dv, bwd=False, nseq=0, G=1):
    """Byte offsets / per-chunk-head sizes of the bf16 workspace regions
    (mirrors WsBf16 in the library: fragment-ordered tiles; the backward adds
    the chunk states Hs and dH (fp16, with fp32 scales Hsc, DHsc per 16 x 32
    block) and R (fp16 fragment blocks with scales Rsc), then dR and A as
    fragment blocks).  A
    packed call (nseq > 0) has H * (T // 64 + nseq) chunk-heads and appends
    its chunk table (int32: nseq + 1 offsets, two slot arrays, the scan order).
    H counts value heads; with G value heads per key head the key-side tiles
    (all but U and the backward's states, R, dH, dR) exist once per key head."""
    NC = H * (T // CH + nseq) if nseq > 0 else B * H * (-(-T // CH))
    gc = (Dk * 4 + 255) // 256 * 256
    key = {"Y", "Qg", "Aqk", "KtT", "GC", "Am", "Amsc"}
    sizes = [("Y", 4 * (Dk // 32) * 1024), ("Qg", 4 * (Dk // 32) * 2048), ("Aqk", 8 * 2048),
             ("KtT", (Dk // 16) * 2 * 2048), ("U", (Dv // 16) * 4 * 1024), ("GC", gc)]
    if bwd:
        hsc = (Dk // 16) * (Dv // 32) * 4
        rsc = 4 * (Dv // 32) * 4
        sizes += [("Hs", Dk * Dv * 2), ("Hsc", hsc), ("Rs", CH * Dv * 2), ("Rsc", rsc), ("DH", Dk * Dv * 2),
                  ("DHsc", hsc),
                  ("DR", (Dv // 16) * 4 * 1024), ("Am", 16 * 512), ("Amsc", 16 * 4)]
    off, out = 0, {}
    for n, per in sizes:
        out[n] = (off, per)
        off += ((NC // G if n in key else NC) * per + 255) // 256 * 256
    if nseq > 0:
        slots = T // CH + nseq
        for n, cnt in (("coff", nseq + 1), ("ct0", slots), ("clen", slots), ("sorder", nseq)):
            out[n] = (off, cnt * 4)
            off += (cnt * 4 + 255) // 256 * 256
    return out, off, NC


def _frag_index(permuted):
    """(lane, e) -> (row, key) inside one 16 x 32 fragment block."""
    lane = np.arange(64)[:, None]
    e = np.arange(8)[None, :]
    row = np.broadcast_to(lane % 16, (64, 8))
    if permuted:
        key = np.where(e < 4, 4 * (lane // 16) + e, 16 + 4 * (lane // 16) + (e - 4))
    else:
        key = 8 * (lane // 16) + e
    return row, np.broadcast_to(key, (64, 8))


def decode_frag_blocks(raw_u16, nrb, nkb, split, permuted):
    """raw bf16 bits of one chunk-head region -> dense (16 nrb, 32 nkb) matrix
    (hi + lo when split)."""
    planes = 2 if split else 1
    blocks = raw_u16.reshape(nrb, nkb, planes, 64, 8)
    vals = bf16_bits_to_f32(blocks).astype(np.float64)
    vals = vals.sum(axis=2) if split else vals[:, :, 0]
    row, key = _frag_index(permuted)
    out = np.zeros((16 * nrb, 32 * nkb))
    for rb in range(nrb):
        for kb in range(nkb):
            out[16 * rb + row, 32 * kb + key] = vals[rb, kb]
    return out


def decode_tiles_f16(raw_f16, raw_scales, ncb, nrb):
    """fp16 16 x 16 blocks [column block ncb][row block nrb] with one scale each
    -> dense (16 nrb, 16 ncb) float64; lane l of a block holds column l % 16 and
    rows 4 (l // 16) + e, e < 4."""
    vals = raw_f16.view(np.float16).astype(np.float64).reshape(ncb, nrb, 64, 4)
    sc = raw_scales.view(np.float32).astype(np.float64).reshape(ncb, nrb)
    lane = np.arange(64)[:, None]
    e = np.arange(4)[None, :]
    col = np.broadcast_to(lane % 16, (64, 4))
    row = np.broadcast_to(4 * (lane // 16) + e, (64, 4))
    out = np.zeros((16 * nrb, 16 * ncb))
    for cb in range(ncb):
        for rb in range(nrb):
            out[16 * rb + row, 16 * cb + col] = vals[cb, rb] * sc[cb, rb]
    return out


def decode_tiles_split(raw_u16, ncb, nrb):
    """split bf16 16 x 16 blocks [column block ncb][row block nrb] (hi 256 values,
    then lo) -> dense (16 nrb, 16 ncb) float64, lanes as in decode_tiles_f16."""
    vals = bf16_bits_to_f32(raw_u16.view(np.uint16).reshape(ncb, nrb, 2, 64, 4)).astype(np.float64).sum(axis=2)
    lane = np.arange(64)[:, None]
    e = np.arange(4)[None, :]
    col = np.broadcast_to(lane % 16, (64, 4))
    row = np.broadcast_to(4 * (lane // 16) + e, (64, 4))
    out = np.zeros((16 * nrb, 16 * ncb))
    for cb in range(ncb):
        for rb in range(nrb):
            out[16 * rb + row, 16 * cb + col] = vals[cb, rb]
    return out


def round_tiles_f16(x):
    """x rounded as the fp16 block copies round it: per 16 x 16 block a power of
    two maps the largest magnitude m = f 2^e (f in [0.5, 1)) to [2^14, 2^15)
    (exponent 15 - e, clamped to +-120; 1 for m = 0), then fp16."""
    out = np.empty_like(x, dtype=np.float64)
    for r0 in range(0, x.shape[0], 16):
        for c0 in range(0, x.shape[1], 16):
            blk = x[r0:r0 + 16, c0:c0 + 16].astype(np.float64)
            m = np.abs(blk).max()
            sh = 0 if m == 0 else int(np.clip(15 - np.frexp(m)[1], -120, 120))
            out[r0:r0 + 16, c0:c0 + 16] = np.ldexp(np.ldexp(blk, sh).astype(np.float16).astype(np.float64), -sh)
    return out


def decode_u_tiles(raw_f32, Dv):
    """fp32 accumulator tiles [Dv/16][4] x (64 lanes x 4) -> dense (64, Dv)."""
    t = raw_f32.reshape(Dv // 16, 4, 64, 4)
    lane = np.arange(64)
    out = np.zeros((64, Dv))
    for vb in range(Dv // 16):
        for i in range(4):
            for u in range(4):
                out[16 * i + 4 * (lane // 16) + u, 16 * vb + lane % 16] = t[vb, i, :, u]
    return out


# --------------------------------------------------------------------------- sequence-parallel scans
def scan_segments(B, T, H, Dv, dtype="bf16"):
    """(nseg, seg_len) the library picks for its state scans (mirrors its rule:
    bf16 problems with fewer than 128 (sequence, 64-wide value slice) scans and
    at least 16 chunks double the segments while the grid stays within 256
    workgroups and a segment keeps 8 chunks or more)."""
    NT = T // CH
    slices = B * H * (Dv // 64)
    n = 1
    if dtype == "bf16" and slices < 128 and NT >= 16:
        while slices * n * 2 <= 256 and n * 2 * 8 <= NT:
            n *= 2
    seg_len = -(-NT // n)
    return -(-NT // seg_len), seg_len


def seg_buffer_bytes(B, T, H, Dk, Dv, dtype="bf16"):
    """Workspace bytes of the segment maps M, N and entry states X (0 if unsegmented)."""
    nseg, _ = scan_segments(B, T, H, Dv, dtype)
    if nseg == 1:
        return 0
    r = lambda n: (n * 4 + 255) // 256 * 256
    nvs = B * H * nseg
    return r(nvs * Dk * Dk) + 2 * r(nvs * Dk * Dv)


def decode_states_f16(raw_f16, raw_scales, NC, Dk, Dv):
    """fp16 chunk states with their per-(16 x 32)-block scales -> (NC, Dk, Dv) float64.

    Each 32-column group is stored in the fragments' permuted order: column
    4 m + e sits at 8 m + e and column 16 + 4 m + e at 8 m + 4 + e (e < 4)."""
    c = np.arange(Dv)
    pos = (c & ~31) + 8 * ((c & 15) >> 2) + 4 * ((c >> 4) & 1) + (c & 3)
    h = raw_f16.view(np.float16).astype(np.float64).reshape(NC, Dk, Dv)[:, :, pos]
    sc = raw_scales.view(np.float32).astype(np.float64).reshape(NC, Dk // 16, Dv // 32)
    return h * np.repeat(np.repeat(sc, 16, axis=1), 32, axis=2)
