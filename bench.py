"""Throughput of the chunkwise GDR-2 operator (forward + gate-aware backward) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu] [--no-decode]
                    [--path stored|recompute]

One step = the forward + gate-aware backward over one batch of the 1.3B-layer
training shape (B=8, H=16, T=4096, d_k=d_v=128, bf16 inputs, fp32 log-decay
and state), inputs resident in HBM before the timed region.  The default
training path keeps the forward's A, chunk states and R for the backward
(gdr2_chunk_fwd_save + gdr2_chunk_bwd_saved); the memory-saving path, where
the backward recomputes them (gdr2_chunk_fwd + gdr2_chunk_bwd), is timed beside
it over the same number of steps.  Prints one JSON
line with tokens/s (B*T per step over the K timed steps), the roofline of the
dominant kernel (per-kernel durations from hipEvents recorded on the launch
stream during the timed steps) and the CPU oracle timed on a bounded sample.
"""

import argparse
import json
import os
import sys
import time

HBM_PEAK_GBS = 8000.0                    # MI355X HBM3E, GB/s
PEAK_TFLOPS = {"fp32": 157.3, "bf16": 2500.0}
MFMA_DTYPE = "bf16"                      # operand type of the path's products (v_mfma_f32_16x16x32_bf16)


def kernel_model(B, T, H, Dk, Dv, stored=True):
    """Algorithmic flops and HBM bytes per launch of each kernel of the bf16 path.

    stored: the forward also writes A, the chunk-start states and R for the
    backward (the saved training path); otherwise the backward recomputes them.

    Per chunk-head (C = 64 tokens of one head); a causal C x C x D product
    counts C^2 D flops (half of the dense 2 C^2 D).  Bytes are each kernel's
    inputs read once plus its outputs written once, in the dtypes they have:
    q/k/v/b/w/dO/o and their gradients bf16, log-decay and its gradient fp32,
    the fragment-ordered workspace tiles as stored (split tiles hi + lo, Y
    single bf16, U fp32), and the backward's copies of the chunk states, their
    gradients and R in fp16 with one fp32 scale per 16 x 32 block, A in fp16
    with one fp32 scale per 16 x 16 block.  Blocks that are zero by causality
    are not stored: two of A_qk's eight fragment blocks (query rows 0..31,
    keys 32..63) and A's six tiles above the diagonal, of which the chunk
    backward's copy skips the two 1 KB pieces that hold nothing else.
    """
    C = 64
    NC = B * H * (T // C)
    NT = T // C
    f, h = 4, 2
    tri, triv = C * C * Dk, C * C * Dv         # causal products
    mm = 2 * C * Dk * Dv                      # one dense (C x Dk) x (Dk x Dv) product
    solve = C ** 3 / 3
    kin, vin = C * Dk * h, C * Dv * h          # bf16 (C x D) tiles
    kf, vf = C * Dk * f, C * Dv * f            # fp32 (C x D) tiles
    st = Dk * Dv * f                          # fp32 state
    st16 = Dk * Dv * h + (Dk // 16) * (Dv // 32) * f   # fp16 state copy + scales
    r16 = C * Dv * h + (C // 16) * (Dv // 32) * f      # fp16 R + scales
    ws_y, ws_q, ws_a = C * Dk * h, C * Dk * 2 * h, C * C * 2 * h * 6 // 8
    ws_k, ws_u, ws_g = C * Dk * 2 * h, C * Dv * f, -(-Dk * f // 256) * 256
    ws_am = 10 * 16 * 16 * h + 10 * f                # fp16 A written: 10 tiles + their scales
    ws_am_rd = 6 * 1024 + (C // 16) * (C // 16) * f   # read by the chunk backward
    ws_dr = C * Dv * 2 * h                            # split bf16 dR
    seq_state = 2 * st / NT                   # S0 read + S_T write, per sequence
    m = {}
    intra_fl = tri + tri + solve + tri + triv
    intra_by = 3 * kin + kf + 2 * vin + ws_y + ws_q + ws_a + ws_k + ws_u + ws_g
    m["fwd_intra"] = (intra_fl, intra_by + (ws_am if stored else 0))
    m["fwd_state"] = (3 * mm + triv, ws_y + ws_q + ws_a + ws_k + ws_u + ws_g + vin + seq_state
                      + (st16 + r16 if stored else 0))
    m["bwd_recompute_intra"] = (intra_fl, intra_by + ws_am)
    m["bwd_recompute_state"] = (2 * mm, ws_y + ws_k + ws_u + ws_g + st / NT + st16 + r16)
    m["bwd_state"] = (triv + 3 * mm, ws_y + ws_q + ws_a + ws_k + ws_g + vin + seq_state + st16 + ws_dr)
    # dZ = A^T dR, dT = -dZ R^T, dA_qk = dO R^T (causal); dZ h^T, dO h^T, R dh^T;
    # the three decay products with dT / dA_qk (causal)
    m["bwd_intra"] = (3 * triv + 3 * mm + 4 * tri,
                      3 * kin + kf + 3 * vin + 2 * st16 + r16 + ws_dr + ws_am_rd + 3 * kin + 2 * vin + kf)
    return {k: (fl * NC, by * NC) for k, (fl, by) in m.items()}


def method_bytes(B, T, H, Dk, Dv):
    """The method's own HBM bytes per launch of each kernel of the bf16 path:
    what the kernel's step of the chunkwise algorithm must move at the least,
    with model-dtype (bf16) operands and fp32 log-decay and state, counted per
    token-head and multiplied by the B * T * H token-heads of one launch.

      fwd_intra  (Gram, solve, auxiliaries; Sec. 3.3, App. C.2): reads q, k, b,
                 v, w (bf16) and g (fp32) = 14 d, writes A_qk (bf16, C values
                 per token) and Y, U (bf16) = 2 C + 4 d          -> 2432 B at d = 128
      fwd_state  (state recurrence with the output fused): reads Y, U, K_tail
                 (bf16, 6 d), writes the chunk states (fp32, 4 d^2 / C per
                 token) and R (bf16, 2 d); the output adds Q_g, A_qk in and
                 o out (2 d + 2 C + 2 d)                         -> 2688 B
      bwd_state  (reverse state recurrence): reads Y, K_tail, Q_g, dO (bf16,
                 8 d) and A_qk (2 C), writes the chunk-state gradients (fp32,
                 4 d^2 / C) and dR (bf16, 2 d)                   -> 2432 B
      bwd_intra  (gate-aware WY VJP and intra-chunk VJP): the backward's own
                 I/O, q, k, v, b, w, dO in (bf16) and g in (fp32) = 16 d,
                 dq, dk, dv, db, dw out (bf16) and dlog_alpha out (fp32) = 14 d
                                                                  -> 3840 B
    These are the per-token figures of the flop and byte accounting of the
    chunkwise form (App. B's products and each step's operands); the
    decomposition's own stored intermediates (split planes, fp32 U and R, the
    per-chunk states read back by the chunk backward) are counted by
    kernel_model instead."""
    C = 64
    d = Dk
    per = {
        "fwd_intra": 14 * d + 2 * C + 4 * d,
        "fwd_state": 6 * d + 4 * Dk * Dv // C + 2 * Dv + (2 * d + 2 * C + 2 * Dv),
        "bwd_state": 8 * d + 2 * C + 4 * Dk * Dv // C + 2 * Dv,
        "bwd_intra": 30 * d,
    }
    per["bwd_recompute_intra"] = per["fwd_intra"]
    per["bwd_recompute_state"] = 6 * d + 4 * Dk * Dv // C + 2 * Dv
    return {k: v * B * T * H for k, v in per.items()}


KERNEL_SOURCES = {"fwd_intra": "gdr2_intra_bf16.hip", "bwd_recompute_intra": "gdr2_intra_bf16.hip",
                  "fwd_state": "gdr2_scan_bf16.hip", "bwd_recompute_state": "gdr2_scan_bf16.hip",
                  "bwd_state": "gdr2_bscan_bf16.hip", "bwd_intra": "gdr2_bchunk_bf16.hip"}
SHARED_HEADERS = ("gdr2_bf16.hpp", "gdr2_kernels.hpp", "gdr2_device.hpp")


def measured_traffic(kernel_id, table="hbm_traffic_B8H16T4096.txt"):
    """HBM bytes per launch of `kernel_id` from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary, or None when there is none or the kernel's source (with the
    shared headers) has changed since the counters were taken."""
    import hashlib
    here = os.path.dirname(os.path.abspath(__file__))
    path = os.path.join(here, "profiles", table)
    src = KERNEL_SOURCES.get(kernel_id)
    if src is None or not os.path.exists(path):
        return None
    h = hashlib.sha256()
    for f in (src,) + SHARED_HEADERS:
        with open(os.path.join(here, "paper_2605_22791_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    digest = h.hexdigest()[:12]
    with open(path) as fh:
        for line in fh:
            parts = line.split()
            if not parts or parts[0].startswith("#") or parts[0] != kernel_id:
                continue
            fetch, write, sha = int(parts[-3]), int(parts[-2]), parts[-1]
            return fetch + write if sha == digest else None
    return None


def _cpu_worker(args):
    """Oracle forward + adjoint on one head (runs in a spawned process); returns
    the two durations in seconds."""
    from oracle import gdr2_recurrent_fwd, gdr2_recurrent_bwd
    q, k, v, la, b, w, do, scale = args
    t0 = time.perf_counter()
    gdr2_recurrent_fwd(q, k, v, la, b, w, None, scale)
    t1 = time.perf_counter()
    gdr2_recurrent_bwd(q, k, v, la, b, w, None, do, None, scale)
    return t1 - t0, time.perf_counter() - t1


def cpu_baseline(d, heads_sample):
    """Time the oracle (fwd + bwd) on batch row 0, first `heads_sample` heads, full T."""
    import multiprocessing as mp
    try:
        ncores = len(os.sched_getaffinity(0))
    except AttributeError:
        ncores = os.cpu_count() or 1
    workers = max(1, min(16, ncores, heads_sample))
    jobs = [(d["q"][0:1, :, h:h + 1], d["k"][0:1, :, h:h + 1], d["v"][0:1, :, h:h + 1],
             d["log_alpha"][0:1, :, h:h + 1], d["b"][0:1, :, h:h + 1], d["w"][0:1, :, h:h + 1],
             d["do"][0:1, :, h:h + 1], d["scale"]) for h in range(heads_sample)]
    env_keep = {k: os.environ.get(k) for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")}
    for k in env_keep:
        os.environ[k] = "1"
    ctx = mp.get_context("spawn")
    with ctx.Pool(workers) as pool:
        pool.map(_cpu_worker, jobs[:1])           # warm the workers' imports
        t0 = time.perf_counter()
        parts = pool.map(_cpu_worker, jobs, chunksize=1)
        wall = time.perf_counter() - t0
    for k, v in env_keep.items():
        if v is None:
            os.environ.pop(k, None)
        else:
            os.environ[k] = v
    H = d["H"]
    tokens = d["T"] * heads_sample / H           # token = one (b, t) position across all H heads
    fwd_share = sum(p[0] for p in parts) / max(1e-12, sum(p[0] + p[1] for p in parts))
    return {"value": tokens / wall, "unit": "tokens/s", "cores": workers, "workers": workers,
            "host_cores": ncores, "kind": "oracle",
            "sample": f"fp64 numpy token recurrence + adjoint, batch row 0, {heads_sample} of {H} heads, "
                      f"T={d['T']} (= {tokens:.0f} tokens of the workload), {workers} single-threaded workers",
            "wall_s": wall, "fwd_value": tokens / (wall * fwd_share)}


def decode_bench(steps, B=256, H=16, D=128, distinct=64):
    """Decode: `steps` one-token recurrent calls on a 256 MiB fp32 state; the
    synthetic token inputs (drawn on the GPU) cycle through `distinct` sets."""
    import torch
    import paper_2605_22791_amd as g2
    gen = torch.Generator(device="cuda").manual_seed(4)
    m = min(steps, distinct)
    n = lambda *s: torch.randn(*s, device="cuda", generator=gen)
    q = torch.nn.functional.normalize(n(m, B, 1, H, D), dim=-1).bfloat16()
    k = torch.nn.functional.normalize(n(m, B, 1, H, D), dim=-1).bfloat16()
    v = n(m, B, 1, H, D).bfloat16()
    la = -torch.nn.functional.softplus(n(m, B, 1, H, D) - 2.0)
    b = torch.sigmoid(n(m, B, 1, H, D)).bfloat16()
    w = torch.sigmoid(n(m, B, 1, H, D)).bfloat16()
    S = torch.zeros(B, H, D, D, device="cuda")
    o = torch.empty(B, 1, H, D, device="cuda", dtype=torch.bfloat16)
    for t in range(min(8, m)):
        g2.gdr2_recurrent_step(q[t], k[t], v[t], la[t], b[t], w[t], S, o=o)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for t in range(steps):
        j = t % m
        g2.gdr2_recurrent_step(q[j], k[j], v[j], la[j], b[j], w[j], S, o=o)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    bytes_step = B * H * (2 * D * D * 4 + 5 * D * 2 + D * 4 + D * 2)
    out = {"steps_per_s": 1000.0 / ms, "us_per_step": ms * 1000.0, "alg_bytes_per_call": bytes_step,
           "hbm_GBs": bytes_step / (ms * 1e-3) / 1e9, "hbm_frac": bytes_step / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
           "config": {"B": B, "H": H, "d": D, "steps": steps}}
    counted = measured_decode_traffic(B)
    if counted is not None:
        out["counter_bytes_per_call"] = counted
        out["counter_GBs"] = counted / (ms * 1e-3) / 1e9
    return out


def measured_decode_traffic(B):
    """FETCH_SIZE + WRITE_SIZE bytes per decode call at batch B from the committed
    rocprofv3 summary (None when it has no row for B)."""
    here = os.path.dirname(os.path.abspath(__file__))
    path = os.path.join(here, "profiles", "recurrent_decode_B256_B512_counters.md")
    if not os.path.exists(path):
        return None
    for line in open(path):
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) >= 5 and cells[0] == str(B):
            return int((float(cells[3]) + float(cells[4])) * 1e6)
    return None


def calibration_copy(mib):
    """One copy-like elementwise kernel (torch.neg) over `mib` MiB of fp32: the
    reference that scales rocprofv3 FETCH_SIZE / WRITE_SIZE to bytes."""
    import torch
    n = mib * (1 << 20) // 4
    src_c = torch.ones(n, device="cuda")
    dst_c = torch.empty_like(src_c)
    torch.cuda.synchronize()
    torch.neg(src_c, out=dst_c)               # one elementwise kernel: n*4 bytes in, n*4 out
    torch.cuda.synchronize()
    print(f"[bench] calibration copy: {mib} MiB read + {mib} MiB written", file=sys.stderr, flush=True)
    del src_c, dst_c


def copy_bandwidth(mib=2048, reps=5):
    """Measured device copy bandwidth (read + write bytes / time) of a plain
    torch copy, reported beside the 8 TB/s spec peak."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    return 2 * n * 4 / (ms * 1e-3) / 1e9


def config3_bench(steps=3, stored=True):
    """Long-context workload (B=1, H=16, T=65536, d=128, S0 != 0): fwd+bwd step
    time, per-kernel times and the state scans' HBM fraction."""
    import torch
    import paper_2605_22791_amd as g2
    from paper_2605_22791_amd.inputs import config
    d = config(3)
    B, T, H, Dk, Dv = d["B"], d["T"], d["H"], d["Dk"], d["Dv"]
    tb = lambda x: torch.from_numpy(x).cuda().to(torch.bfloat16).contiguous()
    q, k, v, b, w, do = (tb(d[n]) for n in ("q", "k", "v", "b", "w", "do"))
    la = torch.from_numpy(d["log_alpha"]).cuda().contiguous()
    S0 = torch.from_numpy(d["S0"]).cuda().contiguous()
    del d
    prob = g2.Gdr2Problem(B, T, H, Dk, Dv, 64, Dk ** -0.5, g2.GDR2_BF16)
    ws = torch.empty(g2.gdr2_chunk_workspace_bytes(prob, 1), dtype=torch.uint8, device="cuda")

    def step():
        g2.gdr2_chunk_fwd(q, k, v, la, b, w, S0, ws=ws, save=stored)
        g2.gdr2_chunk_bwd(q, k, v, la, b, w, S0, do, None, ws=ws, saved=stored)

    step()
    torch.cuda.synchronize()
    g2.gdr2_profile_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    per_kernel = g2.gdr2_profile_collect()
    g2.gdr2_profile_enable(False)
    ms = e0.elapsed_time(e1) / steps
    mbytes = method_bytes(B, T, H, Dk, Dv)
    kern = {}
    for name, (kms, cnt) in per_kernel.items():
        if cnt:
            avg = kms / cnt
            kern[name] = {"avg_us": round(avg * 1e3, 1),
                          "hbm_frac": round(mbytes[name] / (avg * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    return {"workload": "B1 H16 T65536 d128 bf16, S0 != 0", "training_path": "stored" if stored else "recompute",
            "ms_per_step": ms, "tokens_per_s": B * T / (ms * 1e-3), "kernels": kern}


def packed_lengths(total, seed=2024, lo=64, hi=4096):
    """Sequence lengths of a packed batch: log-uniform in [lo, hi] (documents up
    to the 4K training context), drawn until `total` tokens are used (the last
    one takes the remainder)."""
    import numpy as np
    rng = np.random.default_rng(seed)
    out, used = [], 0
    while used < total:
        L = int(np.exp(rng.uniform(np.log(lo), np.log(hi + 1))))
        L = min(L, total - used)
        out.append(L)
        used += L
    return out


def varlen_bench(steps=10, stored=True):
    """Packed variable-length batch with the tokens of the headline step
    (32768 tokens x 16 heads, d = 128, bf16): documents of log-uniform length in
    [64, 4096] (the 4K training context), so most end in a partial chunk.
    fwd+bwd step time and per-kernel averages."""
    import numpy as np
    import torch
    import paper_2605_22791_amd as g2
    from paper_2605_22791_amd.inputs import make_packed
    lengths = packed_lengths(8 * 4096)
    d = make_packed(lengths, 16, 128, 128, seed=31, dtype="bf16", decay_shift=-2.0)
    tb = lambda x: torch.from_numpy(x).cuda().to(torch.bfloat16).contiguous()
    q, k, v, b, w, do = (tb(d[n]) for n in ("q", "k", "v", "b", "w", "do"))
    la = torch.from_numpy(d["log_alpha"]).cuda().contiguous()
    cu = torch.from_numpy(d["cu_seqlens"]).cuda()
    N, T = len(lengths), sum(lengths)
    prob = g2.Gdr2Problem(1, T, 16, 128, 128, 64, d["scale"], g2.GDR2_BF16)
    ws = torch.empty(g2.gdr2_varlen_workspace_bytes(prob, N, 1), dtype=torch.uint8, device="cuda")

    def step():
        g2.gdr2_chunk_fwd_varlen(q, k, v, la, b, w, cu, None, scale=d["scale"], ws=ws, save=stored)
        g2.gdr2_chunk_bwd_varlen(q, k, v, la, b, w, cu, None, do, None, scale=d["scale"], ws=ws, saved=stored)

    for _ in range(2):
        step()
    torch.cuda.synchronize()
    g2.gdr2_profile_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    per_kernel = g2.gdr2_profile_collect()
    g2.gdr2_profile_enable(False)
    ms = e0.elapsed_time(e1) / steps
    chunks = int(sum(-(-L // 64) for L in lengths))
    kern = {n: round(kms / cnt * 1e3, 1) for n, (kms, cnt) in per_kernel.items() if cnt}
    return {"workload": f"packed batch, {N} sequences (log-uniform 64..4096 tokens), T = {T}, H16 d128 bf16",
            "training_path": "stored" if stored else "recompute", "n_seqs": N, "chunks_per_head": chunks,
            "partial_chunks_per_head": int(sum(1 for L in lengths if L % 64)),
            "ms_per_step": ms, "tokens_per_s": T / (ms * 1e-3), "kernels_avg_us": kern}


def grouped_bench(steps=10, stored=True):
    """Grouped value heads: the headline step's 32768 tokens with H = 8 key heads
    shared by Hv = 16 value heads (G = 2), d = 128, bf16.  fwd+bwd step time."""
    import torch
    import paper_2605_22791_amd as g2
    from paper_2605_22791_amd.inputs import make_grouped
    d = make_grouped(8, 4096, 8, 16, 128, 128, seed=41, dtype="bf16", decay_shift=-2.0)
    tb = lambda x: torch.from_numpy(x).cuda().to(torch.bfloat16).contiguous()
    q, k, v, b, w, do = (tb(d[n]) for n in ("q", "k", "v", "b", "w", "do"))
    la = torch.from_numpy(d["log_alpha"]).cuda().contiguous()
    prob = g2.Gdr2Problem(8, 4096, 8, 128, 128, 64, d["scale"], g2.GDR2_BF16, 16)
    ws = torch.empty(g2.gdr2_chunk_workspace_bytes(prob, 1), dtype=torch.uint8, device="cuda")

    def step():
        g2.gdr2_chunk_fwd(q, k, v, la, b, w, None, scale=d["scale"], ws=ws, save=stored)
        g2.gdr2_chunk_bwd(q, k, v, la, b, w, None, do, None, scale=d["scale"], ws=ws, saved=stored)

    for _ in range(2):
        step()
    torch.cuda.synchronize()
    g2.gdr2_profile_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    per_kernel = g2.gdr2_profile_collect()
    g2.gdr2_profile_enable(False)
    ms = e0.elapsed_time(e1) / steps
    kern = {n: round(kms / cnt * 1e3, 1) for n, (kms, cnt) in per_kernel.items() if cnt}
    return {"workload": "grouped value heads B8 T4096 H8 Hv16 d128 bf16", "training_path": "stored" if stored else "recompute",
            "ms_per_step": ms, "tokens_per_s": 8 * 4096 / (ms * 1e-3), "kernels_avg_us": kern}


def fused_bench(steps=10, stored=True):
    """Fused input stage at the headline shape (B8 T4096 H16 d128 bf16): the
    step from the raw projections (q, k unnormalised, the decay projection f,
    a, delta) with normalisation and activation inside the kernels, against
    the same step composed from separate torch passes (normalise q, k, form
    g, run the plain operator, then the two VJPs)."""
    import torch
    import torch.nn.functional as F
    import paper_2605_22791_amd as g2
    from paper_2605_22791_amd.inputs import make_fused
    d = make_fused(8, 4096, 16, 128, 128, seed=51, dtype="bf16")
    tb = lambda x: torch.from_numpy(x).cuda().to(torch.bfloat16).contiguous()
    tf = lambda x: torch.from_numpy(x).cuda().contiguous()
    q, k, v, b, w, do = (tb(d[n]) for n in ("q", "k", "v", "b", "w", "do"))
    f, a, delta = tf(d["f"]), tf(d["a"]), tf(d["delta"])
    sc, eps = d["scale"], d["eps"]
    prob = g2.Gdr2Problem(8, 4096, 16, 128, 128, 64, sc, g2.GDR2_BF16)
    ws_f = torch.empty(g2.gdr2_fused_workspace_bytes(prob, 0, 1), dtype=torch.uint8, device="cuda")
    ws_p = torch.empty(g2.gdr2_chunk_workspace_bytes(prob, 1), dtype=torch.uint8, device="cuda")

    def fused():
        g2.gdr2_fused_fwd(q, k, v, f, a, delta, b, w, None, scale=sc, eps=eps, ws=ws_f, save=stored)
        g2.gdr2_fused_bwd(q, k, v, f, a, delta, b, w, None, do, None, scale=sc, eps=eps, ws=ws_f, saved=stored)

    def composed():
        qf, kf = q.float(), k.float()
        rq = torch.rsqrt((qf * qf).sum(-1, keepdim=True) + eps)
        rk = torch.rsqrt((kf * kf).sum(-1, keepdim=True) + eps)
        A = a.exp()[:, None]
        x = f + delta
        g = (-A * F.softplus(x)).contiguous()
        qn, kn = (qf * rq).bfloat16(), (kf * rk).bfloat16()
        g2.gdr2_chunk_fwd(qn, kn, v, g, b, w, None, scale=sc, ws=ws_p, save=stored)
        gr = g2.gdr2_chunk_bwd(qn, kn, v, g, b, w, None, do, None, scale=sc, ws=ws_p, saved=stored)
        for xf, r, dy in ((qf, rq, gr["dq"]), (kf, rk, gr["dk"])):
            y, dyf = xf * r, dy.float()
            (r * (dyf - y * (y * dyf).sum(-1, keepdim=True))).bfloat16()
        dg = gr["dlog_alpha"]
        df = dg * (-A * torch.sigmoid(x))
        df.sum((0, 1))
        (dg * g).sum((0, 1, 3))

    def timed(fn, prof=False):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        if prof:
            g2.gdr2_profile_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        kern = None
        if prof:
            per_kernel = g2.gdr2_profile_collect()
            g2.gdr2_profile_enable(False)
            kern = {n: round(kms / cnt * 1e3, 1) for n, (kms, cnt) in per_kernel.items() if cnt}
        return e0.elapsed_time(e1) / steps, kern

    ms_f, kern = timed(fused, prof=True)
    ms_c, _ = timed(composed)
    return {"workload": "fused input stage, B8 T4096 H16 d128 bf16 (raw q, k, decay projection f)",
            "training_path": "stored" if stored else "recompute", "ms_per_step": ms_f,
            "tokens_per_s": 8 * 4096 / (ms_f * 1e-3), "kernels_avg_us": kern,
            "composed_ms_per_step": ms_c, "composed": "torch passes for the stage and its VJPs around the plain operator"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the copy-bandwidth, long-context (config 3) and decode side measurements")
    ap.add_argument("--cpu-heads", type=int, default=16)
    ap.add_argument("--path", choices=("stored", "recompute"), default="stored",
                    help="training path of the timed step: the forward keeps A, h and R for the backward "
                         "(stored) or the backward recomputes them (recompute, the memory-saving path); "
                         "the other path is timed too and reported beside")
    ap.add_argument("--calib-copy", type=int, default=0, metavar="MIB",
                    help="run one copy-like elementwise kernel (torch.neg) over MIB MiB of fp32 before the "
                         "timed steps: the reference that scales rocprofv3 FETCH_SIZE / WRITE_SIZE to bytes")
    ap.add_argument("--fused-only", action="store_true",
                    help="time only the fused input stage step (raw projections, B8 T4096 H16) and its composed "
                         "counterpart and print their figures")
    ap.add_argument("--varlen-only", action="store_true",
                    help="time only the packed variable-length batch (32768 tokens, H=16) and print its figures")
    ap.add_argument("--decode-only", action="store_true",
                    help="time only the decode leg (1024 one-token calls) and print its figures")
    ap.add_argument("--decode-batch", type=int, default=256,
                    help="sequences of the decode leg (256: the 256 MiB fp32 state of the decode workload)")
    ap.add_argument("--long-context-only", action="store_true",
                    help="time only the long-context step (B=1, H=16, T=65536) for --steps steps and print "
                         "its figures (not the benchmark line)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)
    if args.decode_only:
        if args.calib_copy > 0:
            calibration_copy(args.calib_copy)
        print(json.dumps(decode_bench(1024, B=args.decode_batch)), flush=True)
        return
    if args.long_context_only:
        print(json.dumps(config3_bench(steps=args.steps, stored=args.path == "stored")), flush=True)
        return
    if args.varlen_only:
        print(json.dumps(varlen_bench(steps=args.steps, stored=args.path == "stored")), flush=True)
        return
    if args.fused_only:
        print(json.dumps(fused_bench(steps=args.steps, stored=args.path == "stored")), flush=True)
        return

    import torch
    import paper_2605_22791_amd as g2
    from paper_2605_22791_amd.inputs import config

    print("[bench] generating config-2 inputs", file=sys.stderr, flush=True)
    d = config(2)
    B, T, H, Dk, Dv = d["B"], d["T"], d["H"], d["Dk"], d["Dv"]
    dev = "cuda"
    tb = lambda x: torch.from_numpy(x).to(dev).to(torch.bfloat16).contiguous()
    q, k, v, b, w, do = (tb(d[n]) for n in ("q", "k", "v", "b", "w", "do"))
    la = torch.from_numpy(d["log_alpha"]).to(dev).contiguous()
    o = torch.empty_like(v)
    ST = torch.empty(B, H, Dk, Dv, device=dev)
    grads = {"dq": torch.empty_like(q), "dk": torch.empty_like(k), "dv": torch.empty_like(v),
             "dlog_alpha": torch.empty_like(la), "db": torch.empty_like(b), "dw": torch.empty_like(w),
             "dS0": torch.empty(B, H, Dk, Dv, device=dev)}
    prob = g2.Gdr2Problem(B, T, H, Dk, Dv, 64, d["scale"], g2.GDR2_BF16)
    ws = torch.empty(g2.gdr2_chunk_workspace_bytes(prob, 1), dtype=torch.uint8, device=dev)

    def make_step(stored):
        def step():
            g2.gdr2_chunk_fwd(q, k, v, la, b, w, None, scale=d["scale"], o=o, S_T=ST, ws=ws, save=stored)
            g2.gdr2_chunk_bwd(q, k, v, la, b, w, None, do, None, scale=d["scale"], grads=grads, ws=ws,
                              saved=stored)
        return step

    stored = args.path == "stored"
    step = make_step(stored)

    if args.calib_copy > 0:
        calibration_copy(args.calib_copy)

    print("[bench] warmup", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K steps, per-kernel hipEvents recorded on the launch stream
    g2.gdr2_profile_enable(True)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_kernel = g2.gdr2_profile_collect()
    g2.gdr2_profile_enable(False)
    ms_total = e0.elapsed_time(e1)
    ms_step = ms_total / args.steps
    tokens_per_s = B * T / (ms_step * 1e-3)
    print(f"[bench] {ms_step:.3f} ms/step ({wall / args.steps * 1e3:.3f} ms wall)", file=sys.stderr, flush=True)

    model = kernel_model(B, T, H, Dk, Dv, stored)
    mbytes = method_bytes(B, T, H, Dk, Dv)
    kern = {}
    for name, (ms, cnt) in per_kernel.items():
        if cnt == 0:
            continue
        avg = ms / cnt
        fl, by = model[name]
        mb = mbytes[name]
        traffic = measured_traffic(name)
        kern[name] = {"avg_us": avg * 1e3, "launches": cnt, "GBs": mb / (avg * 1e-3) / 1e9,
                      "hbm_frac": mb / (avg * 1e-3) / 1e9 / HBM_PEAK_GBS,
                      "TFLOPs": fl / (avg * 1e-3) / 1e12, "alg_bytes": mb, "alg_flops": fl,
                      "decomposition_bytes": by, "traffic": traffic,
                      "traffic_GBs": None if traffic is None else traffic / (avg * 1e-3) / 1e9}
    dom = max(kern, key=lambda n: kern[n]["avg_us"] * kern[n]["launches"])
    kd = kern[dom]
    peak_fl = PEAK_TFLOPS[MFMA_DTYPE]
    ridge = peak_fl * 1e12 / (HBM_PEAK_GBS * 1e9)
    ai = kd["alg_flops"] / kd["alg_bytes"]
    if ai >= ridge:
        roof = {"bound": "mfma", "achieved": kd["TFLOPs"], "peak": peak_fl, "unit": "TFLOP/s",
                "frac": kd["TFLOPs"] / peak_fl}
    else:
        roof = {"bound": "hbm", "achieved": kd["GBs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": kd["GBs"] / HBM_PEAK_GBS}
    traffic = kd["traffic"]
    roof.update({"traffic": traffic, "kernel": dom, "avg_us": kd["avg_us"],
                 "alg_bytes": kd["alg_bytes"], "decomposition_bytes": kd["decomposition_bytes"],
                 "traffic_over_alg": None if traffic is None else traffic / kd["alg_bytes"],
                 "traffic_GBs": kd["traffic_GBs"],
                 "mfma_dtype": MFMA_DTYPE, "arith_intensity": ai, "ridge": ridge})

    # the other training path, same number of steps, no per-kernel events
    other = make_step(not stored)
    for _ in range(args.warmup):
        other()
    torch.cuda.synchronize()
    f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    f0.record()
    for _ in range(args.steps):
        other()
    f1.record()
    torch.cuda.synchronize()
    other_ms = f0.elapsed_time(f1) / args.steps
    print(f"[bench] {'recompute' if stored else 'stored'} path: {other_ms:.3f} ms/step", file=sys.stderr, flush=True)

    fwd_flops = sum(model[n][0] for n in ("fwd_intra", "fwd_state"))
    step_flops = sum(model[n][0] for n in model if n in kern)
    out = {
        "metric": "tokens/s fwd+bwd GDR-2 chunked op (H=16,d=128,T=4096,bf16); % MFMA peak",
        "value": tokens_per_s, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "GDR-2 chunkwise fwd+bwd, 1.3B-layer training shape",
                   "B": B, "H": H, "T": T, "d_k": Dk, "d_v": Dv, "chunk": 64, "io": "bf16",
                   "log_alpha": "fp32", "state": "fp32", "global_batch": B, "seq_len": T,
                   "training_path": args.path},
        "mfma_pct_of_bf16_peak": 100.0 * step_flops / (ms_step * 1e-3) / 1e12 / PEAK_TFLOPS["bf16"],
        "roofline": roof,
        "kernels": {n: {kk: (round(vv, 3) if isinstance(vv, float) else vv) for kk, vv in kv.items()}
                    for n, kv in kern.items()},
        "fwd_ms": sum(kern[n]["avg_us"] for n in ("fwd_intra", "fwd_state") if n in kern) / 1e3,
        "bwd_ms": sum(kern[n]["avg_us"] for n in kern if n.startswith("bwd")) / 1e3,
        "alg_tflops_per_step": step_flops / 1e12, "fwd_alg_tflops": fwd_flops / 1e12,
        "other_path": {"training_path": "recompute" if stored else "stored", "ms_per_step": other_ms,
                       "tokens_per_s": B * T / (other_ms * 1e-3)},
    }
    if not args.no_extra:
        print("[bench] copy bandwidth", file=sys.stderr, flush=True)
        out["copy_GBs"] = copy_bandwidth()
    if not args.no_decode and not args.no_extra:
        print("[bench] decode (1024 one-token calls, B=256)", file=sys.stderr, flush=True)
        out["decode"] = decode_bench(1024)
        # twice the state: larger than the Infinity Cache, so the state read-modify-write runs from HBM
        out["decode_B512"] = decode_bench(1024, B=512)
    if not args.no_extra:
        print("[bench] long context (config 3)", file=sys.stderr, flush=True)
        out["long_context"] = config3_bench(stored=stored)
        print("[bench] packed variable-length batch", file=sys.stderr, flush=True)
        out["varlen"] = varlen_bench(stored=stored)
        print("[bench] grouped value heads", file=sys.stderr, flush=True)
        out["grouped"] = grouped_bench(stored=stored)
        print("[bench] fused input stage", file=sys.stderr, flush=True)
        out["fused"] = fused_bench(stored=stored)
    if not args.no_cpu:
        print("[bench] cpu oracle baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(d, args.cpu_heads)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
