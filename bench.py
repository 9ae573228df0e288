"""Benchmark of the LoGra hot path on one MI355X.

Logging leg (the reported `value`, tokens/s): the 32-block Llama3-8B logging
stream -- per step one batch of B=8 examples of T=2048 padded tokens, valid
lengths uniform on 128..2048, through all 224 linear layers (k_in = k_out = 16,
57,344 projected dims per example): fused projection into the bf16 gradient
store (8 grouped launches of 28 layers, four blocks each) and the 224 per-layer covariance
updates, each kept as its lower triangle (all the preconditioner reads).

The logging leg's "shared_inputs" entry runs the same stream with the
inputs a transformer block shares (q/k/v one x, gate/up one x), which the
projection reads once.  Its "offload" entry runs the stream again with each
step's store rows copied to a pinned host store (out-of-core logging), the
copy enqueued behind the step on the compute stream, so the host is free
while it runs.  Its "pca" entry times the PCA initialisation of the
projections on one of its batches: the KFAC factor SYRKs of the gate layer
(n = 4096 and 14,336) and their top-16 eigenvectors.

Influence leg (reported under "influence", scores/s): 1,024 test gradients
against 500,000 stored training gradients of 57,344 dims -- damped-Cholesky
preconditioning of the test gradients over 224 blocks of 256 (covariances of
4,096 gradients, damping 0.1 x mean eigenvalue), the score GEMM and the
per-query top-100.  Its "out_of_core" entry streams 131,072 of the stored
rows from pinned host memory through two device buffers (the store of the
paper outgrows GPU memory) and compares the rate with a plain copy over the
same link.  Its "relatif" entry times l-RelatIF on the same store: the
self-influence of every training row (once per store) and the score pass with
the 1/sqrt(self) scales applied before the top-100.  Its "vendor_gemm" entry
times torch.matmul (hipBLASLt) and this library's scores-only path on the same
125,000-row slice of the operands: a measured reference beside the published
peak.

All inputs are synthetic, drawn on the device before timing.  Each leg
reports the roofline of its dominant kernel from HIP events recorded on the
launch stream around the timed launches (the logging leg: one pair over each
step's back-to-back launches), and the float64 oracle timed on a bounded
sample on the host (rank 0 only).
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as W  # noqa: E402

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
PCIE_PEAK_GBS = 64.0   # PCIe 5.0 x16, one direction
METRIC = "projected per-example grads/sec (tokens/s) at Llama3-8B shapes; influence scores/sec"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


TRAFFIC_PATH = os.path.join(ROOT, "profiles", "traffic.json")
PROJ_SOURCES = ["paper_2405_13954_amd/csrc/project.hip", "paper_2405_13954_amd/csrc/common.h"]
SCORE_SOURCES = ["paper_2405_13954_amd/csrc/scores.hip", "paper_2405_13954_amd/csrc/common.h"]
SELF_SOURCES = ["paper_2405_13954_amd/csrc/selfinf.hip", "paper_2405_13954_amd/csrc/common.h"]
PCA_SOURCES = ["paper_2405_13954_amd/csrc/pca.hip", "paper_2405_13954_amd/csrc/common.h"]


def source_sha(sources):
    import hashlib
    h = hashlib.sha256()
    for f in sources:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(key, sources):
    """HBM bytes per launch of a kernel from the committed counter summary
    (profiles/traffic.json), or None when the kernel's sources changed since
    the counters were taken."""
    try:
        rec = json.load(open(TRAFFIC_PATH))[key]
    except (OSError, KeyError, ValueError):
        return None, None
    if source_sha(sources) != rec.get("source_sha"):
        return None, None
    return rec["traffic_bytes"], rec["traffic_over_algorithmic"]


def write_traffic(fetch_csv, write_csv):
    """profiles/traffic.json from the counter files of two runs
    `rocprofv3 --pmc FETCH_SIZE` and `rocprofv3 --pmc WRITE_SIZE` (csv) of
    `bench.py --no-cpu-baseline --steps 3 --warmup 1 --inf-passes 1`.  Per
    kernel, the launches with the largest grid are averaged (the full-size
    launches: the scores-only GEMM over all 500,000 rows, the self-influence
    of the store); the SYRK row takes its single-factor launches (n = 14,336).  Reads = 2 x FETCH_SIZE and writes = 1 x WRITE_SIZE (KiB):
    the factors a plain copy of 1 GiB shows (524,288 KiB fetched, 1,048,576
    KiB written).  The stream kernel's grid is the same for every launch (it
    is sized to the resident workgroups), so its row takes the first launches
    in dispatch order instead: the logging leg runs first, 4 steps of 8
    28-layer launches."""
    import collections
    import csv
    import re

    stream = W.WORKLOADS["llama3_8b_stream"]
    log_launches = 4 * (stream.n_layers // (4 * len(stream.layers)))
    # threads of the n = 14,336 SYRK launch: 256 per workgroup slot, slots in groups of
    # 4 x 8 tiles of 256, a multiple of 8 groups
    nt = 14336 // 256
    groups = sum((nt + 7) // 8 - gr // 2 for gr in range((nt + 3) // 4))
    act_cov_grid = (groups + 7) // 8 * 8 * 32 * 256

    def load(path, ctr):
        d = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == ctr and "logra" in r["Kernel_Name"]:
                n = re.sub(r"\(.*", "", r["Kernel_Name"].replace("(anonymous namespace)::", "").replace("void ", ""))
                d[n].append((int(r["Dispatch_Id"]), int(r["Grid_Size"]), float(r["Counter_Value"])))
        out = {}
        for n, v in d.items():
            if n == "logra::k_project_stream":
                vals = [x for _, _, x in sorted(v)[:log_launches]]
            elif n == "logra::k_act_cov_dma":   # the single-factor launch (the grouped one is larger)
                vals = [x for _, g, x in v if g == act_cov_grid]
            else:
                gmax = max(g for _, g, _ in v)
                vals = [x for _, g, x in v if g == gmax]
            out[n] = sum(vals) / len(vals)
        return out

    f, w = load(fetch_csv, "FETCH_SIZE"), load(write_csv, "WRITE_SIZE")
    lens = [W.lengths(W.rng(0, 200, s), stream.B, stream.len_lo, stream.len_hi) for s in range(4)]
    per_tok = sum(2 * (a + b) for _, a, b in stream.layers)
    p_bytes = sum(2 * stream.k_in * (a + b) for _, a, b in stream.layers)
    sc = W.WORKLOADS["llama3_8b_scores"]
    N, Q, D_tot = sc.extra["N_train"], sc.extra["Q"], sc.n_layers * sc.D
    rows = {
        "projection": ("logra::k_project_stream", "k_project_stream",
                       "28 Llama3-8B layers (4 blocks), B=8, T=2048, lengths of steps 0-3, k=16", PROJ_SOURCES,
                       4 * (sum(int(x.sum()) for x in lens) / 4 * per_tok + p_bytes)),
        "projection_k64": ("logra::k_project_tiles<4, true>", "k_project_tiles<4, true> (paired units)",
                           "7 Llama3-8B layers, B=16, T=1024, all valid, k=64", PROJ_SOURCES,
                           16 * 1024 * per_tok + sum(2 * 64 * (a + b) for _, a, b in stream.layers)),
        "scores": ("logra::k_scores_dma", "k_scores_dma", "1,024 x 500,000 x 57,344 bf16", SCORE_SOURCES,
                   (N + Q) * D_tot * 2 + Q * N * 4),
        "self_influence": ("logra::k_self_influence_dma", "k_self_influence_dma",
                           "500,000 x 57,344 bf16, 224 blocks of 256", SELF_SOURCES,
                           N * D_tot * 2 + sc.n_layers * sc.D * 2 * sc.D * 2 + N * 4),
        # the largest launch of the PCA sub-leg: the gate layer's dy (n = 14,336) over one
        # batch; algorithmic = the valid tokens' rows read once + C read once and written once
        "act_cov": ("logra::k_act_cov_dma", "k_act_cov_dma",
                    "gate dy, n = 14,336, one batch (B=8, lengths of step 0)", PCA_SOURCES,
                    int(lens[0].sum()) * 14336 * 2 + 2 * 14336 * 14336 * 4),
    }
    out = {"_about": "HBM traffic per launch from rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE runs of "
                     "bench.py (--no-cpu-baseline --steps 3 --warmup 1 --inf-passes 1), written by "
                     "`python bench.py --write-traffic <FETCH_SIZE csv> <WRITE_SIZE csv>`. Read bytes = "
                     "2 x FETCH_SIZE (KiB x 1024): a plain copy of 1 GiB reads 524,288 KiB of FETCH_SIZE and "
                     "writes 1,048,576 KiB of WRITE_SIZE, so reads are scaled by 2 and writes by 1. source_sha "
                     "covers the kernel's source files; bench.py reports traffic only while it matches."}
    for key, (name, kernel, workload, sources, alg) in rows.items():
        if name not in f or name not in w:
            continue
        rec = {"kernel": kernel, "workload": workload, "source_sha": source_sha(sources),
               "read_bytes": 2 * f[name] * 1024, "write_bytes": w[name] * 1024, "algorithmic_bytes": alg}
        rec["traffic_bytes"] = rec["read_bytes"] + rec["write_bytes"]
        rec["traffic_over_algorithmic"] = rec["traffic_bytes"] / alg
        out[key] = rec
    with open(TRAFFIC_PATH, "w") as fh:
        json.dump(out, fh, indent=1)
        fh.write("\n")
    print(json.dumps(out, indent=1))


class EventTimer:
    """Pairs of HIP events on the launch stream; mean duration per launch in ms.
    A pair may bracket n back-to-back launches (stop(s, n)): each event record
    puts a marker in the queue that holds the next launch for about 10 us, so
    bracketing every launch would add that gap to the work being timed."""

    def __init__(self, torch):
        self.torch = torch
        self.pairs = []

    def start(self):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record()
        return e

    def stop(self, s, n=1):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record()
        self.pairs.append((s, e, n))

    def mean_ms(self):
        return float(np.mean([a.elapsed_time(b) / n for a, b, n in self.pairs])) if self.pairs else float("nan")


# -------------------------------------------------------------------- peaks --
def peaks_leg(args, torch):
    """Measured ceilings beside the published peaks: a sustained bf16 MFMA
    loop on every CU (long enough for the clock to settle) and an HBM read
    stream of 4 GiB (far above the 256 MB MALL), both timed with HIP events;
    the MFMA kernel also reports the core clock it ran at."""
    import paper_2405_13954_amd as P
    L = ctypes.CDLL(os.path.join(os.path.dirname(P.LIB_PATH), "libpaper_logra_peaks.so"))
    L.logra_peak_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p]
    L.logra_peak_mfma_bf16_data.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_void_p]
    L.logra_peak_hbm_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                      ctypes.c_void_p]
    props = torch.cuda.get_device_properties(0)
    cus = props.multi_processor_count
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    groups = cus * 4                                     # four waves per SIMD
    flops_per_iter = groups * 4 * 4 * 32768.0            # waves x 4 MFMAs x 32x32x16x2
    iters = int(args.peak_ms * 1e-3 * BF16_PEAK_TFLOPS * 1e12 / flops_per_iter)
    sink = torch.empty(max(groups, cus * 8), dtype=torch.float32, device="cuda")
    cyc = torch.zeros(2, dtype=torch.int64, device="cuda")
    t = EventTimer(torch)
    for timed in (False, True, True, True):
        e0 = t.start() if timed else None
        assert L.logra_peak_mfma_bf16(groups, iters, ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(cyc.data_ptr()),
                                      stream) == 0
        if timed:
            t.stop(e0)
    torch.cuda.synchronize()
    mfma_tf = flops_per_iter * iters / (t.mean_ms() * 1e-3) / 1e12
    khz = ctypes.c_int(0)
    wall_khz = khz.value if L.logra_peak_wall_clock_khz(ctypes.byref(khz)) == 0 else None

    def clock_of(c):
        cycles, ticks = (int(v) for v in c.cpu())
        return cycles / (ticks / (wall_khz * 1e3)) / 1e9 if wall_khz and ticks > 0 else None

    clock_ghz = clock_of(cyc)
    # the same loop with random bf16 operands that change from one MFMA to the next
    gen = torch.Generator(device="cuda")
    gen.manual_seed(0)
    ops = torch.randn(16 * 16 * 256 * 8, device="cuda", generator=gen).to(torch.bfloat16)   # 1 MiB
    iters_d = iters - iters % 8
    td = EventTimer(torch)
    for timed in (False, True, True, True):
        e0 = td.start() if timed else None
        assert L.logra_peak_mfma_bf16_data(groups, iters_d, ctypes.c_void_p(ops.data_ptr()),
                                           ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(cyc.data_ptr()),
                                           stream) == 0
        if timed:
            td.stop(e0)
    torch.cuda.synchronize()
    mfma_data_tf = flops_per_iter * iters_d / (td.mean_ms() * 1e-3) / 1e12
    data_clock_ghz = clock_of(cyc)
    nbytes = 4 << 30
    buf = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
    modes = {}
    for mode, name in ((0, "grid_stride_loads"), (1, "blocked_nontemporal_loads"), (2, "lds_dma_copies")):
        r = EventTimer(torch)
        for timed in (False, True, True, True, True, True):
            e0 = r.start() if timed else None
            assert L.logra_peak_hbm_read(ctypes.c_void_p(buf.data_ptr()), nbytes, cus * 8, mode,
                                         ctypes.c_void_p(sink.data_ptr()), stream) == 0
            if timed:
                r.stop(e0)
        torch.cuda.synchronize()
        modes[name] = nbytes / (r.mean_ms() * 1e-3) / 1e9
    read_gbs = max(modes.values())
    del buf
    torch.cuda.empty_cache()
    return {"mfma_bf16_tflops": mfma_tf, "mfma_frac_of_spec": mfma_tf / BF16_PEAK_TFLOPS,
            "mfma_ms": t.mean_ms(), "mfma_clock_ghz": clock_ghz,
            "mfma_bf16_data_tflops": mfma_data_tf, "mfma_data_frac_of_spec": mfma_data_tf / BF16_PEAK_TFLOPS,
            "mfma_data_ms": td.mean_ms(), "mfma_data_clock_ghz": data_clock_ghz, "hbm_read_gbs": read_gbs,
            "hbm_read_frac_of_spec": read_gbs / HBM_PEAK_GBS, "hbm_read_gbs_by_method": modes,
            "compute_units": cus,
            "note": "sustained 32x32x16 bf16 MFMA loop on every CU for the time shown, once on one constant "
                    "operand pair (mfma_bf16_*) and once on random operands that change from one MFMA to the "
                    "next (mfma_bf16_data_*, the ceiling for products of real data); a 4 GiB read stream three "
                    "ways, the best taken as the ceiling; published peaks 2,500 TFLOP/s and 8,000 GB/s"}


# ------------------------------------------------------------------ logging --
def logging_leg(args, torch, P):
    w = W.WORKLOADS["llama3_8b_stream"]
    B, T, k = w.B, w.T, w.k_in
    D = w.D
    layers = w.layers
    nl_block = len(layers)
    n_layers = w.n_layers
    D_tot = n_layers * D
    dev = "cuda"
    n_buf = 4   # distinct x/dy buffer sets, cycled over the 32 blocks (each 2.7 GB >> the 256 MB MALL)
    log(f"[log] allocating {n_buf} x/dy block buffers, projections for {n_layers} layers, store")
    gen = W.torch_generator(args.seed, 100)
    bufs = []
    for i in range(n_buf):
        blk = []
        for (_, n_in, n_out) in layers:
            x = torch.empty((B, T, n_in), dtype=torch.bfloat16, device=dev)
            dy = torch.empty((B, T, n_out), dtype=torch.bfloat16, device=dev)
            W.device_normal_(x, w.x_std, gen)
            W.device_normal_(dy, w.dy_std, gen)
            blk.append((x, dy))
        bufs.append(blk)
    projs = []
    for l in range(n_layers):
        _, n_in, n_out = layers[l % nl_block]
        pi = torch.empty((k, n_in), dtype=torch.bfloat16, device=dev)
        po = torch.empty((k, n_out), dtype=torch.bfloat16, device=dev)
        W.device_normal_(pi, 1.0 / np.sqrt(k), gen)
        W.device_normal_(po, 1.0 / np.sqrt(k), gen)
        projs.append((pi, po))
    n_steps = args.warmup + args.steps
    n_rows = max(n_steps * B, B)
    store = torch.empty((n_rows, D_tot), dtype=torch.bfloat16, device=dev)
    S = torch.zeros((n_layers, D, D), dtype=torch.float32, device=dev)
    lens = [W.lengths(W.rng(args.seed, 200, s), B, w.len_lo, w.len_hi) for s in range(n_steps)]
    masks = [torch.from_numpy(W.mask_from_lengths(L, T)).to(dev) for L in lens]
    gb = args.log_group_blocks            # blocks per grouped launch
    n_launch = w.blocks // gb
    nl_launch = gb * nl_block
    shape_descs = (P.LayerDesc * nl_launch)(*[P.LayerDesc(0, 0, 0, 0, 0, ni, no) for _ in range(gb)
                                             for _, ni, no in layers])
    ws_bytes = P.logra_project_layers_ws_size(shape_descs, nl_launch, B, T, k, k)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    L = P.lib()
    g_ld = store.stride(0)

    # descriptor arrays per (step, launch of gb blocks), built once
    def descs(step, li):
        arr = (P.LayerDesc * nl_launch)()
        row0 = step * B
        for bb in range(gb):
            blk = li * gb + bb
            for j in range(nl_block):
                l = blk * nl_block + j
                x, dy = bufs[blk % n_buf][j]
                pi, po = projs[l]
                g = store[row0:row0 + B, l * D:(l + 1) * D]
                arr[bb * nl_block + j] = P.LayerDesc(x.data_ptr(), dy.data_ptr(), pi.data_ptr(), po.data_ptr(),
                                                     g.data_ptr(), x.shape[2], dy.shape[2])
        return arr

    all_descs = [[descs(s, li) for li in range(n_launch)] for s in range(n_steps)]
    proj_timer = EventTimer(torch)
    cov_timer = EventTimer(torch)

    def step(s, timed, descs_of=all_descs, ptimer=proj_timer):
        m = masks[s]
        e0 = ptimer.start() if timed else None   # one pair over the step's back-to-back launches
        for li in range(n_launch):
            rc = L.logra_project_layers(descs_of[s][li], nl_launch, P.BF16, B, T, ctypes.c_void_p(m.data_ptr()),
                                        k, k, P.BF16, g_ld, ctypes.c_void_p(ws.data_ptr()), ws_bytes, stream)
            if rc != 0:
                raise P.LograError(rc, P.logra_last_error())
        if timed:
            ptimer.stop(e0, n_launch)
        rows = store[s * B:(s + 1) * B]
        e0 = cov_timer.start() if timed else None
        rc = L.logra_cov_accumulate_blocks_lower(ctypes.c_void_p(rows.data_ptr()), P.BF16, g_ld, B, D, n_layers,
                                                 ctypes.c_void_p(S.data_ptr()), stream)
        if rc != 0:
            raise P.LograError(rc, P.logra_last_error())
        if timed:
            cov_timer.stop(e0)

    log(f"[log] warmup {args.warmup} steps")
    for s in range(args.warmup):
        step(s, False)
    torch.cuda.synchronize()
    log(f"[log] timing {args.steps} steps")
    t0 = time.perf_counter()
    for s in range(args.warmup, n_steps):
        step(s, True)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    tokens = int(sum(int(L_.sum()) for L_ in lens[args.warmup:]))
    examples = args.steps * B
    # algorithmic bytes of one grouped launch (gb blocks of 7 layers), averaged over timed steps:
    # valid tokens x 2 B x (n_in + n_out) summed over the launch's layers, plus the projections once.
    per_tok = gb * sum(2 * (ni + no) for _, ni, no in layers)
    proj_bytes = gb * sum(2 * k * (ni + no) for _, ni, no in layers)
    bytes_per_launch = tokens / args.steps * per_tok + proj_bytes
    proj_ms = proj_timer.mean_ms()
    achieved = bytes_per_launch / (proj_ms * 1e-3) / 1e9
    traffic, ratio = measured_traffic("projection", PROJ_SOURCES)
    res = {
        "tokens": tokens, "seconds": dt,
        "tokens_per_s": tokens / dt, "examples_per_s": examples / dt,
        "ms_per_step": dt * 1e3 / args.steps,
        "proj_launch_ms": proj_ms, "cov_launch_ms": cov_timer.mean_ms(),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic, "traffic_over_algorithmic": ratio,
                     "kernel": f"logra_project_layers ({nl_launch} Llama3-8B layers = {gb} blocks, B=8 ragged, k=16)",
                     "bytes_per_launch": bytes_per_launch},
    }
    res["roofline"]["copy_gbs"] = copy_bandwidth(torch)
    if args.shared_inputs:
        # the same stream with the inputs a transformer block shares: q/k/v read
        # one x, gate/up read one x (x elements per token 38,912 -> 26,624)
        shared = [[descs(st, li) for li in range(n_launch)] for st in range(n_steps)]
        for st in range(n_steps):
            for li in range(n_launch):
                for bb in range(gb):
                    for j in (1, 2, 5):
                        src = shared[st][li][bb * nl_block + (0 if j < 4 else 4)]
                        d = shared[st][li][bb * nl_block + j]
                        shared[st][li][bb * nl_block + j] = P.LayerDesc(src.x, d.dy, d.p_in, d.p_out, d.g_out,
                                                                        d.n_in, d.n_out)
        sh_timer = EventTimer(torch)
        for st in range(args.warmup):
            step(st, False, shared, sh_timer)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for st in range(args.warmup, n_steps):
            step(st, True, shared, sh_timer)
        torch.cuda.synchronize()
        dt_sh = time.perf_counter() - t1
        x_shared = sum(ni for i, (_, ni, _) in enumerate(layers) if i not in (1, 2, 5))
        per_tok_sh = 2 * (x_shared + sum(no for _, _, no in layers))
        bytes_sh = tokens / args.steps * per_tok_sh * gb + proj_bytes
        res["shared_inputs"] = {
            "tokens_per_s": tokens / dt_sh, "ms_per_step": dt_sh * 1e3 / args.steps,
            "proj_launch_ms": sh_timer.mean_ms(), "bytes_per_token_per_block": per_tok_sh,
            "achieved_gbs": bytes_sh / (sh_timer.mean_ms() * 1e-3) / 1e9,
            "note": "q/k/v and gate/up given one x each, as in a transformer block; the headline value "
                    "uses separate inputs"}
    if args.offload:
        # out-of-core logging: after each step, its B store rows go to a
        # pinned host store.  The copy is enqueued on the compute stream: the
        # blit kernel that moves the rows costs ~20 us in line there, while on
        # a copy stream it shares the CUs with the streaming projection and
        # costs about ten times that.
        host_store = torch.empty((n_rows, D_tot), dtype=torch.bfloat16).pin_memory()
        off_timer = EventTimer(torch)

        def step_off(st, timed):
            step(st, timed, all_descs, off_timer)
            P.logra_offload_rows(store[st * B:(st + 1) * B], host_store[st * B:(st + 1) * B])

        for st in range(args.warmup):
            step_off(st, False)
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        for st in range(args.warmup, n_steps):
            step_off(st, True)
        torch.cuda.synchronize()
        dt_off = time.perf_counter() - t2
        same = bool(torch.equal(host_store.view(torch.int16), store.view(torch.int16).cpu()))
        res["offload"] = {
            "tokens_per_s": tokens / dt_off, "ms_per_step": dt_off * 1e3 / args.steps,
            "proj_launch_ms": off_timer.mean_ms(), "bytes_per_step": B * D_tot * 2,
            "host_store_equal": same,
            "note": "each step's store rows copied to pinned host memory behind the step on the compute "
                    "stream (asynchronous for the host)"}
        del host_store
    if args.pca:
        res["pca"] = pca_sub_leg(args, torch, P, bufs[0], lens[0], masks[0], k)
    sample = None
    if args.cpu_baseline:
        n_b = min(args.cpu_batches, n_buf)
        sample = {"batches": [{"x": [host_bf16(bufs[i][j][0]) for j in range(nl_block)],
                               "dy": [host_bf16(bufs[i][j][1]) for j in range(nl_block)],
                               "mask": W.mask_from_lengths(lens[i], T)} for i in range(n_b)],
                  "p_in": [host_bf16(projs[j][0]) for j in range(nl_block)],
                  "p_out": [host_bf16(projs[j][1]) for j in range(nl_block)],
                  "blocks": w.blocks, "seconds": args.cpu_seconds}
    del bufs, store, S, ws
    torch.cuda.empty_cache()
    return res, sample


def pca_sub_leg(args, torch, P, blk, lens, mask, k):
    """PCA initialisation on the logging workload (Sec. 3.2): the KFAC factor
    SYRK over one batch of B=8 ragged sequences for the gate layer's input x
    (n = 4096) and output gradient dy (n = 14,336), timed over back-to-back
    calls with HIP events; then the top-k eigenvectors of each factor (30 subspace
    iterations), and for dy also its top-64 (the projection width of the k = 64
    block).  Algorithmic flops of a SYRK call: valid tokens x n (n + 1)
    (the upper triangle of the symmetric product).  Then all eleven KFAC
    factors of the block in one grouped launch (block_group), beside the same
    factors as eleven calls."""
    x, dy = blk[4]                      # gate: 4096 -> 14336
    tokens = int(lens.sum())
    out = {"layer": "gate (x: 4096, dy: 14336)", "valid_tokens": tokens, "k": k, "iters": 30}
    for name, a in (("C_F", x), ("C_B", dy)):
        n = a.shape[2]
        C = torch.zeros((n, n), dtype=torch.float32, device="cuda")
        ws = torch.empty(P.logra_act_cov_ws_size(a.shape[0], a.shape[1]), dtype=torch.uint8, device="cuda")
        t = EventTimer(torch)
        P.logra_act_cov_accumulate(a, C, mask=mask, ws=ws)
        e0 = t.start()                  # one pair over back-to-back calls
        for _ in range(args.pca_reps):
            P.logra_act_cov_accumulate(a, C, mask=mask, ws=ws)
        t.stop(e0, args.pca_reps)
        Pk = torch.empty((k, n), dtype=torch.bfloat16, device="cuda")
        pws = torch.empty(P.logra_pca_ws_size(n, k), dtype=torch.uint8, device="cuda")
        te = EventTimer(torch)
        for timed in (False, True):
            e0 = te.start() if timed else None
            P.logra_pca_topk(C, k, Pk, iters=30, ws=pws)
            if timed:
                te.stop(e0)
        k64_ms = None
        if n == 14336:   # the top-64 at the widest factor
            P64 = torch.empty((64, n), dtype=torch.bfloat16, device="cuda")
            pws64 = torch.empty(P.logra_pca_ws_size(n, 64), dtype=torch.uint8, device="cuda")
            t64 = EventTimer(torch)
            for timed in (False, True):
                e0 = t64.start() if timed else None
                P.logra_pca_topk(C, 64, P64, iters=30, ws=pws64)
                if timed:
                    t64.stop(e0)
            torch.cuda.synchronize()
            k64_ms = t64.mean_ms()
            del P64, pws64
        torch.cuda.synchronize()
        flops = float(tokens) * n * (n + 1)
        tf = flops / (t.mean_ms() * 1e-3) / 1e12
        traffic, ratio = measured_traffic("act_cov", PCA_SOURCES) if n == 14336 else (None, None)
        out[name] = {"n": n, "syrk_ms": t.mean_ms(), "pca_topk_ms": te.mean_ms(), "pca_topk_k64_ms": k64_ms,
                     "roofline": {"bound": "mfma", "achieved": tf, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                  "frac": tf / BF16_PEAK_TFLOPS, "flops_per_launch": flops, "traffic": traffic,
                                  "traffic_over_algorithmic": ratio,
                                  "kernel": "k_act_cov_dma (masked bf16 SYRK)"}}
        del C, ws, Pk, pws
    # every KFAC factor of the block in one grouped launch: C_F of the four
    # distinct inputs (q/k/v share one, gate/up share one; here the q, o,
    # gate and down inputs) and C_B of the seven layers
    facts = [blk[0][0], blk[3][0], blk[4][0], blk[6][0]] + [dy_ for _, dy_ in blk]
    Cs = [torch.zeros((a.shape[2], a.shape[2]), dtype=torch.float32, device="cuda") for a in facts]
    ws = torch.empty(P.logra_act_cov_ws_size(facts[0].shape[0], facts[0].shape[1]), dtype=torch.uint8,
                     device="cuda")
    pairs = list(zip(facts, Cs))
    tg, tsep = EventTimer(torch), EventTimer(torch)
    P.logra_act_cov_accumulate_group(pairs, mask=mask, ws=ws)
    e0 = tg.start()
    for _ in range(args.pca_reps):
        P.logra_act_cov_accumulate_group(pairs, mask=mask, ws=ws)
    tg.stop(e0, args.pca_reps)
    e0 = tsep.start()
    for _ in range(args.pca_reps):
        for a, C in pairs:
            P.logra_act_cov_accumulate(a, C, mask=mask, ws=ws)
    tsep.stop(e0, args.pca_reps)
    torch.cuda.synchronize()
    flops = float(tokens) * sum(a.shape[2] * (a.shape[2] + 1) for a in facts)
    tf = flops / (tg.mean_ms() * 1e-3) / 1e12
    out["block_group"] = {
        "factors": [("C_F " if i < 4 else "C_B ") + str(a.shape[2]) for i, a in enumerate(facts)],
        "group_ms": tg.mean_ms(), "separate_calls_ms": tsep.mean_ms(),
        "roofline": {"bound": "mfma", "achieved": tf, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tf / BF16_PEAK_TFLOPS, "flops_per_launch": flops, "traffic": None,
                     "kernel": "k_act_cov_dma over the 11 KFAC factors of one Llama3-8B block (one launch)"}}
    del Cs, ws, pairs
    return out


def copy_bandwidth(torch, nbytes=2 << 30, reps=5):
    """HBM bytes moved per second (read + write) by torch's device-to-device
    copy of `nbytes` (2 GiB, far above the 256 MB MALL): a measured reference
    for what a plain streaming kernel reaches on this GPU, next to the
    published peak."""
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").normal_()
    dst = torch.empty_like(src)
    t = EventTimer(torch)
    dst.copy_(src)
    for _ in range(reps):
        e0 = t.start()
        dst.copy_(src)
        t.stop(e0)
    torch.cuda.synchronize()
    gbs = 2 * nbytes / (t.mean_ms() * 1e-3) / 1e9
    del src, dst
    return gbs


def host_bf16(t):
    import torch
    return t.contiguous().to("cpu").view(torch.int16).numpy().view(np.uint16)


def host_info(threads_used):
    """The host the oracle ran on: usable CPUs, OpenMP threads, threads the
    sample kept busy, CPU model."""
    import oracle
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count()
    return {"cores": int(threads_used), "nproc": nproc, "omp_threads": oracle.num_threads(), "cpu_model": model}


def cpu_logging_baseline(sample):
    """The oracle on the logging step's work: per-example projection of the 7
    layers of a block (Eq. (5)), parallel over (layer, example), and the
    covariance update of their blocks, over the sampled batches, repeated
    until about `seconds` have passed."""
    import oracle
    batches, target = sample["batches"], sample["seconds"]
    toks, passes, t0 = 0, 0, time.perf_counter()
    nl = len(sample["p_in"])
    while True:
        for b in batches:
            gs = oracle.project_factored_layers([(b["x"][j], b["dy"][j], sample["p_in"][j], sample["p_out"][j])
                                                 for j in range(nl)], b["mask"])
            for g in gs:
                oracle.cov_accumulate(g)
            toks += int(b["mask"].sum())
        passes += 1
        if time.perf_counter() - t0 >= target:
            break
    dt = time.perf_counter() - t0
    B, T = batches[0]["mask"].shape
    # each sampled batch goes through one block; the step runs `blocks` blocks
    out = {"value": toks / (dt * sample["blocks"]), "unit": "tokens/s", "kind": "oracle"}
    out.update(host_info(min(oracle.num_threads(), nl * B)))
    out["sample"] = (f"{len(batches)} batches of {B} examples x {T} token slots through the {nl} layers "
                     f"(projection, parallel over {nl} layers x {B} examples, and covariance update) of one "
                     f"block, {passes} passes, {toks} valid tokens in {dt:.1f} s, scaled to {sample['blocks']} blocks")
    return out


# ------------------------------------------------------- k = 64 block leg --
def block_k64_leg(args, torch, P):
    """One Llama3-8B block at k = 64: 7 layers, B = 16, T = 1024, every token
    valid; the fused projection into bf16 rows of 7 x 4,096, then the 7
    covariance blocks of 4,096 x 4,096 (fp32) updated from those rows.  Two
    distinct x / dy sets (2.7 GB each, far above the 256 MB MALL) alternate
    between launches."""
    w = W.WORKLOADS["llama3_8b_block"]
    B, T, k = w.B, w.T, w.k_in
    D, nl = k * k, len(w.layers)
    log(f"[k64] allocating 2 x/dy sets of one block, B={B} T={T} k={k}")
    gen = W.torch_generator(args.seed, 150)
    sets = []
    for _ in range(2):
        st = []
        for (_, ni, no) in w.layers:
            x = torch.empty((B, T, ni), dtype=torch.bfloat16, device="cuda")
            dy = torch.empty((B, T, no), dtype=torch.bfloat16, device="cuda")
            W.device_normal_(x, w.x_std, gen)
            W.device_normal_(dy, w.dy_std, gen)
            st.append((x, dy))
        sets.append(st)
    projs = []
    for (_, ni, no) in w.layers:
        pi = torch.empty((k, ni), dtype=torch.bfloat16, device="cuda")
        po = torch.empty((k, no), dtype=torch.bfloat16, device="cuda")
        W.device_normal_(pi, 1.0 / np.sqrt(k), gen)
        W.device_normal_(po, 1.0 / np.sqrt(k), gen)
        projs.append((pi, po))
    store = torch.empty((B, nl * D), dtype=torch.bfloat16, device="cuda")
    S = torch.zeros((nl, D, D), dtype=torch.float32, device="cuda")
    descs = []
    for st in sets:
        arr = (P.LayerDesc * nl)()
        for j, (_, ni, no) in enumerate(w.layers):
            arr[j] = P.LayerDesc(st[j][0].data_ptr(), st[j][1].data_ptr(), projs[j][0].data_ptr(),
                                 projs[j][1].data_ptr(), store[:, j * D:(j + 1) * D].data_ptr(), ni, no)
        descs.append(arr)
    L = P.lib()
    wsb = P.logra_project_layers_ws_size(descs[0], nl, B, T, k, k)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)

    def project(i):
        rc = L.logra_project_layers(descs[i % 2], nl, P.BF16, B, T, None, k, k, P.BF16, store.stride(0),
                                    ctypes.c_void_p(ws.data_ptr()), wsb, stream)
        if rc != 0:
            raise P.LograError(rc, P.logra_last_error())

    def cov(fn=L.logra_cov_accumulate_blocks_lower):
        rc = fn(ctypes.c_void_p(store.data_ptr()), P.BF16, store.stride(0), B, D, nl,
                ctypes.c_void_p(S.data_ptr()), stream)
        if rc != 0:
            raise P.LograError(rc, P.logra_last_error())

    reps = args.k64_reps
    for i in range(3):
        project(i)
        cov()
    torch.cuda.synchronize()
    pt, ct, st = EventTimer(torch), EventTimer(torch), EventTimer(torch)
    e0 = pt.start()
    for i in range(reps):
        project(i)
    pt.stop(e0, reps)
    e0 = ct.start()
    for _ in range(reps):
        cov()
    ct.stop(e0, reps)
    # the symmetric form of the same update, for reference (not part of the step)
    S.zero_()
    cov(L.logra_cov_accumulate_blocks)
    e0 = st.start()
    for _ in range(reps):
        cov(L.logra_cov_accumulate_blocks)
    st.stop(e0, reps)
    torch.cuda.synchronize()
    tokens = B * T
    per_tok = sum(2 * (ni + no) for _, ni, no in w.layers)
    p_bytes = sum(2 * k * (ni + no) for _, ni, no in w.layers)
    proj_bytes = tokens * per_tok + p_bytes
    proj_ms = pt.mean_ms()
    ach = proj_bytes / (proj_ms * 1e-3) / 1e9
    # covariance kept as its lower triangle (all the preconditioner reads): that
    # triangle read and written once, plus the store rows
    cov_bytes = nl * 4 * 2 * (D * (D + 1) // 2) + B * nl * D * 2
    cov_ms = ct.mean_ms()
    cach = cov_bytes / (cov_ms * 1e-3) / 1e9
    # the symmetric form reads the upper triangle and writes all of S
    sym_bytes = nl * 4 * (D * (D + 1) // 2 + D * D) + B * nl * D * 2
    sym_ms = st.mean_ms()
    traffic, ratio = measured_traffic("projection_k64", PROJ_SOURCES)
    res = {
        "metric": "projected per-example grads/sec (tokens/s), one Llama3-8B block at k=64",
        "value": tokens / ((proj_ms + cov_ms) * 1e-3), "unit": "tokens/s",
        "examples_per_s": B / ((proj_ms + cov_ms) * 1e-3),
        "proj_launch_ms": proj_ms, "cov_launch_ms": cov_ms,
        "cov_symmetric_launch_ms": sym_ms,
        "cov_symmetric_gbs": sym_bytes / (sym_ms * 1e-3) / 1e9,
        "config": {"workload": "llama3_8b_block", "layers": nl, "B": B, "T": T, "k_in": k, "k_out": k,
                   "store": "bf16 rows of 7 x 4,096",
                   "covariance": "7 x 4,096 x 4,096 fp32, lower triangles"},
        "roofline": {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": ach / HBM_PEAK_GBS, "traffic": traffic, "traffic_over_algorithmic": ratio,
                     "kernel": "logra_project_layers (7 Llama3-8B layers, B=16, T=1024, k=64)",
                     "bytes_per_launch": proj_bytes},
        "cov_roofline": {"bound": "hbm", "achieved": cach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": cach / HBM_PEAK_GBS, "bytes_per_launch": cov_bytes,
                         "kernel": "logra_cov_accumulate_blocks_lower (7 blocks of 4,096, 16 bf16 rows)"},
    }
    sample = None
    if args.cpu_baseline:
        nb = args.k64_cpu_examples
        sample = {"x": [host_bf16(sets[0][j][0][:nb]) for j in range(nl)],
                  "dy": [host_bf16(sets[0][j][1][:nb]) for j in range(nl)],
                  "p_in": [host_bf16(p[0]) for p in projs], "p_out": [host_bf16(p[1]) for p in projs],
                  "seconds": args.cpu_seconds / 2}
    del sets, store, S, ws
    torch.cuda.empty_cache()
    return res, sample


def cpu_block_k64_baseline(sample):
    """The oracle on a bounded sample of the k = 64 block: the projection of
    the 7 layers for a few examples (parallel over layer x example) and the
    covariance update of the 7 blocks from those examples' rows."""
    import oracle
    nl = len(sample["x"])
    passes, t0 = 0, time.perf_counter()
    while True:
        gs = oracle.project_factored_layers([(sample["x"][j], sample["dy"][j], sample["p_in"][j],
                                              sample["p_out"][j]) for j in range(nl)])
        for g in gs:
            oracle.cov_accumulate(g)
        passes += 1
        if time.perf_counter() - t0 >= sample["seconds"]:
            break
    dt = time.perf_counter() - t0
    B, T = sample["x"][0].shape[:2]
    out = {"value": passes * B * T / dt, "unit": "tokens/s", "kind": "oracle"}
    out.update(host_info(min(oracle.num_threads(), nl * B)))
    out["sample"] = (f"{B} examples x {T} tokens through the 7 layers at k=64 (projection, parallel over "
                     f"layer x example, and the 7 covariance updates of 4,096 x 4,096), {passes} passes in "
                     f"{dt:.1f} s")
    return out


# ----------------------------------------------------- GPT-2-small leg --
def gpt2_leg(args, torch, P):
    """GPT-2-small logging: 12 blocks x {qkv, out, fc, proj}, B = 32, T = 512,
    lengths U{64..512} (right padding), k = 16, one step = one batch through
    all 48 layers in one grouped launch, into a bf16 store
    of 48 x 256 columns, then the 48 covariance blocks of 256 x 256 updated
    from the step's rows.  Each block has its own x / dy (403 MB per block)."""
    w = W.WORKLOADS["gpt2_small_log"]
    B, T, k = w.B, w.T, w.k_in
    D, nlb = k * k, len(w.layers)
    nl = w.blocks * nlb
    log(f"[gpt2] allocating {w.blocks} blocks x {nlb} layers, B={B} T={T} k={k}")
    gen = W.torch_generator(args.seed, 160)
    tens = []
    for blk in range(w.blocks):
        for (_, ni, no) in w.layers:
            x = torch.empty((B, T, ni), dtype=torch.bfloat16, device="cuda")
            dy = torch.empty((B, T, no), dtype=torch.bfloat16, device="cuda")
            W.device_normal_(x, w.x_std, gen)
            W.device_normal_(dy, w.dy_std, gen)
            pi = torch.empty((k, ni), dtype=torch.bfloat16, device="cuda")
            po = torch.empty((k, no), dtype=torch.bfloat16, device="cuda")
            W.device_normal_(pi, 1.0 / np.sqrt(k), gen)
            W.device_normal_(po, 1.0 / np.sqrt(k), gen)
            tens.append((x, dy, pi, po))
    steps = args.gpt2_warmup + args.gpt2_steps
    lens = [W.lengths(W.rng(args.seed, 500, st), B, w.len_lo, w.len_hi) for st in range(steps)]
    masks = [torch.from_numpy(W.mask_from_lengths(Ls, T)).cuda() for Ls in lens]
    store = torch.empty((steps * B, nl * D), dtype=torch.bfloat16, device="cuda")
    S = torch.zeros((nl, D, D), dtype=torch.float32, device="cuda")
    group = min(nl, P.MAX_GROUP)
    L = P.lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)

    def descs(st, g0):
        n = min(group, nl - g0)
        arr = (P.LayerDesc * n)()
        for j in range(n):
            l = g0 + j
            x, dy, pi, po = tens[l]
            arr[j] = P.LayerDesc(x.data_ptr(), dy.data_ptr(), pi.data_ptr(), po.data_ptr(),
                                 store[st * B:(st + 1) * B, l * D:(l + 1) * D].data_ptr(), x.shape[2], dy.shape[2])
        return arr, n

    all_d = [[descs(st, g0) for g0 in range(0, nl, group)] for st in range(steps)]
    wsb = max(P.logra_project_layers_ws_size(d, n, B, T, k, k) for d, n in all_d[0])
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    pt = EventTimer(torch)

    def step(st, timed):
        e0 = pt.start() if timed else None
        for d, n in all_d[st]:
            rc = L.logra_project_layers(d, n, P.BF16, B, T, ctypes.c_void_p(masks[st].data_ptr()), k, k, P.BF16,
                                        store.stride(0), ctypes.c_void_p(ws.data_ptr()), wsb, stream)
            if rc != 0:
                raise P.LograError(rc, P.logra_last_error())
        if timed:
            pt.stop(e0, len(all_d[st]))
        rows = store[st * B:(st + 1) * B]
        rc = L.logra_cov_accumulate_blocks_lower(ctypes.c_void_p(rows.data_ptr()), P.BF16, store.stride(0), B, D,
                                                 nl, ctypes.c_void_p(S.data_ptr()), stream)
        if rc != 0:
            raise P.LograError(rc, P.logra_last_error())

    for st in range(args.gpt2_warmup):
        step(st, False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for st in range(args.gpt2_warmup, steps):
        step(st, True)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    tokens = int(sum(int(Ls.sum()) for Ls in lens[args.gpt2_warmup:]))
    per_tok = sum(2 * (ni + no) for _, ni, no in w.layers) * (group // nlb)
    p_bytes = sum(2 * k * (ni + no) for _, ni, no in w.layers) * (group // nlb)
    launch_bytes = tokens / args.gpt2_steps * per_tok + p_bytes
    ach = launch_bytes / (pt.mean_ms() * 1e-3) / 1e9
    res = {
        "metric": "projected per-example grads/sec (tokens/s), GPT-2-small logging (48 layers, k=16)",
        "value": tokens / dt, "unit": "tokens/s", "examples_per_s": args.gpt2_steps * B / dt,
        "ms_per_step": dt * 1e3 / args.gpt2_steps, "proj_launch_ms": pt.mean_ms(), "steps": args.gpt2_steps,
        "config": {"workload": "gpt2_small_log", "blocks": w.blocks, "layers": nl, "B": B, "T": T,
                   "len_range": [w.len_lo, w.len_hi], "k_in": k, "k_out": k, "layers_per_launch": group},
        "roofline": {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": ach / HBM_PEAK_GBS, "traffic": None,
                     "kernel": f"logra_project_layers ({group} GPT-2-small layers, B=32 ragged, k=16)",
                     "bytes_per_launch": launch_bytes},
    }
    sample = None
    if args.cpu_baseline:
        sample = {"x": [host_bf16(t[0]) for t in tens[:nlb]], "dy": [host_bf16(t[1]) for t in tens[:nlb]],
                  "p_in": [host_bf16(t[2]) for t in tens[:nlb]], "p_out": [host_bf16(t[3]) for t in tens[:nlb]],
                  "mask": W.mask_from_lengths(lens[0], T), "blocks": w.blocks, "seconds": args.cpu_seconds / 2}
    del tens, store, S, ws
    torch.cuda.empty_cache()
    return res, sample


def cpu_gpt2_baseline(sample):
    """The oracle on one block of one GPT-2-small batch (the 4 layers,
    parallel over layer x example, and their covariance updates), repeated for
    about `seconds`, scaled to the 12 blocks of a step."""
    import oracle
    nl = len(sample["x"])
    toks, passes, t0 = 0, 0, time.perf_counter()
    while True:
        gs = oracle.project_factored_layers([(sample["x"][j], sample["dy"][j], sample["p_in"][j],
                                              sample["p_out"][j]) for j in range(nl)], sample["mask"])
        for g in gs:
            oracle.cov_accumulate(g)
        toks += int(sample["mask"].sum())
        passes += 1
        if time.perf_counter() - t0 >= sample["seconds"]:
            break
    dt = time.perf_counter() - t0
    B, T = sample["mask"].shape
    out = {"value": toks / (dt * sample["blocks"]), "unit": "tokens/s", "kind": "oracle"}
    out.update(host_info(min(oracle.num_threads(), nl * B)))
    out["sample"] = (f"one batch of {B} examples x {T} token slots through the {nl} layers of one block "
                     f"(projection and covariance update), {passes} passes, {toks} valid tokens in {dt:.1f} s, "
                     f"scaled to {sample['blocks']} blocks")
    return out


# ---------------------------------------------------------------- influence --
def influence_leg(args, torch, P):
    w = W.WORKLOADS["llama3_8b_scores"]
    ex = w.extra
    D = w.D
    nb = w.n_layers
    D_tot = nb * D
    N, Q, Nc, topk = args.n_train or ex["N_train"], ex["Q"], ex["N_cov"], ex["topk"]
    dev = "cuda"
    scales = W.block_scales(args.seed, nb, ex["scale_lo"], ex["scale_hi"])
    log(f"[inf] drawing train store {N} x {D_tot}, {Q} test and {Nc} covariance gradients")
    gen = W.torch_generator(args.seed, 300)
    train = torch.empty((N, D_tot), dtype=torch.bfloat16, device=dev)
    W.device_scaled_rows_(train, scales, D, gen)
    test = torch.empty((Q, D_tot), dtype=torch.bfloat16, device=dev)
    W.device_scaled_rows_(test, scales, D, gen)
    covg = torch.empty((Nc, D_tot), dtype=torch.bfloat16, device=dev)
    W.device_scaled_rows_(covg, scales, D, gen)
    S = torch.zeros((nb, D, D), dtype=torch.float32, device=dev)
    P.logra_cov_accumulate_blocks(covg, S, D)
    pre = torch.empty((Q, D_tot), dtype=torch.bfloat16, device=dev)
    pws = torch.empty(P.logra_precondition_ws_size(D, nb, Q), dtype=torch.uint8, device=dev)
    tv = torch.empty((Q, topk), dtype=torch.float32, device=dev)
    ti = torch.empty((Q, topk), dtype=torch.int64, device=dev)
    sws = torch.empty(P.logra_influence_ws_size(Q, N, topk, False), dtype=torch.uint8, device=dev)
    pre_timer, gemm_timer = EventTimer(torch), EventTimer(torch)

    def one_pass(timed):
        e0 = pre_timer.start() if timed else None
        P.logra_precondition_blocks(S, Nc, ex["damp"], test, pre, ws=pws)   # synchronous
        if timed:
            pre_timer.stop(e0)
        e0 = gemm_timer.start() if timed else None
        P.logra_influence_scores(pre, train, scores=None, topk=topk, topk_val=tv, topk_idx=ti, ws=sws)
        if timed:
            gemm_timer.stop(e0)

    log("[inf] warmup pass")
    one_pass(False)
    torch.cuda.synchronize()
    log(f"[inf] timing {args.inf_passes} passes")
    t0 = time.perf_counter()
    for _ in range(args.inf_passes):
        one_pass(True)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / args.inf_passes
    flops = 2.0 * Q * N * D_tot
    # the GEMM alone, from events around a scores-only launch (top-k excluded)
    s_full = sws.view(torch.float32)[: Q * N].view(Q, N)
    only = EventTimer(torch)
    for _ in range(args.inf_passes):
        e0 = only.start()
        P.logra_influence_scores(pre, train, scores=s_full, topk=0)
        only.stop(e0)
    torch.cuda.synchronize()
    gemm_ms = only.mean_ms()
    achieved = flops / (gemm_ms * 1e-3) / 1e12
    traffic, ratio = measured_traffic("scores", SCORE_SOURCES)
    res = {
        "metric": "influence scores/sec (1,024 x 500,000 at 57,344 dims, top-100)",
        "value": Q * N / dt, "unit": "scores/s", "ms_per_pass": dt * 1e3,
        "precondition_ms": pre_timer.mean_ms(), "scores_topk_ms": gemm_timer.mean_ms(),
        "gemm_ms": gemm_ms,
        "config": {"workload": "llama3_8b_scores", "N_train": N, "Q": Q, "D": D_tot, "blocks": nb,
                   "block": D, "N_cov": Nc, "damp": ex["damp"], "topk": topk},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / BF16_PEAK_TFLOPS, "traffic": traffic, "traffic_over_algorithmic": ratio,
                     "kernel": "score GEMM (bf16 MFMA, fp32 accumulation)", "flops_per_launch": flops},
    }
    if args.relatif:
        res["relatif"] = relatif_sub_leg(args, torch, P, S, Nc, ex["damp"], pre, train, topk, sws, tv, ti)
    if args.ooc_rows > 0:
        res["out_of_core"] = out_of_core_sub_leg(args, torch, P, pre, train, topk)
    if args.ooc_file_rows > 0:
        res["store_file"] = store_file_sub_leg(args, torch, P, pre, train, topk)
    if args.vendor_gemm:
        # the same operands through torch's library GEMM (hipBLASLt) and through this
        # library's scores-only path, on a 125,000-row slice (context for the roofline)
        nv = min(N, 125_000)
        sv = torch.empty((Q, nv), dtype=torch.float32, device=dev)
        sb = torch.empty((Q, nv), dtype=torch.bfloat16, device=dev)   # torch keeps the input dtype
        tv_, to_ = EventTimer(torch), EventTimer(torch)
        for timed in (False, True, True, True):
            e0 = tv_.start() if timed else None
            torch.matmul(pre, train[:nv].T, out=sb)
            if timed:
                tv_.stop(e0)
            e0 = to_.start() if timed else None
            P.logra_influence_scores(pre, train[:nv], scores=sv, topk=0)
            if timed:
                to_.stop(e0)
        torch.cuda.synchronize()
        fl = 2.0 * Q * nv * D_tot
        res["vendor_gemm"] = {"rows": nv, "torch_output": "bf16", "torch_matmul_ms": tv_.mean_ms(),
                              "torch_matmul_tflops": fl / tv_.mean_ms() / 1e9,
                              "logra_ms": to_.mean_ms(), "logra_tflops": fl / to_.mean_ms() / 1e9}
        del sv, sb
    sample = None
    if args.cpu_baseline:
        ns = args.cpu_train_rows
        sample = {"S": S[:, :, :].to("cpu").numpy().astype(np.float64), "N": Nc, "damp": ex["damp"],
                  "test": host_bf16(test[:args.cpu_queries]), "train": host_bf16(train[:ns]), "D": D,
                  "topk": topk}
    del train, test, covg, sws
    torch.cuda.empty_cache()
    return res, sample


def relatif_sub_leg(args, torch, P, S, Nc, damp, pre, train, topk, sws, tv, ti):
    """l-RelatIF on the same store: the self-influence of every train row
    (once per store: sum over blocks of g^T (C + lambda I)^{-1} g, two bf16
    MFMA products with the split inverse factor), then the score pass with the
    1/sqrt(self) column scales applied before the top-k."""
    N = train.shape[0]
    nb, D, _ = S.shape
    rsq = torch.empty(N, dtype=torch.float32, device=train.device)
    iws = torch.empty(P.logra_self_influence_ws_size(D, nb), dtype=torch.uint8, device=train.device)
    self_t, scaled_t = EventTimer(torch), EventTimer(torch)
    log("[inf] l-RelatIF: self-influence of the store, scaled score passes")
    for timed in [False] + [True] * args.inf_passes:
        e0 = self_t.start() if timed else None
        P.logra_self_influence_blocks(S, Nc, damp, train, rsqrt_out=rsq, ws=iws)   # synchronous
        if timed:
            self_t.stop(e0)
        e0 = scaled_t.start() if timed else None
        P.logra_influence_scores(pre, train, scores=None, topk=topk, topk_val=tv, topk_idx=ti, ws=sws,
                                 col_scale=rsq)
        if timed:
            scaled_t.stop(e0)
    torch.cuda.synchronize()
    flops = 4.0 * N * nb * D * D
    tf = flops / (self_t.mean_ms() * 1e-3) / 1e12
    traffic, ratio = measured_traffic("self_influence", SELF_SOURCES)
    return {"self_influence_ms": self_t.mean_ms(), "scaled_scores_topk_ms": scaled_t.mean_ms(),
            "roofline": {"bound": "mfma", "achieved": tf, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": tf / BF16_PEAK_TFLOPS, "traffic": traffic, "traffic_over_algorithmic": ratio,
                         "kernel": "self-influence call (inverse factor + bf16 MFMA products)",
                         "flops_per_launch": flops},
            "note": "self-influence runs once per store (timed over the whole call, factorisation "
                    "included); each query batch pays the preconditioner and the scaled score pass"}


def out_of_core_sub_leg(args, torch, P, pre, train, topk):
    """The same scoring with the store in pinned host memory, streamed over
    PCIe in chunks through two device staging buffers while the previous
    chunk is scored.  Bound: the host-to-device link; the reference is a
    plain host-to-device copy of the same bytes."""
    n = min(args.ooc_rows, train.shape[0])
    chunk = min(args.ooc_chunk, n)
    Q, D = pre.shape
    log(f"[inf] out-of-core: {n} rows in pinned host memory, chunks of {chunk}")
    host = torch.empty((n, D), dtype=train.dtype, pin_memory=True)
    host.copy_(train[:n])
    tv = torch.empty((Q, topk), dtype=torch.float32, device=train.device)
    ti = torch.empty((Q, topk), dtype=torch.int64, device=train.device)
    ws = torch.empty(P.logra_influence_stream_ws_size(Q, chunk, D, P.BF16, topk), dtype=torch.uint8,
                     device=train.device)
    ts = []
    for timed in (False, True):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        P.logra_influence_stream(pre, host, topk, tv, ti, chunk, ws=ws)   # synchronous
        if timed:
            ts.append(time.perf_counter() - t0)
    dev_buf = train[:n]          # a plain copy of the same bytes over the same link
    ct = EventTimer(torch)
    for timed in (False, True):
        e0 = ct.start() if timed else None
        dev_buf.copy_(host, non_blocking=True)
        if timed:
            ct.stop(e0)
    torch.cuda.synchronize()
    nbytes = float(n) * D * 2
    sec = float(np.mean(ts))
    gbs = nbytes / sec / 1e9
    copy_gbs = nbytes / (ct.mean_ms() * 1e-3) / 1e9
    del host, ws
    return {"rows": n, "chunk_rows": chunk, "ms_per_pass": sec * 1e3, "scores_per_s": Q * n / sec,
            "roofline": {"bound": "pcie", "achieved": gbs, "peak": PCIE_PEAK_GBS, "unit": "GB/s",
                         "frac": gbs / PCIE_PEAK_GBS, "plain_copy_gbs": copy_gbs,
                         "kernel": "host-to-device stream of the store (copies overlapped with scoring)"}}


def store_file_sub_leg(args, torch, P, pre, train, topk):
    """The disk tier of the out-of-core store: `ooc_file_rows` store rows
    written from the device to a file with write-behind (logra_offload_rows_file,
    two pinned buffers of one batch each), flushed to the device, then scored
    from the file with logra_influence_stream_file (reader thread, pinned
    double buffer, device double buffer).  The file's pages are evicted from
    the page cache (posix_fadvise) before each pass, so the reads come from the
    disk; the bound is the disk's read rate, measured beside it with plain
    sequential reads of the same file into pinned memory."""
    import shutil
    import tempfile
    n = min(args.ooc_file_rows, train.shape[0])
    Q, D = pre.shape
    rb = D * 2
    nbytes = n * rb
    tmpdir = os.environ.get("TMPDIR", tempfile.gettempdir())
    free = shutil.disk_usage(tmpdir).free
    if free < 2 * nbytes:
        return {"skipped": f"{free / 1e9:.1f} GB free in {tmpdir}, need {2 * nbytes / 1e9:.1f}"}
    log(f"[inf] store file: {n} rows ({nbytes / 1e9:.2f} GB) in {tmpdir}")
    fd_, path = tempfile.mkstemp(prefix="logra_store_", dir=tmpdir)
    os.close(fd_)
    batch = args.ooc_file_batch
    try:
        fd = os.open(path, os.O_RDWR | os.O_TRUNC)
        bufs = [torch.empty(batch * rb, dtype=torch.uint8).pin_memory() for _ in range(2)]
        events, stats = [], []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i, r0 in enumerate(range(0, n, batch)):
            if i >= 2:
                events[i - 2].synchronize()
            st, ev = ctypes.c_int(-7), torch.cuda.Event()
            P.logra_offload_rows_file(train[r0:min(n, r0 + batch)], fd, r0 * rb, bufs[i % 2], io_status=st, done=ev)
            events.append(ev)
            stats.append(st)
        torch.cuda.synchronize()
        t_write = time.perf_counter() - t0
        os.fsync(fd)
        t_sync = time.perf_counter() - t0
        os.close(fd)
        assert all(st.value == P.OK for st in stats), "a store write failed"
        # evict the file's pages, so that the stream reads the disk, not the page cache
        fd = os.open(path, os.O_RDONLY)
        os.posix_fadvise(fd, 0, 0, os.POSIX_FADV_DONTNEED)
        os.close(fd)
        chunk = min(args.ooc_file_chunk, n)
        hb = torch.empty(2 * ((chunk * rb + 255) // 256 * 256), dtype=torch.uint8).pin_memory()
        tv = torch.empty((Q, topk), dtype=torch.float32, device=train.device)
        ti = torch.empty((Q, topk), dtype=torch.int64, device=train.device)
        ws = torch.empty(P.logra_influence_stream_file_ws_size(Q, chunk, D, P.BF16, topk), dtype=torch.uint8,
                         device=train.device)
        fd = os.open(path, os.O_RDONLY)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        P.logra_influence_stream_file(pre, fd, 0, n, D, P.BF16, topk, tv, ti, chunk, hb, ws=ws)   # synchronous
        t_stream = time.perf_counter() - t0
        os.posix_fadvise(fd, 0, 0, os.POSIX_FADV_DONTNEED)
        # the disk alone: the same file read sequentially into the same pinned buffer
        view = hb[: chunk * rb].numpy()
        t0 = time.perf_counter()
        for r0 in range(0, n, chunk):
            rows = min(chunk, n - r0)
            os.preadv(fd, [memoryview(view[: rows * rb])], r0 * rb)
        t_read = time.perf_counter() - t0
        os.close(fd)
        gbs, read_gbs = nbytes / t_stream / 1e9, nbytes / t_read / 1e9
        return {"rows": n, "chunk_rows": chunk, "read_mode": "page cache evicted before each pass", "dir": tmpdir,
                "write_gbs": nbytes / t_write / 1e9, "write_gbs_with_fsync": nbytes / t_sync / 1e9,
                "ms_per_pass": t_stream * 1e3, "scores_per_s": Q * n / t_stream,
                "roofline": {"bound": "disk", "achieved": gbs, "peak": read_gbs, "unit": "GB/s",
                             "frac": gbs / read_gbs,
                             "kernel": "store file streamed through the reader thread and two pinned buffers "
                                       "(scoring overlapped)",
                             "peak_is": "plain sequential reads of the same file into pinned memory"}}
    finally:
        os.unlink(path)


def cpu_influence_baseline(sample):
    import oracle
    D = sample["D"]
    nb = sample["S"].shape[0]
    t0 = time.perf_counter()
    pre = np.concatenate([oracle.precondition(sample["S"][l], sample["N"], sample["damp"],
                                              sample["test"][:, l * D:(l + 1) * D])[0] for l in range(nb)], axis=1)
    s = oracle.scores(pre, sample["train"])
    oracle.topk(s, sample["topk"])
    dt = time.perf_counter() - t0
    q, n = s.shape
    out = {"value": q * n / dt, "unit": "scores/s", "kind": "oracle"}
    out.update(host_info(oracle.num_threads()))
    out["sample"] = f"{q} queries x {n} stored gradients (224 blocks preconditioned, scores, top-100); {dt:.1f} s"
    return out


# --------------------------------------------------------------------- main --
def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--inf-passes", type=int, default=3)
    ap.add_argument("--n-train", type=int, default=0, help="override stored-gradient count (testing)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--leg", choices=["all", "log", "influence", "k64", "gpt2"], default="all")
    ap.add_argument("--k64-reps", type=int, default=20, help="timed launches of the k = 64 block leg")
    ap.add_argument("--log-group-blocks", type=int, default=4, choices=(1, 2, 4),
                    help="Llama3-8B blocks (7 layers each) per grouped projection launch of the logging leg")
    ap.add_argument("--no-peaks", dest="peaks", action="store_false",
                    help="skip the measured MFMA and HBM ceilings")
    ap.add_argument("--peak-ms", type=float, default=60.0, help="duration of the MFMA ceiling loop at spec rate")
    ap.add_argument("--k64-cpu-examples", type=int, default=4, help="examples in the k = 64 oracle sample")
    ap.add_argument("--gpt2-steps", type=int, default=10, help="timed steps of the GPT-2-small leg")
    ap.add_argument("--gpt2-warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", dest="cpu_baseline", action="store_false")
    ap.add_argument("--no-relatif", dest="relatif", action="store_false",
                    help="skip the l-RelatIF sub-leg (self-influence + scaled scores)")
    ap.add_argument("--no-shared-inputs", dest="shared_inputs", action="store_false",
                    help="skip the logging pass with the inputs a transformer block shares")
    ap.add_argument("--no-offload", dest="offload", action="store_false",
                    help="skip the logging pass that copies each step's store rows to pinned host memory")
    ap.add_argument("--no-pca", dest="pca", action="store_false",
                    help="skip the PCA sub-leg (KFAC factor SYRK and top-k eigenvectors)")
    ap.add_argument("--pca-reps", type=int, default=3, help="timed SYRK calls per factor")
    ap.add_argument("--ooc-rows", type=int, default=131072,
                    help="rows of the out-of-core sub-leg's pinned host store (0 = skip)")
    ap.add_argument("--ooc-chunk", type=int, default=32768, help="rows per streamed chunk")
    ap.add_argument("--ooc-file-rows", type=int, default=16384,
                    help="rows of the store-file sub-leg (written to TMPDIR, then streamed; 0 = skip)")
    ap.add_argument("--ooc-file-batch", type=int, default=1024, help="rows per write-behind batch")
    ap.add_argument("--ooc-file-chunk", type=int, default=2048, help="rows per chunk read from the store file")
    ap.add_argument("--no-vendor-gemm", dest="vendor_gemm", action="store_false",
                    help="skip timing torch.matmul (hipBLASLt) on a slice of the score GEMM's operands")
    ap.add_argument("--cpu-batches", type=int, default=2, help="logging batches in the oracle sample")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="oracle time bound of the logging sample")
    ap.add_argument("--cpu-queries", type=int, default=256, help="test gradients in the oracle sample")
    ap.add_argument("--cpu-train-rows", type=int, default=20000, help="stored gradients in the oracle sample")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/traffic.json from rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE counter "
                         "files of this benchmark, and exit (no GPU needed)")
    args = ap.parse_args()
    if args.write_traffic:
        write_traffic(*args.write_traffic)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path; a data-parallel run would "
              "give each GPU its own slice of the batches and of the gradient store",
              file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2405_13954_amd as P
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    P.lib()

    out = {"metric": METRIC, "value": None, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": None, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": "llama3_8b_stream", "blocks": 32, "layers": 224, "B": 8, "T": 2048,
                      "len_range": [128, 2048], "k_in": 16, "k_out": 16, "store": "bf16 rows of 57,344",
                      "layers_per_launch": 7 * args.log_group_blocks}}
    log_sample = inf_sample = None
    peaks = None
    if args.peaks:
        log("[peaks] MFMA loop and HBM read stream")
        peaks = peaks_leg(args, torch)
        out["peaks"] = peaks
    if args.leg in ("all", "log"):
        r, log_sample = logging_leg(args, torch, P)
        out.update(value=r["tokens_per_s"], ms_per_step=r["ms_per_step"], examples_per_s=r["examples_per_s"],
                   roofline=r["roofline"], proj_launch_ms=r["proj_launch_ms"], cov_launch_ms=r["cov_launch_ms"])
        for key in ("pca", "shared_inputs", "offload"):
            if key in r:
                out[key] = r[key]
    k64_sample = gpt2_sample = None
    if args.leg in ("all", "k64"):
        r, k64_sample = block_k64_leg(args, torch, P)
        out["llama3_8b_block"] = r
    if args.leg in ("all", "gpt2"):
        r, gpt2_sample = gpt2_leg(args, torch, P)
        out["gpt2_small_log"] = r
    if args.leg in ("all", "influence"):
        r, inf_sample = influence_leg(args, torch, P)
        out["influence"] = r
    if args.cpu_baseline:
        if log_sample is not None:
            log("[cpu] oracle on the logging sample")
            out["cpu_baseline"] = cpu_logging_baseline(log_sample)
        if k64_sample is not None:
            log("[cpu] oracle on the k = 64 block sample")
            out["llama3_8b_block"]["cpu_baseline"] = cpu_block_k64_baseline(k64_sample)
        if gpt2_sample is not None:
            log("[cpu] oracle on the GPT-2-small sample")
            out["gpt2_small_log"]["cpu_baseline"] = cpu_gpt2_baseline(gpt2_sample)
        if inf_sample is not None:
            log("[cpu] oracle on the influence sample")
            out.setdefault("influence", {})["cpu_baseline"] = cpu_influence_baseline(inf_sample)
    if peaks is not None:   # each roofline also against the measured ceiling of its bound
        for r in [out.get("roofline"), out.get("influence", {}).get("roofline"),
                  out.get("influence", {}).get("relatif", {}).get("roofline"),
                  out.get("llama3_8b_block", {}).get("roofline"), out.get("llama3_8b_block", {}).get("cov_roofline"),
                  out.get("gpt2_small_log", {}).get("roofline"),
                  out.get("pca", {}).get("C_F", {}).get("roofline"), out.get("pca", {}).get("C_B", {}).get("roofline"),
                  out.get("pca", {}).get("block_group", {}).get("roofline")]:
            if r:
                ceil = peaks["hbm_read_gbs"] if r["bound"] == "hbm" else peaks["mfma_bf16_tflops"]
                r["frac_of_measured_peak"] = r["achieved"] / ceil
                if r["bound"] == "mfma":
                    r["frac_of_measured_data_peak"] = r["achieved"] / peaks["mfma_bf16_data_tflops"]
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
