"""Throughput of QUASAR's per-step reconstruction on one MI355X.

One step = reconstructing every matrix of the workload once (all of
Algorithm 1 for every group: optional fused EMA, codes for every clip,
weighted fit, score, argmin, emit codes / scale / zero / r), with the inputs
already resident in HBM.  Prints ONE JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c3]

Workloads (paper_2608_13966_amd/synth.py): c1 single fp32 1024x1024 INT4;
c2 Qwen3-0.6B-shaped layer set INT3; c3 Llama-3.1-8B-shaped layer set INT2
g64, 12 clips, fused EMA (default); c4 the same set in NVFP4; c5 32 such
layers INT4 with fused EMA (one simulated training step); c8 the Llama set
in the Rubin INT3 LUT format with the paper's 15 clip factors; c9 the Llama
set in symmetric INT4 g128; c6 / c7 the
Llama-3.1-8B set with fp32 master weights, one fused AdamW step followed by
the INT2 / NVFP4 reconstruction (a step then includes the optimiser update).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0           # MI355X HBM3E, vendor figure
# non-packed VALU issue rate: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz (lane-ops/s)
PEAK_VALU_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
METRIC = "G weights reconstructed/s and achieved HBM GB/s (% of peak), 1 MI355X"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def source_fingerprint() -> str:
    """Hash of the HIP sources: counter readings are only valid for the
    kernels they were taken on."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_13966_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def binned_valu_ops_per_weight(wl, n_cells: int) -> float:
    """VALU lane-operations per weight of the binned INT kernel (the clips'
    moments from per-group threshold-cell sums): per weight, the range (2),
    the position u (1), its bucket (4) and cell (one compare and add: 2),
    the packed cell (1), h and h w as exact integers (conversions, product,
    sum h w^2, two scaled roundings with their high-word corrections, cell
    address: 10), the emitted code, r and pack (5), and the EMA (3); per
    group of G weights, the suffix scan (about 12 per cell), each clip's
    moments from its NB suffix sums and its ratio test (3 NB + 11 per clip)
    and one fit and score per 16 weights (about 45)."""
    K = len(wl.clips)
    qmax = (1 << (wl.bits - 1)) - 1 if wl.fmt == "int_sym" else (1 << wl.bits) - 1
    nb = 2 * qmax if wl.fmt == "int_sym" else qmax
    pre = 10.0 if wl.adamw else (3.0 if wl.ema else 0.0)
    per_group = 12.0 * n_cells + (3.0 * nb + 11.0) * K + 45.0 * (wl.group / 16)
    return 25.0 + pre + per_group / wl.group


def int_kernel_choice(wl):
    """(kernel name, cells) of the INT kernel the library takes for this
    workload's clip grid (quasar_int_path; host-only)."""
    from paper_2608_13966_amd import quasar as Q
    d = Q.Descriptor(8, wl.group, fmt=wl.fmt, bits=wl.bits, group=wl.group, clips=wl.clips,
                     w_dtype=Q.BF16 if wl.w_bf16 else Q.F32)
    if Q.quasar_int_path(d) == 1:
        return "int_cells_kernel", int_cells_count(wl)
    return "int_reconstruct_kernel", 0


def int_cells_count(wl) -> int:
    """Cells per group of the binned kernel: the distinct code thresholds of
    all clips plus one, with the clips' tie thresholds below u = 0 (odd
    qmax) counted once -- in exact arithmetic T(k, b) = (b - qmax/2 - 1/2)
    (2 f_k / qmax) for asymmetric groups and (b - Q - 1/2) (f_k / Q) for
    symmetric ones."""
    import numpy as np
    sym = wl.fmt == "int_sym"
    qmax = (1 << (wl.bits - 1)) - 1 if sym else (1 << wl.bits) - 1
    ts = set()
    for f in wl.clips:
        for b in range(1, (2 * qmax if sym else qmax) + 1):
            t = (b - qmax - 0.5) * f / qmax if sym else (b - qmax / 2 - 0.5) * 2 * f / qmax
            ts.add(round(t, 9))
    return len(ts) + 1


def algorithmic_valu_ops_per_weight(wl) -> float:
    """VALU lane-operations per weight that the method needs as computed here:
    per clip, the code (scale-shift, round, clamp; NVFP4: scale, E2M1 round)
    and the moments (one product and three accumulations; NVFP4 two); per
    weight, the range, the clip-independent moments, the EMA and the emitted
    code and r."""
    K = len(wl.clips)
    # the fused AdamW step: m (2), v (3), sqrt, fma, quotient, w*decay, fma (10);
    # the plain EMA of v: 3
    pre = 10.0 if wl.adamw else (3.0 if wl.ema else 0.0)
    if wl.fmt == "nvfp4":
        return 5.0 * K + 8.0 + pre
    if wl.fmt == "rubin":
        # per weight, once: its cell among the 7K code thresholds (7 levels of
        # a search tree: compare and descend, 14), the exact fixed-point limbs
        # of h and h w (10), range, h, h w, the clip-independent sums and the
        # normalised position (8), the emitted code, codebook lookup and pack
        # (5); per clip and block, each of the 8 codebook entries from two
        # prefix sums (about 30 lane-ops per entry, 8 x 30 / 512 per weight)
        return 37.0 + K * 8.0 * 30.0 / 512.0 + pre
    if wl.fmt in ("int", "int_sym"):
        kname, cells = int_kernel_choice(wl)
        if kname == "int_cells_kernel":
            return binned_valu_ops_per_weight(wl, cells)
    if wl.fmt == "int_sym":
        # per clip: the code (3), one product and two accumulations (3)
        return 6.0 * K + 9.0 + pre
    return 7.0 * K + 9.0 + pre


def algorithmic_bytes_per_weight(wl, amax_pass: bool) -> float:
    """What the method must move per weight: W, v (and g) read once; v' (with
    the EMA), r, the codes and the per-group parameters written once; with the
    fused AdamW step also m read and written and W written back.  The
    per-group diagnostics (chosen clip, score) are off in the benchmark."""
    wb = 2.0 if wl.w_bf16 else 4.0
    rd = wb + 4.0 + (2.0 if wl.ema else 0.0)
    wr = (4.0 if wl.ema else 0.0) + wb
    if wl.adamw:  # + m read and written, W written back; r in bf16
        rd += 4.0
        wr = 4.0 + 4.0 + wb + 2.0
    if wl.fmt == "nvfp4":
        wr += 0.5 + 1.0 / 16.0
        if amax_pass:
            rd += wb  # the tensor absmax pass reads W once more
    elif wl.fmt == "rubin":
        wr += 3.0 / 8.0 + 8.0 / 512.0   # 3-bit indices, 8 codebook bytes per 512 weights
    else:
        wr += wl.bits / 8.0 + 8.0 / wl.group
    return rd + wr


def kernel_bytes_per_weight(wl) -> float:
    """Algorithmic bytes of the reconstruct kernel alone (no absmax pass)."""
    return algorithmic_bytes_per_weight(wl, amax_pass=False)


def cpu_model() -> str:
    """The host CPU's model name (Linux /proc/cpuinfo), or the platform's."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or platform.machine()


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=int(os.environ.get("WORLD_SIZE", "1")))
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", default="c3", choices=["c1", "c2", "c3", "c4", "c5", "c6", "c7", "c8", "c9"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="CPU time (thread-seconds) the oracle baseline aims to spend; the row stride of "
                         "its sample is chosen from a short pilot run")
    ap.add_argument("--no-copy-baseline", action="store_true")
    ap.add_argument("--weighting", default="h", choices=["h", "h2", "none"],
                    help="saliency weighting variant (h: the method's default)")
    ap.add_argument("--param-dtype", default="fp32", choices=["fp32", "fp16", "bf16"],
                    help="deployed precision of the INT dequantiser (s, z)")
    ap.add_argument("--no-cpu-detail", action="store_true",
                    help="skip the oracle's literal fp32 mode and one-thread timings (reported in cpu_baseline)")
    ap.add_argument("--diagnostics", action="store_true",
                    help="report the chosen-clip histogram (GPU, whole step) and the mean score ratio to "
                         "min-max RTN at clip 1.0 (oracle sample)")
    ap.add_argument("--launch", default="batch", choices=["single", "batch"],
                    help="one kernel launch per matrix, or one quasar_reconstruct_batch launch per run of up "
                         "to 16 consecutive matrices (reconstruction workloads; the fused optimiser step "
                         "always launches per matrix)")
    args = ap.parse_args(argv)

    if args.gpus != 1:
        print(f"bench.py: runs on exactly one GPU (asked for {args.gpus}); the reconstruction would shard "
              "by rows or whole matrices with no communication, but no multi-GPU path exists.",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2608_13966_amd import quasar as Q
    from paper_2608_13966_amd import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    Q.lib()  # fail loudly without the HIP library
    wl = synth.workloads()[args.workload]
    stream = torch.cuda.current_stream(dev)

    # ---- inputs resident in HBM ---------------------------------------------
    t0 = time.time()
    mats = []
    for (name, r, c), seed in zip(wl.shapes, wl.seeds):
        W, v, g = synth.gen_matrix(r, c, seed, w_bf16=wl.w_bf16, ema=wl.ema, device=dev)
        mom = None
        if wl.adamw:
            mom, v = synth.gen_adamw_state(r, c, seed, v, device=dev)
        d = Q.Descriptor(r, c, fmt=wl.fmt, bits=wl.bits, group=wl.group, clips=wl.clips,
                         w_dtype=Q.BF16 if wl.w_bf16 else Q.F32, g_dtype=Q.BF16, beta2=wl.beta2,
                         weighting=args.weighting, param_dtype=args.param_dtype)
        out = Q.alloc_outputs(d, W, want_r=not wl.adamw, want_diag=False, has_amax=wl.fmt == "nvfp4")
        if wl.adamw:
            out["r"] = torch.empty(W.shape, dtype=torch.bfloat16, device=dev)
        out["amax"] = torch.zeros(4, dtype=torch.float32, device=dev) if wl.fmt == "nvfp4" else None
        out["amax2"] = torch.zeros(4, dtype=torch.float32, device=dev) if wl.fmt == "nvfp4" else None
        mats.append(dict(name=name, W=W, v=v, g=g, m=mom, d=d, out=out))
    footprint = sum(m["W"].numel() * (m["W"].element_size() + 4 + (2 if wl.ema else 0) + (4 if wl.adamw else 0))
                    for m in mats)
    # workloads that fit in the 256 MB last-level cache are rotated over copies
    copies = 1
    if footprint < (1 << 30):
        copies = min(64, math.ceil((1 << 30) / footprint))
        base = mats
        mats = []
        for ci in range(copies):
            for m in base:
                mm = dict(m)
                if ci:
                    o2 = Q.alloc_outputs(m["d"], m["W"], want_r=True, want_diag=False, has_amax=wl.fmt == "nvfp4")
                    if wl.adamw:
                        o2["r"] = torch.empty(m["W"].shape, dtype=torch.bfloat16, device=dev)
                    for k in ("amax", "amax2"):
                        o2[k] = None if m["out"][k] is None else torch.zeros_like(m["out"][k])
                    mm = dict(name=m["name"], W=m["W"].clone(), v=m["v"].clone(),
                              g=None if m["g"] is None else m["g"].clone(),
                              m=None if m["m"] is None else m["m"].clone(), d=m["d"], out=o2)
                mats.append(mm)
    torch.cuda.synchronize()
    setup_s = time.time() - t0
    n_per_step = wl.n_weights
    per_step = len(mats) // copies

    def launch_absmax(m):
        s = Q.quasar_absmax(m["d"], m["W"], m["out"]["amax"], stream.cuda_stream)
        if s != Q.OK:
            raise Q.QuasarError(s, "quasar_absmax")

    step_no = [0]

    def launch(m):
        o = m["out"]
        if wl.adamw:
            # one optimiser step + reconstruction; NVFP4 takes this step's
            # tensor scale from the previous step's max |W'| by-product
            opt = Q.AdamW(1e-5, 0.9, wl.beta2, 1e-8, 0.01, step_no[0] + 1)
            s = Q.quasar_adamw_reconstruct(m["d"], opt, m["W"], m["m"], m["v"], m["g"], o["codes"], o["scales"],
                                           o["zeros"], o["r"], Q.BF16, None, None, o["tensor_scale"], o["amax"],
                                           o["amax2"], stream.cuda_stream)
            if s != Q.OK:
                raise Q.QuasarError(s, "quasar_adamw_reconstruct")
            if o["amax"] is not None:
                o["amax"], o["amax2"] = o["amax2"], o["amax"]
            return
        s = Q.quasar_reconstruct(m["d"], m["W"], m["v"], m["g"], o["codes"], o["scales"], o["zeros"], o["r"],
                                 None, None, o["tensor_scale"], o["amax"], o["workspace"], o["workspace_bytes"],
                                 stream.cuda_stream)
        if s != Q.OK:
            raise Q.QuasarError(s)

    # ---- launch plan: per matrix, or batched runs of up to MAX_BATCH matrices ----
    nv = wl.fmt == "nvfp4" and not wl.adamw   # the plain NVFP4 path runs its absmax pass every step
    batched = args.launch == "batch"
    plans = []
    for ci in range(copies):
        ms = mats[ci * per_step:(ci + 1) * per_step]
        grps = [ms[i:i + Q.MAX_BATCH] for i in range(0, len(ms), Q.MAX_BATCH)] if batched else [[m] for m in ms]
        plan = []
        for grp in grps:
            arr = None
            if len(grp) > 1 and not wl.adamw:  # the fused step's arrays are built per step (see launch_group)
                arr = (Q.Matrix * len(grp))(*[Q.matrix(m["W"], m["v"], m["g"], m["out"], m["out"]["amax"])
                                              for m in grp])
                if nv:  # the group's absmax passes in one launch as well
                    arr = (arr, Q._ptr_array([m["out"]["amax"] for m in grp]))
            plan.append((grp, arr, sum(m["W"].numel() for m in grp)))
        plans.append(plan)

    def absmax_group(grp, arr):
        if arr is None:
            for m in grp:
                launch_absmax(m)
            return
        s = Q.lib().quasar_absmax_batch(grp[0]["d"].ref, arr[0], len(grp), arr[1], stream.cuda_stream)
        if s != Q.OK:
            raise Q.QuasarError(s, "quasar_absmax_batch")

    def launch_group(grp, arr):
        if wl.adamw and len(grp) > 1:
            # one batched optimiser step + reconstruction; NVFP4 takes this
            # step's tensor scale from the previous step's max |W'| by-products
            opt = Q.AdamW(1e-5, 0.9, wl.beta2, 1e-8, 0.01, step_no[0] + 1)
            am = [Q.AdamWMatrix(m["W"].shape[0], m["W"].shape[1], Q._p(m["W"]), Q._p(m["m"]), Q._p(m["v"]),
                                Q._p(m["g"]), Q._p(m["out"]["codes"]), Q._p(m["out"]["scales"]),
                                Q._p(m["out"]["zeros"]), Q._p(m["out"]["r"]), None, None,
                                Q._p(m["out"]["tensor_scale"]), Q._p(m["out"]["amax"]), Q._p(m["out"]["amax2"]))
                  for m in grp]
            s = Q.quasar_adamw_reconstruct_batch(grp[0]["d"], opt, am, Q.BF16, stream.cuda_stream)
            if s != Q.OK:
                raise Q.QuasarError(s, "quasar_adamw_reconstruct_batch")
            for m in grp:
                o = m["out"]
                if o["amax"] is not None:
                    o["amax"], o["amax2"] = o["amax2"], o["amax"]
            return
        if arr is None:
            launch(grp[0])
            return
        mats_arr = arr[0] if nv else arr
        s = Q.lib().quasar_reconstruct_batch(grp[0]["d"].ref, mats_arr, len(grp), stream.cuda_stream)
        if s != Q.OK:
            raise Q.QuasarError(s, "quasar_reconstruct_batch")

    # ---- plain copy of the same byte count: achievable bandwidth.  Measured
    # before the warmup steps, so that the GPU runs at its working clocks by
    # the time the timed steps start (it is untimed work for the step) -------
    amax_pass = wl.fmt == "nvfp4" and not wl.adamw
    bpw = algorithmic_bytes_per_weight(wl, amax_pass)
    copy_gbps = None
    if not args.no_copy_baseline:
        nbytes = min(int(n_per_step * bpw / 2), 4 << 30)
        src = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        reps = 10
        for _ in range(reps):
            dst.copy_(src)
        b.record(stream)
        torch.cuda.synchronize()
        copy_gbps = 2 * nbytes * reps / (a.elapsed_time(b) * 1e-3) / 1e9
        del src, dst

    # ---- warmup ----------------------------------------------------------------
    if wl.adamw and wl.fmt == "nvfp4":
        for m in mats:
            launch_absmax(m)                        # the first step's tensor amax
    for i in range(args.warmup):
        step_no[0] = i
        for grp, arr, _ in plans[i % copies]:
            if nv:
                absmax_group(grp, arr)
            launch_group(grp, arr)
    torch.cuda.synchronize()

    # ---- timed steps: whole-step events plus one event pair per launch ---------
    ev_start, ev_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    per_launch, per_absmax = [], []
    torch.cuda.synchronize()
    t_wall = time.time()
    ev_start.record(stream)
    for i in range(args.steps):
        step_no[0] = args.warmup + i
        for grp, arr, nw in plans[i % copies]:
            if nv:  # NVFP4: the tensor absmax pass(es), timed on their own
                a0 = torch.cuda.Event(enable_timing=True)
                a0.record(stream)
                absmax_group(grp, arr)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            launch_group(grp, arr)
            b.record(stream)
            per_launch.append((a, b, nw))
            if nv:
                per_absmax.append((a0, a))
    ev_end.record(stream)
    torch.cuda.synchronize()
    wall = time.time() - t_wall
    total_ms = ev_start.elapsed_time(ev_end)
    ms_per_step = total_ms / args.steps
    launch_ms = [a.elapsed_time(b) for a, b, _ in per_launch]
    launch_w = [n for _, _, n in per_launch]

    # per-step kernel time (sum of that step's launches) -> spread over steps
    amax_ms = [a.elapsed_time(b) for a, b in per_absmax]
    step_k = []
    per_step_launches = len(plans[0])
    for i in range(args.steps):
        sl = slice(i * per_step_launches, (i + 1) * per_step_launches)
        step_k.append(sum(launch_ms[sl]) + (sum(amax_ms[sl]) if amax_ms else 0.0))
    step_pct = [round(float(x), 4) for x in np.percentile(step_k, [10, 50, 90])]

    gw_s = n_per_step / (ms_per_step * 1e-3) / 1e9
    gbps = gw_s * bpw
    # dominant kernel: the reconstruct kernel; its algorithmic bytes over the
    # summed launch durations (the NVFP4 absmax pass is timed separately)
    kbpw = kernel_bytes_per_weight(wl)
    absmax_us = (1e3 * sum(a.elapsed_time(b) for a, b in per_absmax) / len(per_absmax)) if per_absmax else None
    k_time = sum(launch_ms) * 1e-3
    k_bytes = sum(launch_w) * kbpw
    k_gbps = k_bytes / k_time / 1e9
    avg_launch_us = 1e3 * sum(launch_ms) / len(launch_ms)

    # ---- CPU oracle on a bounded row sample (reported baseline) ----------------
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        # the CPUs this process may use, at most 16 (the host share of one
        # GPU: worker pools are sized to 16 whatever the host has)
        allowed = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
        threads = max(1, min(16, allowed))

        def oracle_rows(m, step, n_threads=None, fp32_mode=False, diag_out=None):
            nthr = threads if n_threads is None else n_threads
            if wl.fmt == "rubin":  # whole 8-row blocks
                brows = torch.arange(0, m["W"].shape[0] // 8, step, device=dev)
                rows = (brows[:, None] * 8 + torch.arange(8, device=dev)[None, :]).reshape(-1)
            else:
                rows = torch.arange(0, m["W"].shape[0], step, device=dev)
            Ws = synth.to_host(m["W"].index_select(0, rows))
            vh = synth.to_host(m["v"].index_select(0, rows))
            gh = None if m["g"] is None else synth.to_host(m["g"].index_select(0, rows))
            amax = oracle.absmax(synth.to_host(m["W"])) if wl.fmt == "nvfp4" else None
            kw = dict(fmt=wl.fmt, bits=wl.bits, group=wl.group, clips=wl.clips, tensor_amax=amax,
                      n_threads=nthr, weighting=args.weighting, param_dtype=args.param_dtype)
            if wl.adamw:
                mh = synth.to_host(m["m"].index_select(0, rows))
                t1 = time.time()
                oracle.adamw_reconstruct(Ws, mh, vh, gh, lr=1e-5, beta1=0.9, beta2=wl.beta2, eps=1e-8,
                                         weight_decay=0.01, step=1, **kw)
            elif wl.fmt == "rubin":
                t1 = time.time()
                oracle.rubin_reconstruct(Ws, vh, clips=wl.clips, g=gh, beta2=wl.beta2, weighting=args.weighting,
                                         n_threads=nthr)
            else:
                t1 = time.time()
                o = oracle.reconstruct(Ws, vh, g=gh, beta2=wl.beta2, fp32_mode=fp32_mode,
                                       want_diag=diag_out is not None, **kw)
                if diag_out is not None:
                    diag_out.append((o["err"].astype(np.float64), o["diag"][:, 0]))
            return Ws.size, time.time() - t1

        # pilot on the largest matrix, then a stride that spends about
        # --cpu-seconds of thread time over the whole step (the first pilot
        # call warms the oracle's thread pool and caches; the second is timed).
        # Each call has a fixed cost of some milliseconds, so a sample that
        # comes out far too short is taken again with a finer stride.
        big = max(mats[:per_step], key=lambda m: m["W"].numel())
        pilot_step = max(1, big["W"].shape[0] // 32)
        oracle_rows(big, pilot_step)
        pw, pt = oracle_rows(big, pilot_step)
        rate = pw / max(pt, 1e-6)
        step = max(1, math.ceil(n_per_step / (rate * args.cpu_seconds / threads)))
        for attempt in range(2):
            sample_w, t_cpu = 0, 0.0
            for m in mats[:per_step]:
                w_, t_ = oracle_rows(m, step)
                sample_w += w_
                t_cpu += t_
            spent = t_cpu * threads
            if attempt == 1 or step == 1 or spent >= 0.5 * args.cpu_seconds:
                break
            step = max(1, int(step * spent / args.cpu_seconds))
        detail = {}
        if not args.no_cpu_detail and wl.fmt in ("int", "nvfp4", "int_sym") and not wl.adamw:
            # the same sample with the literal fp32 accumulation mode, and a
            # sparser sample on one thread
            fw, ft = 0, 0.0
            for m in mats[:per_step]:
                w_, t_ = oracle_rows(m, step, fp32_mode=True)
                fw += w_
                ft += t_
            detail["fp32_mode_value"] = round(fw / ft / 1e9, 6)
            sw, stt = 0, 0.0
            for m in mats[:per_step]:
                w_, t_ = oracle_rows(m, step * 16, n_threads=1)
                sw += w_
                stt += t_
            detail["single_thread_value"] = round(sw / stt / 1e9, 6)
            detail["single_thread_sample"] = f"rows 0, {16 * step}, ... of every matrix ({sw} weights, {stt:.1f} s)"
        cpu = {"value": round(sample_w / t_cpu / 1e9, 6), "unit": "G weights/s", "cores": threads,
               "kind": "oracle", "host_cpus": os.cpu_count(), "cpus_allowed": allowed, "cpu_model": cpu_model(),
               "threads_rule": "min(16, CPUs this process may use): the host share of one GPU",
               "sample": f"{'block ' if wl.fmt == 'rubin' else ''}rows 0, {step}, {2 * step}, ... of every matrix "
                         f"of {args.workload} ({sample_w} weights, "
                         f"{t_cpu:.1f} s wall = {t_cpu * threads:.0f} thread-s on {threads} threads; "
                         f"fp64 fit/score)", **detail}

    # which roof binds: time per weight at the HBM peak vs at the VALU issue peak
    ops_w = algorithmic_valu_ops_per_weight(wl)
    k_wps = sum(launch_w) / k_time
    t_hbm, t_alu = kbpw / (PEAK_HBM_GBPS * 1e9), ops_w / (PEAK_VALU_TOPS * 1e12)
    traffic = None
    traffic_ratio = None
    prof = None
    try:
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        ent = tr.get("workloads", {}).get(args.workload)
        if ent and tr.get("source_fingerprint") == source_fingerprint():
            # measured HBM bytes per weight (calibrated FETCH_SIZE + WRITE_SIZE) per launch
            traffic = round(ent["bytes_per_weight"] * sum(launch_w) / len(launch_w))
            traffic_ratio = round(ent["bytes_per_weight"] / kbpw, 4)
            if ent.get("rocprof_avg_us") and (args.weighting, args.param_dtype) == ("h", "fp32"):
                # the committed rocprofv3 kernel trace of this workload: its
                # average kernel duration, the frac it gives, and the bench
                # line taken in the same session without the profiler
                pw = ent["rocprof_weights_per_launch"]
                p_wps = pw / (ent["rocprof_avg_us"] * 1e-6)  # weights/s inside the kernel, from the trace
                p_hbm = pw * kbpw / (ent["rocprof_avg_us"] * 1e-6) / 1e9 / PEAK_HBM_GBPS
                prof = {"rocprof_avg_us": ent["rocprof_avg_us"],
                        # the same roof as the line's frac (set below), from the trace's duration
                        "frac": round(ops_w * p_wps / 1e12 / PEAK_VALU_TOPS if t_alu > t_hbm else p_hbm, 4),
                        "hbm_frac": round(p_hbm, 4),
                        "same_session_bench_avg_launch_us": ent.get("bench_avg_launch_us"),
                        "trace_overhead": ent.get("trace_overhead"),
                        "valu_lane_ops_per_weight_measured": ent.get("valu_lane_ops_per_weight"),
                        # the VALU load by the issued count (SQ_INSTS_VALU), at this line's kernel rate
                        "valu_frac_measured": (round(ent["valu_lane_ops_per_weight"] * k_wps / 1e12 / PEAK_VALU_TOPS, 4)
                                               if ent.get("valu_lane_ops_per_weight") else None),
                        "file": f"profiles/{ent['kernel']}_{args.workload}_kernel_stats.txt"}
    except (OSError, ValueError, KeyError):
        pass
    if wl.fmt in ("int", "int_sym"):
        kname = int_kernel_choice(wl)[0]
    else:
        kname = {"nvfp4": "nvfp4_reconstruct_kernel", "rubin": "rubin_reconstruct_kernel"}[wl.fmt]
    if t_alu > t_hbm:
        achieved = ops_w * k_wps / 1e12
        roofline = {"bound": "alu", "achieved": round(achieved, 2), "peak": round(PEAK_VALU_TOPS, 2),
                    "unit": "T VALU lane-ops/s", "frac": round(achieved / PEAK_VALU_TOPS, 4), "traffic": traffic,
                    "hbm_GBps": round(k_gbps, 1), "hbm_frac": round(k_gbps / PEAK_HBM_GBPS, 4)}
    else:
        roofline = {"bound": "hbm", "achieved": round(k_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                    "frac": round(k_gbps / PEAK_HBM_GBPS, 4), "traffic": traffic,
                    "valu_Tops": round(ops_w * k_wps / 1e12, 2),
                    "valu_frac": round(ops_w * k_wps / 1e12 / PEAK_VALU_TOPS, 4)}
    roofline.update({"kernel": kname, "bytes_per_weight": kbpw, "valu_ops_per_weight": ops_w,
                     "traffic_over_algorithmic": traffic_ratio, "avg_launch_us": round(avg_launch_us, 2)})
    if prof is not None:
        roofline["profile"] = prof
    if absmax_us is not None:
        roofline["absmax_avg_launch_us"] = round(absmax_us, 2)
    line = {
        "metric": METRIC, "value": round(gw_s, 3), "unit": "G weights/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"{args.workload}: {wl.description}", "matrices": per_step,
                   "weights_per_step": n_per_step,
                   "format": {"nvfp4": "nvfp4", "rubin": "rubin-int3-lut",
                              "int_sym": f"int{wl.bits}-symmetric"}.get(wl.fmt, f"int{wl.bits}"),
                   "group": wl.group, "clips": len(wl.clips), "fused_ema": wl.ema,
                   "io": (("fp32 W (updated), bf16 r, fp32 m and v, bf16 g" if wl.adamw else
                           ("bf16" if wl.w_bf16 else "fp32") + " W and r, fp32 v" + (", bf16 g" if wl.ema else ""))),
                   "arithmetic": "fp32 codes, fp64 moments/fit/score",
                   "weighting": args.weighting, "param_dtype": args.param_dtype,
                   "cache_rotation_copies": copies,
                   "launch": "batched (up to 16 matrices per launch)" if batched else "one launch per matrix",
                   "launches_per_step": per_step_launches},
        "hbm_GBps": round(gbps, 1), "hbm_pct_peak": round(100 * gbps / PEAK_HBM_GBPS, 2),
        "algorithmic_bytes_per_weight": bpw,
        "copy_GBps": None if copy_gbps is None else round(copy_gbps, 1),
        "hbm_pct_of_copy": None if copy_gbps is None else round(100 * gbps / copy_gbps, 2),
        "step_kernel_ms_p10_p50_p90": step_pct,
        "wall_s_timed": round(wall, 3), "setup_s": round(setup_s, 1),
        "roofline": roofline, "cpu_baseline": cpu,
    }
    if args.diagnostics and not wl.adamw:
        # chosen-clip histogram over every group of one step (GPU), on copies
        # of v so that the timed state is untouched
        hist = np.zeros(len(wl.clips), dtype=np.int64)
        for m in mats[:per_step]:
            o = Q.reconstruct(m["W"], m["v"].clone(), m["g"], fmt=wl.fmt, bits=wl.bits, group=wl.group,
                              clips=wl.clips, beta2=wl.beta2, want_r=False, want_diag=True,
                              weighting=args.weighting, param_dtype=args.param_dtype)
            hist += np.bincount(o["best_clip"].cpu().numpy(), minlength=len(wl.clips))[:len(wl.clips)]
            del o
        clips_arr = np.asarray(wl.clips, dtype=np.float32)
        diag = {"best_clip_histogram": hist.tolist(),
                "frac_groups_clip_below_1": round(float(hist[clips_arr < 1.0].sum() / hist.sum()), 6)}
        if cpu is not None and wl.fmt in ("int", "nvfp4", "int_sym"):
            # mean score of the chosen candidate over that of min-max RTN at
            # clip 1.0 with the standard dequantiser, on a sparse oracle sample
            pairs = []
            for m in mats[:per_step]:
                oracle_rows(m, step * 8, diag_out=pairs)
            err = np.concatenate([a for a, _ in pairs])
            rtn = np.concatenate([b for _, b in pairs])
            ok = rtn > 0
            diag["mean_score_over_rtn"] = round(float(np.mean(err[ok] / rtn[ok])), 6)
            diag["rtn_sample_groups"] = int(ok.sum())
        line["diagnostics"] = diag
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
