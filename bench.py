"""Benchmark of one AMS image-embedding training step on one MI355X.

A step is the whole hot path on one batch already resident in HBM:
ams_dedup -> ams_embed_fwd -> ams_pool_fwd -> ams_pool_bwd -> ams_embed_bwd,
enqueued back to back on one stream.  The same steps through StepPipeline
(batch k + 1's dedup on a second stream beside batch k's pooling and
backward) are reported beside ("pipelined").  Distinct seeded batches rotate
so a batch is never replayed against its own warm cache.  Prints ONE JSON
line.

    python bench.py [--steps K] [--warmup W] [--workload c1_f32] [--mode att]

Throughput = behavior images embedded and pooled per second (fwd + bwd).
Passes after the timed one (none of them enters `value`):
  * per call: events between the five calls of each step;
  * per kernel: the library's own event pairs around every launch
    (ams_timing_enable); the roofline entry is taken for the kernel with the
    largest total time, from its algorithmic flops and bytes per unique image;
  * cold: each step timed alone after a 512 MiB write that evicts the caches.
The CPU baseline is the float64 oracle, timed on this host on one whole batch
of the same workload, repeated for about ten seconds (median run), with the
time of each of its phases and a one-thread run on the batch's first 64
samples.  With the default workload (the 1024-sample float32 step, whose
number is `value`) the line also carries, under "workloads", the same
measurement of the bf16 workloads: the 1024-sample bf16 step (attentive
pooling, sum and max beside) and the 4096-sample step over the 2M-image
table, each with its own roofline entry.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "behavior images embedded+pooled/sec (fwd+bwd), % HBM peak and % MFMA peak"
PEAK_HBM = 8.0e12
PEAK_MFMA = {"f32": 157.3e12, "bf16": 2.5e15}
DEFAULT_WORKLOAD = "c1_f32"
# joint workloads whose image path is another workload's (for its counter record)
JOINT_IMAGE_PATH = {"c4_joint": "c3_long", "c4_mqap": "c3_long"}
OTHER_WORKLOADS = ("c2_bf16", "c3_long")


def mfma_peak(kernel: str, dtype: str) -> float:
    """Dense MFMA peak of the type a kernel's products run in: the split
    float32 layer 1 (l1sk_x3) runs on bf16 MFMA; other float32-storage
    kernels on float32 MFMA."""
    if kernel.endswith("_bf16") or kernel == "l1sk_x3":
        return PEAK_MFMA["bf16"]
    if kernel.endswith("_f32"):
        return PEAK_MFMA["f32"]
    return PEAK_MFMA["bf16" if dtype == "bf16" else "f32"]


def flops_per_unique(dims):
    fwd = 2 * sum(a * b for a, b in zip(dims[:-1], dims[1:]))
    # backward: every weight gradient, plus dH of every layer but the first
    bwd = 2 * sum(a * b for a, b in zip(dims[:-1], dims[1:])) + 2 * sum(
        a * b for a, b in zip(dims[1:-1], dims[2:]))
    return fwd, bwd


# Algorithmic work of the layer-1 GEMM kernels per unique image: 2*F*H flops
# and one read of the image's F-wide feature row.
GEMM_KERNELS = ("l1sk_f32", "l1sk_bf16", "l1rs_bf16", "l1sk_x3", "l1_fwd_f32", "l1_fwd_bf16", "dw1_part_f32",
                "dw1_part_bf16", "dw1_rs_bf16", "dw1_part")


def gemm_work_per_unique(dims, esz):
    return 2 * dims[0] * dims[1], dims[0] * esz


def src_hash():
    h = hashlib.sha256()
    for f in ("embed.hip", "ams_device.h"):
        h.update(open(os.path.join(ROOT, "paper_1711_06505_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def traffic_from_profile(workload: str, kernel: str, unique_count: float):
    """HBM bytes per launch of `kernel` from the committed PMC record, if it
    was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path))
    except Exception:
        return None
    if d.get("source_sha256") != src_hash() or kernel not in d.get("kernels", {}):
        return None
    # bytes scale with the unique rows a launch gathers: per-unique figure of
    # the profiled batch times this run's mean unique count
    return d["kernels"][kernel]["hbm_bytes_per_unique"] * unique_count


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def oracle_phases(batch, n_ids, T_u, Ws, bs, mode):
    """One oracle step, phase by phase (the oracle's own calls, in its order),
    with the wall time of each phase."""
    import numpy as np

    from oracle import oracle
    t = {}
    t0 = time.perf_counter()
    occ = np.concatenate([batch["beh_ids"], batch["ad_ids"]]).astype(np.int32)
    dd = oracle.dedup(occ, n_ids)
    t1 = time.perf_counter()
    rows = np.arange(dd["n_uniq"], dtype=np.int32)
    fw = oracle.mlp_fwd(T_u, rows, Ws, bs)
    t2 = time.perf_counter()
    pf = oracle.pool_fwd(mode, batch["seg_off"], dd["inv"], fw["E"])
    t3 = time.perf_counter()
    pb = oracle.pool_bwd(mode, batch["seg_off"], dd["inv"], dd["n_uniq"], fw["E"], pf, batch["g_u"], batch["g_a"])
    t4 = time.perf_counter()
    oracle.mlp_bwd(T_u, rows, Ws, fw, pb["dE"])
    t5 = time.perf_counter()
    t = {"dedup": t1 - t0, "mlp_fwd": t2 - t1, "pool_fwd": t3 - t2, "pool_bwd": t4 - t3, "mlp_bwd": t5 - t4}
    return t5 - t0, t


def sub_batch(batch, n_samples):
    """The first n_samples samples of a batch (their behaviors, ads and
    upstream gradients)."""
    seg = batch["seg_off"][:n_samples + 1]
    n_beh = int(seg[-1])
    return {"seg_off": seg, "beh_ids": batch["beh_ids"][:n_beh], "ad_ids": batch["ad_ids"][:n_samples],
            "g_u": batch["g_u"][:n_samples], "g_a": batch["g_a"][:n_samples]}


def cpu_baseline(w, batch, mode, min_runs=3, min_seconds=10.0, max_runs=30, one_thread_samples=64):
    import numpy as np

    from oracle import oracle
    from paper_1711_06505_amd import synth
    Ws, bs = synth.make_weights(w)
    occ = synth.occurrences(batch)
    uniq = np.unique(occ)
    T_u = synth.table_rows(w, uniq)
    # repeated until about min_seconds of CPU work, then the median run
    runs = []
    while len(runs) < min_runs or (sum(r[0] for r in runs) < min_seconds and len(runs) < max_runs):
        runs.append(oracle_phases(batch, w.n_images, T_u, Ws, bs, mode))
    runs.sort(key=lambda r: r[0])
    dt, phases = runs[len(runs) // 2]
    times = [r[0] for r in runs]
    n_beh = int(batch["seg_off"][-1])
    threads = oracle.num_threads()
    # one thread, on a bounded sample: the batch's first samples
    sb = sub_batch(batch, one_thread_samples)
    su = np.unique(synth.occurrences(sb))
    oracle.set_threads(1)
    try:
        t1, ph1 = oracle_phases(sb, w.n_images, synth.table_rows(w, su), Ws, bs, mode)
    finally:
        oracle.set_threads(threads)
    n_beh1 = int(sb["seg_off"][-1])
    return {"value": n_beh / dt, "unit": "behavior images/s", "cores": threads,
            "kind": "oracle",
            "sample": f"one whole batch of the same workload ({w.batch} samples, {n_beh} behaviors, "
                      f"{uniq.size} unique images), float64 C oracle with OpenMP, median of {len(runs)} runs "
                      f"(total {sum(times):.1f} s, min {min(times):.2f} s, max {max(times):.2f} s), "
                      f"CPU: {cpu_model()}",
            "phases_s": phases,
            "one_thread": {"value": n_beh1 / t1, "unit": "behavior images/s", "cores": 1, "phases_s": ph1,
                           "sample": f"the batch's first {one_thread_samples} samples ({n_beh1} behaviors, "
                                     f"{su.size} unique images), one run"}}


def bench_peaks(args):
    """Achievable rates of this part: HBM copy and read, gathers of the
    2M-image step's unique rows (8 KB bf16 rows) in the first-layer kernels'
    visit orders, and MFMA loops on operands read from memory.  Each probe is
    timed with events on the stream it is launched on, median of 5 runs."""
    import numpy as np
    import torch

    from oracle import oracle
    from paper_1711_06505_amd import ams, synth

    st = torch.cuda.current_stream()

    def timed(fn, reps=5):
        fn()
        out = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(st)
            fn()
            b.record(st)
            b.synchronize()
            out.append(a.elapsed_time(b) * 1e-3)
        return sorted(out)[len(out) // 2]

    res = {"metric": "achievable peaks", "peak_hbm_bytes_per_s": PEAK_HBM, "peak_mfma_flops": PEAK_MFMA}
    sink = torch.empty(4096 * 256, dtype=torch.int32, device="cuda")
    nb = 1 << 30
    src = torch.empty(nb // 4, dtype=torch.int32, device="cuda").fill_(7)
    dst = torch.empty_like(src)
    for blocks in (1024, 4096):
        t = timed(lambda: ams.ams_peak_copy(src, dst, blocks))
        res[f"copy_1GiB_blocks{blocks}"] = {"bytes_per_s": 2 * nb / t, "seconds": t}
        t = timed(lambda: ams.ams_peak_read(src, blocks, sink))
        res[f"read_1GiB_blocks{blocks}"] = {"bytes_per_s": nb / t, "seconds": t}
    del src, dst
    # the unique rows of the 4096-sample long-behavior batch, table of 2M x 4096 bf16
    w = synth.get("c3_long")
    batch = synth.make_batch(w)
    uniq = oracle.dedup(synth.occurrences(batch), w.n_images)["uniq"]
    rows = torch.from_numpy(np.ascontiguousarray(uniq, dtype=np.int32)).cuda()
    T = torch.empty((w.n_images, w.in_dim), dtype=torch.bfloat16, device="cuda")
    T.view(torch.int16).random_(-32768, 32767)
    row_bytes = w.in_dim * 2
    W = torch.empty(256 * w.in_dim, dtype=torch.bfloat16, device="cuda").normal_()
    patterns = {0: "registers, 16-byte pieces of 32 rows per load (MFMA operand layout)",
                1: "registers, whole 128-byte lines (8 rows per load)",
                2: "registers, whole lines, non-temporal",
                3: "LDS DMA ring, whole lines, non-temporal",
                4: "LDS DMA ring, whole lines, non-temporal, plus a 32 KB weight slice per stage from L2"}
    gather = {}
    for pat, what in patterns.items():
        for blocks in (256, 512):
            t = timed(lambda: ams.ams_peak_gather(T, rows, pat, blocks, sink, W=W))
            gather[f"pattern{pat}_blocks{blocks}"] = {"what": what, "bytes_per_s": rows.numel() * row_bytes / t,
                                                      "seconds": t}
    res["gather_c3_unique_rows"] = {"rows": int(rows.numel()), "row_bytes": row_bytes, "variants": gather,
                                    "note": "512-thread blocks, each a contiguous range of the ascending unique-row list "
                                            "in 256-row tiles, 64 stages of 128 bytes per row, 3 stages in flight"}
    del T, W
    out = torch.empty(4096 * 256, device="cuda")
    for dt, flops in (("bf16", 32768), ("f32", 4096)):
        # random operands (the MFMA rate depends on the data through the clock)
        ops_d = (torch.randn(524288 // 2, device="cuda").to(torch.bfloat16) if dt == "bf16"
                 else torch.randn(524288 // 4, device="cuda"))
        blocks, iters = 1024, (2000 if dt == "bf16" else 250)
        t = timed(lambda: ams.ams_peak_mfma(dt, ops_d, iters, blocks, out))
        total = blocks * 4 * iters * 16 * flops
        res[f"mfma_{dt}_random_operands"] = {"flops_per_s": total / t, "seconds": t,
                                             "frac_of_peak": total / t / PEAK_MFMA[dt]}
    print(json.dumps(res))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--mode", default=None)
    ap.add_argument("--dtype", default=None, choices=("f32", "f32x3", "bf16"),
                    help="override the workload's storage/arithmetic mode (f32x3: float32 storage, "
                         "the 4096-wide forward product on bf16 MFMA with a three-part split)")
    ap.add_argument("--batches", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="with the default workload, leave out the bf16 legs (the 1024-sample step with each "
                         "pooling mode, the 2M-image long-behavior step) added under 'workloads'")
    ap.add_argument("--ops", action="store_true",
                    help="instead of the step, time the widened operations one by one at their real shapes "
                         "(one JSON line each)")
    ap.add_argument("--ops-scaled-only", action="store_true",
                    help="with --ops, time only the aggregators at the 65,536-sample point (for counter runs)")
    ap.add_argument("--peaks", action="store_true",
                    help="instead of the step, time the achievable-peak probes (HBM copy and read, gathers of "
                         "the long-behavior step's unique rows by visit order, MFMA loops) and print one JSON line")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="instead of the step, run a plain device copy of this many MiB "
                         "(calibrates the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1711_06505_amd import ams, synth

    if args.copy_probe_mib:
        n = args.copy_probe_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes_read_per_launch": n * 4, "copy_probe_bytes_written_per_launch": n * 4,
                          "launches": 3}))
        return

    if args.ops:
        torch.cuda.set_device(0)
        ams.load()
        return bench_ops(args)

    if args.peaks:
        torch.cuda.set_device(0)
        ams.load()
        return bench_peaks(args)

    w = synth.get(args.workload)
    if args.dtype and args.dtype != w.dtype:
        if (args.dtype == "bf16") != (w.dtype == "bf16"):
            sys.exit("--dtype may switch between f32 and f32x3 only (bf16 has workloads of its own)")
        w = dataclasses.replace(w, dtype=args.dtype, name=w.name.replace(w.dtype, args.dtype))
    mode = args.mode or w.pools[-1]
    torch.cuda.set_device(0)
    ams.load()
    if w.joint is not None:
        return bench_joint(w, mode, args)

    out = bench_step(w, mode, args)
    if args.workload == DEFAULT_WORKLOAD and not args.no_other_workloads:
        # the bf16 workloads of the same metric, each a leg of its own
        out["workloads"] = {}
        for name in OTHER_WORKLOADS:
            torch.cuda.empty_cache()
            w2 = synth.get(name)
            out["workloads"][name] = bench_step(w2, w2.pools[-1], args, light=True)
    print(json.dumps(out))


def bench_step(w, mode, args, light=False):
    """Times the hot path of workload w (pooling `mode`) and returns its JSON
    record.  light: the value, the other pooling modes, per-kernel times and
    the roofline only (no pipelined, f32x3, cold, per-call or CPU legs)."""
    import torch

    from paper_1711_06505_amd import ams, synth

    # inputs, resident in HBM before timing starts
    T = synth.table_full(w, device="cuda")
    Ws, bs = synth.make_weights(w)
    Wd = [x.cuda() for x in Ws]
    bd = [x.cuda() for x in bs]
    host_batches = [synth.make_batch(w, k=k) for k in range(args.batches)]
    dev_batches = []
    for hb in host_batches:
        dev_batches.append({
            "ids": torch.from_numpy(synth.occurrences(hb)).cuda(),
            "seg_off": torch.from_numpy(hb["seg_off"]).cuda(),
            "dU": torch.from_numpy(hb["g_u"]).cuda(),
            "dA": torch.from_numpy(hb["g_a"]).cuda(),
            "n_beh": int(hb["seg_off"][-1]),
        })
    n_beh_max = max(b["n_beh"] for b in dev_batches)
    step = ams.Step(w.dims, w.dtype, mode, w.batch, n_beh_max)
    step.alloc_workspace(w.n_images)
    stream = torch.cuda.current_stream()

    def one(b, ev=None, st=None):
        st = step if st is None else st
        if ev is not None:
            ev[0].record(stream)
        st.dedup(b["ids"], w.n_images)
        if ev is not None:
            ev[1].record(stream)
        st.embed_fwd(T, Wd, bd)
        if ev is not None:
            ev[2].record(stream)
        st.pool_fwd(b["seg_off"], b["n_beh"])
        st.pool_bwd(b["seg_off"], b["n_beh"], b["dU"], b["dA"])
        if ev is not None:
            ev[3].record(stream)
        st.embed_bwd(T, Wd)
        if ev is not None:
            ev[4].record(stream)

    # unique counts per batch (read once, outside the timed region)
    n_uniq = []
    for b in dev_batches:
        one(b)
        torch.cuda.synchronize()
        assert int(step.dev_status.item()) == 0
        n_uniq.append(int(step.n_uniq.item()))
    for s in range(args.warmup):
        one(dev_batches[s % len(dev_batches)])
    torch.cuda.synchronize()

    # timed region: K whole steps back to back on one stream
    seq = [dev_batches[s % len(dev_batches)] for s in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record(stream)
    for b in seq:
        one(b)
    t_end.record(stream)
    torch.cuda.synchronize()
    ms_total = t_start.elapsed_time(t_end)
    ms_step = ms_total / args.steps
    # the same K steps through StepPipeline (dedup of batch k + 1 on a second
    # stream beside batch k's pooling and backward), reported beside
    ms_step_pipe = None
    if not light:
        pipe = ams.StepPipeline(step, w.n_images)
        pipe.run(seq[:2], T, Wd, bd)
        torch.cuda.synchronize()
        t_start.record(stream)
        last = pipe.run(seq, T, Wd, bd)
        t_end.record(stream)
        torch.cuda.synchronize()
        assert int(pipe.sets[last]["dev_status"].item()) == 0
        ms_step_pipe = t_start.elapsed_time(t_end) / args.steps
        for key in pipe._SET:
            setattr(step, key, pipe.sets[0][key])
    order = [s % len(dev_batches) for s in range(args.steps)]
    beh_total = sum(dev_batches[i]["n_beh"] for i in order)
    uniq_total = sum(n_uniq[i] for i in order)
    value = beh_total / (ms_total * 1e-3)
    # float32 workloads: the same K steps in AMS_F32_X3 mode (float32 storage,
    # the 4096-wide forward product on bf16 MFMA with an exact three-part
    # split), reported beside
    # the workload's other pooling modes: the same steps with each, reported beside
    other_modes = {}
    for m in w.pools:
        if m == mode:
            continue
        stm = ams.Step(w.dims, w.dtype, m, w.batch, n_beh_max)
        stm.alloc_workspace(w.n_images)
        for b in seq[:2]:
            one(b, st=stm)
        torch.cuda.synchronize()
        t_start.record(stream)
        for b in seq:
            one(b, st=stm)
        t_end.record(stream)
        torch.cuda.synchronize()
        assert int(stm.dev_status.item()) == 0
        msm = t_start.elapsed_time(t_end) / args.steps
        other_modes[m] = {"value": beh_total / (msm * args.steps * 1e-3), "ms_per_step": msm}
        del stm
    split3 = None
    if w.dtype == "f32" and not light:
        step3 = ams.Step(w.dims, "f32x3", mode, w.batch, n_beh_max)
        step3.alloc_workspace(w.n_images)
        for b in seq[:2]:
            one(b, st=step3)
        torch.cuda.synchronize()
        t_start.record(stream)
        for b in seq:
            one(b, st=step3)
        t_end.record(stream)
        torch.cuda.synchronize()
        assert int(step3.dev_status.item()) == 0
        ms3 = t_start.elapsed_time(t_end) / args.steps
        split3 = {"value": beh_total / (ms3 * args.steps * 1e-3), "ms_per_step": ms3,
                  "note": "the same steps with dtype f32x3: float32 operands, layer 1's forward product on "
                          "bf16 MFMA with each operand split exactly into three bf16 parts (six part "
                          "products kept, float32-rounding-sized error)"}
        del step3

    # per-call durations: a second pass with events between the calls
    per = None
    if not light:
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
        for s in range(args.steps):
            one(dev_batches[s % len(dev_batches)], evs[s])
        torch.cuda.synchronize()
        per = {"dedup": 0.0, "embed_fwd": 0.0, "pool_fwd_bwd": 0.0, "embed_bwd": 0.0}
        for e in evs:
            per["dedup"] += e[0].elapsed_time(e[1])
            per["embed_fwd"] += e[1].elapsed_time(e[2])
            per["pool_fwd_bwd"] += e[2].elapsed_time(e[3])
            per["embed_bwd"] += e[3].elapsed_time(e[4])
        per = {k: v / args.steps for k, v in per.items()}

    # per-kernel durations: the library's event pairs on the launching stream
    ams.ams_timing_read()                      # drop anything recorded before
    ams.ams_timing_enable(True)
    for s in range(args.steps):
        one(dev_batches[s % len(dev_batches)])
    torch.cuda.synchronize()
    ams.ams_timing_enable(False)
    ktimes = ams.ams_timing_read()
    kernels = {k: {"launches": n, "ms_per_launch": t / n} for k, (n, t) in ktimes.items() if n}

    # cold caches: each step timed alone after a 512 MiB write
    scratch = torch.empty(512 << 18, dtype=torch.float32, device="cuda")
    cold_ms = []
    for s in range(0 if light else args.steps):
        scratch.fill_(float(s))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        one(dev_batches[s % len(dev_batches)])
        e1.record(stream)
        torch.cuda.synchronize()
        cold_ms.append(e0.elapsed_time(e1))
    del scratch
    cold = None
    if cold_ms:
        cold = {"value": beh_total / (sum(cold_ms) * 1e-3), "ms_per_step": sum(cold_ms) / len(cold_ms),
                "note": "each step timed alone after a 512 MiB device write"}

    fwd_f, bwd_f = flops_per_unique(w.dims)
    u_mean = uniq_total / args.steps
    esz = 2 if w.dtype == "bf16" else 4
    step_flops = u_mean * (fwd_f + bwd_f)
    step_bytes = u_mean * 2 * w.in_dim * esz           # the two reads of every unique feature row
    step_peak = PEAK_MFMA["bf16" if w.dtype == "bf16" else "f32"]

    # roofline of the dominant kernel (largest total time over the pass)
    dom = max(ktimes, key=lambda k: ktimes[k][1])
    peak = mfma_peak(dom, w.dtype)
    t_launch = kernels[dom]["ms_per_launch"] * 1e-3
    if dom in GEMM_KERNELS:
        fl_u, by_u = gemm_work_per_unique(w.dims, esz)
        # bound: whichever peak the algorithmic work would take longer on
        bound = "mfma" if fl_u / peak >= by_u / PEAK_HBM else "hbm"
        if bound == "mfma":
            ach, pk, unit, alg = u_mean * fl_u / t_launch / 1e12, peak / 1e12, "TFLOP/s", u_mean * fl_u
        else:
            ach, pk, unit, alg = u_mean * by_u / t_launch / 1e9, PEAK_HBM / 1e9, "GB/s", u_mean * by_u
        roof = {"kernel": dom, "bound": bound, "achieved": ach, "peak": pk, "unit": unit, "frac": ach / pk,
                "traffic": traffic_from_profile(w.name, dom, u_mean),
                "algorithmic_per_launch": alg, "avg_launch_ms": t_launch * 1e3,
                "unit_of_work": f"{fl_u} flop and {by_u} B per unique image, {u_mean:.0f} unique per launch"}
    else:
        roof = {"kernel": dom, "bound": None, "achieved": None, "peak": None, "unit": None, "frac": None,
                "traffic": None, "avg_launch_ms": t_launch * 1e3}
    for k, v in kernels.items():
        if k in GEMM_KERNELS:
            fl_u, _ = gemm_work_per_unique(w.dims, esz)
            v["mfma_frac"] = u_mean * fl_u / (v["ms_per_launch"] * 1e-3) / mfma_peak(k, w.dtype)

    out = {
        "metric": METRIC, "value": value, "unit": "behavior images/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": f"{w.name}: B={w.batch}, lengths {w.lengths}, ids {w.ids} over "
                               f"{w.n_images} images, table {w.n_images}x{w.in_dim} {w.dtype}, "
                               f"MLP {'-'.join(map(str, w.dims))}, pooling {mode}, fwd+bwd",
                   "batch": w.batch, "behaviors_per_step": beh_total / args.steps,
                   "unique_per_step": u_mean, "dedup_ratio": (beh_total + w.batch * args.steps) / uniq_total,
                   "rotating_batches": len(dev_batches)},
        "step_mfma_frac": step_flops / (ms_step * 1e-3) / step_peak,
        "step_hbm_frac": step_bytes / (ms_step * 1e-3) / PEAK_HBM,
        "unique_images_per_s": uniq_total / (ms_total * 1e-3),
        "samples_per_s": w.batch * args.steps / (ms_total * 1e-3),
        "pipelined": None if ms_step_pipe is None else {
            "value": beh_total / (ms_step_pipe * args.steps * 1e-3), "ms_per_step": ms_step_pipe,
            "note": "the same steps through StepPipeline (dedup of the next batch on a second stream)"},
        "f32x3": split3,
        "other_pooling_modes": other_modes or None,
        "cold": cold,
        "per_call_ms": per,
        "kernels": kernels,
        "roofline": roof,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline and not light:
        out["cpu_baseline"] = cpu_baseline(w, host_batches[0], mode)
    if light:
        for k in ("n_gpus", "steps", "warmup", "higher_is_better", "scaling", "vs_baseline", "data", "metric",
                  "unit", "pipelined", "f32x3", "cold", "per_call_ms", "cpu_baseline"):
            out.pop(k, None)
    return out


def bench_joint(w, mode, args):
    """The joint step (image path + ID bags + CTR model + sparse Adagrad), the
    ID tables and accumulators updated in place every step."""
    import numpy as np
    import torch

    from paper_1711_06505_amd import ams, synth

    T = synth.table_full(w, device="cuda")
    Ws, bs = synth.make_weights(w)
    Wd = [x.cuda() for x in Ws]
    bd = [x.cuda() for x in bs]
    cW, cb = synth.make_ctr_weights(w)
    cWd = [x.cuda() for x in cW]
    cbd = [x.cuda() for x in cb]
    n_t = len(w.joint.id_rows)
    tabs = [synth.id_table_full(w, t, device="cuda") for t in range(n_t)]
    accs = [torch.full_like(x, w.joint.acc0) for x in tabs]
    dev_batches = []
    for k in range(args.batches):
        hb = synth.make_batch(w, k=k)
        jb = synth.make_joint(w, hb, k=k)
        dev_batches.append({
            "ids": torch.from_numpy(synth.occurrences(hb)).cuda(),
            "seg_off": torch.from_numpy(hb["seg_off"]).cuda(),
            "id_ids": [torch.from_numpy(synth.joint_occurrences(jb, t)).cuda() for t in range(n_t)],
            "labels": torch.from_numpy(jb["labels"]).cuda(),
            "n_beh": int(hb["seg_off"][-1]),
        })
    n_beh_max = max(b["n_beh"] for b in dev_batches)
    tq = w.joint.query_table if w.joint.query_table >= 0 else None
    js = ams.JointStep(w.dims, w.dtype, mode, w.batch, n_beh_max, w.joint.id_rows, w.joint.id_dim,
                       synth.ctr_dims(w), query_table=tq)
    js.alloc_workspace(w.n_images)
    stream = torch.cuda.current_stream()

    def one(b):
        js.run(b["ids"], w.n_images, T, Wd, bd, b["seg_off"], b["id_ids"], tabs, accs, b["labels"], cWd, cbd,
               w.joint.lr, w.joint.eps)

    n_uniq, n_rows = [], []
    for b in dev_batches:
        one(b)
        torch.cuda.synchronize()
        assert int(js.img.dev_status.item()) == 0 and all(int(x.item()) == 0 for x in js.t_status)
        n_uniq.append(int(js.img.n_uniq.item()))
        n_rows.append(sum(int(x.item()) for x in js.t_nu))
    for s in range(args.warmup):
        one(dev_batches[s % len(dev_batches)])
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for s in range(args.steps):
        one(dev_batches[s % len(dev_batches)])
    t1.record(stream)
    torch.cuda.synchronize()
    ms_total = t0.elapsed_time(t1)
    order = [s % len(dev_batches) for s in range(args.steps)]
    beh_total = sum(dev_batches[i]["n_beh"] for i in order)
    uniq_total = sum(n_uniq[i] for i in order)
    rows_total = sum(n_rows[i] for i in order)
    loss = float(js.loss.item())

    ams.ams_timing_read()
    ams.ams_timing_enable(True)
    for s in range(args.steps):
        one(dev_batches[s % len(dev_batches)])
    torch.cuda.synchronize()
    ams.ams_timing_enable(False)
    ktimes = ams.ams_timing_read()
    kernels = {k: {"launches": n, "ms_per_launch": t / n} for k, (n, t) in ktimes.items() if n}

    esz = 2 if w.dtype == "bf16" else 4
    u_mean = uniq_total / args.steps
    step_peak = PEAK_MFMA["bf16" if w.dtype == "bf16" else "f32"]
    # dominant kernel of the image path: the ID-table kernels run on a side
    # stream beside it, so their event-timed durations include the time they
    # wait for the GPU and overstate their own work
    img = [k for k in ktimes if k in GEMM_KERNELS] or list(ktimes)
    dom = max(img, key=lambda k: ktimes[k][1])
    peak = mfma_peak(dom, w.dtype)
    t_launch = kernels[dom]["ms_per_launch"] * 1e-3
    if dom in GEMM_KERNELS:
        fl_u, by_u = gemm_work_per_unique(w.dims, esz)
        bound = "mfma" if fl_u / peak >= by_u / PEAK_HBM else "hbm"
        if bound == "mfma":
            ach, pk, unit, alg = u_mean * fl_u / t_launch / 1e12, peak / 1e12, "TFLOP/s", u_mean * fl_u
        else:
            ach, pk, unit, alg = u_mean * by_u / t_launch / 1e9, PEAK_HBM / 1e9, "GB/s", u_mean * by_u
        # the joint workloads' image path is the long-sequence step's (same
        # batch, table, weights and kernels): its counter record applies
        rec = JOINT_IMAGE_PATH.get(w.name, w.name)
        roof = {"kernel": dom, "bound": bound, "achieved": ach, "peak": pk, "unit": unit, "frac": ach / pk,
                "traffic": traffic_from_profile(rec, dom, u_mean), "algorithmic_per_launch": alg,
                "avg_launch_ms": t_launch * 1e3,
                "unit_of_work": f"{fl_u} flop and {by_u} B per unique image, {u_mean:.0f} unique per launch"}
        if rec != w.name:
            roof["traffic_record"] = f"profiles/traffic_{rec}.json (the same image-path kernels)"
    else:
        roof = {"kernel": dom, "bound": None, "achieved": None, "peak": None, "unit": None, "frac": None,
                "traffic": None, "avg_launch_ms": t_launch * 1e3}
    for k, v in kernels.items():
        if k in GEMM_KERNELS:
            fl_u, _ = gemm_work_per_unique(w.dims, esz)
            v["mfma_frac"] = u_mean * fl_u / (v["ms_per_launch"] * 1e-3) / mfma_peak(k, w.dtype)
    fwd_f, bwd_f = flops_per_unique(w.dims)
    ms_step = ms_total / args.steps
    out = {
        "metric": METRIC, "value": beh_total / (ms_total * 1e-3), "unit": "behavior images/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": f"{w.name}: B={w.batch}, lengths {w.lengths}, image ids {w.ids} over "
                               f"{w.n_images} images, table {w.n_images}x{w.in_dim} {w.dtype}, MLP "
                               f"{'-'.join(map(str, w.dims))}, pooling {mode}"
                               f"{'' if tq is None else f' + a query channel on ID table {tq} (MultiQueryAttentivePooling)'}"
                               f"; ID tables "
                               f"{'/'.join(str(n) for n in w.joint.id_rows)} x {w.joint.id_dim} fp32 "
                               f"Zipf({w.joint.id_zipf}); CTR MLP {'-'.join(map(str, synth.ctr_dims(w)))} fp32, "
                               f"softmax cross-entropy; sparse Adagrad lr {w.joint.lr}; fwd+bwd+update",
                   "batch": w.batch, "behaviors_per_step": beh_total / args.steps, "unique_per_step": u_mean,
                   "id_rows_touched_per_step": rows_total / args.steps, "rotating_batches": len(dev_batches)},
        "step_mfma_frac": u_mean * (fwd_f + bwd_f) / (ms_step * 1e-3) / step_peak,
        "step_hbm_frac": u_mean * 2 * w.in_dim * esz / (ms_step * 1e-3) / PEAK_HBM,
        "unique_images_per_s": uniq_total / (ms_total * 1e-3),
        "id_rows_per_s": rows_total / (ms_total * 1e-3),
        "samples_per_s": w.batch * args.steps / (ms_total * 1e-3),
        "loss_last_step": loss,
        "kernels": kernels,
        "roofline": roof,
        "cpu_baseline": None,
    }
    print(json.dumps(out))


PEAK_F32_VALU = 157.3e12


def bench_ops(args):
    """The operations beside the step, each timed alone at its real shape on
    inputs resident in HBM: the sum and attentive aggregators at 65,536
    samples, one channel of multiple-query attentive pooling and the
    concatenate aggregator on the long-sequence batch, the Adam update of the
    image model, the CTR model with PReLU and the pre-rank towers at 4096
    samples.  Per op: ms per call over --steps calls (HIP events on the
    launch stream) after --warmup calls, the library's per-kernel times, and
    a roofline entry: compulsory HBM bytes (every input read once, every
    output written once) against 8 TB/s, or for the small fp32 nets their
    multiply-adds against the fp32 vector peak."""
    import numpy as np
    import torch

    from paper_1711_06505_amd import ams, synth
    stream = torch.cuda.current_stream()
    f32, i32 = torch.float32, torch.int32

    def timed(name, fn, shape, bound, work, unit_note):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        ams.ams_timing_read()
        ams.ams_timing_enable(True)
        for _ in range(args.steps):
            fn()
        torch.cuda.synchronize()
        ams.ams_timing_enable(False)
        kt = {k: {"launches": n, "ms_per_launch": t / n} for k, (n, t) in ams.ams_timing_read().items() if n}
        if bound == "hbm":
            ach, pk, unit = work / (ms * 1e-3) / 1e9, PEAK_HBM / 1e9, "GB/s"
        else:
            ach, pk, unit = work / (ms * 1e-3) / 1e12, PEAK_F32_VALU / 1e12, "TFLOP/s"
        print(json.dumps({"op": name, "shape": shape, "ms_per_call": ms, "calls": args.steps,
                          "roofline": {"bound": bound, "achieved": ach, "peak": pk, "unit": unit, "frac": ach / pk,
                                       "work_per_call": work, "unit_of_work": unit_note},
                          "kernels": kt}), flush=True)

    # ---- the aggregators alone at a scale where bandwidth, not latency,
    # bounds them: 65,536 samples with the long-sequence lengths (geometric,
    # mean 200, capped at 500) and image IDs (Zipf 1.05 over 2M), ~12M
    # behaviors; E random (the embedding model is not part of this leg).
    # Algorithmic bytes per the step's units: forward 52 B per behavior (its
    # index and its 48-byte row) + 96 B per sample (U and A), + 4 B per
    # behavior for the attention weights; backward 60 B per occurrence
    # (stable order, inverse index and its 48-byte gradient) + 48 B per
    # unique image (dE), + 8 B per behavior for attention (weights, E row).
    wsc = dataclasses.replace(synth.get("c3_long"), name="pool_scaled", index=31, batch=65_536, stream=-1)
    hb = synth.make_batch(wsc)
    occ = torch.from_numpy(synth.occurrences(hb)).cuda()
    seg = torch.from_numpy(hb["seg_off"]).cuda()
    B, n_beh, D = wsc.batch, int(hb["seg_off"][-1]), 12
    gA_d = torch.from_numpy(hb["g_a"]).cuda()
    gU_d = torch.from_numpy(hb["g_u"]).cuda()
    for mode in ("sum", "att"):
        # (at most n_images distinct images: that capacity always holds)
        st = ams.Step((wsc.in_dim, 256, 64, D), "bf16", mode, B, n_beh, cap=wsc.n_images, cap_checked=True)
        st.dedup(occ, wsc.n_images)
        torch.cuda.synchronize()
        assert int(st.dev_status.item()) == 0
        n_u = int(st.n_uniq.item())
        st.alloc_workspace(wsc.n_images)
        g = torch.Generator(device="cuda").manual_seed(7)
        st.E.copy_(torch.randn(st.E.shape, generator=g, device="cuda") * 0.5)
        shape = f"B={B} (lengths geometric mean 200 cap 500), {n_beh} behaviors, {n_u} unique images, D={D}"
        att = 1 if mode == "att" else 0
        timed(f"pool_scaled_{mode}_fwd", lambda: st.pool_fwd(seg, n_beh), shape, "hbm",
              n_beh * (52 + 4 * att) + B * 96, "52 B per behavior (+4 attention weight) + 96 B per sample")
        st.pool_fwd(seg, n_beh)
        timed(f"pool_scaled_{mode}_bwd", lambda: st.pool_bwd(seg, n_beh, gU_d, gA_d), shape, "hbm",
              (n_beh + B) * 60 + n_u * 48 + n_beh * 8 * att,
              "60 B per occurrence (+8 attention) + 48 B per unique image")
        del st
        torch.cuda.empty_cache()
    if args.ops_scaled_only:
        return

    # ---- pooling variants on the long-sequence batch
    w = synth.get("c3_long")
    hb = synth.make_batch(w)
    occ = torch.from_numpy(synth.occurrences(hb)).cuda()
    seg = torch.from_numpy(hb["seg_off"]).cuda()
    B, n_beh, D = w.batch, int(hb["seg_off"][-1]), 12
    st = ams.Step(w.dims, w.dtype, "att", B, n_beh)
    st.dedup(occ, w.n_images)
    torch.cuda.synchronize()
    n_u = int(st.n_uniq.item())
    cap = st.cap
    g = torch.Generator(device="cuda").manual_seed(5)
    E = torch.randn((cap, D), generator=g, device="cuda") * 0.5
    Q = torch.randn((B, D), generator=g, device="cuda") * 0.5
    U = torch.empty((B, D), device="cuda")
    wq = torch.empty(n_beh, device="cuda")
    dU = torch.randn((B, D), generator=g, device="cuda")
    dQ = torch.empty((B, D), device="cuda")
    dE = torch.zeros((cap, D), device="cuda")
    ws = torch.empty(ams.load().ams_pool_workspace(2, B, n_beh, D, cap), dtype=torch.uint8, device="cuda")

    def mqap():
        ams.ams_pool_query_fwd(seg, n_beh, st.inv, E, Q, U, wq)
        ams.ams_pool_query_bwd(seg, n_beh, st.inv, st.occ_perm, st.uniq_off, st.n_uniq, cap, E, Q, U, wq, dU, dQ,
                               dE, True, ws)
    # fwd: inv, E, Q, seg in; U, w out.  bwd: inv, occ_perm, uniq_off, E, Q, U, w, dU in; dE (read and
    # written: accumulate), dQ out
    fwd_b = n_beh * 4 + n_u * D * 4 + B * D * 4 + (B + 1) * 4 + B * D * 4 + n_beh * 4
    bwd_b = n_beh * 4 * 3 + (n_u + 1) * 4 + n_u * D * 4 * 3 + B * D * 4 * 4
    timed("mqap_query_channel", mqap, f"c3_long batch: B={B}, {n_beh} behaviors, {n_u} unique, D={D}", "hbm",
          fwd_b + bwd_b, "compulsory bytes of the forward and backward (accumulating into dE)")

    Lc = 64
    Uc = torch.empty((B, Lc * D), device="cuda")
    Ac = torch.empty((B, D), device="cuda")
    dUc = torch.randn((B, Lc * D), generator=g, device="cuda")
    dAc = torch.randn((B, D), generator=g, device="cuda")
    wsc = torch.empty(ams.load().ams_pool_workspace(0, B, n_beh, D, cap), dtype=torch.uint8, device="cuda")

    def concat():
        ams.ams_pool_concat_fwd(Lc, seg, n_beh, st.inv, E, Uc, Ac)
        ams.ams_pool_concat_bwd(Lc, seg, n_beh, st.inv, st.occ_perm, st.uniq_off, st.n_uniq, cap, dUc, dAc, dE,
                                wsc)
    kept = int(np.minimum(np.diff(hb["seg_off"]), Lc).sum())
    fwd_b = kept * 4 + (B + 1) * 4 + B * 4 + min(kept + B, n_u) * D * 4 + B * Lc * D * 4 + B * D * 4
    bwd_b = (n_beh + B) * 4 * 2 + (n_u + 1) * 4 + B * Lc * D * 4 + B * D * 4 + n_u * D * 4
    timed("concat_aggregator", concat, f"c3_long batch, Lc={Lc}: U {B}x{Lc * D}", "hbm", fwd_b + bwd_b,
          "compulsory bytes of the forward and backward")
    del st, E, Q, U, wq, dU, dQ, dE, ws, Uc, Ac, dUc, dAc, wsc

    # ---- Adam on the image model's parameters (float32 master + bf16 copy)
    n = sum(o * i + o for i, o in zip((4096, 256, 64), (256, 64, 12)))
    prm = torch.randn(n, generator=g, device="cuda") * 0.05
    grd = torch.randn(n, generator=g, device="cuda") * 1e-3
    m, v = torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
    pb = torch.empty(n, dtype=torch.int16, device="cuda")
    t_step = [0]

    def adam():
        t_step[0] += 1
        ams.ams_adam_update(prm, grd, m, v, 1e-3, t_step[0], param_bf16=pb)
    timed("adam_update", adam, f"{n} parameters (4096-256-64-12), bf16 copy", "hbm", n * 30,
          "30 B per parameter: param, grad, m, v read; param, m, v written; bf16 copy written")

    # ---- CTR model with PReLU and the pre-rank towers, 4096 samples
    rng = np.random.default_rng(3)

    def net(dims, prelu=True):
        Ws = [torch.from_numpy(rng.uniform(-0.1, 0.1, (o, i)).astype(np.float32)).cuda()
              for i, o in zip(dims[:-1], dims[1:])]
        bs = [torch.zeros(o, device="cuda") for o in dims[1:]]
        sl = [torch.full((o,), 0.25, device="cuda") for o in dims[1:-1]] if prelu else None
        dW = [torch.empty_like(x) for x in Ws]
        db = [torch.empty_like(x) for x in bs]
        ds = [torch.empty_like(x) for x in sl] if prelu else None
        return (Ws, bs, sl), (dW, db, ds)

    Bc = 4096
    cd = (60, 200, 80, 2)
    (cW, cb, cs), (cdW, cdb, cds) = net(cd)
    fields = [torch.randn((Bc, 12), generator=g, device="cuda") for _ in range(5)]
    dfields = [torch.empty_like(x) for x in fields]
    labels = torch.from_numpy((rng.random(Bc) < 0.05).astype(np.int32)).cuda()
    loss, prob = torch.zeros(1, device="cuda"), torch.empty((Bc, 2), device="cuda")
    cnet = ams.make_ctr(cd)
    wsn = torch.empty(ams.ams_ctr_workspace(cnet, Bc), dtype=torch.uint8, device="cuda")

    def ctr():
        ams.ams_ctr_fwd_bwd(cnet, fields, labels, cW, cb, loss, prob, cdW, cdb, dfields, wsn, slopes=cs,
                            dslopes=cds)
    macs = sum(i * o for i, o in zip(cd[:-1], cd[1:]))
    timed("ctr_prelu", ctr, f"B={Bc}, CTR MLP {'-'.join(map(str, cd))} PReLU, 5 fields of 12", "alu",
          2.0 * Bc * macs * 3, "2 flop per multiply-add, forward + input gradient + weight gradient")

    ud, ad = (48, 64, 32), (48, 64, 32)
    user, duser = net(ud)
    adn, dad = net(ad)
    uf = [torch.randn((Bc, 12), generator=g, device="cuda") for _ in range(4)]
    af = [torch.randn((Bc, 12), generator=g, device="cuda") for _ in range(4)]
    duf, daf = [torch.empty_like(x) for x in uf], [torch.empty_like(x) for x in af]
    pr = torch.empty(Bc, device="cuda")
    un, an = ams.make_ctr(ud), ams.make_ctr(ad)
    wsd = torch.empty(ams.ams_dssm_workspace(un, an, Bc), dtype=torch.uint8, device="cuda")

    def dssm():
        ams.ams_dssm_fwd_bwd(un, an, uf, af, labels, user, adn, loss, pr, duser, dad, duf, daf, wsd)
    macs = sum(i * o for i, o in zip(ud[:-1], ud[1:])) + sum(i * o for i, o in zip(ad[:-1], ad[1:]))
    timed("prerank_dssm", dssm, f"B={Bc}, towers {'-'.join(map(str, ud))} / {'-'.join(map(str, ad))} PReLU",
          "alu", 2.0 * Bc * macs * 3, "2 flop per multiply-add, forward + input gradient + weight gradient")


if __name__ == "__main__":
    main()
