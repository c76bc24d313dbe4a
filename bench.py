"""Throughput of pooled back-propagation on one MI355X, in connections per second.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one pooled update: forward pass, output and hidden deltas, summed
change and learning-rate/momentum update over one batch (all on the GPU,
inputs resident in HBM).  The headline workload is the deep dense net
512-2048-2048-2048-64 (batch 8192, 524,288 N(0,1) patterns, one epoch = 64
updates), the largest of the five workloads and the one on which the fp32
MFMA fraction is measured.  K updates are timed as one library call over
K x 8192 patterns; before it, W untimed updates warm the clocks, and two
calls identical to the timed one let the library capture its replay graph,
so that the timed call replays it whatever W is.

Under "secondary": the wide dense net 1024-4096-1024 (one epoch), the
NETtalk-shaped one-hot nets 203-80-26 (one update), 203-120-26 at batch 512
(10 epochs) and at batch 16 (2 epochs), the Elman net (64 external inputs +
256 context units, 256 hidden, 64 outputs; 1024 sequence streams, an update
every 8 steps), and the batch-512 NETtalk net with the table sigmoid and
with the range check of the summed changes switched on.

value = connections x patterns presented / wall time (the paper's
definition, section 7.1: bias connections included, update frequency and
cheaper input connections not accounted for).

Per-kernel device times come from a second pass over the same steps in which
the library brackets every launch with HIP events on the stream it runs on
(direct launches, no graph); the dominant kernel's algorithmic work per
launch divided by its average duration gives the roofline entry.  The oracle
(CPU, test infrastructure) is timed on a bounded sample for the CPU
baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "connection-updates/sec (fwd+bwd+update) and % fp32 MFMA peak, 1 MI355X"
PEAK_FP32_MFMA = 157.3e12   # MI355X dense fp32 matrix peak, flop/s
PEAK_HBM = 8.0e12           # MI355X HBM3E, bytes/s
PAPER_GF11_CPS = 9.01e8     # section 6.3, Table 1: 356 processors, tree summation
PRIMARY = "deep-512-2048x3-64"
SECONDARY = ("wide-1024-4096-1024", "nettalk-80-b1024", "nettalk-120-b512", "nettalk-120-b16")
VARIANT_WORKLOAD = "nettalk-120-b512"
SECONDARY_SEQ = ("elman-64+256-256-64",)
GEMM_KINDS = ("forward", "output", "backward", "change", "splitk", "seq_pair", "seq_win")
KERNEL_NAMES = {
    "forward": "gemm_kernel|skinny_kernel<..., EpiSigmoid>",
    "output": "gemm_kernel|skinny_kernel<..., EpiOutputDelta>",
    "backward": "gemm_kernel|skinny_kernel<..., EpiHiddenDelta>",
    "change": "gemm_kernel<..., EpiUpdate>",
    "splitk": "gemm_kernel|skinny_kernel<..., EpiSplitUpdate>",
    "bias": "bias_update_kernel",
    "gather": "onehot_forward_kernel",
    "scatter": "onehot_update_kernel",
    "reduce": "sse_reduce_kernel",
    "fused_fb": "small_fwdbwd_kernel",
    "fused_update": "small_update_kernel",
    "output_finish": "output_finish_kernel",
    "seq_in": "seq_assemble_kernel",
    "seq_pair": "elman_pair_kernel",
    "seq_win": "elman_window_kernel",
}
SMALL_MAX_HIDDEN, SMALL_MAX_OUT, SMALL_MAX_ACTIVE = 256, 64, 32   # the library's fused-path limits


def kind_work(sizes, rows, onehot, n_active, splits_of, parts=("fwd", "bwd")):
    """Algorithmic (flops, HBM bytes) of each kernel kind for one update over `rows` patterns
    (parts: "fwd" the forward pass and output deltas, "bwd" the hidden deltas, changes and updates)."""
    w = {}

    def add(kind, f, b):
        f0, b0 = w.get(kind, (0.0, 0.0))
        w[kind] = (f0 + f, b0 + b)

    L = len(sizes) - 1
    R = float(rows)
    if onehot and L == 2 and sizes[1] <= SMALL_MAX_HIDDEN and sizes[2] <= SMALL_MAX_OUT and n_active <= SMALL_MAX_ACTIVE:
        # The algorithmic bytes of one update are 4 (n_active + n_L) per pattern (indices and
        # targets, read by the forward/backward launch) and 16 per weight (W and V read and
        # written, by the update launch); intermediates (activations, deltas) are not counted.
        n0, H, O = sizes
        add("fused_fb", R * (H * (n_active + 1) + 4 * H * O), 4.0 * R * (n_active + O))
        add("fused_update", R * (2 * (H + 1) * O + H * (n_active + 1)), 16.0 * ((n0 + 1) * H + (H + 1) * O))
        return w
    fwd, bwd = "fwd" in parts, "bwd" in parts
    for l in range(L):
        ni, no = sizes[l], sizes[l + 1]
        if l == 0 and onehot:
            add("gather", R * no * (n_active + 1), 4 * (R * n_active + (ni + 1) * no + R * no))
            add("scatter", R * no * (n_active + 1), 4 * (R * n_active + R * no) + 16 * (ni + 1) * no)
        else:
            if fwd and l == L - 1 and choose_output_splits(rows, no, ni) > 1:
                add("output", 2 * R * ni * no, 4 * (R * ni + (ni + 1) * no))
                add("output_finish", 6 * R * no, 4 * (2 * R * no + no))
            elif fwd and l == L - 1:
                add("output", 2 * R * ni * no, 4 * (R * ni + (ni + 1) * no + 2 * R * no))
            elif fwd:
                add("forward", 2 * R * ni * no, 4 * (R * ni + (ni + 1) * no + R * no))
            upd = 16.0 * ni * no
            if bwd and splits_of(ni, no, rows) > 1:
                add("splitk", 2 * R * ni * no, 4 * (R * ni + R * no) + upd)
            elif bwd:
                add("change", 2 * R * ni * no, 4 * (R * ni + R * no) + upd)
            if bwd:
                add("bias", R * no, 4 * -(-rows // 64) * no + 16 * no)
        if l >= 1 and bwd:
            add("backward", 2 * R * no * ni, 4 * (R * no + ni * no + 2 * R * ni))
    return w


def seq_kind_work(sizes, n_ctx, S, steps, splits_of, built_steps=0, paired=False, window=False):
    """Algorithmic (flops, HBM bytes) per kind of one Elman window: `steps` forward steps of S
    patterns, then one backward pass and update over steps x S rows.  `built_steps` of the steps
    have their input rows built by the first product (reading the flags besides X and the context
    source, writing the rows); the others assemble them first (seq_in).  `paired`: steps 1 ..
    steps - 1 run their hidden layer in one launch with the output layer of the step before
    (seq_pair); the first step's hidden layer and the last step's output layer run alone.
    `window`: the whole forward pass of the window is one launch (seq_win), which reads X, the
    flags, the targets and the weights and writes the input rows, hidden units and output deltas."""
    n_ext = sizes[0] - n_ctx
    if window:
        n0, n1, n2 = sizes
        step = kind_work(sizes, S, False, 0, splits_of, ("fwd",))
        flops = steps * sum(f for f, _ in step.values())
        io = 4.0 * S * (n_ext + 2 + n2 + n0 + n1 + n2)
        w = {"seq_win": (flops, steps * io + 4.0 * ((n0 + 1) * n1 + (n1 + 1) * n2))}
        for k, (f, b) in kind_work(sizes, steps * S, False, 0, splits_of, ("bwd",)).items():
            f0, b0 = w.get(k, (0.0, 0.0))
            w[k] = (f0 + f, b0 + b)
        return w
    rows_bytes = 4.0 * S * (1 + -(-sizes[0] // 4) * 4)          # flags read, rows written
    w = {"seq_in": (0.0, (steps - built_steps) * (4.0 * S * (n_ext + n_ctx) + rows_bytes))}

    def add(kind, f, b):
        f0, b0 = w.get(kind, (0.0, 0.0))
        w[kind] = (f0 + f, b0 + b)

    step = kind_work(sizes, S, False, 0, splits_of, ("fwd",))
    if paired:
        pairs = steps - 1
        add("forward", *step["forward"])
        add("forward", 0.0, (built_steps - pairs) * rows_bytes)
        add("output", *step["output"])
        add("seq_pair", pairs * (step["forward"][0] + step["output"][0]),
            pairs * (step["forward"][1] + step["output"][1] + rows_bytes))
    else:
        if built_steps:
            add("forward", 0.0, built_steps * rows_bytes)
        for _ in range(steps):
            for k, (f, b) in step.items():
                add(k, f, b)
    for k, (f, b) in kind_work(sizes, steps * S, False, 0, splits_of, ("bwd",)).items():
        f0, b0 = w.get(k, (0.0, 0.0))
        w[k] = (f0 + f, b0 + b)
    return w


def choose_output_splits(M, N, K):
    """Mirror of the library's split-K choice for the output layer (products with few tiles and
    K <= 2048 take the skinny kernel, unsplit), for work accounting only."""
    if K <= 2048 and -(-M // 64) * -(-N // 64) < 128:
        return 1
    return choose_splits(M, N, K)


def input_built_in_product(sizes, n_ctx, S):
    """Mirror of the library's choice to build an Elman step's input rows in the first product
    (context copying hidden layer 1 in order, product on the skinny kernel)."""
    return n_ctx > 0 and sizes[0] <= 2048 and -(-S // 64) * -(-sizes[1] // 64) < 128


def elman_pair(sizes, n_ctx, S):
    """Mirror of the library's choice to run an Elman step's hidden layer in one launch with the
    output layer of the step before (one hidden layer, both products on the skinny kernel)."""
    return (len(sizes) == 3 and input_built_in_product(sizes, n_ctx, S) and sizes[1] <= 2048
            and -(-S // 64) * -(-sizes[2] // 64) < 128)


def elman_window(sizes, n_ctx, S):
    """Mirror of the library's choice to run an Elman window's forward pass in one launch (one
    hidden layer whose context copies it in order; sizes within the kernel's limits)."""
    if len(sizes) != 3:
        return False
    n0, n1, n2 = sizes
    n_ext = n0 - n_ctx
    return (S > 0 and 0 < n_ctx <= n1 and n_ext >= 0 and n0 <= 512 and n1 <= 256 and n2 <= 256
            and 4 * n_ext <= 1024 and 4 * n2 <= 1024)


def change_splits(M, N, K):
    """Mirror of the library's split count for a change product (split over blocks, whose last
    block per tile applies the update), for work accounting only."""
    t64 = -(-M // 64) * -(-N // 64)
    if K >= 4096 and 16 <= t64 < 128:
        return min(-(-256 // t64), K // 256)
    if K >= 1024 and -(-M // 64) * -(-N // 64) < 128:
        tiles, chunk = -(-M // 64) * -(-N // 32), 1024
        while chunk > 128 and tiles * -(-K // chunk) < 256:
            chunk //= 2
        if -(-K // chunk) >= 2:
            return -(-K // chunk)
    return choose_splits(M, N, K)


def choose_splits(M, N, K):
    """Mirror of the library's split-K choice, for work accounting only."""
    t128 = -(-M // 128) * -(-N // 128)
    tiles = t128 if (t128 >= 256 or K >= 1024) else -(-M // 64) * -(-N // 64)
    if K < 1024 or tiles >= 512:
        return 1
    s = -(-512 // tiles)
    return max(1, min(s, K // 256))


def schedule(spec, steps):
    """(first pattern, patterns, updates) calls covering `steps` updates in epoch order."""
    per_epoch = -(-spec.n_patterns // spec.batch)
    calls = []
    full, rem = divmod(steps, per_epoch)
    calls += [(0, spec.n_patterns, per_epoch)] * full
    if rem:
        calls.append((0, rem * spec.batch, rem))
    return calls


def step_rows(spec, calls):
    rows = []
    for p0, n, _ in calls:
        for b0 in range(p0, p0 + n, spec.batch):
            rows.append(min(spec.batch, p0 + n - b0))
    return rows


def run_workload(name, steps, warmup, torch, bp, wl, metrics, log, variant=None):
    """Times `steps` pooled updates of a named workload (variant: "table sigmoid" or "range check").

    The timed updates run as the calls of schedule(spec, steps) (one call per epoch, in epoch
    order).  Before them: `warmup` untimed updates (clock warm-up), then the same calls twice,
    so that the library has captured them into its replay graph (it captures the second of two
    identical calls) and the timed calls replay it, whatever `warmup` is."""
    spec = wl.SPECS[name]
    t0 = time.time()
    w = wl.make(name)
    log(f"[{name}] generated {w.n_patterns} patterns in {time.time() - t0:.1f}s")
    dev = torch.device("cuda:0")
    t = torch.from_numpy(w.targets).to(dev)
    x = torch.from_numpy(w.inputs).to(dev) if w.inputs is not None else None
    a = torch.from_numpy(w.active).to(dev) if w.active is not None else None
    net = bp.Net(w.sizes)
    if variant == "table sigmoid":
        net.set_sigmoid(bp.BP_SIGMOID_TABLE)
    elif variant == "range check":
        net.set_fault_limit(1e6)
    elif variant is not None:
        raise ValueError(variant)

    def run(calls):
        for p0, n, _ in calls:
            if a is not None:
                net.train_batches(t[p0:p0 + n], spec.batch, w.lr, w.momentum, active=a[p0:p0 + n], want_sse=False)
            else:
                net.train_batches(t[p0:p0 + n], spec.batch, w.lr, w.momentum, inputs=x[p0:p0 + n], want_sse=False)

    calls = schedule(spec, steps)
    patterns = sum(n for _, n, _ in calls)
    if warmup:
        net.set_weights(w.weights)
        run(schedule(spec, warmup))
    for _ in range(2):                    # the second identical call captures the replay graph
        net.set_weights(w.weights)
        run(calls)
    net.set_weights(w.weights)            # timed run starts from the workload's initial state
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()  # the library's stream (bp.Net enqueues on torch's current stream)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    ev0.record(stream)
    run(calls)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    secs = ev0.elapsed_time(ev1) / 1e3
    log(f"[{name}{' + ' + variant if variant else ''}] {steps} steps, {patterns} patterns in {secs * 1e3:.2f} ms "
        f"(wall {wall * 1e3:.2f} ms)")

    # profile pass: the same steps with every launch bracketed by events.  It
    # runs twice and the second pass is kept: the first creates the library's
    # pooled events, which delays its launches.
    for _ in range(2):
        net.set_weights(w.weights)
        net.profile(True)                 # clears the counts of an earlier pass
        run(calls)
    rep = net.profile_report()
    net.profile(False)
    net.close()

    W = metrics.num_weights(w.sizes)
    cps = W * patterns / secs
    rows = step_rows(spec, calls)
    flops_step = sum(metrics.dense_flops_per_pattern(w.sizes, r) * r for r in rows)
    work = {}
    for r in rows:
        for k, (f, b) in kind_work(w.sizes, r, w.active is not None, 7, change_splits).items():
            f0, b0 = work.get(k, (0.0, 0.0))
            work[k] = (f0 + f, b0 + b)
    kernels, roof, gemm_f, gemm_ms = summarize_kernels(rep, work, name)
    res = {
        "workload": name, "net": "-".join(map(str, w.sizes)), "batch": spec.batch, "patterns": patterns,
        "steps": steps, "warmup": warmup, "seconds": secs, "ms_per_step": secs * 1e3 / steps, "value": cps,
        "mfma_peak_frac": flops_step / secs / PEAK_FP32_MFMA,
        "gemm_mfma_frac": (gemm_f / (gemm_ms / 1e3) / PEAK_FP32_MFMA) if gemm_ms > 0 else None,
        "us_per_update": secs * 1e6 / steps, "roofline": roof, "kernels": kernels,
        "kernel_time_ms": sum(v["total_ms"] for v in kernels.values()),
    }
    if w.active is not None:
        # the whole update against HBM: 16 B per weight (W, V read and written) + 4 (n_active + n_L) B
        # per pattern (indices, targets), over the measured time per update
        upd_bytes = sum(metrics.onehot_bytes_per_update(w.sizes) +
                        r * metrics.onehot_bytes_per_pattern(w.sizes, w.active.shape[1]) for r in rows)
        res["update_hbm"] = {"algorithmic_bytes_per_update": upd_bytes / steps,
                             "achieved_gbps": upd_bytes / secs / 1e9, "frac": upd_bytes / secs / PEAK_HBM}
    if variant:
        res["variant"] = variant
    return res, w


def summarize_kernels(rep, work, name):
    """Per-kind kernel table and the roofline entry of the dominant kind."""
    kernels = {}
    for k, (cnt, ms) in rep.items():
        if cnt == 0:
            continue
        f, b = work.get(k, (0.0, 0.0))
        s = ms / 1e3
        kernels[k] = {"name": KERNEL_NAMES[k], "launches": cnt, "avg_us": ms * 1e3 / cnt, "total_ms": ms,
                      "tflops": f / s / 1e12 if s > 0 else None, "gbps": b / s / 1e9 if s > 0 else None,
                      "flops_per_launch": f / cnt, "bytes_per_launch": b / cnt}
    dom = max(kernels, key=lambda k: kernels[k]["total_ms"])
    dk = kernels[dom]
    f, b = work.get(dom, (0.0, 0.0))
    mfma_bound = f / PEAK_FP32_MFMA >= b / PEAK_HBM
    if mfma_bound:
        ach, peak, unit = dk["tflops"], PEAK_FP32_MFMA / 1e12, "TFLOP/s"
    else:
        ach, peak, unit = dk["gbps"], PEAK_HBM / 1e9, "GB/s"
    roof = {"bound": "mfma" if mfma_bound else "hbm", "kernel": dk["name"], "kind": dom,
            "achieved": ach, "peak": peak, "unit": unit, "frac": ach / peak,
            "avg_launch_us": dk["avg_us"], "work_per_launch": dk["flops_per_launch"] if mfma_bound else dk["bytes_per_launch"],
            "traffic": traffic_for(name, dom)}
    gemm_ms = sum(kernels[k]["total_ms"] for k in GEMM_KINDS if k in kernels)
    gemm_f = sum(work.get(k, (0, 0))[0] for k in GEMM_KINDS)
    return kernels, roof, gemm_f, gemm_ms


def run_seq_workload(name, epochs, torch, bp, wl, metrics, log):
    """Elman training: `epochs` whole passes over the sequence streams, after one untimed epoch."""
    spec = wl.SEQ_SPECS[name]
    t0 = time.time()
    w = wl.make_sequences(name)
    log(f"[{name}] generated {spec.n_steps} steps x {spec.n_streams} streams in {time.time() - t0:.1f}s")
    dev = torch.device("cuda:0")
    x, t, c, m = (torch.from_numpy(a).to(dev) for a in (w.inputs, w.targets, w.cont, w.mask))
    net = bp.Net(w.sizes)
    net.set_context(w.ctx_layer, w.ctx_unit)

    def run():
        for _ in range(epochs):
            net.train_sequences(x, t, c, m, spec.steps_per_update, w.lr, w.momentum, want_sse=False)

    net.set_weights(w.weights)
    net.train_sequences(x, t, c, m, spec.steps_per_update, w.lr, w.momentum, want_sse=False)   # warmup epoch
    net.set_weights(w.weights)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    run()
    ev1.record()
    torch.cuda.synchronize()
    secs = ev0.elapsed_time(ev1) / 1e3
    windows = -(-spec.n_steps // spec.steps_per_update) * epochs
    real = int(w.mask.sum()) * epochs
    log(f"[{name}] {epochs} epoch(s), {windows} updates, {real} patterns ({spec.n_steps * spec.n_streams * epochs} "
        f"with padding) in {secs * 1e3:.2f} ms")
    for _ in range(2):                    # as in run_workload: the second pass is kept
        net.set_weights(w.weights)
        net.profile(True)
        run()
    rep = net.profile_report()
    net.profile(False)
    net.close()
    work = {}
    built = input_built_in_product(w.sizes, spec.n_ctx, spec.n_streams) and spec.steps_per_update > 1
    for w0 in range(0, spec.n_steps, spec.steps_per_update):
        steps = min(spec.steps_per_update, spec.n_steps - w0)
        nb = (steps - 1 if w0 == 0 else steps) if built else 0     # one call per epoch: its first step assembles
        window = elman_window(w.sizes, spec.n_ctx, spec.n_streams)
        paired = not window and built and elman_pair(w.sizes, spec.n_ctx, spec.n_streams)
        for k, (f, b) in seq_kind_work(w.sizes, spec.n_ctx, spec.n_streams, steps, change_splits, nb,
                                       paired, window).items():
            f0, b0 = work.get(k, (0.0, 0.0))
            work[k] = (f0 + epochs * f, b0 + epochs * b)
    kernels, roof, gemm_f, gemm_ms = summarize_kernels(rep, work, name)
    W = metrics.num_weights(w.sizes)
    flops = sum(f for f, _ in work.values())
    res = {
        "workload": name, "net": "-".join(map(str, w.sizes)), "streams": spec.n_streams,
        "steps_per_epoch": spec.n_steps, "steps_per_update": spec.steps_per_update, "epochs": epochs,
        "patterns": real, "patterns_with_padding": spec.n_steps * spec.n_streams * epochs, "seconds": secs,
        "value": W * real / secs, "unit": "connections/s (sequence patterns, padding excluded)",
        "us_per_update": secs * 1e6 / windows, "mfma_peak_frac": flops / secs / PEAK_FP32_MFMA,
        "gemm_mfma_frac": (gemm_f / (gemm_ms / 1e3) / PEAK_FP32_MFMA) if gemm_ms > 0 else None,
        "roofline": roof, "kernels": kernels, "kernel_time_ms": sum(v["total_ms"] for v in kernels.values()),
    }
    return res, w


TRAFFIC_JSON = os.path.join(ROOT, "profiles", "traffic.json")
COPY_BYTES = 1 << 30        # one copy of 1 GiB for the counter calibration


def kernel_source_sha():
    h = hashlib.sha256()
    for f in ("bp_device.h", "bp_kernels.hip", "bp_small.hip", "bp_seq.hip"):
        h.update(open(os.path.join(ROOT, "paper_1801_01554_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def traffic_for(workload, kind):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it matches the current kernels."""
    if not os.path.exists(TRAFFIC_JSON):
        return None
    try:
        with open(TRAFFIC_JSON) as f:
            d = json.load(f)
        if d.get("kernel_source_sha256") != kernel_source_sha():
            return None
        e = d.get("workloads", {}).get(workload, {}).get(kind)
        return e["hbm_bytes_per_launch"] if e else None
    except (OSError, ValueError, KeyError):
        return None


def kind_of_kernel(name):
    """Kernel kind of a rocprofv3 kernel name."""
    import re
    # the epilogue is the template argument named Epi...; the tile shape and a
    # thread count may stand before or after it
    m = re.search(r"(gemm_kernel|skinny_kernel)<[^>]*?\b(Epi\w+)", name)
    if m:
        return {"EpiSigmoid": "forward", "EpiOutputDelta": "output", "EpiPartial": "output",
                "EpiHiddenDelta": "backward", "EpiUpdate": "change", "EpiSplitUpdate": "splitk"}.get(m.group(2))
    for k, v in KERNEL_NAMES.items():
        if "<" not in v and v in name:
            return k
    return None


def summarize_stats(src, out, title, note, cmd):
    """Writes a rocprofv3 --stats kernel_stats.csv as the markdown summary kept in profiles/."""
    import csv
    import re
    lines = [f"# {title}", "", note, "", "Command (on the MI355X box, from /tmp with TMPDIR=/tmp; R = repository root):",
             "", f"    {cmd}", "", "| kernel | calls | total ns | average ns | % | min ns | max ns |",
             "|---|---|---|---|---|---|---|"]
    for r in csv.DictReader(open(src)):
        name = r["Name"].replace("bpk::(anonymous namespace)::", "")
        m = re.search(r"(\w+_kernel(?:<[^>]*>)?|fillBufferAligned|copyBuffer)", name)
        short = m.group(1) if m else name[:60]
        lines.append(f"| `{short}` | {r['Calls']} | {r['TotalDurationNs']} | {float(r['AverageNs']):.0f} | "
                     f"{float(r['Percentage']):.1f} | {r['MinNs']} | {r['MaxNs']} |")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


def summarize_mfma(counter_csv, trace_csv, out, title, note, cmd):
    """Writes the MFMA-pipe utilisation per kernel from a rocprofv3 --pmc GRBM_GUI_ACTIVE
    SQ_VALU_MFMA_BUSY_CYCLES (+ --kernel-trace) run as the markdown summary kept in profiles/:
    the rate of GRBM_GUI_ACTIVE cycles during a dispatch (summed over the 8 XCDs / 8 /
    duration) and the share of those cycles the MFMA pipes were busy
    (SQ_VALU_MFMA_BUSY_CYCLES summed over the 1024 SIMDs / 1024 / (GRBM_GUI_ACTIVE / 8))."""
    import collections
    import csv
    import math
    import re
    dur = {r["Dispatch_Id"]: int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in csv.DictReader(open(trace_csv))}
    per = collections.defaultdict(dict)
    for r in csv.DictReader(open(counter_csv)):
        per[r["Dispatch_Id"]][r["Counter_Name"]] = float(r["Counter_Value"])
        per[r["Dispatch_Id"]]["name"] = r["Kernel_Name"]
        per[r["Dispatch_Id"]]["grid"] = f'{r.get("Grid_Size", r.get("Grid_Size_X", ""))}'
    agg = collections.defaultdict(list)
    for d, v in per.items():
        if d not in dur or "GRBM_GUI_ACTIVE" not in v or "SQ_VALU_MFMA_BUSY_CYCLES" not in v:
            continue
        name = v["name"].replace("bpk::(anonymous namespace)::", "")
        m = re.search(r"(\w+_kernel(?:<[^>]*>)?)", name)
        if not m or "gemm" not in m.group(1) and "skinny" not in m.group(1) and "elman" not in m.group(1):
            continue
        # launches of one kernel differ by shape: grouped by duration to within 10%
        key = (m.group(1), round(math.log(dur[d]) / math.log(1.1)))
        g = v["GRBM_GUI_ACTIVE"] / 8.0
        agg[key].append((dur[d], g / dur[d], v["SQ_VALU_MFMA_BUSY_CYCLES"] / 1024.0 / g))
    lines = [f"# {title}", "", note, "", "Command (on the MI355X box, from /tmp with TMPDIR=/tmp; R = repository root):",
             "", f"    {cmd}", "", "| kernel | dispatches | average µs | active cycles per ns | MFMA busy |", "|---|---|---|---|---|"]
    for (k, _), v in sorted(agg.items(), key=lambda kv: -sum(x[0] for x in kv[1])):
        n = len(v)
        avg = sum(x[0] for x in v) / n
        if n < 4 or avg < 20e3:    # short launches: the counters' window is longer than the dispatch
            continue
        lines.append(f"| `{k}` | {n} | {avg / 1e3:.1f} | {sum(x[1] for x in v) / n:.2f} | "
                     f"{100 * sum(x[2] for x in v) / n:.1f}% |")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


def copy_calibration():
    """Copies a 1 GiB buffer four times (device to device), for the FETCH_SIZE / WRITE_SIZE scale."""
    import torch
    x = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda:0").fill_(1.0)
    y = torch.empty_like(x)
    for _ in range(4):
        y.copy_(x)
    torch.cuda.synchronize()
    print(f"copied {COPY_BYTES} bytes x 4", flush=True)


def counters_to_traffic(workload, fetch_csv, write_csv, calib_fetch_csv, calib_write_csv, command):
    """Turns rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE passes into per-launch HBM bytes in profiles/traffic.json."""
    import csv
    import collections

    def per_kernel(path, counter):
        acc = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] == counter:
                acc[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        return acc

    def copy_factor(path, counter):
        acc = per_kernel(path, counter)
        # the copy is the dispatch with the largest counter value
        name, vals = max(acc.items(), key=lambda kv: max(kv[1]))
        return COPY_BYTES / (max(vals) * 1024.0), name

    ff, fname = copy_factor(calib_fetch_csv, "FETCH_SIZE")
    wf, _ = copy_factor(calib_write_csv, "WRITE_SIZE")
    fetch = per_kernel(fetch_csv, "FETCH_SIZE")
    write = per_kernel(write_csv, "WRITE_SIZE")
    kinds = collections.defaultdict(lambda: [0.0, 0.0, 0])
    for name, vals in fetch.items():
        k = kind_of_kernel(name)
        if k:
            kinds[k][0] += sum(vals) * 1024.0 * ff
            kinds[k][2] += len(vals)
    for name, vals in write.items():
        k = kind_of_kernel(name)
        if k:
            kinds[k][1] += sum(vals) * 1024.0 * wf
    d = {}
    if os.path.exists(TRAFFIC_JSON):
        d = json.load(open(TRAFFIC_JSON))
    sha = kernel_source_sha()
    if d.get("kernel_source_sha256") != sha:
        d = {"kernel_source_sha256": sha, "workloads": {}}
    d["calibration"] = {"copy_bytes": COPY_BYTES, "copy_kernel": fname, "fetch_factor": ff, "write_factor": wf}
    d["workloads"][workload] = {
        k: {"dispatches": n, "fetch_bytes_per_launch": fb / n, "write_bytes_per_launch": wb / n,
            "hbm_bytes_per_launch": (fb + wb) / n} for k, (fb, wb, n) in kinds.items() if n}
    d.setdefault("commands", {})[workload] = command
    with open(TRAFFIC_JSON, "w") as f:
        json.dump(d, f, indent=1)
    print(json.dumps(d["workloads"][workload], indent=1))


def cpu_baseline(w, budget_s, log, max_updates=None):
    """The oracle (double storage) on the host cores: the workload's updates in order (whole
    epochs of batches, momentum carried) until `budget_s` seconds are spent, at least one update,
    at most the workload's own updates (or `max_updates`)."""
    import oracle
    from paper_1801_01554_amd import metrics
    spec = w.spec
    o = oracle.OracleNet(w.sizes, 64)
    o.set_weights(w.weights.astype("float64"))
    per_epoch = -(-w.n_patterns // spec.batch)
    total = per_epoch * spec.epochs if max_updates is None else min(max_updates, per_epoch * spec.epochs)
    t0 = time.perf_counter()
    done, pats = 0, 0
    while done < total:
        b0 = (done % per_epoch) * spec.batch
        n = min(spec.batch, w.n_patterns - b0)
        kw = {"active": w.active[b0:b0 + n]} if w.active is not None else {"x": w.inputs[b0:b0 + n]}
        o.train_epoch(w.targets[b0:b0 + n], spec.batch, w.lr, w.momentum, **kw)
        done += 1
        pats += n
        if time.perf_counter() - t0 >= budget_s:
            break
    secs = time.perf_counter() - t0
    v = metrics.num_weights(w.sizes) * pats / secs
    log(f"[cpu] oracle {done} update(s) of {spec.name}, {pats} patterns in {secs:.2f}s on {oracle.get_threads()} "
        f"threads")
    return {"value": v, "unit": "connections/s", "cores": oracle.get_threads(), "kind": "oracle",
            "sample": f"the first {done} of {per_epoch * spec.epochs} updates of {spec.name} in order ({pats} "
                      f"patterns, batch {spec.batch}), {secs:.2f} s"}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="pooled updates timed (default: the whole workload)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed updates first, to warm the clocks (default 4); two untimed calls identical to "
                         "the timed one always follow, so that the library replays its captured graph in the "
                         "timed call")
    ap.add_argument("--workload", default=PRIMARY)
    ap.add_argument("--no-secondary", action="store_true", help="time the headline workload only")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle time for the baseline")
    ap.add_argument("--copy-calibration", action="store_true", help="only copy 1 GiB four times (counter scale)")
    ap.add_argument("--counters-to-traffic", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "CAL_FETCH", "CAL_WRITE"),
                    help="write per-launch HBM traffic of --workload to profiles/traffic.json")
    ap.add_argument("--command", default="", help="the profiling command recorded with --counters-to-traffic")
    ap.add_argument("--summarize-mfma", nargs=6, metavar=("COUNTER_CSV", "TRACE_CSV", "OUT_MD", "TITLE", "NOTE", "CMD"),
                    help="write the MFMA-busy summary of a rocprofv3 --pmc run")
    ap.add_argument("--summarize-stats", nargs=5, metavar=("STATS_CSV", "OUT_MD", "TITLE", "NOTE", "CMD"),
                    help="format a rocprofv3 kernel_stats.csv as a profiles/ summary")
    args = ap.parse_args()
    if args.summarize_stats:
        summarize_stats(*args.summarize_stats)
        return
    if args.summarize_mfma:
        summarize_mfma(*args.summarize_mfma)
        return
    if args.counters_to_traffic:
        counters_to_traffic(args.workload, *args.counters_to_traffic, args.command)
        return
    if args.copy_calibration:
        copy_calibration()
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (the design notes describe how the "
              "pooled update would shard across GPUs). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    def log(msg):
        print(msg, file=sys.stderr, flush=True)

    import torch
    from paper_1801_01554_amd import bp, metrics
    from paper_1801_01554_amd import workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a ROCm device"
    bp.lib()
    if args.workload in wl.SEQ_SPECS:
        # an Elman workload on its own (profiling runs): one epoch per step
        epochs = args.steps if args.steps is not None else 1
        r, _ = run_seq_workload(args.workload, epochs, torch, bp, wl, metrics, log)
        print(json.dumps({"metric": METRIC, "value": r["value"], "unit": "connections/s", "n_gpus": 1,
                          "steps": epochs, "warmup": 1, "ms_per_step": r["seconds"] * 1e3 / epochs,
                          "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
                          "data": "synthetic", "config": {"workload": args.workload, "net": r["net"],
                                                          "parallelism": "single GPU"},
                          "roofline": r["roofline"], "kernels": r["kernels"]}), flush=True)
        return
    spec = wl.SPECS[args.workload]
    per_epoch = -(-spec.n_patterns // spec.batch)
    steps = args.steps if args.steps is not None else per_epoch * spec.epochs
    warmup = args.warmup if args.warmup is not None else 4
    prim, w = run_workload(args.workload, steps, warmup, torch, bp, wl, metrics, log)
    cpu = cpu_baseline(w, args.cpu_budget, log) if not args.no_cpu else None
    del w
    torch.cuda.empty_cache()

    secondary = []
    if not args.no_secondary:
        for name in SECONDARY:
            if name == args.workload:
                continue
            s2 = wl.SPECS[name]
            pe = -(-s2.n_patterns // s2.batch)
            r, w2 = run_workload(name, pe * s2.epochs, 4, torch, bp, wl, metrics, log)
            if not args.no_cpu:
                r["cpu_baseline"] = cpu_baseline(w2, min(args.cpu_budget, 5.0), log)
            secondary.append(r)
            del w2
            torch.cuda.empty_cache()
        for name in SECONDARY_SEQ:
            r, w2 = run_seq_workload(name, 1, torch, bp, wl, metrics, log)
            secondary.append(r)
            del w2
            torch.cuda.empty_cache()
        sv = wl.SPECS[VARIANT_WORKLOAD]
        for variant in ("table sigmoid", "range check"):
            r, _ = run_workload(VARIANT_WORKLOAD, -(-sv.n_patterns // sv.batch) * sv.epochs, 4, torch, bp, wl,
                                metrics, log, variant=variant)
            secondary.append(r)

    line = {
        "metric": METRIC, "value": prim["value"], "unit": "connections/s", "n_gpus": 1, "steps": steps,
        "warmup": warmup, "ms_per_step": prim["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": args.workload, "net": prim["net"], "batch": spec.batch,
                   "patterns_per_epoch": spec.n_patterns, "patterns_timed": prim["patterns"],
                   "inputs": "one-hot 7x29 window" if spec.onehot else spec.input_kind,
                   "lr": spec.lr, "momentum": spec.momentum, "parallelism": "single GPU"},
        "mfma_peak_frac": prim["mfma_peak_frac"], "gemm_mfma_frac": prim["gemm_mfma_frac"],
        "us_per_update": prim["us_per_update"], "roofline": prim["roofline"], "kernels": prim["kernels"],
        "context": {"paper_gf11_cps": PAPER_GF11_CPS, "note": "GF11, 356 processors, NETtalk 203-60-26 (section 6.3)"},
        "secondary": secondary,
    }
    if prim.get("update_hbm"):
        line["update_hbm"] = prim["update_hbm"]
    if cpu:
        line["cpu_baseline"] = cpu
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
