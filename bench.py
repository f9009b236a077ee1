"""Benchmark of the MI355X forward convolution (Eq. (1)).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-layers] [--no-cpu]
    python bench.py --traffic-run              (under rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE)
    python bench.py --traffic-parse FETCH_DIR WRITE_DIR
    python bench.py --traffic-run --layer all  (under rocprofv3 --pmc, one counter per run)
    python bench.py --model-check FETCH_DIR WRITE_DIR TCP_TCC_DIR LDS_DIR
    python bench.py --rank-sweep [N]           (model rank vs measured time, every layer)
    python bench.py --table1                   (Table 1 layers at batch 1, stride and same padding)

A step is one conv_fwd call (tile selection is cached, so the step is the
kernel launch) on the pointwise layer N=32 C=256 K=64 56x56 1x1 fp32.  Inputs
are seeded uniform[-1,1) synthetic tensors of that shape.  The timed steps
cycle through enough independent In/Out buffer sets (more than twice the
256 MB last-level cache) that every step reads In from HBM and writes Out to
HBM.  The default 500 untimed warm-up steps (about 20 ms) bring the GPU out
of its idle clocks first: a cold start measured up to twice the steady
launch time for the first few milliseconds.

Prints ONE JSON line with the metric, the roofline of the kernel (average
launch duration from HIP events recorded on the launch stream around the
timed region), the HBM traffic measured by the counter passes when they were
taken on the launched kernel's current source and plan, the CPU oracle timed on this host (cpu_baseline),
and a per-layer table for the other layer configurations.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"fp32_mfma_tflops": 157.3, "bf16_mfma_tflops": 2516.6, "hbm_gbs": 8000.0}
HEADLINE = "conv1x1_n32_c256_k64_in56"
MALL_BYTES = 256 * 2 ** 20
FLUSH_BYTES = 512 * 2 ** 20  # read between timed runs: twice the last-level cache
PROTOCOL_RUNS = 50           # timed runs per layer (Sec. 10: 50 runs, the first excluded)
RAMP_S = 0.1                 # back-to-back launches before any timing, independent of --warmup
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_conv1x1_n32_c256_k64_in56.json")
SETS_MAX_BYTES = 16 * 2 ** 30  # device memory of all rotating buffer sets of one layer


def buffer_sets(in_bytes, out_bytes):
    """Number of In/Out buffer sets that back-to-back launches rotate through
    so that each launch reads its In from HBM.  The kernels write Out with
    streaming stores, which the 256 MB last-level cache does not keep, so In
    alone must exceed twice that cache.  (Measured on the 226x226 bf16 layer:
    with four sets, 209 MB of In in all, a launch took 66 us; once anything
    of 48 MB or more passed through the cache between launches, 107 us.)
    Capped at SETS_MAX_BYTES of device memory in all."""
    want = -(-2 * MALL_BYTES // max(1, in_bytes)) + 1
    return max(2, min(want, SETS_MAX_BYTES // max(1, in_bytes + out_bytes)))


def flops(c):
    return 2.0 * c.N * c.K * c.P * c.Q * c.C * c.R * c.S


def alg_bytes(c):
    e = 2 if c.dtype == "bf16" else 4
    return (c.N * c.C * c.H * c.W + c.K * c.C * c.R * c.S) * e + c.N * c.K * c.P * c.Q * 4


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("conv_kernels.hip", "select.cpp"):
        with open(os.path.join(ROOT, "paper_2101_09808_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


KERNEL_FUNCTIONS = {1: "conv_f32_kernel", 2: "conv_f32_dma_kernel", 3: "conv_bf16_kernel",
                    4: "conv1x1_stream_kernel", 5: "conv1x1_stream_loop_kernel", 6: "conv_bf16_tr_kernel",
                    7: "conv1x1_bal_kernel"}


def plan_kernel_hash(c, plan):
    """Hash of what one launch of `plan` runs: the source text of its kernel
    template, the instance line that fixes the template arguments, the launch
    geometry struct, and the plan's tile fields.  Counter figures taken for
    the plan stay valid while this hash does."""
    from paper_2101_09808_amd import conv as B

    src = open(os.path.join(ROOT, "paper_2101_09808_amd", "csrc", "conv_kernels.hip")).read()
    hdr = open(os.path.join(ROOT, "paper_2101_09808_amd", "csrc", "conv_internal.h")).read()
    fam = B.conv_fwd_geometry(*c.key(), plan)["family"]
    name = KERNEL_FUNCTIONS[fam]
    at = src.index("\n" + name + "(")
    begin = src.rindex("\ntemplate <", 0, at)
    end = src.index("\n}\n", at) + 3
    inst = [ln.strip() for ln in src.splitlines() if ln.strip().startswith(("F32_", "BF16_"))
            and "(%d," % plan["variant"] in ln]
    geom = hdr[hdr.index("struct Geom {"):]
    geom = geom[:geom.index("};") + 2]
    tiles = {k: plan[k] for k in ("variant", "tile_k", "tile_rows", "tile_cols", "tile_c", "waves_k",
                                  "waves_px", "grid_order", "split_c")}
    h = hashlib.sha256()
    for part in (src[begin:end], "\n".join(inst), geom, json.dumps(tiles, sort_keys=True)):
        h.update(part.encode())
    return h.hexdigest()[:16]


class LayerRunner:
    """Device buffers and a raw-pointer launcher for one layer: In/Out buffer
    sets rotate (In alone more than twice the 256 MB last-level cache in
    all, see buffer_sets) so that back-to-back launches read In from HBM and
    write Out to HBM."""

    def __init__(self, c, out_bf16=False):
        import torch
        from paper_2101_09808_amd import conv as B
        from paper_2101_09808_amd.workloads import make_inputs

        self.c = c
        In0, Ker0 = make_inputs(c)
        self.nsets = buffer_sets(In0.numel() * In0.element_size(),
                                 c.N * c.K * c.P * c.Q * (2 if out_bf16 else 4))
        dev = torch.device("cuda:0")
        self.Ker = Ker0.to(dev)
        self.ins = [In0.to(dev) for _ in range(self.nsets)]
        odt = torch.bfloat16 if out_bf16 else torch.float32
        self.outs = [torch.empty(c.N, c.K, c.P, c.Q, device=dev, dtype=odt) for _ in range(self.nsets)]
        bf16 = c.dtype == "bf16"
        self.stream = torch.cuda.current_stream()
        sp = self.stream.cuda_stream
        kp = self.Ker.data_ptr()
        ips = [t.data_ptr() for t in self.ins]
        ops = [t.data_ptr() for t in self.outs]
        strided = c.stride != 1 or c.pad != 0
        L = B.lib()
        dt = B.CONV_DTYPE_BF16 if bf16 else B.CONV_DTYPE_F32

        def fn(i):
            if out_bf16:
                st = L.conv_fwd_bf16_out(*c.key(), ips[i], kp, ops[i], sp)
            elif strided:
                st = L.conv_fwd_ex(*c.key(), c.stride, c.stride, c.pad, c.pad, dt, ips[i], kp, ops[i], sp)
            else:
                st = B.conv_fwd_ptr(*c.key(), ips[i], kp, ops[i], sp, bf16)
            if st != B.CONV_OK:
                raise B.ConvError(st, "conv_fwd")

        self.fn = fn
        # checked call through the tensor API first
        if out_bf16:
            B.conv_fwd_bf16_out(self.ins[0], self.Ker, out=self.outs[0])
        elif strided:
            B.conv_fwd_ex(self.ins[0], self.Ker, c.stride, c.pad, out=self.outs[0])
        else:
            (B.conv_fwd_bf16 if bf16 else B.conv_fwd)(self.ins[0], self.Ker, out=self.outs[0])
        torch.cuda.synchronize()

    def ramp(self, seconds=RAMP_S):
        """Launch back to back for a fixed wall time, whatever --warmup says,
        so that the clocks have left their idle state before timing."""
        import torch
        t0 = time.perf_counter()
        i = 0
        while time.perf_counter() - t0 < seconds:
            for _ in range(16):
                self.fn(i % self.nsets)
                i += 1
            torch.cuda.synchronize()
        return i

    def back_to_back(self, steps, warmup, queued=False):
        """Average launch duration from HIP events recorded on the launch
        stream around `steps` back-to-back launches (rotating buffer sets),
        and the host wall time of the same region.  queued: the launches first
        queue up behind a bounded spin kernel, so that for layers shorter than
        the host's per-call time the events still see back-to-back kernels
        (the wall time then includes the spin)."""
        import torch
        for i in range(warmup):
            self.fn(i % self.nsets)
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        if queued:
            torch.cuda._sleep(int(sleep_cycles_per_us() * 60 * steps))
        start.record(self.stream)
        for i in range(steps):
            self.fn(i % self.nsets)
        end.record(self.stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ev_ms = start.elapsed_time(end)
        return dict(mean_kernel_ms=ev_ms / steps, wall_ms_per_step=wall * 1e3 / steps, buffer_sets=self.nsets)

    def cold_runs(self, flush, runs=PROTOCOL_RUNS):
        """The paper's protocol (Sec. 10): one untimed run, then `runs` runs,
        each after a read pass over a 512 MB buffer (twice the last-level
        cache: In, Ker and Out start in HBM) and between its own two HIP
        events on the launch stream.  Returns the per-run times in us."""
        import torch
        self.fn(0)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(runs)]
        sink = torch.empty((), device=flush.device)
        for i, (a, b) in enumerate(evs):
            torch.sum(flush, 0, out=sink)
            a.record(self.stream)
            self.fn(i % self.nsets)
            b.record(self.stream)
        torch.cuda.synchronize()
        return [a.elapsed_time(b) * 1e3 for a, b in evs]


def trace_summary(db_path, limit=20):
    """Kernel table of a rocprofv3 results database (--kernel-trace): per
    kernel name, calls, average / min / max duration in us and workgroups,
    the kernels that took the most total time first."""
    import sqlite3
    db = sqlite3.connect(db_path)
    q = ("select name, count(*), avg(duration), min(duration), max(duration), sum(duration), grid_x, workgroup_x "
         "from kernels group by name order by sum(duration) desc limit ?")
    lines = ["| kernel | calls | avg us | min us | max us | workgroups |", "|---|---|---|---|---|---|"]
    for r in db.execute(q, (limit,)):
        lines.append(f"| {r[0][:110]} | {r[1]} | {r[2] / 1e3:.2f} | {r[3] / 1e3:.2f} | {r[4] / 1e3:.2f} | "
                     f"{r[6] // max(1, r[7])} |")
    return "\n".join(lines)


def progress(msg):
    """A progress line on stderr (stdout carries only the result line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def summary(ts):
    """Mean, median, standard deviation and 95% confidence half-width of the
    mean (Student t) of per-run times in us."""
    import statistics

    from scipy import stats

    n = len(ts)
    mean = statistics.fmean(ts)
    sd = statistics.stdev(ts) if n > 1 else 0.0
    half = float(stats.t.ppf(0.975, n - 1)) * sd / n ** 0.5 if n > 1 else 0.0
    return {"runs": n, "mean_us": mean, "median_us": statistics.median(ts), "min_us": min(ts), "max_us": max(ts),
            "std_us": sd, "ci95_us": [mean - half, mean + half]}


def flush_buffer():
    import torch
    return torch.ones(FLUSH_BYTES // 4, device="cuda:0")


def empty_kernel_floor(flush, runs=PROTOCOL_RUNS):
    """Event-timed duration of a kernel that does nothing (torch's bounded
    spin kernel asked to spin for 0 cycles), measured exactly as cold_runs
    times a layer: the fixed cost any single launch pays between its events."""
    import torch
    stream = torch.cuda.current_stream()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(runs)]
    sink = torch.empty((), device="cuda:0")
    torch.cuda._sleep(0)
    for a, b in evs:
        torch.sum(flush, 0, out=sink)
        a.record(stream)
        torch.cuda._sleep(0)
        b.record(stream)
    torch.cuda.synchronize()
    cold = summary([a.elapsed_time(b) * 1e3 for a, b in evs])
    # back to back, amortised (100 launches queued behind a spin)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(int(sleep_cycles_per_us() * 2000))
    a.record(stream)
    for _ in range(100):
        torch.cuda._sleep(0)
    b.record(stream)
    torch.cuda.synchronize()
    return {"cold": cold, "back_to_back_us": a.elapsed_time(b) * 1e3 / 100}


def observed_sclk(runner, seconds=2.0):
    """Shader clock observed while the layer runs back to back: amd-smi (or
    rocm-smi) sampled from a helper thread during `seconds` of launches.
    Returns the samples in MHz and the tool used, or the reason none was read."""
    import re
    import shutil
    import subprocess
    import threading

    import torch

    cmds = []
    if shutil.which("amd-smi"):
        cmds.append(["amd-smi", "metric", "-g", "0", "-c"])
    if shutil.which("rocm-smi"):
        cmds.append(["rocm-smi", "-d", "0", "--showclocks"])
    if not cmds:
        return {"mhz": None, "tool": None, "note": "no amd-smi or rocm-smi on this host"}
    samples, used, errors = [], [], []
    stop = threading.Event()

    def sample():
        while not stop.is_set():
            for cmd in cmds:
                try:
                    r = subprocess.run(cmd, capture_output=True, text=True, timeout=10)
                except (OSError, subprocess.SubprocessError) as e:
                    errors.append(f"{cmd[0]}: {e}")
                    continue
                txt = r.stdout
                if cmd[0] == "amd-smi":  # one GFX_i clock per XCD: their mean
                    v = [float(x) for x in re.findall(r"GFX_\d+:\s*CLK:\s*([0-9.]+)\s*MHz", txt)]
                else:
                    v = [float(x) for x in re.findall(r"sclk clock level:.*?\(([0-9.]+)\s*Mhz\)", txt, flags=re.I)]
                if v:
                    samples.append(sum(v) / len(v))
                    used.append(cmd[0])
                    break
                errors.append(f"{cmd[0]}: no clock in output ({txt[:80]!r})")

    th = threading.Thread(target=sample, daemon=True)
    th.start()
    t0 = time.perf_counter()
    i = 0
    while time.perf_counter() - t0 < seconds or (not samples and time.perf_counter() - t0 < 3 * seconds):
        for _ in range(32):
            runner.fn(i % runner.nsets)
            i += 1
        torch.cuda.synchronize()
    stop.set()
    th.join(timeout=15)
    if not samples:
        return {"mhz": None, "tool": None, "note": "; ".join(errors[:2]) or "no sample"}
    return {"mhz": samples, "tool": used[0], "note": "sampled while the layer ran back to back"}


def time_layer(c, steps, warmup, queued=False, out_bf16=False):
    """Back-to-back timing of one layer (LayerRunner.back_to_back) after the
    fixed clock ramp."""
    r = LayerRunner(c, out_bf16=out_bf16)
    r.ramp()
    return r.back_to_back(steps, warmup, queued)


COPY_BYTES = 256 * 2 ** 20  # plain device-to-device copy used to scale the HBM byte counters
COPY_REPS = 3
MODEL_CHECK_COMMANDS = [
    f"rocprofv3 --pmc {cnt} --output-format csv -d gpurun_out/model_check_{i} -o m -- python -u bench.py --traffic-run --layer all"
    for i, cnt in enumerate(["FETCH_SIZE", "WRITE_SIZE", "TCP_TCC_READ_REQ_sum", "SQ_INSTS_LDS"])
] + ["python bench.py --model-check gpurun_out/model_check_0 gpurun_out/model_check_1 "
     "gpurun_out/model_check_2 gpurun_out/model_check_3"]
TRAFFIC_COMMANDS = [
    "rocprofv3 --pmc FETCH_SIZE --output-format csv -d gpurun_out/traffic_fetch -o f -- python -u bench.py --traffic-run",
    "rocprofv3 --pmc WRITE_SIZE --output-format csv -d gpurun_out/traffic_write -o w -- python -u bench.py --traffic-run",
    "python bench.py --traffic-parse gpurun_out/traffic_fetch gpurun_out/traffic_write",
]


def traffic_run(layers, launches=6):
    """Workload for the rocprofv3 --pmc counter passes (one counter set per
    run): COPY_REPS plain copies of COPY_BYTES, then `launches` launches of
    each layer's selected plan on rotating buffer sets, layer after layer.
    Inputs are generated on the device so that no other copy kernel runs in
    this process."""
    import torch
    from paper_2101_09808_amd import conv as B

    dev = torch.device("cuda:0")
    src = torch.empty(COPY_BYTES // 4, device=dev).uniform_(-1, 1)
    dst = torch.empty_like(src)
    for _ in range(COPY_REPS):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    for c in layers:
        if c.stride != 1 or c.pad != 0:
            raise ValueError(f"{c.name}: the traffic run launches stride-1 valid layers only")
        bf16 = c.dtype == "bf16"
        edt = torch.bfloat16 if bf16 else torch.float32
        nsets = buffer_sets(c.N * c.C * c.H * c.W * (2 if bf16 else 4), c.N * c.K * c.P * c.Q * 4)
        ins = [torch.empty(c.N, c.C, c.H, c.W, device=dev).uniform_(-1, 1).to(edt) for _ in range(nsets)]
        Ker = torch.empty(c.K, c.C, c.R, c.S, device=dev).uniform_(-1, 1).to(edt)
        outs = [torch.empty(c.N, c.K, c.P, c.Q, device=dev) for _ in range(nsets)]
        torch.cuda.synchronize()
        sp = torch.cuda.current_stream().cuda_stream
        for i in range(launches):
            st = B.conv_fwd_ptr(*c.key(), ins[i % nsets].data_ptr(), Ker.data_ptr(), outs[i % nsets].data_ptr(),
                                sp, bf16)
            if st != B.CONV_OK:
                raise B.ConvError(st, "conv_fwd")
        torch.cuda.synchronize()
        del ins, outs, Ker
        print(f"traffic run: {launches} launches of {c.name}", flush=True)
    print(f"traffic run: {COPY_REPS} copies of {COPY_BYTES} B first", flush=True)


def counter_per_dispatch(d, counter):
    """[(kernel name, counter value summed over instances)] in dispatch order
    from the counter_collection.csv of one rocprofv3 --pmc run."""
    import csv
    import glob

    f = sorted(glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True))
    if not f:
        raise SystemExit(f"no counter_collection.csv under {d}")
    vals = {}
    for r in csv.DictReader(open(f[0])):
        if r["Counter_Name"] != counter:
            continue
        k = int(r["Dispatch_Id"])
        name, v = vals.get(k, (r["Kernel_Name"], 0.0))
        vals[k] = (name, v + float(r["Counter_Value"]))
    return [vals[k] for k in sorted(vals)]


def calibrated(d, counter, unit_bytes, layers, launches):
    """Per layer: bytes per launch implied by `counter` (in units of
    `unit_bytes`), scaled by copy bytes / what the counter reads for the
    plain copies.  The first launch of each layer (which also faults in the
    buffers) is left out."""
    rows = counter_per_dispatch(d, counter)
    # a split plan's launch is two dispatches: the main kernel, then the
    # reduction of its channel ranges, counted together
    conv = []
    for n, v in rows:
        if "convfwd::" not in n:
            continue
        if "splitk_reduce" in n and conv:
            conv[-1] += v
        else:
            conv.append(v)
    # the calibration copies are the process's first copy kernels (later ones,
    # e.g. dtype conversions of the inputs, are not of known size)
    first_conv = next((i for i, (n, _) in enumerate(rows) if "convfwd::" in n), len(rows))
    copy = [v for n, v in rows[:first_conv] if "copy" in n.lower()][:COPY_REPS]
    if len(copy) != COPY_REPS or len(conv) != launches * len(layers):
        raise SystemExit(f"{counter}: expected {COPY_REPS} copy and {launches * len(layers)} conv dispatches, "
                         f"got {len(copy)} and {len(conv)}")
    # counters a plain copy does not move (instruction counts) are not scaled
    factor = COPY_BYTES * COPY_REPS / (sum(copy) * unit_bytes) if sum(copy) > 0 else 1.0
    out = {}
    for i, c in enumerate(layers):
        mine = conv[i * launches + 1:(i + 1) * launches]
        per = sum(mine) / len(mine)
        out[c.name] = {"per_dispatch": per, "bytes_per_launch": per * unit_bytes * factor}
    return factor, sum(copy) / len(copy), out


def traffic_parse(c, fetch_dir, write_dir, out_path, launches=6):
    """HBM bytes per launch of the timed layer from the FETCH_SIZE and
    WRITE_SIZE runs (KiB per dispatch, scaled by the plain copy), stored with
    the hash of the launched kernel's source and plan (plan_kernel_hash)."""
    from paper_2101_09808_amd import conv as B

    res = {}
    for key, counter, d in (("fetch", "FETCH_SIZE", fetch_dir), ("write", "WRITE_SIZE", write_dir)):
        factor, copy_per, per_layer = calibrated(d, counter, 1024.0, [c], launches)
        res[key] = {"kib_per_dispatch": per_layer[c.name]["per_dispatch"], "copy_kib_per_dispatch": copy_per,
                    "factor": factor, "bytes_per_launch": per_layer[c.name]["bytes_per_launch"]}
    dtype_code = B.CONV_DTYPE_BF16 if c.dtype == "bf16" else B.CONV_DTYPE_F32
    plan = B.conv_fwd_plan(*c.key(), dtype=dtype_code)
    out = {"workload": c.name, "kernel_sha": plan_kernel_hash(c, plan), "plan_variant": plan["variant"],
           "copy_bytes": COPY_BYTES, "copy_reps": COPY_REPS,
           "fetch": res["fetch"], "write": res["write"],
           "hbm_bytes_per_launch": res["fetch"]["bytes_per_launch"] + res["write"]["bytes_per_launch"],
           "alg_bytes_per_launch": alg_bytes(c), "commands": TRAFFIC_COMMANDS}
    with open(out_path, "w") as fh:
        json.dump(out, fh, indent=1)
    print(json.dumps(out), flush=True)


MODEL_CHECK_COUNTERS = [("FETCH_SIZE", 1024.0), ("WRITE_SIZE", 1024.0), ("TCP_TCC_READ_REQ_sum", 1.0),
                        ("SQ_INSTS_LDS", 1.0)]
MODEL_CHECK_FILE = os.path.join(ROOT, "profiles", "model_vs_counters")


def model_check_parse(layers, dirs, launches=6):
    """The selector's predicted bytes per level against counters, per layer
    (one counter run per directory, in MODEL_CHECK_COUNTERS order).

    * HBM level (compulsory In + Ker + Out): FETCH_SIZE + WRITE_SIZE, both
      scaled by the plain copy.  MALL hits count as fetches, so this is the
      traffic out of the L2s, an upper bound of the HBM traffic.
    * L2 -> CU traffic: TCP_TCC_READ_REQ (L1 -> L2 read requests), scaled by
      the copy's bytes per request.  Predicted: the LDS level of the model
      (In and Ker tiles staged per workgroup), plus In itself for the
      pointwise streaming kernels, whose In loads go to registers.
    * Operand (REG) level: LDS instructions (SQ_INSTS_LDS, per wave), shown
      beside the predicted operand bytes; the byte figure per instruction
      depends on each kernel's read widths, so only the count is measured.
    """
    from paper_2101_09808_amd import conv as B

    meas = {}
    cal = {}
    for (counter, unit), d in zip(MODEL_CHECK_COUNTERS, dirs):
        factor, copy_per, per_layer = calibrated(d, counter, unit, layers, launches)
        cal[counter] = {"factor": factor, "copy_per_dispatch": copy_per}
        for name, v in per_layer.items():
            meas.setdefault(name, {})[counter] = v
    rows = []
    for c in layers:
        dtype_code = B.CONV_DTYPE_BF16 if c.dtype == "bf16" else B.CONV_DTYPE_F32
        plan = B.conv_fwd_plan(*c.key(), dtype=dtype_code)
        fam = B.conv_fwd_geometry(*c.key(), plan)["family"]
        m = meas[c.name]
        pb = plan["pred_bytes"]
        e = 2 if c.dtype == "bf16" else 4
        in_bytes = c.N * c.C * c.H * c.W * e
        pred_l2cu = pb["lds"] + (in_bytes if fam in (4, 5, 7) else 0)
        out_bytes = c.N * c.K * c.P * c.Q * 4
        hbm = m["FETCH_SIZE"]["bytes_per_launch"] + m["WRITE_SIZE"]["bytes_per_launch"]
        l2cu = m["TCP_TCC_READ_REQ_sum"]["bytes_per_launch"]
        rows.append({"workload": c.name, "plan_variant": plan["variant"], "family": fam,
                     "plan_kernel_sha": plan_kernel_hash(c, plan),
                     "hbm_pred": pb["hbm"], "hbm_meas": hbm, "hbm_ratio": hbm / pb["hbm"],
                     "l2_pred": pb["l2"] + out_bytes, "l2_ratio": hbm / (pb["l2"] + out_bytes),
                     "l2cu_pred": pred_l2cu, "l2cu_meas": l2cu, "l2cu_ratio": l2cu / pred_l2cu,
                     "reg_pred_bytes": pb["reg"], "lds_instructions": m["SQ_INSTS_LDS"]["per_dispatch"],
                     "fetch_bytes": m["FETCH_SIZE"]["bytes_per_launch"],
                     "write_bytes": m["WRITE_SIZE"]["bytes_per_launch"]})
    out = {"kernel_sha": kernel_source_hash(), "calibration": cal, "copy_bytes": COPY_BYTES,
           "copy_reps": COPY_REPS, "launches_per_layer": launches, "layers": rows,
           "commands": MODEL_CHECK_COMMANDS}
    with open(MODEL_CHECK_FILE + ".json", "w") as fh:
        json.dump(out, fh, indent=1)
    lines = ["# Predicted vs measured bytes per level (selected plan of each layer)", "",
             "Commands (MI355X, one GPU, from the repository root), one counter per run:", ""]
    lines += ["    " + x for x in MODEL_CHECK_COMMANDS]
    lines += ["", "Scale factors (plain 256 MiB copy: copy bytes / counter reading): " +
              ", ".join(f"{k} {v['factor']:.4g}" for k, v in cal.items() if k != "SQ_INSTS_LDS"), "",
              "| layer | variant | fabric meas MB | compulsory MB | ratio | L2 level + Out pred MB | ratio |"
              " L2->CU pred MB | L2->CU meas MB | ratio | REG pred MB | LDS instr |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {r['workload']} | {r['plan_variant']} | {r['hbm_meas'] / 1e6:.2f} | {r['hbm_pred'] / 1e6:.2f} | "
                     f"{r['hbm_ratio']:.3f} | {r['l2_pred'] / 1e6:.2f} | {r['l2_ratio']:.3f} | "
                     f"{r['l2cu_pred'] / 1e6:.2f} | {r['l2cu_meas'] / 1e6:.2f} | "
                     f"{r['l2cu_ratio']:.3f} | {r['reg_pred_bytes'] / 1e6:.1f} | {r['lds_instructions']:.4g} |")
    lines += ["", "Fabric: FETCH_SIZE + WRITE_SIZE, the traffic between the XCDs' L2s and the fabric (MALL hits",
              "count as fetches), against the compulsory In + Ker + Out (the model's HBM level) and against the",
              "model's L2 level (per-XCD re-fetches of In and Ker) plus Out.  L2->CU: TCP_TCC_READ_REQ against",
              "the model's LDS level (plus In for the pointwise streaming kernels, which load In into",
              "registers).  REG: predicted operand bytes beside the measured LDS instruction count",
              "(SQ_INSTS_LDS).", ""]
    with open(MODEL_CHECK_FILE + ".md", "w") as fh:
        fh.write("\n".join(lines))
    print(json.dumps(out), flush=True)


# per-plan raw results of the sweeps (large; the committed summaries are the .md
# files beside them and calibration/ratios.txt in the package)
RAW_DIR = os.path.join(ROOT, "gpurun_out")
RANK_JSON = os.path.join(RAW_DIR, "model_rank_sweep.json")
RANK_MD = os.path.join(ROOT, "profiles", "model_rank_sweep.md")


def rank_sample(cands, n=100, top=5, seed=0):
    """Indices (model order) of the plans a rank sweep times: the model's
    `top` best plans plus a uniform sample without replacement of the rest,
    `n` in all (Sec. 9 samples about 100 configurations per operator)."""
    import random
    head = list(range(min(top, len(cands))))
    rest = list(range(len(head), len(cands)))
    return sorted(head + random.Random(seed).sample(rest, max(0, min(n - len(head), len(rest)))))


def ranks(x):
    """Ranks 1..n of the values x, ties sharing their average rank."""
    order = sorted(range(len(x)), key=lambda i: x[i])
    r = [0.0] * len(x)
    i = 0
    while i < len(order):
        j = i
        while j + 1 < len(order) and x[order[j + 1]] == x[order[i]]:
            j += 1
        for t in range(i, j + 1):
            r[order[t]] = (i + j) / 2.0 + 1.0
        i = j + 1
    return r


def spearman(x, y):
    """Spearman rank correlation: Pearson correlation of the tie-averaged ranks."""
    rx, ry = ranks(x), ranks(y)
    n = len(x)
    mx, my = sum(rx) / n, sum(ry) / n
    sxy = sum((a - mx) * (b - my) for a, b in zip(rx, ry))
    sxx = sum((a - mx) ** 2 for a in rx)
    syy = sum((b - my) ** 2 for b in ry)
    return sxy / (sxx * syy) ** 0.5 if sxx > 0 and syy > 0 else float("nan")


def topk_loss(times_in_model_order, k):
    """Loss of performance of the best of the model's top k plans against the
    best plan measured (Sec. 9): time ratio minus one."""
    return min(times_in_model_order[:k]) / min(times_in_model_order) - 1.0


_SLEEP_RATE = []


def sleep_cycles_per_us():
    """Rate of torch.cuda._sleep (a bounded spin kernel) on this device."""
    import torch
    if not _SLEEP_RATE:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(1000)
        e0.record()
        torch.cuda._sleep(2_000_000)
        e1.record()
        torch.cuda.synchronize()
        _SLEEP_RATE.append(2_000_000 / max(1.0, e0.elapsed_time(e1) * 1e3))
    return _SLEEP_RATE[0]


def time_plan(c, plan, ins, outs, Ker, reps=10):
    """Median launch duration of an explicit plan over `reps` launches on
    rotating buffer sets (after two untimed launches), each bracketed by its
    own pair of HIP events on the launch stream.  The launches queue up
    behind a bounded spin kernel and then run back to back, so host time
    between them does not count (a split plan's launch is its two kernels)."""
    import ctypes
    import torch
    from paper_2101_09808_amd import conv as B
    L = B.lib()
    p = B.ConvPlan.from_dict(plan)
    # the plan runs the stride-1 valid problem of c.key(): Out must hold it
    N, C, K, H, W, R, S = c.key()
    if any(t.numel() < N * K * (H - R + 1) * (W - S + 1) for t in outs):
        raise ValueError("Out buffers smaller than the valid convolution's output")
    if any(t.numel() < N * C * H * W for t in ins) or Ker.numel() < K * C * R * S:
        raise ValueError("input buffers smaller than the shape")
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    kp = Ker.data_ptr()
    n = len(ins)

    def fn(i):
        st = L.conv_fwd_with_plan(*c.key(), ins[i % n].data_ptr(), kp, outs[i % n].data_ptr(), ctypes.byref(p), sp)
        if st != B.CONV_OK:
            raise B.ConvError(st, "conv_fwd_with_plan")

    fn(0)
    fn(1)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    torch.cuda._sleep(int(sleep_cycles_per_us() * 300 * reps))  # launches below queue up behind it
    for i, (e0, e1) in enumerate(ev):
        e0.record(stream)
        fn(i + 2)
        e1.record(stream)
    torch.cuda.synchronize()
    t = sorted(e0.elapsed_time(e1) * 1e3 for e0, e1 in ev)
    return t[len(t) // 2]


def all_candidates(c, dt):
    from paper_2101_09808_amd import conv as B
    n = B.lib().conv_fwd_candidates(*c.key(), dt, None, 0)
    return B.conv_fwd_candidates(*c.key(), dtype=dt, cap=max(1, n))


def rank_sweep(configs, n=None, reps=10):
    """Model validation on the GPU (Sec. 9): per layer, time every candidate
    plan (n = None), or the model's top 5 and a uniform sample of the others
    (n plans); report the rank correlation of predicted and measured time
    and the top-1/2/5 loss against the fastest timed plan, plus the
    empirical pick among the top 5 (Sec. 10, MOpt-5)."""
    import torch
    from paper_2101_09808_amd import conv as B
    from paper_2101_09808_amd.workloads import make_inputs
    res = {}
    for c in configs:
        dt = B.CONV_DTYPE_BF16 if c.dtype == "bf16" else B.CONV_DTYPE_F32
        cands = all_candidates(c, dt)
        idx = list(range(len(cands))) if n is None else rank_sample(cands, n=n, seed=c.seed)
        In0, Ker0 = make_inputs(c)
        nsets = buffer_sets(In0.numel() * In0.element_size(), c.N * c.K * c.P * c.Q * 4)
        ins = [In0.cuda() for _ in range(nsets)]
        outs = [torch.empty(c.N, c.K, c.P, c.Q, device="cuda") for _ in range(nsets)]
        Ker = Ker0.cuda()
        for i in range(30):  # clocks up before the first timed plan
            B.conv_fwd_with_plan(ins[i % nsets], Ker, cands[0], out=outs[i % nsets])
        rows = []
        for i in idx:
            p = cands[i]
            us = time_plan(c, p, ins, outs, Ker, reps)
            rows.append({"model_rank": i, "variant": p["variant"], "split_c": p["split_c"],
                         "tile": [p["tile_k"], p["tile_rows"], p["tile_cols"], p["tile_c"]],
                         "grid_order": p["grid_order"], "pred_us": p["pred_total_us"], "rank_us": p["rank_us"],
                         "measured_us": us})
            if len(rows) % 200 == 1 or i < 5:
                print(f"[rank] {c.name} rank {i} v{p['variant']} split {p['split_c']} pred {p['pred_total_us']:.1f} "
                      f"measured {us:.1f} us ({len(rows)}/{len(idx)})", flush=True)
        t = [r["measured_us"] for r in rows]  # model order
        best = min(t)
        res[c.name] = {
            "shape": list(c.key()), "dtype": c.dtype,
            "candidates": len(cands), "sampled": len(rows),
            "spearman_rank_vs_measured": spearman([r["model_rank"] for r in rows], t),
            "spearman_pred_us_vs_measured": spearman([r["pred_us"] for r in rows], t),
            "top1_loss": topk_loss(t, 1), "top2_loss": topk_loss(t, 2), "top5_loss": topk_loss(t, 5),
            "mopt1_us": t[0], "mopt5_us": min(t[:5]), "best_sampled_us": best,
            "best_sampled": min(rows, key=lambda r: r["measured_us"]),
            "plans": rows,
        }
        del ins, outs
        torch.cuda.empty_cache()
    return res


def rank_report(res, title="Model-predicted rank vs measured time (Sec. 9), MI355X",
                command="python bench.py --rank-sweep", intro=""):
    lines = ["# " + title, "",
             (intro + " " if intro else "") +
             "Per layer: every candidate plan the selector scores (or, where marked, the model's 5 best "
             "plus a uniform sample of the others), each the median of 10 launches on rotating buffer sets, "
             "every launch between its own pair of HIP events, queued behind a spin kernel so that they run "
             "back to back (no host time).  Spearman "
             "correlation of the model's order (and of its predicted time) with the measured time; "
             "top-k loss = best of the model's first k plans over the fastest timed plan, "
             "minus 1; MOpt-1 = the selector's plan, MOpt-5 = best of its top 5 (Sec. 10).", "",
             f"Command: `{command}`", "",
             "| layer | candidates | timed | rho(rank) | rho(pred us) | top-1 loss | top-2 loss | top-5 loss "
             "| MOpt-1 us | MOpt-5 us | fastest us (variant, model rank) |",
             "|---|---|---|---|---|---|---|---|---|---|---|"]
    for name, r in res.items():
        b = r["best_sampled"]
        shape = "x".join(str(x) for x in r.get("shape", [])) if name.startswith("heldout") else name
        lines.append(f"| {shape} | {r['candidates']} | {r['sampled']} | {r['spearman_rank_vs_measured']:.2f} | "
                     f"{r['spearman_pred_us_vs_measured']:.2f} | {100 * r['top1_loss']:.1f}% | "
                     f"{100 * r['top2_loss']:.1f}% | {100 * r['top5_loss']:.1f}% | {r['mopt1_us']:.1f} | "
                     f"{r['mopt5_us']:.1f} | {b['measured_us']:.1f} (v{b['variant']}, rank {b['model_rank']}) |")
    return "\n".join(lines) + "\n"


HELDOUT_JSON = os.path.join(RAW_DIR, "model_heldout.json")
HELDOUT_MD = os.path.join(ROOT, "profiles", "model_heldout.md")
TRAIN_JSON = os.path.join(RAW_DIR, "model_train_sweep.json")
TRAIN_MD = os.path.join(ROOT, "profiles", "model_train_sweep.md")
HELDOUT_SEED, TRAIN_SEED = 78, 77


def heldout_layers(n=10, seed=HELDOUT_SEED, n_bf16=None):
    """Seeded random layers.  Seed 77 (the training set) joins the five
    configurations in the per-variant calibration of the selector; seed 78
    (the held-out set) is used for validation only.  `n` fp32 shapes in
    Table 1's range: batch 1-32, 16-512 channels, 7-58 pixels, 1x1 and 3x3
    taps, valid stride 1; then `n_bf16` (default 4 for training, 3 held out)
    bf16 first-layer shapes (32 input channels, 32-64 filters, 3x3, 58-226
    pixels, batch 2-16: the family of the 226x226 layer, whose kernels no
    fp32 layer runs), drawn from a stream of their own so that the fp32
    shapes do not depend on them."""
    import random

    from paper_2101_09808_amd.workloads import ConvShape
    rng = random.Random(seed)
    out = []
    while len(out) < n:
        RS = rng.choice([1, 3, 3])
        N = rng.choice([1, 2, 4, 8, 16, 32])
        C = rng.choice([16, 32, 48, 64, 96, 128, 192, 256, 384, 512])
        K = rng.choice([16, 32, 64, 96, 128, 192, 256, 384, 512])
        HW = rng.randint(7, 58) + RS - 1
        if N * C * HW * HW * 4 > 200e6 or N * K * HW * HW > 40e6:
            continue
        out.append(ConvShape(f"heldout{len(out)}" if seed == HELDOUT_SEED else f"train{len(out)}", N, C, K, HW, HW,
                             RS, RS, "f32", 12000 + 100 * (seed - TRAIN_SEED) + len(out)))
    if n_bf16 is None:
        n_bf16 = 4 if seed == TRAIN_SEED else 3
    rng = random.Random(1000 + seed)
    while len(out) < n + n_bf16:
        N = rng.choice([2, 4, 8, 16])
        K = rng.choice([32, 48, 64])
        HW = rng.choice([56, 112, 168, 224]) + 2  # Out rows divisible by 4, 7, 8 and 14
        if N * K * (HW - 2) ** 2 * 4 > 400e6:
            continue
        out.append(ConvShape(f"heldout{len(out)}" if seed == HELDOUT_SEED else f"train{len(out)}", N, 32, K, HW, HW,
                             3, 3, "bf16", 12000 + 100 * (seed - TRAIN_SEED) + len(out)))
    return out


def heldout_report(res, train=False):
    if train:
        return rank_report(res, title="Model rank vs measured time on the calibration layers (Sec. 9), MI355X",
                           command="python bench.py --train-sweep",
                           intro="Ten seeded random fp32 layers (bench.py heldout_layers, seed 77: batch 1-32, 16-512 "
                                 "channels, 7-58 pixels, 1x1 and 3x3) and four bf16 first layers (32 input channels, "
                                 "3x3, 58-226 pixels) that, with the five configurations, set the selector's "
                                 "per-variant calibration (paper_2101_09808_amd/calibrate.py).")
    return rank_report(res, title="Model rank vs measured time on held-out layers (Sec. 9), MI355X",
                       command="python bench.py --held-out",
                       intro="Ten seeded random fp32 layers (bench.py heldout_layers, seed 78: batch 1-32, 16-512 "
                             "channels, 7-58 pixels, 1x1 and 3x3) and three bf16 first layers (32 input channels, "
                             "3x3, 58-226 pixels) that none of the model's measured constants (calibration "
                             "included) were fitted on.")


BREAKDOWN_COUNTERS = ["GRBM_GUI_ACTIVE", "SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_WAIT_INST_ANY",
                      "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_ACTIVE_INST_VMEM", "SQ_ACTIVE_INST_LDS", "SQ_WAIT_INST_LDS"]
BREAKDOWN_FILE = os.path.join(ROOT, "profiles", "cycle_breakdown_per_layer.md")
BREAKDOWN_COMMANDS = [
    "rocprofv3 --kernel-trace --pmc " + " ".join(BREAKDOWN_COUNTERS) +
    " --output-format csv -d gpurun_out/breakdown -o b -- python -u bench.py --traffic-run --layer all",
    "python bench.py --breakdown-parse gpurun_out/breakdown"]


def breakdown_parse(layers, d, launches=6):
    """Where each layer's waves spend their cycles (one counter pass with the
    kernel trace): MFMA-pipe busy share of the SIMD cycles, the share of
    wave cycles spent waiting on a dependency (memory or LDS), and the clock
    the counters imply.  SQ_WAVE_CYCLES and SQ_WAIT_INST_* count in units of
    four cycles (quad cycles), summed over waves; SQ_BUSY_CYCLES in cycles,
    summed over the chip's 32 shader engines."""
    import csv
    import glob
    cc = sorted(glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True))[0]
    tr = sorted(glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True))[0]
    dur = {int(r["Dispatch_Id"]): int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in csv.DictReader(open(tr))}
    vals, names = {}, {}
    for r in csv.DictReader(open(cc)):
        k = int(r["Dispatch_Id"])
        vals.setdefault(k, {})
        vals[k][r["Counter_Name"]] = vals[k].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        names[k] = r["Kernel_Name"]
    conv = [k for k in sorted(vals) if "convfwd::" in names[k] and "reduce" not in names[k]]
    if len(conv) != launches * len(layers):
        raise SystemExit(f"expected {launches * len(layers)} conv dispatches, got {len(conv)}")
    lines = ["# Where the waves spend their cycles, per layer (selected plans), MI355X", "",
             "One rocprofv3 counter pass with the kernel trace over `bench.py --traffic-run --layer all` "
             "(six launches of each layer's selected plan; the first left out):", ""]
    lines += ["    " + x for x in BREAKDOWN_COMMANDS]
    lines += ["", "* MFMA busy: SQ_VALU_MFMA_BUSY_CYCLES over (SIMDs x kernel cycles), the share of the chip's "
              "MFMA pipe time in use; kernel cycles from the trace duration at the clock below.",
              "* Waiting: SQ_WAIT_INST_ANY over SQ_WAVE_CYCLES, the share of resident-wave time stalled on a "
              "dependency (a load, an LDS read, a barrier); LDS waits separately (SQ_WAIT_INST_LDS).",
              "* Clock: SQ_BUSY_CYCLES / 32 shader engines over the kernel's duration (busy time of the "
              "shader engines, so a lower bound of the clock while the kernel runs).", "",
              "| layer | kernel us | clock GHz (>=) | MFMA busy | waiting | LDS waits | waves |",
              "|---|---|---|---|---|---|---|"]
    rows = {}
    for i, c in enumerate(layers):
        ks = conv[i * launches + 1:(i + 1) * launches]
        us = sum(dur[k] for k in ks) / len(ks) / 1e3
        m = {n: sum(vals[k].get(n, 0.0) for k in ks) / len(ks) for n in BREAKDOWN_COUNTERS}
        ghz = m["SQ_BUSY_CYCLES"] / 32 / (us * 1e3)
        mfma = m["SQ_VALU_MFMA_BUSY_CYCLES"] / (1024 * us * 1e3 * ghz)
        wait = m["SQ_WAIT_INST_ANY"] / max(1.0, m["SQ_WAVE_CYCLES"])
        lwait = m["SQ_WAIT_INST_LDS"] / max(1.0, m["SQ_WAVE_CYCLES"])
        rows[c.name] = {"kernel_us": us, "clock_ghz_lower_bound": ghz, "mfma_busy": mfma, "waiting": wait,
                        "lds_waiting": lwait, "waves": m["SQ_WAVES"], "counters": m}
        lines.append(f"| {c.name} | {us:.1f} | {ghz:.2f} | {100 * mfma:.0f}% | {100 * wait:.0f}% | "
                     f"{100 * lwait:.0f}% | {m['SQ_WAVES']:.0f} |")
    open(BREAKDOWN_FILE, "w").write("\n".join(lines) + "\n")
    json.dump(rows, open(BREAKDOWN_FILE.replace(".md", ".json"), "w"), indent=1)
    print("\n".join(lines), flush=True)


COUNTER_SWEEP_LAYER = "conv3x3_n32_c128_k128_in30"
COUNTER_SWEEP_COUNTERS = [["FETCH_SIZE"], ["TCP_TCC_READ_REQ_sum"], ["SQ_INSTS_LDS", "SQ_LDS_BANK_CONFLICT"]]
COUNTER_SWEEP_JSON = os.path.join(RAW_DIR, "model_counter_sweep.json")
COUNTER_SWEEP_MD = os.path.join(ROOT, "profiles", "model_counter_sweep.md")


def counter_sweep_plans(c, n):
    from paper_2101_09808_amd import conv as B
    dt = B.CONV_DTYPE_BF16 if c.dtype == "bf16" else B.CONV_DTYPE_F32
    cands = all_candidates(c, dt)
    return cands, rank_sample(cands, n=n, seed=c.seed)


def counter_sweep(c, n):
    """Workload of the counter passes: each sampled plan once (after one
    untimed launch of the selected plan), in model order, with a
    synchronisation after each so that dispatches are one plan each."""
    import ctypes

    import torch
    from paper_2101_09808_amd import conv as B
    from paper_2101_09808_amd.workloads import make_inputs
    cands, idx = counter_sweep_plans(c, n)
    In0, Ker0 = make_inputs(c)
    In, Ker = In0.cuda(), Ker0.cuda()
    out = torch.empty(c.N, c.K, c.P, c.Q, device="cuda")
    L = B.lib()
    sp = torch.cuda.current_stream().cuda_stream
    for i in idx:
        p = B.ConvPlan.from_dict(cands[i])
        st = L.conv_fwd_with_plan(*c.key(), In.data_ptr(), Ker.data_ptr(), out.data_ptr(), ctypes.byref(p), sp)
        if st != B.CONV_OK:
            raise B.ConvError(st, "conv_fwd_with_plan")
        torch.cuda.synchronize()
    print(f"counter sweep: {len(idx)} plans of {c.name}", flush=True)


def counter_sweep_parse(c, dirs):
    """Fig. 6 analogue: per plan, the counters of the sweep passes (one pass
    per directory, COUNTER_SWEEP_COUNTERS order) beside the model's levels,
    with the Spearman correlation of each counter with the model's rank, and
    with the measured time where the rank sweep timed the same plans."""
    cands, idx = counter_sweep_plans(c, 100)
    per = {}
    for cnts, d in zip(COUNTER_SWEEP_COUNTERS, dirs):
        for cnt in cnts:
            rows = [v for name, v in counter_per_dispatch(d, cnt) if "convfwd::" in name and "reduce" not in name]
            if len(rows) != len(idx):
                raise SystemExit(f"{cnt}: {len(rows)} conv dispatches for {len(idx)} plans")
            per[cnt] = rows
    timed = {}
    if os.path.exists(RANK_JSON):
        rj = json.load(open(RANK_JSON)).get(c.name, {})
        timed = {r["model_rank"]: r["measured_us"] for r in rj.get("plans", [])}
    plans = []
    for j, i in enumerate(idx):
        p = cands[i]
        row = {"model_rank": i, "variant": p["variant"], "tile": [p["tile_k"], p["tile_rows"], p["tile_cols"]],
               "pred_us": p["pred_total_us"], "pred_lds_bytes": p["pred_bytes"]["lds"],
               "pred_reg_bytes": p["pred_bytes"]["reg"], "pred_l2_bytes": p["pred_bytes"]["l2"],
               "fetch_kib": per["FETCH_SIZE"][j], "l2_to_cu_req": per["TCP_TCC_READ_REQ_sum"][j],
               "lds_instr": per["SQ_INSTS_LDS"][j], "lds_bank_conflict_cycles": per["SQ_LDS_BANK_CONFLICT"][j],
               "measured_us": timed.get(i)}
        plans.append(row)
    rank = [r["model_rank"] for r in plans]
    out = {"layer": c.name, "plans": plans, "spearman": {}, "commands": COUNTER_SWEEP_COMMANDS}
    pairs = [("fetch_kib", "pred_l2_bytes"), ("l2_to_cu_req", "pred_lds_bytes"), ("lds_instr", "pred_reg_bytes"),
             ("lds_bank_conflict_cycles", None)]
    for cnt, pred in pairs:
        v = [r[cnt] for r in plans]
        e = {"vs_model_rank": spearman(rank, v)}
        if pred:
            e["vs_predicted_level"] = spearman([r[pred] for r in plans], v)
        t = [(r["measured_us"], r[cnt]) for r in plans if r["measured_us"] is not None]
        if len(t) > 2:
            e["vs_measured_time"] = spearman([a for a, _ in t], [b for _, b in t])
        out["spearman"][cnt] = e
    conflicts = sum(r["lds_bank_conflict_cycles"] for r in plans) / max(1.0, sum(r["lds_instr"] for r in plans))
    out["bank_conflict_cycles_per_lds_instr"] = conflicts
    os.makedirs(RAW_DIR, exist_ok=True)
    json.dump(out, open(COUNTER_SWEEP_JSON, "w"), indent=1)
    lines = [f"# Counters per plan against the model (Fig. 6 analogue), {c.name}, MI355X", "",
             "The model's 5 best plans and a uniform sample of the other candidates (100 in all), each "
             "launched once under rocprofv3 counter passes (one pass per counter group):", ""]
    lines += ["    " + x for x in COUNTER_SWEEP_COMMANDS]
    lines += ["", "Spearman correlation of each counter with the model's rank, with the model's "
              "prediction of the level it measures, and with the measured time (rank sweep):", "",
              "| counter | level predicted | rho vs model rank | rho vs predicted level | rho vs measured time |",
              "|---|---|---|---|---|"]
    for cnt, pred in pairs:
        e = out["spearman"][cnt]
        f = lambda k: f"{e[k]:.2f}" if k in e else "-"
        lines.append(f"| {cnt} | {pred or '-'} | {f('vs_model_rank')} | {f('vs_predicted_level')} | "
                     f"{f('vs_measured_time')} |")
    sel = plans[0]
    lines += ["", f"LDS bank conflicts: {conflicts:.4f} conflict cycles per LDS instruction over the sample; "
              f"the selected plan (model rank 0, variant {sel['variant']}): "
              f"{sel['lds_bank_conflict_cycles']:.0f} cycles over {sel['lds_instr']:.0f} LDS instructions.", ""]
    lines += ["| model rank | variant | tile k x rows x cols | pred us | measured us | FETCH KiB | L2->CU req | "
              "LDS instr | bank-conflict cycles |", "|---|---|---|---|---|---|---|---|---|"]
    for r in plans[:25]:
        lines.append(f"| {r['model_rank']} | {r['variant']} | {'x'.join(map(str, r['tile']))} | {r['pred_us']:.1f} | "
                     f"{'-' if r['measured_us'] is None else format(r['measured_us'], '.1f')} | "
                     f"{r['fetch_kib']:.0f} | {r['l2_to_cu_req']:.0f} | {r['lds_instr']:.0f} | "
                     f"{r['lds_bank_conflict_cycles']:.0f} |")
    lines.append(f"\n(first 25 of {len(plans)} plans; the parse writes all of them to its per-plan JSON)\n")
    open(COUNTER_SWEEP_MD, "w").write("\n".join(lines))
    print("\n".join(lines[:20]), flush=True)


COUNTER_SWEEP_COMMANDS = [
    f"rocprofv3 --pmc {' '.join(cs)} --output-format csv -d gpurun_out/counter_sweep_{i} -o s -- "
    f"python -u bench.py --counter-sweep --layer {COUNTER_SWEEP_LAYER}"
    for i, cs in enumerate(COUNTER_SWEEP_COUNTERS)
] + [f"python bench.py --counter-sweep-parse gpurun_out/counter_sweep_0 gpurun_out/counter_sweep_1 "
     f"gpurun_out/counter_sweep_2 --layer {COUNTER_SWEEP_LAYER}"]


TABLE1_JSON = os.path.join(ROOT, "profiles", "table1_sweep.json")
TABLE1_MD = os.path.join(ROOT, "profiles", "table1_sweep.md")


def table1_sweep():
    """Every conv2d layer of Table 1 (Yolo-9000, ResNet-18) at batch 1 with
    its stride and same padding: launch time (median of queued launches on
    rotating buffers), achieved rates and the roofline bound of the layer."""
    from paper_2101_09808_amd import conv as B
    from paper_2101_09808_amd.workloads import TABLE1
    rows = {}
    for c in TABLE1:
        lk = time_layer(c, 30, 5, queued=True)["mean_kernel_ms"] * 1e-3
        inner = B.conv_fwd_ex_inner_shape(*c.key(), c.stride, c.pad)
        plan, direct = B.conv_fwd_ex_plan(*c.key(), c.stride, c.pad)
        F, Bt = flops(c), alg_bytes(c)
        t_mfma, t_hbm = F / (PEAK["fp32_mfma_tflops"] * 1e12), Bt / (PEAK["hbm_gbs"] * 1e9)
        bound = "mfma" if t_mfma >= t_hbm else "hbm"
        rows[c.name] = {
            "K": c.K, "C": c.C, "HW": c.H, "RS": c.R, "stride": c.stride, "pad": c.pad,
            "inner_shape": list(inner[:7]), "variant": plan["variant"], "split_c": plan["split_c"],
            "direct": direct, "pred_us": plan["pred_total_us"], "kernel_us": lk * 1e6, "gflops": F / lk / 1e9,
            "pct_fp32_mfma_peak": 100 * F / lk / 1e12 / PEAK["fp32_mfma_tflops"],
            "alg_hbm_gbs": Bt / lk / 1e9, "pct_hbm_peak": 100 * Bt / lk / 1e9 / PEAK["hbm_gbs"],
            "bound": bound, "roofline_frac": max(t_mfma, t_hbm) / lk,
        }
        print(f"[table1] {c.name} {lk * 1e6:.1f} us", flush=True)
    return rows


def table1_report(rows):
    lines = ["# Table 1 conv2d layers at batch 1 (Yolo-9000, ResNet-18), MI355X, fp32", "",
             "Each layer with the table's stride and same padding (R // 2), through conv_fwd_ex: "
             "strided or padded layers are rewritten as a stride-1 valid convolution (inner shape "
             "C', H', R') and run with the selector's plan, which reads the caller's In through the phase "
             "mapping where its kernel can (plan marked d) and otherwise runs on a phase-split or padded "
             "copy of In.  Time = mean of 30 launches queued behind a "
             "spin kernel on rotating buffer sets, from HIP events.  Roofline fraction = time at the "
             "layer's bound (fp32 MFMA 157.3 TFLOP/s or HBM 8 TB/s) over the measured time.  The "
             "depth-wise MobileNet layers are not Eq. (1).", "",
             "Command: `python bench.py --table1`", "",
             "| layer | K | C | H=W | R=S | stride | inner (C', H', R') | plan | us | GFLOP/s | % fp32 peak "
             "| GB/s | bound | roofline frac |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for name, r in rows.items():
        ic = r["inner_shape"]
        lines.append(f"| {name.split('_', 1)[1]} | {r['K']} | {r['C']} | {r['HW']} | {r['RS']} | {r['stride']} | "
                     f"({ic[1]}, {ic[3]}, {ic[5]}) | v{r['variant']}/{r['split_c']}{' d' if r.get('direct') else ''} | "
                     f"{r['kernel_us']:.1f} | "
                     f"{r['gflops']:.0f} | {r['pct_fp32_mfma_peak']:.1f} | {r['alg_hbm_gbs']:.0f} | {r['bound']} | "
                     f"{r['roofline_frac']:.3f} |")
    return "\n".join(lines) + "\n"


def cpu_baseline(c, budget_s=10.0):
    """The fp64 oracle on this host's cores over a bounded batch sample."""
    import numpy as np

    from oracle import conv as oconv
    from paper_2101_09808_amd.workloads import make_inputs

    In, Ker = make_inputs(c)
    In = In.float().numpy()
    Ker = Ker.float().numpy()
    n = 1
    t0 = time.perf_counter()
    oconv.conv_fwd(In[:1], Ker)
    dt = time.perf_counter() - t0
    if dt < budget_s and c.N > 1:
        n = int(min(c.N, max(1, budget_s / max(dt, 1e-6))))
        t0 = time.perf_counter()
        oconv.conv_fwd(np.ascontiguousarray(In[:n]), Ker)
        dt = time.perf_counter() - t0
    reps = 1
    if n == c.N and dt < budget_s:  # the whole layer is cheap: repeat it for a stable rate
        reps = max(1, int(budget_s / max(dt, 1e-6)))
        t0 = time.perf_counter()
        for _ in range(reps):
            oconv.conv_fwd(In, Ker)
        dt = time.perf_counter() - t0
    f = flops(c) * n / c.N * reps
    return {"value": f / dt / 1e9, "unit": "GFLOP/s", "cores": oconv.num_threads(), "kind": "oracle",
            "sample": f"{n} of {c.N} images of {c.name}, {reps} pass(es) (fp64 plain loops, OpenMP over n,k), "
                      f"{dt:.2f} s"}


def cpu_baseline_one_thread(c):
    """The oracle on one host thread over the whole layer."""
    from oracle import conv as oconv
    from paper_2101_09808_amd.workloads import make_inputs

    In, Ker = make_inputs(c)
    In, Ker = In.float().numpy(), Ker.float().numpy()
    prev = oconv.set_num_threads(1)
    try:
        t0 = time.perf_counter()
        oconv.conv_fwd(In, Ker)
        dt = time.perf_counter() - t0
        cores = oconv.num_threads()
    finally:
        oconv.set_num_threads(prev)
    return {"value": flops(c) / dt / 1e9, "unit": "GFLOP/s", "cores": cores, "kind": "oracle",
            "sample": f"all of {c.name}, one pass (fp64 plain loops), {dt:.2f} s"}


def layer_counters():
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated) of each
    layer from the last counter passes, keyed by (layer, plan_kernel_hash):
    a figure is reported only for the plan and kernel source it was taken on."""
    path = MODEL_CHECK_FILE + ".json"
    if not os.path.exists(path):
        return {}
    d = json.load(open(path))
    out = {}
    for row in d.get("layers", []):
        h = row.get("plan_kernel_sha")
        if h and "fetch_bytes" in row:
            out[(row["workload"], h)] = {"fetch_bytes": row["fetch_bytes"], "write_bytes": row["write_bytes"],
                                        "hbm_bytes": row["fetch_bytes"] + row["write_bytes"],
                                        "ratio_to_alg": row.get("hbm_ratio")}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=500)
    ap.add_argument("--no-layers", action="store_true", help="skip the per-layer table")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--layer", default=HEADLINE, help="workload of the timed step ('all': every layer, "
                    "for --traffic-run)")
    ap.add_argument("--traffic-run", action="store_true",
                    help="plain copies + a few launches, for rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs")
    ap.add_argument("--traffic-parse", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="turn the two counter runs into the HBM traffic record read by the benchmark")
    ap.add_argument("--model-check", nargs=4, metavar=("FETCH", "WRITE", "TCP_TCC", "LDS"),
                    help="predicted vs measured bytes per level for every layer, from four counter runs "
                         "of --traffic-run --layer all")
    ap.add_argument("--rank-sweep", nargs="?", const=0, type=int, metavar="N",
                    help="model validation: time every candidate of every layer (or, with N, the model's "
                         "top 5 and a uniform sample of the others, N plans per layer); writes "
                         "profiles/model_rank_sweep.md (per-plan JSON: gpurun_out/)")
    ap.add_argument("--held-out", action="store_true",
                    help="the same validation on seeded random layers that none of the model's measured "
                         "constants were fitted on; writes profiles/model_heldout.md (per-plan JSON: gpurun_out/)")
    ap.add_argument("--train-sweep", action="store_true",
                    help="the same sweep on the seeded random layers that join the five configurations in the "
                         "selector's calibration; writes profiles/model_train_sweep.md (per-plan JSON: gpurun_out/)")
    ap.add_argument("--counter-sweep", nargs="?", const=100, type=int, metavar="N",
                    help="launch the model's top 5 and a sample of the other plans of --layer (N in all) "
                         "once each, for rocprofv3 --pmc counter passes (Fig. 6 analogue)")
    ap.add_argument("--breakdown-parse", metavar="DIR",
                    help="cycle breakdown per layer from one counter pass of --traffic-run --layer all; writes "
                         "profiles/cycle_breakdown_per_layer.{md,json}")
    ap.add_argument("--counter-sweep-parse", nargs="+", metavar="DIR",
                    help="per-plan counters of the --counter-sweep passes against the model's rank and "
                         "levels; writes profiles/model_counter_sweep.md (per-plan JSON: gpurun_out/)")
    ap.add_argument("--trace-summary", metavar="RESULTS_DB",
                    help="host only: the kernel table (calls, average/min/max us, workgroups) of a rocprofv3 "
                         "--kernel-trace results database")
    ap.add_argument("--table1", action="store_true",
                    help="every conv2d layer of Table 1 at batch 1 (stride, same padding); writes "
                         "profiles/table1_sweep.{json,md}")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on exactly one GPU (got --gpus {args.gpus}); "
              "the convolution shards by batch or output channel without communication, "
              "but no multi-GPU run is part of this benchmark.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2101_09808_amd import conv as B
    from paper_2101_09808_amd.workloads import BY_NAME, CONFIGS, STRIDED_CONFIGS, make_inputs

    if args.traffic_parse:  # host-only: reads the counter files of two earlier runs
        traffic_parse(BY_NAME[args.layer], args.traffic_parse[0], args.traffic_parse[1], TRAFFIC_FILE)
        return
    if args.model_check:  # host-only: reads the counter files of four earlier runs
        model_check_parse(list(CONFIGS), args.model_check)
        return
    if args.trace_summary:  # host-only: reads a rocprofv3 results database
        print(trace_summary(args.trace_summary), flush=True)
        return
    if args.breakdown_parse:  # host-only: reads the counter files of one pass
        breakdown_parse(list(CONFIGS), args.breakdown_parse)
        return
    if args.counter_sweep_parse:  # host-only: reads the counter files of the sweep's passes
        counter_sweep_parse(BY_NAME[args.layer if args.layer != HEADLINE else COUNTER_SWEEP_LAYER],
                            args.counter_sweep_parse)
        return
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    B.lib()  # fail loudly if the HIP library is missing
    if args.traffic_run:
        traffic_run(list(CONFIGS) if args.layer == "all" else [BY_NAME[args.layer]])
        return
    if args.table1:
        rows = table1_sweep()
        json.dump({"layers": rows, "_meta": {"kernel_sha": kernel_source_hash(),
                                             "command": "python bench.py --table1"}},
                  open(TABLE1_JSON, "w"), indent=1)
        md = table1_report(rows)
        open(TABLE1_MD, "w").write(md)
        print(md, flush=True)
        return
    if args.held_out or args.train_sweep:
        train = bool(args.train_sweep)
        res = rank_sweep(heldout_layers(seed=TRAIN_SEED if train else HELDOUT_SEED))
        res["_meta"] = {"kernel_sha": kernel_source_hash(),
                        "command": "python bench.py " + ("--train-sweep" if train else "--held-out")}
        os.makedirs(RAW_DIR, exist_ok=True)
        json.dump(res, open(TRAIN_JSON if train else HELDOUT_JSON, "w"), indent=1)
        md = heldout_report({k: v for k, v in res.items() if not k.startswith("_")}, train=train)
        open(TRAIN_MD if train else HELDOUT_MD, "w").write(md)
        print(md, flush=True)
        return
    if args.counter_sweep:
        counter_sweep(BY_NAME[args.layer if args.layer != HEADLINE else COUNTER_SWEEP_LAYER], args.counter_sweep)
        return
    if args.rank_sweep is not None:
        res = rank_sweep(list(CONFIGS) if args.layer in ("all", HEADLINE) else [BY_NAME[args.layer]],
                         n=args.rank_sweep or None)
        res["_meta"] = {"kernel_sha": kernel_source_hash(), "command": "python bench.py --rank-sweep"}
        os.makedirs(RAW_DIR, exist_ok=True)
        json.dump(res, open(RANK_JSON, "w"), indent=1)
        md = rank_report({k: v for k, v in res.items() if not k.startswith("_")})
        open(RANK_MD, "w").write(md)
        print(md, flush=True)
        return
    c = BY_NAME[args.layer]

    dtype_code = B.CONV_DTYPE_BF16 if c.dtype == "bf16" else B.CONV_DTYPE_F32
    plan = B.conv_fwd_plan(*c.key(), dtype=dtype_code)
    runner = LayerRunner(c)
    ramp_launches = runner.ramp()
    r = runner.back_to_back(args.steps, args.warmup)
    flush = flush_buffer()
    cold = summary(runner.cold_runs(flush))
    sclk = observed_sclk(runner)
    del runner
    F, Bt = flops(c), alg_bytes(c)
    ms = r["wall_ms_per_step"]
    value = F / (ms * 1e-3) / 1e9
    kern_s = r["mean_kernel_ms"] * 1e-3
    peak_tf = PEAK["bf16_mfma_tflops"] if c.dtype == "bf16" else PEAK["fp32_mfma_tflops"]
    t_mfma = F / (peak_tf * 1e12)
    t_hbm = Bt / (PEAK["hbm_gbs"] * 1e9)
    if t_mfma >= t_hbm:
        roof = {"bound": "mfma", "achieved": F / kern_s / 1e12, "peak": peak_tf, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": Bt / kern_s / 1e9, "peak": PEAK["hbm_gbs"], "unit": "GB/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = None
    if c.name == HEADLINE and os.path.exists(TRAFFIC_FILE):
        t = json.load(open(TRAFFIC_FILE))
        if t.get("kernel_sha") == plan_kernel_hash(c, plan) and t.get("plan_variant") == plan["variant"]:
            roof["traffic"] = t["hbm_bytes_per_launch"]
    roof["kernel_ms"] = r["mean_kernel_ms"]
    roof["alg_bytes"] = Bt
    roof["alg_flop"] = F
    roof["hbm_gbs_alg"] = Bt / kern_s / 1e9
    roof["hbm_frac_alg"] = roof["hbm_gbs_alg"] / PEAK["hbm_gbs"]
    out = {
        "metric": "conv_fwd GFLOP/s per layer shape + % of MI355X MFMA peak (fp32) on 1 GPU",
        "value": value, "unit": "GFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if c.dtype == "bf16" else "f32",
        "data": "synthetic (seeded uniform[-1,1), Table-1-style layer shape)",
        "config": {"workload": c.name, "N": c.N, "C": c.C, "K": c.K, "H": c.H, "W": c.W, "R": c.R,
                   "S": c.S, "layout": "NCHW/KCRS->NKPQ", "buffer_sets": r["buffer_sets"],
                   "plan": {k: plan[k] for k in ("variant", "tile_k", "tile_rows", "tile_cols", "tile_c",
                                                 "wave_k", "wave_px", "waves_k", "waves_px",
                                                 "grid_order", "num_wg")}},
        "pct_fp32_mfma_peak": 100.0 * F / kern_s / 1e12 / PEAK["fp32_mfma_tflops"],
        "roofline": roof,
        "ramp": {"seconds": RAMP_S, "launches": ramp_launches},
        "protocol": {"cold": cold, "gflops_at_mean": F / (cold["mean_us"] * 1e-6) / 1e9,
                     "pct_fp32_mfma_peak_at_mean": 100 * F / (cold["mean_us"] * 1e-6) / 1e12 / PEAK["fp32_mfma_tflops"],
                     "note": f"1 untimed + {PROTOCOL_RUNS} runs, each after a read pass over "
                             f"{FLUSH_BYTES >> 20} MB and between its own HIP events"},
        "sclk": sclk,
    }
    progress(f"headline {c.name}: {r['mean_kernel_ms'] * 1e3:.1f} us per launch back to back")
    out["empty_kernel_floor"] = empty_kernel_floor(flush)
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(c)
        out["cpu_baseline_1thread"] = cpu_baseline_one_thread(CONFIGS[0])
        progress("CPU oracle baselines done")
    if not args.no_layers:
        layers = {}
        # the bf16 layer with bf16 Out (conv_fwd_bf16_out): half the write
        # traffic; timed before the tuning below replaces any cached plan
        c5 = [lc for lc in CONFIGS if lc.dtype == "bf16"][0]
        lr5 = LayerRunner(c5, out_bf16=True)
        lr5.ramp()
        lk = lr5.back_to_back(50, 5, queued=True)["mean_kernel_ms"] * 1e-3
        cold5 = summary(lr5.cold_runs(flush))
        del lr5
        ab = alg_bytes(c5) - c5.N * c5.K * c5.P * c5.Q * 2
        bf16out_row = {
            "dtype": "bf16", "out_dtype": "bf16", "variant": B.conv_fwd_bf16_out_plan(*c5.key())["variant"],
            "split_c": 1, "kernel_us": lk * 1e6, "gflops": flops(c5) / lk / 1e9,
            "pct_fp32_mfma_peak": 100 * flops(c5) / lk / 1e12 / PEAK["fp32_mfma_tflops"],
            "pct_dtype_mfma_peak": 100 * flops(c5) / lk / 1e12 / PEAK["bf16_mfma_tflops"],
            "alg_hbm_gbs": ab / lk / 1e9, "pct_hbm_peak": 100 * ab / lk / 1e9 / PEAK["hbm_gbs"],
            "cold": cold5,
        }
        counters = layer_counters()
        for lc in CONFIGS:
            try:
                lrun = LayerRunner(lc)
            except B.ConvError as e:
                layers[lc.name] = {"error": str(e)}
                continue
            lrun.ramp()
            lr = lrun.back_to_back(50, 5, queued=True)
            lcold = summary(lrun.cold_runs(flush))
            del lrun
            lk = lr["mean_kernel_ms"] * 1e-3
            lpeak = PEAK["bf16_mfma_tflops"] if lc.dtype == "bf16" else PEAK["fp32_mfma_tflops"]
            lplan = B.conv_fwd_plan(*lc.key(), dtype=B.CONV_DTYPE_BF16 if lc.dtype == "bf16" else B.CONV_DTYPE_F32)
            layers[lc.name] = {
                "dtype": lc.dtype, "variant": lplan["variant"], "split_c": lplan["split_c"],
                "num_wg": lplan["num_wg"],
                "kernel_us": lk * 1e6, "gflops": flops(lc) / lk / 1e9,
                "pct_fp32_mfma_peak": 100 * flops(lc) / lk / 1e12 / PEAK["fp32_mfma_tflops"],
                "pct_dtype_mfma_peak": 100 * flops(lc) / lk / 1e12 / lpeak,
                "alg_hbm_gbs": alg_bytes(lc) / lk / 1e9,
                "pct_hbm_peak": 100 * alg_bytes(lc) / lk / 1e9 / PEAK["hbm_gbs"],
                "cold": lcold,
                "cold_pct_fp32_mfma_peak_at_mean": 100 * flops(lc) / (lcold["mean_us"] * 1e-6) / 1e12
                / PEAK["fp32_mfma_tflops"],
                "traffic": counters.get((lc.name, plan_kernel_hash(lc, lplan))),
            }
            if not args.no_cpu:
                layers[lc.name]["cpu_oracle"] = cpu_baseline(lc, budget_s=3.0)
            # Sec. 10 MOpt-5: the fastest of the model's top 5 plans, kept as
            # the shape's plan by conv_fwd_tune, timed the same way
            In_t, Ker_t = make_inputs(lc)
            _, tplan, _ = B.conv_fwd_tune(In_t.cuda(), Ker_t.cuda(), top_n=5, reps=5)
            del In_t, Ker_t
            tk = time_layer(lc, 50, 5, queued=True)["mean_kernel_ms"] * 1e-3
            layers[lc.name].update({"mopt5_variant": tplan["variant"], "mopt5_split_c": tplan["split_c"],
                                    "mopt5_kernel_us": tk * 1e6, "mopt5_gflops": flops(lc) / tk / 1e9,
                                    "mopt5_pct_hbm_peak": 100 * alg_bytes(lc) / tk / 1e9 / PEAK["hbm_gbs"]})
            progress(f"layer {lc.name}: {lk * 1e6:.1f} us (MOpt-5 {tk * 1e6:.1f} us)")
            torch.cuda.empty_cache()
        layers[c5.name + "_bf16out"] = bf16out_row
        # strided, padded Table 1 layers (conv_fwd_ex: the selected stride-1
        # plan of the polyphase inner problem, reading In through the phase
        # mapping where its kernel can), timed the same way
        for lc in STRIDED_CONFIGS:
            lrun = LayerRunner(lc)
            lrun.ramp()
            lk = lrun.back_to_back(50, 5, queued=True)["mean_kernel_ms"] * 1e-3
            lcold = summary(lrun.cold_runs(flush))
            del lrun
            inner = B.conv_fwd_ex_inner_shape(*lc.key(), lc.stride, lc.pad)
            lplan, ldirect = B.conv_fwd_ex_plan(*lc.key(), lc.stride, lc.pad)
            layers[lc.name] = {
                "dtype": lc.dtype, "stride": lc.stride, "pad": lc.pad, "inner_shape": list(inner[:7]),
                "variant": lplan["variant"], "split_c": lplan["split_c"], "direct": ldirect,
                "kernel_us": lk * 1e6,
                "gflops": flops(lc) / lk / 1e9,
                "pct_fp32_mfma_peak": 100 * flops(lc) / lk / 1e12 / PEAK["fp32_mfma_tflops"],
                "alg_hbm_gbs": alg_bytes(lc) / lk / 1e9,
                "pct_hbm_peak": 100 * alg_bytes(lc) / lk / 1e9 / PEAK["hbm_gbs"],
                "cold": lcold,
            }
            progress(f"layer {lc.name}: {lk * 1e6:.1f} us")
            torch.cuda.empty_cache()
        out["per_layer"] = layers
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
