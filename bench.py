"""Benchmark: images/sec of the sparse MobileNetV2 block stack at mask density
0.25, and its speedup over the same kernels run densely, on one MI355X.

Default workload: 8 stacked stride-1 gated inverted-residual blocks at
32 x 64x64x32 (hidden 192), fp16 storage, synthetic ellipse ("person")
features, every block's mask bias set so that 25% of the positions are active.

A step is one pass of the whole hot path over the batch: for each block the
mask unit, the active / halo lists, gather + expansion, depthwise + projection
+ scatter-add into the identity path.  The input stays resident in HBM and is
not modified; the stack writes a separate output buffer.  Steps run from a
captured HIP graph (--no-graph: eager).  W warm-up steps, then exactly K timed
steps between two device synchronisations.  --unfused times the multi-kernel
chain instead of the one-launch blocks.

Also reported on the same JSON line:
  dense         the same stack with every block dense (no mask, no lists)
  kernels       per-kernel average duration from the start/end events the HIP
                runtime stamps on each launch (eager, separate pass)
  roofline      the dominant kernel's algorithmic bytes per launch / its
                average duration, against the 8 TB/s HBM peak
  cpu_baseline  the CPU oracle (gather/scatter form, fp64, one thread) on a
                bounded sample of the same workload
  sweep         per-block latency of the 32 x 56x56x24 (hidden 144) fp16 block
                at densities 0.1 .. 0.9, sparse and dense
  sweep_pose_stack
                the 8-block pose stack at densities 0.1 .. 0.9 and at per-block
                densities ~ U[0.2, 0.4] (seed 1)
  sweep_parity_block_fp32
                the 1 x 32x32x32 (hidden 192) fp32 block at density 0.5
                (launch-bound)
  chain         the same stack through the kernel chain (the per-block calls'
                kernels), sparse and dense, with per-kernel HBM fractions
  shufflenet    ShuffleNetV2 stride-1 units (gated branch) at 64 x 28x28x116 and
                64 x 14x14x232, bf16, density 0.3: one unit and 3 / 7 units
  timing_protocol
                per-call median / p10 / p90 of the step, 200 calls per mode in
                alternating sparse / dense groups of 20
  cpu_baseline_parallel
                the oracle over the batch's images on all host cores (<= 16)
  mask_variants the stack with G-Softmax mask units against G-Binary ones
  network       a whole MobileNetV2 (64 x 224x224x3 -> 7x7x1280, fp16) with its 10
                stride-1 residual blocks gated, densities ~ U[0.2, 0.6], and dense
  pose_network  the pose network end to end (32 x 256x256x3 ellipse images: a
                MobileNetV2 backbone to 64x64x32, then the 8 stacked blocks; 9
                gated blocks, densities ~ U[0.2, 0.4]), and dense
  bandwidth_probes
                the chain's mask / gather+expand / depthwise+scatter kernels and
                the one-launch block at batches moving >= 512 MB per kernel,
                cache flushed before each call, against a 1 GiB copy
"""
from __future__ import annotations

import argparse
import json
import tempfile
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "images/sec of sparse MobileNetV2 block stack at mask density 0.25; speedup vs dense"
HBM_PEAK_GBS = 8000.0
# what the stack's input feature maps are (the benchmark draws them directly;
# the pose_network report runs the backbone from 256x256x3 images instead)
INPUT_RECIPES = {
    "ellipses": "64x64x32 features drawn directly: 1-2 person ellipses (15-35% of the image each, "
                "own mean + 3 texture blobs) on a flat N(0,0.3) background + N(0,0.05) noise; mask "
                "weights point from background to person mean; standing in for a MobileNetV2 backbone "
                "on 256x256x3 person crops",
    "blobs": "4 random Gaussian blobs per image + N(0,0.05) noise",
}


def traffic_file(kernel):
    return os.path.join(ROOT, "profiles", "%s_pose_stack8_traffic.md" % kernel)


KERNEL_SOURCES = ("paper_1912_03203_amd/csrc/cells.h", "paper_1912_03203_amd/csrc/fused.h",
                  "paper_1912_03203_amd/csrc/kernels.h", "paper_1912_03203_amd/csrc/dynconv.hip")
ONE_LAUNCH = ("k_block_cells", "k_block_fused")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_sha1():
    """Hash of the sources the kernels and their launch shapes are built from:
    measured HBM traffic is only reported while it matches."""
    import hashlib
    h = hashlib.sha1()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(kernel, workload, density):
    """HBM bytes per sparse one-launch block from the committed counter
    summary, or None when it is absent, for another workload, or taken on
    other kernel sources."""
    try:
        with open(traffic_file(kernel)) as f:
            text = f.read()
    except OSError:
        return None
    tag = "<!-- traffic "
    if tag not in text:
        return None
    rec = json.loads(text.split(tag, 1)[1].split(" -->", 1)[0])
    if rec.get("source_sha1") != kernel_source_sha1():
        return None
    if rec.get("workload") != workload or abs(rec.get("density", -1) - density) > 1e-9:
        return None
    return rec


# ------------------------------------------------------------------ HIP events
class HipEvents:
    """Timing events whose raw hipEvent_t handles the library records on its own
    stream.  They are torch events (so the runtime already loaded in the
    process creates them), each recorded once up front so the handle exists."""

    def __init__(self, torch, n):
        self.torch = torch
        self.events = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in self.events:
            e.record()
        torch.cuda.synchronize()
        self.ev = [e.cuda_event for e in self.events]

    def elapsed_ms(self, i, j):
        self.events[j].synchronize()
        return self.events[i].elapsed_time(self.events[j])

    def close(self):
        self.events = []
        self.ev = []


# ------------------------------------------------------------------ setup
def calibrate(dc, inputs, torch, x0_dev, blocks_np, dt, density):
    """Per-block mask bias for the target density (one value, or one per
    block), from the library's own bias-free logits of each block's input
    (offline, before timing)."""
    n, h, w, c = x0_dev.shape
    npos = n * h * w
    shape = dc.shape_of(x0_dev)
    x = x0_dev.clone()
    logits = torch.empty(npos, dtype=torch.float32, device=x.device)
    idx = dc.IndexBuffers.alloc(npos, device=x.device)
    ws_i = torch.empty(dc.indices_workspace_bytes(shape), dtype=torch.uint8, device=x.device)
    out = []
    for wts in blocks_np:
        blk = dc.BlockWeights.from_arrays(wts, dt, device=x.device)
        dc.mask(x, blk.w_mask, 0.0, logits=logits)
        torch.cuda.synchronize()
        d = density[len(out)] if isinstance(density, (list, tuple)) else density
        blk.b_mask = float(inputs.percentile_bias(logits.cpu().numpy(), d))
        m = dc.mask(x, blk.w_mask, blk.b_mask)
        dc.build_indices(m, shape, 1, idx, ws_i)
        ws = torch.empty(dc.block_workspace_bytes(shape, blk, dt), dtype=torch.uint8, device=x.device)
        dc.block_forward(x, x, blk, idx, ws)
        out.append(blk)
    torch.cuda.synchronize()
    return out


class Runner:
    """One timed step (the stack call, input -> output buffer), eager or
    graph-replayed.  The step produces y only (no mask or count outputs, as
    an inference caller runs it); read_counts() runs the same stack once more
    with the per-block counts P, P_d requested."""

    def __init__(self, dc, torch, x0, blocks, flags, use_graph, n_blocks, shuffle=False, network=False):
        self.torch = torch
        self.dc = dc
        self.x0 = x0
        self.blocks = blocks
        self.flags = flags
        self.n_blocks = n_blocks
        if network:
            self.cls = dc.Network
            out = dc.network_output_shape(dc.shape_of(x0), blocks)
            self.y = torch.empty(out.n, out.h, out.w, out.c, dtype=x0.dtype, device=x0.device)
        else:
            self.cls = dc.ShuffleStack if shuffle else dc.Stack
            self.y = torch.empty_like(x0)
        self.stack = self.cls(x0, self.y, blocks, flags=flags)
        # the count reduction is listed last but runs only when counts are requested
        names = self.stack.launch_names()
        self.names = names[:-1] if names and names[-1] == "k_band_counts" else names
        self.n_listed = len(names)
        self.counts = None
        self.graph = None
        if use_graph:
            self.graph = self._capture()

    def eager(self):
        self.stack()

    def read_counts(self):
        torch = self.torch
        if self.flags & self.dc.STACK_DENSE:
            return None
        counts = torch.zeros(self.n_blocks, 2, dtype=torch.int32, device=self.x0.device)
        y = torch.empty_like(self.y)
        self.cls(self.x0, y, self.blocks, flags=self.flags, counts=counts)()
        torch.cuda.synchronize()
        if not torch.equal(y, self.y):
            raise RuntimeError("the stack with counts requested gave another output")
        self.counts = counts
        return counts

    def _capture(self):
        torch = self.torch
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            self.eager()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.eager()
        torch.cuda.synchronize()
        return g

    def step(self):
        if self.graph is not None:
            self.graph.replay()
        else:
            self.eager()

    def timed(self, steps, warmup):
        torch = self.torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            self.step()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / steps


def profile_kernels(dc, torch, runner, steps):
    """Average duration per kernel name from start/end events that the HIP
    runtime stamps on every launch of the library (profiled stack call)."""
    names = runner.names
    ev = HipEvents(torch, 2 * runner.n_listed)
    per_launch = np.zeros(len(names))
    try:
        for _ in range(steps):
            runner.stack.profiled(ev.ev)
            torch.cuda.synchronize()
            per_launch += [ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(len(names))]
    finally:
        ev.close()
    per_launch /= steps
    out = {}
    for name, t in zip(names, per_launch):
        d = out.setdefault(name, [0.0, 0])
        d[0] += t
        d[1] += 1
    return {k: {"avg_us": 1000.0 * v[0] / v[1], "launches": v[1], "total_us": 1000.0 * v[0]}
            for k, v in out.items()}, per_launch


def algorithmic_bytes(name, dense, s, C, E, npos, rows, P, Pd, last=False, bands=0):
    """Bytes one launch must move at minimum (each input read once, each output
    written once); P, Pd are the block's active and dilated counts.  The
    one-launch block reads x and writes y at every position (its output is a
    separate buffer), reads this block's mask and writes the next one's."""
    weights = 2 * E * C * s + 9 * E * s + 4 * (2 * E + C)
    if name == "k_mask_cells":  # x everywhere in, the mask and the per-cell counts out
        return npos * C * s + npos + bands
    if name in ("k_block_fused", "k_block_cells"):
        if dense:  # x read and y written at every position
            return 2 * npos * C * s + weights
        # the fused-block ideal: the mask unit reads x everywhere, the
        # expansion gathers the dilated rows, the residual reads x and writes
        # y at the active rows; this block's mask in, the next one's out
        masks = npos + (0 if last else npos)
        return npos * C * s + Pd * C * s + 2 * P * C * s + masks + weights
    if name == "k_copy16":
        return 2 * npos * C * s
    if name == "k_band_counts":  # per-band (P, P_d) pairs in, the block's sums out
        return 8 * bands + 8
    if dense:
        if name == "k_expand":
            return npos * C * s + npos * E * s + E * C * s + 4 * E
        if name == "k_dw_project":
            return npos * E * s + 2 * npos * C * s + 9 * E * s + E * C * s + 4 * (E + C)
    table = {
        "k_mask": npos * C * s + npos + 4 * C,
        "k_rowcount": npos + 8 * rows,
        "k_rowscan": 8 * rows + 8 * (rows + 1) + 8,
        "k_compact": npos + 8 * rows + 4 * P + 4 * Pd + 36 * P,
        "k_expand": 4 * Pd + Pd * C * s + Pd * E * s + E * C * s + 4 * E,
        "k_dw_project": 40 * P + Pd * E * s + 2 * P * C * s + 9 * E * s + E * C * s + 4 * (E + C),
    }
    return table[name]


def work_counts(wl, counts, t_sp, t_dn):
    """Multiply-accumulates of one step from the device's per-block counts
    (Sec. 3.3): dense F_b = NHW (9E + 2CE) (Eq. 9) and sparse
    F_b,sp = P_d C E + P (9E + EC) (Eq. 10, N_b = P by Eq. 11), summed over
    the blocks; flop rates count two per multiply-accumulate."""
    C, E, nhw = wl.c, wl.e, wl.nhw
    dense = wl.blocks * nhw * (9 * E + 2 * C * E)
    sparse = sum(int(Pd) * C * E + int(P) * (9 * E + E * C) for P, Pd in counts)
    return {"eq9_dense_macs_per_step": int(dense), "eq10_sparse_macs_per_step": int(sparse),
            "mac_ratio_dense_over_sparse": dense / sparse if sparse else None,
            "sparse_tflops": 2.0 * sparse / t_sp / 1e12, "dense_tflops": 2.0 * dense / t_dn / 1e12,
            "P_per_block": [int(P) for P, _ in counts], "Pd_per_block": [int(Pd) for _, Pd in counts]}


def compact_record(result):
    """The benchmark's one-line result: the headline, the roofline of the
    dominant kernel, the work counts, the CPU baseline and one summary number
    per extra report (the full report goes to a file)."""
    r3 = lambda v: None if v is None else float("%.4g" % v)
    keep = ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
            "scaling", "vs_baseline", "dtype", "data", "config", "speedup_vs_dense", "dense", "roofline",
            "work", "cpu_baseline")
    out = {k: result[k] for k in keep if k in result}
    out["per_block_us"] = {k: r3(v) for k, v in result["per_block_us"].items()}
    if "cpu_baseline_parallel" in result:
        c = result["cpu_baseline_parallel"]
        out["cpu_baseline_parallel"] = {"value": r3(c["value"]), "cores": c["cores"], "kind": c["kind"]}
    if "cpu_baseline_dense" in result:
        c = result["cpu_baseline_dense"]
        out["cpu_baseline_dense"] = {"value": r3(c["value"]), "cores": c["cores"], "kind": c["kind"]}
    if "timing_protocol" in result:
        tp = result["timing_protocol"]
        out["timing_protocol"] = {"sparse_median_us": r3(tp["sparse"]["median_us"]),
                                  "dense_median_us": r3(tp["dense"]["median_us"]),
                                  "speedup_median": r3(tp["speedup_median"])}
    extra = {}
    for key in ("sweep_pose_stack", "sweep"):
        if key in result:
            extra[key] = [[r["density"] if not isinstance(r["density"], list) else "U[0.2,0.4]",
                           r3(r["sparse_us"]), r3(r["dense_us"]), r3(r["speedup"])] for r in result[key]["rows"]]
    for key in ("network", "pose_network"):
        if key in result:
            extra[key] = {"images_per_s": r3(result[key]["sparse_images_per_s"]),
                          "speedup_vs_dense": r3(result[key]["speedup_vs_dense"])}
    if "shufflenet" in result:
        extra["shufflenet_speedup"] = {r["workload"]: r3(r["speedup_vs_dense"]) for r in result["shufflenet"]}
    if "chain" in result and "speedup_vs_dense" in result["chain"]:
        extra["chain_speedup_vs_dense"] = r3(result["chain"]["speedup_vs_dense"])
    if extra:
        out["other_reports"] = extra
    return out


def cpu_baseline(inputs, wl, x0_np, blocks_np, density, budget_s=12.0, form="sparse"):
    """The oracle (mask, dilation, index maps, gather/scatter block; fp64; one
    thread) on the first S images of the batch, biases calibrated on that
    sample.  S is sized so the timed run takes about budget_s seconds.
    form="dense": the oracle's dense block with masked output (the plain
    definition, Eq. 1 with the mask of Eq. 3) after the same mask unit."""
    import oracle

    def run(x_nhwc, biases=None, timed=False):
        x = np.ascontiguousarray(x_nhwc.transpose(0, 3, 1, 2)).astype(np.float64)
        N, C, H, W = x.shape
        cal = []
        t = 0.0
        for b, wts in enumerate(blocks_np):
            if biases is None:
                _, s = oracle.mask(x.astype(np.float32), wts["w_m"], 0.0)
                bias = inputs.percentile_bias(s, density)
            else:
                bias = biases[b]
            cal.append(bias)
            t0 = time.perf_counter()
            G, _ = oracle.mask(x.astype(np.float32), wts["w_m"], bias)
            if form == "dense":
                y, _, _ = oracle.block_dense(x, wts, G)
            else:
                Gd = oracle.dilate(G, N, H, W, 1)
                A, D, nbr = oracle.indices(G, Gd, N, H, W)
                y, _, _ = oracle.block_sparse(x, wts, A, D, nbr)
            t += time.perf_counter() - t0
            y_nhwc = inputs.round_to_storage(y.transpose(0, 2, 3, 1), wl.dtype)
            x = np.ascontiguousarray(y_nhwc.transpose(0, 3, 1, 2)).astype(np.float64)
        return cal, t

    cal1, _ = run(x0_np[:1])
    _, t1 = run(x0_np[:1], cal1)
    S = int(max(1, min(wl.n, round(budget_s / max(t1, 1e-3)))))
    sample = x0_np[:S]
    cal, _ = run(sample)
    _, t = run(sample, cal)
    what = ("mask, dense block with masked output" if form == "dense"
            else "mask, dilation, index maps, gather/scatter block")
    return {"value": S / t, "unit": "images/s", "cores": 1, "kind": "oracle",
            "sample": "%d of %d images through all %d blocks (%s; fp64 C loops, one thread); %.1f s"
                      % (S, wl.n, len(blocks_np), what, t)}


def cpu_baseline_parallel(inputs, wl, x0_np, blocks_np, density, budget_s=8.0):
    """The same oracle run over the images of the batch in parallel (images
    are independent; the oracle's C loops run outside the interpreter lock),
    one thread per host core this process may use (at most 16), the batch
    repeated until the run takes about budget_s seconds.  Biases are
    calibrated on the batch first (untimed)."""
    import os
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    # one thread per core this process may use, at most 16 (the host cores
    # that a machine shares per GPU)
    affinity = len(os.sched_getaffinity(0))
    threads = max(1, min(16, affinity))
    x = np.ascontiguousarray(x0_np.transpose(0, 3, 1, 2)).astype(np.float64)
    biases = []
    cur = x
    for wts in blocks_np:
        _, sl = oracle.mask(cur.astype(np.float32), wts["w_m"], 0.0)
        b = inputs.percentile_bias(sl, density)
        biases.append(b)
        N, C, H, W = cur.shape
        G, _ = oracle.mask(cur.astype(np.float32), wts["w_m"], b)
        A, D, nbr = oracle.indices(G, oracle.dilate(G, N, H, W, 1), N, H, W)
        y, _, _ = oracle.block_sparse(cur, wts, A, D, nbr)
        cur = np.ascontiguousarray(inputs.round_to_storage(y.transpose(0, 2, 3, 1), wl.dtype).transpose(0, 3, 1, 2))

    def one(i):
        xi = x[i:i + 1]
        for b, wts in enumerate(blocks_np):
            _, _, H, W = xi.shape
            G, _ = oracle.mask(xi.astype(np.float32), wts["w_m"], biases[b])
            A, D, nbr = oracle.indices(G, oracle.dilate(G, 1, H, W, 1), 1, H, W)
            y, _, _ = oracle.block_sparse(xi, wts, A, D, nbr)
            xi = np.ascontiguousarray(inputs.round_to_storage(y.transpose(0, 2, 3, 1), wl.dtype).transpose(0, 3, 1, 2))
        return 0

    with ThreadPoolExecutor(threads) as pool:
        t0 = time.perf_counter()
        list(pool.map(one, range(x.shape[0])))
        t1 = time.perf_counter() - t0
        reps = int(max(1, round(budget_s / max(t1, 1e-3))))
        t0 = time.perf_counter()
        for _ in range(reps):
            list(pool.map(one, range(x.shape[0])))
        t = time.perf_counter() - t0
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": reps * x.shape[0] / t, "unit": "images/s", "cores": threads, "kind": "oracle",
            "cpu": model, "affinity_cores": affinity,
            "sample": "all %d images x %d repeats through all %d blocks, one image per task on %d threads; %.1f s"
                      % (x.shape[0], reps, len(blocks_np), threads, t)}


def timing_protocol(torch, sp, dn, groups=10, per=20, warm=20):
    """Per-call times of the graph-replayed step: after `warm` calls per mode,
    alternating groups of `per` sparse and `per` dense calls (groups x per
    per mode), each call between two events; median, p10, p90 in us."""
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(per)]
    for _ in range(warm):
        sp.step()
        dn.step()
    torch.cuda.synchronize()
    res = {"sparse": [], "dense": []}
    for _ in range(groups):
        for tag, r in (("sparse", sp), ("dense", dn)):
            for i in range(per):
                ev[i][0].record()
                r.step()
                ev[i][1].record()
            torch.cuda.synchronize()
            res[tag] += [1e3 * ev[i][0].elapsed_time(ev[i][1]) for i in range(per)]
    out = {"calls_per_mode": groups * per, "group": per}
    for tag, v in res.items():
        a = np.asarray(v)
        out[tag] = {"median_us": float(np.median(a)), "p10_us": float(np.percentile(a, 10)),
                    "p90_us": float(np.percentile(a, 90))}
    out["speedup_median"] = out["dense"]["median_us"] / out["sparse"]["median_us"]
    return out


def chain_report(dc, torch, wl, x0, sparse_blocks, dense_blocks, counts, use_graph, steps, warmup,
                 profile_steps):
    """The same stack through the kernel chain (mask, row counts, row scan,
    compaction, gather+expand, depthwise+project+scatter; and expand +
    depthwise-project over all positions for dense): step times and, per
    kernel, the average duration, algorithmic bytes and HBM fraction."""
    sp = Runner(dc, torch, x0, sparse_blocks, dc.STACK_UNFUSED, use_graph, wl.blocks)
    dn = Runner(dc, torch, x0, dense_blocks, dc.STACK_UNFUSED | dc.STACK_DENSE, use_graph, wl.blocks)
    t_sp = sp.timed(steps, warmup)
    t_dn = dn.timed(steps, warmup)
    c_chain = sp.read_counts().cpu().numpy()
    if not np.array_equal(c_chain, counts):
        raise RuntimeError("kernel chain and one-launch blocks disagree on the counts")
    s = 2 if wl.dtype != "f32" else 4
    rows = wl.n * wl.h
    out = {"sparse_ms_per_step": 1e3 * t_sp, "dense_ms_per_step": 1e3 * t_dn, "speedup_vs_dense": t_dn / t_sp,
           "sparse_images_per_s": wl.n / t_sp, "kernels": {}}
    for tag, runner, dense in (("sparse", sp, False), ("dense", dn, True)):
        prof, _ = profile_kernels(dc, torch, runner, profile_steps)
        for k, v in prof.items():
            if dense:
                b = float(algorithmic_bytes(k, True, s, wl.c, wl.e, wl.nhw, rows, wl.nhw, wl.nhw))
            else:
                b = float(np.mean([algorithmic_bytes(k, False, s, wl.c, wl.e, wl.nhw, rows, int(P), int(Pd))
                                   for P, Pd in counts]))
            gbs = b / (v["avg_us"] * 1e-6) / 1e9
            out["kernels"]["%s %s" % (k, tag)] = {"avg_us": v["avg_us"], "launches": v["launches"],
                                                  "algorithmic_bytes": b, "gbs": gbs,
                                                  "hbm_frac": gbs / HBM_PEAK_GBS}
    return out


def mask_variants(dc, torch, wl, x0, sparse_blocks, t_gbinary, use_graph, steps, warmup, profile_steps):
    """The stack with G-Softmax mask units (Sec. 3.1.2, Table 1's G-Softmax
    row) beside the G-Binary stack: step time, and the chain's mask-unit
    kernel in both modes."""
    gs = Runner(dc, torch, x0, sparse_blocks, dc.STACK_GSOFTMAX, use_graph, wl.blocks)
    t_gs = gs.timed(steps, warmup)
    out = {"gbinary_ms_per_step": 1e3 * t_gbinary, "gsoftmax_ms_per_step": 1e3 * t_gs,
           "gsoftmax_images_per_s": wl.n / t_gs, "gsoftmax_over_gbinary": t_gs / t_gbinary}
    for tag, flags in (("gbinary", dc.STACK_UNFUSED), ("gsoftmax", dc.STACK_UNFUSED | dc.STACK_GSOFTMAX)):
        r = Runner(dc, torch, x0, sparse_blocks, flags, False, wl.blocks)
        prof, _ = profile_kernels(dc, torch, r, profile_steps)
        out["chain_k_mask_us_" + tag] = prof["k_mask"]["avg_us"]
    return out


def density_sweep(dc, inputs, torch, steps, warmup, use_graph, flags,
                  workload="mbv2_stage2_block_56x56x24_f16", densities=None):
    """Step time of a stack at each density (one value for every block, or a
    tuple with one value per block), against the same stack dense."""
    wl = inputs.WORKLOADS[workload]
    x_np, blocks_np, _ = inputs.make_block_inputs(wl, 0)
    dt = dc.NAME_TO_DTYPE[wl.dtype]
    x0 = torch.from_numpy(x_np).cuda().to(dt)
    dense_blk = [dc.BlockWeights.from_arrays(b, dt) for b in blocks_np]
    dense_t = Runner(dc, torch, x0, dense_blk, flags | dc.STACK_DENSE, use_graph, wl.blocks).timed(steps, warmup)
    rows = []
    for d in (wl.densities if densities is None else densities):
        blks = calibrate(dc, inputs, torch, x0, blocks_np, dt, d)
        r = Runner(dc, torch, x0, blks, flags, use_graph, wl.blocks)
        t = r.timed(steps, warmup)
        counts = r.read_counts().cpu().numpy()
        rows.append({"density": list(d) if isinstance(d, tuple) else d,
                     "active_frac": [float(c[0]) / wl.nhw for c in counts],
                     "dilated_frac": [float(c[1]) / wl.nhw for c in counts],
                     "sparse_us": 1e6 * t, "dense_us": 1e6 * dense_t, "speedup": dense_t / t,
                     "sparse_images_per_s": wl.n / t, "dense_images_per_s": wl.n / dense_t})
    return {"workload": wl.name, "blocks": wl.blocks, "rows": rows}


def calibrate_shuffle(dc, inputs, torch, x0_dev, branches_np, dt, density):
    """Per-unit mask bias of a ShuffleNetV2 unit stack for the target density,
    from the library's bias-free logits of each unit's branch rows (x2
    zero-extended to the padded width), units run one after another."""
    n, h, w, c = x0_dev.shape
    cb = c // 2
    x = x0_dev.clone()
    logits = torch.empty(n * h * w, dtype=torch.float32, device=x.device)
    out = []
    for wts in branches_np:
        blk = dc.BlockWeights.from_arrays(dc.padded_branch_arrays(wts), dt, device=x.device)
        cp = blk.w_expand.shape[1]
        x2 = torch.zeros(n, h, w, cp, dtype=x.dtype, device=x.device)
        x2[..., :cb] = x[..., cb:]
        dc.mask(x2, blk.w_mask, 0.0, logits=logits)
        torch.cuda.synchronize()
        blk.b_mask = float(inputs.percentile_bias(logits.cpu().numpy(), density))
        y = torch.empty_like(x)
        dc.ShuffleStack(x, y, [blk])()
        x = y
        out.append(blk)
    torch.cuda.synchronize()
    return out


def shuffle_bytes(name, dense, s, C, cp, ep, npos, rows, P, Pd, last):
    """Algorithmic bytes of one launch of the ShuffleNetV2 unit path (C
    channels, branch rows of cp channels, hidden ep)."""
    cb = C // 2
    if name == "k_shuffle_split":
        return npos * (cb + cp) * s
    if name == "k_shuffle_merge":
        return npos * (2 * cb + C) * s + (0 if last else npos * cp * s)
    if name == "k_block_fused":  # branch rows in and out, the unit's own mask computed on chip
        return 2 * npos * cp * s + 2 * ep * cp * s + 9 * ep * s + 4 * (2 * ep + cp)
    return algorithmic_bytes(name, dense, s, cp, ep, npos, rows, P, Pd)


def shufflenet_report(dc, inputs, torch, steps, warmup, use_graph, profile_steps):
    """ShuffleNetV2 1.0x stride-1 units at 28x28x116 and 14x14x232 (batch 64,
    bf16, density 0.3): one unit (latency) and the stage repeats (3 and 7
    units, throughput), sparse against dense, with per-kernel HBM fractions."""
    rows = []
    for name in ("shufflenet_unit_28x28x116_bf16", "shufflenet_unit_14x14x232_bf16",
                 "shufflenet_stage2_3units_28x28x116_bf16", "shufflenet_stage3_7units_14x14x232_bf16"):
        wl = inputs.WORKLOADS[name]
        d = wl.densities[0]
        x_np, br_np, _ = inputs.make_block_inputs(wl, 0)
        dt = dc.NAME_TO_DTYPE[wl.dtype]
        x0 = torch.from_numpy(x_np).cuda().to(dt)
        sp_b = calibrate_shuffle(dc, inputs, torch, x0, br_np, dt, d)
        dn_b = [dc.BlockWeights.from_arrays(dc.padded_branch_arrays(w), dt) for w in br_np]
        sp = Runner(dc, torch, x0, sp_b, 0, use_graph, wl.blocks, shuffle=True)
        dn = Runner(dc, torch, x0, dn_b, dc.STACK_DENSE, use_graph, wl.blocks, shuffle=True)
        t_sp = sp.timed(steps, warmup)
        t_dn = dn.timed(steps, warmup)
        counts = sp.read_counts().cpu().numpy()
        s = 2 if wl.dtype != "f32" else 4
        cp = sp_b[0].w_expand.shape[1]
        ep = sp_b[0].w_expand.shape[0]
        kern = {}
        for tag, runner, dense in (("sparse", sp, False), ("dense", dn, True)):
            prof, per_launch = profile_kernels(dc, torch, runner, profile_steps)
            for k, v in prof.items():
                if dense:
                    b = float(np.mean([shuffle_bytes(k, True, s, wl.c, cp, ep, wl.nhw, wl.n * wl.h, wl.nhw, wl.nhw,
                                                     u == wl.blocks - 1) for u in range(wl.blocks)]))
                else:
                    b = float(np.mean([shuffle_bytes(k, False, s, wl.c, cp, ep, wl.nhw, wl.n * wl.h, int(P), int(Pd),
                                                     u == wl.blocks - 1) for u, (P, Pd) in enumerate(counts)]))
                gbs = b / (v["avg_us"] * 1e-6) / 1e9
                kern["%s %s" % (k, tag)] = {"avg_us": v["avg_us"], "launches": v["launches"],
                                            "algorithmic_bytes": b, "gbs": gbs, "hbm_frac": gbs / HBM_PEAK_GBS}
        dom = max((k for k in kern if k.endswith("sparse")),
                  key=lambda k: kern[k]["avg_us"] * kern[k]["launches"])
        rows.append({"workload": wl.name, "units": wl.blocks, "batch": wl.n, "density": d,
                     "branch_channels_padded": cp, "hidden_padded": ep,
                     "sparse_ms_per_step": 1e3 * t_sp, "dense_ms_per_step": 1e3 * t_dn,
                     "sparse_images_per_s": wl.n / t_sp, "dense_images_per_s": wl.n / t_dn,
                     "speedup_vs_dense": t_dn / t_sp, "per_unit_us": 1e6 * t_sp / wl.blocks,
                     "active_frac": (counts[:, 0] / wl.nhw).tolist(),
                     "dilated_frac": (counts[:, 1] / wl.nhw).tolist(),
                     "sparse_launches": sp.names, "kernels": kern,
                     "roofline": {"bound": "hbm", "kernel": dom, "achieved": kern[dom]["gbs"],
                                  "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": kern[dom]["hbm_frac"]}})
    return rows


def calibrate_network(dc, inputs, torch, x0, layers, dens, dt, labels=None):
    """Mask bias of every gated block of a whole network for its target
    density, from the library's bias-free logits of the block's input, the
    layers run one after another (offline, before timing).  With person
    labels (the pose network), each gated block's mask weights are first set
    to point from the background to the people in its own input features
    (inputs.person_mask_weights)."""
    cur = x0
    biases = []
    gi = 0
    rng = np.random.default_rng(11)
    for L in layers:
        if L.get("gated") and labels is not None:
            L["w_m"] = inputs.person_mask_weights(rng, cur.float().cpu().numpy(), labels)
        one = dc.NetworkWeights([L], dt, biases=[0.0] if L.get("gated") else None)
        if L.get("gated"):
            n, h, w, c = cur.shape
            logits = torch.empty(n * h * w, dtype=torch.float32, device=cur.device)
            w_m = torch.from_numpy(np.asarray(L["w_m"], np.float32)).to(cur.device)
            dc.mask(cur, w_m, 0.0, logits=logits)
            torch.cuda.synchronize()
            b = float(inputs.percentile_bias(logits.cpu().numpy(), dens[gi]))
            biases.append(b)
            one.set_bias(0, b)
            gi += 1
        out = dc.network_output_shape(dc.shape_of(cur), one)
        nxt = torch.empty(out.n, out.h, out.w, out.c, dtype=cur.dtype, device=cur.device)
        dc.Network(cur, nxt, one)()
        cur = nxt
    torch.cuda.synchronize()
    return biases


def network_report(dc, inputs, torch, steps, warmup, use_graph, profile_steps, kind="mobilenetv2"):
    """A whole network against the same network run dense.  "mobilenetv2":
    the MobileNetV2 feature extractor (batch 64, 224x224x3 -> 7x7x1280, fp16),
    17 blocks, the 10 stride-1 residual blocks gated with densities
    ~ U[0.2, 0.6].  "pose": the pose network (batch 32, 256x256x3 ellipse
    images -> 64x64x32, fp16): a MobileNetV2 backbone, then 8 stacked
    stride-1 blocks; 9 gated blocks with densities ~ U[0.2, 0.4], their mask
    units pointed at the people (set during calibration)."""
    labels = None
    if kind == "pose":
        n, h, w = 32, 256, 256
        x_np, layers, dens, labels = inputs.make_pose_network_inputs(0, n, dtype="f16")
        name = "pose_network_256_b32_f16"
    else:
        n, h, w = 64, 224, 224
        x_np, layers, dens = inputs.make_network_inputs(0, n, h, w, dtype="f16")
        name = "mobilenetv2_224_b64_f16"
    dt = torch.float16
    x0 = torch.from_numpy(x_np).cuda().to(dt)
    biases = calibrate_network(dc, inputs, torch, x0, layers, dens, dt, labels)
    sp_net = dc.NetworkWeights(layers, dt, biases=biases)
    dn_net = dc.NetworkWeights(layers, dt, biases=None)
    ng = sp_net.ngated
    sp = Runner(dc, torch, x0, sp_net, 0, use_graph, ng, network=True)
    dn = Runner(dc, torch, x0, dn_net, dc.STACK_DENSE, use_graph, ng, network=True)
    t_sp = sp.timed(steps, warmup)
    t_dn = dn.timed(steps, warmup)
    counts = sp.read_counts().cpu().numpy()
    npos = []
    sh = dc.shape_of(x0)
    for L in layers:
        one = dc.NetworkWeights([L], dt, biases=[0.0] if L.get("gated") else None)
        if L.get("gated"):
            npos.append(sh.n * sh.h * sh.w)
        sh = dc.network_output_shape(sh, one)
    prof_sp, _ = profile_kernels(dc, torch, sp, profile_steps)
    prof_dn, _ = profile_kernels(dc, torch, dn, profile_steps)

    def top(prof):
        return {k: {"avg_us": v["avg_us"], "launches": v["launches"], "total_us": v["total_us"]}
                for k, v in sorted(prof.items(), key=lambda kv: -kv[1]["total_us"])}
    return {"workload": name, "batch": n, "input": [h, w, 3], "output": [sh.h, sh.w, sh.c],
            "gated_blocks": ng, "target_density": dens.tolist(),
            "active_frac": [float(c[0]) / p for c, p in zip(counts, npos)],
            "dilated_frac": [float(c[1]) / p for c, p in zip(counts, npos)],
            "sparse_ms_per_step": 1e3 * t_sp, "dense_ms_per_step": 1e3 * t_dn,
            "sparse_images_per_s": n / t_sp, "dense_images_per_s": n / t_dn, "speedup_vs_dense": t_dn / t_sp,
            "kernels_sparse": top(prof_sp), "kernels_dense": top(prof_dn)}


def bandwidth_probes(dc, inputs, torch, reps=5):
    """HBM-scale timing of the bandwidth-bound kernels.  At the benchmark
    shapes a kernel moves 10-70 MB, which the 256 MB Infinity Cache holds; here
    the batch is scaled until each probed kernel moves at least 512 MB, and a
    512 MB scratch buffer is rewritten before every call so that its data
    comes from HBM.  Reference: a 1 GiB device-to-device copy (2 GiB moved)."""
    out = {}
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")

    def flush():
        scratch.fill_(1)

    # copy bandwidth
    a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ts = []
    for _ in range(reps):
        flush()
        e0.record()
        b.copy_(a)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e-3)
    copy_gbs = 2 * a.numel() / min(ts) / 1e9
    out["copy"] = {"bytes": 2 * a.numel(), "best_us": 1e6 * min(ts), "gbs": copy_gbs,
                   "hbm_frac": copy_gbs / HBM_PEAK_GBS}
    del a, b

    def probe(tag, wl, rep, flags, density, kernels):
        x_np, blocks_np, _ = inputs.make_block_inputs(wl, 0)
        dt = dc.NAME_TO_DTYPE[wl.dtype]
        base = torch.from_numpy(x_np).cuda().to(dt)
        blk = calibrate(dc, inputs, torch, base, blocks_np[:1], dt, density)[0] if density else \
            dc.BlockWeights.from_arrays(blocks_np[0], dt)
        x = base.repeat(rep, 1, 1, 1).contiguous()
        y = torch.empty_like(x)
        counts = torch.zeros(1, 2, dtype=torch.int32, device="cuda")
        st = dc.Stack(x, y, [blk], flags=flags, counts=None if flags & dc.STACK_DENSE else counts)
        names = st.launch_names()
        ev = HipEvents(torch, 2 * len(names))
        best = {}
        try:
            for _ in range(reps):
                flush()
                st.profiled(ev.ev)
                torch.cuda.synchronize()
                for i, n in enumerate(names):
                    if n in kernels:
                        t = ev.elapsed_ms(2 * i, 2 * i + 1) * 1e-3
                        best[n] = min(best.get(n, t), t)
        finally:
            ev.close()
        npos = x.shape[0] * x.shape[1] * x.shape[2]
        rows = x.shape[0] * x.shape[1]
        s = 2 if wl.dtype != "f32" else 4
        dense = bool(flags & dc.STACK_DENSE)
        P, Pd = (npos, npos) if dense else (int(v) for v in counts[0].cpu())
        for n, t in best.items():
            nb = algorithmic_bytes(n, dense, s, wl.c, wl.e, npos, rows, P, Pd, last=True)
            if n == "k_block_fused" and not dense:
                nb -= npos  # the patch kernel's one-block stack computes its own mask: no mask read
            out["%s %s" % (n, tag)] = {"batch": x.shape[0], "density": None if dense else P / npos,
                                       "dilated": None if dense else Pd / npos, "bytes": nb,
                                       "best_us": 1e6 * t, "gbs": nb / t / 1e9,
                                       "hbm_frac": nb / t / 1e9 / HBM_PEAK_GBS,
                                       "copy_frac": nb / t / 1e9 / copy_gbs}
        del x, y

    stage2 = inputs.WORKLOADS["mbv2_stage2_block_56x56x24_f16"]
    pose = inputs.WORKLOADS["pose_stack8_64x64x32_f16"]
    chain = ("k_mask", "k_expand", "k_dw_project")
    probe("dense, 2048 x 56x56x24", stage2, 64, dc.STACK_UNFUSED | dc.STACK_DENSE, None, chain)
    probe("sparse d=0.25, 2048 x 56x56x24", stage2, 64, dc.STACK_UNFUSED, 0.25, chain)
    probe("dense, 1024 x 64x64x32", pose, 32, dc.STACK_DENSE, None, ONE_LAUNCH)
    probe("sparse d=0.25, 1024 x 64x64x32", pose, 32, 0, 0.25, ONE_LAUNCH + ("k_mask_cells",))
    del scratch
    torch.cuda.empty_cache()
    return out


def traffic_pass(dc, torch, wl, x0, sparse_blocks, dense_blocks, reps=3):
    """Launch sequence for one HBM-counter run (FETCH_SIZE or WRITE_SIZE):
    (1) the kernel chain's plain copy (k_copy16, input -> output buffer, a
    known number of bytes each way) as the counter's calibration, (2) the
    sparse stack, (3) the dense stack; eager, synchronised after each."""
    y = torch.empty_like(x0)
    chain = dc.Stack(x0, y, sparse_blocks[:1], flags=dc.STACK_UNFUSED)
    assert chain.launch_names()[0] == "k_copy16"
    sp = Runner(dc, torch, x0, sparse_blocks, 0, False, wl.blocks)
    dn = Runner(dc, torch, x0, dense_blocks, dc.STACK_DENSE, False, wl.blocks)
    for run in (chain, sp.eager, dn.eager):
        for _ in range(reps):
            run()
            torch.cuda.synchronize()
    s = 2 if wl.dtype != "f32" else 4
    print(json.dumps({"workload": wl.name, "copy_bytes": wl.nhw * wl.c * s, "reps": reps,
                      "blocks": wl.blocks, "counts": sp.read_counts().cpu().numpy().tolist(),
                      "source_sha1": kernel_source_sha1()}), flush=True)


def _counter_rows(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def summarize_traffic(args):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE (KiB) of the copy, the sparse and
    the dense one-launch block, each counter scaled by what it reads for the
    copy of known size; written as the committed traffic summary."""
    fetch_csv, write_csv = args.summarize_traffic
    from paper_1912_03203_amd import inputs
    wl = inputs.WORKLOADS[args.workload]
    s = 2 if wl.dtype != "f32" else 4
    copy_bytes = wl.nhw * wl.c * s
    kern = args.traffic_kernel
    out = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        groups = {"copy": [], "sparse": [], "dense": []}
        for row in _counter_rows(path):
            if row["Counter_Name"] != counter:
                continue
            name = row["Kernel_Name"]
            v = float(row["Counter_Value"])
            if "k_copy16" in name:
                groups["copy"].append(v)
            elif kern in name:
                # template argument DENSE: mangled "...<kernel>I<type>Lb1E..."
                # or demangled "<kernel><type, true, ...>"
                if "<" in name:
                    dense = name.split("<", 1)[1].split(",")[1].strip() == "true"
                else:
                    dense = "Lb1E" in name.split(kern, 1)[1][:12]
                groups["dense" if dense else "sparse"].append(v)
        if not all(groups.values()):
            raise SystemExit("%s: missing dispatches in %s" % (counter, path))
        out[counter] = {k: (float(np.mean(v)), len(v)) for k, v in groups.items()}
    f_fetch = copy_bytes / (1024.0 * out["FETCH_SIZE"]["copy"][0])
    f_write = copy_bytes / (1024.0 * out["WRITE_SIZE"]["copy"][0])
    kib = {k: (out["FETCH_SIZE"][k][0], out["WRITE_SIZE"][k][0]) for k in ("copy", "sparse", "dense")}
    by = {k: 1024.0 * (kib[k][0] * f_fetch + kib[k][1] * f_write) for k in ("sparse", "dense")}
    rec = {"kernel": kern, "workload": wl.name, "density": args.density,
           "source_sha1": kernel_source_sha1(), "sparse_bytes": by["sparse"], "dense_bytes": by["dense"],
           "fetch_scale": f_fetch, "write_scale": f_write}
    lines = [
        "# HBM traffic of %s: 8-block pose stack, 32 x 64x64x32, hidden 192, fp16, density %.2f"
        % (kern, args.density),
        "",
        "Two counter runs of the same launch sequence (`bench.py --traffic-pass`: a plain copy of "
        "%d bytes each way, the sparse stack, the dense stack, 3 times each). Each counter is scaled "
        "by the ratio of the copy's known size to what the counter reads for it." % copy_bytes,
        "",
        "Commands ($REPO: the repository root; $OUT: any output directory):",
        "",
        "```",
        "cd /tmp && export TMPDIR=/tmp && timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE --output-format csv "
        "-d $OUT/traffic_fetch -o run -- python3 $REPO/bench.py --traffic-pass",
        "cd /tmp && export TMPDIR=/tmp && timeout -s KILL 120 rocprofv3 --pmc WRITE_SIZE --output-format csv "
        "-d $OUT/traffic_write -o run -- python3 $REPO/bench.py --traffic-pass",
        "python3 $REPO/bench.py --summarize-traffic $OUT/traffic_fetch/run_counter_collection.csv "
        "$OUT/traffic_write/run_counter_collection.csv",
        "```",
        "",
        "| dispatches | n | FETCH_SIZE KiB | WRITE_SIZE KiB | scaled bytes |",
        "|---|---:|---:|---:|---:|",
        "| k_copy16 (calibration) | %d | %.1f | %.1f | %d read + %d written |"
        % (out["FETCH_SIZE"]["copy"][1], kib["copy"][0], kib["copy"][1], copy_bytes, copy_bytes),
        "| %s sparse | %d | %.1f | %.1f | %.0f |"
        % (kern, out["FETCH_SIZE"]["sparse"][1], kib["sparse"][0], kib["sparse"][1], by["sparse"]),
        "| %s dense | %d | %.1f | %.1f | %.0f |"
        % (kern, out["FETCH_SIZE"]["dense"][1], kib["dense"][0], kib["dense"][1], by["dense"]),
        "",
        "Scale factors: FETCH_SIZE x %.4f, WRITE_SIZE x %.4f." % (f_fetch, f_write),
        "",
        "<!-- traffic %s -->" % json.dumps(rec),
        "",
    ]
    with open(traffic_file(kern), "w") as f:
        f.write("\n".join(lines))
    print(json.dumps(rec))


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="pose_stack8_64x64x32_f16")
    ap.add_argument("--density", type=float, default=0.25)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--unfused", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-chain", action="store_true", help="skip the kernel-chain report")
    ap.add_argument("--no-shufflenet", action="store_true", help="skip the ShuffleNetV2 unit report")
    ap.add_argument("--no-probes", action="store_true", help="skip the HBM-scale bandwidth probes")
    ap.add_argument("--no-network", action="store_true", help="skip the whole-MobileNetV2 report")
    ap.add_argument("--profile-steps", type=int, default=20)
    ap.add_argument("--report", help="where the full JSON report goes "
                                     "(default: bench_report.json in the system's temporary directory); stdout "
                                     "gets the compact line")
    ap.add_argument("--traffic-pass", action="store_true",
                    help="untimed launches for an HBM-counter run: a plain copy of known size, "
                         "then the sparse and the dense stack")
    ap.add_argument("--traffic-kernel", default="k_block_cells",
                    help="the one-launch kernel whose dispatches --summarize-traffic reads")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the traffic summary from the counter CSVs of two --traffic-pass runs")
    ap.add_argument("--section", choices=("network", "pose_network", "shufflenet", "probes"),
                    help="run only this report (for a kernel trace of it) and print its JSON object")
    args = ap.parse_args()
    if args.summarize_traffic:
        summarize_traffic(args)
        return

    if args.gpus != 1:
        print("bench.py measures one GPU: the gated-block path runs on a single MI355X "
              "(batch sharding across GPUs needs no exchange and is not launched here); "
              "use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_1912_03203_amd import dynconv as dc
    from paper_1912_03203_amd import inputs

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    dc.load()
    if args.section:
        g = not args.no_graph
        if args.section == "shufflenet":
            out = shufflenet_report(dc, inputs, torch, args.steps, args.warmup, g, args.profile_steps)
        elif args.section == "probes":
            out = bandwidth_probes(dc, inputs, torch)
        else:
            kind = "pose" if args.section == "pose_network" else "mobilenetv2"
            out = network_report(dc, inputs, torch, args.steps, args.warmup, g, args.profile_steps, kind)
        print(json.dumps({args.section: out}))
        return
    wl = inputs.WORKLOADS[args.workload]
    dt = dc.NAME_TO_DTYPE[wl.dtype]
    use_graph = not args.no_graph
    log("workload %s density %.2f steps %d warmup %d graph %s" % (wl.name, args.density, args.steps,
                                                                 args.warmup, use_graph))
    x_np, blocks_np, _ = inputs.make_block_inputs(wl, args.seed)
    x0 = torch.from_numpy(x_np).cuda().to(dt)
    sparse_blocks = calibrate(dc, inputs, torch, x0, blocks_np, dt, args.density)
    dense_blocks = [dc.BlockWeights.from_arrays(w, dt) for w in blocks_np]
    if args.traffic_pass:
        traffic_pass(dc, torch, wl, x0, sparse_blocks, dense_blocks)
        return

    base_flags = dc.STACK_UNFUSED if args.unfused else 0
    sp = Runner(dc, torch, x0, sparse_blocks, base_flags, use_graph, wl.blocks)
    dn = Runner(dc, torch, x0, dense_blocks, base_flags | dc.STACK_DENSE, use_graph, wl.blocks)
    if use_graph:  # replays must reproduce the eager step bit for bit
        for r in (sp, dn):
            r.eager()
            torch.cuda.synchronize()
            ref = r.y.clone()
            for _ in range(3):
                r.y.zero_()
                r.step()
                torch.cuda.synchronize()
                if not torch.equal(r.y, ref):
                    raise RuntimeError("graph replay differs from the eager step")
    log("timing sparse (%s)" % " ".join(sorted(set(sp.names))))
    t_sp = sp.timed(args.steps, args.warmup)
    log("timing dense")
    t_dn = dn.timed(args.steps, args.warmup)
    counts = sp.read_counts().cpu().numpy()
    npos = wl.nhw
    active = (counts[:, 0] / npos).tolist()
    dilated = (counts[:, 1] / npos).tolist()
    log("sparse %.1f us/step, dense %.1f us/step, speedup %.2fx" % (1e6 * t_sp, 1e6 * t_dn, t_dn / t_sp))

    # per-kernel profile (runtime-stamped events on each launch)
    prof_sp, _ = profile_kernels(dc, torch, sp, args.profile_steps)
    prof_dn, _ = profile_kernels(dc, torch, dn, args.profile_steps)
    s = 2 if wl.dtype != "f32" else 4
    rows = wl.n * wl.h
    if "k_block_cells" in sp.names:
        # cells of 2 x 8 positions
        bands = wl.n * -(-wl.h // 2) * -(-wl.w // 8)
    else:
        # patches of the one-launch block: column strips of at most 32, R rows,
        # at most `own` positions and `region` ring-included slots
        own, region = (256, 340) if wl.c <= 32 else (128, 208) if wl.c <= 64 else (64, 108)
        strips = -(-wl.w // 32)
        wu = -(-wl.w // strips)
        pr = max(1, min(own // wu, region // (wu + 2) - 2, 50, wl.h))
        bands = wl.n * -(-wl.h // pr) * -(-wl.w // wu)

    def avg_bytes(name, dense):
        if dense:
            return float(algorithmic_bytes(name, True, s, wl.c, wl.e, npos, rows, npos, npos))
        per = [algorithmic_bytes(name, False, s, wl.c, wl.e, npos, rows, int(P), int(Pd),
                                 last=(b == wl.blocks - 1), bands=bands)
               for b, (P, Pd) in enumerate(counts)]
        return float(np.mean(per))

    for prof, dense in ((prof_sp, False), (prof_dn, True)):
        for k, v in prof.items():
            v["algorithmic_bytes"] = avg_bytes(k, dense)
            v["gbs"] = v["algorithmic_bytes"] / (v["avg_us"] * 1e-6) / 1e9
    dom = max(prof_sp, key=lambda k: prof_sp[k]["total_us"])
    bytes_per_launch = prof_sp[dom]["algorithmic_bytes"]
    achieved = prof_sp[dom]["gbs"]
    kernel_sum_us = float(sum(v["total_us"] for v in prof_sp.values()))

    result = {
        "metric": METRIC,
        "value": wl.n / t_sp,
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * t_sp,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "input_recipe": INPUT_RECIPES[wl.features],
                   "batch": wl.n, "h": wl.h, "w": wl.w, "c": wl.c,
                   "hidden": wl.e, "blocks": wl.blocks, "density": args.density,
                   "graph": use_graph, "seed": args.seed,
                   "execution": "kernel chain" if args.unfused else "one launch per block"},
        "speedup_vs_dense": t_dn / t_sp,
        "dense": {"value": wl.n / t_dn, "ms_per_step": 1e3 * t_dn},
        "per_block_us": {"sparse": 1e6 * t_sp / wl.blocks, "dense": 1e6 * t_dn / wl.blocks},
        "active_frac": active,
        "dilated_frac": dilated,
        "kernels": {"sparse": prof_sp, "dense": prof_dn, "sparse_kernel_sum_us": kernel_sum_us},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "algorithmic_bytes_per_launch": bytes_per_launch,
                     "avg_us_per_launch": prof_sp[dom]["avg_us"]},
        "work": work_counts(wl, counts, t_sp, t_dn),
    }
    rec = measured_traffic(dom, wl.name, args.density) if dom in ONE_LAUNCH else None
    if rec is not None:
        result["roofline"]["traffic"] = rec["sparse_bytes"]
        result["roofline"]["traffic_dense"] = rec["dense_bytes"]
    log("timing protocol")
    result["timing_protocol"] = timing_protocol(torch, sp, dn)
    if not args.no_chain and not args.unfused:
        log("kernel chain")
        result["chain"] = chain_report(dc, torch, wl, x0, sparse_blocks, dense_blocks, counts, use_graph,
                                       min(args.steps, 50), min(args.warmup, 5), args.profile_steps)
    if not args.unfused:
        log("mask variants")
        result["mask_variants"] = mask_variants(dc, torch, wl, x0, sparse_blocks, t_sp, use_graph,
                                                min(args.steps, 100), min(args.warmup, 10), args.profile_steps)
    if not args.no_network:
        log("whole network")
        result["network"] = network_report(dc, inputs, torch, min(args.steps, 30), min(args.warmup, 5), use_graph,
                                           min(args.profile_steps, 5))
        log("pose network")
        result["pose_network"] = network_report(dc, inputs, torch, min(args.steps, 30), min(args.warmup, 5),
                                                use_graph, min(args.profile_steps, 5), "pose")
    if not args.no_probes:
        log("bandwidth probes")
        result["bandwidth_probes"] = bandwidth_probes(dc, inputs, torch)
    if not args.no_shufflenet:
        log("shufflenet units")
        result["shufflenet"] = shufflenet_report(dc, inputs, torch, min(args.steps, 100), min(args.warmup, 10),
                                                 use_graph, args.profile_steps)
    if not args.no_sweep:
        log("density sweep")
        sw_steps, sw_warm = min(args.steps, 100), min(args.warmup, 10)
        result["sweep"] = density_sweep(dc, inputs, torch, sw_steps, sw_warm, use_graph, base_flags)
        pose_d = (0.1, 0.25, 0.5, 0.75, 0.9)
        mixed = tuple(float(v) for v in np.random.default_rng(1).uniform(0.2, 0.4, size=wl.blocks))
        result["sweep_pose_stack"] = density_sweep(dc, inputs, torch, sw_steps, sw_warm, use_graph, base_flags,
                                                   "pose_stack8_64x64x32_f16", pose_d + (mixed,))
        result["sweep_parity_block_fp32"] = density_sweep(dc, inputs, torch, sw_steps, sw_warm, use_graph,
                                                          base_flags, "mbv2_block_32x32x32_f32")
    if not args.no_cpu:
        log("cpu baseline (oracle)")
        result["cpu_baseline"] = cpu_baseline(inputs, wl, x_np, blocks_np, args.density)
        log("cpu baseline (oracle, all host cores)")
        result["cpu_baseline_parallel"] = cpu_baseline_parallel(inputs, wl, x_np, blocks_np, args.density)
        log("cpu baseline (dense oracle)")
        result["cpu_baseline_dense"] = cpu_baseline(inputs, wl, x_np, blocks_np, args.density, budget_s=8.0,
                                                    form="dense")
    report = args.report or os.path.join(tempfile.gettempdir(), "bench_report.json")
    os.makedirs(os.path.dirname(os.path.abspath(report)), exist_ok=True)
    with open(report, "w") as f:
        json.dump(result, f, indent=1)
    log("full report: %s" % report)
    print(json.dumps(compact_record(result)), flush=True)


if __name__ == "__main__":
    main()
