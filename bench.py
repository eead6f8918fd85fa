#!/usr/bin/env python3
"""Benchmark: fused Λ24(12) dequantize + GEMV at batch 1 on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config c2_4096x4096]

A step is one GEMV y = W x of the workload matrix in the served layout
(Planes14, 4.80 b/w records + fp16 per-block scales), with W and x resident in
HBM.  The timed region is exactly K steps, bracketed by a device
synchronisation on both sides and timed with HIP events on the launch stream
(created without the system-scope fence, which timing does not need).
The matrix is held in n replicas (same codes, distinct buffers, ≥ 1 GiB in
all); step j reads replica j mod n.  Right before the timed steps, replays
of the replicas the timed region does not read (or, when K leaves fewer than
512 MiB of them, of every replica) stream ≥ 512 MiB, twice the 256 MB
Infinity Cache, so no replica the timed region reads can still be cached: its
bytes come from HBM.  The timed steps are enqueued behind those replays
without waiting for them, and the replays last at least twice (three times
for single launches) as many launches as the timed region, so the host has
submitted the timed launches before the device reaches them (checked, and
reported): K launches one by one when the host has enqueued them all in
time, else one graph of K launches; the interval then holds the K kernels
back to back.  The line
states the timed bytes, the working set and the fewest bytes streamed between
a replica's previous read and its timed read, both launch forms' times, and
the same GEMV timed over one whole ≥ 1 GiB cycle of replicas beside it.

Printed: one JSON line with the metric (served-weight GB/s of the Planes14
GEMV), µs per GEMV, the roofline against MI355X's 8 TB/s, every arm of the
layout comparison (four layouts, FP16 GEMV control, no-weights control;
interleaved, 7 rounds, first 2 discarded, medians), the prologue-mode and
phase breakdowns, the decoder-layer, batch, large-matrix and launch-floor
sections, and the CPU oracle timed on a bounded sample of the same workload.
"""
import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published peak
REPLICA_BYTES = 1 << 30        # working set per arm: 4× the 256 MB Infinity Cache
EVICT_BYTES = 512 << 20        # streamed right before a timed replay: 2× that cache
# rotated arms that mix the two forms: the activation is rotated inside the
# GEMV's prologue up to this K, this many workgroups and from this many units
# per wave (each workgroup redoes the whole transform, which pays while K is
# small, the workgroups few, and each wave's stream long enough to hide it
# behind the record loads in flight), by the separate rotation kernel
# otherwise (bench layer_8b.rotation_sites measures both forms at every site)
ROT_IN_KERNEL_MAX_K = 5120
ROT_IN_KERNEL_MAX_TILES = 512
ROT_IN_KERNEL_MIN_UNITS = 16


def rotate_in_kernel(m, K):
    d = m.desc
    tiles = -(-d.M // d.tile_rows)
    groups = -(-d.nb // d.lane_cols)
    units = -(-groups // min(8, groups))
    return (K <= ROT_IN_KERNEL_MAX_K and tiles <= ROT_IN_KERNEL_MAX_TILES
            and units >= ROT_IN_KERNEL_MIN_UNITS)
ARMS = ["planes14", "slot32", "planes12x", "planes12x_inline", "golay70", "golay70_inline",
        "fp16", "noweights"]
CONFIGS = {"c1_768x1536": (768, 1536), "c2_4096x4096": (4096, 4096),
           "c4_8192x8192": (8192, 8192)}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[1])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--config", default="c2_4096x4096", choices=sorted(CONFIGS))
    ap.add_argument("--arms", default=",".join(ARMS))
    ap.add_argument("--rounds", type=int, default=7)
    ap.add_argument("--discard", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-layer", action="store_true",
                    help="skip the 8B-layer comparison (separate vs fused launches vs FP16)")
    ap.add_argument("--layer-steps", type=int, default=300)
    ap.add_argument("--no-batch", action="store_true",
                    help="skip the batched GEMV sweep (B = 1, 2, 4, 8, 16)")
    ap.add_argument("--no-step14b", action="store_true",
                    help="skip the 14B-class decode step (40 layers + fp16 head, Leech vs FP16)")
    ap.add_argument("--step14b-layers", type=int, default=40)
    ap.add_argument("--batch-14b", action="store_true",
                    help="also time batched launches at the 14B-class fused projection shapes")
    ap.add_argument("--sweep", action="store_true",
                    help="also time square Planes14 GEMVs from 1024x1024 to 16384x16384")
    ap.add_argument("--no-large", action="store_true",
                    help="skip the large single GEMVs (16384x16384, 32768x16384, 152064x5120)")
    ap.add_argument("--no-floor", action="store_true",
                    help="skip the launch-floor probe (one-element fill, one-block GEMV)")
    ap.add_argument("--floor-steps", type=int, default=2000)
    ap.add_argument("--no-arms-c4", action="store_true",
                    help="skip the 8192x8192 layout sweep (four layouts, both exception "
                         "decoders, FP16 and no-weights controls)")
    ap.add_argument("--geometry-sweep", action="store_true",
                    help="only time the candidate tile geometries of the decoder projection "
                         "shapes (Planes14) and print them as one JSON line")
    ap.add_argument("--geometry-all", action="store_true",
                    help="with --geometry-sweep: time a broad set of geometries (every lane_cols, "
                         "tile heights in steps of 4 or 8) on the decoder shapes and 14 more")
    ap.add_argument("--calib-mib", type=int, default=0,
                    help="first run a plain device-to-device copy of this many MiB, 5 times: "
                         "the known-size reference that scales the HBM byte counters")
    return ap.parse_args()


class Arm:
    """One arm: a list of replica launchers, each enqueueing one GEMV."""

    def __init__(self, name, launchers, served_bytes, desc=None, mats=None):
        self.name, self.launchers, self.served_bytes, self.desc = name, launchers, served_bytes, desc
        self.mats = mats
        self._graphs = {}

    def run(self, k, start=0):
        n = len(self.launchers)
        for s in range(start, start + k):
            self.launchers[s % n]()

    def graph(self, torch, k, start=0):
        """A HIP graph of k consecutive GEMVs over replicas start, start + 1, …
        (mod n), captured once: replaying it enqueues the k kernels without k
        host round trips."""
        key = (k, start)
        if key not in self._graphs:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                self.run(k, start)
            self._graphs[key] = g
        return self._graphs[key]

    def evict_plan(self, k):
        """The replay that precedes a timed replay of k GEMVs from replica 0:
        (start, length) of the replicas it reads, and the fewest bytes streamed
        between a timed replica's previous read and its timed read.  It reads
        only the replicas the timed region does not read when those hold
        ≥ EVICT_BYTES, else one whole cycle from replica 0."""
        n, b = len(self.launchers), max(self.served_bytes, 1)
        if (n - k) * b >= EVICT_BYTES:
            return k, n - k, (n - k) * b
        return 0, n, (n - 1) * b


def build_arms(args, torch, P, synth, config=None):
    M, K = CONFIGS[config or args.config]
    dev = torch.device("cuda:0")
    t0 = time.time()
    inp = synth.make_gemv_inputs(M, K, seed=args.seed, name=config or args.config)
    cb = P.Codebook(12)
    dcb = P.DeviceCodebook(cb, dev)
    cls, sm, lv = cb.fields_from_points(inp.z)
    log(f"[bench] inputs {M}x{K} (Kpad {inp.Kpad}) ready in {time.time() - t0:.1f}s")
    x = torch.from_numpy(inp.x).to(dev)
    y = torch.empty(M, dtype=torch.float32, device=dev)
    arms = {}
    wanted = args.arms.split(",")
    base_desc = None
    mat14 = None
    for name in ("planes14", "slot32", "planes12x", "golay70"):
        if name not in wanted and f"{name}_inline" not in wanted and name != "planes14":
            continue
        mat = P.LeechMatrix.from_fields(dcb, P.LAYOUTS[name], cls, inp.gain, sm, lv, inp.scale, dev)
        served = mat.desc.served_bytes
        reps = max(1, math.ceil(REPLICA_BYTES / served))
        mats = [mat] + [P.LeechMatrix(mat.desc, mat.main.clone(), mat.side0.clone(),
                                      mat.side1.clone(), mat.scale.clone(), dcb)
                        for _ in range(reps - 1)]
        arms[name] = Arm(name, [(lambda m=m: m.gemv(x, y)) for m in mats], served, mat.desc, mats)
        if name == "planes14":
            base_desc, mat14 = mat.desc, mat
        if name in ("planes12x", "golay70") and f"{name}_inline" in wanted:
            # the plain decoder: exceptions decoded in the loop (the mode is
            # read when a launch is enqueued, so graphs keep it)
            def inline(m):
                P.set_exception_mode(P.EXC_INLINE)
                try:
                    m.gemv(x, y)
                finally:
                    P.set_exception_mode(P.EXC_HOISTED)
            arms[f"{name}_inline"] = Arm(f"{name}_inline", [(lambda m=m: inline(m)) for m in mats],
                                         served, mat.desc)
        log(f"[bench] {name}: {served} served bytes/GEMV, {reps} replicas")
    if "fp16" in wanted:
        # FP16 control on the same weights, decoded on the device
        z, _, _ = mat14.decode()
        zf = z.float()
        fac = torch.from_numpy(inp.scale.astype("float32")).to(dev) / zf.pow(2).sum(-1).sqrt()
        W = (zf * fac[..., None]).reshape(M, inp.Kpad).half().contiguous()
        del z, zf
        served = W.numel() * 2
        reps = max(1, math.ceil(REPLICA_BYTES / served))
        Ws = [W] + [W.clone() for _ in range(reps - 1)]
        arms["fp16"] = Arm("fp16", [(lambda w=w: P.fp16_gemv(w, x, y)) for w in Ws], served, None, Ws)
        log(f"[bench] fp16: {served} bytes/GEMV, {reps} replicas")
    if "noweights" in wanted:
        arms["noweights"] = Arm("noweights", [lambda: P.noweights_ctrl(base_desc, x, y)], 0)
    return inp, arms, y


def verify_arms(torch, inp, arms, y):
    """Every arm's output, before any timing (as §3.1 checks every arm first):
    each replica of each layout gives the Planes14 output bit for bit (all
    layouts sum in one order); the FP16 control agrees within
    max_r |Δy_r| / (‖W_r‖·‖x‖) ≤ 2e-3, with ‖W_r‖ from the block scales (each
    block direction has unit norm, centroids 1); the no-weights control writes
    one value, Σx, on every row."""
    import numpy as np
    res = {"replicas_checked": 0}

    def out(launch):
        launch()
        torch.cuda.synchronize()
        return y.clone()

    ref = out(arms["planes14"].launchers[0])
    if not bool(torch.isfinite(ref).all()):
        sys.exit("verification failed: planes14 output is not finite")
    same = []
    for name, arm in arms.items():
        if name in ("fp16", "noweights"):
            continue
        for i, launch in enumerate(arm.launchers):
            if not torch.equal(out(launch).view(torch.int32), ref.view(torch.int32)):
                sys.exit(f"verification failed: {name} replica {i} differs from planes14")
            res["replicas_checked"] += 1
        same.append(name)
    res["bit_identical_to_planes14"] = same
    if "fp16" in arms:
        w_norm = np.sqrt((inp.scale.astype(np.float64) ** 2).sum(axis=1))
        x_norm = float(np.linalg.norm(inp.x.astype(np.float64)))
        worst = 0.0
        for i, launch in enumerate(arms["fp16"].launchers):
            d = (out(launch) - ref).abs().double().cpu().numpy()
            worst = max(worst, float((d / (w_norm * x_norm)).max()))
            res["replicas_checked"] += 1
        if not worst <= 2e-3:
            sys.exit(f"verification failed: fp16 control differs by {worst:.3g} (normalised)")
        res["fp16_max_normalised_diff"] = worst
    if "noweights" in arms:
        yn = out(arms["noweights"].launchers[0])
        if not (bool(torch.isfinite(yn).all()) and bool((yn == yn[0]).all())):
            sys.exit("verification failed: no-weights control rows differ")
        res["noweights_rows_equal"] = True
    log(f"[bench] verified before timing: {res}")
    return res


_HIP = None


def hip_runtime():
    """The HIP runtime PyTorch already loaded (looked up by its soname, never
    loaded a second time), or None."""
    global _HIP
    if _HIP is None:
        import ctypes
        try:
            _HIP = ctypes.CDLL("libamdhip64.so.7", mode=os.RTLD_NOLOAD)
        except OSError:
            _HIP = False
    return _HIP or None


class TimingEvent:
    """A HIP event for timing only: created with hipEventDisableSystemFence,
    so recording it writes back and invalidates no caches (the kernels between
    two such events see the caches as they would without them, and the
    markers' own cost shrinks).  Falls back to torch.cuda.Event where the
    runtime cannot be looked up; `kind` says which."""
    FLAGS = 0x20000000  # hipEventDisableSystemFence

    def __init__(self, torch):
        import ctypes
        self._c = ctypes
        self.hip = hip_runtime()
        if self.hip is None:
            self.kind = "torch.cuda.Event"
            self.ev = torch.cuda.Event(enable_timing=True)
            return
        self.kind = "hipEvent, no system fence"
        self.ev = ctypes.c_void_p()
        rc = self.hip.hipEventCreateWithFlags(ctypes.byref(self.ev), ctypes.c_uint(self.FLAGS))
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed: {rc}")

    def record(self, stream):
        if self.hip is None:
            self.ev.record(stream)
            return
        rc = self.hip.hipEventRecord(self.ev, self._c.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed: {rc}")

    def query(self):
        if self.hip is None:
            return self.ev.query()
        return self.hip.hipEventQuery(self.ev) == 0

    def elapsed_time(self, other):
        if self.hip is None:
            return self.ev.elapsed_time(other.ev)
        ms = self._c.c_float()
        rc = self.hip.hipEventElapsedTime(self._c.byref(ms), self.ev, other.ev)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed: {rc}")
        return ms.value

    def __del__(self):
        if getattr(self, "hip", None) is not None:
            self.hip.hipEventDestroy(self.ev)


_LAST_AHEAD = [True]


def lead_reps(steps, lead_len, factor=2):
    """Replays of a lead graph of lead_len launches to put ahead of a timed
    region of `steps` launches: the device then works through at least
    factor × steps launches before it reaches the timed region, time in which
    the host submits the timed launches (a cold graph's submission can take
    longer than the device takes to run its kernels)."""
    return max(1, -(-factor * steps // max(1, lead_len)))


def timed_replay(torch, lead, g, reps=2):
    """ms of one replay of graph g, timed with HIP events (TimingEvent) on the
    current stream.  The device is synchronised first; then `lead` (a graph,
    or None) is replayed `reps` times untimed and the events and g are
    enqueued behind it without waiting, so the device is still busy with the
    lead while the host submits g: the timed interval holds g's kernels back
    to back and not the host's submission of the graph.  Whether the host had
    submitted all of g before the device reached the first event is kept in
    _LAST_AHEAD.  The device is synchronised again before the events are
    read."""
    st = torch.cuda.current_stream()
    e0, e1 = TimingEvent(torch), TimingEvent(torch)
    torch.cuda.synchronize()
    if lead is not None:
        for _ in range(reps):
            lead.replay()
    e0.record(st)
    g.replay()
    _LAST_AHEAD[0] = not e0.query()
    e1.record(st)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1)


def time_arm(torch, arm, steps):
    """ms for `steps` GEMVs: one replay of a graph holding exactly `steps`
    launches (replicas 0, 1, …), timed with HIP events on the stream the
    kernels run on, between device synchronisations.  It is enqueued right
    behind replays of arm.evict_plan(steps), which streams the replicas the
    timed region does not read (≥ 512 MiB, twice the Infinity Cache), so that
    the timed replicas are read from HBM, and which keeps the device busy for
    at least twice the timed launches while the host submits them; an arm
    without weight bytes leads with replays of its own graph.  The timed graph
    is replayed once before the lead: a graph's first replay after other work
    runs its kernels about 0.5 µs slower each, which the timed replay should
    not carry."""
    g = arm.graph(torch, steps)
    lead, length = g, steps
    if arm.served_bytes:
        start, length, _ = arm.evict_plan(steps)
        lead = arm.graph(torch, length, start)
    g.replay()
    return timed_replay(torch, lead, g, lead_reps(steps, length))


def time_arm_stream(torch, arm, steps):
    """ms for `steps` GEMVs launched one by one on the stream (no graph),
    enqueued behind replays of the eviction graph of arm.evict_plan(steps)
    (at least three times the timed launches), and whether every launch was
    enqueued before the device reached the timed region (the first event
    still pending when the host had enqueued the last launch): then the
    interval holds the kernels back to back, neither the host's launch calls
    nor a graph's start."""
    start, length, _ = arm.evict_plan(steps)
    lead = arm.graph(torch, length, start)
    st = torch.cuda.current_stream()
    e0, e1 = TimingEvent(torch), TimingEvent(torch)
    torch.cuda.synchronize()
    for _ in range(max(2, lead_reps(steps, length, 3))):
        lead.replay()
    e0.record(st)
    arm.run(steps)
    e1.record(st)
    ahead = not e0.query()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1), ahead


def cycle_us(torch, arm, replays=3):
    """µs per GEMV over one whole cycle of the arm's replicas (≥ 1 GiB), median
    of `replays` timed replays, each led by an untimed one."""
    n = len(arm.launchers)
    g = arm.graph(torch, n)
    out = [timed_replay(torch, g, g, lead_reps(n, n)) * 1e3 / n for _ in range(replays)]
    return statistics.median(out)


def arms_table(args, torch, arms, inp):
    """§3.1's comparison: every arm timed as a k-GEMV replay, arms interleaved
    in a fixed order for args.rounds rounds, the first args.discard dropped;
    medians with min and max, and the median of the per-round ratios against
    the FP16 control."""
    k_arm = max(200, args.steps // 4)
    per_round = {n: [] for n in arms}
    for r in range(args.rounds):
        for n, a in arms.items():
            per_round[n].append(time_arm(torch, a, k_arm) * 1e3 / k_arm)
        log(f"[bench] {inp.M}x{inp.K} round {r + 1}/{args.rounds} done")
    kept = {n: v[args.discard:] for n, v in per_round.items()}
    table = {}
    for n, v in kept.items():
        med = statistics.median(v)
        row = {"us_per_gemv": round(med, 3), "min_us": round(min(v), 3), "max_us": round(max(v), 3),
               "served_bytes": arms[n].served_bytes}
        if arms[n].served_bytes:
            row["GBps"] = round(arms[n].served_bytes / (med * 1e-6) / 1e9, 1)
            row["pct_hbm_peak"] = round(100 * row["GBps"] / HBM_PEAK_GBS, 1)
            row["bits_per_weight"] = round(8 * arms[n].served_bytes / (inp.M * inp.Kpad), 3)
        if "fp16" in kept:
            ratios = [f / t for f, t in zip(kept["fp16"], v)]
            row["vs_fp16"] = round(statistics.median(ratios), 3)
        table[n] = row
    return table


def prologue_table(args, torch, P, arm):
    """µs per GEMV of the arm under each prologue mode (the order in which
    waves request their records; leech_set_prologue_mode), as cold-replica
    timed replays of 200 launches, modes interleaved over 5 rounds: the
    measurement behind the automatic choice."""
    k = 200
    res = {m: [] for m in ("auto", 0, 1, 2)}
    graphs = {}
    try:
        for m in res:
            P.set_prologue_mode(P.PROLOGUE_AUTO if m == "auto" else m)
            arm._graphs.clear()
            start, len_ev, _ = arm.evict_plan(k)
            graphs[m] = (arm.graph(torch, len_ev, start), arm.graph(torch, k))
        arm._graphs.clear()
    finally:
        P.set_prologue_mode(P.PROLOGUE_AUTO)
    for _ in range(5):
        for m, (ev, g) in graphs.items():
            g.replay()
            res[m].append(timed_replay(torch, ev, g, lead_reps(k, len_ev)) * 1e3 / k)
    del graphs
    return {str(m): round(statistics.median(v), 3) for m, v in res.items()}


def phase_table(torch, P, arm, x, y, steps=20):
    """Where a launch's time goes: `steps` back-to-back Planes14 launches over
    the arm's replicas (as the timed region: a graph behind the eviction
    replay), each recording per-workgroup stamps of the 100 MHz real-time
    counter (leech_gemv_phases: start, staging barrier passed, each wave's last
    unit decoded, last store).  Medians over launches of: the gap between one
    launch's last store and the next one's first workgroup start; the spread
    of workgroup starts; and, per workgroup (median over workgroups), the
    prologue (start to barrier), the loop (barrier to the last wave's last
    unit) and the tail (to the last store); beside them the event-timed µs per
    launch, the stamped span of all launches, and what the event window holds
    beyond it (its markers and the graph's start)."""
    import numpy as np
    mats = arm.mats
    n = len(mats)
    d = mats[0].desc
    tiles = -(-d.M // d.tile_rows)
    waves = min(8, -(-d.nb // d.lane_cols))
    st = torch.full((steps, tiles, 11), -1, dtype=torch.int64, device=x.device)
    g = torch.cuda.CUDAGraph()
    mats[0].gemv_phases(x, y, st[0])
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        for i in range(steps):
            mats[i % n].gemv_phases(x, y, st[i])
    start, length, _ = arm.evict_plan(steps)
    lead = arm.graph(torch, length, start)
    g.replay()
    ms = timed_replay(torch, lead, g, lead_reps(steps, length))
    s = st.cpu().numpy().astype(np.float64)
    del g
    t0, t1, t10 = s[:, :, 0], s[:, :, 1], s[:, :, 10]
    tw = s[:, :, 2:2 + waves].max(axis=2)
    starts, ends = t0.min(axis=1), t10.max(axis=1)
    span_ticks = ends[-1] - starts[0]
    # the real-time counter runs at 100 MHz; the event-timed interval also
    # holds the two event markers and the first launch's start, which the
    # stamps do not: their difference is the window's own cost
    us = lambda v: round(float(v) / 100.0, 3)  # noqa: E731
    med = lambda v: us(np.median(v))  # noqa: E731
    return {"launches": steps, "workgroups": tiles, "waves": waves,
            "event_us_per_launch": round(ms * 1e3 / steps, 3),
            "stamped_us_first_start_to_last_store": us(span_ticks),
            "event_window_minus_stamped_us": round(ms * 1e3 - span_ticks / 100.0, 3),
            "gap_between_launches_us": med(starts[1:] - ends[:-1]),
            "workgroup_start_spread_us": med(t0.max(axis=1) - starts),
            "prologue_us": med(np.median(t1 - t0, axis=1)),
            "loop_us": med(np.median(tw - t1, axis=1)),
            "tail_us": med(np.median(t10 - tw, axis=1)),
            "first_start_to_last_store_us": med(ends - starts),
            "span_us_by_launch": [us(v) for v in ends - starts],
            "gap_us_by_launch": [us(v) for v in starts[1:] - ends[:-1]]}


def shader_clock(torch, arm, seconds=1.0):
    """The shader clock while the arm's GEMVs run back to back: the current
    level of /sys/class/drm/card*/device/pp_dpm_sclk, sampled every 20 ms
    during about `seconds` of graph replays (median and range in MHz), or None
    where the file cannot be read."""
    import glob
    import re
    import threading
    paths = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
    samples, stop = [], []

    def poll():
        while not stop:
            for p in paths:
                try:
                    for line in open(p).read().splitlines():
                        m = re.match(r"\s*\d+:\s*(\d+)\s*[Mm][Hh]z\s*\*", line)
                        if m:
                            samples.append(int(m.group(1)))
                except OSError:
                    pass
            time.sleep(0.02)

    if not paths:
        return None
    n = len(arm.launchers)
    g = arm.graph(torch, n)
    g.replay()
    torch.cuda.synchronize()
    th = threading.Thread(target=poll)
    th.start()
    t0 = time.time()
    while time.time() - t0 < seconds:
        for _ in range(10):
            g.replay()
        torch.cuda.synchronize()
    stop.append(1)
    th.join()
    if not samples:
        return None
    return {"median_MHz": statistics.median(samples), "min_MHz": min(samples),
            "max_MHz": max(samples), "samples": len(samples),
            "source": "pp_dpm_sclk during back-to-back GEMV replays", "max_rated_MHz": 2400}


# One 8B-class decoder layer at batch 1: (name, rows, K), K padded to 24.
LAYER_8B = [("q", 4096, 4096), ("k", 1024, 4096), ("v", 1024, 4096), ("o", 4096, 4096),
            ("gate", 14336, 4096), ("up", 14336, 4096), ("down", 4096, 14336)]
FUSED_8B = [("qkv", ["q", "k", "v"]), ("o", ["o"]), ("gate_up", ["gate", "up"]), ("down", ["down"])]


def bench_layer(args, torch, P, synth):
    """µs per decoder layer: seven Planes14 GEMVs, the same weights in four
    fused launches (q/k/v and gate/up row-concatenated, §3.4), and seven FP16
    GEMVs; each timed as one graph replay of args.layer_steps layers walking
    ≥ 1 GiB of replicas."""
    import numpy as np
    dev = torch.device("cuda:0")
    cb = P.Codebook(12)
    dcb = P.DeviceCodebook(cb, dev)
    t0 = time.time()
    parts = {}
    for i, (name, M, K) in enumerate(LAYER_8B):
        inp = synth.make_gemv_inputs(M, K, seed=1000 + i, name=f"layer8b-{name}")
        parts[name] = inp
    log(f"[bench] 8B layer inputs ready in {time.time() - t0:.1f}s")
    xs = {K: torch.from_numpy(synth.make_activation(K, seed=1, name=f"layer8b-x{K}")).to(dev)
          for K in {K for _, _, K in LAYER_8B}}
    cen = (1.0, 1.0)

    def xfor(inp):
        return xs[inp.K]

    def leech(names):
        z = np.concatenate([parts[n].z for n in names])
        gain = np.concatenate([parts[n].gain for n in names])
        scale = np.concatenate([parts[n].scale for n in names])
        cls, sm, lv = cb.fields_from_points(z)
        return P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, gain, sm, lv, scale, dev)

    sep = {n: leech([n]) for n, _, _ in LAYER_8B}
    fused = {f: (leech(ns), [parts[n].M for n in ns]) for f, ns in FUSED_8B}
    layer_bytes = sum(m.desc.served_bytes for m in sep.values())
    reps = max(1, math.ceil(REPLICA_BYTES / layer_bytes))

    def clone(m):
        return P.LeechMatrix(m.desc, m.main.clone(), m.side0.clone(), m.side1.clone(),
                             m.scale.clone(), dcb)

    ys = {n: torch.empty(parts[n].M, dtype=torch.float32, device=dev) for n in parts}
    yf = {f: torch.empty(sum(r), dtype=torch.float32, device=dev) for f, (_, r) in fused.items()}
    sep_r = [sep] + [{n: clone(m) for n, m in sep.items()} for _ in range(reps - 1)]
    fus_r = [fused] + [{f: (clone(m), r) for f, (m, r) in fused.items()} for _ in range(reps - 1)]

    def run_sep(i):
        for n, m in sep_r[i % reps].items():
            m.gemv(xfor(parts[n]), ys[n], centroids=cen)

    def run_fused(i):
        for f, (m, rows) in fus_r[i % reps].items():
            m.gemv_grouped(xfor(parts[dict(FUSED_8B)[f][0]]), rows, [cen] * len(rows), yf[f])

    # FP16 arm: the same layer as binary16 weights (decoded on the device)
    fp = {}
    for n, m in sep.items():
        z, _, _ = m.decode()
        zf = z.float()
        inp = parts[n]
        fac = torch.from_numpy(inp.scale.astype("float32")).to(dev) / zf.pow(2).sum(-1).sqrt()
        fp[n] = (zf * fac[..., None]).reshape(inp.M, inp.Kpad).half().contiguous()
        del z, zf
    fp_bytes = sum(w.numel() * 2 for w in fp.values())
    fp_reps = max(1, math.ceil(REPLICA_BYTES / fp_bytes))
    fp_r = [fp] + [{n: w.clone() for n, w in fp.items()} for _ in range(fp_reps - 1)]

    def run_fp(i):
        for n, w in fp_r[i % fp_reps].items():
            P.fp16_gemv(w, xfor(parts[n]), ys[n])

    # rotated arm: every fused site first rotates its activation (§2.3, §6;
    # one rotation per site, shared by the site's groups), then runs its GEMV
    sites = [(f, parts[dict(FUSED_8B)[f][0]]) for f, _ in FUSED_8B]
    raw = {f: xfor(inp)[:inp.K] for f, inp in sites}
    signs = {f: torch.from_numpy(synth.make_signs(inp.K, seed=2, name=f"layer8b-{f}")).to(dev)
             for f, inp in sites}
    xrot = {f: torch.empty(inp.Kpad, dtype=torch.float16, device=dev) for f, inp in sites}

    def run_fused_rot(i):
        for f, (m, rows) in fus_r[i % reps].items():
            P.rotate_x(raw[f], signs[f], m.Kpad, out=xrot[f])
            m.gemv_grouped(xrot[f], rows, [cen] * len(rows), yf[f])

    # the same, with each GEMV rotating its activation in its own prologue
    def run_fused_rotk(i):
        for f, (m, rows) in fus_r[i % reps].items():
            m.gemv_rotated(raw[f], signs[f], rows, [cen] * len(rows), yf[f])

    # in the prologue where rotate_in_kernel says so, a separate rotation otherwise
    def run_fused_rotmix(i):
        for f, (m, rows) in fus_r[i % reps].items():
            if rotate_in_kernel(m, raw[f].numel()):
                m.gemv_rotated(raw[f], signs[f], rows, [cen] * len(rows), yf[f])
            else:
                P.rotate_x(raw[f], signs[f], m.Kpad, out=xrot[f])
                m.gemv_grouped(xrot[f], rows, [cen] * len(rows), yf[f])

    # outputs agree (fused rows are the separate rows, within f32 rounding)
    run_sep(0)
    run_fused(0)
    torch.cuda.synchronize()
    ysep = torch.cat([ys[n] for n in ("q", "k", "v")])
    rel = float(((yf["qkv"] - ysep).abs().max() / ysep.abs().max()).item())
    res = {}
    for name, fn, nrep in (("separate", run_sep, reps), ("fused", run_fused, reps),
                           ("fused_rot", run_fused_rot, reps), ("fused_rotk", run_fused_rotk, reps),
                           ("fused_rotmix", run_fused_rotmix, reps), ("fp16", run_fp, fp_reps)):
        steps = args.layer_steps
        g = torch.cuda.CUDAGraph()
        fn(0)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            for i in range(steps):
                fn(i)
        meds = [timed_replay(torch, g, g) * 1e3 / steps for _ in range(3)]
        res[name] = round(statistics.median(meds), 2)
        log(f"[bench] 8B layer {name}: {res[name]} us/layer ({nrep} replicas)")
        del g
    return {"workload": "one 8B-class decoder layer at batch 1 (q, o 4096x4104; k, v 1024x4104; "
                        "gate, up 14336x4104; down 4096x14352), Planes14",
            "served_bytes": layer_bytes, "us_separate_7_launches": res["separate"],
            "us_fused_4_launches": res["fused"],
            "us_fused_with_rotation_8_launches": res["fused_rot"],
            "us_fused_with_rotation_in_kernel_4_launches": res["fused_rotk"],
            "us_fused_with_rotation_mixed": res["fused_rotmix"],
            "us_fp16_7_launches": res["fp16"],
            "fusion_saves": round(1 - res["fused"] / res["separate"], 4),
            "fused_vs_fp16": round(res["fp16"] / res["fused"], 3),
            "fused_GBps": round(layer_bytes / (res["fused"] * 1e-6) / 1e9, 1),
            "qkv_fused_vs_separate_max_rel_diff": rel}


# One 14B-class decoder layer: hidden 5120, 40 query heads and 8 KV heads of
# dimension 128, FFN 17408; and the fp16 output head (vocabulary 152064).
MODEL_14B = [("q", 5120, 5120), ("k", 1024, 5120), ("v", 1024, 5120), ("o", 5120, 5120),
             ("gate", 17408, 5120), ("up", 17408, 5120), ("down", 5120, 17408)]
HEAD_14B = (152064, 5120)


def replay_us(torch, fn, reps):
    """µs per call of fn(i), i = 0..reps-1, captured once in a HIP graph:
    median of three timed replays after one untimed replay."""
    fn(0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(reps):
            fn(i)
    meds = [timed_replay(torch, g, g) * 1e3 / reps for _ in range(3)]
    del g
    return statistics.median(meds)


def bench_step14b(args, torch, P, synth):
    """One batch-1 decode step of a 14B-class model through its projections
    (§3.1's "one token through the projections", at 14B shapes): 40 layers of
    seven Leech-coded GEMVs each, then the fp16 output head, which is the same
    in every arm.  Arms: Planes14 in 280 launches; Planes14 fused (q/k/v and
    gate/up row-concatenated, 160 launches); the fused arm behind the
    activation rotation of each of the four sites (160 more launches); and FP16
    weights in 280 launches.  One layer's codes are drawn and every layer
    holds its own copy in distinct buffers (8.8 GB of Leech bytes, 28 GB of
    FP16), so every step streams from HBM."""
    import numpy as np
    L = args.step14b_layers
    dev = torch.device("cuda:0")
    cb = P.Codebook(12)
    dcb = P.DeviceCodebook(cb, dev)
    t0 = time.time()
    parts = {name: synth.make_gemv_inputs(M, K, seed=2000 + i, name=f"step14b-{name}")
             for i, (name, M, K) in enumerate(MODEL_14B)}
    log(f"[bench] 14B layer inputs ready in {time.time() - t0:.1f}s")
    xs = {K: torch.from_numpy(synth.make_activation(K, seed=4, name=f"step14b-x{K}")).to(dev)
          for K in {K for _, _, K in MODEL_14B}}
    cen = (1.0, 1.0)

    def leech(names):
        z = np.concatenate([parts[n].z for n in names])
        gain = np.concatenate([parts[n].gain for n in names])
        scale = np.concatenate([parts[n].scale for n in names])
        cls, sm, lv = cb.fields_from_points(z)
        return P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, gain, sm, lv, scale, dev)

    def clone(m):
        return P.LeechMatrix(m.desc, m.main.clone(), m.side0.clone(), m.side1.clone(),
                             m.scale.clone(), dcb)

    sep0 = {n: leech([n]) for n, _, _ in MODEL_14B}
    fus0 = {f: (leech(ns), [parts[n].M for n in ns]) for f, ns in FUSED_8B}
    leech_bytes = sum(m.desc.served_bytes for m in sep0.values())
    sep = [sep0] + [{n: clone(m) for n, m in sep0.items()} for _ in range(L - 1)]
    fus = [fus0] + [{f: (clone(m), r) for f, (m, r) in fus0.items()} for _ in range(L - 1)]
    fp0 = {}
    for n, m in sep0.items():
        z, _, _ = m.decode()
        zf = z.float()
        inp = parts[n]
        fac = torch.from_numpy(inp.scale.astype("float32")).to(dev) / zf.pow(2).sum(-1).sqrt()
        fp0[n] = (zf * fac[..., None]).reshape(inp.M, inp.Kpad).half().contiguous()
        del z, zf
    fp = [fp0] + [{n: w.clone() for n, w in fp0.items()} for _ in range(L - 1)]
    fp_bytes = sum(w.numel() * 2 for w in fp0.values())
    gen = torch.Generator(device=dev)
    gen.manual_seed(5)
    head = (torch.randn(HEAD_14B, generator=gen, device=dev) * 0.02).half()
    y_head = torch.empty(HEAD_14B[0], dtype=torch.float32, device=dev)
    x_head = xs[HEAD_14B[1]][:HEAD_14B[1]]
    ys = {n: torch.empty(parts[n].M, dtype=torch.float32, device=dev) for n in parts}
    yf = {f: torch.empty(sum(r), dtype=torch.float32, device=dev) for f, (_, r) in fus0.items()}
    site_inp = {f: parts[dict(FUSED_8B)[f][0]] for f, _ in FUSED_8B}
    raw = {f: xs[inp.K][:inp.K] for f, inp in site_inp.items()}
    signs = {f: torch.from_numpy(synth.make_signs(inp.K, seed=6, name=f"step14b-{f}")).to(dev)
             for f, inp in site_inp.items()}
    xrot = {f: torch.empty(inp.Kpad, dtype=torch.float16, device=dev)
            for f, inp in site_inp.items()}
    log(f"[bench] 14B step: {L} layers resident, {L * leech_bytes / 1e9:.2f} GB Planes14, "
        f"{L * fp_bytes / 1e9:.2f} GB FP16, head {head.numel() * 2 / 1e9:.3f} GB")

    def run_head():
        P.fp16_gemv(head, x_head, y_head)

    def step_sep(_):
        for layer in sep:
            for n, m in layer.items():
                m.gemv(xs[parts[n].K], ys[n], centroids=cen)
        run_head()

    def step_fused(_):
        for layer in fus:
            for f, (m, rows) in layer.items():
                m.gemv_grouped(xs[site_inp[f].K], rows, [cen] * len(rows), yf[f])
        run_head()

    def step_fused_rot(_):
        for layer in fus:
            for f, (m, rows) in layer.items():
                P.rotate_x(raw[f], signs[f], m.Kpad, out=xrot[f])
                m.gemv_grouped(xrot[f], rows, [cen] * len(rows), yf[f])
        run_head()

    def step_fused_rotk(_):
        for layer in fus:
            for f, (m, rows) in layer.items():
                m.gemv_rotated(raw[f], signs[f], rows, [cen] * len(rows), yf[f])
        run_head()

    def step_fused_rotmix(_):
        for layer in fus:
            for f, (m, rows) in layer.items():
                if rotate_in_kernel(m, raw[f].numel()):
                    m.gemv_rotated(raw[f], signs[f], rows, [cen] * len(rows), yf[f])
                else:
                    P.rotate_x(raw[f], signs[f], m.Kpad, out=xrot[f])
                    m.gemv_grouped(xrot[f], rows, [cen] * len(rows), yf[f])
        run_head()

    def step_fp(_):
        for layer in fp:
            for n, w in layer.items():
                P.fp16_gemv(w, xs[parts[n].K], ys[n])
        run_head()

    transcode = bench_transcode(torch, P, dcb, parts, dev)

    res = {}
    for name, fn in (("separate", step_sep), ("fused", step_fused), ("fused_rot", step_fused_rot),
                     ("fused_rotk", step_fused_rotk), ("fused_rotmix", step_fused_rotmix),
                     ("fp16", step_fp)):
        res[name] = round(replay_us(torch, fn, 3), 1)
        log(f"[bench] 14B step {name}: {res[name]} us")
    head_us = round(replay_us(torch, lambda _: run_head(), 20), 1)
    leech_fused = res["fused"] - head_us
    return {"workload": f"14B-class decode step at batch 1: {L} layers x (q, o 5120x5136; k, v "
                        f"1024x5136; gate, up 17408x5136; down 5120x17424) Planes14, then the fp16 "
                        f"head 152064x5120 (same in every arm)",
            "layers": L, "planes14_bytes": L * leech_bytes, "fp16_bytes": L * fp_bytes,
            "head_bytes": head.numel() * 2,
            "us_separate_280": res["separate"], "us_fused_160": res["fused"],
            "us_fused_with_rotation_320": res["fused_rot"],
            "us_fused_with_rotation_in_kernel_160": res["fused_rotk"],
            "us_fused_with_rotation_mixed": res["fused_rotmix"],
            "us_fp16_280": res["fp16"],
            "us_head": head_us,
            "fp16_vs_fused": round(res["fp16"] / res["fused"], 3),
            "fp16_vs_fused_with_rotation": round(res["fp16"] / res["fused_rot"], 3),
            "fp16_vs_fused_with_rotation_mixed": round(res["fp16"] / res["fused_rotmix"], 3),
            "fp16_vs_fused_with_rotation_in_kernel": round(res["fp16"] / res["fused_rotk"], 3),
            "leech_part_GBps_fused": round(L * leech_bytes / (leech_fused * 1e-6) / 1e9, 1),
            "transcode": transcode}


BLOCKS_4B = 150_681_600     # blocks of the paper's 4B model (§3.1), for the time to unfold it


def bench_transcode(torch, P, dcb, parts, dev):
    """Load-time unfolding of one 14B layer (§2.2): format-v1 codes -> Planes14
    streams.  GPU: the transcoder over the seven projections, codes resident
    in HBM, median of five passes.  Host: the library's multithreaded decode of
    the codes to fields plus the Planes14 expansion, once."""
    import numpy as np
    cb = dcb.cb
    codes = {}
    for n, inp in parts.items():
        cls, sm, lv = cb.fields_from_points(inp.z)
        codes[n] = P.index_encode(cb, cls, inp.gain, sm, lv)
    blocks = sum(c.size for c in codes.values())
    d_codes = {n: torch.from_numpy(c.view(np.int64)).to(dev) for n, c in codes.items()}
    descs = {n: P.planes14_desc(c.shape[0], c.shape[1] * 24) for n, c in codes.items()}
    mains = {n: torch.empty(d.main_bytes, dtype=torch.uint8, device=dev) for n, d in descs.items()}
    bad = torch.zeros(len(codes), dtype=torch.int32, device=dev)

    def run():
        for i, n in enumerate(codes):
            P._lib.transcode_planes14(descs[n], dcb.index.data_ptr(), d_codes[n].data_ptr(),
                                      mains[n].data_ptr(), bad[i:].data_ptr(),
                                      torch.cuda.current_stream().cuda_stream)
    run()
    torch.cuda.synchronize()
    if int(bad.sum().item()):
        raise RuntimeError("transcoder rejected valid codes")
    times = []
    for _ in range(5):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e3)
    gpu_us = statistics.median(times)
    t0 = time.perf_counter()
    for n, c in codes.items():
        f = P.index_decode(cb, c)
        P.expand_layout(cb, P.PLANES14, *f)
    host_s = time.perf_counter() - t0
    moved = blocks * (8 + 14)
    log(f"[bench] transcode {blocks} blocks: GPU {gpu_us:.0f} us, host {host_s:.2f} s")
    return {"blocks": blocks, "gpu_us": round(gpu_us, 1),
            "gpu_Mblocks_per_s": round(blocks / gpu_us, 1),
            "gpu_GBps_codes_in_records_out": round(moved / (gpu_us * 1e-6) / 1e9, 1),
            "host_s_decode_and_expand": round(host_s, 3), "host_threads": os.cpu_count(),
            "host_Mblocks_per_s": round(blocks / host_s / 1e6, 2),
            "gpu_s_for_4B_model_blocks": round(BLOCKS_4B / blocks * gpu_us * 1e-6, 4),
            "host_s_for_4B_model_blocks": round(BLOCKS_4B / blocks * host_s, 2)}


def bench_batch(args, torch, P, synth, inp, arms, batches=(1, 2, 4, 8, 16)):
    """Batched GEMV (§6 "Batching") on the bench workload in Planes14: µs per
    launch of Y = W X for B activations (each block decoded once for up to 16
    of them), walking the same replicas as the Planes14 arm, with the
    library's default products (the matrix cores for B > 1) and, for B > 1,
    with v_dot2 per activation (dot2_us); the largest normalised
    difference of Y[0] and Y[B-1] from their single GEMVs; beside
    it the FP16 weights through the library GEMM (torch.matmul, hipBLASLt) on
    the same B, as the batched FP16 reference."""
    import numpy as np
    dev = torch.device("cuda:0")
    p14 = arms["planes14"]
    reps = len(p14.launchers)
    leech = p14.mats
    res = {}
    fp = arms.get("fp16")
    for B in batches:
        X = torch.from_numpy(np.stack([synth.make_activation(inp.K, seed=50 + b, name="bench-batch")
                                       for b in range(B)])).to(dev)
        Y = torch.empty((B, inp.M), dtype=torch.float32, device=dev)
        leech[0].gemv_batch(X, Y)
        diff = 0.0
        for b in {0, B - 1}:
            y1 = leech[0].gemv(X[b].contiguous())
            diff = max(diff, float((Y[b] - y1).abs().max() / y1.abs().max()))
        us = replay_us(torch, lambda i: leech[i % reps].gemv_batch(X, Y), args.layer_steps)
        mx = B > 1
        row = {"us": round(us, 2), "us_per_vector": round(us / B, 3),
               "weight_GBps": round(p14.served_bytes / (us * 1e-6) / 1e9, 1),
               "products": "mfma" if mx else "dot2", "max_norm_diff_vs_single": diff}
        if B > 1:
            P.set_batch_mode(P.BATCH_DOT2)
            try:
                us_d = replay_us(torch, lambda i: leech[i % reps].gemv_batch(X, Y),
                                 args.layer_steps)
            finally:
                P.set_batch_mode(P.BATCH_AUTO)
            row["dot2_us"] = round(us_d, 2)
            row["dot2_vs_default"] = round(us_d / us, 3)
        if fp is not None:
            Ws = fp.mats
            Xt = X.t().contiguous()
            Yf = torch.empty((inp.M, B), dtype=torch.float16, device=dev)
            # eager launches: the library GEMM is kept out of graph capture
            for i in range(10):
                torch.matmul(Ws[i % len(Ws)], Xt, out=Yf)
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for i in range(args.layer_steps):
                torch.matmul(Ws[i % len(Ws)], Xt, out=Yf)
            e1.record()
            torch.cuda.synchronize()
            us_fp = e0.elapsed_time(e1) * 1e3 / args.layer_steps
            row["fp16_gemm_us"] = round(us_fp, 2)
            row["fp16_vs_planes14"] = round(us_fp / us, 3)
        res[f"B{B}"] = row
        log(f"[bench] batch B={B}: {row}")
    return res


BATCH_14B = [("q/k/v fused", 7168, 5136), ("o", 5120, 5136), ("gate/up fused", 34816, 5136),
             ("down", 5120, 17424)]


def bench_batch_14b(args, torch, P, synth, batches=(4, 16)):
    """Batched launches (§6 "Batching") at the 14B-class fused projection
    shapes, Planes14 in the library's geometry: µs per launch of Y = W X for B
    activations on the matrix cores (the default) and with v_dot2, graph
    replay of args.layer_steps launches over replicas of >= 1 GiB."""
    import numpy as np
    dev = torch.device("cuda:0")
    dcb = P.DeviceCodebook(P.Codebook(12), dev)
    res = {}
    for i, (name, M, K) in enumerate(BATCH_14B):
        inp = synth.make_gemv_inputs(M, K, seed=2000 + i, name=f"batch14b-{name}")
        cls, sm, lv = dcb.cb.fields_from_points(inp.z)
        m0 = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
        reps = max(1, math.ceil(REPLICA_BYTES / m0.desc.served_bytes))
        mats = [m0] + [P.LeechMatrix(m0.desc, m0.main.clone(), m0.side0.clone(),
                                     m0.side1.clone(), m0.scale.clone(), dcb)
                       for _ in range(reps - 1)]
        row = {"geometry": f"{m0.desc.lane_cols}x{m0.desc.tile_rows}", "replicas": reps}
        for B in batches:
            X = torch.from_numpy(np.stack([synth.make_activation(K, seed=60 + b, name="batch14b")
                                           for b in range(B)])).to(dev)
            Y = torch.empty((B, M), dtype=torch.float32, device=dev)
            row[f"B{B}_us"] = round(replay_us(torch, lambda j: mats[j % reps].gemv_batch(X, Y),
                                              args.layer_steps), 2)
            P.set_batch_mode(P.BATCH_DOT2)
            try:
                row[f"B{B}_dot2_us"] = round(replay_us(
                    torch, lambda j: mats[j % reps].gemv_batch(X, Y), args.layer_steps), 2)
            finally:
                P.set_batch_mode(P.BATCH_AUTO)
        key = f"{name} {M}x{K}"
        res[key] = row
        log(f"[bench] batch 14B {key}: {row}")
        del mats, m0
        torch.cuda.empty_cache()
    return res


def bench_rotation(args, torch, P, synth, widths=(4096, 14336, 17408)):
    """µs per activation rotation (blockwise Walsh–Hadamard, fp16 in and out)
    at the 8B and 14B site widths: one graph replay of args.layer_steps
    launches, median of three replays (the launch gap included)."""
    dev = torch.device("cuda:0")
    res = {}
    for K in widths:
        x = torch.from_numpy(synth.make_activation(K, seed=3, name=f"rot{K}")[:K].copy()).to(dev)
        sg = torch.from_numpy(synth.make_signs(K, seed=3, name=f"rot{K}")).to(dev)
        Kpad = synth.padded_k(K)
        out = torch.empty(Kpad, dtype=torch.float16, device=dev)
        P.rotate_x(x, sg, Kpad, out=out)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(args.layer_steps):
                P.rotate_x(x, sg, Kpad, out=out)
        meds = [timed_replay(torch, g, g) * 1e3 / args.layer_steps for _ in range(3)]
        n = K & -K
        res[f"K{K}"] = {"us": round(statistics.median(meds), 3), "block": n, "workgroups": K // n}
        log(f"[bench] rotation K={K}: {res[f'K{K}']}")
        del g
    return res


# GEMV shapes (rows, K) of the 8B and 14B rotation sites (q/k/v and gate/up
# row-concatenated): the activation rotated by the separate kernel, or inside
# the GEMV's prologue.
ROT_SITES = [(4096, 4096), (6144, 4096), (28672, 4096), (4096, 14336),
             (7168, 5120), (34816, 5120), (5120, 17408)]


def bench_rotation_sites(args, torch, P, synth):
    """µs per site: the GEMV on a pre-rotated activation, rotate_x then the
    GEMV, and gemv_rotated (the rotation in the GEMV's prologue); each a graph
    replay of args.layer_steps calls walking ≥ 1 GiB of weight replicas."""
    dev = torch.device("cuda:0")
    dcb = P.DeviceCodebook(P.Codebook(12), dev)
    res = {}
    for M, K in ROT_SITES:
        inp = synth.make_gemv_inputs(M, K, seed=7, name=f"rotsite-{M}x{K}")
        cls, sm, lv = dcb.cb.fields_from_points(inp.z)
        m0 = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
        reps = max(1, math.ceil(REPLICA_BYTES / m0.desc.served_bytes))
        mats = [m0] + [P.LeechMatrix(m0.desc, m0.main.clone(), m0.side0.clone(),
                                     m0.side1.clone(), m0.scale.clone(), dcb)
                       for _ in range(reps - 1)]
        x = torch.from_numpy(inp.x[:K].copy()).to(dev)
        sg = torch.from_numpy(synth.make_signs(K, seed=7, name=f"rotsite-{M}x{K}")).to(dev)
        xr = P.rotate_x(x, sg, inp.Kpad)
        y = torch.empty(M, dtype=torch.float32, device=dev)
        n = args.layer_steps
        row = {
            "gemv_us": replay_us(torch, lambda i: mats[i % reps].gemv(xr, y), n),
            "rotate_then_gemv_us": replay_us(
                torch, lambda i: (P.rotate_x(x, sg, inp.Kpad, out=xr), mats[i % reps].gemv(xr, y)), n),
            "gemv_rotated_us": replay_us(
                torch, lambda i: mats[i % reps].gemv_rotated(x, sg, y=y), n),
        }
        row = {k: round(v, 2) for k, v in row.items()}
        row["lane_cols"] = m0.desc.lane_cols
        res[f"{M}x{K}"] = row
        log(f"[bench] rotation site {M}x{K}: {row}")
        del mats, m0
        torch.cuda.empty_cache()
    return res


# Large single GEMVs, where the fixed cost of a launch (its dispatch gap, the
# first loads' latency, the reduction) is small against the stream.
LARGE = [(16384, 16384), (32768, 16384), (152064, 5120)]


def bench_large(args, torch, P, synth):
    """µs and served GB/s of the Planes14 GEMV on large matrices, next to the
    FP16 control on the same decoded weights: each a graph replay over ≥ 1 GiB
    of replicas, after the Planes14 output is checked against the FP16
    control's (max_r |Δy_r| / (‖W_r‖·‖x‖) ≤ 2e-3)."""
    import numpy as np
    dev = torch.device("cuda:0")
    dcb = P.DeviceCodebook(P.Codebook(12), dev)
    res = {}
    for M, K in LARGE:
        t0 = time.time()
        inp = synth.make_gemv_inputs(M, K, seed=5, name=f"large-{M}x{K}")
        cls, sm, lv = dcb.cb.fields_from_points(inp.z)
        m0 = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
        del cls, sm, lv
        sb = m0.desc.served_bytes
        reps = max(1, math.ceil(REPLICA_BYTES / sb))
        mats = [m0] + [P.LeechMatrix(m0.desc, m0.main.clone(), m0.side0.clone(), m0.side1.clone(),
                                     m0.scale.clone(), dcb) for _ in range(reps - 1)]
        x = torch.from_numpy(inp.x).to(dev)
        y = torch.empty(M, dtype=torch.float32, device=dev)
        y16 = torch.empty(M, dtype=torch.float32, device=dev)
        z, _, _ = m0.decode()
        zf = z.float()
        del z
        fac = torch.from_numpy(inp.scale.astype("float32")).to(dev) / zf.pow(2).sum(-1).sqrt()
        W = (zf * fac[..., None]).reshape(M, inp.Kpad).half().contiguous()
        del zf, fac
        m0.gemv(x, y)
        P.fp16_gemv(W, x, y16)
        torch.cuda.synchronize()
        w_norm = np.sqrt((inp.scale.astype(np.float64) ** 2).sum(axis=1))
        x_norm = float(np.linalg.norm(inp.x.astype(np.float64)))
        diff = float(((y - y16).abs().double().cpu().numpy() / (w_norm * x_norm)).max())
        if not diff <= 2e-3:
            sys.exit(f"verification failed: large {M}x{K} planes14 vs fp16 {diff:.3g}")
        fr = max(1, math.ceil(REPLICA_BYTES / (W.numel() * 2)))
        Ws = [W] + [W.clone() for _ in range(fr - 1)]
        n = 100
        us = replay_us(torch, lambda i: mats[i % reps].gemv(x, y), n)
        usf = replay_us(torch, lambda i: P.fp16_gemv(Ws[i % fr], x, y16), n)
        row = {"Kpad": inp.Kpad, "lane_cols": m0.desc.lane_cols, "served_bytes": sb,
               "us": round(us, 2), "GBps": round(sb / us / 1e3, 1),
               "pct_hbm_peak": round(100 * sb / us / 1e3 / HBM_PEAK_GBS, 1),
               "fp16_us": round(usf, 2), "fp16_GBps": round(W.numel() * 2 / usf / 1e3, 1),
               "fp16_vs_planes14": round(usf / us, 3), "max_normalised_diff_vs_fp16": diff}
        res[f"{M}x{K}"] = row
        log(f"[bench] large {M}x{K}: {row} ({time.time() - t0:.0f}s)")
        del mats, m0, Ws, W, inp
        torch.cuda.empty_cache()
    return res


# Decoder projection shapes (rows, Kpad) of the 8B and 14B layers, fused
# (q/k/v, gate/up) and separate, and the layout sweep's square shape.
GEOMETRY_SHAPES = [(4096, 4104), (1024, 4104), (6144, 4104), (14336, 4104), (28672, 4104),
                   (4096, 14352), (5120, 5136), (1024, 5136), (7168, 5136), (17408, 5136),
                   (34816, 5136), (5120, 17424), (8192, 8208)]
GEOMETRY_SHAPES_MORE = [(3072, 3096), (2048, 2064), (12288, 12312), (6144, 6168), (10240, 5136),
                        (20480, 5136), (24576, 4104), (8192, 4104), (4096, 8208), (16384, 4104),
                        (2560, 5136), (12288, 4104), (3584, 4104), (9216, 4104)]
# the broad set of --geometry-all: (lane_cols, tile heights)
GEOMETRY_ALL = {1: [16, 24, 32, 40, 48, 56, 64], 2: [8, 12, 16, 20, 24, 28, 32], 3: [8, 12, 16, 20],
                4: [4, 8, 12, 16], 8: [4, 8], 16: [4]}


def geometry_candidates(M, Kpad, n=6):
    """The n geometries (lane_cols, tile_rows) of least cost under a simple
    ranking, ceil(tiles / 256) · (units per wave + 3), plus the power-of-two
    tile of the same lane_cols."""
    nb = Kpad // 24
    cands = []
    for C in (1, 2, 3, 4, 8, 16):
        for R in range(4, 64 // C + 1, 4):
            tiles = -(-M // R)
            groups = -(-nb // C)
            waves = min(8, groups)
            cost = -(-tiles // 256) * (-(-groups // waves) + 3)
            cands.append((cost, -tiles, -R * C, C, R))
    cands.sort()
    out = [(c, r) for *_, c, r in cands[:n]]
    for C in (1, 2, 4, 8, 16):
        if (C, 64 // C) not in out and any(c == C for c, _ in out):
            out.append((C, 64 // C))
    return out


def bench_geometry(args, torch, P, synth):
    """µs per Planes14 GEMV of each candidate tile geometry on the decoder
    projection shapes: the measurement behind the library's geometry rule.
    Codes are drawn once (Planes14's time does not depend on them) and tiled
    into each shape; every geometry's y is first checked against the library
    choice's (normalised difference ≤ 2e-3); each timing is a graph replay over
    ≥ 512 MiB of replicas, geometries interleaved over three rounds, medians.
    --geometry-all times the broad set GEOMETRY_ALL on these shapes and on
    GEOMETRY_SHAPES_MORE."""
    import numpy as np
    dev = torch.device("cuda:0")
    dcb = P.DeviceCodebook(P.Codebook(12), dev)
    pool = synth.make_gemv_inputs(512, 24 * 512, seed=11, name="geometry-pool")
    pcls, psm, plv = dcb.cb.fields_from_points(pool.z)
    pcls, psm, plv = pcls.reshape(-1), psm.reshape(-1), plv.reshape(-1, 24)
    pgain, pscale = pool.gain.reshape(-1), pool.scale.reshape(-1)
    rng = np.random.default_rng(12)
    res = {}
    shapes = GEOMETRY_SHAPES + (GEOMETRY_SHAPES_MORE if args.geometry_all else [])
    for M, Kpad in shapes:
        t0 = time.time()
        nb = Kpad // 24
        pick = rng.integers(0, pcls.size, M * nb)
        cls, sm = pcls[pick].reshape(M, nb), psm[pick].reshape(M, nb)
        lv, gain = plv[pick].reshape(M, nb, 24), pgain[pick].reshape(M, nb)
        scale = pscale[pick].reshape(M, nb)
        x = torch.from_numpy(synth.make_activation(Kpad, seed=13, name="geometry")).to(dev)
        y = torch.empty(M, dtype=torch.float32, device=dev)
        lib = P.layout_geometry(M, Kpad)
        geos = ([(c, r) for c, rs in GEOMETRY_ALL.items() for r in rs] if args.geometry_all
                else geometry_candidates(M, Kpad))
        if lib not in geos:
            geos.insert(0, lib)
        mats, yref = {}, None
        w_norm = torch.from_numpy(np.sqrt((scale.astype(np.float64) ** 2).sum(1))).to(dev)
        x_norm = float(x.double().norm())
        for geo in [lib] + [g for g in geos if g != lib]:
            m0 = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, gain, sm, lv, scale, dev,
                                           geometry=geo)
            m0.gemv(x, y)
            torch.cuda.synchronize()
            if yref is None:
                yref = y.clone()
            d = float(((y - yref).abs().double() / (w_norm * x_norm)).max())
            if not d <= 2e-3:
                sys.exit(f"verification failed: geometry {geo} at {M}x{Kpad}: {d:.3g}")
            reps = max(1, math.ceil((REPLICA_BYTES // 2) / m0.desc.served_bytes))
            mats[geo] = [m0] + [P.LeechMatrix(m0.desc, m0.main.clone(), m0.side0, m0.side1,
                                              m0.scale.clone(), dcb) for _ in range(reps - 1)]
        steps = 200 if M * nb < 2_000_000 else 60
        times = {g: [] for g in mats}
        for _ in range(3):
            for g, ms in mats.items():
                times[g].append(replay_us(torch, lambda i, ms=ms: ms[i % len(ms)].gemv(x, y),
                                          steps))
        row = {f"{c}x{r}": round(statistics.median(v), 2) for (c, r), v in times.items()}
        best = min(row, key=row.get)
        res[f"{M}x{Kpad}"] = {"library": f"{lib[0]}x{lib[1]}", "best": best, "us": row}
        log(f"[bench] geometry {M}x{Kpad}: library {lib}, best {best}, {row} "
            f"({time.time() - t0:.0f}s)")
        del mats, yref
        torch.cuda.empty_cache()
    return res


SWEEP = [1024, 2048, 3072, 4096, 6144, 8192, 12288, 16384]


def bench_sweep(args, torch, P, synth):
    """Square Planes14 GEMVs from 1024² to 16384² next to the FP16 control
    (random fp16 weights of the same shape: its time depends on the bytes
    only), each a graph replay over ≥ 1 GiB of replicas: where the fixed cost
    of a launch stops mattering."""
    dev = torch.device("cuda:0")
    dcb = P.DeviceCodebook(P.Codebook(12), dev)
    res = {}
    for n in SWEEP:
        inp = synth.make_gemv_inputs(n, n, seed=8, name=f"sweep-{n}")
        cls, sm, lv = dcb.cb.fields_from_points(inp.z)
        m0 = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
        del cls, sm, lv
        sb = m0.desc.served_bytes
        reps = max(1, math.ceil(REPLICA_BYTES / sb))
        mats = [m0] + [P.LeechMatrix(m0.desc, m0.main.clone(), m0.side0.clone(), m0.side1.clone(),
                                     m0.scale.clone(), dcb) for _ in range(reps - 1)]
        x = torch.from_numpy(inp.x).to(dev)
        y = torch.empty(n, dtype=torch.float32, device=dev)
        W = torch.randn(n, inp.Kpad, device=dev, dtype=torch.float16)
        fr = max(1, math.ceil(REPLICA_BYTES / (W.numel() * 2)))
        Ws = [W] + [W.clone() for _ in range(fr - 1)]
        steps = 300 if sb < 5e7 else 100
        us = replay_us(torch, lambda i: mats[i % reps].gemv(x, y), steps)
        usf = replay_us(torch, lambda i: P.fp16_gemv(Ws[i % fr], x, y), steps)
        row = {"Kpad": inp.Kpad, "lane_cols": m0.desc.lane_cols, "served_bytes": sb,
               "us": round(us, 2), "GBps": round(sb / us / 1e3, 1),
               "pct_hbm_peak": round(100 * sb / us / 1e3 / HBM_PEAK_GBS, 1),
               "fp16_us": round(usf, 2), "fp16_GBps": round(W.numel() * 2 / usf / 1e3, 1)}
        res[str(n)] = row
        log(f"[bench] sweep {n}x{n}: {row}")
        del mats, m0, Ws, W, inp
        torch.cuda.empty_cache()
    return res


def measured_traffic(config):
    """HBM bytes per launch of the Planes14 GEMV from the committed counter
    runs (FETCH_SIZE + WRITE_SIZE, each scaled by a known-size copy), or None
    when the kernel source has changed since those runs or the workload was not
    profiled."""
    import hashlib
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
        src = open(os.path.join(ROOT, "paper_2609_02652_amd", "csrc", "kernels.hip"), "rb").read()
    except OSError:
        return None
    if rec.get("kernels_sha256") != hashlib.sha256(src).hexdigest():
        return None
    c = rec.get("configs", {}).get(config)
    return c["traffic_bytes"] if c else None


def bench_floor(args, torch, P, synth):
    """The per-launch floor under graph replay: µs per launch of a one-element
    torch fill (the smallest kernel the runtime launches), of the no-weights
    control and of the Planes14 GEMV on one 24-wide block (one tile, one
    unit), and of both at the bench shape with a single cache-resident copy
    of the records.  Each is one replay of a graph of args.floor_steps
    launches, best of five; the bench shape's fraction of peak with the fill's
    floor taken out is reported beside it."""
    dev = torch.device("cuda:0")
    n = args.floor_steps

    def per_launch(fn):
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(n):
                fn()
        best = min(timed_replay(torch, g, g) * 1e3 / n for _ in range(5))
        del g
        return round(best, 3)

    t = torch.zeros(1, device=dev)
    out = {"launches_per_graph": n, "fill_one_element_us": per_launch(lambda: t.fill_(1.0))}
    dcb = P.DeviceCodebook(P.Codebook(12), dev)
    for tag, (M, K) in (("one_block", (64, 24)), ("bench_shape_cached", CONFIGS[args.config])):
        inp = synth.make_gemv_inputs(M, K, seed=args.seed, name="launch-floor")
        cls, sm, lv = dcb.cb.fields_from_points(inp.z)
        m = P.LeechMatrix.from_fields(dcb, P.PLANES14, cls, inp.gain, sm, lv, inp.scale, dev)
        x = torch.from_numpy(inp.x).to(dev)
        y = torch.empty(M, dtype=torch.float32, device=dev)
        out[tag] = {"M": M, "K": K,
                    "planes14_us": per_launch(lambda: m.gemv(x, y)),
                    "noweights_us": per_launch(lambda: P.noweights_ctrl(m.desc, x, y))}
    log(f"[bench] launch floor: {out}")
    return out


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(inp, seconds):
    """The oracle as it stands, on the host: (a) decode
    every block from its fields, form the f64 weights and multiply, and (b)
    the f64 matvec alone on the decoded weights, each repeated for about a
    quarter of `seconds`, once with the BLAS pool held to one thread and once
    with it on every core this process may use.  numpy runs the decode and the
    weights on one thread either way.  The reported value is (a) on every
    core; the four legs are listed beside it."""
    from threadpoolctl import threadpool_limits
    from oracle import decode as D
    cls, sm, lv = D.fields_from_points(inp.z)           # setup, not timed
    served = inp.M * inp.nb * 16
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    W0 = D.weights64(cls, inp.gain, inp.scale, D.decode_fields(cls, sm, lv))

    def full():
        z = D.decode_fields(cls, sm, lv)
        W = D.weights64(cls, inp.gain, inp.scale, z)
        return D.gemv64(W, inp.x)

    def matvec():
        return D.gemv64(W0, inp.x)

    def timed(fn, threads, budget, warm):
        with threadpool_limits(limits=threads):
            if warm:
                fn()
            n, t0 = 0, time.perf_counter()
            while True:
                fn()
                n += 1
                el = time.perf_counter() - t0
                if el >= budget or n >= 100000:
                    break
        return el / n * 1e6, n

    legs = {}
    for name, fn in (("decode_and_matvec", full), ("matvec_only", matvec)):
        for label, threads in (("1_thread", 1), ("all_cores", cores)):
            us, n = timed(fn, threads, seconds / 4, fn is matvec)
            legs[f"{name}_{label}"] = {"us_per_gemv": round(us, 1), "threads": threads,
                                       "repeats": n, "GBps_served_equiv": round(served / us / 1e3, 4)}
    main = legs["decode_and_matvec_all_cores"]
    return {"value": main["GBps_served_equiv"], "unit": "GB/s", "cores": cores,
            "kind": "oracle",
            "sample": f"full {inp.M}x{inp.K} GEMVs on the host (oracle decode_fields + weights64 + "
                      f"gemv64, f64; BLAS on {cores} threads), {main['repeats']} repeats; "
                      f"GB/s of Planes14 served bytes",
            "us_per_gemv": main["us_per_gemv"], "legs": legs,
            "cpu_model": cpu_model(), "os_cpu_count": os.cpu_count(), "affinity_cores": cores}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; the GEMV shards by "
                          "rows or by K across GPUs (see the design notes) but no multi-GPU "
                          "path is built", "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    import paper_2609_02652_amd as P
    from paper_2609_02652_amd import synth
    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU (torch.cuda.is_available() is False)")
    if args.geometry_sweep:
        print(json.dumps({"geometry_sweep": bench_geometry(args, torch, P, synth)}), flush=True)
        return
    if args.calib_mib:
        n = args.calib_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] copy reference: 5 × {n} bytes read and written")
        del src, dst
    inp, arms, y_arms = build_arms(args, torch, P, synth)
    main_arm = arms["planes14"]
    verified = verify_arms(torch, inp, arms, y_arms)

    # warmup every arm (eager, then its graphs), then the contract's timed
    # region: K Planes14 GEMVs from replica 0, after the replay that evicts
    # them from the Infinity Cache
    k_arm = max(50, args.steps // 4)
    for a in arms.values():
        a.run(args.warmup)
        a.graph(torch, k_arm).replay()
    main_arm.graph(torch, args.steps).replay()
    torch.cuda.synchronize()
    log(f"[bench] warmup done; timing {args.steps} planes14 steps")
    # the K launches one by one behind a lead replay, when the host enqueues
    # them all before the device reaches them; else one graph of K launches
    ms_graph = time_arm(torch, main_arm, args.steps)
    graph_ahead = _LAST_AHEAD[0]
    ms_stream, ahead = time_arm_stream(torch, main_arm, args.steps)
    ms = ms_stream if ahead else ms_graph
    us = ms * 1e3 / args.steps
    gbs = main_arm.served_bytes / (us * 1e-6) / 1e9
    ev_start, ev_len, between = main_arm.evict_plan(args.steps)
    n_rep = len(main_arm.launchers)
    timed = {"launch": "stream, enqueued ahead" if ahead else "graph",
             "events": TimingEvent(torch).kind,
             "us_per_gemv_stream": round(ms_stream * 1e3 / args.steps, 3),
             "stream_enqueued_ahead": ahead,
             "us_per_gemv_graph": round(ms_graph * 1e3 / args.steps, 3),
             "graph_enqueued_ahead": graph_ahead,
             "timed_bytes": args.steps * main_arm.served_bytes,
             "working_set_bytes": n_rep * main_arm.served_bytes,
             "evict_replay": {"first_replica": ev_start, "launches": ev_len,
                              "bytes": ev_len * main_arm.served_bytes},
             "timed_replicas_read_by_evict_replay": ev_len == n_rep,
             "min_bytes_between_reads": between}
    cyc = cycle_us(torch, main_arm)
    timed["whole_cycle"] = {"launches": n_rep, "bytes": n_rep * main_arm.served_bytes,
                            "us_per_gemv": round(cyc, 3),
                            "GBps": round(main_arm.served_bytes / (cyc * 1e-6) / 1e9, 1)}
    clock = shader_clock(torch, main_arm)
    log(f"[bench] timed region {timed}; shader clock {clock}")

    prologue = {f"{inp.M}x{inp.K}": prologue_table(args, torch, P, main_arm)}
    log(f"[bench] prologue modes {prologue}")
    x_main = torch.from_numpy(inp.x).to(main_arm.mats[0].main.device)
    phases = {f"{inp.M}x{inp.K}": phase_table(torch, P, main_arm, x_main, y_arms)}
    log(f"[bench] phases {phases}")

    # layout comparison: arms interleaved in fixed order, rounds, first discarded
    table = arms_table(args, torch, arms, inp)
    table_c4 = None
    if not args.no_arms_c4 and args.config != "c4_8192x8192":
        for a in arms.values():
            a._graphs.clear()
        torch.cuda.synchronize()
        inp4, arms4, y4 = build_arms(args, torch, P, synth, "c4_8192x8192")
        verify_arms(torch, inp4, arms4, y4)
        for a in arms4.values():
            a.run(args.warmup)
        table_c4 = {"workload": f"single GEMV W {inp4.M}x{inp4.K} (Kpad {inp4.Kpad}), every layout "
                                f"of the same codes and both controls",
                    "lane_cols": arms4["planes14"].desc.lane_cols,
                    "arms": arms_table(args, torch, arms4, inp4)}
        prologue[f"{inp4.M}x{inp4.K}"] = prologue_table(args, torch, P, arms4["planes14"])
        log(f"[bench] prologue modes {prologue}")
        x4 = torch.from_numpy(inp4.x).to(y4.device)
        phases[f"{inp4.M}x{inp4.K}"] = phase_table(torch, P, arms4["planes14"], x4, y4)
        log(f"[bench] phases {phases}")
        del arms4, y4
        torch.cuda.empty_cache()

    batch = None
    if not args.no_batch:
        batch = bench_batch(args, torch, P, synth, inp, arms)
    layer = None
    if not args.no_layer:
        for a in arms.values():
            a._graphs.clear()
        torch.cuda.synchronize()
        layer = bench_layer(args, torch, P, synth)
        layer["rotation"] = bench_rotation(args, torch, P, synth)
        layer["rotation_sites"] = bench_rotation_sites(args, torch, P, synth)
    step14b = None
    if not args.no_step14b:
        for a in arms.values():
            a._graphs.clear()
        torch.cuda.synchronize()
        step14b = bench_step14b(args, torch, P, synth)

    large = None
    if not args.no_large:
        for a in arms.values():
            a._graphs.clear()
        torch.cuda.synchronize()
        large = bench_large(args, torch, P, synth)

    batch14b = None
    if args.batch_14b:
        for a in arms.values():
            a._graphs.clear()
        torch.cuda.synchronize()
        batch14b = bench_batch_14b(args, torch, P, synth)

    sweep = None
    if args.sweep:
        for a in arms.values():
            a._graphs.clear()
        torch.cuda.synchronize()
        sweep = bench_sweep(args, torch, P, synth)

    floor = None
    if not args.no_floor:
        for a in arms.values():
            a._graphs.clear()
        torch.cuda.synchronize()
        floor = bench_floor(args, torch, P, synth)
        f = floor["fill_one_element_us"]
        if us > f:
            floor["pct_hbm_peak_above_fill_floor"] = round(
                100 * main_arm.served_bytes / ((us - f) * 1e-6) / 1e9 / HBM_PEAK_GBS, 1)

    cpu = None
    if not args.no_cpu_baseline:
        log(f"[bench] timing the CPU oracle for ~{args.cpu_seconds:.0f}s")
        cpu = cpu_baseline(inp, args.cpu_seconds)

    out = {
        "metric": "Leech GEMV µs + served-weight GB/s (% HBM peak), batch 1, 4.80 bpw",
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms / args.steps, 6),
        "us_per_gemv": round(us, 3),
        "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic: uniform Λ24(12) points, fp16 |N(0,1)|·0.02 block scales, fp16 N(0,1) x",
        "config": {"workload": f"single GEMV W {inp.M}x{inp.K} (Kpad {inp.Kpad}), Planes14 + fp16 "
                               f"block scales, batch 1", "M": inp.M, "K": inp.K, "Kpad": inp.Kpad,
                   "layout": "planes14", "lane_cols": main_arm.desc.lane_cols,
                   "served_bytes_per_gemv": main_arm.served_bytes,
                   "replicas": len(main_arm.launchers),
                   "timed_bytes": timed["timed_bytes"]},
        "timed_region": timed,
        "shader_clock": clock,
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(args.config)},
        "arms": table,
        "arms_c4": table_c4,
        "prologue_modes_us": prologue,
        "phases": phases,
        "verified": verified,
        "batch": batch,
        "layer_8b": layer,
        "step_14b": step14b,
        "large": large,
        "batch_14b": batch14b,
        "sweep": sweep,
        "launch_floor": floor,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
