"""Benchmark of the InfiniPot-V compression pass on one MI355X.

One step = one whole pass (TaR + VaN scores, keep-set selection, in-place
compaction) over every (stream, layer, KV head) slice of a synthetic cache,
through the C ABI's ipv_compress; further steps through ipv_compress_timed
give the per-kernel times. Each step compresses its own replica of the
cache, all resident in HBM before the timed region, so nothing is restored
inside it; a 1 GiB write and read evict the caches before warm-up and before
timing. Prints one JSON line.

  python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--workload 7b-class-28L]
                  [--mode tar_reverse,van_reverse,tar_adjacent,head_shared,uniform_select]
  python bench.py --workload streaming-16x16 --stream   # the whole frame stream: ipv_ckv_step per frame, then ipv_ckv_stream
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import synth  # noqa: E402
from synth import workloads as W  # noqa: E402

METRIC = "compression-pass latency (us) + achieved HBM GB/s (% of peak), 1 MI355X"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCES = os.path.join(ROOT, "paper_2506_15745_amd", "csrc")
PEAK_HBM_GBPS = 8000.0
# the recent-key table runs in one launch with the VaN tiles; the TaR tiles follow
STEP_NAMES = ("table_van", "tar_sweep", "pool", "select", "compact")
# with consecutive-frame TaR the prev-row walks run with the VaN tiles, then the TaR rows
STEP_NAMES_ADJACENT = ("prev_van", "adjacent_tar", "pool", "select", "compact")
MODE_BITS = {"tar_reverse": 1, "van_reverse": 2, "tar_adjacent": 4, "head_shared": 8, "uniform_select": 16}
# the oracle's bits for the same variants (the two sides define them separately)
ORACLE_MODE = {"tar_reverse": "TAR_REVERSE", "van_reverse": "VAN_REVERSE", "tar_adjacent": "TAR_ADJACENT",
               "head_shared": "HEAD_SHARED", "uniform_select": "UNIFORM"}


def parse_mode(text: str) -> int:
    bits = 0
    for name in filter(None, text.split(",")):
        if name not in MODE_BITS:
            raise SystemExit("unknown mode %r (known: %s)" % (name, ", ".join(MODE_BITS)))
        bits |= MODE_BITS[name]
    return bits


class Hip:
    """The few HIP runtime calls the benchmark makes itself (events)."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]

    # Timing events only: recording one skips the system-scope fence (a cache
    # write-back and invalidation that would otherwise land between the passes
    # and kernels being timed); elapsed times are read after a device-wide
    # synchronize.
    DISABLE_SYSTEM_FENCE = 0x20000000  # hipEventDisableSystemFence

    def event(self):
        e = ctypes.c_void_p()
        if self.lib.hipEventCreateWithFlags(ctypes.byref(e), self.DISABLE_SYSTEM_FENCE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")
        return e.value

    def elapsed_ms(self, a, b) -> float:
        ms = ctypes.c_float()
        if self.lib.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value


def pct(xs, q):
    xs = sorted(xs)
    return xs[min(len(xs) - 1, int(round(q * (len(xs) - 1))))]


def make_cache(w: W.Workload):
    sts = [synth.fresh_cache(w.seeds[s], w.layers, w.kv_heads, w.capacity, w.head_dim, w.grid_h, w.grid_w,
                             w.n_tokens, w.dtype, w.rho_specs[s], w.value_sigma) for s in range(w.streams)]
    st = lambda a: np.ascontiguousarray(np.stack([getattr(s, a) for s in sts]))
    return st("K"), st("V"), st("frame_idx"), st("patch_idx")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def parity_record(w, K, V, fr, pa, alpha, mode, got):
    """The oracle's verdict on one GPU pass over the same input bytes (the
    acceptance rule of oracle/compare.py): largest score errors, keep-set
    differences split into near-threshold and unexplained rows, and whether
    the compaction equals the oracle's gather of the GPU's keep set bit for
    bit. got: host copies of the pass's tar, van, keep_idx and compacted K, V,
    frame_idx, patch_idx."""
    import oracle
    from oracle import compare

    om = sum(getattr(oracle, ORACLE_MODE[k]) for k, b in MODE_BITS.items() if mode & b)
    n, C, r = w.n_tokens, w.budget, w.recent_frames
    out = {"slices": int(np.prod(K.shape[:3]))}
    if mode & MODE_BITS["uniform_select"]:
        sel = oracle.select(None, None, fr, n, C, alpha, r, mode=om)
        differ = np.any(got["keep"] != sel.keep_idx, axis=-1)
        out.update({"keep": "bit-exact (frame ids only)", "slices_differing": int(differ.sum()),
                    "unexplained_rows": int((got["keep"] != sel.keep_idx).sum())})
    else:
        tar64 = oracle.tar_scores(K, fr, pa, n, r, w.grid_h, w.grid_w, mode=om)
        van64, _ = oracle.van_scores(V, fr, pa, n, w.grid_h, w.grid_w, w.cv_tau)
        sel = oracle.select(tar64.astype(np.float32), van64.astype(np.float32), fr, n, C, alpha, r, mode=om)
        et, ev = compare.score_errors(got["tar"], tar64, n), compare.score_errors(got["van"], van64, n)
        if mode & MODE_BITS["head_shared"]:
            H = K.shape[2]
            tar64 = np.repeat(tar64.sum(axis=2, keepdims=True), H, axis=2)
            van64 = np.repeat(van64.sum(axis=2, keepdims=True), H, axis=2)
        ks = compare.keep_stats(got["keep"], sel.keep_idx, sel.cut_tar, sel.cut_van, tar64, van64)
        own = oracle.select(np.ascontiguousarray(got["tar"]), np.ascontiguousarray(got["van"]), fr, n, C, alpha, r,
                            mode=om)
        out.update({"tar_max_abs_err": et["max_abs"], "tar_tol_used": round(et["max_tol_frac"], 6),
                    "van_max_abs_err": ev["max_abs"], "van_tol_used": round(ev["max_tol_frac"], 6),
                    "slices_differing": ks["slices_differing"], "mismatched_rows": ks["mismatched_rows"],
                    "near_threshold_rows": ks["near_threshold_rows"], "unexplained_rows": ks["unexplained_rows"],
                    "keep_equals_oracle_on_gpu_scores": bool(np.array_equal(own.keep_idx, got["keep"]))})
    Ko, Vo, fo, po = oracle.compact(K, V, fr, pa, n, np.ascontiguousarray(got["keep"]))
    out["compaction_bit_exact"] = bool(
        np.array_equal(got["K"][..., :C, :].view(np.uint8), Ko[..., :C, :].view(np.uint8))
        and np.array_equal(got["V"][..., :C, :].view(np.uint8), Vo[..., :C, :].view(np.uint8))
        and np.array_equal(got["fr"][..., :C], fo[..., :C]) and np.array_equal(got["pa"][..., :C], po[..., :C]))
    return out


def cpu_baseline(w, K, V, fr, pa, alpha, seconds, mode=0):
    """The CPU oracle on the same workload, on this host's cores; for the tiny
    and 7B-class caches also on one thread."""
    import oracle

    def passes(budget_s, max_runs):
        # whole passes on fresh copies of the cache (the pass is in place) until
        # budget_s of oracle time have been spent; the copies are not timed
        times = []
        Kc, Vc, fc, pc = K.copy(), V.copy(), fr.copy(), pa.copy()
        while not times or (sum(times) < budget_s and len(times) < max_runs):
            for dst, src in ((Kc, K), (Vc, V), (fc, fr), (pc, pa)):
                np.copyto(dst, src)
            t = time.perf_counter()
            oracle.compress_inplace(Kc, Vc, fc, pc, w.n_tokens, w.budget, alpha, w.recent_frames, w.grid_h, w.grid_w,
                                    w.cv_tau, mode)
            times.append(time.perf_counter() - t)
        return times

    threads = oracle.max_threads()
    times = passes(seconds, 1000)
    t = statistics.median(times)
    out = {"value": round(w.algorithmic_bytes() / t / 1e9, 3), "unit": "GB/s", "cores": threads,
           "kind": "oracle", "latency_us": round(t * 1e6, 1), "cpu_model": cpu_model(), "nproc": os.cpu_count(),
           "sample": "whole %s pass, median of %d runs (%.1f s of oracle time)" % (w.name, len(times), sum(times))}
    if w.name in (W.TINY.name, W.SEVEN_B.name):
        oracle.set_threads(1)
        try:
            one = passes(3.0, 3)
        finally:
            oracle.set_threads(threads)
        t1 = statistics.median(one)
        out["single_thread"] = {"value": round(w.algorithmic_bytes() / t1 / 1e9, 3), "unit": "GB/s",
                                "latency_us": round(t1 * 1e6, 1), "runs": len(one)}
    return out


def code_only(src: str) -> str:
    """C++ source without its comments and with whitespace runs folded: what
    the compiler sees (string and character literals kept as they are)."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash() -> str:
    """Hash of the HIP sources' code (comments and layout ignored): counter
    readings are valid only for this code."""
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(KERNEL_SOURCES)):
        if not name.endswith((".hip", ".hpp", ".h")):
            continue
        with open(os.path.join(KERNEL_SOURCES, name), encoding="utf-8") as f:
            h.update(name.encode() + b"\0" + code_only(f.read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(step: str):
    """HBM bytes per launch of a step's kernel, from the committed counter
    readings (rocprofv3 FETCH_SIZE/WRITE_SIZE, scaled by the copy-kernel
    calibration), or None when they were taken on other kernel sources."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_hash") != kernel_source_hash():
        return None
    e = t.get("kernels", {}).get(step)
    return None if e is None else int(e["fetch_bytes"] + e["write_bytes"])


def summarize(paths):
    """Text summary of rocprofv3 result databases (kernel trace or counters)."""
    import sqlite3
    for path in paths:
        con = sqlite3.connect(path)
        print("# %s" % os.path.basename(path))
        try:
            rows = con.execute("select counter_name, kernel_name, count(*), avg(value) from counters_collection "
                               "group by counter_name, kernel_name order by counter_name, kernel_name").fetchall()
        except sqlite3.Error:
            rows = []
        if rows:
            print("%-12s %8s %14s  %s" % ("counter", "calls", "avg per call", "kernel"))
            for c, k, n, v in rows:
                print("%-12s %8d %14.1f  %s" % (c, n, v, k[:110]))
            continue
        rows = con.execute("select name, count(*), avg(duration), min(duration), max(duration), sum(duration) "
                           "from kernels group by name order by sum(duration) desc").fetchall()
        total = sum(r[5] for r in rows) or 1
        print("%8s %10s %10s %10s %7s  %s" % ("calls", "avg_us", "min_us", "max_us", "time%", "kernel"))
        for name, n, avg, mn, mx, tot in rows:
            print("%8d %10.2f %10.2f %10.2f %6.1f%%  %s" % (n, avg / 1e3, mn / 1e3, mx / 1e3, 100 * tot / total,
                                                          name[:110]))


STEP_KERNELS = {"table_van": "k_table_van<", "tar_sweep": "k_score_sweep<", "select": "k_select<",
                "compact": "k_compact<"}


def write_traffic(fetch_db, write_db, cal_fetch_db, cal_write_db):
    """profiles/traffic.json from two counter runs of the benchmark and two of
    the copy probe: per step kernel, HBM bytes per launch = FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch) times the factor that maps the copy
    probe's counters onto its known size."""
    import sqlite3

    def per_kernel(path, counter):
        con = sqlite3.connect(path)
        rows = con.execute("select kernel_name, avg(value) from counters_collection where counter_name = ? "
                           "group by kernel_name", (counter,)).fetchall()
        return {k: v for k, v in rows}

    copy_kib = (360 << 20) / 1024
    cal = {}
    for counter, db in (("FETCH_SIZE", cal_fetch_db), ("WRITE_SIZE", cal_write_db)):
        copies = [v for k, v in per_kernel(db, counter).items() if "copyBuffer" in k]
        cal[counter] = copy_kib / max(copies)
    fetch, write = per_kernel(fetch_db, "FETCH_SIZE"), per_kernel(write_db, "WRITE_SIZE")
    out = {"source_hash": kernel_source_hash(), "calibration": cal, "kernels": {}}
    for step, pat in STEP_KERNELS.items():
        f = [v for k, v in fetch.items() if pat in k]
        w_ = [v for k, v in write.items() if pat in k]
        if f and w_:
            out["kernels"][step] = {"fetch_bytes": int(f[0] * cal["FETCH_SIZE"] * 1024),
                                    "write_bytes": int(w_[0] * cal["WRITE_SIZE"] * 1024)}
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(out, fh, indent=1)
    print(json.dumps(out))


def copy_probe():
    """A plain device-to-device copy of 360 MiB, three times: the known-size
    reference for scaling the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    src = torch.ones((360 << 20) // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": src.numel() * 4, "copies": 3}))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=W.SEVEN_B.name)
    ap.add_argument("--alpha", type=float, default=None)
    ap.add_argument("--mode", default="", help="comma-separated variant modes (default: the method as published)")
    ap.add_argument("--stream", action="store_true",
                    help="streaming workloads: time whole frame streams through ipv_ckv_step (steps = streams)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true", help="only run the counter-calibration copy")
    ap.add_argument("--summarize", nargs="+", metavar="DB", help="print summaries of rocprofv3 result databases")
    ap.add_argument("--traffic", nargs=4, metavar=("FETCH_DB", "WRITE_DB", "CAL_FETCH_DB", "CAL_WRITE_DB"),
                    help="write profiles/traffic.json from counter runs")
    args = ap.parse_args()
    if args.summarize:
        summarize(args.summarize)
        return
    if args.traffic:
        write_traffic(*args.traffic)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the pass shards by (stream, layer, KV head) with no communication, "
              "so only --gpus 1 is supported", file=sys.stderr)
        sys.exit(2)

    if args.copy_probe:
        copy_probe()
        return

    import torch
    from paper_2506_15745_amd import ipv

    w = W.BY_NAME[args.workload]
    alpha = w.alphas[0] if args.alpha is None else args.alpha
    mode = parse_mode(args.mode)
    if args.stream:
        stream_main(args, w, alpha, mode)
        return
    names = STEP_NAMES_ADJACENT if mode & MODE_BITS["tar_adjacent"] else STEP_NAMES
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    hip = Hip()

    K, V, fr, pa = make_cache(w)
    kind = torch.bfloat16 if w.dtype == synth.BF16 else torch.float32
    to_dev = lambda a, bf=False: (torch.from_numpy(a).view(kind) if bf else torch.from_numpy(a)).to(dev)
    pristine = (to_dev(K, True), to_dev(V, True), to_dev(fr), to_dev(pa))
    # replicas: warm-up, the timed steps, then the per-kernel (event) steps
    ev_steps = min(args.steps, 10)
    reps = args.warmup + args.steps + ev_steps
    replicas = [tuple(t.clone() for t in pristine) for _ in range(reps)]
    comp = ipv.Compressor(pristine[0], w.grid_h, w.grid_w, w.budget)
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)  # 1 GiB

    def evict(v):
        # a write then a read of 1 GiB: caches end up holding clean flush data,
        # so a timed pass neither hits cached cache rows nor pays for writing
        # back dirty lines left by earlier work
        flush.fill_(v)
        flush.sum()

    # copy ceiling: a plain device-to-device copy of the K and V bytes
    kv_bytes = 2 * pristine[0].numel() * pristine[0].element_size()
    src = torch.empty(kv_bytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    copy_gbps = 2 * kv_bytes * 10 / (time.perf_counter() - t) / 1e9
    del src, dst

    events = [[hip.event() for _ in range(6)] for _ in range(reps)]
    ev_structs = [ipv.Events(*e) for e in events]

    def step(i, timed_kernels=False):
        Kd, Vd, fd, pd = replicas[i]
        if timed_kernels:
            ipv.ipv_compress_timed(Kd, Vd, fd, pd, w.n_tokens, w.budget, alpha, w.recent_frames, w.cv_tau,
                                   comp.tar, comp.van, comp.keep_idx, comp.ws, w.grid_h, w.grid_w, ev_structs[i],
                                   mode=mode)
        else:
            ipv.ipv_compress(Kd, Vd, fd, pd, w.n_tokens, w.budget, alpha, w.recent_frames, w.cv_tau, comp.tar,
                             comp.van, comp.keep_idx, comp.ws, w.grid_h, w.grid_w, mode=mode)

    evict(1.0)
    for i in range(args.warmup):
        step(i)
    # an event at every pass boundary of the timed loop: pass j's latency is the
    # time from its start to the next pass's start (or the end), so the
    # latencies add up to the loop's device time
    record = hip.lib.hipEventRecord
    record.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    bounds = [hip.event() for _ in range(args.steps + 1)]
    cur = torch.cuda.current_stream().cuda_stream
    evict(2.0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for j, i in enumerate(range(args.warmup, args.warmup + args.steps)):
        record(bounds[j], cur)
        step(i)
    record(bounds[args.steps], cur)
    enqueue = time.perf_counter() - t0  # host time to enqueue the timed passes
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    pass_us = [hip.elapsed_ms(bounds[j], bounds[j + 1]) * 1e3 for j in range(args.steps)]
    # per-kernel breakdown on further replicas, with events between the kernels
    evict(3.0)
    for i in range(args.warmup + args.steps, reps):
        step(i, timed_kernels=True)
    torch.cuda.synchronize()

    timed = range(args.warmup + args.steps, reps)
    step_us = {name: statistics.mean(hip.elapsed_ms(events[i][k], events[i][k + 1]) * 1e3 for i in timed)
               for k, name in enumerate(names)}
    # warm passes: each replica restored from the pristine cache right before
    # its pass (as when the model has just written the cache), no eviction;
    # two events around each pass, the restores outside them
    warm_ev = [(hip.event(), hip.event()) for _ in timed]
    for (a, b), i in zip(warm_ev, timed):
        for dst, src in zip(replicas[i], pristine):
            dst.copy_(src)
        record(a, cur)
        step(i)
        record(b, cur)
    torch.cuda.synchronize()
    warm_us = [hip.elapsed_ms(a, b) * 1e3 for a, b in warm_ev]
    errors = comp.device_errors()
    uniform = bool(mode & MODE_BITS["uniform_select"])
    if w.cv_tau is None or uniform:
        del step_us["pool"]  # no pooling kernel runs: its events are back to back
    if uniform:  # frame ids decide: no score kernels run
        for k in names[:2]:
            del step_us[k]

    ms_per_step = wall / args.steps * 1e3
    algo = w.algorithmic_bytes()
    if uniform:  # no scores read: only the compaction's read and write of the kept rows
        algo = w.streams * w.layers * w.kv_heads * w.head_dim * w.elem_bytes * 4 * w.budget
    value = algo / (ms_per_step * 1e-3) / 1e9
    B, L, H = w.streams, w.layers, w.kv_heads
    row = w.head_dim * w.elem_bytes
    n_recent = min(w.n_tokens, w.recent_frames * w.p)
    if w.n_tokens % w.p:
        n_recent = (w.recent_frames - 1) * w.p + w.n_tokens % w.p
    slices = B * L * H
    if uniform:
        algo_by_step = {}
    elif mode & MODE_BITS["tar_adjacent"]:
        # every V row beside the walks (which read 8 B of metadata per row); then the past K rows
        algo_by_step = {"prev_van": slices * w.n_tokens * (row + 8),
                        "adjacent_tar": slices * (w.n_tokens - n_recent) * row}
    else:
        # recent K rows for the table and every V row; then the past K rows
        algo_by_step = {"table_van": slices * (w.n_tokens + n_recent) * row,
                        "tar_sweep": slices * (w.n_tokens - n_recent) * row}
    algo_by_step["compact"] = slices * 4 * w.budget * row
    dom = max(algo_by_step, key=lambda k: step_us[k])
    achieved = algo_by_step[dom] / (step_us[dom] * 1e-6) / 1e9

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == synth.BF16 else "f32",
        "data": "synthetic (seeded AR(1) keys, log-normal-scaled values)",
        "config": {"workload": w.name, "streams": B, "layers": L, "kv_heads": H, "head_dim": w.head_dim,
                   "tokens_per_frame": w.p, "n_tokens": w.n_tokens, "budget": w.budget,
                   "recent_frames": w.recent_frames, "alpha": alpha, "parallelism": "single GPU",
                   **({"mode": args.mode} if mode else {})},
        "latency_us": {"wall_mean": round(ms_per_step * 1e3, 2), "events_mean": round(statistics.mean(pass_us), 2),
                       "p50": round(pct(pass_us, 0.5), 2), "p99": round(pct(pass_us, 0.99), 2),
                       "source": "events at the timed loop's pass boundaries",
                       "warm_mean": round(statistics.mean(warm_us), 2), "warm_p50": round(pct(warm_us, 0.5), 2),
                       "warm_source": "events around passes on caches restored right before them, no eviction",
                       "host_enqueue_per_pass": round(enqueue / args.steps * 1e6, 2)},
        "pct_of_peak_hbm": round(100 * value / PEAK_HBM_GBPS, 2),
        "tokens_per_s": round(B * w.n_tokens / (ms_per_step * 1e-3), 1),
        "rows_per_s": round(B * L * H * w.n_tokens / (ms_per_step * 1e-3), 1),
        "algorithmic_bytes": algo,
        "step_us_mean": {k: round(v, 2) for k, v in step_us.items()},
        "step_GBps": {k: round(v / (step_us[k] * 1e-6) / 1e9, 1) for k, v in algo_by_step.items()},
        "copy_ceiling_GBps": round(copy_gbps, 1),
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "algorithmic_bytes": algo_by_step[dom], "traffic": measured_traffic(dom)},
        "device_errors": errors,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, K, V, fr, pa, alpha, args.cpu_seconds, mode)
        # the last replica's pass (same input bytes as every pass) against the oracle
        Kd, Vd, fd, pd = replicas[reps - 1]
        host = lambda t: (t.view(torch.int16).cpu().numpy().view(np.uint16) if t.dtype == torch.bfloat16
                          else t.cpu().numpy())
        got = {"tar": comp.tar.cpu().numpy(), "van": comp.van.cpu().numpy(), "keep": comp.keep_idx.cpu().numpy(),
               "K": host(Kd), "V": host(Vd), "fr": fd.cpu().numpy(), "pa": pd.cpu().numpy()}
        out["cpu_baseline"]["parity"] = parity_record(w, K, V, fr, pa, alpha, mode, got)
    print(json.dumps(out), flush=True)


def stream_main(args, w, alpha, mode):
    """The workload's whole frame stream, one frame per ipv_ckv_step (append,
    and the pass whenever a stream reaches the cap). All frames are resident
    in HBM before timing; each timed step is one whole stream from an empty
    cache; events bracket every step that runs the pass."""
    import torch
    from paper_2506_15745_amd import ipv

    if not w.stream_frames:
        raise SystemExit("--stream needs a streaming workload")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    hip = Hip()
    p, F, L, H, D = w.p, w.stream_frames, w.layers, w.kv_heads, w.head_dim
    kind = torch.bfloat16 if w.dtype == synth.BF16 else torch.float32
    st = synth.Stream(w.seeds[0], L, H, F * p, D, w.grid_h, w.grid_w, w.dtype, w.rho_specs[0], tuple(w.value_sigma))
    st.append(F)

    def frames_of(a):  # [L, H, F*p, D] host -> [F, 1, L, H, p, D] device, frame-major
        t = torch.from_numpy(a)
        t = (t.view(kind) if kind == torch.bfloat16 else t).to(dev)
        return t.view(L, H, F, p, D).permute(2, 0, 1, 3, 4).contiguous().unsqueeze(1)

    Kf, Vf = frames_of(st.K), frames_of(st.V)
    del st
    cap, C = w.n_tokens, w.budget
    S = cap + p
    Kd = torch.zeros((1, L, H, S, D), dtype=kind, device=dev)
    Vd = torch.zeros_like(Kd)
    fd = torch.full((1, L, H, S), -1, dtype=torch.int32, device=dev)
    pd = torch.full_like(fd, -1)
    comp = ipv.Compressor(Kd, w.grid_h, w.grid_w, C)
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    # which steps run the pass (the trigger is a host-side count)
    fires, n = [], 0
    for f in range(F):
        n += p
        fires.append(n >= cap)
        n = C if n >= cap else n
    passes = sum(fires)
    ev = [[(hip.event(), hip.event()) for _ in range(passes)] for _ in range(args.steps)]
    stream_ev = [(hip.event(), hip.event()) for _ in range(args.steps)]
    record = hip.lib.hipEventRecord
    record.argtypes = [ctypes.c_void_p, ctypes.c_void_p]

    def one_stream(events=None, bracket=None):
        n = 0
        k = 0
        cur = torch.cuda.current_stream().cuda_stream
        if bracket:
            record(bracket[0], cur)
        for f in range(F):
            if events and fires[f]:
                record(events[k][0], cur)
            n, fired = ipv.ipv_ckv_step(Kd, Vd, fd, pd, n, Kf[f], Vf[f], f, 0, cap, C, alpha, w.recent_frames,
                                        w.cv_tau, comp.tar, comp.van, comp.keep_idx, comp.ws, w.grid_h, w.grid_w,
                                        mode=mode)
            if events and fired:
                record(events[k][1], cur)
                k += 1
        if bracket:
            record(bracket[1], cur)

    flush.fill_(1.0)
    flush.sum()
    for _ in range(args.warmup):
        one_stream()
    torch.cuda.synchronize()
    flush.fill_(2.0)
    flush.sum()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        one_stream(ev[i], stream_ev[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # the same streams through the library's own loop: one call per stream
    native_ev = [(hip.event(), hip.event()) for _ in range(args.steps)]
    native_passes = set()
    for i in range(-1, args.steps):
        cur = torch.cuda.current_stream().cuda_stream
        if i >= 0:
            record(native_ev[i][0], cur)
        n_end, fired = ipv.ipv_ckv_stream(Kd, Vd, fd, pd, 0, Kf, Vf, 0, cap, C, alpha, w.recent_frames, w.cv_tau,
                                          comp.tar, comp.van, comp.keep_idx, comp.ws, w.grid_h, w.grid_w, mode=mode)
        if i >= 0:
            record(native_ev[i][1], cur)
        native_passes.add(fired)
    torch.cuda.synchronize()
    if native_passes != {passes}:
        raise SystemExit("ipv_ckv_stream ran %s passes per stream, expected %d" % (native_passes, passes))
    native_ms = statistics.mean(hip.elapsed_ms(a, b) for a, b in native_ev)
    errors = comp.device_errors()
    pass_us = [hip.elapsed_ms(a, b) * 1e3 for run in ev for a, b in run]
    stream_ms = [hip.elapsed_ms(a, b) for a, b in stream_ev]
    pass_mean = statistics.mean(pass_us)
    algo = w.algorithmic_bytes()
    value = algo / (pass_mean * 1e-6) / 1e9
    stream_mean = statistics.mean(stream_ms)
    append_us = (stream_mean * 1e3 - sum(pass_us) / args.steps) / (F - passes)
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == synth.BF16 else "f32",
        "data": "synthetic (seeded AR(1) keys, log-normal-scaled values)",
        "config": {"workload": w.name, "streams": 1, "layers": L, "kv_heads": H, "head_dim": D,
                   "tokens_per_frame": p, "frames": F, "mem_cap": cap, "budget": C,
                   "recent_frames": w.recent_frames, "alpha": alpha, "parallelism": "single GPU",
                   "step": "one whole stream through ipv_ckv_step, one call per frame", **({"mode": args.mode} if mode else {})},
        "latency_us": {"pass_mean": round(pass_mean, 2), "pass_p50": round(pct(pass_us, 0.5), 2),
                       "pass_p99": round(pct(pass_us, 0.99), 2)},
        "pct_of_peak_hbm": round(100 * value / PEAK_HBM_GBPS, 2),
        "stream": {"passes_per_stream": passes, "stream_ms_mean": round(stream_mean, 3),
                   "compression_ms_per_stream": round(sum(pass_us) / args.steps / 1e3, 3),
                   "append_us_mean": round(append_us, 2),
                   "tokens_per_s": round(F * p / (stream_mean * 1e-3), 1),
                   "ipv_ckv_stream_ms_mean": round(native_ms, 3),
                   "ipv_ckv_stream_tokens_per_s": round(F * p / (native_ms * 1e-3), 1)},
        "algorithmic_bytes_per_pass": algo,
        "roofline": {"bound": "hbm", "kernel": "whole pass (ipv_ckv_step that fires)", "achieved": round(value, 1),
                     "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": round(value / PEAK_HBM_GBPS, 4),
                     "algorithmic_bytes": algo, "traffic": None},
        "device_errors": errors,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
