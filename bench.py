#!/usr/bin/env python3
"""Benchmark of the replay hot path on one MI355X.

One step = prioritized selection (prefix scan, B draws, importance-sampling
weights) + collection of the B selected L-step windows of every column +
priority-update scatter, on a synthetic table resident in HBM (default
workload: MAT-shaped, N=500000 trajectories x T=200 steps, B=8192, L=32).
Inputs are generated and inserted before the timed region.

Prints one JSON line.  `value` is trajectory-steps gathered per second over
the whole step; `roofline` rates the gather kernel (the dominant kernel)
against its bandwidth peak from HIP events around each gather launch in the
timed region; `cpu_baseline` is the plain CPU oracle timed on a bounded
sample of the same workload.

  python bench.py [--steps K] [--warmup W] [--workload mat|gato-host|dt|dt-full|tiny|select-stress|topk|...]
  python bench.py --workload mat-insert   # insertion through the index manager (own metric)
  python bench.py --workload shard-select # one GPU's share of selection over 8 shards (own metric)
  python bench.py --calibrate     # plain copy kernel of known size, for counter scaling
  python bench.py --ceilings      # HBM read / write / copy rates of plain kernels
"""
import argparse
import dataclasses
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "trajectory-steps gathered/sec + gather GB/s as % of HBM / host-link peak"
HBM_PEAK_GBS = 8000.0           # MI355X HBM3E
HOST_LINK_PEAK_GBS = 63.0       # PCIe Gen5 x16 per direction: 32 GT/s * 16 * 128/130 / 8
GATHER_SRC = os.path.join(ROOT, "paper_2310_05205_amd", "csrc", "collect.hip")
PIPELINE_MIN_BATCH = 128 << 20  # batch bytes from which steps overlap select/update with the gather


class HipEvents:
    """HIP events for timing, created with hipEventDisableSystemFence: recording
    one does not write back and invalidate caches, so bracketing a kernel
    neither stalls the stream nor adds that flush to the measured interval."""

    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        h = ctypes.CDLL("libamdhip64.so.7")  # the runtime torch and libgear.so share
        vp = ctypes.c_void_p
        h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp), ctypes.c_uint]
        h.hipEventRecord.argtypes = [vp, vp]
        h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
        h.hipEventDestroy.argtypes = [vp]
        h.hipStreamWaitEvent.argtypes = [vp, vp, ctypes.c_uint]
        self.h = h
        self.made = []

    def _ok(self, rc, what):
        if rc != 0:
            raise RuntimeError("%s failed (%d)" % (what, rc))

    def create(self):
        e = ctypes.c_void_p()
        self._ok(self.h.hipEventCreateWithFlags(ctypes.byref(e), self.DISABLE_SYSTEM_FENCE), "hipEventCreateWithFlags")
        self.made.append(e)
        return e

    def record(self, e, stream_handle):
        self._ok(self.h.hipEventRecord(e, ctypes.c_void_p(stream_handle)), "hipEventRecord")

    def wait(self, stream_handle, e):
        """Work enqueued on the stream after this waits for event e."""
        self._ok(self.h.hipStreamWaitEvent(ctypes.c_void_p(stream_handle), e, 0), "hipStreamWaitEvent")

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        self._ok(self.h.hipEventElapsedTime(ctypes.byref(ms), a, b), "hipEventElapsedTime")
        return ms.value

    def close(self):
        for e in self.made:
            self.h.hipEventDestroy(e)
        self.made = []


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="mat",
                    choices=["mat", "gato-host", "dt", "dt-full", "tiny", "select-stress", "topk", "mat-insert",
                             "shard-select"])
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing (profiling runs)")
    ap.add_argument("--serial", action="store_true",
                    help="issue every step in order on one stream (default for batches under 128 MiB)")
    ap.add_argument("--pipeline", action="store_true",
                    help="overlap select/update with the gather on two streams whatever the batch size")
    ap.add_argument("--graph", action="store_true",
                    help="capture the timed steps into one HIP graph and replay it (steps in order on one stream; "
                         "only workloads whose calls replay correctly from a capture)")
    ap.add_argument("--strategy", choices=["fifo", "lifo", "uniform", "prioritized", "topk"],
                    help="select with this one of the workload's strategies instead of its first")
    ap.add_argument("--fused", action="store_true",
                    help="FIFO, LIFO and uniform workloads: each step is one gear_select_collect launch "
                         "(selection computed inside the gather)")
    ap.add_argument("--group", type=int, default=4,
                    help="steps per cross-stream handshake when select/update overlap the gather")
    ap.add_argument("--legs", default="all", choices=["all", "headline"],
                    help="default MAT run: also measure the host-link, whole-trajectory and selection legs")
    ap.add_argument("--incremental", action="store_true",
                    help="keep the selection sum tree current across updates (no rescan per step)")
    ap.add_argument("--global-min", action="store_true",
                    help="IS weights normalised over the whole table (GEAR_OPT_IS_GLOBAL_MIN)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target oracle time for the CPU baseline")
    ap.add_argument("--calibrate", action="store_true", help="run a plain copy kernel of known size and exit")
    ap.add_argument("--ceilings", action="store_true", help="measure plain read/write/copy HBM rates and exit")
    args = ap.parse_args()
    if args.group < 1:
        ap.error("--group must be at least 1")
    return args


def workload(name):
    from gen import configs
    return {"mat": configs.MAT, "gato-host": configs.GATO_HOST, "dt": configs.DT, "dt-full": configs.DT_FULL,
            "tiny": configs.TINY,
            "select-stress": configs.SELECT_STRESS, "topk": configs.TOPK_STRESS}[name]


def calibrate():
    """A plain elementwise copy (bitwise_not of int64) of 2 GiB: reads and
    writes exactly 2 GiB per launch, for scaling FETCH_SIZE/WRITE_SIZE."""
    import torch
    n = (2 << 30) // 8
    a = torch.zeros(n, dtype=torch.int64, device="cuda")
    b = torch.empty_like(a)
    for _ in range(5):
        torch.bitwise_not(a, out=b)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate": "bitwise_not int64", "bytes_read_per_launch": n * 8,
                      "bytes_written_per_launch": n * 8, "launches": 5}))


def ceilings():
    """HBM rates of plain torch kernels on 8 GiB buffers (no gather, no
    replay): a read-only reduction, a fill, and an elementwise copy.  They
    bound what a kernel that reads and writes HBM can reach on this device.
    Then plain copies of the gather's own sizes, which show what launch,
    ramp and drain cost at those sizes."""
    import torch
    n = (8 << 30) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    sh = torch.cuda.current_stream().cuda_stream
    hev = HipEvents()
    out = {}
    tests = [("read (sum)", lambda: torch.sum(a), n * 4),
             ("write (fill)", lambda: b.fill_(2.0), n * 4),
             ("copy (neg)", lambda: torch.neg(a, out=b), 2 * n * 4)]
    for name, fn, nbytes in tests:
        for _ in range(3):
            fn()
        e0, e1 = hev.create(), hev.create()
        hev.record(e0, sh)
        for _ in range(10):
            fn()
        hev.record(e1, sh)
        torch.cuda.synchronize()
        ms = hev.elapsed_ms(e0, e1) / 10
        out[name] = {"GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1), "ms": round(ms, 4),
                     "frac_of_8TB/s": round(nbytes / (ms * 1e-3) / 8e12, 4)}
    # Copies of the gather's own sizes, from and to a fresh 1 GiB region each
    # time (eight regions, more than the 256 MB last-level cache holds), as
    # the gather reads windows no earlier step touched: the DT-shaped whole
    # trajectories (51.2 MB each way) and the MAT windows (277.9 MB each way).
    region = (1 << 30) // 4
    sized = {}
    for label, nbytes in (("dt-full 51.2 MB", 51_200_000), ("mat 277.9 MB", 277_872_640)):
        m = nbytes // 4
        for kind in ("runtime copy", "elementwise"):
            def run(k, kind=kind, m=m):
                src = a[(k % 8) * region:(k % 8) * region + m]
                dst = b[((k + 3) % 8) * region:((k + 3) % 8) * region + m]
                if kind == "runtime copy":
                    dst.copy_(src)
                else:
                    torch.neg(src, out=dst)
            for k in range(3):
                run(k)
            e0, e1 = hev.create(), hev.create()
            hev.record(e0, sh)
            reps = 16
            for k in range(reps):
                run(k)
            hev.record(e1, sh)
            torch.cuda.synchronize()
            ms = hev.elapsed_ms(e0, e1) / reps
            sized["%s, %s" % (label, kind)] = {"GB/s": round(2 * nbytes / (ms * 1e-3) / 1e9, 1), "us": round(ms * 1e3, 2),
                                               "frac_of_8TB/s": round(2 * nbytes / (ms * 1e-3) / 8e12, 4)}
    hev.close()
    print(json.dumps({"ceilings": out, "bytes_per_buffer": n * 4, "gather_sized_copies": sized}))


def source_sha(path):
    """Hash of a source's code: line comments and blank lines left out, so
    that a comment edit does not invalidate counters taken on the same code."""
    with open(path) as f:
        code = [l.split("//", 1)[0].rstrip() for l in f]
    return hashlib.sha256("\n".join(l for l in code if l).encode()).hexdigest()


def profiled_traffic(kernel_key, workload_name):
    """HBM bytes per gather launch from the committed counter summary, if it
    was taken on the current gather source; else None."""
    path = os.path.join(ROOT, "profiles", "gather_%s_counters.txt" % workload_name)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("source_sha256") != source_sha(GATHER_SRC) or vals.get("kernel") != kernel_key:
        return None
    try:
        return float(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def host_link_extras(t, w, idx, start, outs, dev):
    """Context for a gather from a pinned host table.

    link_h2d_copy_gbs: a plain pinned-to-device copy of 1 GiB
    (hipMemcpyAsync, through torch), the host link's empirical ceiling.
    cpu_staged: the CPU-driven transfer that zero-copy replaces (Sec. 4.4):
    host threads copy the same B windows out of the pinned table into a pinned
    staging buffer, then one host-to-device copy per column.  Its batch is
    compared byte for byte with the zero-copy gather's (`outs`, produced from
    the same `idx` and `start`)."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np
    import torch

    s = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    nb = 1 << 30
    src = torch.empty(nb, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(nb, dtype=torch.uint8, device=dev)
    for _ in range(2):
        dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    reps = 5
    e0.record(s)
    for _ in range(reps):
        dst.copy_(src, non_blocking=True)
    e1.record(s)
    torch.cuda.synchronize()
    h2d_gbs = nb * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst

    B, L = w.B, w.L
    hidx = idx.cpu().numpy()
    hstart = start.cpu().numpy()
    ncols = len(w.elem_bytes)
    views = [t.column_view(c) for c in range(ncols)]
    stage = [torch.empty(B * L * e, dtype=torch.uint8, pin_memory=True) for e in w.elem_bytes]
    stage_np = [x.numpy().reshape(B, L * e) for x, e in zip(stage, w.elem_bytes)]
    dev_out = [torch.empty(B * L * e, dtype=torch.uint8, device=dev) for e in w.elem_bytes]
    threads = max(1, min(16, os.cpu_count() or 1))

    def gather(lo, hi):
        for c, e in enumerate(w.elem_bytes):
            v, sn = views[c], stage_np[c]
            for b in range(lo, hi):
                i, s0 = int(hidx[b]), int(hstart[b])
                sn[b] = v[i, s0 * e:(s0 + L) * e]

    ranges = [(B * k // threads, B * (k + 1) // threads) for k in range(threads)]
    times = []
    with ThreadPoolExecutor(threads) as ex:
        for _ in range(3):
            t0 = time.perf_counter()
            list(ex.map(lambda r: gather(*r), ranges))
            for c in range(ncols):
                dev_out[c].copy_(stage[c], non_blocking=True)
            torch.cuda.synchronize()
            times.append(time.perf_counter() - t0)
    same = all(bool(torch.equal(dev_out[c], outs[c])) for c in range(ncols))
    ms = float(np.median(times)) * 1e3
    batch_bytes = B * L * sum(w.elem_bytes)
    return {"link_h2d_copy_gbs": round(h2d_gbs, 1),
            "cpu_staged": {"ms_per_batch": round(ms, 3), "gbs": round(batch_bytes / (ms * 1e-3) / 1e9, 2),
                           "threads": threads, "matches_zero_copy": same,
                           "note": "host threads gather the windows into pinned staging, then one H2D copy "
                                   "per column; median of 3 batches"}}


def torch_context(t, w, dev):
    """The same selection done with PyTorch's own GPU operators, on a copy of
    the table's priorities, timed with events over 20 calls: torch.multinomial
    (weighted draws with replacement, fp32 weights) for prioritized
    selection, torch.topk for TopK.  Context only: neither reproduces the
    exact draws or tie order, and neither is the baseline."""
    import torch

    p = torch.from_numpy(t.priorities().astype("int64")).to(dev)
    strat = w.strategies[0]
    if strat == 3:
        x = p.to(torch.float32)
        fn = lambda: torch.multinomial(x, w.B, replacement=True)
        name = "torch_multinomial_us"
    elif strat == 4:
        fn = lambda: torch.topk(p, w.B)
        name = "torch_topk_us"
    else:
        return None
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(20):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return {name: round(e0.elapsed_time(e1) * 1e3 / 20, 2),
            "note": "PyTorch operator on the same priorities, for scale; the GPU select is stages_ms.select"}


def cpu_baseline(w, target_s, global_min=False):
    """The oracle, single-threaded, on a bounded sample: repeated steps of
    the same workload (select over all N priorities, IS weights, collection
    of the B selected windows, update), collecting from a compact host table
    that holds only the trajectories the first selection picks."""
    import numpy as np

    import gen
    import oracle

    ring = oracle.Store([], w.N, w.T)      # the priority array after all of w's insertions
    ring.insert([], gen.insert_priorities(w.prio, w.seed, 0, w.n_insert))
    p, next_seq = ring.priority, ring.next_seq
    seed = gen.select_seed(w.seed, 0)
    strat = w.strategies[0]
    updates = strat in (oracle.PRIORITIZED, oracle.TOPK)  # as in the GPU step
    st, idx, start, _ = oracle.select(strat, p, next_seq, w.T, w.B, w.L, seed, w.beta, True, global_min=global_min)
    assert st == oracle.OK
    ks = gen.slot_insertion(idx, next_seq, w.N)
    rows = [gen.fill_rows_list_cpu(c, ci, w.seed, w.T, ks) for ci, c in enumerate(w.columns)]
    local = np.arange(w.B, dtype=np.int64)
    newp = gen.update_priorities(w.prio, w.seed, 0, w.B)
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), model)
    except OSError:
        pass
    # The timed loop runs on one core of those this thread may use.
    allowed = sorted(os.sched_getaffinity(0))
    core = allowed[-1]
    os.sched_setaffinity(0, {core})
    try:
        reps = 0
        t0 = time.perf_counter()
        while True:
            st, oidx, ostart, ow = oracle.select(strat, p, next_seq, w.T, w.B, w.L, seed, w.beta, True,
                                                 global_min=global_min)
            if rows:
                st2, outs = oracle.collect(rows, w.T, local, ostart, w.L)
                del outs
            if updates:
                oracle.update(p, oidx, newp)
            reps += 1
            el = time.perf_counter() - t0
            if el >= target_s:
                break
    finally:
        os.sched_setaffinity(0, set(allowed))
    return {"value": w.B * w.L * reps / el, "unit": "trajectory-steps/s", "cores": 1, "kind": "oracle",
            "sample": "%d repetitions of one step (%s select over all %d slots, collect of "
                      "the %d selected %d-step windows from a compact host table of the selected "
                      "trajectories%s) in %.1f s on one host core"
                      % (reps, {0: "FIFO", 1: "LIFO", 2: "uniform", 3: "prioritized", 4: "TopK"}[strat], w.N, w.B,
                         w.L, ", update" if updates else "", el),
            "pinned_core": core, "nproc": os.cpu_count(), "host_cpu": model}


def run_insert(args):
    """Insertion through the index manager on the MAT-shaped HBM table, full
    and in steady state (every new trajectory releases a victim), once with
    FIFO and once with LIFO removal.  Per step and removal:
      write_rows  allocate B indices, write B device-resident trajectories into
                  them with gear_write_rows (one scatter kernel per column),
                  commit B with device-side priorities;
      insert      the same through one gear_insert call;
    and, FIFO only, the client's own scatter through the column views (torch
    indexing) in place of gear_write_rows.  Prints one JSON line with its own
    metric: trajectories inserted per second by the write_rows path, FIFO."""
    import numpy as np
    import torch

    import gen
    from gen import configs
    from gen.fill import fill_table
    from paper_2310_05205_amd import gear

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    w = configs.MAT
    dev = torch.device("cuda", 0)
    sh = torch.cuda.current_stream(dev).cuda_stream
    B, K, W = w.B, args.steps, args.warmup
    row_bytes = w.T * sum(w.elem_bytes)
    # B new trajectories, generated in HBM: insertions N .. N+B-1 of the workload.
    rows = [torch.empty((B, w.T * c.elem_bytes), dtype=torch.uint8, device=dev) for c in w.columns]
    for ci, c in enumerate(w.columns):
        gen.fill_rows_gpu(c, ci, w.seed, w.T, w.n_insert, B, rows[ci].data_ptr(), sh)
    ptrs = [r.data_ptr() for r in rows]
    prio = torch.from_numpy(gen.insert_priorities(w.prio, w.seed, w.n_insert, B)).to(dev)
    hev = HipEvents()

    def timed(fn, stages=1):
        for _ in range(W):
            fn(None)
        torch.cuda.synchronize()
        evs = [[hev.create() for _ in range(stages + 1)] for _ in range(K)]
        t0 = time.perf_counter()
        for k in range(K):
            fn(evs[k])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = [float(np.mean([hev.elapsed_ms(e[j], e[j + 1]) for e in evs])) for j in range(stages)]
        return wall, ms

    results = {}
    for removal, name in ((gear.GEAR_FIFO, "fifo"), (gear.GEAR_LIFO, "lifo")):
        t = gear.Table(w.elem_bytes, w.N, w.T, gear.GEAR_DEVICE, 0)
        t.use_allocator(removal, w.N)
        fill_table(w, lambda n, p_, q_: t.insert(p_, q_), device=0)
        views = [t.column_view(c) for c in range(len(w.columns))]

        def write_rows_step(ev):
            if ev:
                hev.record(ev[0], sh)
            idx = t.allocate(B)
            if ev:
                hev.record(ev[1], sh)
            gear.gear_write_rows(t.handle, idx, ptrs, sh)
            if ev:
                hev.record(ev[2], sh)
            t.commit(idx, prio)
            if ev:
                hev.record(ev[3], sh)

        def insert_step(ev):
            if ev:
                hev.record(ev[0], sh)
            t.insert(ptrs, prio)
            if ev:
                hev.record(ev[1], sh)

        def client_step(ev):
            if ev:
                hev.record(ev[0], sh)
            idx = t.allocate(B)
            d_idx = torch.from_numpy(idx).to(dev)
            for c, r in enumerate(rows):
                views[c][d_idx] = r
            if ev:
                hev.record(ev[1], sh)
            t.commit(idx, prio)

        wall_w, (a_ms, w_ms, c_ms) = timed(write_rows_step, 3)
        wall_i, (i_ms,) = timed(insert_step, 1)
        r = {"write_rows_path": {"trajectories_per_s": round(B * K / wall_w, 1), "ms_per_step": round(wall_w * 1e3 / K, 5),
                                 "allocate_ms": round(a_ms, 5), "write_ms": round(w_ms, 5), "commit_ms": round(c_ms, 5),
                                 "write_GBps": round(2 * B * row_bytes / (w_ms * 1e-3) / 1e9, 1)},
             "gear_insert": {"trajectories_per_s": round(B * K / wall_i, 1), "ms_per_call": round(i_ms, 5),
                             "GBps": round(2 * B * row_bytes / (i_ms * 1e-3) / 1e9, 1)}}
        if removal == gear.GEAR_FIFO:
            wall_c, (s_ms,) = timed(client_step, 1)
            r["client_torch_scatter"] = {"trajectories_per_s": round(B * K / wall_c, 1),
                                         "allocate_and_scatter_ms": round(s_ms, 5)}
        committed, pending, free = t.allocator_info()
        assert committed == w.N and pending == 0
        if t.sync() != 0:
            raise SystemExit("device status set during the insert steps")
        del views
        t.close()
        results[name] = r
    hev.close()
    fifo = results["fifo"]["write_rows_path"]
    line = {
        "metric": "trajectories inserted/sec through allocate + in-place write + commit",
        "value": fifo["trajectories_per_s"], "unit": "trajectories/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": fifo["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u8", "data": "synthetic",
        "config": {"workload": "mat-insert N=500000 T=200 B=8192 (table full, FIFO then LIFO removal)", "N": w.N,
                   "T": w.T, "B": B, "elem_bytes": w.elem_bytes, "table_bytes": w.table_bytes,
                   "parallelism": "1 GPU"},
        "by_removal": results,
        "roofline": {"bound": "hbm", "achieved": fifo["write_GBps"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(fifo["write_GBps"] / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "scatter_rows_kernel", "algorithmic_bytes_per_launch": 2 * B * row_bytes,
                     "note": "bytes of the three per-column launches of one gear_write_rows call, "
                             "over the events around that call"},
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


def run_shard(args):
    """One GPU's share of selection over G = 8 shards, each shaped like the
    MAT priorities (500000 log-normal priorities; the other shards' totals
    are taken equal to this one's).  Times, per call: the shard total, the
    shard's prioritized select of B = 8192 draws, IS weights over the
    all-reduced priorities, and the merge of 8 sorted top-8192 lists; plus a
    plain prioritized select of the same table.  Prints one JSON line."""
    import numpy as np
    import torch

    import gen
    from gen import configs
    from paper_2310_05205_amd import gear

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    w = configs.MAT
    G, g, B, K = 8, 3, w.B, 8192
    dev = torch.device("cuda", 0)
    sh = torch.cuda.current_stream(dev).cuda_stream
    t = gear.Table([], w.N, 1, gear.GEAR_DEVICE, 0)   # priorities only: windows of one step
    t.insert([], gen.insert_priorities(w.prio, w.seed, 0, w.N))
    totals = torch.zeros(G, dtype=torch.int64, device=dev)
    t.shard_total(totals[g:g + 1])
    torch.cuda.synchronize()
    totals.fill_(int(totals[g].item()))
    local, _, _ = t.select(gear.GEAR_TOPK, K, 1, 0)
    lp = torch.from_numpy(t.priorities().view(np.int32)).to(dev)[local]
    gidx = torch.stack([local + h * w.N for h in range(G)])
    gprio = torch.stack([lp for _ in range(G)])
    idx = torch.empty(B, dtype=torch.int64, device=dev)
    start = torch.empty(B, dtype=torch.int32, device=dev)
    selp = torch.empty(B, dtype=torch.int32, device=dev)
    wts = torch.empty(B, dtype=torch.float32, device=dev)
    midx = torch.empty(K, dtype=torch.int64, device=dev)
    mstart = torch.empty(K, dtype=torch.int32, device=dev)
    hev = HipEvents()
    K_, W = args.steps, args.warmup

    def timed(fn):
        for i in range(W):
            fn(i)
        torch.cuda.synchronize()
        a, b = hev.create(), hev.create()
        hev.record(a, sh)
        for i in range(K_):
            fn(W + i)
        hev.record(b, sh)
        torch.cuda.synchronize()
        return hev.elapsed_ms(a, b) * 1e3 / K_

    out = {
        "shard_total_us": timed(lambda i: gear.gear_shard_total(t.handle, totals[g:g + 1].data_ptr(), sh)),
        "select_shard_us": timed(lambda i: gear.gear_select_shard(t.handle, G, g, totals.data_ptr(), g * w.N, B, 1,
                                                                  gen.select_seed(w.seed, i), idx.data_ptr(),
                                                                  start.data_ptr(), selp.data_ptr(), sh)),
        "is_weights_us": timed(lambda i: gear.gear_is_weights(t.handle, selp.data_ptr(), B, w.beta, wts.data_ptr(), sh)),
        "topk_merge_us": timed(lambda i: gear.gear_topk_merge(gprio.data_ptr(), gidx.data_ptr(), G, K, w.T, w.L,
                                                              gen.select_seed(w.seed, i), midx.data_ptr(),
                                                              mstart.data_ptr(), 0, 0, sh)),
        "plain_select_us": timed(lambda i: gear.gear_select(t.handle, gear.GEAR_PRIORITIZED, B, 1,
                                                            gen.select_seed(w.seed, i), w.beta, idx.data_ptr(),
                                                            start.data_ptr(), wts.data_ptr(), sh)),
    }
    if t.sync() != 0:
        raise SystemExit("device status set during the shard steps")
    hev.close()
    t.close()
    line = {
        "metric": "sharded selection, one GPU's share: draws resolved per second by this shard",
        "value": round(B / (out["select_shard_us"] * 1e-6), 1), "unit": "draws/s", "n_gpus": 1, "steps": K_,
        "warmup": W, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": "shard-select G=8 shards of N=500000 log-normal priorities, B=8192, TopK K=8192",
                   "G": G, "g": g, "N_per_shard": w.N, "B": B, "K": K, "parallelism": "1 GPU (shard 3 of 8)"},
        "per_call_us": {k: round(v, 2) for k, v in out.items()},
        "note": "the all-gather of 8 totals, the all-reduce of B priorities and the gather of 8 top-K lists "
                "are the caller's collectives and are not timed here; select_shard rescans only when dirty",
        "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


class Step:
    """One workload's step on a table, issued through the C ABI with its
    arguments built once: select into buffer set k, collect from set k into
    batch set k, update the priorities of set k's draws.  The sets (indices,
    starts, weights and one batch buffer per column) are used in turn, so
    no batch line is still cached from the step before."""

    def __init__(self, t, w, nsets, iters, dev, options=0):
        import numpy as np
        import torch

        import gen
        from paper_2310_05205_amd import gear

        self.gear, self.lib = gear, gear.lib()
        self.tab = ctypes.c_void_p(t.handle)
        self.options = options
        self.B, self.L = w.B, w.L
        self.strategy = w.strategies[0]
        self.updates = self.strategy in (gear.GEAR_PRIORITIZED, gear.GEAR_TOPK)
        self.weights = bool(w.weights)
        self.beta = ctypes.c_float(w.beta)
        self.ncols = len(w.elem_bytes)
        B, L = w.B, w.L
        self.idx = [torch.empty(B, dtype=torch.int64, device=dev) for _ in range(nsets)]
        self.start = [torch.empty(B, dtype=torch.int32, device=dev) for _ in range(nsets)]
        self.wts = [torch.empty(B, dtype=torch.float32, device=dev) for _ in range(nsets)]
        self.outs = [[torch.empty(B * L * e, dtype=torch.uint8, device=dev) for e in w.elem_bytes]
                     for _ in range(nsets)]
        vp = lambda x: ctypes.c_void_p(x.data_ptr())
        self.ip = [vp(x) for x in self.idx]
        self.sp = [vp(x) for x in self.start]
        self.wp = [vp(x) if self.weights else None for x in self.wts]
        self.op = [gear._ptr_array([o.data_ptr() for o in outs]) for outs in self.outs]
        self.seeds = [ctypes.c_uint64(gen.select_seed(w.seed, it)) for it in range(iters)]
        if self.updates:
            self.newp = torch.from_numpy(np.stack([gen.update_priorities(w.prio, w.seed, it, B)
                                                   for it in range(iters)])).to(dev)
            self.np_ = [vp(self.newp[it]) for it in range(iters)]

    def _ok(self, rc, what):
        if rc != 0:
            raise RuntimeError("%s failed: %s" % (what, self.gear.gear_last_error()))

    def select(self, it, k, sh):
        self._ok(self.lib.gear_select(self.tab, self.strategy, self.B, self.L, self.seeds[it], self.beta, self.ip[k],
                                      self.sp[k], self.wp[k], sh), "gear_select")

    def collect(self, k, sh):
        self._ok(self.lib.gear_collect(self.tab, self.ip[k], self.sp[k], self.B, self.L, None, self.ncols, self.op[k],
                                       sh), "gear_collect")

    def update(self, it, k, sh):
        self._ok(self.lib.gear_update_priorities(self.tab, self.ip[k], self.np_[it], self.B, sh),
                 "gear_update_priorities")

    def select_collect(self, it, k, sh):
        """FIFO, LIFO or uniform selection and its gather in one launch."""
        self._ok(self.lib.gear_select_collect(self.tab, self.strategy, self.B, self.L, self.seeds[it], self.ip[k],
                                              self.sp[k], self.wp[k], None, self.ncols, self.op[k], sh),
                 "gear_select_collect")

    def share_cus(self, on):
        """Gathers enqueued from now on leave room for the other stream (on) or not."""
        opts = self.options | (self.gear.GEAR_OPT_GATHER_SHARE_CU if on else 0)
        self._ok(self.lib.gear_table_set_options(self.tab, ctypes.c_uint32(opts)), "gear_table_set_options")


def concurrent_streams(dev, tries=8):
    """Two streams from torch's pool (default priority, like every stream
    here) whose work runs concurrently.  HIP spreads streams over a few
    hardware queues, and two streams on one queue run one after the other:
    pipelined steps then take as long as serial ones.  A pair passes if, in
    both directions, a tiny kernel on one finishes while a 1 GiB copy on the
    other is still running.  Each stream first runs a tiny kernel of its
    own: the first work on a fresh stream starts late, which failed the check
    for pairs that overlap well (ratios 0.8-2.4 cold, 0.1 warmed), so that
    every try could fail and the steps fell back to one stream."""
    import torch
    big = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    small = torch.zeros(16, dtype=torch.float32, device=dev)

    def finishes_inside(a, b):
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record(b)
        with torch.cuda.stream(b):
            big.mul_(1.0)
        e[1].record(b)
        a.wait_event(e[0])
        with torch.cuda.stream(a):
            small.add_(1.0)
        e[2].record(a)
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[2]) < 0.5 * e[0].elapsed_time(e[1])

    torch.cuda.synchronize()
    for _ in range(tries):
        a, b = torch.cuda.Stream(dev), torch.cuda.Stream(dev)
        for s in (a, b):
            with torch.cuda.stream(s):
                small.add_(0.0)
        torch.cuda.synchronize()
        if finishes_inside(a, b) and finishes_inside(b, a):
            del big, small
            return a, b
    return None  # e.g. under a counter-collecting profiler, which serialises dispatches


def capturable(w, options):
    """Whether a step of w (select, collect, and the update of prioritized or
    TopK draws) replays correctly from a HIP graph capture: the calls whose
    captures gear.h lists as replaying correctly."""
    from paper_2310_05205_amd import gear
    strategy = w.strategies[0]
    if options & gear.GEAR_OPT_INCREMENTAL_TREE:
        return strategy in (gear.GEAR_FIFO, gear.GEAR_LIFO, gear.GEAR_UNIFORM)
    if strategy == gear.GEAR_PRIORITIZED:
        return w.N <= gear.GEAR_SMALL_SELECT_MAX_N and w.B <= gear.GEAR_SMALL_SELECT_MAX_B
    return True


# Sizes of a pipeline's first groups.  The gather stream waits for the first
# group's selections and updates before it can start, about 23 us per step
# on an idle GPU, so the pipeline starts with one step, then two, then
# `group` per handshake.  Beside gathers that hold 4 workgroups per CU the
# selection stream is no faster than the gathers, and it would then fall
# behind a growing group; during the ramp the gathers therefore run with
# GEAR_OPT_GATHER_SHARE_CU, which halves the selection chain's time beside
# them.  MAT steps, one table, configurations alternated in one process:
# 100.1-100.5 against 102.1-102.4 us per step over 20 steps, and 96.6-96.9
# against 97.0-97.4 over 100.  With the option in every group the 20-step
# figure is the same, and the 100-step one up to 0.7 us worse.
RAMP = (1, 2)


def pipeline_groups(n, group, ramp=RAMP):
    """Positions 0..n-1 split into handshake groups: the ramp's sizes (at most
    `group` each), then `group` steps per group."""
    if group < 1:
        raise ValueError("a handshake group holds at least one step")
    sizes = [min(r, group) for r in ramp]
    out, j, g = [], 0, 0
    while j < n:
        size = sizes[g] if g < len(sizes) else group
        out.append(list(range(j, min(n, j + size))))
        j += size
        g += 1
    return out


def set_reuse_waits(groups, nsets):
    """For each group, the earlier groups whose gathers the selection stream
    must see finished before it writes the group's buffer sets (a step at
    position j uses set j % nsets)."""
    last, waits = {}, []
    for g, js in enumerate(groups):
        waits.append(sorted({last[j % nsets] for j in js if j % nsets in last}))
        for j in js:
            last[j % nsets] = g
    return waits


def run_steps(t, w, K, W, dev, pipelined, group=4, stage_steps=50, serial_too=False, options=0, timed_every=1,
              graph=False):
    """W untimed steps, then K timed ones, of workload w on table t.

    Serial: select, collect and update of each step on one stream, in turn
    over two buffer sets.
    Pipelined: select and update on a second stream S, collect on the
    current stream C, in groups over 2*group buffer sets: one step, two,
    then `group` steps per group (RAMP).  S issues the selects and updates
    of a group, with one event after the last select (before the last
    update); C waits for that event once and runs the group's gathers, then
    records one event, which S waits for before it reuses those buffer sets
    in a later group.  Recording the event before the last update took
    0.5 us off a MAT step over 20 steps and 0.8 us over 100.
    Every select still follows the previous step's update on S, so each step
    draws exactly what the serial order draws; the selects and updates of
    the next group overlap this group's gathers.  A cross-stream wait and a
    marker between two gathers cost about 6 us (measured on gfx950 with
    64 MB copies), which the groups pay once per group instead of per step.

    Returns wall time, the mean gather launch time in the timed region, a
    per-stage breakdown from a one-stream loop after the timed region, and,
    with serial_too, the serial step time.  Gather launches are timed with
    HIP events on C: serially, an event before and after the gather of every
    timed_every-th step (each marker costs the stream about 2 us, which in a
    launch-bound step of a few microseconds would dominate what is measured);
    pipelined, an event after C's wait and the group's closing event, which
    bracket the group's gathers and nothing else.

    graph (serial steps only): the K timed steps are captured into one HIP
    graph before the timed region, and the timed region replays it once.
    Events cannot be recorded inside the graph, so the gather time then
    comes from the stage loop after the timed region."""
    import numpy as np
    import torch

    if graph and pipelined:
        raise ValueError("graph replay takes steps issued in order on one stream")
    pair = concurrent_streams(dev) if pipelined else None
    fallback = pipelined and pair is None
    pipelined = pair is not None    # no two streams run concurrently: steps in order on one stream
    nsets = 2 * group if pipelined else 2
    step = Step(t, w, nsets, W + K, dev, options)
    hev = HipEvents()
    if pipelined:
        gather_stream, side = pair
        C, S = ctypes.c_void_p(gather_stream.cuda_stream), ctypes.c_void_p(side.cuda_stream)
    elif graph:
        capture_stream = torch.cuda.Stream(dev)  # capture needs a stream other than the default one
        C = ctypes.c_void_p(capture_stream.cuda_stream)
        S = C
    else:
        C = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
        S = C
    ngroups = len(pipeline_groups(max(K, W), group))
    sel_done = [hev.create() for _ in range(ngroups)]
    col_begin = [hev.create() for _ in range(ngroups)]
    col_done = [hev.create() for _ in range(ngroups)]
    ev = [(hev.create(), hev.create()) for _ in range((K + timed_every - 1) // timed_every)]

    def loop_serial(its, timed):
        for j, it in enumerate(its):
            k = j % nsets
            mark = timed and j % timed_every == 0
            step.select(it, k, C)
            if mark:
                hev.record(ev[j // timed_every][0], C.value)
            if step.ncols:
                step.collect(k, C)
            if mark:
                hev.record(ev[j // timed_every][1], C.value)
            if step.updates:
                step.update(it, k, C)

    def loop_pipe(its):
        its = list(its)
        groups = pipeline_groups(len(its), group)
        for g, (js, waits) in enumerate(zip(groups, set_reuse_waits(groups, nsets))):
            for p in waits:
                hev.wait(S.value, col_done[p])
            for n, j in enumerate(js):
                step.select(its[j], j % nsets, S)
                if n == len(js) - 1:
                    # The gathers read the selected indices and starts, never
                    # the priorities: they need not wait for the last update.
                    hev.record(sel_done[g], S.value)
                if step.updates:
                    step.update(its[j], j % nsets, S)
            hev.wait(C.value, sel_done[g])
            hev.record(col_begin[g], C.value)
            step.share_cus(g < len(RAMP))
            for j in js:
                step.collect(j % nsets, C)
            hev.record(col_done[g], C.value)
        step.share_cus(False)
        return len(groups)

    if pipelined:
        loop_pipe(range(W))
    else:
        loop_serial(range(W), False)
    torch.cuda.synchronize()
    if t.sync() != 0:
        raise SystemExit("device status set during warm-up")
    if graph:
        hip_graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(hip_graph, stream=capture_stream, capture_error_mode="relaxed"):
            loop_serial(range(W, W + K), False)
        torch.cuda.synchronize()
    t0 = time.perf_counter()
    if graph:
        hip_graph.replay()
        ng = 0
    else:
        ng = loop_pipe(range(W, W + K)) if pipelined else loop_serial(range(W, W + K), True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    status = t.sync()
    if status != 0:
        raise SystemExit("device status %d set during the timed steps" % status)
    if graph:
        col_ms = None  # from the stage loop below
    elif pipelined:
        col_ms = sum(hev.elapsed_ms(col_begin[g], col_done[g]) for g in range(ng)) / K
    else:
        col_ms = float(np.mean([hev.elapsed_ms(a, b) for a, b in ev]))
    res = {"wall_s": wall, "collect_ms": col_ms, "step": step, "buffer_sets": nsets, "pipelined": pipelined,
           "fallback": fallback}
    if pipelined and ng > 1:
        # Gather-stream time between one group's last gather and the next
        # group's first: the handshake plus any wait for S.  About 9-13 us
        # when the streams overlap; one group of selects and updates (about
        # 100 us) when they run one after the other.
        res["gather_stream_gap_us"] = float(np.median([hev.elapsed_ms(col_done[g - 1], col_begin[g]) * 1e3
                                                       for g in range(1, ng)]))
    if serial_too and pipelined:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        loop_serial(range(W, W + K), False)
        torch.cuda.synchronize()
        res["serial_ms_per_step"] = (time.perf_counter() - t0) * 1e3 / K

    # Stage breakdown: one stream, events around every stage.
    nb = min(K, stage_steps)
    sev = [[hev.create() for _ in range(4)] for _ in range(nb)]
    for j in range(nb):
        it, k, e = W + j, j % nsets, sev[j]
        hev.record(e[0], C.value)
        step.select(it, k, C)
        hev.record(e[1], C.value)
        if step.ncols:
            step.collect(k, C)
        hev.record(e[2], C.value)
        if step.updates:
            step.update(it, k, C)
        hev.record(e[3], C.value)
    torch.cuda.synchronize()
    if t.sync() != 0:
        raise SystemExit("device status set during the stage loop")
    stages = {"select": [hev.elapsed_ms(e[0], e[1]) for e in sev],
              "collect": [hev.elapsed_ms(e[1], e[2]) for e in sev],
              "update": [hev.elapsed_ms(e[2], e[3]) for e in sev]}
    res["stages_mean"] = {k: float(np.mean(v)) for k, v in stages.items()}
    if graph:
        res["collect_ms"] = res["stages_mean"]["collect"]
    res["stages_pct"] = {k: [round(float(x), 5) for x in np.percentile(v, [10, 50, 90])] for k, v in stages.items()
                         if (k != "update" or step.updates) and (k != "collect" or step.ncols)}
    hev.close()
    return res


def incremental_leg(t, w, dev, K=50, W=5):
    """The same MAT table with the sum tree kept current by the updates
    (GEAR_OPT_INCREMENTAL_TREE: selects skip the rescan), K steps in order
    on one stream: the serial step and the select and update stage times.
    The headline keeps the rescan per select that the method describes."""
    from paper_2310_05205_amd import gear

    t.set_options(gear.GEAR_OPT_INCREMENTAL_TREE)
    r = run_steps(t, w, K, W, dev, False, stage_steps=K, options=gear.GEAR_OPT_INCREMENTAL_TREE)
    t.set_options(0)
    del r["step"]
    sm, pct = r["stages_mean"], r["stages_pct"]
    return {"tree": "incremental", "steps": K, "serial_ms_per_step": round(r["wall_s"] * 1e3 / K, 5),
            "select_us": round(sm["select"] * 1e3, 2), "update_us": round(sm["update"] * 1e3, 2),
            "collect_us": round(sm["collect"] * 1e3, 2),
            "select_us_p10_p50_p90": [round(x * 1e3, 2) for x in pct["select"]],
            "note": "steps in order on one stream on the headline table, the gathers timed by events"}


def gather_roofline(w, col_ms, workload_key):
    """Roofline object of the gather: algorithmic bytes per launch over the
    mean event-timed launch duration."""
    batch_bytes = w.B * w.L * sum(w.elem_bytes)
    if w.host_table:
        alg, peak, bound = batch_bytes, HOST_LINK_PEAK_GBS, "host-link"   # bytes crossing the link
    else:
        alg, peak, bound = 2 * batch_bytes, HBM_PEAK_GBS, "hbm"            # window bytes read + batch written
    achieved = alg / (col_ms * 1e-3) / 1e9
    return {"bound": bound, "achieved": round(achieved, 1), "peak": peak, "unit": "GB/s",
            "frac": round(achieved / peak, 4), "traffic": profiled_traffic("collect_kernel", workload_key),
            "kernel": "collect_kernel", "algorithmic_bytes_per_launch": alg, "avg_launch_ms": round(col_ms, 5)}


def make_table(w, dev_index=0):
    from gen.fill import fill_table
    from paper_2310_05205_amd import gear
    t = gear.Table(w.elem_bytes, w.N, w.T, gear.GEAR_HOST_PINNED if w.host_table else gear.GEAR_DEVICE, dev_index)
    fill_table(w, lambda n, ptrs, prio: t.insert(ptrs, prio), device=dev_index)
    return t


def host_link_leg(dev, steps=10, warmup=2):
    """Gato-like table (31.5 GB) in pinned host memory, read zero-copy:
    prioritized select, gather of 1024 windows of 64 steps (805.8 MB over
    the host link), update."""
    from gen import configs
    w = configs.GATO_HOST
    t0 = time.perf_counter()
    t = make_table(w)
    setup = time.perf_counter() - t0
    try:
        r = run_steps(t, w, steps, warmup, dev, pipelined=False, stage_steps=steps)
        roof = gather_roofline(w, r["collect_ms"], "gato-host")
        st = r["step"]
        link = host_link_extras(t, w, st.idx[0], st.start[0], st.outs[0], dev)
        if not link["cpu_staged"]["matches_zero_copy"]:
            raise SystemExit("the CPU-staged batch differs from the zero-copy batch")
    finally:
        t.close()
    return {"workload": w.name, "residency": "pinned-host", "achieved_gbs": roof["achieved"],
            "peak_gbs": HOST_LINK_PEAK_GBS, "frac": roof["frac"], "gate": 0.70,
            "link_h2d_copy_gbs": link["link_h2d_copy_gbs"],
            "frac_of_h2d_copy": round(roof["achieved"] / link["link_h2d_copy_gbs"], 4),
            "avg_launch_ms": roof["avg_launch_ms"], "link_bytes_per_launch": roof["algorithmic_bytes_per_launch"],
            "traffic": roof["traffic"], "steps": steps, "ms_per_step": round(r["wall_s"] * 1e3 / steps, 4),
            "cpu_staged": link["cpu_staged"], "table_setup_s": round(setup, 1)}


def run_fused(t, w, K, W, dev, graph=False, timed_every=4):
    """K steps of gear_select_collect (FIFO, LIFO or uniform selection and
    its gather in one launch) in order on one stream, after W untimed ones,
    over two buffer sets.  Eager: HIP events around every timed_every-th
    launch.  graph: the K steps captured into one HIP graph before the timed
    region, which replays it once.  Returns wall seconds and the mean event-
    timed launch (None with graph)."""
    import numpy as np
    import torch

    step = Step(t, w, 2, W + K, dev)
    hev = HipEvents()
    ev = [(hev.create(), hev.create()) for _ in range((K + timed_every - 1) // timed_every)]
    if graph:
        cs = torch.cuda.Stream(dev)
        C = ctypes.c_void_p(cs.cuda_stream)
    else:
        C = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)

    def loop(its, timed):
        for j, it in enumerate(its):
            mark = timed and j % timed_every == 0
            if mark:
                hev.record(ev[j // timed_every][0], C.value)
            step.select_collect(it, j % 2, C)
            if mark:
                hev.record(ev[j // timed_every][1], C.value)

    if graph:
        with torch.cuda.stream(cs):
            loop(range(W), False)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cs, capture_error_mode="relaxed"):
            loop(range(W, W + K), False)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        g.replay()
    else:
        loop(range(W), False)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        loop(range(W, W + K), True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = None if graph else float(np.mean([hev.elapsed_ms(a, b) for a, b in ev]))
    hev.close()
    if t.sync() != 0:
        raise SystemExit("device status set during the fused select-and-gather steps")
    return wall, ms


def dt_legs(dev, launches=64, sets=8, window_steps=200):
    """DT-shaped table (6.55 GB, HBM).

    Whole trajectories: uniform selection of 512 whole trajectories (L = T =
    1000), 51.2 MB read and written per gather.  The selections of `sets`
    batches are made first; then `launches` gathers run back to back,
    cycling over those batches and their output buffers (8 x 51.2 MB, more
    than the last-level cache holds), between two HIP events on their stream.

    20-step windows on the same table: `window_steps` steps of a uniform
    select of 512 windows and their gather (2.05 MB), in order on one stream,
    then the same steps captured into one HIP graph and replayed.  These
    steps are launch-bound."""
    import torch
    from gen import configs
    w = configs.DT_FULL
    t = make_table(w)
    try:
        windows = dt_windows(t, dev, window_steps)
        step = Step(t, w, sets, sets, dev)
        C = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
        for k in range(sets):
            step.select(k, k, C)
        for k in range(sets):
            step.collect(k, C)
        hev = HipEvents()
        a, b = hev.create(), hev.create()
        hev.record(a, C.value)
        for k in range(launches):
            step.collect(k % sets, C)
        hev.record(b, C.value)
        torch.cuda.synchronize()
        col_ms = hev.elapsed_ms(a, b) / launches
        # The same batches selected inside the gather launch (uniform draws
        # computed per piece, no index list read first), back to back.
        a2, b2 = hev.create(), hev.create()
        hev.record(a2, C.value)
        for k in range(launches):
            step.select_collect(k % sets, k % sets, C)
        hev.record(b2, C.value)
        torch.cuda.synchronize()
        fused_ms = hev.elapsed_ms(a2, b2) / launches
        hev.close()
        if t.sync() != 0:
            raise SystemExit("device status set during the whole-trajectory gathers")
    finally:
        t.close()
    roof = gather_roofline(w, col_ms, "dt-full")
    full = {"workload": w.name, "achieved_gbs": roof["achieved"], "peak_gbs": HBM_PEAK_GBS, "frac": roof["frac"],
            "gate": 0.70, "avg_launch_ms": roof["avg_launch_ms"],
            "algorithmic_bytes_per_launch": roof["algorithmic_bytes_per_launch"], "traffic": roof["traffic"],
            "launches": launches, "batches": sets}
    fused = gather_roofline(w, fused_ms, "dt-full")
    full["select_collect"] = {"avg_launch_ms": fused["avg_launch_ms"], "achieved_gbs": fused["achieved"],
                              "frac": fused["frac"],
                              "note": "gear_select_collect: the uniform selection computed inside the gather launch, "
                                      "the same bytes per launch"}
    return full, windows


def dt_windows(t, dev, K, W=10):
    """The DT 20-step-window steps on table t (which holds the DT trajectories)."""
    from gen import configs
    w = configs.DT
    eager = run_steps(t, w, K, W, dev, pipelined=False, stage_steps=20, timed_every=4)
    replay = run_steps(t, w, K, W, dev, pipelined=False, stage_steps=20, graph=True)
    f_wall, f_ms = run_fused(t, w, K, W, dev)
    g_wall, _ = run_fused(t, w, K, W, dev, graph=True)
    ts = w.B * w.L * K
    return {"workload": w.name, "strategy": "uniform", "steps": K,
            "eager_us_per_step": round(eager["wall_s"] * 1e6 / K, 2),
            "eager_value": round(ts / eager["wall_s"], 1),
            "graph_us_per_step": round(replay["wall_s"] * 1e6 / K, 2),
            "graph_value": round(ts / replay["wall_s"], 1),
            "unit": "trajectory-steps/s",
            "gather_avg_us": round(eager["collect_ms"] * 1e3, 2),
            "select_collect": {"eager_us_per_step": round(f_wall * 1e6 / K, 2), "eager_value": round(ts / f_wall, 1),
                               "graph_us_per_step": round(g_wall * 1e6 / K, 2), "graph_value": round(ts / g_wall, 1),
                               "launch_avg_us": round(f_ms * 1e3, 2)},
            "note": "eager: select and gather issued in order on one stream, events around every 4th gather; "
                    "graph: the same steps captured into one HIP graph before the timed region and replayed once; "
                    "select_collect: each step one gear_select_collect launch, eager and from a graph"}


def selection_leg(dev, iters=100, warmup=5):
    """Selection without collection on 2^22 Pareto(1.5) priorities, each
    iteration a select of B = 8192 and an update of those draws:
    prioritized with IS weights, then TopK of the 8192 highest.  Rated
    against HBM with the bytes the method must move: the scan's 4N-byte read
    of the priorities plus the select's outputs (idx 8 B, start 4 B, weight
    4 B per draw), and for the update the idx and value read and the
    priority written (16 B per draw)."""
    from gen import configs
    out = {}
    for w, key in ((configs.SELECT_STRESS, "prioritized"), (configs.TOPK_STRESS, "topk")):
        t = make_table(w)
        try:
            r = run_steps(t, w, iters, warmup, dev, pipelined=False, stage_steps=iters)
        finally:
            t.close()
        sel_ms, upd_ms = r["stages_mean"]["select"], r["stages_mean"]["update"]
        sel_bytes = 4 * w.N + w.B * (8 + 4 + (4 if w.weights else 0))
        upd_bytes = 16 * w.B
        out[key] = {"workload": w.name, "select_us": round(sel_ms * 1e3, 2), "update_us": round(upd_ms * 1e3, 2),
                    "samples_per_s": round(w.B / (sel_ms * 1e-3), 1),
                    "select_algorithmic_bytes": sel_bytes,
                    "select_frac_of_hbm": round(sel_bytes / (sel_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                    "update_algorithmic_bytes": upd_bytes,
                    "update_frac_of_hbm": round(upd_bytes / (upd_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                    "select_us_p10_p50_p90": [round(x * 1e3, 2) for x in r["stages_pct"]["select"]],
                    "iterations": iters}
    return out


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: there is no multi-GPU path here (requested %d GPUs, WORLD_SIZE=%d)"
              % (args.gpus, world), file=sys.stderr)
        sys.exit(2)
    if args.calibrate:
        calibrate()
        return
    if args.ceilings:
        ceilings()
        return
    if args.workload == "mat-insert":
        run_insert(args)
        return
    if args.workload == "shard-select":
        run_shard(args)
        return

    import torch

    from paper_2310_05205_amd import gear

    w = workload(args.workload)
    if args.strategy:
        code = {"fifo": 0, "lifo": 1, "uniform": 2, "prioritized": 3, "topk": 4}[args.strategy]
        if code not in w.strategies:
            print("bench.py --strategy: %s is not one of the %s workload's strategies" % (args.strategy, w.name),
                  file=sys.stderr)
            sys.exit(2)
        w = dataclasses.replace(w, strategies=(code,) + tuple(x for x in w.strategies if x != code))
    opts = (gear.GEAR_OPT_INCREMENTAL_TREE if args.incremental else 0) | \
        (gear.GEAR_OPT_IS_GLOBAL_MIN if args.global_min else 0)
    if args.graph and not capturable(w, opts):
        print("bench.py --graph: the %s steps cannot be replayed from a HIP graph capture (prioritized selection "
              "over more than %d slots, or with the incremental tree, decides per call how to keep its sum tree)"
              % (w.name, gear.GEAR_SMALL_SELECT_MAX_N), file=sys.stderr)
        sys.exit(2)
    if args.fused and (w.strategies[0] not in (gear.GEAR_FIFO, gear.GEAR_LIFO, gear.GEAR_UNIFORM) or not w.elem_bytes):
        print("bench.py --fused: only FIFO, LIFO and uniform workloads with columns (%s is not)" % w.name,
              file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    gear.lib()  # fails loudly if the library is not built
    dev = torch.device("cuda", 0)
    t = make_table(w)
    if opts:
        t.set_options(opts)
    K, W = args.steps, args.warmup
    strategy = w.strategies[0]
    # Steps whose gather dominates (a batch of at least PIPELINE_MIN_BATCH
    # bytes from a device table) are pipelined over two streams.  Smaller
    # batches are launch-bound, and the cross-stream handshakes cost more
    # than the overlap saves (DT 20-step windows: 24.2 against 12.0 us per
    # step); a pinned host table's gather takes milliseconds; so those steps,
    # and selection-only workloads, run in order on one stream.
    batch = w.B * w.L * sum(w.elem_bytes)
    if args.fused:
        wall, ms = run_fused(t, w, K, W, dev, graph=args.graph, timed_every=1 if batch >= PIPELINE_MIN_BATCH else 4)
        t.close()
        line = {"metric": METRIC, "value": round(w.B * w.L * K / wall, 1), "unit": "trajectory-steps/s",
                "n_gpus": 1, "steps": K, "warmup": W, "ms_per_step": round(wall * 1e3 / K, 5),
                "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u64",
                "data": "synthetic",
                "config": {"workload": w.name, "N": w.N, "T": w.T, "B": w.B, "L": w.L,
                           "strategy": {0: "fifo", 1: "lifo", 2: "uniform"}[strategy],
                           "steps_issued": "one gear_select_collect launch per step, "
                                           + ("replayed from a HIP graph" if args.graph else "in order on one stream")},
                "roofline": gather_roofline(w, ms, args.workload) if ms is not None else None,
                "cpu_baseline": None}
        print(json.dumps(line), flush=True)
        return
    pipelined = (batch >= PIPELINE_MIN_BATCH and not w.host_table and not args.serial) or args.pipeline
    if args.graph:
        pipelined = False
    # Short serial steps are launch-bound: time every fourth gather only.
    timed_every = 1 if pipelined or batch >= PIPELINE_MIN_BATCH else 4
    r = run_steps(t, w, K, W, dev, pipelined, group=args.group, serial_too=pipelined, options=opts,
                  timed_every=timed_every, graph=args.graph)
    if r["fallback"]:
        print("bench.py: no two streams ran concurrently; the steps ran in order on one stream", file=sys.stderr)
    pipelined = r["pipelined"]
    prioritized = strategy in (gear.GEAR_PRIORITIZED, gear.GEAR_TOPK)
    roof = gather_roofline(w, r["collect_ms"], args.workload) if w.elem_bytes else None
    context = torch_context(t, w, dev) if prioritized else None
    link = None
    if w.host_table and w.elem_bytes:
        st = r["step"]
        link = host_link_extras(t, w, st.idx[0], st.start[0], st.outs[0], dev)
        if not link["cpu_staged"]["matches_zero_copy"]:
            raise SystemExit("the CPU-staged batch differs from the zero-copy batch")
        link["zero_copy_frac_of_h2d_copy"] = round(roof["achieved"] / link["link_h2d_copy_gbs"], 4)
    del r["step"]
    incremental = None
    if args.workload == "mat" and not (args.incremental or args.global_min) and args.legs == "all":
        incremental = incremental_leg(t, w, dev)
    t.close()

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args.cpu_seconds, args.global_min)

    B, L = w.B, w.L
    sm = r["stages_mean"]
    line = {
        "metric": METRIC, "value": round(B * L * K / r["wall_s"], 1), "unit": "trajectory-steps/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(r["wall_s"] * 1e3 / K, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": w.name, "N": w.N, "T": w.T, "B": B, "L": L,
                   "columns": {c.name: "%s[%d]" % (c.dtype, c.m) for c in w.columns},
                   "elem_bytes": w.elem_bytes, "table_bytes": w.table_bytes,
                   "residency": "pinned-host" if w.host_table else "hbm",
                   "strategy": {0: "fifo", 1: "lifo", 2: "uniform", 3: "prioritized", 4: "topk"}[strategy],
                   "is_weights": bool(w.weights), "parallelism": "1 GPU",
                   "tree": "incremental" if args.incremental and not args.global_min else "rescan per select",
                   "is_normalisation": "table minimum" if args.global_min else "batch minimum",
                   "steps_issued": "two streams, select/update overlapping the gather" if pipelined
                   else "one HIP graph of the timed steps, captured before the timed region and replayed once"
                   if args.graph else "one stream, in order", "batch_buffer_sets": r["buffer_sets"],
                   "steps_per_handshake": args.group if pipelined else None,
                   "first_groups": [min(x, args.group) for x in RAMP] if pipelined else None,
                   "gathers_timed": "in the stage loop after the timed region (no events inside a graph)"
                   if args.graph else "every step's" if timed_every == 1 else "every %dth step's" % timed_every},
        "roofline": roof,
        "cpu_baseline": cpu,
        "stages_ms": {"select": round(sm["select"], 5),
                      "collect": round(sm["collect"], 5) if w.elem_bytes else None,
                      "update": round(sm["update"], 5) if prioritized else None,
                      "note": "from a one-stream loop with events around every stage, after the timed region"},
        "stages_ms_p10_p50_p90": r["stages_pct"],
        "selection_samples_per_s": round(B / (sm["select"] * 1e-3), 1),
        "batch_bytes": B * L * sum(w.elem_bytes),
    }
    if pipelined:
        line["serial_ms_per_step"] = round(r["serial_ms_per_step"], 5)
        line["gather_stream_gap_us_median"] = round(r["gather_stream_gap_us"], 2) if "gather_stream_gap_us" in r else None
        line["serial_value"] = round(B * L / (r["serial_ms_per_step"] * 1e-3), 1)
    if link is not None:
        line["host_link"] = link
    if context is not None:
        line["torch_context"] = context
    if args.workload == "mat" and not (args.incremental or args.global_min) and args.legs == "all":
        # The other gates, measured in the same run after the headline table is closed.
        line["host_link"] = host_link_leg(dev)
        line["dt_full"], line["dt_windows"] = dt_legs(dev)
        line["selection"] = selection_leg(dev)
        line["incremental_tree"] = incremental
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
