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
    ap.add_argument("--incremental", action="store_true",
                    help="keep the selection sum tree current across updates (no rescan per step)")
    ap.add_argument("--global-min", action="store_true",
                    help="IS weights normalised over the whole table (GEAR_OPT_IS_GLOBAL_MIN)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="target oracle time for the CPU baseline")
    ap.add_argument("--calibrate", action="store_true", help="run a plain copy kernel of known size and exit")
    ap.add_argument("--ceilings", action="store_true", help="measure plain read/write/copy HBM rates and exit")
    return ap.parse_args()


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
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


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
    from tests.helpers import oracle_priorities

    p, next_seq = oracle_priorities(w)
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

    import numpy as np
    import torch

    import gen
    from gen.fill import fill_table
    from paper_2310_05205_amd import gear

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    gear.lib()  # fails loudly if the library is not built
    w = workload(args.workload)
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream

    host_table = w.host_table
    t = gear.Table(w.elem_bytes, w.N, w.T, gear.GEAR_HOST_PINNED if host_table else gear.GEAR_DEVICE, 0)
    fill_table(w, lambda n, ptrs, prio: t.insert(ptrs, prio), device=0)
    opts = (gear.GEAR_OPT_INCREMENTAL_TREE if args.incremental else 0) | \
        (gear.GEAR_OPT_IS_GLOBAL_MIN if args.global_min else 0)
    if opts:
        t.set_options(opts)

    K, W = args.steps, args.warmup
    B, L = w.B, w.L
    strategy = w.strategies[0]
    prioritized = strategy in (gear.GEAR_PRIORITIZED, gear.GEAR_TOPK)  # steps that update priorities
    idx = torch.empty(B, dtype=torch.int64, device=dev)
    start = torch.empty(B, dtype=torch.int32, device=dev)
    wts = torch.empty(B, dtype=torch.float32, device=dev)
    outs = [torch.empty(B * L * e, dtype=torch.uint8, device=dev) for e in w.elem_bytes]
    out_ptrs = [o.data_ptr() for o in outs]
    newp = torch.from_numpy(np.stack([gen.update_priorities(w.prio, w.seed, it, B) for it in range(W + K)])).to(dev)
    seeds = [gen.select_seed(w.seed, it) for it in range(W + K)]
    batch_bytes = B * L * sum(w.elem_bytes)

    def step(it):
        gear.gear_select(t.handle, strategy, B, L, seeds[it], w.beta, idx.data_ptr(), start.data_ptr(),
                         wts.data_ptr() if w.weights else 0, sh)
        if outs:
            gear.gear_collect(t.handle, idx.data_ptr(), start.data_ptr(), B, L, None, out_ptrs, sh)
        if prioritized:
            gear.gear_update_priorities(t.handle, idx.data_ptr(), newp[it].data_ptr(), B, sh)

    for it in range(W):
        step(it)
    torch.cuda.synchronize()
    if t.sync() != 0:
        raise SystemExit("device status set during warm-up")

    # Timed region: K whole steps; HIP events on the same stream bracket each
    # gather launch.
    hev = HipEvents()
    ev = [(hev.create(), hev.create()) for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        it = W + k
        gear.gear_select(t.handle, strategy, B, L, seeds[it], w.beta, idx.data_ptr(), start.data_ptr(),
                         wts.data_ptr() if w.weights else 0, sh)
        hev.record(ev[k][0], sh)
        if outs:
            gear.gear_collect(t.handle, idx.data_ptr(), start.data_ptr(), B, L, None, out_ptrs, sh)
        hev.record(ev[k][1], sh)
        if prioritized:
            gear.gear_update_priorities(t.handle, idx.data_ptr(), newp[it].data_ptr(), B, sh)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    status = t.sync()
    if status != 0:
        raise SystemExit("device status %d set during the timed steps" % status)
    wall = t1 - t0
    col_ms = float(np.mean([hev.elapsed_ms(a, b) for a, b in ev]))

    # Stage breakdown, after the timed region (events around every stage).
    nb = min(K, 50)
    sev = [[hev.create() for _ in range(4)] for _ in range(nb)]
    for k in range(nb):
        it = W + k
        e = sev[k]
        hev.record(e[0], sh)
        gear.gear_select(t.handle, strategy, B, L, seeds[it], w.beta, idx.data_ptr(), start.data_ptr(),
                         wts.data_ptr() if w.weights else 0, sh)
        hev.record(e[1], sh)
        if outs:
            gear.gear_collect(t.handle, idx.data_ptr(), start.data_ptr(), B, L, None, out_ptrs, sh)
        hev.record(e[2], sh)
        if prioritized:
            gear.gear_update_priorities(t.handle, idx.data_ptr(), newp[it].data_ptr(), B, sh)
        hev.record(e[3], sh)
    torch.cuda.synchronize()
    sel_all = [hev.elapsed_ms(e[0], e[1]) for e in sev]
    col_all = [hev.elapsed_ms(e[1], e[2]) for e in sev]
    upd_all = [hev.elapsed_ms(e[2], e[3]) for e in sev]
    sel_ms = float(np.mean(sel_all))
    upd_ms = float(np.mean(upd_all))
    pct = {name: [round(float(x), 5) for x in np.percentile(v, [10, 50, 90])]
           for name, v in (("select", sel_all), ("collect", col_all), ("update", upd_all))
           if name != "update" or prioritized}
    hev.close()

    if host_table:
        alg_bytes = batch_bytes                  # bytes crossing the host link
        peak, bound = HOST_LINK_PEAK_GBS, "host-link"
    else:
        alg_bytes = 2 * batch_bytes              # window bytes read + batch bytes written
        peak, bound = HBM_PEAK_GBS, "hbm"
    roof = None
    if outs:
        achieved = alg_bytes / (col_ms * 1e-3) / 1e9
        roof = {"bound": bound, "achieved": round(achieved, 1), "peak": peak, "unit": "GB/s",
                "frac": round(achieved / peak, 4),
                "traffic": profiled_traffic("collect_kernel", args.workload),
                "kernel": "collect_kernel", "algorithmic_bytes_per_launch": alg_bytes,
                "avg_launch_ms": round(col_ms, 5)}

    context = torch_context(t, w, dev) if strategy in (gear.GEAR_PRIORITIZED, gear.GEAR_TOPK) else None

    link = None
    if host_table and outs:
        link = host_link_extras(t, w, idx, start, outs, dev)
        if not link["cpu_staged"]["matches_zero_copy"]:
            raise SystemExit("the CPU-staged batch differs from the zero-copy batch")
        link["zero_copy_frac_of_h2d_copy"] = round(roof["achieved"] / link["link_h2d_copy_gbs"], 4)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args.cpu_seconds, args.global_min)

    steps_per_s = B * L * K / wall
    line = {
        "metric": METRIC, "value": round(steps_per_s, 1), "unit": "trajectory-steps/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(wall * 1e3 / K, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": w.name, "N": w.N, "T": w.T, "B": B, "L": L,
                   "columns": {c.name: "%s[%d]" % (c.dtype, c.m) for c in w.columns},
                   "elem_bytes": w.elem_bytes, "table_bytes": w.table_bytes,
                   "residency": "pinned-host" if host_table else "hbm",
                   "strategy": {0: "fifo", 1: "lifo", 2: "uniform", 3: "prioritized", 4: "topk"}[strategy],
                   "is_weights": bool(w.weights), "parallelism": "1 GPU",
                   "tree": "incremental" if args.incremental and not args.global_min else "rescan per select",
                   "is_normalisation": "table minimum" if args.global_min else "batch minimum"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "stages_ms": {"select": round(sel_ms, 5), "collect": round(col_ms, 5),
                      "update": round(upd_ms, 5) if prioritized else None,
                      "note": "select/update from a separate loop after the timed region"},
        "stages_ms_p10_p50_p90": pct,
        "selection_samples_per_s": round(B / (sel_ms * 1e-3), 1),
        "batch_bytes": batch_bytes,
    }
    if link is not None:
        line["host_link"] = link
    if context is not None:
        line["torch_context"] = context
    t.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
