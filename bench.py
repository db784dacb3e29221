"""Benchmark of the MAPS scheduler core on one MI355X.

One step = the whole hot path over one batch already resident in HBM:
calibrate (per-bucket conformal quantiles and the bound of every resident,
arrival and queued request) -> project (occupancy snapshot of every decoder)
-> place (every arrival x decoder peak, with the per-pair peak matrix written,
and the choice per arrival) -> local order (queue order and admitted prefix).

Prints one JSON line: arrival x decoder placement evaluations per second over
the whole step, the placement pass against the HBM roofline (algorithmic
bytes / its HIP-event time), and the CPU oracle timed on the host as a
baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, vendor figure
DEFAULT_WORKLOAD = "large"     # 256 decoders x 4096 residents, 262,144 arrivals
PLACE_SAMPLE = 5               # placement bracketed by timing events on every 5th timed step
BREAKDOWN_STEPS = 10           # untimed steps with an event at every phase boundary
PLACEMENT_SOURCES = ("paper_2609_15359_amd/csrc/place.hip", "paper_2609_15359_amd/csrc/maps_internal.hpp",
                     "paper_2609_15359_amd/csrc/order_core.hpp")


def placement_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in PLACEMENT_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic(workload_name: str):
    """HBM bytes of one placement pass from the committed counter summary
    (FETCH_SIZE and WRITE_SIZE, scaled by a plain copy of known size), or None
    when there is none for this workload or the placement code changed since."""
    path = os.path.join(ROOT, "profiles", f"place_traffic_{workload_name}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256") != placement_source_hash():
        return None
    return rec.get("placement_bytes")


def placement_bytes(D: int, A: int, u_max: int, W: int, events) -> int:
    """Algorithmic bytes of one placement pass: every input read once and
    every output written once.  Pair matrix 4 B/pair; arrivals 8 B in and
    13 B out (choice, peak, overflow, flags); per decoder its header, capacity
    and queue length, and its dense profile (4 B per entry, u_max + 1 entries
    rounded up to 4) or, for bounds too long for a profile, its rank words
    (8 B each) and its E+1 records (16 B each)."""
    P = (u_max + 4) & ~3 if u_max + 1 <= 16384 else 0
    if P:
        snap = D * (4 * P + 32 + 8)
    else:
        snap = sum(8 * W + 16 * (int(e) + 1) + 32 + 8 for e in events)
    return 4 * D * A + (8 + 13) * A + snap


def cpu_baseline(batch, budget_s: float = 20.0):
    """The single-threaded C oracle's whole step on the same batch, timed; also
    returns its last result, which the timed GPU step is checked against."""
    import oracle
    o = oracle.Oracle()
    t0 = time.perf_counter()
    runs = 0
    while True:
        ref = oracle.step(batch, o, want_pairs=True)
        runs += 1
        if time.perf_counter() - t0 > budget_s / 2 or runs >= 5:
            break
    dt = (time.perf_counter() - t0) / runs
    pairs = batch.decoders * batch.arrivals
    out = {"value": pairs / dt, "unit": "pair-evaluations/s", "cores": 1, "kind": "oracle",
           "sample": f"the full workload, {runs} step(s) of the single-threaded C oracle "
                     f"(calibrate, bound, project, place with pair matrix, local order), "
                     f"{dt * 1e3:.1f} ms per step"}
    out["all_cores"] = cpu_placement_all_cores(batch, o)
    return out, ref


def verify_step(ws, ref) -> dict:
    """Every output of the timed GPU step against the oracle's step on the same
    batch, element by element (all are integers): quantiles, counts, bounds,
    base peaks, choices, chosen peaks, overflows, flags, the whole pair-peak
    matrix, local orders and admitted prefixes.  Exits non-zero on any
    difference."""
    import numpy as np
    got = {"q": ws.out["q"], "count": ws.out["count"], "U": ws.out["U"], "base_peak": ws.base_peak,
           "choice": ws.placement.choice, "chosen_peak": ws.placement.chosen_peak,
           "chosen_overflow": ws.placement.chosen_overflow, "flags": ws.placement.flags,
           "pair_peak": ws.placement.pair_peak, "order": ws.order, "admitted": ws.admitted}
    want = {"q": ref.q, "count": ref.count, "U": ref.U, "base_peak": ref.base_peak, "choice": ref.place.choice,
            "chosen_peak": ref.place.chosen_peak, "chosen_overflow": ref.place.chosen_overflow,
            "flags": ref.place.flags, "pair_peak": ref.place.pair_peak, "order": ref.order,
            "admitted": ref.admitted}
    compared = 0
    for k, t in got.items():
        g = t.cpu().numpy().astype(np.int64)
        w = np.asarray(want[k]).astype(np.int64)
        if g.shape != w.shape or not np.array_equal(g, w):
            bad = int(np.count_nonzero(g != w)) if g.shape == w.shape else -1
            print(f"bench.py: the timed step's {k} differs from the oracle ({bad} entries)", file=sys.stderr)
            sys.exit(3)
        compared += g.size
    return {"verified": True, "entries_compared": compared,
            "against": "the C oracle's step on the same batch (every output, the pair matrix included)"}


def cpu_placement_all_cores(batch, o, max_threads: int = 16):
    """The oracle's placement pass (every pair peak and every choice; the pair
    matrix itself not kept, so that page faults of a fresh 0.5 GB array do not
    dominate) on one thread, then split over decoders across the host's cores:
    one thread per shard of decoders, each a call of the same single-threaded
    C oracle (ctypes releases the interpreter lock during the call)."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    threads = max(1, min(max_threads, len(os.sched_getaffinity(0))))
    U = oracle.step(batch, o, want_pairs=False).U
    U_res, U_arr, _ = batch.split_bounds(U)

    def run(ds):
        lo, hi = int(batch.seg_off[ds[0]]), int(batch.seg_off[ds[-1] + 1])
        seg = batch.seg_off[ds[0]:ds[-1] + 2] - lo
        o.place(seg, batch.res_prompt[lo:hi], batch.res_gen[lo:hi], U_res[lo:hi], batch.capacity[ds],
                batch.queue_len[ds], batch.arr_prompt, U_arr, want_pairs=False)

    t0 = time.perf_counter()
    run(np.arange(batch.decoders))
    t1 = time.perf_counter() - t0
    shards = [s for s in np.array_split(np.arange(batch.decoders), threads) if s.size]
    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(run, shards))
    tn = time.perf_counter() - t0
    pairs = batch.decoders * batch.arrivals
    return {"value": pairs / tn, "unit": "pair-evaluations/s", "cores": threads, "kind": "oracle",
            "one_core_value": pairs / t1,
            "sample": f"the placement pass alone (every pair peak and choice, the pair matrix not kept) on the full "
                      f"workload: {t1 * 1e3:.1f} ms on one thread, {tn * 1e3:.1f} ms with the decoders split into "
                      f"{len(shards)} shards on {threads} threads"}


WINDOW = 500   # Sec. 4: calibration over a sliding window of the 500 most recent requests


def window_calibration(b, cpu: bool, calls: int = 20):
    """Sliding-window calibration of every bounded request of the batch
    (maps_calibrate_window, window 500): residents bounded at earlier points of
    the completion log, arrivals and queued requests after all of it.  Timed
    with fence-free HIP events around each call, inputs resident in HBM."""
    import numpy as np
    import torch

    import workload
    import paper_2609_15359_amd as maps
    ap = b.apply_pred()
    seen = workload.window_seen(b)
    dev = lambda x, t=torch.int32: torch.from_numpy(np.ascontiguousarray(x)).to(t).cuda()  # noqa: E731
    pred, truth, edges, apd, sn = dev(b.cal_pred), dev(b.cal_truth), dev(b.edges), dev(ap), dev(seen, torch.int64)
    n, nb, m = pred.numel(), edges.numel() + 1, apd.numel()
    ws = torch.empty(maps.calibrate_window_workspace_bytes(n, nb), dtype=torch.uint8, device="cuda")
    U = torch.empty(m, dtype=torch.int32, device="cuda")
    err = maps.new_error_word()

    def call():
        maps.calibrate_window(pred, truth, edges, WINDOW, b.alpha_ppm, apd, sn, b.u_max, dev_err=err,
                              workspace=ws, U=U, want_q=False)
    for _ in range(3):
        call()
    torch.cuda.synchronize()
    ev = [(TimingEvent(), TimingEvent()) for _ in range(calls)]
    for e0, e1 in ev:
        e0.record()
        call()
        e1.record()
    torch.cuda.synchronize()
    ms = statistics.median(e0.elapsed_time(e1) for e0, e1 in ev)
    if int(err.item()) != 0:
        raise SystemExit(f"window calibration raised {maps.error_names(int(err.item()))}")
    nbytes = 8 * n + 16 * m   # log (pred, truth) in; per request pred and seen in, bound out
    out = {"log": n, "buckets": nb, "window": WINDOW, "requests": m, "ms": ms, "requests_per_s": m / (ms * 1e-3),
           "roofline": {"bound": "hbm", "achieved": nbytes / (ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": nbytes},
           "note": "median of per-call HIP events over the five launches of one call"}
    if cpu:
        import oracle
        o = oracle.Oracle()
        idx = np.arange(0, m, max(1, m // 30000))
        t0 = time.perf_counter()
        o.calibrate_window(b.cal_pred, b.cal_truth, b.edges, WINDOW, b.alpha_ppm, ap[idx], seen[idx], b.u_max)
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": idx.size / dt, "unit": "requests/s", "cores": 1, "kind": "oracle",
                               "sample": f"{idx.size} evenly spaced requests of the same batch, single-threaded C "
                                         f"oracle (each request's window sorted), {dt:.2f} s"}
    return out


BLOCK = 16     # tokens per KV block for Algorithm 1 on block counts (PagedAttention's default block)


def static_placement(b, db, U_res, U_arr, cpu: bool, calls: int = 10):
    """Algorithm 1 on block counts for the batch: the runtime state from the
    residents, then every arrival against it (independent) and one after
    another with reservation.  HIP events around each call."""
    import numpy as np
    import torch

    import paper_2609_15359_amd as maps
    D, A = b.decoders, b.arrivals
    n = int(db.seg_off[-1].item())
    err = maps.new_error_word()
    st = [torch.empty(D, dtype=torch.int64, device="cuda") for _ in range(3)]
    outs = (torch.empty(A, dtype=torch.int32, device="cuda"), torch.empty(A, dtype=torch.int64, device="cuda"),
            torch.empty(A, dtype=torch.uint8, device="cuda"), torch.empty(D, dtype=torch.int64, device="cuda"),
            torch.empty(D, dtype=torch.int32, device="cuda"))
    calls_of = {
        "rsc_state": lambda: maps.rsc_state(db.seg_off, db.res_prompt, db.res_gen, U_res, db.capacity, BLOCK,
                                            dev_err=err, out=st),
        "independent": lambda: maps.place_static(st[2], db.queue_len, BLOCK, db.arr_prompt, U_arr, dev_err=err,
                                                 out=outs),
        "reserve": lambda: maps.place_static(st[2], db.queue_len, BLOCK, db.arr_prompt, U_arr, reserve=True,
                                             dev_err=err, out=outs),
    }
    ms = {}
    for name, fn in calls_of.items():
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        ev = [(TimingEvent(), TimingEvent()) for _ in range(calls if name != "reserve" else 3)]
        for e0, e1 in ev:
            e0.record()
            fn()
            e1.record()
        torch.cuda.synchronize()
        ms[name] = statistics.median(e0.elapsed_time(e1) for e0, e1 in ev)
    if int(err.item()) != 0:
        raise SystemExit(f"static placement raised {maps.error_names(int(err.item()))}")
    feasible = float(np.mean(outs[2].cpu().numpy() & 1))
    out = {"block_size": BLOCK, "decoders": D, "arrivals": A, "residents": n, "ms": ms,
           "independent_pairs_per_s": D * A / (ms["independent"] * 1e-3),
           "reserve_arrivals_per_s": A / (ms["reserve"] * 1e-3),
           "reserve_feasible_fraction": feasible,
           "note": "independent: every arrival against the reported state; reserve: arrivals in order, each "
                   "reserving its B_need and joining the queue (a serial chain, one wavefront)"}
    if cpu:
        import oracle
        o = oracle.Oracle()
        Ur, Ua = U_res.cpu().numpy(), U_arr.cpu().numpy()
        t0 = time.perf_counter()
        _, _, be = o.rsc_state(b.seg_off, b.res_prompt, b.res_gen, Ur, b.capacity, BLOCK)
        t_rsc = time.perf_counter() - t0
        k = min(A, 20000)
        t0 = time.perf_counter()
        o.place_static(be, b.queue_len, BLOCK, b.arr_prompt[:k], Ua[:k])
        t_ind = time.perf_counter() - t0
        t0 = time.perf_counter()
        o.place_static(be, b.queue_len, BLOCK, b.arr_prompt, Ua, reserve=True)
        t_res = time.perf_counter() - t0
        out["cpu_baseline"] = {"rsc_state_ms": t_rsc * 1e3, "independent_pairs_per_s": D * k / t_ind,
                               "reserve_arrivals_per_s": A / t_res, "cores": 1, "kind": "oracle",
                               "sample": f"runtime state of all {n} residents; {k} arrivals independent; all {A} "
                                         "arrivals with reservation; single-threaded C oracle"}
    return out


def block_placement(b, db, U_res, U_arr, cpu: bool, calls: int = 10):
    """Projected placement in blocks of BLOCK tokens for the batch: the block
    snapshot of every decoder, then every pair's peak in blocks (the matrix
    written) and the choices.  HIP events around each call."""
    import numpy as np
    import torch

    import paper_2609_15359_amd as maps
    D, A = b.decoders, b.arrivals
    err = maps.new_error_word()
    state = {}

    def proj():
        state["snap"], state["base"], _ = maps.project_blocks(db.seg_off, db.res_prompt, db.res_gen, U_res, db.u_max,
                                                              BLOCK, dev_err=err, base_peak=state.get("base"))
    proj()
    out = maps.Placement(choice=torch.empty(A, dtype=torch.int32, device="cuda"),
                         chosen_peak=torch.empty(A, dtype=torch.int32, device="cuda"),
                         chosen_overflow=torch.empty(A, dtype=torch.int32, device="cuda"),
                         flags=torch.empty(A, dtype=torch.uint8, device="cuda"),
                         pair_peak=torch.empty((D, A), dtype=torch.int32, device="cuda"), dev_err=err)
    snap = state["snap"]

    def project_again():   # into the same buffers: no allocation in the timed call
        maps.project_blocks(db.seg_off, db.res_prompt, db.res_gen, U_res, db.u_max, BLOCK, dev_err=err,
                            base_peak=state["base"], snapshot=snap)

    calls_of = {"project_blocks": project_again,
                "place_blocks": lambda: maps.place_blocks(snap, db.capacity, db.queue_len, db.arr_prompt, U_arr,
                                                          dev_err=err, out=out)}
    ms = {}
    for name, fn in calls_of.items():
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        ev = [(TimingEvent(), TimingEvent()) for _ in range(calls)]
        for e0, e1 in ev:
            e0.record()
            fn()
            e1.record()
        torch.cuda.synchronize()
        ms[name] = statistics.median(e0.elapsed_time(e1) for e0, e1 in ev)
    if int(err.item()) != 0:
        raise SystemExit(f"block placement raised {maps.error_names(int(err.item()))}")
    res = {"block_size": BLOCK, "decoders": D, "arrivals": A, "ms": ms,
           "pairs_per_s": D * A / (ms["place_blocks"] * 1e-3),
           "snapshot_mb": snap.data.numel() / 1e6,
           "feasible_fraction": float(np.mean(out.flags.cpu().numpy() & 1)),
           "note": "peaks, capacities and overflow in blocks; the pair matrix always written; the block snapshot "
                   "is read through L2 (about 150 B per event at 16 tokens per block)"}
    if cpu:
        import oracle
        o = oracle.Oracle()
        k = min(A, 65536)
        Ur, Ua = U_res.cpu().numpy(), U_arr.cpu().numpy()
        t0 = time.perf_counter()
        o.place_blocks(b.seg_off, b.res_prompt, b.res_gen, Ur, b.capacity, b.queue_len, BLOCK, b.arr_prompt[:k],
                       Ua[:k], want_pairs=True)
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": D * k / dt, "unit": "pair-evaluations/s", "cores": 1, "kind": "oracle",
                               "sample": f"every decoder against the first {k} arrivals (dense occupancy in blocks "
                                         f"per decoder, then each pair), single-threaded C oracle, {dt:.2f} s"}
    return res


class TimingEvent:
    """A HIP event made only for timing: created with hipEventDisableSystemFence,
    so recording it costs no system-scope cache write-back and invalidation
    (which, recorded between kernels, adds microseconds to what it brackets).
    Recorded on torch's current stream through the HIP runtime torch loaded."""

    _hip = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        import ctypes
        if TimingEvent._hip is None:
            TimingEvent._hip = ctypes.CDLL("libamdhip64.so")
        self._ev = ctypes.c_void_p()
        rc = TimingEvent._hip.hipEventCreateWithFlags(ctypes.byref(self._ev), ctypes.c_uint(self.DISABLE_SYSTEM_FENCE))
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")

    def record(self):
        import ctypes
        import torch
        rc = TimingEvent._hip.hipEventRecord(self._ev, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_time(self, end: "TimingEvent") -> float:
        """Milliseconds from this event to `end` (both recorded and complete)."""
        import ctypes
        ms = ctypes.c_float()
        if TimingEvent._hip.hipEventSynchronize(end._ev) != 0:
            raise RuntimeError("hipEventSynchronize failed")
        rc = TimingEvent._hip.hipEventElapsedTime(ctypes.byref(ms), self._ev, end._ev)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(ms.value)


def copy_probe(nbytes: int):
    """A plain device copy of known size (for scaling HBM byte counters)."""
    import torch
    src = torch.empty(nbytes // 4, dtype=torch.int32, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0, help="run only a plain copy of this many bytes")
    ap.add_argument("--window-only", action="store_true", help="run only the sliding-window calibration leg "
                                                               "(for profiling its kernels)")
    ap.add_argument("--graph", action="store_true", help="replay one HIP graph per phase instead of "
                                                         "launching every kernel from the host")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (--gpus {args.gpus} requested); "
              "the multi-GPU split is described in DESIGN.md", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return

    import numpy as np
    import torch

    import workload
    import paper_2609_15359_amd as maps
    from paper_2609_15359_amd import pipeline

    b = workload.make(args.workload)
    if args.window_only:
        print(json.dumps({"window_calibration": window_calibration(b, cpu=False)}), flush=True)
        return
    D, A = b.decoders, b.arrivals
    db = pipeline.to_device(b)
    ws = pipeline.Workspaces(db, want_pairs=True)
    # placement and local order in one call: the final selection and the
    # local orders share a launch
    phases = pipeline.step_phases(db, ws, fused=True)
    names = pipeline.PHASES_FUSED

    ws.dev_err.zero_()
    for fn in phases:   # one eager step: the reference for the replayed graphs
        fn()
    eager = (ws.placement.choice.clone(), ws.placement.pair_peak.sum(dtype=torch.int64), ws.order.clone())
    graphs = pipeline.StepGraphs(db, ws, fused=True) if args.graph else None

    def one_step(ev=None, place_ev=None):
        """One step; `ev` brackets every phase, `place_ev` only placement.
        Timing events are created without the system-scope fence."""
        if graphs is not None:
            graphs.replay(ev if ev else ([None, None, place_ev[0], place_ev[1]] if place_ev else None))
            return
        for i, fn in enumerate(phases):
            if ev:
                ev[i].record()
            if place_ev and i == 2:
                place_ev[0].record()
            fn()
            if place_ev and i == 2:
                place_ev[1].record()
        if ev:
            ev[-1].record()

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    bits = int(ws.dev_err.item()) & 0xFFFFFFFF
    if bits:
        raise SystemExit(f"device value errors: {maps.error_names(bits)}")

    # timed region: exactly K steps, bracketed by synchronization.  Placement
    # is bracketed by timing events on every PLACE_SAMPLE-th step (the
    # roofline's kernel time, measured live); the per-phase breakdown is
    # taken after the timed region, so that its events do not slow the steps
    # that are timed.
    sampled = [k for k in range(args.steps) if k % PLACE_SAMPLE == 0]
    place_events = {k: (TimingEvent(), TimingEvent()) for k in sampled}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        one_step(place_ev=place_events.get(k))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    if not (torch.equal(eager[0], ws.placement.choice) and torch.equal(eager[2], ws.order)
            and int(eager[1]) == int(ws.placement.pair_peak.sum(dtype=torch.int64))):
        raise SystemExit("replayed steps differ from the eager step")
    place_ms = statistics.mean(a.elapsed_time(b) for a, b in place_events.values())
    events = [[TimingEvent() for _ in range(len(names) + 1)] for _ in range(BREAKDOWN_STEPS)]
    for ev in events:
        one_step(ev)
    torch.cuda.synchronize()
    parts = {name: statistics.median(ev[i].elapsed_time(ev[i + 1]) for ev in events)
             for i, name in enumerate(names)}

    # algorithmic bytes of the placement pass, from the snapshot's own event counts
    hdr = ws.snapshot[256:256 + 64 * D].view(torch.int32).view(D, 16).cpu().numpy()
    events_per_decoder = hdr[:, 4]
    W = (((db.u_max + 1) // 32 + 1) + 1) & ~1
    nbytes = placement_bytes(D, A, db.u_max, W, events_per_decoder)
    achieved = nbytes / (place_ms * 1e-3) / 1e9
    feasible = float(np.mean(ws.placement.flags.cpu().numpy() & 1))

    result = {
        "metric": "arrival x decoder peak-KV placement evals/sec",
        "value": D * A / (ms_per_step * 1e-3),
        "unit": "pair-evaluations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": f"{b.workload.name}: {workload.describe(b.workload)}; "
                               f"capacities {list(b.workload.capacities)} tokens, alpha_ppm {b.alpha_ppm}, "
                               f"u_max {b.u_max}; per-pair peak matrix written",
                   "decoders": D, "arrivals": A, "pairs": D * A,
                   "launch": "one HIP graph per phase" if args.graph else "host launches"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": recorded_traffic(args.workload),
                     "kernel": "maps_place_order (place_records, then place_finish_order: placement's final "
                               "selection and every local order in one launch)",
                     "algorithmic_bytes": nbytes, "place_ms": place_ms},
        "breakdown_ms": parts,
        "breakdown_note": f"median of {BREAKDOWN_STEPS} untimed steps with a timing event (no system "
                          "fence) at every phase boundary",
        "place_samples": len(place_events),
        "mean_events_per_decoder": float(np.mean(events_per_decoder)),
        "feasible_fraction": feasible,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"], ref = cpu_baseline(b)
    else:
        import oracle
        ref = oracle.step(b, oracle.Oracle(), want_pairs=True)
    # the outputs of the last timed step (the breakdown steps rewrote the same values)
    result.update(verify_step(ws, ref))
    # the next rows on the path: sliding-window calibration and Algorithm 1 on block counts, same batch
    result["window_calibration"] = window_calibration(b, cpu=not args.no_cpu_baseline)
    nr, na = db.n_res, db.n_arr
    result["static_placement"] = static_placement(b, db, ws.out["U"][:nr], ws.out["U"][nr:nr + na],
                                                  cpu=not args.no_cpu_baseline)
    result["block_placement"] = block_placement(b, db, ws.out["U"][:nr], ws.out["U"][nr:nr + na],
                                                cpu=not args.no_cpu_baseline)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
