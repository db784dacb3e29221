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
LEGS = ("window", "static", "blocks", "commit", "incremental", "appa", "record")
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
    import oracle
    o = oracle.Oracle()
    idx = np.arange(0, m, max(1, m // 30000))
    t0 = time.perf_counter()
    _, U_ref = o.calibrate_window(b.cal_pred, b.cal_truth, b.edges, WINDOW, b.alpha_ppm, ap[idx], seen[idx],
                                  b.u_max)
    dt = time.perf_counter() - t0
    if not np.array_equal(U.cpu().numpy()[idx], U_ref):
        raise SystemExit("window calibration differs from the oracle")
    out["verified"] = True
    out["verified_note"] = f"{idx.size} evenly spaced requests' bounds against the oracle"
    if cpu:
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
           "reserve_bound": "latency: a serial chain, each arrival's choice waits on the state its predecessors left",
           "reserve_feasible_fraction": feasible,
           "note": "independent: every arrival against the reported state; reserve: arrivals in order, each "
                   "reserving its B_need and joining the queue (a serial chain, one wavefront)"}
    import oracle
    o = oracle.Oracle()
    Ur, Ua = U_res.cpu().numpy(), U_arr.cpu().numpy()
    t0 = time.perf_counter()
    state_ref = o.rsc_state(b.seg_off, b.res_prompt, b.res_gen, Ur, b.capacity, BLOCK)
    t_rsc = time.perf_counter() - t0
    be = state_ref[2]
    k = min(A, 20000)
    t0 = time.perf_counter()
    o.place_static(be, b.queue_len, BLOCK, b.arr_prompt[:k], Ua[:k])
    t_ind = time.perf_counter() - t0
    t0 = time.perf_counter()
    res_ref = o.place_static(be, b.queue_len, BLOCK, b.arr_prompt, Ua, reserve=True)
    t_res = time.perf_counter() - t0
    # the last call made was the reserving one: its outputs, and the state, against the oracle
    for got, want in zip(list(st) + list(outs), list(state_ref) + list(res_ref)):
        if not np.array_equal(got.cpu().numpy().astype(np.int64), np.asarray(want).astype(np.int64)):
            raise SystemExit("Algorithm 1 on block counts differs from the oracle")
    out["verified"] = True
    out["verified_note"] = "the runtime state and every arrival of the reserving chain against the oracle"
    if cpu:
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
    # the slice arrays placement reads (rank words, residue maxima, class counts, sums, event records), not the
    # projection's own copies of tau, N, OB and the suffix maxima: 16 B per record slot, a decoder's slots
    # being its residents + 1 rounded up to a multiple of 4
    slots = ((np.diff(np.asarray(b.seg_off, dtype=np.int64)) + 1 + 3) // 4) * 4
    snap_read = snap.data.numel() - 16 * int(slots.sum())
    res = {"block_size": BLOCK, "decoders": D, "arrivals": A, "ms": ms,
           "pairs_per_s": D * A / (ms["place_blocks"] * 1e-3),
           "snapshot_mb": snap.data.numel() / 1e6,
           # the pair matrix written once, the snapshot arrays placement reads read once, 21 B per arrival in and out
           "roofline": _hbm_roofline(4 * D * A + snap_read + 21 * A, ms["place_blocks"],
                                     "maps_place_blocks (blocks_order, blocks_pairs, blocks_finish)"),
           "feasible_fraction": float(np.mean(out.flags.cpu().numpy() & 1)),
           "note": "peaks, capacities and overflow in blocks; the pair matrix always written; the block snapshot "
                   "is read through L2 (about 160 B per event at 16 tokens per block)"}
    import oracle
    o = oracle.Oracle()
    k = min(A, 65536)
    Ur, Ua = U_res.cpu().numpy(), U_arr.cpu().numpy()
    t0 = time.perf_counter()
    ref = o.place_blocks(b.seg_off, b.res_prompt, b.res_gen, Ur, b.capacity, b.queue_len, BLOCK, b.arr_prompt[:k],
                         Ua[:k], want_pairs=True)
    dt = time.perf_counter() - t0
    checks = ((out.choice[:k], ref.choice), (out.chosen_peak[:k], ref.chosen_peak),
              (out.chosen_overflow[:k], ref.chosen_overflow), (out.flags[:k], ref.flags),
              (out.pair_peak[:, :k], ref.pair_peak), (state["base"], ref.base_peak))
    for got, want in checks:
        if not np.array_equal(got.cpu().numpy().astype(np.int64), want.astype(np.int64)):
            raise SystemExit("placement in blocks differs from the oracle")
    res["verified"] = True
    res["verified_note"] = f"every output of the first {k} arrivals (their pair-matrix columns included) and the " \
                           "base peaks against the oracle"
    if cpu:
        res["cpu_baseline"] = {"value": D * k / dt, "unit": "pair-evaluations/s", "cores": 1, "kind": "oracle",
                               "sample": f"every decoder against the first {k} arrivals (dense occupancy in blocks "
                                         f"per decoder, then each pair), single-threaded C oracle, {dt:.2f} s"}
    return res


def _hbm_roofline(nbytes: int, ms: float, kernel: str) -> dict:
    achieved = nbytes / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "algorithmic_bytes": nbytes, "kernel": kernel}


def _median_ms(fn, calls: int, warm: int = 2) -> float:
    """Median over `calls` of fence-free HIP events around fn() on the current stream."""
    import torch
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    ev = [(TimingEvent(), TimingEvent()) for _ in range(calls)]
    for e0, e1 in ev:
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    return statistics.median(e0.elapsed_time(e1) for e0, e1 in ev)


def _walks(hdr, A: int, U_arr, groups: int = 8, tile: int = 8192):
    """How the placement kernel walks each (arrival tile, decoder group) of a
    launch with 8 groups and tiles of 8,192 arrivals, from the decoder headers
    (hot window, flat region start) and the tile's bound range: 'flat' needs
    no event data, 'hot' reads the rank word and PMX, 'full' also tests the
    thresholds (the rule of the kernel's tile choice, restated on the host)."""
    import numpy as np
    D = hdr.shape[0]
    Dg = (D + groups - 1) // groups
    out = {"flat": 0, "hot": 0, "full": 0}
    for g in range(groups):
        h = hdr[g * Dg:(g + 1) * Dg]
        if h.shape[0] == 0:
            continue
        lo, hi, fl = int(h[:, 6].max()), int(h[:, 7].min()), max(int(h[:, 8].max()), int(h[:, 6].max()))
        for a0 in range(0, A, tile):
            u = U_arr[a0:a0 + tile]
            if (u < 0).any():
                out["full"] += 1
                continue
            t_lo, t_hi = int(u.min()), int(u.max())
            if t_lo >= fl and t_hi <= hi:
                out["flat"] += 1
            elif t_lo >= lo and t_hi <= hi:
                out["hot"] += 1
            else:
                out["full"] += 1
    return out


def record_path(cpu: bool, calls: int = 20):
    """The general placement path at the headline shape: workload
    large_growing (256 decoders x 4,096 residents, 262,144 arrivals, the pair
    matrix written), whose decoders' occupancy peaks mid-horizon, so that
    tiles take the event-record walks.  The placement pass (maps_place_order)
    timed alone with HIP events on inputs already projected; its outputs are
    checked against the oracle's step on the same batch."""
    import numpy as np
    import torch

    import workload
    from paper_2609_15359_amd import pipeline
    b = workload.make("large_growing")
    D, A = b.decoders, b.arrivals
    db = pipeline.to_device(b)
    ws = pipeline.Workspaces(db, want_pairs=True)
    phases = pipeline.step_phases(db, ws, fused="project")
    for fn in phases:
        fn()
    torch.cuda.synchronize()
    if int(ws.dev_err.item()) != 0:
        raise SystemExit("large_growing raised device errors")
    ms = _median_ms(phases[2], calls)
    hdr = ws.snapshot[256:256 + 64 * D].view(torch.int32).view(D, 16).cpu().numpy()
    W = (((db.u_max + 1) // 32 + 1) + 1) & ~1
    nbytes = placement_bytes(D, A, db.u_max, W, hdr[:, 4])
    achieved = nbytes / (ms * 1e-3) / 1e9
    U_arr = ws.out["U"][db.n_res:db.n_res + db.n_arr].cpu().numpy()
    out = {"workload": f"large_growing: {workload.describe(b.workload)}; residents early in outputs of "
                       f"LN(8.5, 1.0) tokens, prompts LN(4, 1)", "decoders": D, "arrivals": A, "pairs": D * A,
           "place_ms": ms, "pairs_per_s": D * A / (ms * 1e-3),
           "mean_events_per_decoder": float(np.mean(hdr[:, 4])),
           "walks": _walks(hdr, A, U_arr),
           "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": achieved / HBM_PEAK_GBS, "traffic": recorded_traffic("large_growing"),
                        "algorithmic_bytes": nbytes,
                        "kernel": "maps_place (place_records, then place_finish)"}}
    import oracle
    o = oracle.Oracle()
    t0 = time.perf_counter()
    ref = oracle.step(b, o, want_pairs=True)
    dt = time.perf_counter() - t0
    out.update({k: v for k, v in verify_step(ws, ref).items() if k != "against"})
    if cpu:
        out["cpu_baseline"] = {"value": D * A / dt, "unit": "pair-evaluations/s", "cores": 1, "kind": "oracle",
                               "sample": f"one whole step of the single-threaded C oracle on the same batch, "
                                         f"{dt:.2f} s"}
    return out


def sequential_commit(b, db, snap, U_arr, ref, cpu: bool, k: int = 65536, check: int = 3000):
    """Placement with sequential commit on the headline batch: the first k
    arrivals in order, each committed to its decoder's projected occupancy
    and queue before the next (a serial chain: one workgroup).  The first
    `check` outputs are compared with the oracle, given the oracle's own
    bounds (later arrivals never change earlier ones)."""
    import numpy as np
    import torch

    import oracle
    import paper_2609_15359_amd as maps
    D = b.decoders
    ap = db.arr_prompt[:k].contiguous()
    aU = U_arr[:k].contiguous()
    err = maps.new_error_word()
    out = maps.CommitPlacement(choice=torch.empty(k, dtype=torch.int32, device="cuda"),
                               chosen_peak=torch.empty(k, dtype=torch.int64, device="cuda"),
                               chosen_overflow=torch.empty(k, dtype=torch.int64, device="cuda"),
                               flags=torch.empty(k, dtype=torch.uint8, device="cuda"),
                               queue_out=torch.empty(D, dtype=torch.int32, device="cuda"), dev_err=err)
    wsb = torch.empty(maps.place_commit_workspace_bytes(D, db.u_max), dtype=torch.uint8, device="cuda")
    fn = lambda: maps.place_commit(snap, db.capacity, db.queue_len, ap, aU, workspace=wsb, out=out)  # noqa: E731
    ms = _median_ms(fn, 3, warm=1)
    if int(err.item()) != 0:
        raise SystemExit(f"sequential commit raised {maps.error_names(int(err.item()))}")
    o = oracle.Oracle()
    Ur, Ua, _ = b.split_bounds(ref.U)
    t0 = time.perf_counter()
    r, _ = o.place_commit(b.seg_off, b.res_prompt, b.res_gen, Ur, b.capacity, b.queue_len, b.arr_prompt[:check],
                          Ua[:check])
    dt = time.perf_counter() - t0
    got = {"choice": out.choice, "chosen_peak": out.chosen_peak, "chosen_overflow": out.chosen_overflow,
           "flags": out.flags}
    for name, t in got.items():
        if not np.array_equal(t[:check].cpu().numpy().astype(np.int64), getattr(r, name).astype(np.int64)):
            print(f"bench.py: sequential commit's {name} differs from the oracle", file=sys.stderr)
            sys.exit(3)
    res = {"decoders": D, "arrivals": k, "ms": ms, "arrivals_per_s": k / (ms * 1e-3),
           "workspace_mb": wsb.numel() / 1e6, "verified": True,
           "bound": "latency: a serial chain, each arrival is evaluated against the curves its predecessors left",
           "verified_note": f"the first {check} arrivals' choices, peaks, overflows and flags against the oracle",
           "feasible_fraction": float(np.mean(out.flags.cpu().numpy() & 1)),
           "note": "arrivals in order; per arrival one peak lookup per decoder (dense curves plus block floors), "
                   "a workgroup argmin, then the commit on [0, U] of the chosen decoder: a serial chain"}
    if cpu:
        res["cpu_baseline"] = {"value": check / dt, "unit": "arrivals/s", "cores": 1, "kind": "oracle",
                               "sample": f"the first {check} arrivals of the same batch (dense curves rebuilt over "
                                         f"the whole step axis at every commit), single-threaded C oracle, "
                                         f"{dt:.2f} s"}
    return res


def appa_simulation(cpu: bool, rhos: int = 64):
    """App. A: 10,000 synthetic requests on N = 4 decoders of C = 50,000
    tokens, theta = 0.85, t_tok = 1 ms, round robin and Algorithm 1 routing
    at `rhos` utilisations from 0.5 to 1.3, all in one call (one wavefront
    per simulation); bounds from maps_calibrate on the workload's calibration
    pairs.  Four simulations are checked against the oracle."""
    import numpy as np
    import torch

    import oracle
    import paper_2609_15359_amd as maps
    import workload.appa as appa
    w = appa.make()
    dev = lambda x, t=torch.int32: torch.from_numpy(np.ascontiguousarray(x)).to(t).cuda()  # noqa: E731
    q, _, U, err = maps.calibrate(dev(w.cal_pred), dev(w.cal_truth), dev(w.edges), appa.ALPHA_PPM, dev(w.pred),
                                  appa.U_MAX)
    grid = np.linspace(0.5, 1.3, rhos)
    arr = np.stack([w.arrivals(r) for r in grid for _ in (0, 1)])
    pol = np.array([p for _ in grid for p in (0, 1)], np.int32)
    arr_d, pol_d, pr, ou = dev(arr, torch.int64), dev(pol), dev(w.prompt), dev(w.output)
    S = arr.shape[0]
    sim = maps.simulate(appa.N_DECODERS, appa.CAPACITY, appa.THETA_PPM, arr_d, pr, ou, U, pol_d, dev_err=err)
    wsb = torch.empty(maps.library().maps_simulate_workspace_size(appa.N_DECODERS, w.n, S), dtype=torch.uint8,
                      device="cuda")
    fn = lambda: maps.simulate(appa.N_DECODERS, appa.CAPACITY, appa.THETA_PPM, arr_d, pr, ou, U, pol_d,  # noqa
                               dev_err=err, workspace=wsb, out=sim)
    ms = _median_ms(fn, 3, warm=1)
    if int(err.item()) != 0:
        raise SystemExit(f"simulation raised {maps.error_names(int(err.item()))}")
    o = oracle.Oracle()
    qo, _ = o.calibrate(w.cal_pred, w.cal_truth, w.edges, appa.ALPHA_PPM)
    Uo = o.apply_bounds(w.pred, w.edges, qo, appa.U_MAX)
    fin = sim.finish_ms.cpu().numpy()
    st = sim.stats.cpu().numpy()
    span = sim.span.cpu().numpy()
    checked = [int(np.argmin(np.abs(grid - r))) * 2 + p for r in (0.96, 1.05) for p in (0, 1)]
    t0 = time.perf_counter()
    for s in checked:
        r = o.simulate(appa.N_DECODERS, appa.CAPACITY, appa.THETA_PPM, arr[s], w.prompt, w.output, Uo, int(pol[s]))
        ok = (np.array_equal(fin[s], r.finish_ms) and np.array_equal(st[s, 0], r.hp_time)
              and np.array_equal(st[s, 1], r.hp_max) and np.array_equal(st[s, 2], r.hp_count)
              and np.array_equal(st[s, 3], r.max_queue) and np.array_equal(st[s, 4], r.queue_area)
              and np.array_equal(span[s], r.span))
        if not ok:
            print(f"bench.py: simulation {s} differs from the oracle", file=sys.stderr)
            sys.exit(3)
    dt = (time.perf_counter() - t0) / len(checked)

    def summary(s):
        T = int(span[s, 1] - span[s, 0])
        lat = fin[s] - arr[s]
        return {"rho": round(float(grid[s // 2]), 3), "policy": ["round_robin", "algorithm1"][int(pol[s])],
                "f_hp": [round(float(x) / T, 4) for x in st[s, 0]], "B_hp_ms": st[s, 1].tolist(),
                "C_hp": st[s, 2].tolist(), "max_queue": st[s, 3].tolist(),
                "mean_e2e_ms": float(lat.mean()), "p99_e2e_ms": float(np.percentile(lat, 99))}
    res = {"simulations": S, "requests": w.n, "decoders": appa.N_DECODERS, "capacity": appa.CAPACITY,
           "theta": appa.THETA_PPM / 1e6, "ms": ms, "simulations_per_s": S / (ms * 1e-3),
           "bound": "latency: one wavefront per simulation, event after event",
           "simulated_requests_per_s": S * w.n / (ms * 1e-3), "verified": True,
           "verified_note": f"simulations {checked} (rho 0.96 and 1.05, both policies) against the oracle in full",
           "at": [summary(s) for s in checked],
           "note": "synthetic lognormal lengths stand in for BurstGPT; event to event per wavefront"}
    if cpu:
        res["cpu_baseline"] = {"value": 1.0 / dt, "unit": "simulations/s", "cores": 1, "kind": "oracle",
                               "sample": f"{len(checked)} of the simulations, one millisecond at a time, "
                                         f"single-threaded C oracle, {dt:.3f} s each"}
    return res


def incremental_window(b, ref, cpu: bool, batches: int = 64, window: int = 500):
    """The headline batch's 1,000,000 calibration pairs appended as a
    completion log in `batches` batches to the incremental window state
    (64 buckets, window 500), then the bounds of every resident, arrival and
    queued request from the state: each append and the bound call timed with
    HIP events.  The final bounds of a sample of requests are checked against
    the oracle's window calibration with every request having seen the log."""
    import numpy as np
    import torch

    import oracle
    import paper_2609_15359_amd as maps
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(torch.int32).cuda()  # noqa: E731
    pred, truth, ap = dev(b.cal_pred), dev(b.cal_truth), dev(b.apply_pred())
    n = pred.numel()
    cuts = np.linspace(0, n, batches + 1).astype(np.int64)
    st = maps.WindowState(dev(b.edges), window)
    U = torch.empty(ap.numel(), dtype=torch.int32, device="cuda")
    ws = torch.empty(maps.library().maps_window_append_workspace_size(int(cuts[1] - cuts[0]) + 1, st.nb),
                     dtype=torch.uint8, device="cuda")
    ev = [(TimingEvent(), TimingEvent()) for _ in range(batches)]
    st.reset()
    torch.cuda.synchronize()
    for j, (e0, e1) in enumerate(ev):
        e0.record()
        st.append(pred[cuts[j]:cuts[j + 1]], truth[cuts[j]:cuts[j + 1]], workspace=ws)
        e1.record()
    torch.cuda.synchronize()
    append_ms = statistics.median(e0.elapsed_time(e1) for e0, e1 in ev)
    bounds_ms = _median_ms(lambda: st.bounds(b.alpha_ppm, ap, b.u_max, U=U), 10)
    if int(st.dev_err.item()) != 0:
        raise SystemExit("incremental window raised device errors")
    o = oracle.Oracle()
    apn = b.apply_pred()
    idx = np.arange(0, apn.size, max(1, apn.size // 20000))
    t0 = time.perf_counter()
    _, Uo = o.calibrate_window(b.cal_pred, b.cal_truth, b.edges, window, b.alpha_ppm, apn[idx],
                               np.full(idx.size, n), b.u_max)
    dt = time.perf_counter() - t0
    if not np.array_equal(U.cpu().numpy()[idx], Uo):
        print("bench.py: incremental window bounds differ from the oracle", file=sys.stderr)
        sys.exit(3)
    m = apn.size
    res = {"log": n, "batches": batches, "batch_size": int(cuts[1] - cuts[0]), "buckets": st.nb, "window": window,
           "append_ms": append_ms, "appended_per_s": (cuts[1] - cuts[0]) / (append_ms * 1e-3),
           "bounds_ms": bounds_ms, "requests": m, "bounds_per_s": m / (bounds_ms * 1e-3),
           # the bounds call: prediction in, bound out per request, every ring slot read once
           "roofline": _hbm_roofline(8 * m + 4 * st.nb * window, bounds_ms,
                                     "maps_window_bounds (win_select, win_bounds)"),
           "verified": True,
           "verified_note": f"{idx.size} evenly spaced requests' bounds after the last batch against the oracle"}
    if cpu:
        res["cpu_baseline"] = {"value": idx.size / dt, "unit": "requests/s", "cores": 1, "kind": "oracle",
                               "sample": f"{idx.size} requests, each calibrated on the last {window} completions of "
                                         f"its bucket (a sort per request), single-threaded C oracle, {dt:.2f} s"}
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
    ap.add_argument("--legs", default="all", help="comma-separated legs to run after the step ("
                    + ", ".join(LEGS) + "), 'all' or 'none' (for profiling the step alone)")
    args = ap.parse_args()
    legs = set(LEGS) if args.legs == "all" else set() if args.legs == "none" else set(args.legs.split(","))
    if legs - set(LEGS):
        ap.error(f"unknown legs: {sorted(legs - set(LEGS))}")
    if args.gpus != 1:
        print(f"bench.py: one GPU only (--gpus {args.gpus} requested); placement would shard by arrivals, "
              "each GPU holding a replica of the snapshot, but no multi-GPU path is built", file=sys.stderr)
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
    # projection and local order in one call (each decoder's workgroup orders
    # its queue after projecting it), then placement
    phases = pipeline.step_phases(db, ws, fused="project")
    names = pipeline.PHASES_PROJECT_ORDER

    ws.dev_err.zero_()
    for fn in phases:   # one eager step: the reference for the replayed graphs
        fn()
    eager = (ws.placement.choice.clone(), ws.placement.pair_peak.sum(dtype=torch.int64), ws.order.clone())
    graphs = pipeline.StepGraphs(db, ws, fused="project") if args.graph else None

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
                     "kernel": "maps_place (place_records, then place_finish: each arrival's best group); "
                               "the local orders run inside the projection's launch (maps_project_order)",
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
    # the next rows on the path, on the same batch
    cpu = not args.no_cpu_baseline
    nr, na = db.n_res, db.n_arr
    U_res, U_arr = ws.out["U"][:nr], ws.out["U"][nr:nr + na]
    if "window" in legs:
        result["window_calibration"] = window_calibration(b, cpu=cpu)
    if "static" in legs:
        result["static_placement"] = static_placement(b, db, U_res, U_arr, cpu=cpu)
    if "blocks" in legs:
        result["block_placement"] = block_placement(b, db, U_res, U_arr, cpu=cpu)
    if "commit" in legs:
        snap = maps.Snapshot(data=ws.snapshot, D=D, n_total=nr, u_max=db.u_max)
        result["sequential_commit"] = sequential_commit(b, db, snap, U_arr, ref, cpu=cpu)
    if "incremental" in legs:
        result["incremental_window"] = incremental_window(b, ref, cpu=cpu)
    if "appa" in legs:
        result["appa_simulation"] = appa_simulation(cpu=cpu)
    if "record" in legs:
        result["record_path"] = record_path(cpu=cpu)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
