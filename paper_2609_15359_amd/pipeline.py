"""One pass of the whole scheduler core over a batch: calibrate -> bound every
resident, arrival and queued request -> project -> place -> order.  Chains
the library calls of the binding; the tensors are only sliced, never computed
on here."""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

from . import (POLICY_MQ, Placement, Snapshot, calibrate, local_order, new_error_word, place, place_order,
               place_workspace_bytes, project, project_order)


@dataclass
class DeviceBatch:
    """A batch's arrays resident in device memory."""
    alpha_ppm: int
    u_max: int
    max_wait_ms: int
    cal_pred: torch.Tensor
    cal_truth: torch.Tensor
    edges: torch.Tensor
    apply_pred: torch.Tensor      # residents | arrivals | queued requests
    n_res: int
    n_arr: int
    seg_off: torch.Tensor
    res_prompt: torch.Tensor
    res_gen: torch.Tensor
    arr_prompt: torch.Tensor
    capacity: torch.Tensor
    queue_len: torch.Tensor
    q_off: torch.Tensor
    q_prompt: torch.Tensor
    q_wait_ms: torch.Tensor

    @property
    def decoders(self) -> int:
        return int(self.capacity.numel())


def to_device(batch, device="cuda") -> DeviceBatch:
    """Copy a host batch (numpy arrays, see workload.gen.Batch) to the device."""
    def t(x, dtype):
        return torch.from_numpy(np.ascontiguousarray(x)).to(device=device, dtype=dtype)
    i32, i64 = torch.int32, torch.int64
    return DeviceBatch(
        alpha_ppm=int(batch.alpha_ppm), u_max=int(batch.u_max), max_wait_ms=int(batch.max_wait_ms),
        cal_pred=t(batch.cal_pred, i32), cal_truth=t(batch.cal_truth, i32), edges=t(batch.edges, i32),
        apply_pred=t(batch.apply_pred(), i32), n_res=int(batch.res_pred.size),
        n_arr=int(batch.arr_pred.size), seg_off=t(batch.seg_off, i64),
        res_prompt=t(batch.res_prompt, i32), res_gen=t(batch.res_gen, i32),
        arr_prompt=t(batch.arr_prompt, i32), capacity=t(batch.capacity, i32),
        queue_len=t(batch.queue_len, i32), q_off=t(batch.q_off, i64),
        q_prompt=t(batch.q_prompt, i32), q_wait_ms=t(batch.q_wait_ms, i32))


@dataclass
class StepOutputs:
    q: torch.Tensor
    count: torch.Tensor
    U: torch.Tensor
    snapshot: Snapshot
    base_peak: torch.Tensor
    placement: Placement
    order: torch.Tensor
    admitted: torch.Tensor
    dev_err: torch.Tensor

    def bounds(self, db: DeviceBatch):
        """Views of U for residents, arrivals and queued requests."""
        nr, na = db.n_res, db.n_arr
        return self.U[:nr], self.U[nr:nr + na], self.U[nr + na:]


class Workspaces:
    """Device buffers reused across steps of one batch shape."""

    def __init__(self, db: DeviceBatch, want_pairs: bool = True):
        from . import library, snapshot_bytes
        dev = db.capacity.device
        D, A = db.decoders, db.n_arr
        nb = db.edges.numel() + 1
        lib = library()
        self.cal = torch.empty(max(int(lib.maps_calibrate_workspace_size(db.cal_pred.numel(), nb)), 1),
                               dtype=torch.uint8, device=dev)
        self.place = torch.empty(max(place_workspace_bytes(D, A, db.u_max), 1), dtype=torch.uint8,
                                 device=dev)
        self.snapshot = torch.empty(snapshot_bytes(D, db.n_res, db.u_max), dtype=torch.uint8, device=dev)
        self.out = {"q": torch.empty(nb, dtype=torch.int32, device=dev),
                    "count": torch.empty(nb, dtype=torch.int32, device=dev),
                    "U": torch.empty(db.apply_pred.numel(), dtype=torch.int32, device=dev)}
        self.base_peak = torch.empty(D, dtype=torch.int32, device=dev)
        self.dev_err = new_error_word(dev)
        self.placement = Placement(
            choice=torch.empty(A, dtype=torch.int32, device=dev),
            chosen_peak=torch.empty(A, dtype=torch.int32, device=dev),
            chosen_overflow=torch.empty(A, dtype=torch.int32, device=dev),
            flags=torch.empty(A, dtype=torch.uint8, device=dev),
            pair_peak=torch.empty((D, A), dtype=torch.int32, device=dev) if want_pairs else None,
            dev_err=self.dev_err)
        self.order = torch.empty(db.q_prompt.numel(), dtype=torch.int32, device=dev)
        self.admitted = torch.empty(D, dtype=torch.int32, device=dev)


PHASES = ("calibrate", "project", "place", "local_order")
# with placement and local order in one call (maps_place_order)
PHASES_FUSED = ("calibrate", "project", "place+local_order")
# with projection and local order in one call (maps_project_order), then placement
PHASES_PROJECT_ORDER = ("calibrate", "project+local_order", "place")


def phase_names(fused) -> tuple:
    return {False: PHASES, True: PHASES_FUSED, "project": PHASES_PROJECT_ORDER}[fused]


def step_phases(db: DeviceBatch, ws: Workspaces, want_pairs: bool = True, capacity=None,
                policy: int = POLICY_MQ, rr_offset: int = 0, fused: bool = False):
    """The step as one callable per phase (PHASES order; PHASES_FUSED with
    fused=True, PHASES_PROJECT_ORDER with fused="project").  Each enqueues its
    library calls on the current stream and writes only into `ws`, so a phase
    can also be captured into a graph and replayed."""
    cap = db.capacity if capacity is None else capacity
    err = ws.dev_err
    nr, na = db.n_res, db.n_arr
    U = ws.out["U"]
    snap = Snapshot(data=ws.snapshot, D=db.decoders, n_total=nr, u_max=db.u_max)

    def cal():
        calibrate(db.cal_pred, db.cal_truth, db.edges, db.alpha_ppm, db.apply_pred, db.u_max,
                  dev_err=err, workspace=ws.cal, out=ws.out)

    def proj():
        project(db.seg_off, db.res_prompt, db.res_gen, U[:nr], db.u_max, snapshot=ws.snapshot, dev_err=err,
                base_peak=ws.base_peak)

    def pla():
        place(snap, cap, db.queue_len, db.arr_prompt, U[nr:nr + na], policy=policy, rr_offset=rr_offset,
              want_pairs=want_pairs, workspace=ws.place, out=ws.placement)

    def loc():
        local_order(snap, cap, db.q_off, db.q_prompt, U[nr + na:], db.q_wait_ms, db.max_wait_ms, dev_err=err,
                    order=ws.order, admitted=ws.admitted)

    def pla_loc():
        place_order(snap, cap, db.queue_len, db.arr_prompt, U[nr:nr + na], db.q_off, db.q_prompt, U[nr + na:],
                    db.q_wait_ms, db.max_wait_ms, policy=policy, rr_offset=rr_offset, want_pairs=want_pairs,
                    workspace=ws.place, out=ws.placement, order=ws.order, admitted=ws.admitted)

    def proj_loc():
        project_order(db.seg_off, db.res_prompt, db.res_gen, U[:nr], db.u_max, cap, db.q_off, db.q_prompt,
                      U[nr + na:], db.q_wait_ms, db.max_wait_ms, snapshot=ws.snapshot, dev_err=err,
                      base_peak=ws.base_peak, order=ws.order, admitted=ws.admitted)

    if fused == "project":
        return [cal, proj_loc, pla]
    return [cal, proj, pla_loc] if fused else [cal, proj, pla, loc]


def outputs(db: DeviceBatch, ws: Workspaces) -> StepOutputs:
    """The step's results as they stand in `ws`."""
    return StepOutputs(q=ws.out["q"], count=ws.out["count"], U=ws.out["U"],
                       snapshot=Snapshot(data=ws.snapshot, D=db.decoders, n_total=db.n_res, u_max=db.u_max),
                       base_peak=ws.base_peak, placement=ws.placement, order=ws.order, admitted=ws.admitted,
                       dev_err=ws.dev_err)


def step(db: DeviceBatch, ws: Workspaces | None = None, want_pairs: bool = True, capacity=None,
         policy: int = POLICY_MQ, rr_offset: int = 0, fused: bool = False) -> StepOutputs:
    """Enqueue the whole hot path for one batch on the current stream."""
    ws = ws or Workspaces(db, want_pairs)
    for fn in step_phases(db, ws, want_pairs, capacity, policy, rr_offset, fused):
        fn()
    return outputs(db, ws)


class StepGraphs:
    """The step captured as one HIP graph per phase, then replayed on the
    current stream.  The phases run once eagerly first, so that every kernel
    attribute is set before capture; all buffers live in `ws`."""

    def __init__(self, db: DeviceBatch, ws: Workspaces, **kw):
        phases = step_phases(db, ws, **kw)
        self.n_phases = len(phases)
        for fn in phases:
            fn()
        torch.cuda.synchronize()
        self.graphs = []
        for fn in phases:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                fn()
            self.graphs.append(g)
        torch.cuda.synchronize()

    def replay(self, events=None):
        """One step; with events (one per phase plus one, None where no
        event is wanted), the phase boundaries are recorded on the current
        stream."""
        for i, g in enumerate(self.graphs):
            if events is not None and events[i] is not None:
                events[i].record()
            g.replay()
        if events is not None and events[-1] is not None:
            events[-1].record()
