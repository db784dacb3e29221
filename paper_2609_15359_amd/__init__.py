"""Python binding of the MAPS scheduler core for MI355X (gfx950).

Thin ctypes front end of ``libmaps.so`` (C ABI in ``include/maps.h``): every
function below marshals torch device tensors into the library call of the same
name and enqueues it on the current HIP stream.  All computation happens in
the library's HIP kernels; there is no CPU path.  PyTorch only supplies device
memory and the stream.

Steps (paper sections): calibrate -- Sec. 3.2 (uncertainty-aware calibration);
project -- Sec. 3.3 / App. A (KV occupancy projection); place -- Sec. 3.3,
Algorithm 1 (global memory-aware placement); local_order -- Sec. 3.3, Eq. (7)
(local SJF order with starvation promotion and admission).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(HERE, "libmaps.so")

Q_INF = 2**31 - 1
POLICY_MQ, POLICY_MC = 0, 1
MAX_LOCAL_QUEUE = 2048
ERR_BITS = {
    1: "NEG_LEN", 2: "EDGES_UNSORTED", 4: "INT32_RANGE", 8: "SEG_OFFSETS",
    16: "BOUND_RANGE", 32: "SNAPSHOT", 64: "QUEUE_TOO_LONG", 128: "TOO_MANY", 256: "WAIT_TIMEOUT",
    512: "SEEN_RANGE", 1024: "BLOCK_RANGE", 2048: "SIM_INPUT", 4096: "SIM_READY",
}
MAX_RESERVE_DECODERS = 1024
MAX_BLOCKS_U_MAX = 131072
MAX_BLOCK_SIZE = 64
MAX_WINDOW = 4096
MAX_WINDOW_BUCKETS = 1024
MAX_U_MAX = (1 << 24) - 64
MAX_SIM_DECODERS = 8
MAX_SIM_READY = 1024
MAX_COMMIT_DECODERS = 8192
MAX_COMMIT_U_MAX = 1 << 20


class MapsError(RuntimeError):
    """A library call returned a negative status or flagged a value error."""


_c = ctypes
_vp, _i32, _i64, _sz = _c.c_void_p, _c.c_int32, _c.c_int64, _c.c_size_t
_SIGNATURES = {
    "maps_calibrate_workspace_size": (_sz, [_i64, _i32]),
    "maps_calibrate": (_i32, [_vp, _vp, _i64, _vp, _i32, _i32, _vp, _vp, _vp, _i64, _i32, _vp,
                              _vp, _vp, _sz, _vp]),
    "maps_calibrate_window_workspace_size": (_sz, [_i64, _i32]),
    "maps_calibrate_window": (_i32, [_vp, _vp, _i64, _vp, _i32, _i32, _i32, _vp, _vp, _i64, _i32, _vp, _vp,
                                     _vp, _vp, _sz, _vp]),
    "maps_blocks_snapshot_bytes": (_sz, [_i32, _i64, _i32, _i32]),
    "maps_project_blocks": (_i32, [_i32, _vp, _vp, _vp, _vp, _i64, _i32, _i32, _vp, _sz, _vp, _vp, _vp]),
    "maps_place_blocks": (_i32, [_vp, _vp, _i32, _i64, _i32, _i32, _vp, _vp, _vp, _vp, _i64, _i32, _i64, _vp, _vp,
                                 _vp, _vp, _vp, _vp, _vp]),
    "maps_rsc_state": (_i32, [_i32, _vp, _i64, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _vp]),
    "maps_place_static": (_i32, [_i32, _vp, _vp, _i32, _vp, _vp, _i64, _i32, _i64, _i32, _vp, _vp, _vp, _vp, _vp,
                                 _vp, _vp]),
    "maps_snapshot_bytes": (_sz, [_i32, _i64, _i32]),
    "maps_project_workspace_size": (_sz, [_i32, _i64, _i32]),
    "maps_project": (_i32, [_i32, _vp, _i64, _vp, _vp, _vp, _i32, _vp, _sz, _vp, _vp, _vp, _sz, _vp]),
    "maps_place_workspace_size": (_sz, [_i32, _i64, _i32]),
    "maps_place": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _vp, _i64, _i32, _i64, _vp, _vp, _vp, _vp,
                          _vp, _vp, _vp, _sz, _vp]),
    "maps_local_order_workspace_size": (_sz, [_i32, _i64]),
    "maps_local_order": (_i32, [_vp, _i32, _i32, _vp, _vp, _i64, _vp, _vp, _vp, _i32, _vp, _vp, _vp,
                                _vp, _sz, _vp]),
    "maps_place_order": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _vp, _i64, _i32, _i64, _vp, _vp, _vp, _vp,
                                _vp, _vp, _i64, _vp, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _sz, _vp]),
    "maps_place_commit_workspace_size": (_sz, [_i32, _i32]),
    "maps_place_commit": (_i32, [_vp, _i32, _i32, _vp, _vp, _vp, _vp, _i64, _i32, _i64, _vp, _vp, _vp, _vp, _vp,
                                 _vp, _vp, _sz, _vp]),
    "maps_simulate_workspace_size": (_sz, [_i32, _i64, _i32]),
    "maps_simulate": (_i32, [_i32, _i64, _i32, _i64, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                             _sz, _vp]),
    "maps_window_state_bytes": (_sz, [_i32, _i32]),
    "maps_window_append_workspace_size": (_sz, [_i64, _i32]),
    "maps_window_reset": (_i32, [_vp, _sz, _i32, _i32, _vp]),
    "maps_window_append": (_i32, [_vp, _sz, _i32, _i32, _vp, _vp, _i64, _vp, _vp, _vp, _sz, _vp]),
    "maps_window_bounds": (_i32, [_vp, _sz, _i32, _i32, _i32, _vp, _vp, _i64, _i32, _vp, _vp, _vp, _vp]),
    "maps_calibrate_noalloc": (_i32, [_vp, _vp, _i64, _vp, _i32, _i32, _vp, _vp, _vp, _i64, _i32, _vp, _vp, _vp]),
    "maps_project_order": (_i32, [_i32, _vp, _i64, _vp, _vp, _vp, _i32, _vp, _sz, _vp, _vp, _vp, _i64, _vp, _vp, _vp,
                                  _i32, _vp, _vp, _vp, _vp]),
    "maps_capacity_tokens": (_i32, [_vp, _i32, _i64, _vp, _vp, _vp]),
    "maps_status_string": (_c.c_char_p, [_i32]),
}
EXPORTS = tuple(_SIGNATURES)

_LIB = None


def library():
    """The loaded ``libmaps.so``; raises if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIBRARY):
            raise MapsError(f"{LIBRARY} is not built: run paper_2609_15359_amd.build.build() "
                            "(hipcc for gfx950); there is no fallback path")
        lib = ctypes.CDLL(LIBRARY)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = lib
    return _LIB


def status_string(status: int) -> str:
    return library().maps_status_string(int(status)).decode()


def _check(status: int, what: str):
    if status != 0:
        raise MapsError(f"{what}: {status_string(status)} ({status})")


def _dev(t: torch.Tensor, dtype: torch.dtype, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device.type != "cuda":
        raise MapsError(f"{name} must be a device tensor (got {t.device})")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise MapsError(f"{name} must be contiguous")
    return t


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _workspace(nbytes: int, device, given=None):
    if given is not None and given.numel() >= nbytes:
        return given
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def new_error_word(device=None) -> torch.Tensor:
    """A zeroed device word for the MAPS_ERR_* bits (int32 storage of a uint32)."""
    return torch.zeros(1, dtype=torch.int32, device=device or "cuda")


def error_names(bits: int) -> list[str]:
    return [name for b, name in ERR_BITS.items() if bits & b]


def check_errors(dev_err: torch.Tensor):
    """Synchronizes and raises MapsError if any value-error bit is set."""
    bits = int(dev_err.item()) & 0xFFFFFFFF
    if bits:
        raise MapsError("device value error: " + ", ".join(error_names(bits)))


def capacity_tokens(capacity_bytes: torch.Tensor, bytes_per_token: int, dev_err=None) -> torch.Tensor:
    """KV capacity in bytes -> tokens, floor(C / b) (App. A: tokens map to
    bytes by model constants); int64 device tensor in, int32 out."""
    capacity_bytes = _dev(capacity_bytes, torch.int64, "capacity_bytes")
    dev = capacity_bytes.device
    out = torch.empty(capacity_bytes.numel(), dtype=torch.int32, device=dev)
    err = new_error_word(dev) if dev_err is None else dev_err
    _check(library().maps_capacity_tokens(_ptr(capacity_bytes), capacity_bytes.numel(), int(bytes_per_token),
                                          _ptr(out), _ptr(err), _stream(dev)), "maps_capacity_tokens")
    if dev_err is None:
        check_errors(err)
    return out


# ---------------------------------------------------------------------------
# 1. calibration (Sec. 3.2)
# ---------------------------------------------------------------------------

def calibrate(pred, truth, edges, alpha_ppm: int, apply_pred=None, u_max: int = 0,
              dev_err=None, workspace=None, out=None):
    """Per-bucket conformal quantiles q[nb], bucket sizes, and bounds for apply_pred."""
    pred = _dev(pred, torch.int32, "pred")
    dev = pred.device
    truth = _dev(truth, torch.int32, "truth")
    edges = _dev(edges, torch.int32, "edges")
    nb = edges.numel() + 1
    n = pred.numel()
    if truth.numel() != n:
        raise MapsError("pred and truth differ in length")
    m = 0 if apply_pred is None else _dev(apply_pred, torch.int32, "apply_pred").numel()
    q = torch.empty(nb, dtype=torch.int32, device=dev) if out is None else out["q"]
    cnt = torch.empty(nb, dtype=torch.int32, device=dev) if out is None else out["count"]
    U = (torch.empty(m, dtype=torch.int32, device=dev) if out is None else out["U"]) if m else None
    err = new_error_word(dev) if dev_err is None else dev_err
    lib = library()
    ws_bytes = lib.maps_calibrate_workspace_size(n, nb)
    ws = _workspace(ws_bytes, dev, workspace)
    st = lib.maps_calibrate(_ptr(pred), _ptr(truth), n, _ptr(edges) if nb > 1 else None, nb,
                            int(alpha_ppm), _ptr(q), _ptr(cnt), _ptr(apply_pred) if m else None, m,
                            int(u_max), _ptr(U), _ptr(err), _ptr(ws), ws.numel(), _stream(dev))
    _check(st, "maps_calibrate")
    return q, cnt, U, err


def calibrate_window_workspace_bytes(n: int, nb: int) -> int:
    return int(library().maps_calibrate_window_workspace_size(int(n), int(nb)))


def calibrate_window(pred, truth, edges, window: int, alpha_ppm: int, apply_pred, apply_seen, u_max: int,
                     dev_err=None, workspace=None, q=None, U=None, want_q: bool = True):
    """Sliding-window calibration: each request's bound from the `window` most
    recent completions of its bucket among the first apply_seen[j] entries of
    the completion log (pred, truth).  Returns (q or None, U, dev_err)."""
    pred = _dev(pred, torch.int32, "pred")
    dev = pred.device
    truth = _dev(truth, torch.int32, "truth")
    edges = _dev(edges, torch.int32, "edges")
    apply_pred = _dev(apply_pred, torch.int32, "apply_pred")
    apply_seen = _dev(apply_seen, torch.int64, "apply_seen")
    nb, n, m = edges.numel() + 1, pred.numel(), apply_pred.numel()
    if truth.numel() != n or apply_seen.numel() != m:
        raise MapsError("pred/truth or apply_pred/apply_seen differ in length")
    if want_q and q is None:
        q = torch.empty(m, dtype=torch.int32, device=dev)
    U = torch.empty(m, dtype=torch.int32, device=dev) if U is None else U
    err = new_error_word(dev) if dev_err is None else dev_err
    lib = library()
    ws = _workspace(lib.maps_calibrate_window_workspace_size(n, nb), dev, workspace)
    st = lib.maps_calibrate_window(_ptr(pred), _ptr(truth), n, _ptr(edges) if nb > 1 else None, nb, int(window),
                                   int(alpha_ppm), _ptr(apply_pred), _ptr(apply_seen), m, int(u_max),
                                   _ptr(q) if want_q else None, _ptr(U), _ptr(err), _ptr(ws), ws.numel(),
                                   _stream(dev))
    _check(st, "maps_calibrate_window")
    return (q if want_q else None), U, err


class WindowState:
    """Incremental sliding-window calibration: per length bucket the count of
    completions appended and a ring of the last `window` scores, kept in
    device memory (Sec. 3.2; Sec. 4 uses a window of 500)."""

    def __init__(self, edges: torch.Tensor, window: int, device=None):
        self.edges = _dev(edges, torch.int32, "edges")
        self.nb = edges.numel() + 1
        self.window = int(window)
        dev = edges.device if device is None else device
        lib = library()
        nbytes = int(lib.maps_window_state_bytes(self.nb, self.window))
        if nbytes == 0:
            raise MapsError("invalid (buckets, window)")
        self.state = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        self.dev_err = new_error_word(dev)
        self.q = torch.empty(self.nb, dtype=torch.int32, device=dev)
        self._ws = None
        self.reset()

    def reset(self):
        _check(library().maps_window_reset(_ptr(self.state), self.state.numel(), self.nb, self.window,
                                           _stream(self.state.device)), "maps_window_reset")

    def append(self, pred, truth, workspace=None):
        pred = _dev(pred, torch.int32, "pred")
        truth = _dev(truth, torch.int32, "truth")
        k = pred.numel()
        if truth.numel() != k:
            raise MapsError("pred and truth differ in length")
        lib = library()
        need = int(lib.maps_window_append_workspace_size(k, self.nb))
        if workspace is None:
            if self._ws is None or self._ws.numel() < need:
                self._ws = torch.empty(max(need, 1), dtype=torch.uint8, device=self.state.device)
            workspace = self._ws
        st = lib.maps_window_append(_ptr(self.state), self.state.numel(), self.nb, self.window, _ptr(pred),
                                    _ptr(truth), k, _ptr(self.edges) if self.nb > 1 else None, _ptr(self.dev_err),
                                    _ptr(workspace), workspace.numel(), _stream(self.state.device))
        _check(st, "maps_window_append")

    def bounds(self, alpha_ppm: int, apply_pred=None, u_max: int = 0, U=None):
        """Per-bucket quantiles of the current windows and the bounds of apply_pred."""
        m = 0 if apply_pred is None else _dev(apply_pred, torch.int32, "apply_pred").numel()
        if m and U is None:
            U = torch.empty(m, dtype=torch.int32, device=self.state.device)
        st = library().maps_window_bounds(_ptr(self.state), self.state.numel(), self.nb, self.window, int(alpha_ppm),
                                          _ptr(self.edges) if self.nb > 1 else None, _ptr(apply_pred) if m else None,
                                          m, int(u_max), _ptr(self.q), _ptr(U) if m else None, _ptr(self.dev_err),
                                          _stream(self.state.device))
        _check(st, "maps_window_bounds")
        return self.q, U


# ---------------------------------------------------------------------------
# 2. projection (Sec. 3.3, App. A)
# ---------------------------------------------------------------------------

def snapshot_bytes(D: int, n_total: int, u_max: int) -> int:
    return int(library().maps_snapshot_bytes(int(D), int(n_total), int(u_max)))


def project(seg_off, prompt, generated, upper, u_max: int, snapshot=None, dev_err=None,
            base_peak=None):
    """Occupancy snapshot of D decoders and their base peaks."""
    seg_off = _dev(seg_off, torch.int64, "seg_off")
    dev = seg_off.device
    D = seg_off.numel() - 1
    n = prompt.numel()
    for name, t in (("prompt", prompt), ("generated", generated), ("upper", upper)):
        _dev(t, torch.int32, name)
        if t.numel() != n:
            raise MapsError("prompt, generated and upper differ in length")
    nbytes = snapshot_bytes(D, n, u_max)
    if nbytes == 0:
        raise MapsError("invalid snapshot size arguments")
    snap = snapshot if snapshot is not None else torch.empty(nbytes, dtype=torch.uint8, device=dev)
    bp = torch.empty(D, dtype=torch.int32, device=dev) if base_peak is None else base_peak
    err = new_error_word(dev) if dev_err is None else dev_err
    st = library().maps_project(D, _ptr(seg_off), n, _ptr(prompt), _ptr(generated), _ptr(upper),
                                int(u_max), _ptr(snap), snap.numel(), _ptr(bp), _ptr(err), None, 0,
                                _stream(dev))
    _check(st, "maps_project")
    return Snapshot(data=snap, D=D, n_total=n, u_max=int(u_max)), bp, err


@dataclass
class Snapshot:
    data: torch.Tensor
    D: int
    n_total: int
    u_max: int


# ---------------------------------------------------------------------------
# 3. placement (Sec. 3.3, Algorithm 1)
# ---------------------------------------------------------------------------

@dataclass
class Placement:
    choice: torch.Tensor
    chosen_peak: torch.Tensor
    chosen_overflow: torch.Tensor
    flags: torch.Tensor
    pair_peak: torch.Tensor | None
    dev_err: torch.Tensor


def place_workspace_bytes(D: int, A: int, u_max: int) -> int:
    return int(library().maps_place_workspace_size(int(D), int(A), int(u_max)))


def place(snapshot: Snapshot, capacity, queue_len, a_prompt, a_upper, policy: int = POLICY_MQ,
          rr_offset: int = 0, want_pairs: bool = True, dev_err=None, workspace=None,
          out: Placement | None = None) -> Placement:
    """Choice of decoder for every arrival, and optionally every pair's peak."""
    capacity = _dev(capacity, torch.int32, "capacity")
    dev = capacity.device
    queue_len = _dev(queue_len, torch.int32, "queue_len")
    a_prompt = _dev(a_prompt, torch.int32, "a_prompt")
    a_upper = _dev(a_upper, torch.int32, "a_upper")
    D, A = snapshot.D, a_prompt.numel()
    if capacity.numel() != D or queue_len.numel() != D or a_upper.numel() != A:
        raise MapsError("capacity/queue_len must have D entries and a_upper A entries")
    if out is None:
        out = Placement(
            choice=torch.empty(A, dtype=torch.int32, device=dev),
            chosen_peak=torch.empty(A, dtype=torch.int32, device=dev),
            chosen_overflow=torch.empty(A, dtype=torch.int32, device=dev),
            flags=torch.empty(A, dtype=torch.uint8, device=dev),
            pair_peak=torch.empty((D, A), dtype=torch.int32, device=dev) if want_pairs else None,
            dev_err=new_error_word(dev) if dev_err is None else dev_err)
    lib = library()
    ws = _workspace(lib.maps_place_workspace_size(D, A, snapshot.u_max), dev, workspace)
    st = lib.maps_place(_ptr(snapshot.data), D, snapshot.u_max, _ptr(capacity), _ptr(queue_len),
                        _ptr(a_prompt), _ptr(a_upper), A, int(policy), int(rr_offset),
                        _ptr(out.choice), _ptr(out.chosen_peak), _ptr(out.chosen_overflow),
                        _ptr(out.flags), _ptr(out.pair_peak), _ptr(out.dev_err), _ptr(ws),
                        ws.numel(), _stream(dev))
    _check(st, "maps_place")
    return out


def place_commit_workspace_bytes(D: int, u_max: int) -> int:
    return int(library().maps_place_commit_workspace_size(int(D), int(u_max)))


@dataclass
class CommitPlacement:
    choice: torch.Tensor
    chosen_peak: torch.Tensor       # int64
    chosen_overflow: torch.Tensor   # int64
    flags: torch.Tensor
    queue_out: torch.Tensor
    dev_err: torch.Tensor


def place_commit(snapshot: Snapshot, capacity, queue_len, a_prompt, a_upper, policy: int = POLICY_MQ,
                 rr_offset: int = 0, dev_err=None, workspace=None,
                 out: CommitPlacement | None = None) -> CommitPlacement:
    """Arrivals placed one after another, each committed to its decoder's
    projected occupancy and queue before the next (Sec. 3.3, Algorithm 1)."""
    capacity = _dev(capacity, torch.int32, "capacity")
    dev = capacity.device
    queue_len = _dev(queue_len, torch.int32, "queue_len")
    a_prompt = _dev(a_prompt, torch.int32, "a_prompt")
    a_upper = _dev(a_upper, torch.int32, "a_upper")
    D, A = snapshot.D, a_prompt.numel()
    if capacity.numel() != D or queue_len.numel() != D or a_upper.numel() != A:
        raise MapsError("capacity/queue_len must have D entries and a_upper A entries")
    if out is None:
        out = CommitPlacement(choice=torch.empty(A, dtype=torch.int32, device=dev),
                              chosen_peak=torch.empty(A, dtype=torch.int64, device=dev),
                              chosen_overflow=torch.empty(A, dtype=torch.int64, device=dev),
                              flags=torch.empty(A, dtype=torch.uint8, device=dev),
                              queue_out=torch.empty(D, dtype=torch.int32, device=dev),
                              dev_err=new_error_word(dev) if dev_err is None else dev_err)
    lib = library()
    ws = _workspace(lib.maps_place_commit_workspace_size(D, snapshot.u_max), dev, workspace)
    st = lib.maps_place_commit(_ptr(snapshot.data), D, snapshot.u_max, _ptr(capacity), _ptr(queue_len),
                               _ptr(a_prompt), _ptr(a_upper), A, int(policy), int(rr_offset), _ptr(out.choice),
                               _ptr(out.chosen_peak), _ptr(out.chosen_overflow), _ptr(out.flags),
                               _ptr(out.queue_out), _ptr(out.dev_err), _ptr(ws), ws.numel(), _stream(dev))
    _check(st, "maps_place_commit")
    return out


def project_order(seg_off, prompt, generated, upper, u_max: int, capacity, q_off, q_prompt, q_upper, q_wait_ms=None,
                  max_wait_ms: int = 2**31 - 1, snapshot=None, dev_err=None, base_peak=None, order=None,
                  admitted=None):
    """maps_project then maps_local_order in one launch: (snapshot, base_peak,
    order, admitted, dev_err)."""
    seg_off = _dev(seg_off, torch.int64, "seg_off")
    dev = seg_off.device
    D = seg_off.numel() - 1
    n = prompt.numel()
    for name, t in (("prompt", prompt), ("generated", generated), ("upper", upper)):
        _dev(t, torch.int32, name)
        if t.numel() != n:
            raise MapsError("prompt, generated and upper differ in length")
    capacity = _dev(capacity, torch.int32, "capacity")
    q_off = _dev(q_off, torch.int64, "q_off")
    q_prompt = _dev(q_prompt, torch.int32, "q_prompt")
    q_upper = _dev(q_upper, torch.int32, "q_upper")
    if q_wait_ms is not None:
        _dev(q_wait_ms, torch.int32, "q_wait_ms")
    total = q_prompt.numel()
    if capacity.numel() != D or q_off.numel() != D + 1 or q_upper.numel() != total:
        raise MapsError("capacity must have D entries, q_off D+1 and q_upper as many as q_prompt")
    nbytes = snapshot_bytes(D, n, u_max)
    snap = snapshot if snapshot is not None else torch.empty(nbytes, dtype=torch.uint8, device=dev)
    bp = torch.empty(D, dtype=torch.int32, device=dev) if base_peak is None else base_peak
    order = torch.empty(total, dtype=torch.int32, device=dev) if order is None else order
    admitted = torch.empty(D, dtype=torch.int32, device=dev) if admitted is None else admitted
    err = new_error_word(dev) if dev_err is None else dev_err
    st = library().maps_project_order(D, _ptr(seg_off), n, _ptr(prompt), _ptr(generated), _ptr(upper), int(u_max),
                                      _ptr(snap), snap.numel(), _ptr(bp), _ptr(capacity), _ptr(q_off), total,
                                      _ptr(q_prompt), _ptr(q_upper), _ptr(q_wait_ms), int(max_wait_ms), _ptr(order),
                                      _ptr(admitted), _ptr(err), _stream(dev))
    _check(st, "maps_project_order")
    return Snapshot(data=snap, D=D, n_total=n, u_max=int(u_max)), bp, order, admitted, err


# ---------------------------------------------------------------------------
# 4. local order (Sec. 3.3, Eq. (7); App. A, Eq. (10))
# ---------------------------------------------------------------------------

def local_order(snapshot: Snapshot, capacity, q_off, q_prompt, q_upper, q_wait_ms=None,
                max_wait_ms: int = 2**31 - 1, dev_err=None, order=None, admitted=None):
    """New order of every decoder's queue and the admitted prefix length."""
    capacity = _dev(capacity, torch.int32, "capacity")
    dev = capacity.device
    q_off = _dev(q_off, torch.int64, "q_off")
    q_prompt = _dev(q_prompt, torch.int32, "q_prompt")
    q_upper = _dev(q_upper, torch.int32, "q_upper")
    if q_wait_ms is not None:
        _dev(q_wait_ms, torch.int32, "q_wait_ms")
    D, total = snapshot.D, q_prompt.numel()
    if q_off.numel() != D + 1 or q_upper.numel() != total:
        raise MapsError("q_off must have D+1 entries and q_upper as many as q_prompt")
    order = torch.empty(total, dtype=torch.int32, device=dev) if order is None else order
    admitted = torch.empty(D, dtype=torch.int32, device=dev) if admitted is None else admitted
    err = new_error_word(dev) if dev_err is None else dev_err
    st = library().maps_local_order(_ptr(snapshot.data), D, snapshot.u_max, _ptr(capacity),
                                    _ptr(q_off), total, _ptr(q_prompt), _ptr(q_upper),
                                    _ptr(q_wait_ms), int(max_wait_ms), _ptr(order), _ptr(admitted),
                                    _ptr(err), None, 0, _stream(dev))
    _check(st, "maps_local_order")
    return order, admitted, err


# ---------------------------------------------------------------------------
# 3c. projected placement in blocks
# ---------------------------------------------------------------------------

@dataclass
class BlockSnapshot:
    data: torch.Tensor      # uint8 device buffer
    seg_off: torch.Tensor   # the residents' segment offsets it was built from
    D: int
    n_total: int
    u_max: int
    block_size: int


def project_blocks(seg_off, prompt, generated, upper, u_max: int, block_size: int, dev_err=None, base_peak=None,
                   snapshot: "BlockSnapshot | None" = None):
    """Block snapshot of D decoders and their base peaks in blocks (into the
    buffer of `snapshot` when one is given)."""
    seg_off = _dev(seg_off, torch.int64, "seg_off")
    dev = seg_off.device
    D = seg_off.numel() - 1
    n = prompt.numel()
    for name, t in (("prompt", prompt), ("generated", generated), ("upper", upper)):
        _dev(t, torch.int32, name)
        if t.numel() != n:
            raise MapsError("prompt, generated and upper differ in length")
    lib = library()
    nbytes = lib.maps_blocks_snapshot_bytes(D, n, int(u_max), int(block_size))
    if nbytes == 0:
        raise MapsError("D, u_max or block_size out of range for the block snapshot")
    if snapshot is not None and snapshot.data.numel() >= nbytes:
        snap = snapshot.data
    else:
        snap = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    base = torch.empty(D, dtype=torch.int32, device=dev) if base_peak is None else base_peak
    err = new_error_word(dev) if dev_err is None else dev_err
    st = lib.maps_project_blocks(D, _ptr(seg_off), _ptr(prompt), _ptr(generated), _ptr(upper), n, int(u_max),
                                 int(block_size), _ptr(snap), nbytes, _ptr(base), _ptr(err), _stream(dev))
    _check(st, "maps_project_blocks")
    return BlockSnapshot(snap, seg_off, D, n, int(u_max), int(block_size)), base, err


def place_blocks(snapshot: BlockSnapshot, capacity, queue_len, a_prompt, a_upper, policy: int = POLICY_MQ,
                 rr_offset: int = 0, dev_err=None, out: Placement | None = None) -> Placement:
    """Placement with peaks, capacities floor(C/S) and overflow in blocks; the
    pair matrix [D][A] is always written."""
    capacity = _dev(capacity, torch.int32, "capacity")
    dev = capacity.device
    queue_len = _dev(queue_len, torch.int32, "queue_len")
    a_prompt = _dev(a_prompt, torch.int32, "a_prompt")
    a_upper = _dev(a_upper, torch.int32, "a_upper")
    D, A = snapshot.D, a_prompt.numel()
    if capacity.numel() != D or queue_len.numel() != D or a_upper.numel() != A:
        raise MapsError("capacity/queue_len must have D entries and a_upper A entries")
    if out is None:
        out = Placement(
            choice=torch.empty(A, dtype=torch.int32, device=dev),
            chosen_peak=torch.empty(A, dtype=torch.int32, device=dev),
            chosen_overflow=torch.empty(A, dtype=torch.int32, device=dev),
            flags=torch.empty(A, dtype=torch.uint8, device=dev),
            pair_peak=torch.empty((D, A), dtype=torch.int32, device=dev),
            dev_err=new_error_word(dev) if dev_err is None else dev_err)
    st = library().maps_place_blocks(_ptr(snapshot.data), _ptr(snapshot.seg_off), D, snapshot.n_total,
                                     snapshot.u_max, snapshot.block_size, _ptr(capacity), _ptr(queue_len),
                                     _ptr(a_prompt), _ptr(a_upper), A, int(policy), int(rr_offset), _ptr(out.choice),
                                     _ptr(out.chosen_peak), _ptr(out.chosen_overflow), _ptr(out.flags),
                                     _ptr(out.pair_peak), _ptr(out.dev_err), _stream(dev))
    _check(st, "maps_place_blocks")
    return out


# ---------------------------------------------------------------------------
# 3b. Algorithm 1 on block counts
# ---------------------------------------------------------------------------

def rsc_state(seg_off, prompt, generated, upper, capacity, block_size: int, dev_err=None, out=None, in_flight=None):
    """Runtime state per decoder in blocks: (b_free, b_res, b_eff, dev_err), int64 [D].
    in_flight (optional uint8 per request): prompt KV still in transfer."""
    seg_off = _dev(seg_off, torch.int64, "seg_off")
    dev = seg_off.device
    D = seg_off.numel() - 1
    n = prompt.numel()
    for name, t in (("prompt", prompt), ("generated", generated), ("upper", upper)):
        _dev(t, torch.int32, name)
        if t.numel() != n:
            raise MapsError("prompt, generated and upper differ in length")
    capacity = _dev(capacity, torch.int32, "capacity")
    if capacity.numel() != D:
        raise MapsError("capacity must have D entries")
    if in_flight is not None:
        _dev(in_flight, torch.uint8, "in_flight")
        if in_flight.numel() != n:
            raise MapsError("in_flight must have one entry per request")
    bf, br, be = out if out is not None else [torch.empty(D, dtype=torch.int64, device=dev) for _ in range(3)]
    err = new_error_word(dev) if dev_err is None else dev_err
    st = library().maps_rsc_state(D, _ptr(seg_off), n, _ptr(prompt), _ptr(generated), _ptr(upper), _ptr(in_flight),
                                  _ptr(capacity),
                                  int(block_size), _ptr(bf), _ptr(br), _ptr(be), _ptr(err), _stream(dev))
    _check(st, "maps_rsc_state")
    return bf, br, be, err


def place_static(b_eff, queue_len, block_size: int, a_prompt, a_upper, policy: int = POLICY_MQ, rr_offset: int = 0,
                 reserve: bool = False, dev_err=None, out=None, want_state: bool = True):
    """Algorithm 1 per arrival against (b_eff, queue_len); with `reserve` each
    dispatch reserves its B_need and joins its queue before the next.  Returns
    (choice, b_need, flags, b_eff_after, queue_after, dev_err)."""
    b_eff = _dev(b_eff, torch.int64, "b_eff")
    dev = b_eff.device
    queue_len = _dev(queue_len, torch.int32, "queue_len")
    a_prompt = _dev(a_prompt, torch.int32, "a_prompt")
    a_upper = _dev(a_upper, torch.int32, "a_upper")
    D, A = b_eff.numel(), a_prompt.numel()
    if queue_len.numel() != D or a_upper.numel() != A:
        raise MapsError("queue_len must have D entries and a_upper A entries")
    if out is None:
        out = (torch.empty(A, dtype=torch.int32, device=dev), torch.empty(A, dtype=torch.int64, device=dev),
               torch.empty(A, dtype=torch.uint8, device=dev),
               torch.empty(D, dtype=torch.int64, device=dev) if want_state else None,
               torch.empty(D, dtype=torch.int32, device=dev) if want_state else None)
    choice, need, flags, b_after, q_after = out
    err = new_error_word(dev) if dev_err is None else dev_err
    st = library().maps_place_static(D, _ptr(b_eff), _ptr(queue_len), int(block_size), _ptr(a_prompt), _ptr(a_upper),
                                     A, int(policy), int(rr_offset), int(bool(reserve)), _ptr(choice), _ptr(need),
                                     _ptr(flags), _ptr(b_after), _ptr(q_after), _ptr(err), _stream(dev))
    _check(st, "maps_place_static")
    return choice, need, flags, b_after, q_after, err


# ---------------------------------------------------------------------------
# 3 + 4. placement and local order in two launches
# ---------------------------------------------------------------------------

def place_order(snapshot: Snapshot, capacity, queue_len, a_prompt, a_upper, q_off, q_prompt, q_upper,
                q_wait_ms=None, max_wait_ms: int = 2**31 - 1, policy: int = POLICY_MQ, rr_offset: int = 0,
                want_pairs: bool = True, dev_err=None, workspace=None, out: Placement | None = None,
                order=None, admitted=None):
    """place() then local_order() on the same snapshot, with the final
    selection and the local orders in one launch; returns (Placement, order,
    admitted)."""
    capacity = _dev(capacity, torch.int32, "capacity")
    dev = capacity.device
    queue_len = _dev(queue_len, torch.int32, "queue_len")
    a_prompt = _dev(a_prompt, torch.int32, "a_prompt")
    a_upper = _dev(a_upper, torch.int32, "a_upper")
    q_off = _dev(q_off, torch.int64, "q_off")
    q_prompt = _dev(q_prompt, torch.int32, "q_prompt")
    q_upper = _dev(q_upper, torch.int32, "q_upper")
    if q_wait_ms is not None:
        _dev(q_wait_ms, torch.int32, "q_wait_ms")
    D, A, total = snapshot.D, a_prompt.numel(), q_prompt.numel()
    if capacity.numel() != D or queue_len.numel() != D or a_upper.numel() != A:
        raise MapsError("capacity/queue_len must have D entries and a_upper A entries")
    if q_off.numel() != D + 1 or q_upper.numel() != total:
        raise MapsError("q_off must have D+1 entries and q_upper as many as q_prompt")
    if out is None:
        out = Placement(
            choice=torch.empty(A, dtype=torch.int32, device=dev),
            chosen_peak=torch.empty(A, dtype=torch.int32, device=dev),
            chosen_overflow=torch.empty(A, dtype=torch.int32, device=dev),
            flags=torch.empty(A, dtype=torch.uint8, device=dev),
            pair_peak=torch.empty((D, A), dtype=torch.int32, device=dev) if want_pairs else None,
            dev_err=new_error_word(dev) if dev_err is None else dev_err)
    order = torch.empty(total, dtype=torch.int32, device=dev) if order is None else order
    admitted = torch.empty(D, dtype=torch.int32, device=dev) if admitted is None else admitted
    lib = library()
    ws = _workspace(lib.maps_place_workspace_size(D, A, snapshot.u_max), dev, workspace)
    st = lib.maps_place_order(_ptr(snapshot.data), D, snapshot.u_max, _ptr(capacity), _ptr(queue_len),
                              _ptr(a_prompt), _ptr(a_upper), A, int(policy), int(rr_offset),
                              _ptr(out.choice), _ptr(out.chosen_peak), _ptr(out.chosen_overflow),
                              _ptr(out.flags), _ptr(out.pair_peak), _ptr(q_off), total, _ptr(q_prompt),
                              _ptr(q_upper), _ptr(q_wait_ms), int(max_wait_ms), _ptr(order), _ptr(admitted),
                              _ptr(out.dev_err), _ptr(ws), ws.numel(), _stream(dev))
    _check(st, "maps_place_order")
    return out, order, admitted


# ---------------------------------------------------------------------------
# 5. KV pressure under round-robin or MAPS routing (App. A)
# ---------------------------------------------------------------------------

@dataclass
class Simulation:
    finish_ms: torch.Tensor   # int64 [S][n]
    routed: torch.Tensor      # int32 [S][n]
    stats: torch.Tensor       # int64 [S][5][N]: hp_time, hp_max, hp_count, max_queue, queue_area
    span: torch.Tensor        # int64 [S][2]: first arrival, last completion
    dev_err: torch.Tensor


def simulate(N: int, C: int, theta_ppm: int, arrival_ms, prompt, output, bound, policy, dev_err=None,
             workspace=None, out: Simulation | None = None) -> Simulation:
    """S simulations (rows of arrival_ms, one policy each: 0 round robin, 1
    Algorithm 1) of the same requests on N decoders of C tokens."""
    arrival_ms = _dev(arrival_ms, torch.int64, "arrival_ms")
    dev = arrival_ms.device
    if arrival_ms.dim() != 2:
        raise MapsError("arrival_ms must be [S][n]")
    S, n = arrival_ms.shape
    for name, t in (("prompt", prompt), ("output", output), ("bound", bound)):
        _dev(t, torch.int32, name)
        if t.numel() != n:
            raise MapsError(f"{name} must have n entries")
    policy = _dev(policy, torch.int32, "policy")
    if policy.numel() != S:
        raise MapsError("policy must have S entries")
    if out is None:
        out = Simulation(finish_ms=torch.empty((S, n), dtype=torch.int64, device=dev),
                         routed=torch.empty((S, n), dtype=torch.int32, device=dev),
                         stats=torch.empty((S, 5, N), dtype=torch.int64, device=dev),
                         span=torch.empty((S, 2), dtype=torch.int64, device=dev),
                         dev_err=new_error_word(dev) if dev_err is None else dev_err)
    lib = library()
    ws = _workspace(lib.maps_simulate_workspace_size(int(N), int(n), int(S)), dev, workspace)
    st = lib.maps_simulate(int(N), int(C), int(theta_ppm), int(n), int(S), _ptr(arrival_ms), _ptr(prompt),
                           _ptr(output), _ptr(bound), _ptr(policy), _ptr(out.finish_ms), _ptr(out.routed),
                           _ptr(out.stats), _ptr(out.span), _ptr(out.dev_err), _ptr(ws), ws.numel(), _stream(dev))
    _check(st, "maps_simulate")
    return out
