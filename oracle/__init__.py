"""CPU oracle of the MAPS scheduler core -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  It wraps ``maps_oracle.c`` (plain C, built with
gcc) through ctypes and never touches the GPU library.

Functions follow the paper's steps (Sec. 3.2 calibration, Sec. 3.3 and App. A
occupancy and admission, Algorithm 1 placement); see the C source for the
definitions each one writes out.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "maps_oracle.c")
LIBRARY = os.path.join(HERE, "liboracle.so")
Q_INF = np.iinfo(np.int32).max
POLICY_MQ, POLICY_MC = 0, 1

_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")
_i64p = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_u8p = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")


def build(source: str = SOURCE, output: str = LIBRARY, strict: bool = True) -> str:
    """Compile the oracle with gcc into a shared library and return its path."""
    cmd = ["gcc", "-O2", "-std=c11", "-shared", "-fPIC", "-Wall",
           *(["-Werror"] if strict else []), source, "-o", output]
    subprocess.run(cmd, check=True)
    return output


def _nullable(ptr_type):
    """ndpointer that also accepts None (passed as NULL)."""
    class _Nullable(ptr_type):
        @classmethod
        def from_param(cls, obj):
            if obj is None:
                return None
            return super().from_param(obj)
    return _Nullable


def _declare(lib):
    i64n, i32n, u8n = _nullable(_i64p), _nullable(_i32p), _nullable(_u8p)
    c = ctypes
    lib.oracle_bucket.argtypes = [c.c_int32, _i32p, c.c_int32]
    lib.oracle_bucket.restype = c.c_int32
    lib.oracle_conformal_rank.argtypes = [c.c_int64, c.c_int32]
    lib.oracle_conformal_rank.restype = c.c_int64
    lib.oracle_calibrate.argtypes = [_i32p, _i32p, c.c_int64, _i32p, c.c_int32, c.c_int32,
                                     _i32p, _i32p]
    lib.oracle_calibrate.restype = c.c_int
    lib.oracle_apply_bounds.argtypes = [_i32p, c.c_int64, _i32p, c.c_int32, _i32p, c.c_int32,
                                        _i32p]
    lib.oracle_apply_bounds.restype = None
    lib.oracle_calibrate_window.argtypes = [_i32p, _i32p, c.c_int64, _i32p, c.c_int32, c.c_int32,
                                            c.c_int32, _i32p, _i64p, c.c_int64, c.c_int32, _i32p,
                                            _i32p]
    lib.oracle_calibrate_window.restype = c.c_int
    lib.oracle_occupancy.argtypes = [_i32p, _i32p, _i32p, c.c_int64, c.c_int64, _i64p]
    lib.oracle_occupancy.restype = c.c_int
    lib.oracle_project.argtypes = [c.c_int32, _i64p, _i32p, _i32p, _i32p, _i64p]
    lib.oracle_project.restype = c.c_int
    lib.oracle_place.argtypes = [c.c_int32, _i64p, _i32p, _i32p, _i32p, _i32p, _i32p,
                                 c.c_int64, _i32p, _i32p, i64n, c.c_int32, c.c_int64,
                                 _i32p, _i64p, _i64p, _u8p, i64n, i64n]
    lib.oracle_place.restype = c.c_int
    lib.oracle_occupancy_blocks.argtypes = [_i32p, _i32p, _i32p, c.c_int64, c.c_int32, c.c_int64, _i64p]
    lib.oracle_occupancy_blocks.restype = c.c_int
    lib.oracle_place_blocks.argtypes = [c.c_int32, _i64p, _i32p, _i32p, _i32p, _i32p, _i32p, c.c_int32,
                                        c.c_int64, _i32p, _i32p, c.c_int32, c.c_int64,
                                        _i32p, _i64p, _i64p, _u8p, i64n, i64n]
    lib.oracle_place_blocks.restype = c.c_int
    lib.oracle_rsc_state.argtypes = [c.c_int32, _i64p, _i32p, _i32p, _i32p, u8n, _i32p, c.c_int32, _i64p, _i64p,
                                     _i64p]
    lib.oracle_rsc_state.restype = c.c_int
    lib.oracle_place_static.argtypes = [c.c_int32, _i64p, _i32p, c.c_int32, c.c_int64, _i32p, _i32p, c.c_int32,
                                        c.c_int64, c.c_int32, _i32p, _i64p, _u8p, i64n, i32n]
    lib.oracle_place_static.restype = c.c_int
    lib.oracle_place_commit.argtypes = [c.c_int32, _i64p, _i32p, _i32p, _i32p, _i32p, _i32p, c.c_int64,
                                        _i32p, _i32p, c.c_int32, c.c_int64, _i32p, _i64p, _i64p, _u8p, i32n]
    lib.oracle_place_commit.restype = c.c_int
    lib.oracle_simulate.argtypes = [c.c_int32, c.c_int64, c.c_int32, c.c_int64, _i64p, _i32p, _i32p, _i32p,
                                    c.c_int32, _i64p, _i32p, _i64p, _i64p, _i64p, _i64p, _i64p, _i64p]
    lib.oracle_simulate.restype = c.c_int
    lib.oracle_local_order.argtypes = [c.c_int32, _i64p, _i32p, _i32p, _i32p, _i32p, _i64p,
                                       _i32p, _i32p, i32n, c.c_int32, c.c_int32, _i32p, _i32p]
    lib.oracle_local_order.restype = c.c_int
    lib.oracle_bruteforce_peak.argtypes = [c.c_int64, _i32p, _i32p, _i32p, c.c_int64, _i32p,
                                           _i32p]
    lib.oracle_bruteforce_peak.restype = c.c_int64
    return lib


_LIB = None


def load(path: str | None = None):
    """Load the oracle library (building it first if it is not built)."""
    global _LIB
    if path is not None:
        return _declare(ctypes.CDLL(path))
    if _LIB is None:
        if not os.path.exists(LIBRARY):
            build()
        _LIB = _declare(ctypes.CDLL(LIBRARY))
    return _LIB


def _i32(x):
    return np.ascontiguousarray(x, dtype=np.int32)


def _i64(x):
    return np.ascontiguousarray(x, dtype=np.int64)


class Oracle:
    """numpy front end of one oracle library (the default build, or a variant)."""

    def __init__(self, lib=None):
        self.lib = lib if lib is not None else load()

    # -- calibration (Sec. 3.2) --------------------------------------------
    def bucket(self, pred: int, edges) -> int:
        e = _i32(edges) if len(edges) else np.zeros(1, np.int32)
        return int(self.lib.oracle_bucket(int(pred), e, len(edges) + 1))

    def conformal_rank(self, n: int, alpha_ppm: int) -> int:
        return int(self.lib.oracle_conformal_rank(int(n), int(alpha_ppm)))

    def calibrate(self, pred, truth, edges, alpha_ppm: int):
        pred, truth = _i32(pred), _i32(truth)
        nb = len(edges) + 1
        e = _i32(edges) if len(edges) else np.zeros(1, np.int32)
        q = np.zeros(nb, np.int32)
        cnt = np.zeros(nb, np.int32)
        rc = self.lib.oracle_calibrate(pred, truth, pred.size, e, nb, int(alpha_ppm), q, cnt)
        if rc:
            raise ValueError(f"oracle_calibrate failed ({rc})")
        return q, cnt

    def calibrate_window(self, pred, truth, edges, window: int, alpha_ppm: int, apply_pred, seen,
                         u_max: int):
        """Sliding-window calibration (Sec. 3.2, Sec. 4): each request's own set
        is the `window` most recent completions of its bucket among the first
        seen[j] log entries.  Returns (q, U) per request."""
        pred, truth = _i32(pred), _i32(truth)
        apply_pred, seen = _i32(apply_pred), _i64(seen)
        e = _i32(edges) if len(edges) else np.zeros(1, np.int32)
        q = np.zeros(apply_pred.size, np.int32)
        U = np.zeros(apply_pred.size, np.int32)
        rc = self.lib.oracle_calibrate_window(pred, truth, pred.size, e, len(edges) + 1, int(window),
                                              int(alpha_ppm), apply_pred, seen, apply_pred.size,
                                              int(u_max), q, U)
        if rc:
            raise ValueError(f"oracle_calibrate_window failed ({rc})")
        return q, U

    def apply_bounds(self, pred, edges, q, u_max: int):
        pred = _i32(pred)
        e = _i32(edges) if len(edges) else np.zeros(1, np.int32)
        U = np.zeros(pred.size, np.int32)
        self.lib.oracle_apply_bounds(pred, pred.size, e, len(edges) + 1, _i32(q), int(u_max), U)
        return U

    # -- occupancy (Sec. 3.3, App. A) --------------------------------------
    def occupancy(self, p, g, U, T: int):
        O = np.zeros(int(T) + 1, np.int64)
        rc = self.lib.oracle_occupancy(_i32(p), _i32(g), _i32(U), len(p), int(T), O)
        if rc:
            raise ValueError(f"oracle_occupancy failed ({rc})")
        return O

    def project(self, seg_off, p, g, U):
        seg_off = _i64(seg_off)
        D = seg_off.size - 1
        base = np.zeros(D, np.int64)
        rc = self.lib.oracle_project(D, seg_off, _i32(p), _i32(g), _i32(U), base)
        if rc:
            raise ValueError(f"oracle_project failed ({rc})")
        return base

    # -- placement (Algorithm 1) -------------------------------------------
    def place(self, seg_off, p, g, U, capacity, queue_len, a_p, a_U, policy=POLICY_MQ,
              rr_offset=0, a_index=None, want_pairs=True):
        seg_off = _i64(seg_off)
        D = seg_off.size - 1
        a_p, a_U = _i32(a_p), _i32(a_U)
        A = a_p.size
        out = PlaceResult(
            choice=np.zeros(A, np.int32), chosen_peak=np.zeros(A, np.int64),
            chosen_overflow=np.zeros(A, np.int64), flags=np.zeros(A, np.uint8),
            pair_peak=np.zeros((D, A), np.int64) if want_pairs else None,
            base_peak=np.zeros(D, np.int64))
        rc = self.lib.oracle_place(
            D, seg_off, _i32(p), _i32(g), _i32(U), _i32(capacity), _i32(queue_len),
            A, a_p, a_U, None if a_index is None else _i64(a_index), int(policy), int(rr_offset),
            out.choice, out.chosen_peak, out.chosen_overflow, out.flags,
            None if out.pair_peak is None else out.pair_peak.reshape(-1), out.base_peak)
        if rc:
            raise ValueError(f"oracle_place failed ({rc})")
        return out

    # -- projected peak in blocks (Sec. 3.3, Eq. (6)) -------------------------
    def occupancy_blocks(self, p, g, U, S: int, T: int):
        OB = np.zeros(T + 1, np.int64)
        p = _i32(p)
        rc = self.lib.oracle_occupancy_blocks(p, _i32(g), _i32(U), p.size, int(S), int(T), OB)
        if rc:
            raise ValueError(f"oracle_occupancy_blocks failed ({rc})")
        return OB

    def place_blocks(self, seg_off, p, g, U, capacity, queue_len, S: int, a_p, a_U, policy=POLICY_MQ,
                     rr_offset=0, want_pairs=True):
        """Placement with every count in blocks of S tokens (peaks, capacities
        floor(C/S), overflow); the same result fields as place()."""
        seg_off = _i64(seg_off)
        D = seg_off.size - 1
        a_p, a_U = _i32(a_p), _i32(a_U)
        A = a_p.size
        out = PlaceResult(
            choice=np.zeros(A, np.int32), chosen_peak=np.zeros(A, np.int64),
            chosen_overflow=np.zeros(A, np.int64), flags=np.zeros(A, np.uint8),
            pair_peak=np.zeros((D, A), np.int64) if want_pairs else None,
            base_peak=np.zeros(D, np.int64))
        rc = self.lib.oracle_place_blocks(
            D, seg_off, _i32(p), _i32(g), _i32(U), _i32(capacity), _i32(queue_len), int(S), A, a_p, a_U,
            int(policy), int(rr_offset), out.choice, out.chosen_peak, out.chosen_overflow, out.flags,
            None if out.pair_peak is None else out.pair_peak.reshape(-1), out.base_peak)
        if rc:
            raise ValueError(f"oracle_place_blocks failed ({rc})")
        return out

    # -- Algorithm 1 on block counts (Sec. 3.3, Eq. (6)) ---------------------
    def rsc_state(self, seg_off, p, g, U, capacity, S: int, in_flight=None):
        """(B_free, B_res, B_eff) per decoder in blocks of S tokens; in_flight
        (optional, one flag per request) marks requests whose prompt KV is
        still being transferred (whole budget reserved, nothing held)."""
        seg_off = _i64(seg_off)
        D = seg_off.size - 1
        out = [np.zeros(D, np.int64) for _ in range(3)]
        fl = None if in_flight is None else np.ascontiguousarray(in_flight, dtype=np.uint8)
        rc = self.lib.oracle_rsc_state(D, seg_off, _i32(p), _i32(g), _i32(U), fl, _i32(capacity), int(S), *out)
        if rc:
            raise ValueError(f"oracle_rsc_state failed ({rc})")
        return tuple(out)

    def place_static(self, b_eff, queue_len, S: int, a_p, a_U, policy=POLICY_MQ, rr_offset=0, reserve=False):
        """Algorithm 1 per arrival; with `reserve`, each dispatch reserves its
        B_need and joins the queue before the next.  Returns (choice, b_need,
        flags, b_eff_after, queue_after)."""
        b_eff = _i64(b_eff)
        D = b_eff.size
        a_p, a_U = _i32(a_p), _i32(a_U)
        A = a_p.size
        choice = np.zeros(A, np.int32)
        need = np.zeros(A, np.int64)
        flags = np.zeros(A, np.uint8)
        b_after = np.zeros(D, np.int64)
        q_after = np.zeros(D, np.int32)
        rc = self.lib.oracle_place_static(D, b_eff, _i32(queue_len), int(S), A, a_p, a_U, int(policy),
                                          int(rr_offset), int(bool(reserve)), choice, need, flags, b_after, q_after)
        if rc:
            raise ValueError(f"oracle_place_static failed ({rc})")
        return choice, need, flags, b_after, q_after

    # -- placement with sequential commit (Sec. 3.3, Algorithm 1) -----------
    def place_commit(self, seg_off, p, g, U, capacity, queue_len, a_p, a_U, policy=POLICY_MQ, rr_offset=0):
        """Arrivals in order, each committed to its decoder's projected
        occupancy (and queue) before the next.  Returns a PlaceResult (no pair
        matrix, no base peaks) and the queue lengths after the batch."""
        seg_off = _i64(seg_off)
        D = seg_off.size - 1
        a_p, a_U = _i32(a_p), _i32(a_U)
        A = a_p.size
        out = PlaceResult(choice=np.zeros(A, np.int32), chosen_peak=np.zeros(A, np.int64),
                          chosen_overflow=np.zeros(A, np.int64), flags=np.zeros(A, np.uint8), pair_peak=None,
                          base_peak=np.zeros(0, np.int64))
        q_after = np.zeros(D, np.int32)
        rc = self.lib.oracle_place_commit(D, seg_off, _i32(p), _i32(g), _i32(U), _i32(capacity), _i32(queue_len),
                                          A, a_p, a_U, int(policy), int(rr_offset), out.choice, out.chosen_peak,
                                          out.chosen_overflow, out.flags, q_after)
        if rc:
            raise ValueError(f"oracle_place_commit failed ({rc})")
        return out, q_after

    # -- App. A pressure simulation --------------------------------------------
    def simulate(self, N: int, C: int, theta_ppm: int, arrival_ms, prompt, output, bound=None, policy: int = 0):
        """Round-robin (policy 0) or Algorithm 1 (policy 1) routing of the
        requests onto N decoders of C tokens, one millisecond at a time.
        Returns a SimResult."""
        arrival_ms = _i64(arrival_ms)
        prompt, output = _i32(prompt), _i32(output)
        n = prompt.size
        bound = np.full(n, -1, np.int32) if bound is None else _i32(bound)
        r = SimResult(finish_ms=np.zeros(n, np.int64), routed=np.zeros(n, np.int32),
                      hp_time=np.zeros(N, np.int64), hp_max=np.zeros(N, np.int64), hp_count=np.zeros(N, np.int64),
                      max_queue=np.zeros(N, np.int64), queue_area=np.zeros(N, np.int64),
                      span=np.zeros(2, np.int64))
        rc = self.lib.oracle_simulate(int(N), int(C), int(theta_ppm), n, arrival_ms, prompt, output, bound,
                                      int(policy), r.finish_ms, r.routed, r.hp_time, r.hp_max, r.hp_count,
                                      r.max_queue, r.queue_area, r.span)
        if rc:
            raise ValueError(f"oracle_simulate failed ({rc})")
        return r

    # -- local order (Sec. 3.3, Eq. (7); App. A, Eq. (10)) -------------------
    def local_order(self, seg_off, p, g, U, capacity, q_off, q_p, q_U, q_wait, max_wait_ms,
                    u_max):
        seg_off, q_off = _i64(seg_off), _i64(q_off)
        D = seg_off.size - 1
        order = np.zeros(int(q_off[-1]), np.int32)
        admitted = np.zeros(D, np.int32)
        rc = self.lib.oracle_local_order(
            D, seg_off, _i32(p), _i32(g), _i32(U), _i32(capacity), q_off, _i32(q_p), _i32(q_U),
            None if q_wait is None else _i32(q_wait), int(max_wait_ms), int(u_max), order,
            admitted)
        if rc:
            raise ValueError(f"oracle_local_order failed ({rc})")
        return order, admitted

    # -- brute force (tiny inputs) -------------------------------------------
    def bruteforce_peak(self, p, g, U, q=(), V=()):
        q, V = _i32(q), _i32(V)
        qq = q if q.size else np.zeros(1, np.int32)
        VV = V if V.size else np.zeros(1, np.int32)
        return int(self.lib.oracle_bruteforce_peak(len(p), _i32(p), _i32(g), _i32(U),
                                                   q.size, qq, VV))


@dataclass
class PlaceResult:
    choice: np.ndarray
    chosen_peak: np.ndarray
    chosen_overflow: np.ndarray
    flags: np.ndarray
    pair_peak: np.ndarray | None
    base_peak: np.ndarray


@dataclass
class SimResult:
    finish_ms: np.ndarray
    routed: np.ndarray
    hp_time: np.ndarray
    hp_max: np.ndarray
    hp_count: np.ndarray
    max_queue: np.ndarray
    queue_area: np.ndarray
    span: np.ndarray


@dataclass
class StepResult:
    q: np.ndarray
    count: np.ndarray
    U: np.ndarray
    base_peak: np.ndarray
    place: PlaceResult
    order: np.ndarray
    admitted: np.ndarray


def step(batch, oracle: Oracle | None = None, capacity=None, want_pairs=True, policy=POLICY_MQ,
         rr_offset=0) -> StepResult:
    """The whole hot path on the CPU for one synthetic batch: calibrate, bound
    every resident, arrival and queued request, project, place, order."""
    o = oracle or Oracle()
    cap = batch.capacity if capacity is None else capacity
    q, cnt = o.calibrate(batch.cal_pred, batch.cal_truth, batch.edges, batch.alpha_ppm)
    U = o.apply_bounds(batch.apply_pred(), batch.edges, q, batch.u_max)
    U_res, U_arr, U_q = batch.split_bounds(U)
    base = o.project(batch.seg_off, batch.res_prompt, batch.res_gen, U_res)
    pl = o.place(batch.seg_off, batch.res_prompt, batch.res_gen, U_res, cap, batch.queue_len,
                 batch.arr_prompt, U_arr, policy=policy, rr_offset=rr_offset,
                 want_pairs=want_pairs)
    order, admitted = o.local_order(batch.seg_off, batch.res_prompt, batch.res_gen, U_res, cap,
                                    batch.q_off, batch.q_prompt, U_q, batch.q_wait_ms,
                                    batch.max_wait_ms, batch.u_max)
    return StepResult(q=q, count=cnt, U=U, base_peak=base, place=pl, order=order,
                      admitted=admitted)
