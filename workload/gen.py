"""Seeded synthetic inputs for the scheduler core.

This module only draws random inputs; it computes none of the scheduler's
quantities (no residual, quantile, bound, occupancy, peak or ordering).  Both
the GPU path and the CPU oracle consume exactly the arrays produced here.

Per request the generator draws a prompt length, a true output length and a
speculative prediction ``pred = max(1, rint(true * exp(sigma * z)))``, the
synthetic stand-in for the device-side predictor (Sec. 3.1).  A resident
request has already generated ``g = floor(f * true)`` tokens, f ~ U[0, 1): it
is partway through its true output.  Upper bounds are not drawn here: they are
what calibration computes from ``pred``.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass

import numpy as np

from .configs import WORKLOADS, LogNormal, PromptMix, Workload

INT32_MAX = np.iinfo(np.int32).max


def _lognormal(rng: np.random.Generator, n: int, m: LogNormal) -> np.ndarray:
    z = rng.standard_normal(n)
    return np.clip(np.rint(np.exp(m.mu + m.sigma * z)), m.lo, m.hi).astype(np.int32)


def _prompts(rng: np.random.Generator, n: int, pm: PromptMix) -> np.ndarray:
    p = _lognormal(rng, n, pm.base)
    if pm.long_frac > 0.0:
        is_long = rng.random(n) < pm.long_frac
        longs = rng.integers(pm.long_lo, pm.long_hi + 1, size=n, dtype=np.int64)
        p = np.where(is_long, longs, p).astype(np.int32)
    return p


def _predict(rng: np.random.Generator, true: np.ndarray, sigma: float) -> np.ndarray:
    z = rng.standard_normal(true.size)
    pred = np.rint(true.astype(np.float64) * np.exp(sigma * z))
    return np.clip(pred, 1, INT32_MAX).astype(np.int32)


@dataclass
class Batch:
    """One batch of scheduler input, all int32 token counts unless noted."""
    workload: Workload
    alpha_ppm: int
    u_max: int
    max_wait_ms: int
    # calibration set D_cal (Sec. 3.2)
    cal_pred: np.ndarray
    cal_truth: np.ndarray
    edges: np.ndarray            # nb-1 ascending bucket edges on pred
    # residents, decoder-major segments
    seg_off: np.ndarray          # int64 [D+1]
    res_prompt: np.ndarray
    res_gen: np.ndarray
    res_pred: np.ndarray
    # arrivals J_i
    arr_prompt: np.ndarray
    arr_pred: np.ndarray
    # decoders
    capacity: np.ndarray         # C_k, tokens
    queue_len: np.ndarray        # Q_k
    # pending local queues, decoder-major segments
    q_off: np.ndarray            # int64 [D+1]
    q_prompt: np.ndarray
    q_pred: np.ndarray
    q_wait_ms: np.ndarray

    @property
    def decoders(self) -> int:
        return int(self.capacity.size)

    @property
    def arrivals(self) -> int:
        return int(self.arr_prompt.size)

    def apply_pred(self) -> np.ndarray:
        """Predictions that calibration turns into bounds, in the order
        residents | arrivals | queued requests."""
        return np.concatenate([self.res_pred, self.arr_pred, self.q_pred]).astype(np.int32)

    def split_bounds(self, U: np.ndarray):
        """Inverse of :meth:`apply_pred` on the bound array."""
        nr, na = self.res_pred.size, self.arr_pred.size
        return U[:nr], U[nr:nr + na], U[nr + na:]

    def arrays(self) -> dict:
        return {k: v for k, v in self.__dict__.items() if isinstance(v, np.ndarray)}


def make(name_or_workload, alpha_ppm: int | None = None, seed: int | None = None) -> Batch:
    """Draw the batch of one workload.  Deterministic in (workload, seed)."""
    w = WORKLOADS[name_or_workload] if isinstance(name_or_workload, str) else name_or_workload
    seed = w.seed if seed is None else seed
    alpha_ppm = w.alphas_ppm[0] if alpha_ppm is None else alpha_ppm
    s_cal, s_res, s_arr, s_dec, s_q = np.random.SeedSequence(seed).spawn(5)

    rng = np.random.Generator(np.random.PCG64(s_cal))
    truth = _lognormal(rng, w.n_cal, w.output)
    cal_pred = _predict(rng, truth, w.pred_sigma)
    nb = w.buckets
    if w.n_cal > 0 and nb > 1:
        sp = np.sort(cal_pred)
        edges = sp[(np.arange(1, nb, dtype=np.int64) * w.n_cal) // nb].astype(np.int32)
    else:
        edges = np.zeros(max(nb - 1, 0), dtype=np.int32)

    D, n = w.decoders, w.residents
    rng = np.random.Generator(np.random.PCG64(s_res))
    res_prompt = _prompts(rng, D * n, w.prompt)
    res_true = _lognormal(rng, D * n, w.output)
    res_pred = _predict(rng, res_true, w.pred_sigma)
    res_gen = np.floor(rng.random(D * n) * w.gen_frac * res_true).astype(np.int32)
    seg_off = np.arange(D + 1, dtype=np.int64) * n

    rng = np.random.Generator(np.random.PCG64(s_arr))
    arr_prompt = _prompts(rng, w.arrivals, w.prompt)
    arr_true = _lognormal(rng, w.arrivals, w.output)
    arr_pred = _predict(rng, arr_true, w.pred_sigma)

    rng = np.random.Generator(np.random.PCG64(s_dec))
    capacity = rng.choice(np.asarray(w.capacities, dtype=np.int64), size=D).astype(np.int32)
    if w.queue_fixed is not None:
        queue_len = np.full(D, w.queue_fixed, dtype=np.int32)
    else:
        queue_len = rng.integers(0, w.queue_max + 1, size=D).astype(np.int32)

    rng = np.random.Generator(np.random.PCG64(s_q))
    nq = int(queue_len.sum())
    q_off = np.zeros(D + 1, dtype=np.int64)
    q_off[1:] = np.cumsum(queue_len, dtype=np.int64)
    q_prompt = _prompts(rng, nq, w.prompt)
    q_true = _lognormal(rng, nq, w.output)
    q_pred = _predict(rng, q_true, w.pred_sigma)
    q_wait = np.floor(rng.exponential(w.wait_mean_ms, size=nq)).astype(np.int32)

    return Batch(workload=w, alpha_ppm=int(alpha_ppm), u_max=w.u_max, max_wait_ms=w.max_wait_ms,
                 cal_pred=cal_pred, cal_truth=truth, edges=edges,
                 seg_off=seg_off, res_prompt=res_prompt, res_gen=res_gen, res_pred=res_pred,
                 arr_prompt=arr_prompt, arr_pred=arr_pred,
                 capacity=capacity, queue_len=queue_len,
                 q_off=q_off, q_prompt=q_prompt, q_pred=q_pred, q_wait_ms=q_wait)


def window_seen(batch: Batch, seed: int | None = None) -> np.ndarray:
    """For sliding-window calibration: how many entries of the completion log
    (the calibration pairs, oldest first) each bounded request had seen when
    its bound was taken, in :meth:`Batch.apply_pred` order.  Residents were
    bounded at earlier times, uniform over the log; arrivals and queued
    requests see all of it.  int64."""
    seed = batch.workload.seed if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(5,))))
    n = batch.cal_pred.size
    res = rng.integers(0, n + 1, size=batch.res_pred.size, dtype=np.int64)
    rest = np.full(batch.arr_pred.size + batch.q_pred.size, n, dtype=np.int64)
    return np.concatenate([res, rest])


def manifest(batch: Batch) -> dict:
    """SHA-256 of every input array (bytes in native little-endian order)."""
    return {k: hashlib.sha256(np.ascontiguousarray(v).tobytes()).hexdigest()
            for k, v in sorted(batch.arrays().items())}


def heldout(name_or_workload, n: int, seed: int):
    """Fresh (pred, truth) pairs from a workload's length model, for coverage checks."""
    w = WORKLOADS[name_or_workload] if isinstance(name_or_workload, str) else name_or_workload
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7919])))
    truth = _lognormal(rng, n, w.output)
    return _predict(rng, truth, w.pred_sigma), truth
