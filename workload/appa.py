"""Seeded synthetic inputs of the App. A pressure simulation.

App. A simulates 10,000 requests on N = 4 decoders of C = 50,000 KV tokens
with t_tok = 1 ms and a high-pressure threshold of 0.85, drawing prompt and
output lengths from the empirical BurstGPT distributions and arrivals from a
Poisson process whose rate sets the utilisation rho = lambda E[L_out] t_tok / N.
The BurstGPT trace is not available here; its stand-in is the heavy-tailed
lognormal length model of the other workloads (prompt LN(6, 1) on [16, 4096],
output LN(6, 1.2) on [1, 8192], prediction noise 0.3).  As in App. A one
realisation is fixed (lengths and unit-rate inter-arrival gaps) and only the
load varies: arrival i comes at floor(G_i / lambda) ms, G_i the sum of the
first i + 1 unit-rate exponential gaps.  Calibration pairs are drawn from the
same model, so that the bounds MAPS routes by come from the calibration step.
Input generation only: nothing of the simulation is computed here.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

N_DECODERS = 4
CAPACITY = 50_000
THETA_PPM = 850_000
N_REQUESTS = 10_000
U_MAX = 8192
ALPHA_PPM = 100_000


@dataclass
class SimWorkload:
    prompt: np.ndarray       # int32 [n], L_p
    output: np.ndarray       # int32 [n], L_out
    pred: np.ndarray         # int32 [n], speculative prediction of L_out
    gaps: np.ndarray         # float64 [n], unit-rate exponential inter-arrival gaps
    cal_pred: np.ndarray     # int32, calibration pairs (prediction, observed length)
    cal_truth: np.ndarray
    edges: np.ndarray        # int32, equal-frequency bucket edges on cal_pred

    @property
    def n(self) -> int:
        return int(self.prompt.size)

    def mean_output(self) -> float:
        return float(self.output.astype(np.float64).mean())

    def arrivals(self, rho: float, N: int = N_DECODERS) -> np.ndarray:
        """Arrival times (int64 ms) at utilisation rho: lambda = rho N / E[L_out] per ms."""
        lam = rho * N / self.mean_output()
        return np.floor(np.cumsum(self.gaps) / lam).astype(np.int64)


def _lengths(rng, n, mu, sigma, lo, hi):
    return np.clip(np.rint(np.exp(mu + sigma * rng.standard_normal(n))), lo, hi).astype(np.int32)


def make(n: int = N_REQUESTS, seed: int = 7, n_cal: int = 20_000, buckets: int = 8) -> SimWorkload:
    ss = np.random.SeedSequence(seed).spawn(3)
    r_req, r_arr, r_cal = (np.random.default_rng(s) for s in ss)
    prompt = _lengths(r_req, n, 6.0, 1.0, 16, 4096)
    output = _lengths(r_req, n, 6.0, 1.2, 1, U_MAX)
    pred = np.clip(np.rint(output * np.exp(0.3 * r_req.standard_normal(n))), 1, 2**31 - 1).astype(np.int32)
    gaps = r_arr.exponential(1.0, size=n)
    cal_truth = _lengths(r_cal, n_cal, 6.0, 1.2, 1, U_MAX)
    cal_pred = np.clip(np.rint(cal_truth * np.exp(0.3 * r_cal.standard_normal(n_cal))), 1,
                       2**31 - 1).astype(np.int32)
    s = np.sort(cal_pred)
    edges = np.array([s[(j * n_cal) // buckets] for j in range(1, buckets)], np.int32)
    return SimWorkload(prompt, output, pred, gaps, cal_pred, cal_truth, edges)
