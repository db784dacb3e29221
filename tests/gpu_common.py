"""Shared helpers of the GPU parity tests: run the HIP path and the CPU oracle
on the same seeded batch and compare every output element by element."""
from __future__ import annotations

import sys

import numpy as np

import oracle
import workload
from workload.gen import Batch

Q_INF = 2**31 - 1


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def gpu_step(b: Batch, capacity=None, want_pairs=True, policy=0, rr_offset=0, fused=False):
    """The whole step on the GPU; fused=True makes placement and local order
    one call (maps_place_order); fused="project" makes projection and local
    order one call (maps_project_order), as the benchmark does."""
    import torch

    import paper_2609_15359_amd as maps
    from paper_2609_15359_amd import pipeline
    db = pipeline.to_device(b)
    cap = None if capacity is None else torch.from_numpy(np.ascontiguousarray(capacity, np.int32)).cuda()
    out = pipeline.step(db, want_pairs=want_pairs, capacity=cap, policy=policy, rr_offset=rr_offset, fused=fused)
    torch.cuda.synchronize()
    bits = int(out.dev_err.item()) & 0xFFFFFFFF
    pl = out.placement
    res = dict(
        err=bits, errors=maps.error_names(bits),
        q=out.q.cpu().numpy(), count=out.count.cpu().numpy(), U=out.U.cpu().numpy(),
        base_peak=out.base_peak.cpu().numpy(),
        choice=pl.choice.cpu().numpy(), chosen_peak=pl.chosen_peak.cpu().numpy(),
        chosen_overflow=pl.chosen_overflow.cpu().numpy(), flags=pl.flags.cpu().numpy(),
        pair_peak=None if pl.pair_peak is None else pl.pair_peak.cpu().numpy(),
        order=out.order.cpu().numpy(), admitted=out.admitted.cpu().numpy())
    # the snapshot's decoder headers (16 int32 each: slice offset lo/hi, total lo/hi, E, base peak,
    # hot window low, hot window high, flat region start, PMX_E, padding), behind its 256-byte header
    D = b.decoders
    res["dec_hdr"] = out.snapshot.data[256:256 + 64 * D].view(torch.int32).view(D, 16).cpu().numpy()
    return res


def oracle_step(b: Batch, capacity=None, want_pairs=True, policy=0, rr_offset=0, o=None):
    r = oracle.step(b, o, capacity=capacity, want_pairs=want_pairs, policy=policy, rr_offset=rr_offset)
    return dict(q=r.q, count=r.count, U=r.U, base_peak=r.base_peak, choice=r.place.choice,
                chosen_peak=r.place.chosen_peak, chosen_overflow=r.place.chosen_overflow,
                flags=r.place.flags, pair_peak=r.place.pair_peak, order=r.order, admitted=r.admitted)


def assert_same(name, got, want):
    got = np.asarray(got)
    want = np.asarray(want)
    assert got.shape == want.shape, f"{name}: shape {got.shape} != {want.shape}"
    eq = got.astype(np.int64) == want.astype(np.int64)
    if not eq.all():
        bad = np.argwhere(~eq)
        i = tuple(bad[0])
        raise AssertionError(f"{name}: {bad.shape[0]} of {eq.size} differ; first at {i}: "
                             f"gpu {got[i]} oracle {want[i]}")


def compare_all(g, o, pairs=True):
    for k in ("q", "count", "U", "base_peak", "choice", "chosen_peak", "chosen_overflow", "flags",
              "order", "admitted"):
        assert_same(k, g[k], o[k])
    if pairs and g["pair_peak"] is not None and o["pair_peak"] is not None:
        assert_same("pair_peak", g["pair_peak"], o["pair_peak"])


def fit_capacity(b: Batch, o_res: dict, seed: int = 99) -> np.ndarray:
    """Capacities with headroom over the oracle's base peaks, so that both the
    feasible branch and the fallback are taken: C_d = base_d + h_d,
    h_d ~ U{0 .. 2 median(p_a + U_a)} over arrivals with a bound."""
    _, U_arr, _ = b.split_bounds(o_res["U"])
    ok = U_arr >= 0
    med = int(np.median(b.arr_prompt[ok].astype(np.int64) + U_arr[ok])) if ok.any() else 0
    rng = np.random.default_rng(seed)
    h = rng.integers(0, 2 * med + 1, size=b.decoders)
    return np.minimum(o_res["base_peak"] + h, 2**31 - 1).astype(np.int32)


def custom_batch(*, cal_pred, cal_truth, edges, alpha_ppm, u_max, seg_off, res_prompt, res_gen, res_pred,
                 arr_prompt, arr_pred, capacity, queue_len=None, q_off=None, q_prompt=None, q_pred=None,
                 q_wait_ms=None, max_wait_ms=1000) -> Batch:
    """A hand-made batch with the same fields as a generated one."""
    i32 = lambda x: np.ascontiguousarray(x, dtype=np.int32)  # noqa: E731
    D = len(capacity)
    if q_off is None:
        q_off = np.zeros(D + 1, np.int64)
        q_prompt = q_pred = q_wait_ms = np.zeros(0, np.int32)
    if queue_len is None:
        queue_len = np.diff(np.asarray(q_off, np.int64))
    w = workload.WORKLOADS["tiny"]
    return Batch(workload=w, alpha_ppm=int(alpha_ppm), u_max=int(u_max), max_wait_ms=int(max_wait_ms),
                 cal_pred=i32(cal_pred), cal_truth=i32(cal_truth), edges=i32(edges),
                 seg_off=np.ascontiguousarray(seg_off, np.int64), res_prompt=i32(res_prompt),
                 res_gen=i32(res_gen), res_pred=i32(res_pred), arr_prompt=i32(arr_prompt),
                 arr_pred=i32(arr_pred), capacity=i32(capacity), queue_len=i32(queue_len),
                 q_off=np.ascontiguousarray(q_off, np.int64), q_prompt=i32(q_prompt), q_pred=i32(q_pred),
                 q_wait_ms=i32(q_wait_ms))
