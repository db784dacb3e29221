"""Placement with sequential commit on the GPU (maps_place_commit) against
the CPU oracle, bit for bit: arrivals in order, each committed to its
decoder's projected occupancy and queue before the next (Sec. 3.3, Algorithm
1).  Random ragged decoders and arrival mixes, both policies, round-robin
arrivals, capacity ties, the seeded workloads (literal and with room), the
single-arrival case against maps_place, and the device error bits."""
import numpy as np
import pytest

import oracle
import workload
from tests.gpu_common import assert_same, fit_capacity, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def orc():
    return oracle.Oracle()


def _cuda(x, dtype=np.int32):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=dtype)).cuda()


def _gpu(seg, p, g, U, u_max, cap, Q, a_p, a_U, policy=0, rr=0):
    import torch

    import paper_2609_15359_amd as maps
    snap, _, err = maps.project(_cuda(seg, np.int64), _cuda(p), _cuda(g), _cuda(U), u_max)
    out = maps.place_commit(snap, _cuda(cap), _cuda(Q), _cuda(a_p), _cuda(a_U), policy, rr, dev_err=err)
    torch.cuda.synchronize()
    return dict(choice=out.choice.cpu().numpy(), chosen_peak=out.chosen_peak.cpu().numpy(),
                chosen_overflow=out.chosen_overflow.cpu().numpy(), flags=out.flags.cpu().numpy(),
                queue_out=out.queue_out.cpu().numpy(), err=int(err.item()) & 0xFFFFFFFF)


def _compare(g, r, q_after, tag):
    assert g["err"] == 0, tag
    for f in ("choice", "chosen_peak", "chosen_overflow", "flags"):
        assert_same(f"{tag} {f}", g[f], getattr(r, f))
    assert_same(f"{tag} queue_out", g["queue_out"], q_after)


def _random_case(rng, D, nmax, A, u_max):
    counts = rng.integers(0, nmax + 1, size=D)
    seg = np.zeros(D + 1, np.int64)
    seg[1:] = np.cumsum(counts)
    n = int(seg[-1])
    U = rng.integers(0, u_max + 1, size=n)
    g = rng.integers(0, u_max + 1, size=n)           # g may exceed U: remaining length 0
    p = rng.integers(0, 3000, size=n)
    a_p = rng.integers(0, 3000, size=A)
    a_U = np.where(rng.random(A) < 0.1, -1, rng.integers(0, u_max + 1, size=A))
    return seg, p, g, U, a_p, a_U


@pytest.mark.parametrize("D,nmax,A,u_max", [(1, 5, 40, 50), (3, 30, 300, 2000), (17, 200, 700, 9000),
                                            (64, 40, 2100, 1023), (300, 8, 900, 70),
                                            # ranges longer than the chain's LDS stage, many floor blocks
                                            (4, 60, 500, 40000),
                                            # more decoders than threads: no lookups ahead
                                            (1100, 3, 250, 2500),
                                            # the most decoders the chain takes: the smallest LDS stage
                                            (8192, 2, 60, 100)])
def test_random(orc, D, nmax, A, u_max):
    rng = np.random.default_rng(D * 1000 + A)
    seg, p, g, U, a_p, a_U = _random_case(rng, D, nmax, A, u_max)
    base = orc.project(seg, p, g, U)
    # capacities around the base peaks plus a few arrivals: both branches, and queue growth matters
    cap = (base + rng.integers(0, 4 * (3000 + u_max), size=D)).astype(np.int32)
    Q = rng.integers(0, 5, size=D)
    for policy in (0, 1):
        rr = int(rng.integers(0, 1000))
        r, q_after = orc.place_commit(seg, p, g, U, cap, Q, a_p, a_U, policy=policy, rr_offset=rr)
        got = _gpu(seg, p, g, U, u_max, cap, Q, a_p, a_U, policy, rr)
        _compare(got, r, q_after, f"D={D} A={A} policy={policy}")
        say(f"[commit] D={D} A={A} policy={policy}: feasible {np.mean(r.flags & 1):.3f}")


def test_ties_and_empty_decoders(orc):
    # identical decoders (every key ties: lowest index first, then queue growth spreads them), empty decoders
    D = 6
    seg = np.array([0, 2, 4, 4, 6, 8, 8], np.int64)
    p = np.array([10, 20] * 4)
    g = np.array([1, 2] * 4)
    U = np.array([5, 7] * 4)
    a_p = np.full(40, 3)
    a_U = np.full(40, 4)
    cap = np.full(D, 10**6)
    for policy in (0, 1):
        r, q_after = orc.place_commit(seg, p, g, U, cap, np.zeros(D), a_p, a_U, policy=policy)
        got = _gpu(seg, p, g, U, 16, cap, np.zeros(D), a_p, a_U, policy)
        _compare(got, r, q_after, f"ties policy={policy}")


def test_single_arrival_is_maps_place(orc):
    import torch

    import paper_2609_15359_amd as maps
    rng = np.random.default_rng(5)
    seg, p, g, U, a_p, a_U = _random_case(rng, 9, 50, 1, 3000)
    a_U[:] = 1234
    cap = rng.integers(0, 300000, size=9)
    Q = rng.integers(0, 4, size=9)
    got = _gpu(seg, p, g, U, 3000, cap, Q, a_p, a_U)
    snap, _, err = maps.project(_cuda(seg, np.int64), _cuda(p), _cuda(g), _cuda(U), 3000)
    pl = maps.place(snap, _cuda(cap), _cuda(Q), _cuda(a_p), _cuda(a_U), dev_err=err)
    torch.cuda.synchronize()
    assert int(got["choice"][0]) == int(pl.choice[0]) and int(got["chosen_peak"][0]) == int(pl.chosen_peak[0])
    assert int(got["flags"][0]) == int(pl.flags[0])


@pytest.mark.parametrize("name,arrivals", [("tiny", None), ("small", None), ("medium", 6000), ("large", 3000)])
def test_workload(orc, name, arrivals):
    """The seeded workloads (bounds from the oracle's calibration of the
    batch): literal capacities, where every decoder is overloaded and each
    arrival takes the largest slack, and capacities with room; medium and
    large on their first arrivals (the oracle derives a decoder's maxima over
    the whole step axis at every commit)."""
    b = workload.make(name)
    o = oracle.step(b, orc, want_pairs=False)
    U_res, U_arr, _ = b.split_bounds(o.U)
    k = b.arrivals if arrivals is None else arrivals
    ap, aU = b.arr_prompt[:k], U_arr[:k]
    fit = fit_capacity(b, {"U": o.U, "base_peak": o.base_peak})
    for tag, cap in (("literal", b.capacity), ("room", fit)):
        r, q_after = orc.place_commit(b.seg_off, b.res_prompt, b.res_gen, U_res, cap, b.queue_len, ap, aU,
                                      rr_offset=11)
        got = _gpu(b.seg_off, b.res_prompt, b.res_gen, U_res, b.u_max, cap, b.queue_len, ap, aU, 0, 11)
        _compare(got, r, q_after, f"{name} {tag}")
        say(f"[commit] {name} {tag}: {k} arrivals, feasible fraction {np.mean(r.flags & 1):.3f}")


def test_error_bits():
    seg = np.array([0, 2], np.int64)
    ok = _gpu(seg, [5, 1], [0, 0], [3, 3], 10, [100], [0], [1, 2], [3, 4])
    assert ok["err"] == 0
    assert _gpu(seg, [5, 1], [0, 0], [3, 3], 10, [100], [0], [-1, 2], [3, 4])["err"] & 1
    assert _gpu(seg, [5, 1], [0, 0], [3, 3], 10, [100], [0], [-1, 2], [-1, 4])["err"] == 0   # no bound: RR
    assert _gpu(seg, [5, 1], [0, 0], [3, 3], 10, [-100], [0], [1, 2], [3, 4])["err"] & 1
    assert _gpu(seg, [5, 1], [0, 0], [3, 3], 10, [100], [-3], [1, 2], [3, 4])["err"] & 1
    assert _gpu(seg, [5, 1], [0, 0], [3, 3], 10, [100], [0], [1, 2], [3, 11])["err"] & 16


def test_snapshot_mismatch_is_reported():
    import torch

    import paper_2609_15359_amd as maps
    seg = np.array([0, 2], np.int64)
    snap, _, err = maps.project(_cuda(seg, np.int64), _cuda([5, 1]), _cuda([0, 0]), _cuda([3, 3]), 10)
    torch.cuda.synchronize()
    wrong = maps.Snapshot(data=snap.data, D=1, n_total=2, u_max=12)   # built for u_max 10
    e = maps.new_error_word()
    maps.place_commit(wrong, _cuda([100]), _cuda([0]), _cuda([1]), _cuda([3]), dev_err=e)
    torch.cuda.synchronize()
    assert int(e.item()) & 32
