"""Algorithm 1 on block counts on the GPU (maps_rsc_state, maps_place_static)
against the CPU oracle, bit for bit: the runtime state of every decoder in
blocks, and each arrival's B_need, choice and flags, both against the
reported state (independent arrivals) and with each dispatch reserving its
B_need and joining its queue before the next (the paper's atomic
reservation).  Hand-worked example, random ragged shapes (decoder tiles, the
1,024-decoder limit of the reserving kernel, empty batches), the five seeded
workloads at block size 16, and the device error bits."""
import numpy as np
import pytest

import oracle
import workload
from tests.gpu_common import assert_same, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def orc():
    return oracle.Oracle()


def _cuda(x, dtype=np.int32):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=dtype)).cuda()


def _rsc(seg, p, g, U, cap, S, in_flight=None):
    import torch

    import paper_2609_15359_amd as maps
    fl = None if in_flight is None else _cuda(in_flight, np.uint8)
    bf, br, be, err = maps.rsc_state(_cuda(seg, np.int64), _cuda(p), _cuda(g), _cuda(U), _cuda(cap), S,
                                     in_flight=fl)
    torch.cuda.synchronize()
    return bf.cpu().numpy(), br.cpu().numpy(), be.cpu().numpy(), int(err.item()) & 0xFFFFFFFF


def _static(B, Q, S, a_p, a_U, policy=0, rr=0, reserve=False):
    import torch

    import paper_2609_15359_amd as maps
    r = maps.place_static(_cuda(B, np.int64), _cuda(Q), S, _cuda(a_p), _cuda(a_U), policy, rr, reserve)
    torch.cuda.synchronize()
    return tuple(t.cpu().numpy() for t in r[:5]) + (int(r[5].item()) & 0xFFFFFFFF,)


def _compare(got, want, tag):
    for name, g, w in zip(("choice", "b_need", "flags", "b_eff_after", "queue_after"), got[:5], want):
        assert_same(f"{tag} {name}", g, w)


def test_hand_worked_example():
    from tests.oracle_pins import golden
    gd = golden("place_static_hand.json")
    r = gd["rsc"]
    bf, br, be, err = _rsc(r["seg_off"], r["p"], r["g"], r["U"], r["capacity"], r["S"])
    assert err == 0
    assert bf.tolist() == r["b_free"] and br.tolist() == r["b_res"] and be.tolist() == r["b_eff"]
    pl = gd["place"]
    for mode, reserve in (("no_reserve", False), ("reserve", True)):
        ch, need, fl, ba, qa, err = _static(pl["b_eff"], pl["queue_len"], pl["S"], pl["a_p"], pl["a_U"],
                                            reserve=reserve)
        assert err == 0
        assert ch.tolist() == pl[mode]["choice"] and need.tolist() == pl["b_need"] and fl.tolist() == pl["flags"]
        assert ba.tolist() == pl[mode]["b_eff_after"] and qa.tolist() == pl[mode]["queue_after"]


# (D, A): one decoder, ragged arrival counts, decoder tiles of 2,048 (independent only), the reserving limit
SHAPES = [(1, 1), (3, 0), (5, 63), (7, 65), (64, 5000), (257, 3001), (1024, 20000), (3000, 9000), (5000, 700)]


@pytest.mark.parametrize("D,A", SHAPES, ids=[f"D{s[0]}-A{s[1]}" for s in SHAPES])
@pytest.mark.parametrize("policy", [0, 1])
def test_ragged_shapes(orc, D, A, policy):
    rng = np.random.default_rng(31 * D + A + policy)
    S = int(rng.choice([1, 16, 37]))
    B = rng.integers(-3000, 6000, size=D)
    B[: min(D, 3)] = B[0]   # ties
    Q = rng.integers(0, 8, size=D)
    a_p = rng.integers(0, 20000, size=A)
    a_U = rng.integers(-3, 40000, size=A)
    for reserve in (False, True):
        if reserve and D > 1024:
            continue
        say(f"[static] D={D} A={A} S={S} policy={policy} reserve={reserve}")
        want = orc.place_static(B, Q, S, a_p, a_U, policy, 2**33 + 5, reserve)
        got = _static(B, Q, S, a_p, a_U, policy, 2**33 + 5, reserve)
        assert got[5] == 0
        _compare(got, want, f"D{D} A{A} reserve={reserve}")


@pytest.mark.parametrize("case", ["wide", "alternating", "long_queues", "spread"])
@pytest.mark.parametrize("policy", [0, 1])
def test_reserve_key_widths(orc, case, policy):
    """The reserving chain takes each run of 64 arrivals with 32-bit keys when
    its needs sum to less than 2^21 blocks and the queues stay below 2^21,
    else with 64-bit keys: runs of huge needs only, narrow and wide runs in
    turn, queues past 2^21, and decoders 2^21 blocks or more below the largest
    B_eff (their 32-bit keys saturate) with some decoders feasible."""
    rng = np.random.default_rng(len(case) * 7 + policy)
    D, A, S = 200, 1000, 1
    B = rng.integers(-3000, 6000, size=D)
    Q = rng.integers(0, 8, size=D)
    a_p = rng.integers(0, 20000, size=A)
    a_U = rng.integers(-3, 40000, size=A)
    if case == "wide":
        a_p = rng.integers(10**6, 10**8, size=A)
    elif case == "alternating":
        huge = (np.arange(A) // 64) % 2 == 1
        a_p = np.where(huge, rng.integers(10**6, 10**8, size=A), rng.integers(0, 200, size=A))
        a_U = np.where(huge, a_U, rng.integers(-1, 300, size=A))
    elif case == "long_queues":
        Q = rng.integers(2**21 - 40, 2**21 + 40, size=D)
        a_p = rng.integers(0, 200, size=A)
        a_U = rng.integers(-1, 300, size=A)
    else:   # spread: half the decoders near the largest B_eff, the rest 2^21 or more below, a few at the edge
        B = np.concatenate([rng.integers(10**9, 10**9 + 5000, size=D // 2),
                            rng.integers(-10**9, 10**9 - 10**7, size=D - D // 2)])
        B[-5:] = B[: D // 2].max() - 2**21 + np.arange(-2, 3)
        a_p = rng.integers(0, 300, size=A)
        a_U = rng.integers(-1, 1000, size=A)
    a_p, a_U = a_p.astype(np.int32), a_U.astype(np.int32)
    want = orc.place_static(B, Q, S, a_p, a_U, policy, 7, True)
    got = _static(B, Q, S, a_p, a_U, policy, 7, True)
    assert got[5] == 0
    _compare(got, want, f"key widths {case} policy={policy}")


def test_water_filling_with_reservation(orc):
    """Every decoder feasible throughout: shortest queues fill level by level."""
    D, A = 37, 5000
    Q = np.random.default_rng(5).integers(0, 9, size=D)
    a = np.random.default_rng(6).integers(0, 500, size=(2, A))
    got = _static(np.full(D, 10**12), Q, 16, a[0], a[1], reserve=True)
    slots = sorted((int(Q[d]) + m, d) for d in range(D) for m in range(A))
    assert got[0].tolist() == [d for _, d in slots[:A]]
    _compare(got, orc.place_static(np.full(D, 10**12), Q, 16, a[0], a[1], reserve=True), "water filling")


@pytest.mark.parametrize("name", ["tiny", "small", "medium", "large", "xlarge"])
def test_workload_block16(orc, name):
    """The seeded workloads at block size 16: the runtime state from the
    residents (bounds from the oracle's calibration of the batch) and every
    arrival, independent and with reservation; and a variant whose
    capacities leave room (both branches of Algorithm 1)."""
    b = workload.make(name)
    o = oracle.step(b, orc, want_pairs=False)
    U_res, U_arr, _ = b.split_bounds(o.U)
    say(f"[static] {name}: D={b.decoders} A={b.arrivals}")
    want_state = orc.rsc_state(b.seg_off, b.res_prompt, b.res_gen, U_res, b.capacity, 16)
    got_state = _rsc(b.seg_off, b.res_prompt, b.res_gen, U_res, b.capacity, 16)
    assert got_state[3] == 0
    for nm, g, w in zip(("b_free", "b_res", "b_eff"), got_state[:3], want_state):
        assert_same(nm, g, w)
    be = want_state[2]
    need_med = int(np.median((b.arr_prompt.astype(np.int64) + np.maximum(U_arr, 0) + 15) // 16))
    roomy = be - be.min() + np.random.default_rng(3).integers(0, 40 * need_med + 1, size=b.decoders)
    for tag, B in (("literal", be), ("roomy", roomy)):
        for reserve in (False, True):
            want = orc.place_static(B, b.queue_len, 16, b.arr_prompt, U_arr, 0, 7, reserve)
            got = _static(B, b.queue_len, 16, b.arr_prompt, U_arr, 0, 7, reserve)
            assert got[5] == 0
            _compare(got, want, f"{name} {tag} reserve={reserve}")
            say(f"[static] {name} {tag} reserve={reserve}: feasible fraction {np.mean(want[2] & 1):.3f}")


def test_error_bits():
    _, _, _, err = _rsc([0, 2], [5, -1], [0, 0], [3, 3], [100], 16)
    assert err & 1
    _, _, _, err = _rsc([0, 5], [5, 1], [0, 0], [3, 3], [100], 16)
    assert err & 8
    _, _, _, err = _rsc([0, 1], [5], [0], [3], [-100], 16)
    assert err & 1
    got = _static([2**53, 5], [0, 0], 16, [1, 2], [3, 4], reserve=True)
    assert got[5] & 1024
    got = _static([5, 5], [0, 0], 16, [-1, 2], [3, 4], reserve=False)
    assert got[5] & 1
    got = _static([5, 5], [0, 0], 16, [-1, 2], [3, 4], reserve=True)
    assert got[5] & 1


@pytest.mark.parametrize("S", [1, 3, 16])
def test_staged_reservation(orc, S):
    """Requests whose prompt KV is still in transfer (whole budget reserved,
    nothing held) mixed with residents: random ragged decoders and the large
    workload with a tenth of its residents in flight."""
    rng = np.random.default_rng(60 + S)
    for trial in range(20):
        D = int(rng.integers(1, 40))
        counts = rng.integers(0, 700, size=D)
        seg = np.zeros(D + 1, np.int64)
        seg[1:] = np.cumsum(counts)
        n = int(seg[-1])
        p = rng.integers(0, 5000, size=n)
        g = rng.integers(0, 3000, size=n)
        U = np.where(rng.random(n) < 0.1, -1, rng.integers(0, 9000, size=n))
        fl = (rng.random(n) < 0.3).astype(np.uint8)
        cap = rng.integers(0, 2**31 - 1, size=D)
        got = _rsc(seg, p, g, U, cap, S, fl)
        assert got[3] == 0
        want = orc.rsc_state(seg, p, g, U, cap, S, in_flight=fl)
        for nm, gg, w in zip(("b_free", "b_res", "b_eff"), got[:3], want):
            assert_same(f"{nm} trial {trial}", gg, w)
    b = workload.make("large")
    o = oracle.step(b, orc, want_pairs=False)
    U_res, _, _ = b.split_bounds(o.U)
    fl = (np.random.default_rng(7).random(U_res.size) < 0.1).astype(np.uint8)
    got = _rsc(b.seg_off, b.res_prompt, b.res_gen, U_res, b.capacity, S, fl)
    assert got[3] == 0
    want = orc.rsc_state(b.seg_off, b.res_prompt, b.res_gen, U_res, b.capacity, S, in_flight=fl)
    for nm, gg, w in zip(("b_free", "b_res", "b_eff"), got[:3], want):
        assert_same(f"large {nm}", gg, w)
