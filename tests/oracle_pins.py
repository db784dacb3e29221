"""Pins of the CPU oracle to facts fixed outside the oracle itself.

Each ``pin_*`` function takes an :class:`oracle.Oracle` and raises
AssertionError when the oracle disagrees with
  * a worked example computed by hand from the paper's definitions
    (``tests/golden/*.json``, each citing its passage),
  * a closed form or a special case that reduces to a textbook rule
    (Algorithm 1's static block test, order statistics),
  * an invariant of the definitions (coverage, monotonicity, peak bounds),
  * or a brute force written here in pure Python on tiny inputs.
The same functions run against deliberately broken builds of the oracle in
``test_oracle_mutants.py``, which shows each plausible mistake fails a pin.
"""
from __future__ import annotations

import json
import math
import os
from fractions import Fraction

import numpy as np

import workload

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
Q_INF = np.iinfo(np.int32).max


def golden(name: str) -> dict:
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------------------
# pure-Python brute force (tiny inputs)
# ---------------------------------------------------------------------------

def py_remaining(U, g):
    return max(int(U) - int(g), 0)


def py_occupancy(p, g, U, t):
    """Tokens held at step t by the residents (p+g+t while t <= R)."""
    return sum(int(pi) + int(gi) + t for pi, gi, Ui in zip(p, g, U) if t <= py_remaining(Ui, gi))


def py_peak(p, g, U, extra=()):
    """max over steps of residents plus extra (q, V) requests holding q+t for t <= V."""
    T = max([py_remaining(Ui, gi) for gi, Ui in zip(g, U)] + [V for _, V in extra] + [0])
    best = 0
    for t in range(T + 1):
        occ = py_occupancy(p, g, U, t) + sum(q + t for q, V in extra if t <= V)
        best = max(best, occ)
    return best


def _rng(seed):
    return np.random.default_rng(seed)


def _tiny_decoders(rng, D, nmax, umax, pmax):
    counts = rng.integers(0, nmax + 1, size=D)
    seg = np.zeros(D + 1, np.int64)
    seg[1:] = np.cumsum(counts)
    n = int(seg[-1])
    p = rng.integers(0, pmax + 1, size=n).astype(np.int32)
    U = rng.integers(0, umax + 1, size=n).astype(np.int32)
    g = rng.integers(0, umax + 3, size=n).astype(np.int32)     # g may exceed U
    return seg, p, g, U


# ---------------------------------------------------------------------------
# calibration (Sec. 3.2)
# ---------------------------------------------------------------------------

def pin_calibrate_golden(o):
    gd = golden("calibrate_hand.json")
    for case in gd["cases"]:
        q, cnt = o.calibrate(gd["pred"], gd["truth"], gd["edges"], case["alpha_ppm"])
        want = [Q_INF if v == "inf" else v for v in case["q"]]
        assert q.tolist() == want, (case, q)
        assert cnt.tolist() == case["count"], (case, cnt)
        for n_b, k in zip(case["count"], case["k"]):
            assert o.conformal_rank(n_b, case["alpha_ppm"]) == k
    ap = gd["apply"]
    q, _ = o.calibrate(gd["pred"], gd["truth"], gd["edges"], ap["alpha_ppm"])
    U = o.apply_bounds(ap["pred"], gd["edges"], q, gd["u_max"])
    assert U.tolist() == ap["U"], U
    ai = gd["apply_inf"]
    q, _ = o.calibrate(gd["pred"], gd["truth"], gd["edges"], ai["alpha_ppm"])
    U = o.apply_bounds(ai["pred"], gd["edges"], q, gd["u_max"])
    assert U.tolist() == ai["U"], U
    rt = gd["rank_threshold"]
    for n, k in zip(rt["n"], rt["k"]):
        assert o.conformal_rank(n, rt["alpha_ppm"]) == k, (n, k)


def pin_rank_is_ceiling(o):
    """k is the least integer with k >= (1 - alpha)(n + 1) (exact rationals)."""
    rng = _rng(11)
    alphas = [1, 50000, 100000, 250000, 333333, 500000, 999999] + list(rng.integers(1, 10**6, 20))
    ns = [0, 1, 2, 3, 8, 9, 10, 19, 99, 500, 3999999, 4000000] + list(rng.integers(0, 10**7, 20))
    for a in alphas:
        for n in ns:
            k = o.conformal_rank(int(n), int(a))
            x = (1 - Fraction(int(a), 10**6)) * (int(n) + 1)
            assert k >= x and k - 1 < x, (a, n, k)


def pin_quantile_order_statistic(o):
    """q_b is the k-th smallest score: #{s <= q} >= k and #{s < q} < k."""
    rng = _rng(12)
    for trial in range(30):
        n = int(rng.integers(0, 300))
        pred = rng.integers(0, 60, size=n).astype(np.int32)
        truth = rng.integers(0, 90, size=n).astype(np.int32)
        nb = int(rng.integers(1, 6))
        edges = np.sort(rng.integers(0, 60, size=nb - 1)).astype(np.int32)
        alpha = int(rng.choice([50000, 100000, 200000, 500000]))
        q, cnt = o.calibrate(pred, truth, edges, alpha)
        b = np.array([int(np.sum(edges <= v)) for v in pred], dtype=np.int64)
        s = np.maximum(0, truth.astype(np.int64) - pred.astype(np.int64))
        for j in range(nb):
            sj = s[b == j]
            assert cnt[j] == sj.size
            k = math.ceil((1 - Fraction(alpha, 10**6)) * (sj.size + 1))
            if k > sj.size:
                assert q[j] == Q_INF
            else:
                assert np.sum(sj <= q[j]) >= k and np.sum(sj < q[j]) < k, (trial, j)


def pin_quantile_special_cases(o):
    # every score zero: the quantile is 0 and the bound is the prediction itself
    pred = np.arange(1, 21, dtype=np.int32) * 10
    q, _ = o.calibrate(pred, pred - 5, [100], 100000)
    assert q.tolist() == [0, 0]
    U = o.apply_bounds(pred, [100], q, 10**6)
    assert U.tolist() == pred.tolist()
    # one bucket (no edges): the paper's single global quantile
    truth = pred + np.arange(20, dtype=np.int32)
    q, cnt = o.calibrate(pred, truth, [], 100000)
    assert cnt.tolist() == [20] and q.tolist() == [18]      # k = ceil(0.9*21) = 19 -> 19th smallest of 0..19
    # a duplicated edge leaves an empty bucket: infinite quantile, bound u_max
    q, cnt = o.calibrate(pred, truth, [100, 100], 100000)
    assert cnt[1] == 0 and q[1] == Q_INF
    # bucket boundaries: an edge equal to the prediction sends it up
    assert o.bucket(99, [100, 200]) == 0
    assert o.bucket(100, [100, 200]) == 1
    assert o.bucket(10**6, [100, 200]) == 2


def pin_quantile_monotone_in_alpha(o):
    b = workload.make("small")
    q05, _ = o.calibrate(b.cal_pred, b.cal_truth, b.edges, 50000)
    q10, _ = o.calibrate(b.cal_pred, b.cal_truth, b.edges, 100000)
    assert np.all(q05.astype(np.int64) >= q10.astype(np.int64))
    assert np.any(q05 != q10)
    pred = b.apply_pred()
    U05 = o.apply_bounds(pred, b.edges, q05, b.u_max)
    U10 = o.apply_bounds(pred, b.edges, q10, b.u_max)
    assert np.all(U05 >= U10)


def pin_coverage(o):
    """Eq. (5): held-out coverage P(L <= U) >= 1 - alpha within sampling error,
    and calibration-set coverage of every finite bucket quantile >= 1 - alpha."""
    for name, alpha in (("small", 50000), ("small", 100000), ("medium", 100000)):
        b = workload.make(name)
        q, cnt = o.calibrate(b.cal_pred, b.cal_truth, b.edges, alpha)
        pred, truth = workload.heldout(name, 200000, seed=5)
        U = o.apply_bounds(pred, b.edges, q, b.u_max)
        a = alpha / 1e6
        cov = float(np.mean(truth <= U))
        assert cov >= 1 - a - 3 * math.sqrt(a * (1 - a) / truth.size), (name, alpha, cov)
        assert cov <= 1 - a + 0.03, (name, alpha, cov)       # calibrated, not vacuous
        s = np.maximum(0, b.cal_truth.astype(np.int64) - b.cal_pred)
        bk = np.searchsorted(b.edges, b.cal_pred, side="right")
        for j in range(b.edges.size + 1):
            if q[j] != Q_INF:
                assert np.mean(s[bk == j] <= q[j]) >= 1 - a


# ---------------------------------------------------------------------------
# sliding-window calibration (Sec. 3.2; Sec. 4: the 500 most recent requests)
# ---------------------------------------------------------------------------

def py_window_quantile(pred, truth, edges, window, alpha_ppm, p, seen):
    """Brute force: walk the log back from entry seen-1, keep the scores of the
    request's bucket until `window` are found, take the k-th smallest."""
    if p < 0:
        return -1
    b = sum(1 for e in edges if e <= p)
    got = []
    i = seen - 1
    while i >= 0 and len(got) < window:
        if sum(1 for e in edges if e <= pred[i]) == b:
            got.append(max(0, int(truth[i]) - int(pred[i])))
        i -= 1
    k = math.ceil((1 - Fraction(alpha_ppm, 10**6)) * (len(got) + 1))
    return sorted(got)[k - 1] if k <= len(got) else Q_INF


def pin_window_golden(o):
    gd = golden("calibrate_window_hand.json")
    r = gd["requests"]
    for case in gd["cases"]:
        q, U = o.calibrate_window(gd["pred"], gd["truth"], gd["edges"], case["window"], case["alpha_ppm"],
                                  r["pred"], r["seen"], gd["u_max"])
        assert q.tolist() == [Q_INF if v == "inf" else v for v in case["q"]], (case, q)
        assert U.tolist() == case["U"], (case, U)


def pin_window_bruteforce(o):
    rng = _rng(31)
    for trial in range(40):
        n = int(rng.integers(0, 45))
        pred = rng.integers(0, 50, size=n).astype(np.int32)
        truth = rng.integers(0, 80, size=n).astype(np.int32)
        nb = int(rng.integers(1, 4))
        edges = np.sort(rng.integers(0, 50, size=nb - 1)).astype(np.int32)
        window = int(rng.choice([1, 2, 5, 9, 60]))
        alpha = int(rng.choice([50000, 100000, 250000, 500000, 900000]))
        m = 60
        ap = rng.integers(-2, 60, size=m).astype(np.int32)
        seen = rng.integers(0, n + 1, size=m).astype(np.int64)
        u_max = 70
        q, U = o.calibrate_window(pred, truth, edges, window, alpha, ap, seen, u_max)
        for j in range(m):
            want = py_window_quantile(pred, truth, edges, window, alpha, int(ap[j]), int(seen[j]))
            assert q[j] == want, (trial, j, q[j], want)
            if ap[j] < 0:
                assert U[j] == -1
            else:
                assert U[j] == (u_max if want == Q_INF else min(int(ap[j]) + want, u_max)), (trial, j)


def pin_window_closed_forms(o):
    """One bucket.  Scores equal to the log position: the set of a request
    that saw c completions is positions c-n_w .. c-1, so q = c - n_w + k - 1.
    Scores n - i (falling): q = n - c + k."""
    n, window, alpha = 300, 40, 100000
    i = np.arange(n, dtype=np.int32)
    pred = np.full(n, 10, np.int32)
    seen = np.arange(n + 1, dtype=np.int64)
    ap = np.full(n + 1, 10, np.int32)
    for truth, form in ((pred + i, lambda c, nw, k: c - nw + k - 1), (pred + (n - i), lambda c, nw, k: n - c + k)):
        q, _ = o.calibrate_window(pred, truth, [], window, alpha, ap, seen, 10**6)
        for c in range(n + 1):
            nw = min(c, window)
            k = math.ceil((1 - Fraction(alpha, 10**6)) * (nw + 1))
            assert q[c] == (form(c, nw, k) if k <= nw else Q_INF), (c, q[c])


def pin_window_reduces_to_fixed_set(o):
    """A window at least as long as the log, every request after the last
    completion: the set is the whole bucket, the quantile of numpy's sort."""
    b = workload.make("small")
    n = b.cal_pred.size
    ap = b.apply_pred()[:2000]
    q, U = o.calibrate_window(b.cal_pred, b.cal_truth, b.edges, n, b.alpha_ppm, ap,
                              np.full(ap.size, n, np.int64), b.u_max)
    s = np.maximum(0, b.cal_truth.astype(np.int64) - b.cal_pred)
    bk = np.searchsorted(b.edges, b.cal_pred, side="right")
    qb = []
    for j in range(b.edges.size + 1):
        sj = np.sort(s[bk == j])
        k = math.ceil((1 - Fraction(b.alpha_ppm, 10**6)) * (sj.size + 1))
        qb.append(int(sj[k - 1]) if k <= sj.size else Q_INF)
    want = np.where(ap < 0, -1, np.array(qb)[np.searchsorted(b.edges, np.maximum(ap, 0), side="right")])
    assert np.array_equal(q, want)
    assert np.array_equal(U, o.apply_bounds(ap, b.edges, np.array(qb, np.int32), b.u_max))


def pin_window_coverage(o):
    """Eq. (5) online: each completion, bounded from the window of the ones
    before it (500 most recent, Sec. 4), is covered with probability at least
    1 - alpha; a smaller alpha never gives a smaller bound."""
    for name, alpha in (("small", 100000), ("small", 50000)):
        b = workload.make(name)
        n = b.cal_pred.size
        seen = np.arange(n, dtype=np.int64)
        q, U = o.calibrate_window(b.cal_pred, b.cal_truth, b.edges, 500, alpha, b.cal_pred, seen, b.u_max)
        warm = np.arange(n) >= min(n // 2, 2 * 500 * (b.edges.size + 1))   # windows mostly full
        a = alpha / 1e6
        cov = float(np.mean(b.cal_truth[warm] <= U[warm]))
        m = int(warm.sum())
        assert cov >= 1 - a - 3 * math.sqrt(a * (1 - a) / m), (name, cov)
        assert cov <= 1 - a + 0.03, (name, cov)
        q2, U2 = o.calibrate_window(b.cal_pred, b.cal_truth, b.edges, 500, 2 * alpha, b.cal_pred, seen, b.u_max)
        assert np.all(q.astype(np.int64) >= q2) and np.all(U >= U2)


# ---------------------------------------------------------------------------
# Algorithm 1 on block counts (Sec. 3.3, Eq. (6)), with and without reservation
# ---------------------------------------------------------------------------

def py_place_static(B, Q, S, a_p, a_U, policy, rr_offset, reserve):
    """Brute force of Algorithm 1: explicit loops, Python integers."""
    B, Q = [int(x) for x in B], [int(x) for x in Q]
    D = len(B)
    out = []
    for a, (p, U) in enumerate(zip(a_p, a_U)):
        if U < 0:
            d = (rr_offset + a) % D
            out.append((d, -1, 2))
            if reserve:
                Q[d] += 1
            continue
        need = -(-(int(p) + int(U)) // S)
        feas = [d for d in range(D) if need <= B[d]]
        if policy == 0 and feas:
            d = min(feas, key=lambda x: (Q[x], x))
        else:
            d = min(range(D), key=lambda x: (-B[x], x))
        out.append((d, need, 1 if need <= B[d] else 0))
        if reserve:
            B[d] -= need
            Q[d] += 1
    return out, B, Q


def pin_static_golden(o):
    gd = golden("place_static_hand.json")
    r = gd["rsc"]
    bf, br, be = o.rsc_state(r["seg_off"], r["p"], r["g"], r["U"], r["capacity"], r["S"])
    assert bf.tolist() == r["b_free"] and br.tolist() == r["b_res"] and be.tolist() == r["b_eff"], (bf, br, be)
    pl = gd["place"]
    for mode, reserve in (("no_reserve", False), ("reserve", True)):
        ch, need, fl, ba, qa = o.place_static(pl["b_eff"], pl["queue_len"], pl["S"], pl["a_p"], pl["a_U"],
                                              reserve=reserve)
        assert ch.tolist() == pl[mode]["choice"], (mode, ch)
        assert need.tolist() == pl["b_need"] and fl.tolist() == pl["flags"], (mode, need, fl)
        assert ba.tolist() == pl[mode]["b_eff_after"] and qa.tolist() == pl[mode]["queue_after"], (mode, ba, qa)


def pin_static_bruteforce(o):
    rng = _rng(41)
    for trial in range(60):
        D = int(rng.integers(1, 7))
        A = int(rng.integers(0, 40))
        S = int(rng.choice([1, 2, 16, 33]))
        B = rng.integers(-20, 60, size=D)
        Q = rng.integers(0, 4, size=D)
        a_p = rng.integers(0, 300, size=A)
        a_U = rng.integers(-2, 300, size=A)
        for policy in (0, 1):
            for reserve in (False, True):
                ch, need, fl, ba, qa = o.place_static(B, Q, S, a_p, a_U, policy, 5, reserve)
                want, wB, wQ = py_place_static(B, Q, S, a_p, a_U, policy, 5, reserve)
                assert [(int(c), int(n), int(f)) for c, n, f in zip(ch, need, fl)] == want, (trial, policy, reserve)
                assert ba.tolist() == wB and qa.tolist() == wQ, (trial, policy, reserve)


def pin_static_water_filling(o):
    """With reservation and every decoder feasible for every arrival, the
    shortest-queue choice fills queues level by level: arrival i takes the
    i-th smallest slot (Q_d + m, d), m = 0, 1, ..."""
    rng = _rng(42)
    for trial in range(10):
        D = int(rng.integers(1, 9))
        A = int(rng.integers(1, 200))
        Q = rng.integers(0, 6, size=D)
        slots = sorted((int(Q[d]) + m, d) for d in range(D) for m in range(A))
        ch, _, fl, _, qa = o.place_static(np.full(D, 10**12), Q, 16, rng.integers(0, 100, size=A),
                                          rng.integers(0, 100, size=A), reserve=True)
        assert ch.tolist() == [d for _, d in slots[:A]], trial
        assert np.all(fl == 1) and qa.tolist() == (Q + np.bincount(ch, minlength=D)).tolist()


def pin_static_state_and_invariants(o):
    rng = _rng(43)
    seg, p, g, U, cap = _static_decoders(rng)
    for S in (1, 16):
        bf, br, be = o.rsc_state(seg, p, g, U, cap, S)
        for d in range(seg.size - 1):
            sl = slice(seg[d], seg[d + 1])
            held = sum(-(-(int(x) + int(y)) // S) for x, y in zip(p[sl], g[sl]))
            assert bf[d] == int(cap[d]) // S - held and br[d] >= 0 and be[d] == bf[d] - br[d]
            if S == 1:   # block size 1: B_eff = C - sum(p + max(g, U)), U < 0 counting as g
                assert be[d] == int(cap[d]) - sum(int(x) + max(int(y), int(u)) for x, y, u in zip(p[sl], g[sl], U[sl]))
    A = 300
    a_p = rng.integers(0, 2000, size=A)
    a_U = rng.integers(-1, 3000, size=A)
    Q = rng.integers(0, 5, size=seg.size - 1)
    ch, need, fl, ba, qa = o.place_static(be, Q, 16, a_p, a_U, reserve=True)
    bound = a_U >= 0
    for d in range(seg.size - 1):
        assert be[d] - ba[d] == need[bound & (ch == d)].sum()
        assert qa[d] - Q[d] == np.sum(ch == d)
    ch0, _, fl0, _, _ = o.place_static(be, Q, 16, a_p[:1], a_U[:1], reserve=False)
    assert ch0[0] == ch[0] and fl0[0] == fl[0]


def _static_decoders(rng, D=6):
    counts = rng.integers(0, 30, size=D)
    seg = np.zeros(D + 1, np.int64)
    seg[1:] = np.cumsum(counts)
    n = int(seg[-1])
    return (seg, rng.integers(0, 500, size=n), rng.integers(0, 400, size=n), rng.integers(-1, 600, size=n),
            rng.integers(0, 40000, size=D))


def pin_static_reduces_to_projection(o):
    """Block size 1, every resident with remaining length T and every arrival
    bound T: the projected peak test is exactly B_need <= B_eff, and the
    largest slack is the largest B_eff (Algorithm 1 is the projected rule's
    special case), so both oracles choose alike."""
    rng = _rng(44)
    for trial in range(10):
        D = int(rng.integers(1, 6))
        T = int(rng.integers(1, 200))
        counts = rng.integers(0, 8, size=D)
        seg = np.zeros(D + 1, np.int64)
        seg[1:] = np.cumsum(counts)
        n = int(seg[-1])
        p = rng.integers(0, 300, size=n)
        g = rng.integers(0, 100, size=n)
        U = g + T
        sums = np.add.reduceat(np.concatenate([p + U, [0]]), seg[:-1])[:D] * (counts > 0)
        cap = (sums + rng.integers(0, 800, size=D)).astype(np.int32)
        Q = rng.integers(0, 4, size=D)
        A = 50
        a_p = rng.integers(0, 400, size=A)
        a_U = np.where(rng.random(A) < 0.1, -1, T)
        pr = o.place(seg, p, g, U, cap, Q, a_p, a_U, want_pairs=False)
        _, _, be = o.rsc_state(seg, p, g, U, cap, 1)
        ch, _, fl, _, _ = o.place_static(be, Q, 1, a_p, a_U)
        assert np.array_equal(ch, pr.choice) and np.array_equal(fl, pr.flags), trial


# ---------------------------------------------------------------------------
# projected peak in blocks (Sec. 3.3, Eq. (6))
# ---------------------------------------------------------------------------

def py_peak_blocks(p, g, U, S, extra=()):
    """Brute force: every step t, every request's blocks ceil(tokens / S)."""
    R = [py_remaining(u, gg) for u, gg in zip(U, g)]
    T = max(list(R) + [int(u) for _, u in extra] + [0])
    best = 0
    for t in range(T + 1):
        occ = sum(-(-(int(pp) + int(gg) + t) // S) for pp, gg, r in zip(p, g, R) if t <= r)
        occ += sum(-(-(int(ap) + t) // S) for ap, au in extra if t <= au)
        best = max(best, occ)
    return best


def pin_blocks_golden(o):
    gd = golden("place_blocks_hand.json")
    OB = o.occupancy_blocks(gd["p"], gd["g"], gd["U"], gd["S"], gd["occupancy_T"])
    assert OB.tolist() == gd["occupancy"], OB
    r = o.place_blocks(gd["seg_off"], gd["p"], gd["g"], gd["U"], gd["capacity"], gd["queue_len"], gd["S"],
                       gd["a_p"], gd["a_U"])
    assert r.pair_peak.tolist() == gd["pair_peak"] and r.choice.tolist() == gd["choice"], (r.pair_peak, r.choice)
    assert r.chosen_peak.tolist() == gd["chosen_peak"] and r.chosen_overflow.tolist() == gd["chosen_overflow"]
    assert r.flags.tolist() == gd["flags"] and r.base_peak.tolist() == gd["base_peak"]


def pin_blocks_bruteforce(o):
    rng = _rng(51)
    for trial in range(40):
        S = int(rng.choice([1, 2, 3, 16, 37]))
        D = int(rng.integers(1, 4))
        seg, p, g, U = _tiny_decoders(rng, D, 6, 60, 80)
        A = int(rng.integers(1, 8))
        a_p = rng.integers(0, 80, size=A)
        a_U = rng.integers(-1, 70, size=A)
        cap = rng.integers(0, 60, size=D)
        r = o.place_blocks(seg, p, g, U, cap, np.zeros(D, np.int32), S, a_p, a_U)
        for d in range(D):
            sl = slice(seg[d], seg[d + 1])
            assert r.base_peak[d] == py_peak_blocks(p[sl], g[sl], U[sl], S), (trial, d)
            for a in range(A):
                want = -1 if a_U[a] < 0 else py_peak_blocks(p[sl], g[sl], U[sl], S, [(a_p[a], a_U[a])])
                assert r.pair_peak[d, a] == want, (trial, d, a, S)


def pin_blocks_reduce_to_tokens(o):
    """Block size 1 is the token rule, output for output."""
    rng = _rng(52)
    for trial in range(10):
        D = int(rng.integers(1, 6))
        seg, p, g, U = _tiny_decoders(rng, D, 20, 300, 400)
        A = 40
        a_p = rng.integers(0, 400, size=A)
        a_U = rng.integers(-1, 300, size=A)
        cap = rng.integers(0, 3000, size=D)
        Q = rng.integers(0, 3, size=D)
        for policy in (0, 1):
            rb = o.place_blocks(seg, p, g, U, cap, Q, 1, a_p, a_U, policy, 9)
            rt = o.place(seg, p, g, U, cap, Q, a_p, a_U, policy, 9)
            for f in ("choice", "chosen_peak", "chosen_overflow", "flags", "pair_peak", "base_peak"):
                assert np.array_equal(getattr(rb, f), getattr(rt, f)), (trial, policy, f)


def pin_blocks_invariants(o):
    """base <= peak <= base + ceil((p+U)/S); peak >= ceil((p+U)/S); peak in
    blocks >= ceil(peak in tokens / S); monotone in p and U."""
    rng = _rng(53)
    seg, p, g, U = _tiny_decoders(rng, 4, 30, 500, 600)
    A = 200
    a_p = rng.integers(0, 600, size=A)
    a_U = rng.integers(0, 500, size=A)
    cap = np.full(4, 10**6)
    Q = np.zeros(4, np.int32)
    for S in (4, 16):
        rb = o.place_blocks(seg, p, g, U, cap, Q, S, a_p, a_U)
        rt = o.place(seg, p, g, U, cap, Q, a_p, a_U)
        need = -(-(a_p.astype(np.int64) + a_U) // S)
        for d in range(4):
            pk = rb.pair_peak[d]
            assert np.all(pk >= rb.base_peak[d]) and np.all(pk <= rb.base_peak[d] + need) and np.all(pk >= need)
            assert np.all(pk >= -(-rt.pair_peak[d] // S))
        r2 = o.place_blocks(seg, p, g, U, cap, Q, S, a_p + 5, a_U)
        r3 = o.place_blocks(seg, p, g, U, cap, Q, S, a_p, a_U + 7)
        assert np.all(r2.pair_peak >= rb.pair_peak) and np.all(r3.pair_peak >= rb.pair_peak)


# ---------------------------------------------------------------------------
# occupancy and placement (Sec. 3.3, App. A, Algorithm 1)
# ---------------------------------------------------------------------------

def pin_place_golden(o):
    gd = golden("place_hand.json")
    seg = np.array(gd["seg_off"], np.int64)
    p, g, U = gd["prompt"], gd["generated"], gd["upper"]
    for d in range(seg.size - 1):
        lo, hi = seg[d], seg[d + 1]
        occ = o.occupancy(p[lo:hi], g[lo:hi], U[lo:hi], len(gd["occupancy"][d]) - 1)
        assert occ.tolist() == gd["occupancy"][d], (d, occ)
    assert o.project(seg, p, g, U).tolist() == gd["base_peak"]
    for policy, key in ((0, "mq"), (1, "mc")):
        r = o.place(seg, p, g, U, gd["capacity"], gd["queue_len"], gd["a_prompt"], gd["a_upper"],
                    policy=policy, rr_offset=gd["rr_offset"])
        assert r.pair_peak.tolist() == gd["pair_peak"], r.pair_peak
        assert r.base_peak.tolist() == gd["base_peak"]
        for f in ("choice", "chosen_peak", "chosen_overflow", "flags"):
            assert getattr(r, f).tolist() == gd[key][f], (key, f, getattr(r, f))


def pin_occupancy_bruteforce(o):
    rng = _rng(21)
    for trial in range(40):
        seg, p, g, U = _tiny_decoders(rng, 1, 9, 15, 30)
        T = max([py_remaining(u, gg) for u, gg in zip(U, g)] + [0]) + 3
        occ = o.occupancy(p, g, U, T)
        want = [py_occupancy(p, g, U, t) for t in range(T + 1)]
        assert occ.tolist() == want, trial
        assert occ[-1] == 0 and occ[0] == int(np.sum(p.astype(np.int64) + g))


def pin_place_bruteforce(o):
    """Every pair peak equals the step-by-step maximum (Python), every choice
    the rule of Algorithm 1 applied to those peaks."""
    rng = _rng(22)
    for trial in range(25):
        D = int(rng.integers(1, 5))
        seg, p, g, U = _tiny_decoders(rng, D, 6, 12, 20)
        A = int(rng.integers(1, 12))
        ap = rng.integers(0, 20, size=A).astype(np.int32)
        aU = rng.integers(-1, 15, size=A).astype(np.int32)
        cap = rng.integers(0, 150, size=D).astype(np.int32)
        Q = rng.integers(0, 3, size=D).astype(np.int32)
        rr = int(rng.integers(0, 7))
        for policy in (0, 1):
            r = o.place(seg, p, g, U, cap, Q, ap, aU, policy=policy, rr_offset=rr)
            for d in range(D):
                lo, hi = seg[d], seg[d + 1]
                assert r.base_peak[d] == py_peak(p[lo:hi], g[lo:hi], U[lo:hi])
            for a in range(A):
                if aU[a] < 0:
                    assert all(r.pair_peak[d, a] == -1 for d in range(D))
                    assert r.choice[a] == (rr + a) % D and r.flags[a] == 2
                    assert r.chosen_peak[a] == -1 and r.chosen_overflow[a] == 0
                    continue
                peaks = []
                for d in range(D):
                    lo, hi = seg[d], seg[d + 1]
                    pk = py_peak(p[lo:hi], g[lo:hi], U[lo:hi], [(int(ap[a]), int(aU[a]))])
                    assert r.pair_peak[d, a] == pk, (trial, d, a)
                    peaks.append(pk)
                slack = [int(cap[d]) - peaks[d] for d in range(D)]
                feas = [d for d in range(D) if slack[d] >= 0]
                if policy == 0 and feas:
                    want = min(feas, key=lambda d: (int(Q[d]), d))
                else:
                    want = max(range(D), key=lambda d: (slack[d], -d))
                assert r.choice[a] == want, (trial, policy, a)
                assert r.chosen_peak[a] == peaks[want]
                assert r.chosen_overflow[a] == max(0, -slack[want])
                assert r.flags[a] == (1 if slack[want] >= 0 else 0)


def pin_bruteforce_peak(o):
    """The oracle's term-by-term brute force (residents plus extra requests
    that start now, each summed at every step) against the Python one, and
    against its closed forms: no request gives 0, one extra request alone
    gives q + V (Sec. 3.3: a request's footprint grows to p + U)."""
    rng = _rng(23)
    assert o.bruteforce_peak([], [], []) == 0
    for q, V in ((0, 0), (5, 0), (3, 9), (100, 250)):
        assert o.bruteforce_peak([], [], [], [q], [V]) == q + V
    for trial in range(40):
        _, p, g, U = _tiny_decoders(rng, 1, 7, 14, 25)
        m = int(rng.integers(0, 4))
        q = rng.integers(0, 25, size=m).astype(np.int32)
        V = rng.integers(0, 16, size=m).astype(np.int32)
        want = py_peak(p, g, U, [(int(a), int(b)) for a, b in zip(q, V)])
        assert o.bruteforce_peak(p, g, U, q, V) == want, trial


def pin_place_closed_forms(o):
    # empty decoder: peak = p_a + U_a
    seg = np.array([0, 0], np.int64)
    z = np.zeros(0, np.int32)
    ap = np.array([0, 5, 7, 100], np.int32)
    aU = np.array([0, 3, 0, 250], np.int32)
    r = o.place(seg, z, z, z, [10**6], [0], ap, aU)
    assert r.pair_peak[0].tolist() == (ap + aU).tolist()
    # one resident (P = p+g, R): U_a >= R -> max(P+R + p_a+R, p_a+U_a); else max(P+R, P+U_a + p_a+U_a)
    rng = _rng(23)
    for _ in range(200):
        pr, gr, Ur = (int(x) for x in rng.integers(0, 50, size=3))
        pa, Ua = (int(x) for x in rng.integers(0, 60, size=2))
        P, R = pr + gr, max(Ur - gr, 0)
        want = max(P + R + pa + R, pa + Ua) if Ua >= R else max(P + R, P + Ua + pa + Ua)
        r = o.place(np.array([0, 1], np.int64), [pr], [gr], [Ur], [10**6], [0], [pa], [Ua])
        assert r.pair_peak[0, 0] == want, (pr, gr, Ur, pa, Ua)


def pin_place_invariants(o):
    b = workload.make("tiny")
    rng = _rng(24)
    seg = b.seg_off
    p, g = b.res_prompt, b.res_gen
    U = np.minimum(b.res_pred + rng.integers(0, 200, size=b.res_pred.size), b.u_max).astype(np.int32)
    ap = b.arr_prompt
    aU = np.minimum(b.arr_pred + 50, b.u_max).astype(np.int32)
    r = o.place(seg, p, g, U, b.capacity, b.queue_len, ap, aU)
    base = r.base_peak[:, None]
    pp = r.pair_peak
    assert np.all(pp >= base)                                # the arrival never lowers the peak
    assert np.all(pp >= (ap + aU)[None, :])                  # the arrival's own footprint
    assert np.all(pp <= base + (ap + aU)[None, :])
    static = np.array([np.sum(p[seg[d]:seg[d + 1]].astype(np.int64) + g[seg[d]:seg[d + 1]]
                              + np.maximum(U[seg[d]:seg[d + 1]].astype(np.int64) - g[seg[d]:seg[d + 1]], 0))
                       for d in range(seg.size - 1)])
    assert np.all(pp <= static[:, None] + (ap + aU)[None, :])   # static reservation bound
    r1 = o.place(seg, p, g, U, b.capacity, b.queue_len, ap + 1, aU)
    r2 = o.place(seg, p, g, U, b.capacity, b.queue_len, ap, aU + 1)
    assert np.all(r1.pair_peak >= pp) and np.all(r2.pair_peak >= pp)
    for d in range(seg.size - 1):
        lo, hi = seg[d], seg[d + 1]
        T = int(np.max(np.maximum(U[lo:hi].astype(np.int64) - g[lo:hi], 0)))
        occ = o.occupancy(p[lo:hi], g[lo:hi], U[lo:hi], T + 5)
        assert np.all(occ[T + 1:] == 0) and occ[T] > 0         # empty once every bound has run out
        assert r.base_peak[d] == occ.max()


def pin_place_reduces_to_algorithm1(o):
    """When every resident and the arrival have the same remaining length, the
    projected test is Algorithm 1's block test at S = 1: B_need = p_a + U_a,
    B_eff = C - sum(p_r + U_r); MQ among feasible, else argmax B_eff."""
    rng = _rng(25)
    for trial in range(40):
        D = int(rng.integers(1, 6))
        T = int(rng.integers(0, 30))
        counts = rng.integers(0, 5, size=D)
        seg = np.zeros(D + 1, np.int64)
        seg[1:] = np.cumsum(counts)
        n = int(seg[-1])
        p = rng.integers(0, 40, size=n).astype(np.int32)
        g = rng.integers(0, 20, size=n).astype(np.int32)
        U = (g + T).astype(np.int32)                          # R = T for everyone
        A = int(rng.integers(1, 8))
        ap = rng.integers(0, 40, size=A).astype(np.int32)
        aU = np.full(A, T, np.int32)
        cap = rng.integers(0, 400, size=D).astype(np.int32)
        Q = rng.integers(0, 4, size=D).astype(np.int32)
        r = o.place(seg, p, g, U, cap, Q, ap, aU)
        B_res = np.array([int(np.sum(p[seg[d]:seg[d + 1]].astype(np.int64) + U[seg[d]:seg[d + 1]]))
                          for d in range(D)])
        B_eff = cap.astype(np.int64) - B_res
        for a in range(A):
            need = int(ap[a]) + int(aU[a])                    # ceil((L_prom + L_up) / S), S = 1
            feas = [d for d in range(D) if need <= B_eff[d]]
            if feas:
                want = min(feas, key=lambda d: (int(Q[d]), d))
            else:
                want = max(range(D), key=lambda d: (int(B_eff[d]), -d))
            assert r.choice[a] == want, (trial, a)
            assert r.chosen_peak[a] == B_res[want] + need


def pin_round_robin_and_ties(o):
    seg = np.array([0, 1, 2, 3, 4], np.int64)
    one = np.array([5, 5, 5, 5], np.int32)
    r = o.place(seg, one, np.zeros(4, np.int32), one, [100] * 4, [2, 2, 2, 2],
                [1] * 6, [-1, 3, -5, 3, -1, -1], rr_offset=6)
    assert r.choice.tolist() == [(6 + 0) % 4, 0, (6 + 2) % 4, 0, (6 + 4) % 4, (6 + 5) % 4]
    r = o.place(seg, one, np.zeros(4, np.int32), one, [0] * 4, [2, 1, 1, 2], [1], [3], policy=0)
    assert r.choice.tolist() == [0] and r.flags.tolist() == [0]          # all infeasible, equal slack
    r = o.place(seg, one, np.zeros(4, np.int32), one, [100] * 4, [2, 1, 1, 2], [1], [3], policy=0)
    assert r.choice.tolist() == [1] and r.flags.tolist() == [1]          # min queue, lowest index
    r = o.place(seg, one, np.zeros(4, np.int32), one, [100, 101, 101, 100], [0] * 4, [1], [3], policy=1)
    assert r.choice.tolist() == [1]                                      # max slack, lowest index
    # every pair peak is 12 (5+t resident and 1+t arrival up to t=3); a peak equal to the
    # capacity is feasible (B_need <= B_eff in Algorithm 1, K+M <= C in Eq. (10))
    r = o.place(seg, one, np.zeros(4, np.int32), one, [11, 12, 13, 13], [0, 1, 5, 5], [1], [3], policy=0)
    assert r.pair_peak[:, 0].tolist() == [12] * 4
    assert r.choice.tolist() == [1] and r.flags.tolist() == [1] and r.chosen_overflow.tolist() == [0]


# ---------------------------------------------------------------------------
# local order and admission (Sec. 3.3 Eq. (7), App. A Eq. (10))
# ---------------------------------------------------------------------------

def pin_local_order_golden(o):
    gd = golden("local_order_hand.json")
    for key, wait in (("with_wait", gd["q_wait_ms"]), ("without_wait", None)):
        order, adm = o.local_order(gd["seg_off"], gd["prompt"], gd["generated"], gd["upper"],
                                   gd["capacity"], gd["q_off"], gd["q_prompt"], gd["q_upper"],
                                   wait, gd["max_wait_ms"], gd["u_max"])
        assert order.tolist() == gd[key]["order"], (key, order)
        assert adm.tolist() == gd[key]["admitted"], (key, adm)


def pin_local_order_bruteforce(o):
    rng = _rng(31)
    for trial in range(25):
        D = int(rng.integers(1, 4))
        seg, p, g, U = _tiny_decoders(rng, D, 4, 10, 15)
        qc = rng.integers(0, 7, size=D)
        qoff = np.zeros(D + 1, np.int64)
        qoff[1:] = np.cumsum(qc)
        nq = int(qoff[-1])
        qp = rng.integers(0, 12, size=nq).astype(np.int32)
        qU = rng.integers(-1, 9, size=nq).astype(np.int32)
        qw = rng.integers(0, 2000, size=nq).astype(np.int32)
        u_max, max_wait = 9, 1000
        cap = rng.integers(0, 160, size=D).astype(np.int32)
        for wait in (qw, None):
            order, adm = o.local_order(seg, p, g, U, cap, qoff, qp, qU, wait, max_wait, u_max)
            for d in range(D):
                lo, hi = int(qoff[d]), int(qoff[d + 1])
                Ue = [u_max if int(x) < 0 else int(x) for x in qU[lo:hi]]
                prom = [wait is not None and int(wait[lo + i]) >= max_wait for i in range(hi - lo)]
                want = sorted(range(hi - lo), key=lambda i: (0, i) if prom[i] else (1, Ue[i]))
                assert order[lo:hi].tolist() == want, (trial, d)
                rp, rg, rU = p[seg[d]:seg[d + 1]], g[seg[d]:seg[d + 1]], U[seg[d]:seg[d + 1]]
                peaks = [py_peak(rp, rg, rU, [(int(qp[lo + i]), Ue[i]) for i in want[:k]])
                         for k in range(hi - lo + 1)]
                assert all(x <= y for x, y in zip(peaks, peaks[1:]))   # adding never lowers the peak
                k_ok = [k for k in range(hi - lo + 1) if peaks[k] <= cap[d]]
                assert adm[d] == (max(k_ok) if k_ok else 0), (trial, d, peaks, cap[d])


# ---------------------------------------------------------------------------
# placement with sequential commit (Sec. 3.3: each dispatch reserves its
# demand before the next request is placed; Algorithm 1)
# ---------------------------------------------------------------------------

def py_place_commit(seg, p, g, U, cap, Q, ap, aU, policy, rr):
    """Arrivals in order; every pair peak by brute force over the residents
    plus the arrivals already committed to the decoder plus the arrival."""
    D = len(seg) - 1
    Q = [int(x) for x in Q]
    committed = [[] for _ in range(D)]
    out = []
    for a in range(len(ap)):
        if aU[a] < 0:
            d = (rr + a) % D
            Q[d] += 1
            out.append((d, -1, 0, 2))
            continue
        peaks = []
        for d in range(D):
            lo, hi = seg[d], seg[d + 1]
            peaks.append(py_peak(p[lo:hi], g[lo:hi], U[lo:hi], committed[d] + [(int(ap[a]), int(aU[a]))]))
        slack = [int(cap[d]) - peaks[d] for d in range(D)]
        feas = [d for d in range(D) if slack[d] >= 0]
        if policy == 0 and feas:
            d = min(feas, key=lambda k: (Q[k], k))
        else:
            d = max(range(D), key=lambda k: (slack[k], -k))
        out.append((d, peaks[d], max(0, -slack[d]), 1 if slack[d] >= 0 else 0))
        committed[d].append((int(ap[a]), int(aU[a])))
        Q[d] += 1
    return out, Q


def pin_commit_bruteforce(o):
    rng = _rng(31)
    for trial in range(30):
        D = int(rng.integers(1, 5))
        seg, p, g, U = _tiny_decoders(rng, D, 5, 10, 15)
        A = int(rng.integers(1, 10))
        ap = rng.integers(0, 15, size=A).astype(np.int32)
        aU = rng.integers(-1, 12, size=A).astype(np.int32)
        cap = rng.integers(0, 160, size=D).astype(np.int32)
        Q = rng.integers(0, 3, size=D).astype(np.int32)
        rr = int(rng.integers(0, 5))
        for policy in (0, 1):
            r, q_after = o.place_commit(seg, p, g, U, cap, Q, ap, aU, policy=policy, rr_offset=rr)
            want, want_q = py_place_commit(seg, p, g, U, cap, Q, ap, aU, policy, rr)
            got = list(zip(r.choice.tolist(), r.chosen_peak.tolist(), r.chosen_overflow.tolist(), r.flags.tolist()))
            assert got == want, (trial, policy, got, want)
            assert q_after.tolist() == want_q, (trial, policy)


def pin_commit_reduces_to_static_reserve(o):
    """Every resident and every arrival with the same remaining length T: the
    projected peak is the sum of the demands plus the arrival's, so sequential
    commit is Algorithm 1 with reservation at block size 1 (B_need = p + T <=
    B_eff, B_eff reduced by each dispatch's need, shortest queue, else largest
    B_eff)."""
    rng = _rng(32)
    for trial in range(30):
        D = int(rng.integers(1, 6))
        T = int(rng.integers(0, 9))
        counts = rng.integers(0, 4, size=D)
        seg = np.zeros(D + 1, np.int64)
        seg[1:] = np.cumsum(counts)
        n = int(seg[-1])
        p = rng.integers(0, 20, size=n).astype(np.int32)
        g = rng.integers(0, 6, size=n).astype(np.int32)
        U = (g + T).astype(np.int32)
        A = int(rng.integers(1, 12))
        ap = rng.integers(0, 20, size=A).astype(np.int32)
        aU = np.where(rng.random(A) < 0.15, -1, T).astype(np.int32)
        cap = rng.integers(0, 200, size=D).astype(np.int32)
        Q = rng.integers(0, 3, size=D).astype(np.int32)
        _, _, be = o.rsc_state(seg, p, g, U, cap, 1)
        for policy in (0, 1):
            r, q_after = o.place_commit(seg, p, g, U, cap, Q, ap, aU, policy=policy, rr_offset=3)
            ch, need, fl, _, q_static = o.place_static(be, Q, 1, ap, aU, policy=policy, rr_offset=3, reserve=True)
            assert r.choice.tolist() == ch.tolist(), (trial, policy)
            assert r.flags.tolist() == fl.tolist(), (trial, policy)
            assert q_after.tolist() == q_static.tolist()


def pin_commit_single_decoder_and_first_arrival(o):
    """With one decoder every arrival lands on it, and its chosen peak is the
    brute-force peak of the residents plus every arrival so far; the first
    arrival of any batch sees the snapshot alone (the independent placement)."""
    rng = _rng(33)
    for trial in range(20):
        seg, p, g, U = _tiny_decoders(rng, 1, 6, 10, 15)
        A = int(rng.integers(1, 8))
        ap = rng.integers(0, 15, size=A).astype(np.int32)
        aU = rng.integers(0, 12, size=A).astype(np.int32)
        r, q_after = o.place_commit(seg, p, g, U, [10**6], [0], ap, aU)
        for a in range(A):
            assert r.choice[a] == 0
            assert r.chosen_peak[a] == o.bruteforce_peak(p, g, U, ap[:a + 1], aU[:a + 1]), (trial, a)
        assert q_after.tolist() == [A]
        D = int(rng.integers(1, 5))
        seg, p, g, U = _tiny_decoders(rng, D, 5, 10, 15)
        cap = rng.integers(0, 150, size=D).astype(np.int32)
        Q = rng.integers(0, 3, size=D).astype(np.int32)
        ind = o.place(seg, p, g, U, cap, Q, ap[:1], aU[:1])
        r, _ = o.place_commit(seg, p, g, U, cap, Q, ap, aU)
        assert r.choice[0] == ind.choice[0] and r.chosen_peak[0] == ind.chosen_peak[0]
        # committing never lowers a later pair's peak below its independent value
        ind = o.place(seg, p, g, U, cap, Q, ap, aU)
        assert np.all(r.chosen_peak >= ind.pair_peak[r.choice, np.arange(A)])


# ---------------------------------------------------------------------------
# staged reservation (appendix on the global algorithm: the prompt part of a
# dispatch's reservation is released once the prompt KV reaches the decoder)
# ---------------------------------------------------------------------------

def pin_staged_reservation(o):
    """A request still in transfer holds nothing and reserves its whole budget
    ceil((p+U)/S) (its prompt's blocks without a bound); once its prompt has
    arrived (g = 0) its prompt blocks are held and only the rest stays
    reserved, so B_eff does not move at the transfer; B_free does."""
    rng = _rng(34)
    for trial in range(30):
        D = int(rng.integers(1, 4))
        seg, p, g, U = _tiny_decoders(rng, D, 6, 40, 60)
        U = np.where(rng.random(U.size) < 0.2, -1, U).astype(np.int32)
        cap = rng.integers(0, 400, size=D).astype(np.int32)
        S = int(rng.choice([1, 2, 3, 16]))
        fl = (rng.random(U.size) < 0.5).astype(np.uint8)
        bf, br, be = o.rsc_state(seg, p, g, U, cap, S, in_flight=fl)
        for d in range(D):
            held = res = 0
            for r in range(seg[d], seg[d + 1]):
                if fl[r]:
                    res += -(-(int(p[r]) + max(int(U[r]), 0)) // S)
                else:
                    now = -(-(int(p[r]) + int(g[r])) // S)
                    held += now
                    if U[r] >= 0:
                        res += max(-(-(int(p[r]) + int(U[r])) // S) - now, 0)
            assert bf[d] == int(cap[d]) // S - held and br[d] == res and be[d] == bf[d] - br[d], (trial, d)
        # the transfer: every in-flight request lands with g = 0; B_eff unchanged where U >= 0
        g0 = np.where(fl == 1, 0, g).astype(np.int32)
        bf2, br2, be2 = o.rsc_state(seg, p, g0, U, cap, S)
        if np.all(U[fl == 1] >= 0):
            assert be2.tolist() == be.tolist(), trial
        # in-flight requests are exactly the dispatches of Algorithm 1 with reservation
    seg = np.array([0, 2], np.int64)
    bf, br, be = o.rsc_state(seg, [5, 7], [0, 0], [10, 3], [100], 4, in_flight=[1, 1])
    assert (bf[0], br[0], be[0]) == (25, 4 + 3, 25 - 7)


# ---------------------------------------------------------------------------
# App. A pressure simulation
# ---------------------------------------------------------------------------

def py_simulate(N, C, theta_ppm, arr, prompt, output, bound, policy):
    """The same millisecond-by-millisecond definition, written with Python
    deques: release, FIFO admission, arrivals, record, one token per decoder."""
    from collections import deque
    n = len(arr)
    M = [int(prompt[i]) + int(output[i]) for i in range(n)]
    need = [int(prompt[i]) + int(bound[i]) for i in range(n)]
    ready = [deque() for _ in range(N)]
    fifo = [deque() for _ in range(N)]
    K = [0] * N
    R = [0] * N
    left = [int(x) for x in output]
    rel = [None] * N
    fin = [0] * n
    routed = [0] * n
    hp_t, hp_m, hp_c, mq, qa, run = ([0] * N for _ in range(6))
    t, nxt, done = int(arr[0]), 0, 0
    last = t
    while True:
        for d in range(N):
            if rel[d] is not None:
                K[d] -= M[rel[d]]
                fin[rel[d]] = t
                last = t
                rel[d] = None
                done += 1
        if done == n:
            break
        if all(not ready[d] and not fifo[d] for d in range(N)) and nxt < n and arr[nxt] > t:
            run = [0] * N
            t = int(arr[nxt])
        for d in range(N):
            while fifo[d] and K[d] + M[fifo[d][0]] <= C:
                i = fifo[d].popleft()
                if policy == 1 and bound[i] >= 0:
                    R[d] -= need[i]
                K[d] += M[i]
                ready[d].append(i)
        while nxt < n and arr[nxt] == t:
            i = nxt
            nxt += 1
            if policy == 1 and bound[i] >= 0:
                beff = [C - K[k] - R[k] for k in range(N)]
                feas = [k for k in range(N) if need[i] <= beff[k]]
                d = min(feas, key=lambda k: (len(fifo[k]), k)) if feas else max(range(N), key=lambda k: (beff[k], -k))
            else:
                d = i % N
            routed[i] = d
            if not fifo[d] and K[d] + M[i] <= C:
                K[d] += M[i]
                ready[d].append(i)
            else:
                fifo[d].append(i)
                if policy == 1 and bound[i] >= 0:
                    R[d] += need[i]
        for d in range(N):
            if K[d] * 10**6 >= theta_ppm * C:
                hp_c[d] += run[d] == 0
                run[d] += 1
                hp_t[d] += 1
                hp_m[d] = max(hp_m[d], run[d])
            else:
                run[d] = 0
            qa[d] += len(fifo[d])
            mq[d] = max(mq[d], len(fifo[d]))
        for d in range(N):
            if ready[d]:
                i = ready[d].popleft()
                left[i] -= 1
                if left[i] == 0:
                    rel[d] = i
                else:
                    ready[d].append(i)
        t += 1
    return dict(finish_ms=fin, routed=routed, hp_time=hp_t, hp_max=hp_m, hp_count=hp_c, max_queue=mq,
                queue_area=qa, span=[int(arr[0]), last])


SIM_FIELDS = ("finish_ms", "routed", "hp_time", "hp_max", "hp_count", "max_queue", "queue_area", "span")


def pin_simulate_golden(o):
    for c in golden("simulate_hand.json")["cases"]:
        r = o.simulate(c["N"], c["C"], c["theta_ppm"], c["arrival_ms"], c["prompt"], c["output"], c["bound"],
                       c["policy"])
        for f in SIM_FIELDS:
            assert getattr(r, f).tolist() == c[f], (c["name"], f, getattr(r, f))


def _sim_case(rng, n_max=14):
    N = int(rng.integers(1, 4))
    C = int(rng.choice([16, 20, 25, 32, 40]))   # divisors of 10^6: K / C can equal theta exactly
    n = int(rng.integers(1, n_max))
    arr = np.cumsum(rng.integers(0, 4, size=n)).astype(np.int64) + int(rng.integers(0, 3))
    prompt = rng.integers(0, 8, size=n).astype(np.int32)
    output = rng.integers(1, 9, size=n).astype(np.int32)
    output = np.minimum(output, C - prompt).astype(np.int32)
    bound = np.where(rng.random(n) < 0.2, -1, output + rng.integers(-2, 4, size=n)).astype(np.int32)
    bound = np.where(bound < -1, 0, bound).astype(np.int32)
    theta = int(rng.integers(1, 10**6 + 1)) if rng.random() < 0.3 else 10**6 * int(rng.integers(1, C + 1)) // C
    return N, C, theta, arr, prompt, output, bound


def pin_simulate_bruteforce(o):
    rng = _rng(41)
    for trial in range(60):
        N, C, theta, arr, prompt, output, bound = _sim_case(rng)
        for policy in (0, 1):
            r = o.simulate(N, C, theta, arr, prompt, output, bound, policy)
            want = py_simulate(N, C, theta, arr, prompt, output, bound, policy)
            for f in SIM_FIELDS:
                assert getattr(r, f).tolist() == want[f], (trial, policy, f)


def pin_simulate_closed_forms(o):
    """One request alone completes after its output length; two requests
    admitted together share the decoder one token at a time (the first of x
    tokens completes at 2x - 1 when x <= y, the second at 2y when y < x, the
    last at x + y); without memory pressure each decoder is work conserving;
    Algorithm 1 without any bound is round robin."""
    r = o.simulate(1, 100, 500000, [7], [30], [25])
    assert r.finish_ms.tolist() == [32] and r.hp_time.tolist() == [25] and r.hp_count.tolist() == [1]
    for x in range(1, 6):
        for y in range(1, 6):
            r = o.simulate(1, 1000, 10**6, [0, 0], [0, 0], [x, y])
            want = [2 * x - 1, x + y] if x <= y else [x + y, 2 * y]
            assert r.finish_ms.tolist() == want, (x, y)
    rng = _rng(42)
    for trial in range(20):
        N = int(rng.integers(1, 4))
        n = int(rng.integers(1, 12))
        out = rng.integers(1, 9, size=n).astype(np.int32)
        pr = rng.integers(0, 5, size=n).astype(np.int32)
        r = o.simulate(N, 10**6, 10**6, np.zeros(n, np.int64), pr, out)
        assert r.routed.tolist() == [i % N for i in range(n)]
        for d in range(N):
            mine = [i for i in range(n) if i % N == d]
            if mine:
                assert max(r.finish_ms[mine]) == int(out[mine].sum()), (trial, d)
        N, C, theta, arr, prompt, output, bound = _sim_case(rng)
        r0 = o.simulate(N, C, theta, arr, prompt, output, None, 0)
        r1 = o.simulate(N, C, theta, arr, prompt, output, None, 1)
        for f in SIM_FIELDS:
            assert getattr(r0, f).tolist() == getattr(r1, f).tolist(), (trial, f)
        assert np.all(r0.finish_ms >= arr + output)
        assert np.all(r0.hp_max <= r0.hp_time) and np.all(r0.hp_count <= r0.hp_time)
        assert np.all(r0.hp_time <= r0.span[1] - r0.span[0]) and r0.span[1] == r0.finish_ms.max()


ALL_PINS = [
    pin_calibrate_golden, pin_rank_is_ceiling, pin_quantile_order_statistic,
    pin_quantile_special_cases, pin_quantile_monotone_in_alpha, pin_coverage,
    pin_window_golden, pin_window_bruteforce, pin_window_closed_forms, pin_window_reduces_to_fixed_set,
    pin_window_coverage,
    pin_static_golden, pin_static_bruteforce, pin_static_water_filling, pin_static_state_and_invariants,
    pin_static_reduces_to_projection,
    pin_blocks_golden, pin_blocks_bruteforce, pin_blocks_reduce_to_tokens, pin_blocks_invariants,
    pin_place_golden, pin_occupancy_bruteforce, pin_bruteforce_peak, pin_place_bruteforce, pin_place_closed_forms,
    pin_place_invariants, pin_place_reduces_to_algorithm1, pin_round_robin_and_ties,
    pin_local_order_golden, pin_local_order_bruteforce,
    pin_commit_bruteforce, pin_commit_reduces_to_static_reserve, pin_commit_single_decoder_and_first_arrival,
    pin_staged_reservation,
    pin_simulate_golden, pin_simulate_bruteforce, pin_simulate_closed_forms,
]
