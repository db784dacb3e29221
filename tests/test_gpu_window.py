"""Sliding-window calibration on the GPU (maps_calibrate_window) against the
CPU oracle, bit for bit: each request calibrated on the most recent
completions of its bucket that it had seen (Sec. 3.2; Sec. 4 uses a window of
the 500 most recent).  Ragged logs around the 4,096-entry chunks and the
1,536-position select runs, windows from 1 to the maximum, empty logs and
buckets, the seeded workloads (sampled requests at the two largest), and the
device error bits."""
import numpy as np
import pytest

import oracle
import workload
from tests.gpu_common import assert_same, say

pytestmark = pytest.mark.gpu
Q_INF = 2**31 - 1


@pytest.fixture(scope="module")
def orc():
    return oracle.Oracle()


def _cuda(x, dtype=np.int32):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=dtype)).cuda()


def _gpu(pred, truth, edges, window, alpha, ap, seen, u_max):
    import torch

    import paper_2609_15359_amd as maps
    q, U, err = maps.calibrate_window(_cuda(pred), _cuda(truth), _cuda(edges), window, alpha, _cuda(ap),
                                      _cuda(seen, np.int64), u_max)
    torch.cuda.synchronize()
    return q.cpu().numpy(), U.cpu().numpy(), int(err.item()) & 0xFFFFFFFF


def test_hand_worked_example():
    from tests.oracle_pins import golden
    gd = golden("calibrate_window_hand.json")
    r = gd["requests"]
    for case in gd["cases"]:
        q, U, err = _gpu(gd["pred"], gd["truth"], gd["edges"], case["window"], case["alpha_ppm"], r["pred"],
                         r["seen"], gd["u_max"])
        assert err == 0
        assert q.tolist() == [Q_INF if v == "inf" else v for v in case["q"]], case
        assert U.tolist() == case["U"], case


# (n, nb, window): chunk and run boundaries, single entries, one bucket, windows 1 .. max
RAGGED = [(0, 3, 500), (1, 1, 1), (5, 2, 3), (4095, 7, 500), (4096, 7, 500), (4097, 40, 1600), (9000, 2, 1),
          (20000, 7, 4096), (30001, 64, 500), (70000, 5, 2000), (50000, 1024, 500)]


@pytest.mark.parametrize("n,nb,window", RAGGED, ids=[f"n{r[0]}-nb{r[1]}-w{r[2]}" for r in RAGGED])
def test_ragged_logs(orc, n, nb, window):
    rng = np.random.default_rng(7 * n + nb + window)
    pred = rng.integers(0, 3000, size=n).astype(np.int32)
    truth = (pred + rng.integers(-800, 2500, size=n)).clip(0).astype(np.int32)
    edges = np.sort(rng.integers(0, 3000, size=nb - 1)).astype(np.int32)
    if nb > 3:
        edges[1] = edges[2]          # a duplicated edge: an empty bucket
    m = 20000
    ap = rng.integers(-3, 3500, size=m).astype(np.int32)
    seen = rng.integers(0, n + 1, size=m).astype(np.int64)
    seen[:50] = n
    seen[50:100] = 0
    for alpha in (100000, 50000):
        say(f"[window] n={n} nb={nb} W={window} alpha={alpha}")
        qo, Uo = orc.calibrate_window(pred, truth, edges, window, alpha, ap, seen, 4000)
        q, U, err = _gpu(pred, truth, edges, window, alpha, ap, seen, 4000)
        assert err == 0
        assert_same("q", q, qo)
        assert_same("U", U, Uo)


def test_every_position_of_one_bucket(orc):
    """One bucket, every seen count from 0 to n: all select runs and the
    partial windows at the start of the log."""
    rng = np.random.default_rng(3)
    n = 5000
    pred = rng.integers(0, 100, size=n).astype(np.int32)
    truth = rng.integers(0, 100000, size=n).astype(np.int32)   # 17-bit scores
    seen = np.arange(n + 1, dtype=np.int64)
    ap = np.full(n + 1, 50, np.int32)
    for window in (1, 2, 500, 1537):
        qo, Uo = orc.calibrate_window(pred, truth, [], window, 100000, ap, seen, 2**30)
        q, U, err = _gpu(pred, truth, [], window, 100000, ap, seen, 2**30)
        assert err == 0
        assert_same(f"q (window {window})", q, qo)
        assert_same(f"U (window {window})", U, Uo)


def test_fixed_set_special_case(orc):
    """A window as long as the log and every request after the last
    completion: the fixed-set bound of maps_calibrate."""
    import paper_2609_15359_amd as maps
    b = workload.make("small")
    n = b.cal_pred.size
    ap = b.apply_pred()
    seen = np.full(ap.size, n, np.int64)
    q, U, err = _gpu(b.cal_pred, b.cal_truth, b.edges, maps.MAX_WINDOW, b.alpha_ppm, ap, seen, b.u_max)
    assert err == 0
    # each bucket of small holds at most 4,096 completions, so the window covers it
    assert np.bincount(np.searchsorted(b.edges, b.cal_pred, side="right")).max() <= maps.MAX_WINDOW
    qb, _ = orc.calibrate(b.cal_pred, b.cal_truth, b.edges, b.alpha_ppm)
    assert_same("U", U, orc.apply_bounds(ap, b.edges, qb, b.u_max))


@pytest.mark.parametrize("name", ["tiny", "small", "medium", "large", "xlarge"])
def test_workload_window_500(orc, name):
    """The seeded workloads: every bounded request of the step (residents at
    earlier points of the log, arrivals and queued requests after all of it),
    window 500 as in Sec. 4.  Full comparison up to medium; at large and
    xlarge the oracle computes 50,000 sampled requests one by one, and every
    request's bound is checked against its quantile."""
    b = workload.make(name)
    ap = b.apply_pred()
    seen = workload.window_seen(b)
    say(f"[window] {name}: log {b.cal_pred.size}, {b.edges.size + 1} buckets, {ap.size} requests")
    q, U, err = _gpu(b.cal_pred, b.cal_truth, b.edges, 500, b.alpha_ppm, ap, seen, b.u_max)
    assert err == 0
    if ap.size <= 200000:
        idx = np.arange(ap.size)
    else:
        rng = np.random.default_rng(11)
        idx = np.unique(np.concatenate([rng.choice(ap.size, 50000, replace=False), np.arange(200),
                                        np.arange(ap.size - 200, ap.size)]))
    qo, Uo = orc.calibrate_window(b.cal_pred, b.cal_truth, b.edges, 500, b.alpha_ppm, ap[idx], seen[idx], b.u_max)
    assert_same("q", q[idx], qo)
    assert_same("U", U[idx], Uo)
    ok = ap >= 0
    fin = ok & (q != Q_INF)
    assert np.all(U[~ok] == -1) and np.all(q[~ok] == -1)
    assert np.all(U[ok & (q == Q_INF)] == b.u_max)
    assert np.array_equal(U[fin], np.minimum(ap[fin].astype(np.int64) + q[fin], b.u_max))


def test_error_bits():
    import paper_2609_15359_amd as maps
    pred = np.array([5, 6, 7], np.int32)
    truth = np.array([9, 9, 9], np.int32)
    _, _, err = _gpu(pred, truth, [], 10, 100000, [1, 2], [0, 4], 100)
    assert err & 512, maps.error_names(err)
    _, _, err = _gpu(pred, truth, [], 10, 100000, [1, 2], [-1, 0], 100)
    assert err & 512
    _, _, err = _gpu(np.array([5, -6, 7], np.int32), truth, [], 10, 100000, [1], [3], 100)
    assert err & 1
    _, _, err = _gpu(pred, truth, [9, 3], 10, 100000, [1], [3], 100)
    assert err & 2
    # no prediction: no bucket, no seen check
    q, U, err = _gpu(pred, truth, [], 10, 100000, [-1], [99], 100)
    assert err == 0 and q.tolist() == [-1] and U.tolist() == [-1]


# ---------------------------------------------------------------------------
# incremental window state (maps_window_reset / append / bounds)
# ---------------------------------------------------------------------------

def _bucket_reps(edges):
    """One prediction per non-empty bucket range: 0 for bucket 0 (when the
    first edge is above 0), each distinct edge for the bucket it opens."""
    reps, buckets = [], []
    e = list(int(x) for x in edges)
    if not e or e[0] > 0:
        reps.append(0)
        buckets.append(0)
    for j, x in enumerate(e):
        if j + 1 < len(e) and e[j + 1] == x:
            continue           # duplicated edge: the bucket it opens is empty
        reps.append(x)
        buckets.append(j + 1)
    return np.array(reps, np.int32), buckets


def _check_state(orc, st, pred, truth, edges, window, alpha, ap, u_max, tag):
    import torch
    n = len(pred)
    q, U = st.bounds(alpha, _cuda(ap), u_max)
    torch.cuda.synchronize()
    assert int(st.dev_err.item()) == 0, tag
    _, want_U = orc.calibrate_window(pred, truth, edges, window, alpha, ap, np.full(len(ap), n), u_max)
    assert_same(f"{tag} U", U.cpu().numpy(), want_U)
    reps, buckets = _bucket_reps(edges)
    want_q, _ = orc.calibrate_window(pred, truth, edges, window, alpha, reps, np.full(len(reps), n), u_max)
    assert_same(f"{tag} q", q.cpu().numpy()[buckets], want_q)


@pytest.mark.parametrize("nb,window", [(1, 1), (3, 7), (8, 500), (64, 500), (200, 4096)])
def test_incremental_window(orc, nb, window):
    """Completions appended in batches of 0 to 3 windows (chunk edges, a
    bucket wrapping its ring within one batch and across batches); after each
    append every bucket's quantile and a batch of bounds equal the window
    calibration of the whole log so far."""
    import paper_2609_15359_amd as maps
    rng = np.random.default_rng(nb * 31 + window)
    total = 40000 if window < 4096 else 60000
    pred = rng.integers(0, 5000, size=total).astype(np.int32)
    truth = (pred + rng.integers(-900, 3000, size=total)).clip(0).astype(np.int32)
    edges = np.sort(rng.integers(0, 5000, size=nb - 1)).astype(np.int32)
    if nb > 3:
        edges[1] = edges[2]   # a duplicated edge: an empty bucket
    ap = np.concatenate([rng.integers(-1, 6000, size=3000 if window <= 500 else 300), [-1, 0]]).astype(np.int32)
    st = maps.WindowState(_cuda(edges), window)
    _check_state(orc, st, pred[:0], truth[:0], edges, window, 100000, ap, 8000, "empty log")
    n = 0
    sizes = [0, 1, 1023, 1024, 1025, window - 1, window, window + 1, 3 * window, 4096, 5000]
    for step, k in enumerate(sizes + list(rng.integers(0, 3 * window + 2, size=8))):
        k = int(min(k, total - n))
        st.append(_cuda(pred[n:n + k]), _cuda(truth[n:n + k]))
        n += k
        for alpha in (50000, 100000):
            _check_state(orc, st, pred[:n], truth[:n], edges, window, alpha, ap, 8000, f"nb={nb} w={window} n={n}")
    say(f"[window-state] nb={nb} window={window}: {n} completions appended in {step + 1} batches")


@pytest.mark.parametrize("top", [0, 255, 65535, 2**24 - 1, 2**24, 2**31 - 1])
def test_incremental_window_score_range(orc, top):
    """Scores from 0 up to `top` (all zero; the largest in the lowest, second,
    third and top byte): the selection starts at the highest byte the largest
    score uses, and every start gives the oracle's quantiles."""
    import paper_2609_15359_amd as maps
    rng = np.random.default_rng(top % 1000003)
    n, window = 6000, 37
    pred = rng.integers(0, 5000, size=n).astype(np.int32)
    score = rng.integers(0, top + 1, size=n, dtype=np.int64)
    score[rng.integers(0, n, size=50)] = top   # the largest score is present
    truth = np.minimum(pred.astype(np.int64) + score, 2**31 - 1).astype(np.int32)
    edges = np.array([1000, 3000], np.int32)
    ap = np.concatenate([rng.integers(-1, 6000, size=500), [-1, 0]]).astype(np.int32)
    st = maps.WindowState(_cuda(edges), window)
    done = 0
    for k in (1000, 37, 4963):
        st.append(_cuda(pred[done:done + k]), _cuda(truth[done:done + k]))
        done += k
        for alpha in (50000, 500000):
            _check_state(orc, st, pred[:done], truth[:done], edges, window, alpha, ap, 2**31 - 1,
                         f"top={top} n={done}")


def test_incremental_window_chunk_prefix_paths(orc):
    """Appends of exactly 1,024 chunks of 1,024 completions (the largest whose
    per-chunk prefix stays in LDS), of one completion more (the prefix written
    over the workspace column) and a small one after them."""
    import paper_2609_15359_amd as maps
    rng = np.random.default_rng(1025)
    sizes = [1024 * 1024, 1024 * 1024 + 1, 3000]
    total = sum(sizes)
    pred = rng.integers(0, 5000, size=total).astype(np.int32)
    truth = (pred + rng.integers(-900, 3000, size=total)).clip(0).astype(np.int32)
    edges = np.array([300, 800, 1500, 2500, 2600, 4000, 4900], np.int32)
    ap = np.concatenate([rng.integers(-1, 6000, size=300), [-1, 0]]).astype(np.int32)
    st = maps.WindowState(_cuda(edges), 500)
    n = 0
    for k in sizes:
        st.append(_cuda(pred[n:n + k]), _cuda(truth[n:n + k]))
        n += k
        _check_state(orc, st, pred[:n], truth[:n], edges, 500, 100000, ap, 8000, f"chunks n={n}")


def test_incremental_window_bounds_past_one_pass(orc):
    """A bound call on more requests than one pass of the bound kernel's grid
    covers (2,048 workgroups x 256 requests, three passes and a ragged tail):
    the quantiles against the oracle's window calibration and every bound
    against the oracle's Eq. (4) from those quantiles."""
    import torch

    import paper_2609_15359_amd as maps
    rng = np.random.default_rng(8192)
    n, window = 20000, 500
    pred = rng.integers(0, 5000, size=n).astype(np.int32)
    truth = (pred + rng.integers(-900, 3000, size=n)).clip(0).astype(np.int32)
    edges = np.array([700, 1400, 2900, 4100], np.int32)
    st = maps.WindowState(_cuda(edges), window)
    st.append(_cuda(pred), _cuda(truth))
    m = 3 * 2048 * 256 + 777
    ap = rng.integers(-2, 7000, size=m).astype(np.int32)
    q, U = st.bounds(50000, _cuda(ap), 6000)
    torch.cuda.synchronize()
    assert int(st.dev_err.item()) == 0
    reps, buckets = _bucket_reps(edges)
    want_q, _ = orc.calibrate_window(pred, truth, edges, window, 50000, reps, np.full(len(reps), n), 6000)
    got_q = q.cpu().numpy()
    assert_same("q", got_q[buckets], want_q)
    assert_same("U", U.cpu().numpy(), orc.apply_bounds(ap, edges, got_q, 6000))


def test_incremental_window_large(orc):
    """The large workload's 1,000,000 calibration pairs as the completion log,
    appended in 16 batches, window 500, 64 buckets; the bounds of every
    resident, arrival and queued request after the last batch (the state
    calibration of the batch, against the oracle with every request having
    seen the whole log) and sampled requests after each batch."""
    import paper_2609_15359_amd as maps
    b = workload.make("large")
    ap = b.apply_pred()
    st = maps.WindowState(_cuda(b.edges), 500)
    n_all = b.cal_pred.size
    cuts = np.linspace(0, n_all, 17).astype(np.int64)
    idx = np.arange(0, ap.size, 97)
    for j in range(16):
        st.append(_cuda(b.cal_pred[cuts[j]:cuts[j + 1]]), _cuda(b.cal_truth[cuts[j]:cuts[j + 1]]))
        n = int(cuts[j + 1])
        _check_state(orc, st, b.cal_pred[:n], b.cal_truth[:n], b.edges, 500, b.alpha_ppm, ap[idx], b.u_max,
                     f"large after {n}")
    _check_state(orc, st, b.cal_pred, b.cal_truth, b.edges, 500, b.alpha_ppm, ap, b.u_max, "large all")


def test_incremental_window_errors():
    import torch

    import paper_2609_15359_amd as maps
    st = maps.WindowState(_cuda([10, 20]), 5)
    st.append(_cuda([1, -2]), _cuda([3, 4]))
    torch.cuda.synchronize()
    assert int(st.dev_err.item()) & 1
    st = maps.WindowState(_cuda([20, 10]), 5)
    st.append(_cuda([1, 2]), _cuda([3, 4]))
    torch.cuda.synchronize()
    assert int(st.dev_err.item()) & 2
    st = maps.WindowState(_cuda([10, 20]), 5)
    st.state[:4] = 0    # not a reset state
    st.bounds(100000)
    torch.cuda.synchronize()
    assert int(st.dev_err.item()) & 32
