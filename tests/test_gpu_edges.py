"""Edge cases of the HIP path against the oracle: empty and ragged inputs,
ties, degenerate bounds, the capacity boundary, decoders too large for LDS,
long queues, and every device value-error bit (which must be reported
without the kernels leaving their buffers)."""
import zlib

import numpy as np
import pytest

import oracle
import workload
from tests.gpu_common import assert_same, compare_all, custom_batch, gpu_step, oracle_step, say

pytestmark = pytest.mark.gpu
Q_INF = 2**31 - 1


@pytest.fixture(scope="module")
def orc():
    return oracle.Oracle()


def _cuda(x, dtype=np.int32):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=dtype)).cuda()


def _calib_gpu(pred, truth, edges, alpha, apply_pred, u_max):
    import torch

    import paper_2609_15359_amd as maps
    q, cnt, U, err = maps.calibrate(_cuda(pred), _cuda(truth), _cuda(edges), alpha,
                                    _cuda(apply_pred) if len(apply_pred) else None, u_max)
    torch.cuda.synchronize()
    return (q.cpu().numpy(), cnt.cpu().numpy(), None if U is None else U.cpu().numpy(),
            int(err.item()) & 0xFFFFFFFF)


CAL_CASES = {
    "all_zero_scores": dict(n=3000, nb=4, alpha=100000, zero=True),
    "heavy_ties": dict(n=5000, nb=8, alpha=100000, tie=True),
    "single_bucket": dict(n=2000, nb=1, alpha=50000),
    "small_buckets_k_gt_n": dict(n=40, nb=8, alpha=100000),
    "empty_set": dict(n=0, nb=4, alpha=100000),
    "wide_scores_4_passes": dict(n=20000, nb=16, alpha=100000, wide=True),
    "many_buckets_global_hist": dict(n=50000, nb=200, alpha=100000),
    "very_many_buckets_global_edges": dict(n=60000, nb=9000, alpha=200000),
    "buckets_1024_sorted_path": dict(n=40000, nb=1024, alpha=100000),
    "buckets_1025_all_bucket_path": dict(n=40000, nb=1025, alpha=100000),
    "one_bucket_holds_most": dict(n=120000, nb=8, alpha=50000, skew=True),
    "alpha_1ppm": dict(n=4000, nb=4, alpha=1),
    "alpha_999999ppm": dict(n=4000, nb=4, alpha=999999),
    "duplicate_edges": dict(n=4000, nb=6, alpha=100000, dup=True),
    # residuals in prediction order: each chunk of 4,096 falls in one or two
    # buckets, so runs are far longer than a wavefront
    "sorted_pred_long_runs": dict(n=30000, nb=4, alpha=100000, sort=True),
    "ragged_last_chunk": dict(n=4097, nb=3, alpha=100000),
    "chunks_at_limit": dict(n=1024 * 4096, nb=128, alpha=100000),
    "one_past_chunk_limit": dict(n=1024 * 4096 + 1, nb=16, alpha=50000),
}


@pytest.mark.parametrize("case", list(CAL_CASES), ids=list(CAL_CASES))
def test_calibrate_cases(orc, case):
    c = CAL_CASES[case]
    rng = np.random.default_rng(zlib.crc32(case.encode()))
    n, nb = c["n"], c["nb"]
    pred = rng.integers(1, 5000, size=n).astype(np.int32)
    truth = (pred + rng.integers(-2000, 3000, size=n)).clip(0).astype(np.int32)
    if c.get("zero"):
        truth = (pred - rng.integers(0, 50, size=n)).clip(0).astype(np.int32)
    if c.get("tie"):
        truth = (pred + rng.choice([0, 7, 7, 7, 100], size=n)).astype(np.int32)
    if c.get("wide"):
        truth = (pred.astype(np.int64) + rng.integers(0, 2**30, size=n)).clip(0, 2**31 - 1).astype(np.int32)
    edges = np.sort(rng.integers(0, 5000, size=nb - 1)).astype(np.int32)
    if c.get("dup"):
        edges = np.array([100, 100, 100, 2000, 9000][: nb - 1], np.int32)
    if c.get("skew"):
        edges = np.array([4000, 4100, 4200, 4300, 4400, 4500, 4600], np.int32)[: nb - 1]
    if c.get("sort"):
        order = np.argsort(pred, kind="stable")
        pred, truth = pred[order], truth[order]
    u_max = 65536
    ap = np.concatenate([rng.integers(-3, 10**6, size=3000), [-1, 0, 1, 2**31 - 1]]).astype(np.int32)
    say(f"[edge] calibrate {case}: n={n} nb={nb}")
    q, cnt, U, err = _calib_gpu(pred, truth, edges, c["alpha"], ap, u_max)
    assert err == 0
    qo, co = orc.calibrate(pred, truth, edges, c["alpha"])
    assert_same("q", q, qo)
    assert_same("count", cnt, co)
    assert_same("U", U, orc.apply_bounds(ap, edges, qo, u_max))


def _decoders(rng, D, nmax, u_max, pmax=3000, empty_every=3):
    counts = rng.integers(0, nmax + 1, size=D)
    counts[::empty_every] = 0
    seg = np.zeros(D + 1, np.int64)
    seg[1:] = np.cumsum(counts)
    n = int(seg[-1])
    p = rng.integers(0, pmax, size=n).astype(np.int32)
    pred = rng.integers(0, u_max // 2, size=n).astype(np.int32)
    g = rng.integers(0, u_max // 2, size=n).astype(np.int32)
    return seg, p, g, pred


def _queues(rng, D, qmax, u_max):
    qc = rng.integers(0, qmax + 1, size=D)
    qoff = np.zeros(D + 1, np.int64)
    qoff[1:] = np.cumsum(qc)
    nq = int(qoff[-1])
    return (qoff, rng.integers(0, 3000, size=nq).astype(np.int32),
            rng.integers(-5, u_max, size=nq).astype(np.int32), rng.integers(0, 2000, size=nq).astype(np.int32))


SHAPES = [  # (D, max residents, A, max queue)
    (1, 50, 1, 3), (3, 200, 1025, 40), (9, 300, 5000, 64), (17, 100, 9000, 0), (64, 40, 70000, 10),
    # more decoders than the final selection stages capacities for in LDS (16,384), and more than a
    # 16-bit decoder index holds in the groups' partial choices (65,536)
    (16500, 2, 300, 1), (70000, 1, 100, 0),
]


@pytest.mark.parametrize("D,nmax,A,qmax", SHAPES, ids=[f"D{s[0]}-A{s[2]}" for s in SHAPES])
@pytest.mark.parametrize("policy", [0, 1])
def test_ragged_shapes(orc, D, nmax, A, qmax, policy):
    """Uneven decoder groups, ragged arrival tiles, empty decoders and queues,
    g >= U residents, zero and missing bounds, bounds above u_max."""
    rng = np.random.default_rng(1000 * D + A + policy)
    u_max = 4096
    seg, p, g, pred = _decoders(rng, D, nmax, u_max)
    arr_pred = rng.integers(-2, u_max + 500, size=A).astype(np.int32)
    arr_pred[: min(A, 5)] = [0, -1, u_max, u_max + 7, 3][: min(A, 5)]
    qoff, qp, qpred, qw = _queues(rng, D, qmax, u_max)
    cal_pred = rng.integers(1, 3000, size=3000).astype(np.int32)
    cal_truth = (cal_pred + rng.integers(-500, 1500, size=3000)).clip(0).astype(np.int32)
    b = custom_batch(cal_pred=cal_pred, cal_truth=cal_truth, edges=[300, 900, 2000], alpha_ppm=100000,
                     u_max=u_max, seg_off=seg, res_prompt=p, res_gen=g, res_pred=pred,
                     arr_prompt=rng.integers(0, 3000, size=A), arr_pred=arr_pred,
                     capacity=rng.integers(0, 400000, size=D), queue_len=rng.integers(0, 4, size=D),
                     q_off=qoff, q_prompt=qp, q_pred=qpred, q_wait_ms=qw)
    o0 = oracle_step(b, o=orc, want_pairs=False)
    cap = (o0["base_peak"] + rng.integers(0, 20000, size=D)).astype(np.int32)
    for capacity in (None, cap):
        o = oracle_step(b, capacity=capacity, policy=policy, rr_offset=2**40 + 3, o=orc)
        for fused in (False, True, "project"):
            gg = gpu_step(b, capacity=capacity, policy=policy, rr_offset=2**40 + 3, fused=fused)
            assert gg["err"] == 0, gg["errors"]
            compare_all(gg, o)


@pytest.mark.parametrize("want_pairs", [False, True])
@pytest.mark.parametrize("policy", [0, 1])
def test_record_path(orc, policy, want_pairs):
    """u_max above the dense-profile limit (16,384 entries): placement answers
    every pair from the rank words and event records instead."""
    rng = np.random.default_rng(77 + 2 * policy + want_pairs)
    D, nmax, A, qmax, u_max = 9, 300, 5000, 20, 20000
    seg, p, g, pred = _decoders(rng, D, nmax, u_max)
    arr_pred = rng.integers(-2, u_max + 500, size=A).astype(np.int32)
    qoff, qp, qpred, qw = _queues(rng, D, qmax, u_max)
    b = custom_batch(cal_pred=np.arange(1, 41), cal_truth=np.arange(1, 41) + 7, edges=[20], alpha_ppm=100000,
                     u_max=u_max, seg_off=seg, res_prompt=p, res_gen=g, res_pred=pred,
                     arr_prompt=rng.integers(0, 3000, size=A), arr_pred=arr_pred,
                     capacity=rng.integers(0, 400000, size=D), queue_len=rng.integers(0, 4, size=D),
                     q_off=qoff, q_prompt=qp, q_pred=qpred, q_wait_ms=qw)
    o0 = oracle_step(b, o=orc, want_pairs=False)
    cap = (o0["base_peak"] + rng.integers(0, 30000, size=D)).astype(np.int32)
    o = oracle_step(b, capacity=cap, policy=policy, want_pairs=want_pairs, o=orc)
    gg = gpu_step(b, capacity=cap, policy=policy, want_pairs=want_pairs)
    assert gg["err"] == 0, gg["errors"]
    compare_all(gg, o, pairs=want_pairs)


@pytest.mark.parametrize("policy", [0, 1])
def test_record_path_growing_occupancy(orc, policy):
    """Residents with long remaining lengths and small prompts: the occupancy
    grows until the first event, so for short bounds the line S + U (N + 1)
    exceeds the running maximum and placement must read the cold records."""
    rng = np.random.default_rng(91 + policy)
    D, u_max, A = 5, 20000, 4000
    counts = [3, 40, 1, 200, 0]
    seg = np.zeros(D + 1, np.int64)
    seg[1:] = np.cumsum(counts)
    n = int(seg[-1])
    p = rng.integers(0, 20, size=n).astype(np.int32)
    g = rng.integers(0, 5, size=n).astype(np.int32)
    pred = rng.integers(5000, u_max, size=n).astype(np.int32)
    arr = rng.integers(-1, 9000, size=A).astype(np.int32)
    b = custom_batch(cal_pred=[5], cal_truth=[5], edges=[], alpha_ppm=100000, u_max=u_max, seg_off=seg,
                     res_prompt=p, res_gen=g, res_pred=pred, arr_prompt=rng.integers(0, 500, size=A),
                     arr_pred=arr, capacity=rng.integers(0, 60000, size=D), queue_len=[2, 0, 1, 3, 0])
    b.cal_pred = np.arange(1, 21, dtype=np.int32)
    b.cal_truth = b.cal_pred.copy()
    o = oracle_step(b, policy=policy, o=orc)
    gg = gpu_step(b, policy=policy)
    assert gg["err"] == 0, gg["errors"]
    compare_all(gg, o)


def hot_windows(b, U):
    """Each decoder's hot window and flat region recomputed on the host from
    the definitions: events tau_e (distinct remaining lengths), N_e and S_e
    over R >= tau_e, PMX_e = max(0, max_{i<e} S_i + tau_i (N_i + 1)), the
    threshold T_e (the smallest bound with S_e + U (N_e + 1) > PMX_e), and the
    bounds landing on e < E, (tau_{e-1}, tau_e], that reach it (after the last
    event S_E = N_E = 0 and max(PMX_E, U) is exact); the window lies above
    event 0's such range and below the first one of a later event.  The flat
    region starts past the first event e* with PMX_e = PMX_E.  Returns rows
    (hot_lo, hot_hi, flat_lo, PMX_E)."""
    big = 2**31 - 1
    out = []
    for d in range(b.decoders):
        lo, hi = int(b.seg_off[d]), int(b.seg_off[d + 1])
        p = b.res_prompt[lo:hi].astype(np.int64)
        g = b.res_gen[lo:hi].astype(np.int64)
        R = np.maximum(U[lo:hi].astype(np.int64) - g, 0)
        tau = np.unique(R)
        E = tau.size
        N = np.array([(R >= t).sum() for t in tau] + [0], np.int64)
        S = np.array([(p + g)[R >= t].sum() for t in tau] + [0], np.int64)
        pmx = [0]
        for e in range(E):
            pmx.append(max(pmx[-1], int(S[e] + tau[e] * (N[e] + 1))))
        win_lo, first = 0, None
        for e in range(E):
            n1 = int(N[e]) + 1
            T = 0 if S[e] > pmx[e] else min((pmx[e] - int(S[e])) // n1 + 1, big)
            lo_e = 0 if e == 0 else int(tau[e - 1]) + 1
            hi_e = int(tau[e])
            start = max(T, lo_e)
            if start > hi_e:
                continue
            if e == 0:
                win_lo = hi_e + 1
            elif first is None:
                first = start
        estar = next(e for e in range(E + 1) if pmx[e] == pmx[E])
        flat_lo = 0 if estar == 0 else int(tau[estar - 1]) + 1
        out.append((win_lo, (big if first is None else first) - 1, flat_lo, pmx[E]))
    return np.array(out, np.int64)


def window_batch(seed):
    """Record-path decoders of four kinds in groups of two: growing occupancy
    (short prompts, long remaining lengths: cold ranges right above the first
    event), long prompts (a window far above u_max), a single resident, and no
    resident; every arrival has a bound, spread over [1, u_max]."""
    rng = np.random.default_rng(seed)
    D, u_max, A = 16, 20000, 20000
    kinds = [0, 1, 1, 1, 2, 1, 0, 0, 3, 1, 1, 2, 0, 3, 1, 0]
    counts = [[30, 300, 1, 0][k] for k in kinds]
    seg = np.zeros(D + 1, np.int64)
    seg[1:] = np.cumsum(counts)
    p, g, pred = [], [], []
    for k, c in zip(kinds, counts):
        if k == 0:
            p.append(rng.integers(0, 20, c)); g.append(rng.integers(0, 5, c)); pred.append(rng.integers(5000, u_max, c))
        else:
            p.append(rng.integers(5000, 100000, c)); g.append(rng.integers(0, 50, c)); pred.append(rng.integers(1, u_max, c))
    b = custom_batch(cal_pred=np.arange(1, 21), cal_truth=np.arange(1, 21), edges=[], alpha_ppm=100000, u_max=u_max,
                     seg_off=seg, res_prompt=np.concatenate(p), res_gen=np.concatenate(g),
                     res_pred=np.concatenate(pred), arr_prompt=rng.integers(0, 500, size=A),
                     arr_pred=np.sort(rng.integers(1, u_max + 1, size=A)), capacity=rng.integers(0, 3 * 10**6, size=D),
                     queue_len=rng.integers(0, 4, size=D))
    return b


def test_hot_window_headers(orc):
    """The projection's hot window, flat region start and PMX_E of every
    decoder equal the ones recomputed from the definitions (a window too wide
    would skip a needed cold record)."""
    b = window_batch(5)
    o = oracle_step(b, o=orc)
    gg = gpu_step(b)
    assert gg["err"] == 0, gg["errors"]
    want = hot_windows(b, o["U"][: b.res_pred.size])
    got = gg["dec_hdr"][:, 6:10].astype(np.int64)
    say("hot windows and flat regions", got.tolist())
    assert np.array_equal(got, want), (got, want)
    # some decoders have a usable flat region, others (growing occupancy) not
    assert (want[:, 2] <= want[:, 1]).any() and (want[:, 2] > want[:, 1]).any()


@pytest.mark.parametrize("policy", [0, 1])
def test_hot_walk_mixed_with_full_walk(orc, policy):
    """Arrival tiles sorted by bound fall inside, across and outside the hot
    windows of their decoder groups, so both walks run in one launch."""
    b = window_batch(6 + policy)
    o = oracle_step(b, policy=policy, o=orc)
    gg = gpu_step(b, policy=policy)
    assert gg["err"] == 0, gg["errors"]
    compare_all(gg, o)


def test_capacity_boundary_and_ties(orc):
    """A peak equal to the capacity is feasible; equal queues and equal slacks
    go to the lowest decoder; all-infeasible arrivals take the largest slack."""
    rng = np.random.default_rng(7)
    D, u_max = 6, 1000
    seg = np.array([0, 4, 8, 12, 16, 20, 24], np.int64)   # identical decoders
    p = np.tile(rng.integers(0, 500, size=4), D).astype(np.int32)
    g = np.zeros(24, np.int32)
    pred = np.tile(rng.integers(0, 400, size=4), D).astype(np.int32)
    A = 300
    b = custom_batch(cal_pred=[10, 20, 30], cal_truth=[10, 20, 30], edges=[], alpha_ppm=500000, u_max=u_max,
                     seg_off=seg, res_prompt=p, res_gen=g, res_pred=pred,
                     arr_prompt=rng.integers(0, 300, size=A), arr_pred=rng.integers(0, 600, size=A),
                     capacity=np.full(D, 10**6), queue_len=[3, 1, 1, 2, 1, 5])
    o0 = oracle_step(b, o=orc)
    peaks = o0["pair_peak"][0]
    at_peak = np.full(D, int(peaks[0]), np.int32)          # arrival 0 lands exactly on the capacity
    for capacity in (at_peak, np.zeros(D, np.int32),
                     np.array([peaks.min()] * 3 + [peaks.max()] * 3, np.int32)):
        o = oracle_step(b, capacity=capacity, o=orc)
        gg = gpu_step(b, capacity=capacity)
        assert gg["err"] == 0
        compare_all(gg, o)
    o = oracle_step(b, capacity=at_peak, o=orc)
    assert o["flags"][0] == 1 and o["chosen_peak"][0] == at_peak[0] and o["chosen_overflow"][0] == 0


def test_decoder_too_large_for_lds(orc):
    """20,000 residents with mostly distinct remaining lengths: projection runs
    on the decoder's HBM slice and placement reads its records from HBM."""
    rng = np.random.default_rng(11)
    u_max = 65535
    n_big = 20000
    seg = np.array([0, 10, n_big + 10, n_big + 40], np.int64)
    n = int(seg[-1])
    p = rng.integers(0, 100, size=n).astype(np.int32)
    g = np.zeros(n, np.int32)
    pred = rng.permutation(u_max)[:n].astype(np.int32)
    A = 3000
    b = custom_batch(cal_pred=[5], cal_truth=[5], edges=[], alpha_ppm=100000, u_max=u_max, seg_off=seg,
                     res_prompt=p, res_gen=g, res_pred=pred, arr_prompt=rng.integers(0, 1000, size=A),
                     arr_pred=rng.integers(-1, u_max, size=A), capacity=[2**31 - 1, 10**9, 10**8],
                     queue_len=[0, 1, 2])
    # the one calibration score is 0 at k = ceil(0.9 * 2) = 2 > 1 -> infinite quantile, so every
    # bound is u_max; use a bound-preserving set instead: 20 zero scores
    b.cal_pred = np.arange(1, 21, dtype=np.int32)
    b.cal_truth = b.cal_pred.copy()
    o = oracle_step(b, o=orc)
    gg = gpu_step(b)
    assert gg["err"] == 0, gg["errors"]
    compare_all(gg, o)
    say(f"[edge] big decoder: base peaks {o['base_peak'].tolist()}")


def test_local_queues_long_and_promoted(orc):
    rng = np.random.default_rng(13)
    D, u_max = 4, 8192
    seg = np.array([0, 100, 200, 200, 300], np.int64)
    n = 300
    qlens = [2048, 1, 0, 700]
    qoff = np.zeros(D + 1, np.int64)
    qoff[1:] = np.cumsum(qlens)
    nq = int(qoff[-1])
    qw = rng.integers(0, 3000, size=nq).astype(np.int32)
    qw[qoff[3]:qoff[4]] = 5000                       # every request of decoder 3 promoted
    qpred = rng.integers(-3, u_max, size=nq).astype(np.int32)
    qpred[:500] = 77                                 # long run of equal bounds
    b = custom_batch(cal_pred=np.arange(1, 41), cal_truth=np.arange(1, 41) + 3, edges=[20], alpha_ppm=100000,
                     u_max=u_max, seg_off=seg, res_prompt=rng.integers(0, 2000, size=n),
                     res_gen=rng.integers(0, 100, size=n), res_pred=rng.integers(0, 4000, size=n),
                     arr_prompt=[5, 6], arr_pred=[10, 20], capacity=[0, 1, 2, 3],
                     q_off=qoff, q_prompt=rng.integers(0, 500, size=nq), q_pred=qpred, q_wait_ms=qw)
    o0 = oracle_step(b, o=orc)
    for capacity in (o0["base_peak"] + np.array([10**6, 0, 5000, 10**7]), np.full(D, 2**31 - 1),
                     np.zeros(D)):
        capacity = np.minimum(capacity, 2**31 - 1).astype(np.int32)
        o = oracle_step(b, capacity=capacity, o=orc)
        gg = gpu_step(b, capacity=capacity)
        assert gg["err"] == 0, gg["errors"]
        compare_all(gg, o)
        say(f"[edge] long queues: admitted {o['admitted'].tolist()}")


# ---------------------------------------------------------------------------
# device value errors: reported in the error word, kernels stay in bounds
# ---------------------------------------------------------------------------

def _project(seg, p, g, U, u_max):
    import torch

    import paper_2609_15359_amd as maps
    snap, base, err = maps.project(_cuda(seg, np.int64), _cuda(p), _cuda(g), _cuda(U), u_max)
    torch.cuda.synchronize()
    return snap, base, int(err.item()) & 0xFFFFFFFF


def test_error_bits():
    import torch

    import paper_2609_15359_amd as maps
    bits = maps.ERR_BITS
    inv = {v: k for k, v in bits.items()}
    # calibration: negative lengths, unsorted edges
    *_, err = _calib_gpu([5, -1, 3], [4, 5, 6], [10, 2], 100000, [1, 2], 100)
    assert err & inv["NEG_LEN"] and err & inv["EDGES_UNSORTED"]
    # projection: negative lengths, decreasing offsets, remaining length above u_max, int32 range
    _, _, err = _project([0, 2], [1, -5], [0, 0], [3, 3], 100)
    assert err & inv["NEG_LEN"]
    _, _, err = _project([0, 2, 1, 3], [1, 1, 1], [0, 0, 0], [3, 3, 3], 100)
    assert err & inv["SEG_OFFSETS"]
    _, _, err = _project([0, 5, 9], [1] * 3, [0] * 3, [3] * 3, 100)       # offsets past n_total
    assert err & inv["SEG_OFFSETS"]
    _, _, err = _project([0, 1], [1], [0], [5000], 100)
    assert err & inv["BOUND_RANGE"]
    _, _, err = _project([0, 3], [2**30, 2**30, 2**30], [0, 0, 0], [1, 1, 1], 100)
    assert err & inv["INT32_RANGE"]
    # placement: snapshot built for another u_max; negative prompt and capacity; peak overflow
    snap, base, err = _project([0, 2], [10, 20], [0, 0], [5, 6], 100)
    assert err == 0
    wrong = maps.Snapshot(data=snap.data, D=snap.D, n_total=snap.n_total, u_max=200)
    pl = maps.place(wrong, _cuda([100]), _cuda([0]), _cuda([1, 2]), _cuda([3, 4]))
    torch.cuda.synchronize()
    assert int(pl.dev_err.item()) & inv["SNAPSHOT"]
    pl = maps.place(snap, _cuda([-1]), _cuda([0]), _cuda([-1, 2]), _cuda([3, 2**31 - 10]))
    torch.cuda.synchronize()
    e = int(pl.dev_err.item())
    assert e & inv["NEG_LEN"] and e & inv["INT32_RANGE"]
    # local order: queue longer than the limit, bad offsets
    n = maps.MAX_LOCAL_QUEUE + 1
    _, adm, err = maps.local_order(snap, _cuda([100]), _cuda([0, n], np.int64), _cuda(np.ones(n)),
                                   _cuda(np.ones(n)))
    torch.cuda.synchronize()
    assert int(err.item()) & inv["QUEUE_TOO_LONG"] and int(adm.item()) == 0
    _, _, err = maps.local_order(snap, _cuda([100]), _cuda([0, 5], np.int64), _cuda(np.ones(3)),
                                 _cuda(np.ones(3)))
    torch.cuda.synchronize()
    assert int(err.item()) & inv["SEG_OFFSETS"]


def test_empty_arrival_batch():
    import torch

    import paper_2609_15359_amd as maps
    snap, _, _ = _project([0, 2], [10, 20], [0, 0], [5, 6], 100)
    pl = maps.place(snap, _cuda([100]), _cuda([0]), _cuda([]), _cuda([]))
    torch.cuda.synchronize()
    assert pl.choice.numel() == 0 and int(pl.dev_err.item()) == 0


def test_empty_arrival_batch_with_queues(orc):
    """maps_place_order with no arrivals still orders and admits every local
    queue (one empty)."""
    import torch

    import paper_2609_15359_amd as maps
    seg, p, g, U = [0, 2, 2, 3], [10, 20, 30], [0, 0, 5], [5, 6, 40]
    snap, _, _ = _project(seg, p, g, U, 100)
    qoff = np.array([0, 3, 3, 5], np.int64)
    qp = np.array([7, 3, 9, 1, 2], np.int32)
    qU = np.array([50, -1, 4, 9, 9], np.int32)
    cap = np.array([120, 50, 100], np.int32)
    pl, order, admitted = maps.place_order(snap, _cuda(cap), _cuda([0, 0, 0]), _cuda([]), _cuda([]),
                                           _cuda(qoff, np.int64), _cuda(qp), _cuda(qU))
    torch.cuda.synchronize()
    assert pl.choice.numel() == 0 and int(pl.dev_err.item()) == 0
    want_order, want_adm = orc.local_order(np.array(seg, np.int64), np.array(p, np.int32), np.array(g, np.int32),
                                           np.array(U, np.int32), cap, qoff, qp, qU, None, 2**31 - 1, 100)
    assert_same("order", order.cpu().numpy(), want_order)
    assert_same("admitted", admitted.cpu().numpy(), want_adm)


@pytest.mark.parametrize("spins", ["0", "3"])
def test_calibrate_fused_launch_selects_missing_quantiles(orc, spins, monkeypatch):
    """The bounds written by workgroups of the selection's own launch: with the
    bounded wait cut to almost nothing (set from the host), the apply
    workgroups find quantiles not yet published and select them themselves;
    every quantile, count and bound is still the oracle's."""
    monkeypatch.setenv("MAPS_CAL_SPIN_LIMIT", spins)
    for name in ("small", "large"):
        b = workload.make(name)
        ap = b.apply_pred()
        q, cnt, U, err = _calib_gpu(b.cal_pred, b.cal_truth, b.edges, b.alpha_ppm, ap, b.u_max)
        assert err == 0
        qo, co = orc.calibrate(b.cal_pred, b.cal_truth, b.edges, b.alpha_ppm)
        assert_same(f"{name} q", q, qo)
        assert_same(f"{name} count", cnt, co)
        assert_same(f"{name} U", U, orc.apply_bounds(ap, b.edges, qo, b.u_max))
