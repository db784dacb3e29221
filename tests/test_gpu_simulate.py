"""The App. A pressure simulation on the GPU (maps_simulate, one wavefront
per simulation, event to event) against the CPU oracle (one millisecond at a
time), bit for bit: completion times, routing, high-pressure time, longest
interval, interval count, queue maxima and areas, span.  Hand-worked
timelines, random small cases (both policies, thresholds hit exactly,
queueing), the App. A setup at full size over a utilisation sweep, limits and
the device error bits."""
import numpy as np
import pytest

import oracle
import workload.appa as appa
from tests.gpu_common import assert_same, say
from tests.oracle_pins import SIM_FIELDS, _sim_case, golden

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def orc():
    return oracle.Oracle()


def _cuda(x, dtype=np.int32):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=dtype)).cuda()


def _gpu(N, C, theta, arrivals, prompt, output, bound, policies):
    """One call: row s of `arrivals` with policy policies[s]."""
    import torch

    import paper_2609_15359_amd as maps
    arr = np.atleast_2d(np.asarray(arrivals, np.int64))
    r = maps.simulate(N, C, theta, _cuda(arr, np.int64), _cuda(prompt), _cuda(output), _cuda(bound),
                      _cuda(policies))
    torch.cuda.synchronize()
    st = r.stats.cpu().numpy()
    out = []
    for s in range(arr.shape[0]):
        out.append(dict(finish_ms=r.finish_ms[s].cpu().numpy(), routed=r.routed[s].cpu().numpy(),
                        hp_time=st[s, 0], hp_max=st[s, 1], hp_count=st[s, 2], max_queue=st[s, 3],
                        queue_area=st[s, 4], span=r.span[s].cpu().numpy()))
    return out, int(r.dev_err.item()) & 0xFFFFFFFF


def _compare(g, r, tag):
    for f in SIM_FIELDS:
        assert_same(f"{tag} {f}", g[f], getattr(r, f))


def test_hand_worked(orc):
    for c in golden("simulate_hand.json")["cases"]:
        got, err = _gpu(c["N"], c["C"], c["theta_ppm"], [c["arrival_ms"]], c["prompt"], c["output"], c["bound"],
                        [c["policy"]])
        assert err == 0
        for f in SIM_FIELDS:
            assert np.asarray(got[0][f]).tolist() == c[f], (c["name"], f)


def test_random_small(orc):
    rng = np.random.default_rng(77)
    for trial in range(150):
        N, C, theta, arr, prompt, output, bound = _sim_case(rng, n_max=40)
        got, err = _gpu(N, C, theta, [arr, arr], prompt, output, bound, [0, 1])
        assert err == 0, trial
        for pol in (0, 1):
            _compare(got[pol], orc.simulate(N, C, theta, arr, prompt, output, bound, pol), f"trial {trial} p{pol}")


@pytest.mark.parametrize("N", [1, 3, 8])
def test_heavy_queueing(orc, N):
    """Many requests at once on tight decoders: long FIFO queues, many
    admissions per completion, ready queues of tens of requests."""
    rng = np.random.default_rng(N)
    n = 3000
    prompt = rng.integers(0, 200, size=n).astype(np.int32)
    output = rng.integers(1, 400, size=n).astype(np.int32)
    bound = (output + rng.integers(-50, 200, size=n)).clip(-1).astype(np.int32)
    C = 6000
    arr = np.sort(rng.integers(0, 20000, size=n)).astype(np.int64)
    burst = np.zeros(n, np.int64)   # everything at t = 0
    got, err = _gpu(N, C, 700000, [arr, arr, burst, burst], prompt, output, bound, [0, 1, 0, 1])
    assert err == 0
    for s, (a, pol) in enumerate(((arr, 0), (arr, 1), (burst, 0), (burst, 1))):
        _compare(got[s], orc.simulate(N, C, 700000, a, prompt, output, bound, pol), f"N={N} case {s}")


def test_appendix_a_setup(orc):
    """App. A: 10,000 requests, N = 4, C = 50,000 tokens, theta = 0.85,
    t_tok = 1 ms, bounds from the oracle's calibration of the synthetic
    predictor, over a sweep of utilisation."""
    w = appa.make()
    q, _ = orc.calibrate(w.cal_pred, w.cal_truth, w.edges, appa.ALPHA_PPM)
    U = orc.apply_bounds(w.pred, w.edges, q, appa.U_MAX)
    rhos = [0.8, 0.9, 0.96, 1.0, 1.05, 1.1]
    arr = [w.arrivals(r) for r in rhos for _ in (0, 1)]
    pols = [p for _ in rhos for p in (0, 1)]
    got, err = _gpu(appa.N_DECODERS, appa.CAPACITY, appa.THETA_PPM, arr, w.prompt, w.output, U, pols)
    assert err == 0
    for s, (a, pol) in enumerate(zip(arr, pols)):
        r = orc.simulate(appa.N_DECODERS, appa.CAPACITY, appa.THETA_PPM, a, w.prompt, w.output, U, pol)
        _compare(got[s], r, f"rho={rhos[s // 2]} policy={pol}")
        T = r.span[1] - r.span[0]
        say(f"[appa] rho={rhos[s // 2]} policy={pol}: f_hp {np.round(r.hp_time / T, 3).tolist()} "
            f"max queue {r.max_queue.tolist()}")


def test_error_bits():
    ok, err = _gpu(1, 10, 500000, [[0, 1]], [2, 3], [4, 5], [4, 5], [0])
    assert err == 0
    _, err = _gpu(1, 10, 500000, [[0, 1]], [2, 8], [4, 5], [4, 5], [0])    # 8 + 5 > C
    assert err & 2048
    _, err = _gpu(1, 10, 500000, [[3, 1]], [2, 3], [4, 5], [4, 5], [0])    # arrival times decrease
    assert err & 2048
    _, err = _gpu(1, 10, 500000, [[0, 1]], [2, 3], [4, 0], [4, 5], [0])    # an empty output
    assert err & 2048
    n = 1100   # more admitted requests at once than a ready queue holds
    _, err = _gpu(1, 10**6, 500000, [np.zeros(n)], np.zeros(n), np.full(n, 3), np.full(n, 3), [0])
    assert err & 4096
