"""Projected placement in blocks of S tokens on the GPU (maps_project_blocks,
maps_place_blocks) against the CPU oracle, bit for bit: base peaks, every
pair peak and every choice in blocks.  Hand-worked example, block size 1
against the token path, random ragged decoders with bounds past u_max and
outran residents, block sizes 1 to 64, the seeded workloads at block size 16
(literal and with room), and the device error bits."""
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


def _gpu(seg, p, g, U, u_max, S, cap, Q, a_p, a_U, policy=0, rr=0):
    import torch

    import paper_2609_15359_amd as maps
    snap, base, err = maps.project_blocks(_cuda(seg, np.int64), _cuda(p), _cuda(g), _cuda(U), u_max, S)
    pl = maps.place_blocks(snap, _cuda(cap), _cuda(Q), _cuda(a_p), _cuda(a_U), policy, rr, dev_err=err)
    torch.cuda.synchronize()
    return dict(base=base.cpu().numpy(), choice=pl.choice.cpu().numpy(), chosen_peak=pl.chosen_peak.cpu().numpy(),
                chosen_overflow=pl.chosen_overflow.cpu().numpy(), flags=pl.flags.cpu().numpy(),
                pair_peak=pl.pair_peak.cpu().numpy(), err=int(err.item()) & 0xFFFFFFFF)


def _compare(g, r, cols=None, tag=""):
    sel = slice(None) if cols is None else cols
    assert_same(f"{tag} base_peak", g["base"], r.base_peak)
    assert_same(f"{tag} pair_peak", g["pair_peak"][:, sel], r.pair_peak)
    for f in ("choice", "chosen_peak", "chosen_overflow", "flags"):
        assert_same(f"{tag} {f}", g[f][sel], getattr(r, f))


def test_hand_worked_example(orc):
    from tests.oracle_pins import golden
    gd = golden("place_blocks_hand.json")
    got = _gpu(gd["seg_off"], gd["p"], gd["g"], gd["U"], 100, gd["S"], gd["capacity"], gd["queue_len"], gd["a_p"],
               gd["a_U"])
    assert got["err"] == 0
    assert got["pair_peak"].tolist() == gd["pair_peak"] and got["choice"].tolist() == gd["choice"]
    assert got["chosen_peak"].tolist() == gd["chosen_peak"] and got["flags"].tolist() == gd["flags"]
    assert got["chosen_overflow"].tolist() == gd["chosen_overflow"] and got["base"].tolist() == gd["base_peak"]


CASES = [  # (D, max residents, A, u_max, S)
    (1, 40, 700, 50, 1), (3, 200, 1025, 4096, 16), (5, 300, 3000, 4096, 2), (17, 120, 5000, 20000, 37),
    (9, 64, 4097, 300, 64), (4, 0, 100, 100, 16),
    # decoders with more distinct remaining lengths than the projection's LDS records hold (about
    # 1,000 at S = 64, 2,700 at S = 16 with u_max 60,000), or with 65,536 residents or more: their
    # arrays stay in HBM, beside decoders that fit
    (3, 4000, 2000, 30000, 64), (4, 10000, 1200, 60000, 16), (1, 200000, 300, 1000, 16),
    # two whole sort tiles of 8,192 arrivals and a ragged third, bounds up to the largest u_max (sorted in
    # ranges of four steps)
    (6, 150, 16461, 131072, 16),
]


@pytest.mark.parametrize("D,nmax,A,u_max,S", CASES, ids=[f"D{c[0]}-A{c[2]}-u{c[3]}-S{c[4]}" for c in CASES])
@pytest.mark.parametrize("policy", [0, 1])
def test_ragged(orc, D, nmax, A, u_max, S, policy):
    rng = np.random.default_rng(97 * D + A + S + policy)
    counts = rng.integers(0, nmax + 1, size=D)
    counts[0] = 0 if D > 1 else counts[0]      # an empty decoder
    seg = np.zeros(D + 1, np.int64)
    seg[1:] = np.cumsum(counts)
    n = int(seg[-1])
    p = rng.integers(0, 5000, size=n).astype(np.int32)
    U = rng.integers(0, u_max + 1, size=n).astype(np.int32)
    g = rng.integers(0, u_max + 3, size=n).astype(np.int32)      # some outran their bound
    a_p = rng.integers(0, 5000, size=A).astype(np.int32)
    a_U = rng.integers(-1, u_max + 1, size=A).astype(np.int32)
    a_U[: min(A, 3)] = [u_max + 40, 0, u_max][: min(A, 3)]       # a bound past u_max, zero, u_max
    Q = rng.integers(0, 4, size=D).astype(np.int32)
    r0 = orc.place_blocks(seg, p, g, U, np.zeros(D, np.int32), Q, S, a_p, a_U, policy, 11, want_pairs=False)
    cap = ((r0.base_peak + rng.integers(0, 200, size=D)) * S).astype(np.int32)
    say(f"[blocks] D={D} A={A} u_max={u_max} S={S} policy={policy}")
    want = orc.place_blocks(seg, p, g, U, cap, Q, S, a_p, a_U, policy, 11)
    got = _gpu(seg, p, g, U, u_max, S, cap, Q, a_p, a_U, policy, 11)
    assert got["err"] == 0
    _compare(got, want, tag=f"D{D} S{S}")


def test_block_size_one_is_the_token_path(orc):
    """S = 1: the block path's outputs equal the token path's, kernel for kernel."""
    import torch

    import paper_2609_15359_amd as maps
    b = workload.make("small")
    U = oracle.step(b, orc, want_pairs=False).U
    U_res, U_arr, _ = b.split_bounds(U)
    got = _gpu(b.seg_off, b.res_prompt, b.res_gen, U_res, b.u_max, 1, b.capacity, b.queue_len, b.arr_prompt, U_arr)
    snap, base, err = maps.project(_cuda(b.seg_off, np.int64), _cuda(b.res_prompt), _cuda(b.res_gen), _cuda(U_res),
                                   b.u_max)
    pl = maps.place(snap, _cuda(b.capacity), _cuda(b.queue_len), _cuda(b.arr_prompt), _cuda(U_arr), dev_err=err)
    torch.cuda.synchronize()
    assert got["err"] == 0 and int(err.item()) == 0
    assert_same("base", got["base"], base.cpu().numpy())
    for f in ("choice", "chosen_peak", "chosen_overflow", "flags", "pair_peak"):
        assert_same(f, got[f], getattr(pl, f).cpu().numpy())


@pytest.mark.parametrize("name", ["tiny", "small", "medium", "large", "xlarge"])
def test_workload_block16(orc, name):
    """The seeded workloads at block size 16 with their own bounds: every
    output in full up to large; at xlarge 2,000 sampled arrivals against
    every decoder (the oracle's matrix would not fit the host)."""
    b = workload.make(name)
    U = oracle.step(b, orc, want_pairs=False).U
    U_res, U_arr, _ = b.split_bounds(U)
    say(f"[blocks] {name}: D={b.decoders} A={b.arrivals}")
    got = _gpu(b.seg_off, b.res_prompt, b.res_gen, U_res, b.u_max, 16, b.capacity, b.queue_len, b.arr_prompt, U_arr)
    assert got["err"] == 0
    if b.arrivals * b.decoders <= 70_000_000:
        want = orc.place_blocks(b.seg_off, b.res_prompt, b.res_gen, U_res, b.capacity, b.queue_len, 16,
                                b.arr_prompt, U_arr)
        _compare(got, want, tag=name)
    else:
        rng = np.random.default_rng(2)
        cols = np.sort(rng.choice(np.flatnonzero(U_arr >= 0), 2000, replace=False))
        want = orc.place_blocks(b.seg_off, b.res_prompt, b.res_gen, U_res, b.capacity, b.queue_len, 16,
                                b.arr_prompt[cols], U_arr[cols])
        _compare(got, want, cols, tag=name)
    # with room: capacities a little above each decoder's base peak (both branches)
    cap = ((got["base"].astype(np.int64) + np.random.default_rng(4).integers(0, 600, size=b.decoders)) * 16)
    cap = np.minimum(cap, 2**31 - 1).astype(np.int32)
    if b.arrivals * b.decoders <= 5_000_000:
        got2 = _gpu(b.seg_off, b.res_prompt, b.res_gen, U_res, b.u_max, 16, cap, b.queue_len, b.arr_prompt, U_arr)
        want2 = orc.place_blocks(b.seg_off, b.res_prompt, b.res_gen, U_res, cap, b.queue_len, 16, b.arr_prompt,
                                 U_arr)
        _compare(got2, want2, tag=f"{name} with room")
        say(f"[blocks] {name} with room: feasible fraction {np.mean(want2.flags & 1):.3f}")


def test_error_bits():
    got = _gpu([0, 2], [5, -1], [0, 0], [3, 3], 100, 16, [100], [0], [1], [2])
    assert got["err"] & 1
    got = _gpu([0, 2], [5, 1], [0, 0], [3, 300], 100, 16, [100], [0], [1], [2])
    assert got["err"] & 16
    got = _gpu([0, 5], [5, 1], [0, 0], [3, 3], 100, 16, [100], [0], [1], [2])
    assert got["err"] & 8
    # placement's own inputs: a negative prompt (of an arrival with a bound), capacity or queue length
    ok = _gpu([0, 2], [5, 1], [0, 0], [3, 3], 100, 16, [100], [0], [1], [2])
    assert ok["err"] == 0
    assert _gpu([0, 2], [5, 1], [0, 0], [3, 3], 100, 16, [100], [0], [-1], [2])["err"] == 1
    assert _gpu([0, 2], [5, 1], [0, 0], [3, 3], 100, 16, [100], [0], [-1], [-1])["err"] == 0   # no bound: RR
    assert _gpu([0, 2], [5, 1], [0, 0], [3, 3], 100, 16, [-5], [0], [1], [2])["err"] == 1
    assert _gpu([0, 2], [5, 1], [0, 0], [3, 3], 100, 16, [100], [-2], [1], [2])["err"] == 1
    # a pair peak beyond INT32_MAX blocks at S = 1 (prompt near INT32_MAX plus the residents)
    big = _gpu([0, 1], [5], [0], [3], 100, 1, [100], [0], [2**31 - 8], [50])
    assert big["err"] & 4


def test_snapshot_mismatch_is_reported():
    """maps_place_blocks called with arguments other than those the snapshot
    was built for (block size, u_max, n_total, D, per-decoder resident counts,
    a buffer never written) raises SNAPSHOT and reads no slice; the matching
    call raises nothing."""
    import dataclasses

    import torch

    import paper_2609_15359_amd as maps
    rng = np.random.default_rng(5)
    D, A, S, u_max = 4, 300, 16, 500
    seg = np.array([0, 30, 30, 75, 120], np.int64)
    n = int(seg[-1])
    p = rng.integers(0, 900, size=n).astype(np.int32)
    g = rng.integers(0, 50, size=n).astype(np.int32)
    U = rng.integers(0, u_max, size=n).astype(np.int32) + g
    a_p = rng.integers(0, 900, size=A).astype(np.int32)
    a_U = rng.integers(0, u_max + 1, size=A).astype(np.int32)
    snap, _, err = maps.project_blocks(_cuda(seg, np.int64), _cuda(p), _cuda(g), _cuda(U), u_max, S)
    torch.cuda.synchronize()
    assert int(err.item()) == 0

    def place(sn, d=D):
        e = maps.new_error_word(snap.data.device)
        maps.place_blocks(sn, _cuda(np.full(d, 10**6)), _cuda(np.zeros(d)), _cuda(a_p), _cuda(a_U), dev_err=e)
        torch.cuda.synchronize()
        return int(e.item()) & 0xFFFFFFFF

    assert place(snap) == 0
    moved = seg.copy()
    moved[2] += 1                                    # one resident moved from decoder 2 to decoder 1
    bad = [dataclasses.replace(snap, block_size=S + 1), dataclasses.replace(snap, u_max=u_max + 1),
           dataclasses.replace(snap, n_total=n + 1), dataclasses.replace(snap, seg_off=_cuda(moved, np.int64)),
           dataclasses.replace(snap, data=torch.zeros_like(snap.data))]
    for sn in bad:
        assert place(sn) & 32, sn
    wider = dataclasses.replace(snap, D=D + 1, seg_off=_cuda(np.append(seg, n), np.int64))
    assert place(wider, D + 1) & 32
    assert place(snap) == 0
