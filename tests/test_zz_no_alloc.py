"""The allocation-free calibration entry point (maps_calibrate_noalloc),
called through the C ABI, against maps_calibrate on the same inputs: two
calls in a row, the second with a smaller input (the shared scratch keeps the
first call's contents), plus its size limit."""
import ctypes

import numpy as np
import pytest

import workload

pytestmark = pytest.mark.gpu


def _cuda(x, dtype=np.int32):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x, dtype=dtype)).cuda()


def _noalloc(pred, truth, edges, alpha, ap, u_max):
    import torch

    import paper_2609_15359_amd as maps
    nb = edges.numel() + 1
    q = torch.empty(nb, dtype=torch.int32, device="cuda")
    cnt = torch.empty(nb, dtype=torch.int32, device="cuda")
    U = torch.empty(ap.numel(), dtype=torch.int32, device="cuda")
    err = maps.new_error_word()
    p = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    st = maps.library().maps_calibrate_noalloc(p(pred), p(truth), pred.numel(), p(edges), nb, alpha, p(q), p(cnt),
                                               p(ap), ap.numel(), u_max, p(U), p(err),
                                               ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, maps.status_string(st)
    torch.cuda.synchronize()
    return q.cpu().numpy(), cnt.cpu().numpy(), U.cpu().numpy(), int(err.item())


def _with_workspace(pred, truth, edges, alpha, ap, u_max):
    import torch

    import paper_2609_15359_amd as maps
    q, cnt, U, err = maps.calibrate(pred, truth, edges, alpha, ap, u_max)
    torch.cuda.synchronize()
    return q.cpu().numpy(), cnt.cpu().numpy(), U.cpu().numpy(), int(err.item())


def test_noalloc_matches_workspace_call_twice():
    big = workload.make("large")      # 1,000,000 residuals, 64 buckets, 1.3M bounds
    small = workload.make("small")    # 20,000 residuals, 16 buckets
    for b in (big, small):
        args = (_cuda(b.cal_pred), _cuda(b.cal_truth), _cuda(b.edges), b.alpha_ppm, _cuda(b.apply_pred()), b.u_max)
        got = _noalloc(*args)
        want = _with_workspace(*args)
        assert got[3] == 0 and want[3] == 0
        for name, g, w in zip(("q", "count", "U"), got[:3], want[:3]):
            assert np.array_equal(g, w), name


def test_noalloc_size_limit():
    import torch

    import paper_2609_15359_amd as maps
    lib = maps.library()
    assert lib.maps_calibrate_workspace_size(1 << 20, 1024) <= 8 << 20
    null = ctypes.c_void_p(0)
    # beyond the scratch array: rejected before anything is enqueued (pointers are not read)
    st = lib.maps_calibrate_noalloc(null, null, 1 << 24, null, 1024, 100000, null, null, null, 0, 10, null, null,
                                    ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == -2
