"""The C-ABI library builds for gfx950, loads, and exports every entry point
that include/maps.h declares; its host-side argument checks answer without a
GPU (no kernel is launched on any of these paths)."""
import ctypes
import os
import re

import pytest

import paper_2609_15359_amd as maps

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "maps.h")


def declared():
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(maps_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(maps.LIBRARY):
        pytest.fail("libmaps.so is not built; run __graft_entry__.build()")
    return maps.library()


def test_header_declares_the_four_steps():
    names = declared()
    for n in ("maps_calibrate", "maps_project", "maps_place", "maps_local_order"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    raw = ctypes.CDLL(maps.LIBRARY)
    for name in declared():
        assert hasattr(raw, name), name
    assert sorted(maps.EXPORTS) == declared()


def test_library_is_built_for_gfx950():
    with open(maps.LIBRARY, "rb") as f:
        blob = f.read()
    assert b"gfx950" in blob


def test_size_queries(lib):
    # header 256 B + D decoder headers + D*P profile entries + per decoder a
    # slice of W/2 16-byte units of rank words and at most n_d + 3 units of
    # event arrays + 64 spare units; P = 0 once u_max + 1 > 16384
    def want(D, n, u_max):
        W = (((u_max + 1) // 32 + 1) + 1) & ~1
        P = (u_max + 4) & ~3 if u_max + 1 <= 16384 else 0
        a = lambda x: (x + 255) // 256 * 256
        return 256 + a(D * 64) + a(D * P * 4) + (n + D * (3 + W // 2) + 64) * 16
    D, n = 4, 100
    for u_max in (0, 1, 8192, 16383, 16384, 65535):
        assert lib.maps_snapshot_bytes(D, n, u_max) == want(D, n, u_max), u_max
    assert lib.maps_snapshot_bytes(0, n, u_max) == 0
    assert lib.maps_snapshot_bytes(D, n, (1 << 24) - 63) == 0
    assert lib.maps_snapshot_bytes(D, n, (1 << 24) - 64) > 0
    # scores in bucket order (4 B per residual) up to 1,024 buckets, scores and
    # bucket ids (6 B per residual) beyond
    assert lib.maps_calibrate_workspace_size(1000, 4) >= 1000 * 4
    assert lib.maps_calibrate_workspace_size(1000, 2000) >= 1000 * 6
    assert lib.maps_place_workspace_size(256, 262144, 32768) >= 262144 * 12
    assert lib.maps_project_workspace_size(4, 100, 8192) == 0
    assert lib.maps_local_order_workspace_size(4, 100) == 0


def test_status_strings(lib):
    assert maps.status_string(0) == "ok"
    assert "alpha" in maps.status_string(-3)
    assert maps.status_string(-99) == "unknown status"


def _v(x):
    return ctypes.c_void_p(x)


def test_host_argument_errors_without_gpu(lib):
    """Invalid sizes, alpha, policy, NULL pointers and short buffers are refused
    synchronously, before anything is enqueued."""
    fake = _v(0x1000)  # never dereferenced: every call below fails its host checks
    # calibrate: alpha outside (0, 1e6), nb < 1, n < 0, NULL outputs
    assert lib.maps_calibrate(fake, fake, 10, fake, 2, 0, fake, fake, None, 0, 10, None, fake, fake, 1 << 20, None) == -3
    assert lib.maps_calibrate(fake, fake, 10, fake, 2, 1000000, fake, fake, None, 0, 10, None, fake, fake, 1 << 20, None) == -3
    assert lib.maps_calibrate(fake, fake, 10, fake, 0, 100000, fake, fake, None, 0, 10, None, fake, fake, 1 << 20, None) == -2
    assert lib.maps_calibrate(fake, fake, -1, fake, 2, 100000, fake, fake, None, 0, 10, None, fake, fake, 1 << 20, None) == -2
    assert lib.maps_calibrate(fake, fake, 10, fake, 2, 100000, None, fake, None, 0, 10, None, fake, fake, 1 << 20, None) == -1
    assert lib.maps_calibrate(fake, fake, 10, fake, 2, 100000, fake, fake, None, 0, 10, None, fake, fake, 8, None) == -4
    # project: D < 1, u_max too large, short snapshot buffer
    assert lib.maps_project(0, fake, 0, fake, fake, fake, 10, fake, 1 << 20, fake, fake, None, 0, None) == -2
    assert lib.maps_project(1, fake, 0, fake, fake, fake, 1 << 24, fake, 1 << 20, fake, fake, None, 0, None) == -2
    assert lib.maps_project(4, fake, 100, fake, fake, fake, 8192, fake, 64, fake, fake, None, 0, None) == -7
    assert lib.maps_project(4, None, 100, fake, fake, fake, 8192, fake, 1 << 20, fake, fake, None, 0, None) == -1
    # place: policy, negative rr_offset, NULL outputs
    args = [fake, 4, 8192, fake, fake, fake, fake, 10]
    assert lib.maps_place(*args, 7, 0, fake, fake, fake, fake, None, fake, fake, 1 << 20, None) == -6
    assert lib.maps_place(*args, 0, -1, fake, fake, fake, fake, None, fake, fake, 1 << 20, None) == -2
    assert lib.maps_place(*args, 0, 0, None, fake, fake, fake, None, fake, fake, 1 << 20, None) == -1
    # local order: D < 1, NULL queue offsets
    assert lib.maps_local_order(fake, 0, 10, fake, fake, 0, fake, fake, None, 0, fake, fake, fake, None, 0, None) == -2
    assert lib.maps_local_order(fake, 2, 10, fake, None, 0, fake, fake, None, 0, fake, fake, fake, None, 0, None) == -1
    # placement with local order: either argument set refused, nothing enqueued
    po = [fake, 4, 8192, fake, fake, fake, fake, 10]
    tail = [fake, 5, fake, fake, fake, 1000, fake, fake, fake, fake, 1 << 20, None]
    assert lib.maps_place_order(*po, 7, 0, fake, fake, fake, fake, None, *tail) == -6
    assert lib.maps_place_order(*po, 0, 0, fake, fake, fake, fake, None, None, *tail[1:]) == -1
    assert lib.maps_place_order(*po, 0, 0, fake, fake, fake, fake, None, fake, -1, *tail[2:]) == -2
    # sliding-window calibration: window and bucket limits, alpha, NULL, short workspace
    wa = lambda n, nb, w, a, ws: lib.maps_calibrate_window(fake, fake, n, fake, nb, w, a, fake, fake, 10, 100,
                                                         None, fake, fake, fake, ws, None)
    assert wa(100, 4, 0, 100000, 1 << 24) == -2
    assert wa(100, 4, maps.MAX_WINDOW + 1, 100000, 1 << 24) == -2
    assert wa(100, maps.MAX_WINDOW_BUCKETS + 1, 500, 100000, 1 << 24) == -2
    assert wa(-1, 4, 500, 100000, 1 << 24) == -2
    assert wa(2**31, 4, 500, 100000, 1 << 24) == -2
    assert wa(100, 4, 500, 0, 1 << 24) == -3
    assert wa(100, 4, 500, 100000, 16) == -4
    assert lib.maps_calibrate_window(fake, fake, 100, fake, 4, 500, 100000, fake, None, 10, 100, None, fake, fake,
                                     fake, 1 << 24, None) == -1
    # the workspace holds the scores three times over (grouped, by bucket, and their
    # log indices) plus a quantile per position of every bucket
    assert lib.maps_calibrate_window_workspace_size(100000, 64) >= 100000 * 18
    # byte capacities: D < 1, bytes per token < 1, NULL
    assert lib.maps_capacity_tokens(fake, 0, 131072, fake, fake, None) == -2
    assert lib.maps_capacity_tokens(fake, 4, 0, fake, fake, None) == -2
    assert lib.maps_capacity_tokens(None, 4, 131072, fake, fake, None) == -1
    assert lib.maps_capacity_tokens(fake, 4, 131072, fake, None, None) == -1


def test_binding_refuses_host_tensors(lib):
    import torch
    x = torch.zeros(4, dtype=torch.int32)
    with pytest.raises(maps.MapsError):
        maps.calibrate(x, x, torch.zeros(1, dtype=torch.int32), 100000)
