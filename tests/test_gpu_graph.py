"""The step captured as HIP graphs (one per phase) and replayed: every replay,
with eager work and synchronizations between them, gives the eager step's
results bit for bit."""
import numpy as np
import pytest

import workload
from tests.gpu_common import assert_same

pytestmark = pytest.mark.gpu


def _snapshot_all(db, ws):
    pl = ws.placement
    return {"q": ws.out["q"], "count": ws.out["count"], "U": ws.out["U"], "base_peak": ws.base_peak,
            "choice": pl.choice, "chosen_peak": pl.chosen_peak, "chosen_overflow": pl.chosen_overflow,
            "flags": pl.flags, "pair_peak": pl.pair_peak, "order": ws.order, "admitted": ws.admitted}


@pytest.mark.parametrize("fused", [False, True, "project"])
@pytest.mark.parametrize("name", ["small", "medium"])
def test_graph_replays_match_eager(name, fused):
    import torch

    from paper_2609_15359_amd import pipeline
    b = workload.make(name)
    db = pipeline.to_device(b)
    ws = pipeline.Workspaces(db, want_pairs=True)
    pipeline.step(db, ws, fused=fused)
    torch.cuda.synchronize()
    want = {k: v.cpu().numpy().copy() for k, v in _snapshot_all(db, ws).items()}
    assert int(ws.dev_err.item()) == 0

    graphs = pipeline.StepGraphs(db, ws, fused=fused)
    other = pipeline.Workspaces(db, want_pairs=True)   # eager work between replays
    for r in range(3):
        for t in _snapshot_all(db, ws).values():
            t.fill_(-7 if t.dtype != torch.uint8 else 7)
        torch.cuda.synchronize()
        graphs.replay()
        torch.cuda.synchronize()
        got = {k: v.cpu().numpy() for k, v in _snapshot_all(db, ws).items()}
        for k in want:
            assert_same(f"replay {r}: {k}", got[k], want[k])
        pipeline.step(db, other, policy=1, rr_offset=r)
        torch.cuda.synchronize()
    assert int(ws.dev_err.item()) == 0
