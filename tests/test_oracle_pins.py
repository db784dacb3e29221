"""The CPU oracle against hand-worked examples, closed forms, invariants and
brute force (no GPU)."""
import pytest

import oracle
from tests import oracle_pins as pins


@pytest.fixture(scope="module")
def o():
    return oracle.Oracle()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(o, pin):
    pin(o)


def test_oracle_step_runs_on_every_small_workload(o):
    import workload
    for name in ("tiny", "small", "medium"):
        b = workload.make(name)
        r = oracle.step(b, o, want_pairs=False)
        assert r.place.choice.min() >= 0 and r.place.choice.max() < b.decoders
        assert r.order.size == b.q_prompt.size
