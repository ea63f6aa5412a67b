"""The fp64 oracle against facts other than itself (no GPU)."""
import pytest

import oracle_pins as P
from paper_2608_12629_amd.synth import make_workload, raw_bits


@pytest.mark.parametrize("pin", P.FAST_PINS + P.KNN_PINS, ids=lambda f: f.__name__)
def test_pin(oracle, pin):
    pin(oracle)


def test_pin_sklearn_lloyd(oracle):
    P.pin_sklearn_lloyd(oracle)


# Scaled-down versions of the five workloads (same recipe, smaller N/K) for the
# objective-monotonicity invariant.
SCALED = [
    dict(cfg=1, N=8192, K=64),
    dict(cfg=2, N=8192, K=128),
    dict(cfg=3, N=16384, K=256),
    dict(cfg=4, B=4, N=2048),
    dict(cfg=5, N=2048, K=128),
]


@pytest.mark.parametrize("kw", SCALED, ids=lambda kw: f"cfg{kw['cfg']}")
def test_objective_monotone_on_workloads(oracle, kw):
    kw = dict(kw)
    w = make_workload(kw.pop("cfg"), **kw)
    P.pin_monotone(oracle, [(w, raw_bits(w.X), w.dtype)])
