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
    dict(wl=1, N=8192, K=64),
    dict(wl=2, N=8192, K=128),
    dict(wl=3, N=16384, K=256),
    dict(wl=4, B=4, N=2048),
    dict(wl=5, N=2048, K=128),
]


@pytest.mark.parametrize("kw", SCALED, ids=["blobs_f32", "blobs_bf16", "zipf_bf16", "batched_f16", "subspace_bf16"])
def test_objective_monotone_on_workloads(oracle, kw):
    kw = dict(kw)
    w = make_workload(kw.pop("wl"), **kw)
    P.pin_monotone(oracle, [(w, raw_bits(w.X), w.dtype)])
