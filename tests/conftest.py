"""Shared pytest configuration: the `gpu` marker and parity helpers."""
from __future__ import annotations

import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

GOLDEN = os.path.join(ROOT, "tests", "golden")

# Model tolerance per round: |gpu - oracle| <= REL * max(|oracle|, rms(oracle row)).
REL_TOL = 1e-5


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")


def assert_models_close(got, ref, rel=REL_TOL, what="model", mask=None):
    """Elementwise check of fp32 models against the fp64 oracle.

    The floor rms(row) keeps entries that cancel towards zero after mixing
    from demanding a relative accuracy no fp32 computation has.  `mask` (bool,
    same shape) drops entries the caller has shown to be ambiguous.
    """
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    ref2 = ref.reshape(ref.shape[0], -1) if ref.ndim > 1 else ref[None, :]
    rms = np.sqrt(np.mean(ref2 * ref2, axis=1, keepdims=True))
    scale = np.maximum(np.abs(ref2), rms)
    err = np.abs(got.reshape(ref2.shape) - ref2)
    bad = err > rel * scale
    if mask is not None:
        bad &= ~np.asarray(mask).reshape(ref2.shape)
    if bad.any():
        r, c = np.argwhere(bad)[0]
        worst = np.max(err / np.where(scale > 0, scale, 1.0))
        raise AssertionError(
            f"{what}: {int(bad.sum())} of {bad.size} entries off; first at row {r} col {c}: "
            f"got {got.reshape(ref2.shape)[r, c]!r} want {ref2[r, c]!r}; worst rel {worst:.3e}")


@pytest.fixture(scope="session")
def golden_dir():
    return GOLDEN
