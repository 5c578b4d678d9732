import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (HIP device visible)")
    config.addinivalue_line("markers", "slow: longer CPU test")


def lane_rel_err(got, want):
    """Elementwise |got - want| / max(|want_p|, max_p |want_p|) per lane, the
    lane-norm scale used for gradient comparisons; non-finite classes must
    agree (the error is then 0) or the error is inf."""
    got = np.atleast_2d(np.asarray(got, dtype=np.float64))
    want = np.atleast_2d(np.asarray(want, dtype=np.float64))
    fin = np.isfinite(want)
    scale = np.max(np.where(fin, np.abs(want), 0.0), axis=1, keepdims=True)
    scale = np.maximum(np.abs(np.where(fin, want, 0.0)), scale)
    err = np.abs(got - want)
    with np.errstate(invalid="ignore", divide="ignore"):
        rel = np.where(scale > 0, err / scale, err)
    same_class = (np.isnan(got) & np.isnan(want)) | (np.isposinf(got) & np.isposinf(want)) | \
        (np.isneginf(got) & np.isneginf(want))
    rel = np.where(fin & np.isfinite(got), rel, np.where(same_class, 0.0, np.inf))
    return rel


def rel_err(got, want):
    """|got - want| / |want| elementwise with matching non-finite classes."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    with np.errstate(invalid="ignore", divide="ignore"):
        r = np.abs(got - want) / np.where(want != 0, np.abs(want), 1.0)
    same_class = (np.isnan(got) & np.isnan(want)) | (np.isposinf(got) & np.isposinf(want)) | \
        (np.isneginf(got) & np.isneginf(want))
    fin = np.isfinite(got) & np.isfinite(want)
    return np.where(fin, r, np.where(same_class, 0.0, np.inf))


@pytest.fixture(scope="session")
def oracle_mod():
    import oracle
    oracle.build(force=False)
    return oracle


def record(name, **fields):
    """Print a parity record and, when NDVM_PARITY_LOG names a file, append
    it there as one JSON line (the GPU runs collect these into a summary)."""
    import json
    rec = dict(test=name, **fields)
    print("PARITY", json.dumps(rec, sort_keys=True), flush=True)
    path = os.environ.get("NDVM_PARITY_LOG")
    if path:
        os.makedirs(os.path.dirname(os.path.abspath(path)), exist_ok=True)
        with open(path, "a") as f:
            f.write(json.dumps(rec, sort_keys=True) + "\n")
