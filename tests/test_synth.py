"""The seeded generator draws what its recipe says (shapes, dtypes, ranges,
structure), and its method-free codebook spread matches the residual spread
the oracle actually sees."""
import numpy as np
import pytest

from oracle import codec
from paper_2606_05484_amd import synth


def test_c1_shapes_and_dtypes():
    x = synth.codec_inputs("c1")
    assert x["X"].shape == (512, 256) and x["X"].dtype == np.float32
    assert x["U"].shape == (256, 32) and x["U"].dtype == np.float32
    assert x["A"].shape == (1024, 16) and x["B"].shape == (16, 256)
    assert x["C"].shape == (2, 64, 32)
    assert np.all(x["C"][:, 0] == 0)
    assert x["ids"].dtype == np.int32 and x["ids"].min() >= 0 and x["ids"].max() < 1024
    U = x["U"].astype(np.float64)
    assert np.abs(U.T @ U - np.eye(32)).max() < 1e-6
    assert abs(x["C"][:, 1:].std() - 0.02) < 2e-3


def test_determinism():
    a = synth.codec_inputs("c1")
    b = synth.codec_inputs("c1")
    for key in ("X", "U", "A", "B", "ids", "C", "dXhat", "dZ", "G"):
        assert np.array_equal(a[key], b[key])


def test_zipf_head_mass():
    rng = np.random.default_rng(0)
    ids = synth.zipf_ids(rng, 32000, 200000)
    p = 1.0 / np.arange(1, 32001) ** 1.1
    p /= p.sum()
    # id 0 frequency matches the finite-support Zipf(1.1) mass within 3 sigma
    f0 = np.mean(ids == 0)
    assert abs(f0 - p[0]) < 3 * np.sqrt(p[0] * (1 - p[0]) / ids.size)
    assert ids.max() < 32000


def test_bf16_storage_roundtrip():
    x = synth.codec_inputs("c3")
    assert x["X"].dtype == np.uint16 and x["X"].shape == (8192, 1024)
    v = synth.as_f64(x["X"], "bf16")
    assert np.isfinite(v).all()
    assert 0.05 < np.sqrt(np.mean(v ** 2)) < 1.0


@pytest.mark.parametrize("name", ["c3"])
def test_codebook_sigma_matches_oracle_residual_spread(name):
    """Reading of 'N(0, residual-std per stage)': sigma_l = rms(X) for every
    stage.  The per-coordinate rms of the oracle's actual residual before each
    stage must agree within 10%."""
    x = synth.codec_inputs(name)
    X = synth.as_f64(x["X"], "bf16")
    A = synth.as_f64(x["A"], "bf16")
    B = synth.as_f64(x["B"], "bf16")
    codes, _, rs = codec.encode(X, x["ids"], x["U"], A, B, x["C"], operand="bf16")
    for l in range(x["L"]):
        rms = np.sqrt(rs[:, l].mean() / x["r"])
        assert abs(rms / x["cb_sigma"] - 1) < 0.10, (l, rms, x["cb_sigma"])
