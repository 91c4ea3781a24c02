"""The oracle's quantized outputs for seeded workload-shaped tensors against
the SHA-256 digests stored in tests/golden/quant_digests.json (written by the
oracle-only script beside it): a regression fixture for the oracle itself.
The digests are not a second source of truth; the oracle's pins are its
other tests."""
import pytest

from golden import quant_digests as G


@pytest.mark.parametrize("name", list(G.CASES))
def test_oracle_matches_stored_digest(name):
    stored = G.load()["cases"][name]
    fmt, rows, cols, sigma, seed, stream, heavy = G.CASES[name]
    assert (stored["format"], stored["rows"], stored["cols"], stored["seed"], stored["stream"],
            stored["heavy_tail"]) == (fmt, rows, cols, seed, stream, heavy)
    assert G.oracle_digest(name) == stored["sha256"]
