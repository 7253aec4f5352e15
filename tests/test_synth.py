"""The seeded input generators: exactness of the fast paths (no method arithmetic here)."""

import numpy as np

from synth.streams import _zipf_cdf, _zipf_draw, _zipf_guide, last_event_time


def test_guided_zipf_draw_equals_binary_search():
    """The guide-table inverse CDF returns exactly the binary-search ranks."""
    for n_ranks, s in [(1000, 1.2), (200_000, 0.8), (50_000, 1.0), (3, 0.5)]:
        cdf = _zipf_cdf(n_ranks, s)
        g = _zipf_guide(cdf)
        a = _zipf_draw(np.random.default_rng(7), cdf, 300_000)
        b = _zipf_draw(np.random.default_rng(7), cdf, 300_000, g)
        assert np.array_equal(a, b)
        assert a.min() >= 0 and a.max() < n_ranks


def test_last_event_time_matches_direct_scan():
    rng = np.random.default_rng(3)
    src = rng.integers(0, 40, 500)
    dst = rng.integers(0, 40, 500)
    t = np.sort(rng.random(500) * 9).astype(np.float32)
    ref = np.zeros(50, np.float32)
    for e in range(500):
        ref[src[e]] = t[e]
        ref[dst[e]] = t[e]
    assert np.array_equal(last_event_time(src, dst, t, 50), ref)
