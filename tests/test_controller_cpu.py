"""The library's host-side runtime controller (Eq. 6-9) against the oracle's, on the CPU (no GPU call)."""

import os

import numpy as np
import pytest

from oracle import controller as O
from paper_2608_16305_amd import mtgnn as M

pytestmark = pytest.mark.skipif(not os.path.exists(M.LIB_PATH), reason="libmtgnn.so not built")


@pytest.mark.parametrize("seed", range(6))
def test_native_controller_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    cfg = dict(alpha=float(rng.uniform(0.05, 1)), beta=float(rng.uniform(0.05, 1)), tau_g=float(rng.uniform(0.5, 1.2)),
               tau_c=float(rng.uniform(1.0, 2.0)), interval=int(rng.integers(1, 6)))
    nat = M.Controller(**cfg)
    ora = O.Controller(cfg["alpha"], cfg["beta"], cfg["tau_g"], cfg["tau_c"], cfg["interval"])
    g = np.abs(rng.standard_normal(200)) * np.exp(-np.arange(200) / 80)   # decaying gradient norms
    c = 1 + 0.2 * rng.standard_normal(200)
    c[rng.integers(0, 200, 15)] *= 3                                      # load spikes
    c = np.abs(c)
    for r in range(200):
        b, s, h = nat.decide(r)
        assert b == int(ora.boundary(r))
        assert s == (ora.sync(r) if ora.boundary(r) else 0), r
        assert h == ora.heavy(r), r
        nat.observe(g[r], c[r])
        ora.observe(g[r], c[r])
        assert nat.state() == (ora.g_bar, ora.g_last, ora.c_bar, ora.c_prev)


def test_native_controller_rejects_bad_config_and_values():
    with pytest.raises(M.MtgnnError):
        M.Controller(alpha=0.0, beta=0.5, tau_g=1.0, tau_c=1.0, interval=1)
    with pytest.raises(M.MtgnnError):
        M.Controller(alpha=0.5, beta=0.5, tau_g=1.0, tau_c=1.0, interval=0)
    c = M.Controller(alpha=0.5, beta=0.5, tau_g=1.0, tau_c=1.0, interval=2)
    with pytest.raises(M.MtgnnError):
        c.observe(float("nan"), 1.0)
    with pytest.raises(M.MtgnnError):
        c.observe(1.0, -1.0)
