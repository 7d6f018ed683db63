"""The stage-4 fit of the package against the oracle's fit (same algorithm,
written independently: vectorised numpy vs. plain loops).  Parameters,
assignment and derived quantities must agree."""
import numpy as np
import pytest

from oracle import fit as ofit
from paper_2608_13057_amd import fit as pfit


def _data(seed, m=60, noise=0.05, tile=False):
    rng = np.random.default_rng(seed)
    G = rng.integers(1, 33, m).astype(float)
    n = rng.choice([1, 8, 32, 64, 100, 128, 129, 200, 256, 512, 1024, 2048], m)
    N = G * n
    T = G * np.ceil(n / 128)
    t = np.array([ofit.cost(g, nn, 30.0, 4.0, 25.0, 0.015, 1.3 if tile else 0.0, tt if tile else None)
                  for g, nn, tt in zip(G, N, T)])
    t = t * (1 + noise * rng.standard_normal(m))
    return G, N, T, t


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("tile", [False, True])
def test_fit_matches_oracle(seed, tile):
    G, N, T, t = _data(seed, tile=tile)
    o = ofit.fit_max_affine(G, N, t, T_tiles=T if tile else None)
    p = pfit.fit(G, N, t, T=T if tile else None)
    keys = ["a", "b", "c", "beta", "n_star", "err_mean", "sse"] + (["b2"] if tile else [])
    for k in keys:
        assert p[k] == pytest.approx(o[k], rel=1e-9, abs=1e-9), k
    assert list(p["flat"].astype(int)) == [1 - v for v in o["assign"]]
    assert p["iterations"] == o["iterations"]


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("tile", [False, True])
def test_restart_fit_matches_oracle(seed, tile):
    G, N, T, t = _data(seed, m=40, noise=0.08, tile=tile)
    o = ofit.fit_restarts(G, N, t, T_tiles=T if tile else None)
    p = pfit.fit_restarts(G, N, t, T=T if tile else None)
    keys = ["a", "b", "c", "beta", "sse"] + (["b2"] if tile else [])
    for k in keys:
        assert p[k] == pytest.approx(o[k], rel=1e-9, abs=1e-9), k
    assert list(p["flat"].astype(int)) == [1 - v for v in o["assign"]]


def test_degenerate_flags():
    good = dict(a=30.0, b=4.0, c=25.0, beta=0.015, b2=None, sse=1.0)
    assert pfit.degenerate(good) is None
    assert "b" in pfit.degenerate(dict(good, b=-1.0))
    assert "beta" in pfit.degenerate(dict(good, beta=float("nan")))
    assert "b2" in pfit.degenerate(dict(good, b2=-0.5))
    assert "Eq. 1" in pfit.degenerate(dict(good, b2=0.1, sse=2.0), eq1=dict(good, sse=1.5))


def test_predict_and_n_star_of_G():
    prm = dict(a=30.0, b=4.0, c=25.0, beta=0.015, b2=None)
    assert pfit.predict(prm, 2, 100) == pytest.approx(ofit.cost(2, 100, 30.0, 4.0, 25.0, 0.015))
    # at n*(G) tokens per slot the two pieces are equal
    G = np.array([1.0, 4.0, 16.0])
    ns = pfit.n_star_of_G(prm, G)
    assert np.allclose(30.0 + 4.0 * G, 25.0 + 0.015 * G * ns)


def test_mixed_regime_classifier():
    # 5 of 6 activated slots flat, 90% of pairs on the linear slot
    r = pfit.mixed_regime([10, 20, 5, 30, 15, 720, 0], n_star=156)
    assert r["mixed"] and r["flat_slots"] == pytest.approx(5 / 6) and r["linear_pairs"] == pytest.approx(0.9)
    assert not pfit.mixed_regime([300, 400], n_star=156)["mixed"]
