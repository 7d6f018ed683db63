"""Pins for the cost-model oracle (Eq. 1, Eq. 2, the fixed-charge objective
of Sec. 3.1) and the calibration fit (appendix "Calibration details")."""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import fit

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def test_toy_example_makespans():
    """Fig. 1(b): token balancing 105 us, activation balancing 69 us, time
    balancing 60 us, 1.75x, with per-GPU time max(bG, beta N).  b = 105/7 and
    beta = 0.1 follow from the printed numbers (7 floors per GPU under token
    balancing; the 690-token hot GPU under activation balancing)."""
    g = GOLD["toy_example"]
    b, beta = g["token_balancing_us"] / (1 + g["n_cold"]), 0.1
    hot, cold, nc = g["hot_tokens"], g["cold_tokens"], g["n_cold"]
    # token balancing: every expert split in half
    tb = fit.makespan([(1 + nc, (hot + nc * cold) / 2)] * 2, 0, b, 0, beta)
    # activation balancing: whole experts, max G = 4 (hot + 3 cold) vs 3 cold
    ab = fit.makespan([(4, hot + 3 * cold), (3, 3 * cold)], 0, b, 0, beta)
    # time balancing: split only the hot expert
    tm = fit.makespan([(4, hot / 2 + 3 * cold)] * 2, 0, b, 0, beta)
    assert (tb, ab, tm) == pytest.approx((g["token_balancing_us"], g["activation_balancing_us"],
                                          g["time_balancing_us"]))
    assert tb / tm == pytest.approx(g["speedup"])
    # brute force over all whole-or-halved assignments of the 7 experts:
    # the best makespan is the printed time-balanced 60 us
    best = np.inf
    for choice in itertools.product(range(3), repeat=1 + nc):  # 0: GPU0, 1: GPU1, 2: split in half
        G = [0, 0]
        N = [0.0, 0.0]
        for e, c in enumerate(choice):
            n = hot if e == 0 else cold
            if c == 2:
                G = [G[0] + 1, G[1] + 1]
                N = [N[0] + n / 2, N[1] + n / 2]
            else:
                G[c] += 1
                N[c] += n
        best = min(best, fit.makespan(list(zip(G, N)), 0, b, 0, beta))
    assert best == pytest.approx(g["time_balancing_us"])


def test_n_star_is_b_over_beta_in_table():
    for r in GOLD["tab_params"]["rows"]:
        assert r["b"] / r["beta"] == pytest.approx(r["n_star"], rel=0.01)


def test_roofline_bytes():
    g = GOLD["roofline_bytes"]
    assert 3 * g["d_model"] * g["d_ff"] * g["bytes_per_param"] / 1e6 == pytest.approx(g["printed_MB"], abs=0.05)


def _grid(a, b, c, beta, b2=None, M=128):
    G, N, T, t = [], [], [], []
    for g in (1, 2, 4, 8, 16, 32):
        for n in (1, 8, 32, 64, 128, 200, 256, 512, 1024, 2048):
            tiles = g * -(-n // M)
            G.append(g)
            N.append(g * n)
            T.append(tiles)
            t.append(fit.cost(g, g * n, a, b, c, beta, b2 or 0.0, tiles if b2 else None))
    return G, N, T, t


def test_fit_recovers_noise_free_parameters():
    a, b, c, beta = 30.0, 5.0, 20.0, 0.02
    G, N, T, t = _grid(a, b, c, beta)
    r = fit.fit_max_affine(G, N, t)
    assert (r["a"], r["b"], r["c"], r["beta"]) == pytest.approx((a, b, c, beta), rel=1e-9)
    assert r["n_star"] == pytest.approx(b / beta, rel=1e-9)
    assert r["err_mean"] < 1e-10


def test_tile_aware_fit_recovers_b2():
    a, b, b2, c, beta = 35.0, 4.0, 1.3, 34.0, 0.015
    G, N, T, t = _grid(a, b, c, beta, b2)
    r = fit.fit_max_affine(G, N, t, T_tiles=T)
    assert (r["a"], r["b"], r["b2"], r["c"], r["beta"]) == pytest.approx((a, b, b2, c, beta), rel=1e-8)


def test_fit_noisy_is_close():
    rng = np.random.default_rng(0)
    a, b, c, beta = 30.0, 5.0, 20.0, 0.02
    G, N, T, t = _grid(a, b, c, beta)
    t = [v * (1 + 0.03 * rng.standard_normal()) for v in t]
    r = fit.fit_max_affine(G, N, t)
    assert r["b"] == pytest.approx(b, rel=0.15) and r["beta"] == pytest.approx(beta, rel=0.1)


def test_fit_never_beats_brute_force():
    rng = np.random.default_rng(1)
    for trial in range(20):
        m = 9
        G = rng.integers(1, 8, m).astype(float)
        N = G * rng.integers(1, 500, m)
        t = [fit.cost(g, n, 10, 3, 5, 0.05) * (1 + 0.05 * rng.standard_normal()) for g, n in zip(G, N)]
        r = fit.fit_max_affine(G, N, t)
        best = fit.brute_force_best(G, N, t)
        assert r["sse"] >= best - 1e-9 * max(1.0, best)


def test_fit_equals_brute_force_on_separated_data():
    G = [1, 2, 3, 4, 1, 2, 3, 4]
    N = [1, 2, 3, 4, 2000, 4000, 6000, 8000]
    t = [fit.cost(g, n, 10, 3, 5, 0.05) for g, n in zip(G, N)]
    r = fit.fit_max_affine(G, N, t)
    assert r["sse"] == pytest.approx(fit.brute_force_best(G, N, t), abs=1e-9)


def _mostly_flat(seed, m=10):
    """Points of which about 80% sit in the flat regime, so that the median
    split of N/G starts half of the flat points in the linear piece."""
    rng = np.random.default_rng(seed)
    G = rng.integers(1, 9, m).astype(float)
    n = np.where(rng.random(m) < 0.8, rng.integers(1, 60, m), rng.integers(300, 2000, m)).astype(float)
    N = G * n
    t = np.array([fit.cost(g, nn, 40.0, 6.0, 20.0, 0.05) for g, nn in zip(G, N)]) * (1 + 0.03 * rng.standard_normal(m))
    return G, N, t


@pytest.mark.parametrize("seed", range(40))
def test_restarts_bounded_by_brute_force_and_median_start(seed):
    """The restarted fit never beats the exhaustive optimum and never does
    worse than the median start alone."""
    G, N, t = _mostly_flat(seed)
    med = fit.fit_max_affine(G, N, t)
    r = fit.fit_restarts(G, N, t)
    best = fit.brute_force_best(G, N, t)
    assert r["sse"] >= best * (1 - 1e-9)
    assert r["sse"] <= med["sse"] * (1 + 1e-12)


@pytest.mark.parametrize("seed", [3, 38, 40])
def test_restarts_reach_the_optimum_where_the_median_start_does_not(seed):
    """On data where alternation from the median split stops in a worse
    local optimum, one of the single-breakpoint starts reaches the
    exhaustive optimum."""
    G, N, t = _mostly_flat(seed)
    best = fit.brute_force_best(G, N, t)
    assert fit.fit_max_affine(G, N, t)["sse"] > best * 1.01
    assert fit.fit_restarts(G, N, t)["sse"] == pytest.approx(best, rel=1e-9)


def test_run_keeps_its_lowest_sse_iterate():
    """A run capped at one round returns that round's fit; more rounds never
    give a larger SSE than fewer (the lowest-SSE iterate is kept)."""
    G, N, t = _mostly_flat(38)
    prev = None
    for k in range(1, 8):
        r = fit.fit_max_affine(G, N, t, iters=k)
        if prev is not None:
            assert r["sse"] <= prev + 1e-9
        prev = r["sse"]


@pytest.mark.parametrize("seed", range(30))
def test_tile_aware_fit_never_worse_than_eq1(seed):
    """Eq. 2 contains Eq. 1 (b2 = 0), so its restarted fit, which also starts
    from the Eq. 1 fit, never ends with a larger SSE.  Unless that start is
    the winner (not a least-squares fit of any assignment), it never beats
    the exhaustive optimum over Eq. 2's assignments either."""
    G, N, t = _mostly_flat(seed)
    rng = np.random.default_rng(100 + seed)
    T = G * np.ceil(N / G / 64.0) + rng.integers(0, 2, len(G))  # tile counts with some noise
    e1 = fit.fit_restarts(G, N, t)
    e2 = fit.fit_restarts(G, N, t, T)
    assert e2["sse"] <= e1["sse"] * (1 + 1e-12)
    # brute force over the 2^m assignments with the tile regressor in the flat piece
    m = len(t)
    best = np.inf
    for mask in range(1 << m):
        lin = np.array([(mask >> i) & 1 for i in range(m)], bool)
        pf = np.full(m, -np.inf)
        pl = np.full(m, -np.inf)
        if (~lin).any():
            X = np.stack([np.ones(m), G, T - G], 1)[~lin]
            cf = np.linalg.lstsq(X, t[~lin], rcond=None)[0] if len({tuple(r) for r in X.tolist()}) >= 2 else \
                np.array([t[~lin].mean(), 0.0, 0.0])
            pf = cf[0] + cf[1] * G + cf[2] * (T - G)
        if lin.any():
            X = np.stack([np.ones(m), N], 1)[lin]
            cl = np.linalg.lstsq(X, t[lin], rcond=None)[0] if len({tuple(r) for r in X.tolist()}) >= 2 else \
                np.array([t[lin].mean(), 0.0])
            pl = cl[0] + cl[1] * N
        best = min(best, float(((np.maximum(pf, pl) - t) ** 2).sum()))
    if (e2["a"], e2["b"], e2["c"], e2["beta"], e2["b2"]) != (e1["a"], e1["b"], e1["c"], e1["beta"], 0.0):
        assert e2["sse"] >= best * (1 - 1e-9) - 1e-9


def test_start_parameters_are_round_zero():
    """With no alternation rounds the fit returns the start parameters, and
    its SSE is that of the max-affine prediction written out by hand."""
    G = np.array([1.0, 2.0, 4.0, 8.0])
    N = np.array([4.0, 900.0, 40.0, 4000.0])
    T = np.array([1.0, 8.0, 4.0, 64.0])
    t = np.array([50.0, 80.0, 70.0, 260.0])
    p = dict(a=40.0, b=5.0, c=20.0, beta=0.05, b2=1.0)
    r = fit.fit_max_affine(G, N, t, T, iters=0, start=p)
    assert (r["a"], r["b"], r["c"], r["beta"], r["b2"]) == (40.0, 5.0, 20.0, 0.05, 1.0)
    # flat a + bG + b2 (T - G): 45, 56, 60, 136; linear c + beta N: 20.2, 65, 22, 220
    pred = np.array([45.0, 65.0, 60.0, 220.0])
    assert r["sse"] == pytest.approx(float(((pred - t) ** 2).sum()))
    assert r["assign"] == [0, 1, 0, 1]
