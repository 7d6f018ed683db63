"""Pins for the tempo_fast solver (Sec. 4.2) and its candidates, on the CPU:
feasibility, the ensemble's guarantee against the token LP, Theorem 1's
additive bound for the round-robin placement, the beta -> 0 limit (Lemma 2)
against a brute-force semi-matching, near-optimality against a MILP optimum
on tiny instances, and the plan it emits reproducing its shares through the
stage-1 oracle."""
import itertools
import math

import numpy as np
import pytest

import oracle
from paper_2608_13057_amd import solver


def _instance(rng, E, ng, extra, full=False, s=1.1, pairs=None):
    R = np.ones((E, ng), bool) if full else np.zeros((E, ng), bool)
    if not full:
        R[np.arange(E), np.arange(E) % ng] = True
        for e in rng.choice(E, size=min(extra, E), replace=False):
            R[e, rng.integers(0, ng)] = True
    pairs = pairs or int(rng.integers(1, 50 * E))
    n = np.bincount(rng.zipf(s, size=pairs) % E, minlength=E).astype(np.int64)
    return n, R


def _model(rng):
    return solver.CostModel(float(rng.uniform(0, 50)), float(rng.uniform(0.5, 10)), float(rng.uniform(0, 80)),
                            float(rng.uniform(0.01, 0.2)))


def _feasible(x, n, R):
    assert x.dtype.kind == "i" and (x >= 0).all()
    assert np.array_equal(x.sum(axis=1), n)
    assert (x[~R] == 0).all()


@pytest.mark.parametrize("seed", range(30))
def test_candidates_feasible_and_ensemble_guarantee(seed):
    rng = np.random.default_rng(seed)
    n, R = _instance(rng, int(rng.integers(2, 80)), int(rng.integers(1, 9)), int(rng.integers(0, 20)),
                     full=seed % 5 == 0)
    m = _model(rng)
    x, info = solver.tempo_fast(n, R, m, return_info=True)
    for y in (x, solver.token_lp(n, R), solver.uniform_split(n, R), solver.greedy_seed(n, R, m)):
        _feasible(y, n, R)
    ms = solver.makespan(x, m)
    assert ms <= 1.01 * solver.makespan(solver.token_lp(n, R), m) + 1e-9
    assert ms <= info["heuristic"] + 1e-9
    assert ms >= solver.lower_bound(n, R.shape[1], m) - 1e-9
    rr = solver.round_robin(n, R)
    if rr is not None:
        _feasible(rr, n, R)
        assert ms <= 1.01 * solver.makespan(rr, m) + 1e-9


@pytest.mark.parametrize("seed", range(30))
def test_round_robin_additive_bound(seed):
    """Theorem 1 under full replication: M(A3) <= OPT + beta n_max (n_max >=
    b / beta) or + b, checked against a lower bound on OPT."""
    rng = np.random.default_rng(100 + seed)
    n, R = _instance(rng, int(rng.integers(1, 200)), int(rng.integers(1, 17)), 0, full=True)
    m = _model(rng)
    rr = solver.round_robin(n, R)
    lb = solver.lower_bound(n, R.shape[1], m)
    assert solver.makespan(rr, m) <= lb + max(m.b, m.beta * float(n.max())) + 1e-9


@pytest.mark.parametrize("seed", range(25))
def test_activation_limit_is_semi_matching_optimum(seed):
    """beta -> 0 (c = beta = 0): the objective is a + b max_g G_g (Lemma 2);
    the optimum assigns every active expert to one replica -- brute force
    over those assignments on small instances."""
    rng = np.random.default_rng(200 + seed)
    E, ng = int(rng.integers(2, 9)), int(rng.integers(2, 4))
    n, R = _instance(rng, E, ng, int(rng.integers(0, E + 1)), pairs=int(rng.integers(1, 200)))
    m = solver.CostModel(5.0, 3.0, 0.0, 0.0)
    act = np.nonzero(n > 0)[0]
    best = math.inf
    for choice in itertools.product(*[np.nonzero(R[e])[0] for e in act]):
        best = min(best, np.bincount(np.array(choice, dtype=np.int64), minlength=ng).max())
    got = solver.makespan(solver.tempo_fast(n, R, m), m)
    assert got == pytest.approx(m.a + m.b * best)


def _milp_opt(n, R, m):
    from scipy.optimize import Bounds, LinearConstraint, milp

    E, ng = R.shape
    idx = np.argwhere(R)
    k = len(idx)
    # variables: x (k, integer), z (k, binary), T
    nv = 2 * k + 1
    c = np.zeros(nv)
    c[-1] = 1
    rows, lo, hi = [], [], []
    for e in range(E):
        r = np.zeros(nv)
        r[:k][idx[:, 0] == e] = 1
        rows.append(r), lo.append(n[e]), hi.append(n[e])
    for j in range(k):
        r = np.zeros(nv)
        r[j] = 1
        r[k + j] = -n[idx[j, 0]]
        rows.append(r), lo.append(-np.inf), hi.append(0)
    for g in range(ng):
        r = np.zeros(nv)
        r[k:2 * k][idx[:, 1] == g] = m.b
        r[-1] = -1
        rows.append(r), lo.append(-np.inf), hi.append(-m.a)
        r = np.zeros(nv)
        r[:k][idx[:, 1] == g] = m.beta
        r[-1] = -1
        rows.append(r), lo.append(-np.inf), hi.append(-m.c)
    integ = np.r_[np.ones(2 * k), 0]
    ub = np.r_[n[idx[:, 0]].astype(float), np.ones(k), np.inf]
    res = milp(c, constraints=LinearConstraint(np.array(rows), lo, hi), integrality=integ,
               bounds=Bounds(np.zeros(nv), ub), options={"time_limit": 20})
    assert res.success
    return res.fun


def test_near_optimal_on_tiny_instances():
    """Against the MILP optimum (splits allowed) on 40 tiny instances: the
    paper reports a mean ratio of 1.005 and a worst of 1.033 on its traces."""
    rng = np.random.default_rng(300)
    ratios = []
    for _ in range(40):
        E, ng = int(rng.integers(3, 11)), int(rng.integers(2, 5))
        n, R = _instance(rng, E, ng, int(rng.integers(0, E)), pairs=int(rng.integers(5, 400)))
        m = _model(rng)
        opt = _milp_opt(n, R, m)
        ratios.append(solver.makespan(solver.tempo_fast(n, R, m), m) / opt)
    ratios = np.array(ratios)
    print(f"tempo_fast / MILP optimum: mean {ratios.mean():.4f} max {ratios.max():.4f}")
    assert ratios.min() >= 1 - 1e-6
    assert ratios.mean() <= 1.02 and ratios.max() <= 1.10


def test_plan_reproduces_shares_through_stage1():
    """The plan of each GPU, fed to the stage-1 oracle with the batch's ids,
    places exactly x[e, gpu] pairs on the GPU's slots of expert e."""
    rng = np.random.default_rng(400)
    E, ng, K, T = 32, 4, 4, 300
    ids = (rng.zipf(1.2, size=(T, K)) % E).astype(np.int32)
    n = np.bincount(ids.reshape(-1), minlength=E)
    R = np.zeros((E, ng), bool)
    R[np.arange(E), np.arange(E) % ng] = True
    for e in np.argsort(-n)[:6]:
        R[e, (e + 1) % ng] = True
        R[e, (e + 2) % ng] = True
    m = solver.CostModel(30.0, 5.0, 10.0, 0.08)
    x = solver.tempo_fast(n, R, m)
    for gpu in range(ng):
        # the GPU's slots: one per expert it holds, and a second slot for the
        # first of them (two local slots of one expert)
        held = np.nonzero(R[:, gpu])[0]
        se = np.r_[held, held[:1]].astype(np.int32)
        sw, rw, rr = solver.plan_for_gpu(x, se, gpu)
        d = oracle.dispatch(ids, T, E, 16, se, sw, rw, rr)
        for e in held:
            assert d["slot_counts"][se == e].sum() == x[e, gpu], (gpu, e)
