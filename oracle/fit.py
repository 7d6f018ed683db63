"""Oracle for the cost model and its calibration fit (TEST INFRASTRUCTURE ONLY).

* :func:`cost` -- the two-piece max-affine per-GPU cost of Eq. 1,
  t = max(a + b*G, c + beta*N), and the tile-aware form of Eq. 2,
  t = max(a + b*G + b2*(T - G), c + beta*N).
* :func:`makespan` -- the objective of the fixed-charge dispatch problem
  (Sec. 3.1): the maximum over GPUs of the per-GPU cost.
* :func:`fit_max_affine` -- the calibration fit of the appendix "Calibration
  details": two-piece max-affine regression by alternating assignment,
  at most 50 iterations, ordinary least squares per piece.  Written as plain
  loops over the points; the least-squares step uses numpy.linalg.lstsq.

Readings where the paper is silent: the initial assignment puts a point in the
flat piece when its tokens-per-activation N/G is at most the median of N/G;
each point is re-assigned to the piece whose prediction is larger (ties go to
the flat piece); iteration stops when no point changes piece or after 50
rounds, and the run's result is its lowest-SSE iterate; a piece with fewer
than two distinct regressor rows keeps slope 0 and its intercept is the mean;
an empty piece never wins a point.  n* = b/beta.

:func:`fit_restarts` -- the same alternation restarted from every
single-breakpoint split of the points by N/G (flat iff N/G <= tau, for each
distinct tau, and all-flat / all-linear) besides the median split, keeping the
lowest SSE; for the tile-aware form also from the assignment of the Eq. 1 fit
and from the Eq. 1 fit itself taken as a tile-aware fit with b2 = 0 (Eq. 2
contains Eq. 1), so the tile-aware fit never ends with a larger SSE.
"""
from __future__ import annotations

import math

import numpy as np


def cost(G, N, a, b, c, beta, b2=0.0, T=None):
    """Per-GPU cost (Eq. 1, or Eq. 2 when b2 and the tile count T are given)."""
    flat = a + b * G + (b2 * (T - G) if T is not None else 0.0)
    return max(flat, c + beta * N)


def makespan(loads, a, b, c, beta):
    """max over GPUs g of cost(G_g, N_g); loads = [(G_g, N_g), ...]."""
    return max(cost(G, N, a, b, c, beta) for (G, N) in loads)


def _lstsq_piece(X_rows, t_vals):
    """Least squares of t on the regressor rows (first column = 1)."""
    if len(t_vals) == 0:
        return None
    X = np.array(X_rows, dtype=np.float64)
    y = np.array(t_vals, dtype=np.float64)
    coef = np.zeros(X.shape[1])
    distinct = {tuple(r) for r in X.tolist()}
    if len(distinct) < 2:
        coef[0] = float(np.mean(y))
        return coef
    sol, *_ = np.linalg.lstsq(X, y, rcond=None)
    return sol


def fit_max_affine(G, N, t, T_tiles=None, iters: int = 50, init=None, start=None):
    """Alternating-assignment fit.  Returns dict(a, b, c, beta, [b2],
    n_star, err_mean, err_max, sse, iterations, assign).  `start`, when
    given, is a parameter dict (a, b, c, beta, [b2]) taken as round 0: its
    SSE competes for the lowest-SSE iterate and its larger-prediction
    assignment is the initial one."""
    G = [float(v) for v in G]
    N = [float(v) for v in N]
    t = [float(v) for v in t]
    m = len(t)
    tile = T_tiles is not None
    Tt = [float(v) for v in T_tiles] if tile else None
    if init is None:
        ratios = [N[i] / G[i] for i in range(m)]
        med = float(np.median(ratios))
        assign = [0 if ratios[i] <= med else 1 for i in range(m)]  # 0 = flat, 1 = linear
    else:
        assign = list(init)
    cf = cl = None
    it = 0
    best = None  # (sse, cf, cl, assignment that produced them, round)
    if start is not None:
        cf = [start["a"], start["b"]] + ([start.get("b2", 0.0)] if tile else [])
        cl = [start["c"], start["beta"]]
        assign, sse = [], 0.0
        for i in range(m):
            pf = cf[0] + cf[1] * G[i] + (cf[2] * (Tt[i] - G[i]) if tile else 0.0)
            pl = cl[0] + cl[1] * N[i]
            assign.append(0 if pf >= pl else 1)
            sse += (max(pf, pl) - t[i]) ** 2
        best = (sse, np.array(cf, np.float64), np.array(cl, np.float64), list(assign), 0)
    for it in range(1, iters + 1):
        fx, fy, lx, ly = [], [], [], []
        for i in range(m):
            if assign[i] == 0:
                fx.append([1.0, G[i], Tt[i] - G[i]] if tile else [1.0, G[i]])
                fy.append(t[i])
            else:
                lx.append([1.0, N[i]])
                ly.append(t[i])
        cf = _lstsq_piece(fx, fy)
        cl = _lstsq_piece(lx, ly)
        new = []
        sse = 0.0
        for i in range(m):
            pf = -math.inf if cf is None else (cf[0] + cf[1] * G[i] + (cf[2] * (Tt[i] - G[i]) if tile else 0.0))
            pl = -math.inf if cl is None else cl[0] + cl[1] * N[i]
            new.append(0 if pf >= pl else 1)
            sse += (max(pf, pl) - t[i]) ** 2
        if best is None or sse < best[0]:
            best = (sse, cf, cl, list(assign), it)
        if new == assign:
            break
        assign = new
    _, cf, cl, assign, _ = best
    a, b = (float(cf[0]), float(cf[1])) if cf is not None else (float("nan"), float("nan"))
    b2 = float(cf[2]) if (cf is not None and tile) else 0.0
    c, beta = (float(cl[0]), float(cl[1])) if cl is not None else (float("nan"), float("nan"))
    pred = []
    for i in range(m):
        pf = -math.inf if cf is None else a + b * G[i] + (b2 * (Tt[i] - G[i]) if tile else 0.0)
        pl = -math.inf if cl is None else c + beta * N[i]
        pred.append(max(pf, pl))
    rel = [abs(pred[i] - t[i]) / t[i] for i in range(m)]
    out = dict(a=a, b=b, c=c, beta=beta, n_star=(b / beta if beta not in (0.0,) and cl is not None else float("nan")),
               err_mean=float(np.mean(rel)), err_max=float(np.max(rel)),
               sse=float(sum((pred[i] - t[i]) ** 2 for i in range(m))), iterations=it, assign=assign)
    if tile:
        out["b2"] = b2
    return out


def fit_restarts(G, N, t, T_tiles=None, iters: int = 50):
    """fit_max_affine from the median split and from every single-breakpoint
    split by N/G (flat iff N/G <= tau over the distinct ratios, plus
    all-flat and all-linear); with tile counts also from the Eq. 1 fit's
    assignment and from the Eq. 1 fit itself with b2 = 0.  Returns the
    lowest-SSE result (ties: the earliest start)."""
    m = len(t)
    ratios = [float(N[i]) / float(G[i]) for i in range(m)]
    starts = [(None, None)]
    for tau in sorted(set(ratios)) + [-math.inf]:
        starts.append(([0 if ratios[i] <= tau else 1 for i in range(m)], None))
    if T_tiles is not None:
        eq1 = fit_restarts(G, N, t, None, iters)
        starts.append((eq1["assign"], None))
        starts.append((None, dict(eq1, b2=0.0)))
    best = None
    for init, start in starts:
        r = fit_max_affine(G, N, t, T_tiles, iters, init, start)
        if best is None or r["sse"] < best["sse"]:
            best = r
    return best


def brute_force_best(G, N, t):
    """Exhaustive search over all 2^m assignments of points to pieces (m small):
    for each, fit both pieces by least squares and score the max-affine SSE.
    Returns the lowest SSE."""
    m = len(t)
    best = math.inf
    for mask in range(1 << m):
        fx, fy, lx, ly = [], [], [], []
        for i in range(m):
            if (mask >> i) & 1:
                lx.append([1.0, float(N[i])])
                ly.append(float(t[i]))
            else:
                fx.append([1.0, float(G[i])])
                fy.append(float(t[i]))
        cf = _lstsq_piece(fx, fy)
        cl = _lstsq_piece(lx, ly)
        sse = 0.0
        for i in range(m):
            pf = -math.inf if cf is None else cf[0] + cf[1] * G[i]
            pl = -math.inf if cl is None else cl[0] + cl[1] * N[i]
            sse += (max(pf, pl) - t[i]) ** 2
        best = min(best, sse)
    return best
