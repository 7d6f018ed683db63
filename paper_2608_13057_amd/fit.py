"""Stage 4: the two-piece max-affine cost model of one GPU's MoE block and its
calibration fit.

* Eq. 1:  t = max(a + b*G, c + beta*N)  -- G activated local slots, N pairs.
* Eq. 2:  t = max(a + b*G + b2*(T - G), c + beta*N), T = sum of M-tiles.
* Fit (appendix "Calibration details"): two-piece max-affine regression by
  alternating assignment, at most 50 rounds, ordinary least squares per piece.
  Readings where the paper is silent: start with the points whose N/G is at
  most the median in the flat piece; re-assign each point to the piece with
  the larger prediction (ties to the flat piece); stop when nothing moves and
  keep the run's lowest-SSE iterate; a piece with fewer than two distinct
  regressor rows has slope 0 and the mean as intercept; an empty piece never
  wins a point.  fit_restarts repeats the alternation from every
  single-breakpoint split by N/G (and, for Eq. 2, from the Eq. 1 fit's
  assignment and from the Eq. 1 fit itself with b2 = 0, which Eq. 2
  contains, so Eq. 2 never ends with a larger SSE) and keeps the lowest SSE.
* degenerate(): a fit whose parameters are not a usable profile (a negative
  or undefined a, b, c, beta or b2, or an Eq. 2 fit worse than Eq. 1) is
  reported as such rather than tabulated (the paper reports a negative fitted
  b as a degenerate negative control, Sec. 5.2).
* n* = b / beta (the printed n* of the paper's parameter table is b/beta), and
  n*(G) = (a - c + b G) / (beta G), the per-slot tokens at which G equally
  loaded slots flip from the flat to the linear piece.
* Bootstrap confidence interval of b (resampling points), the paper's
  identifiability check (Sec. 5.2).
* Mixed-regime classifier (Sec. 2.4): a batch is mixed when >= 20% of its
  activated slots are flat (c_s <= n*) and >= 20% of its pairs sit on
  linear slots.
"""
from __future__ import annotations

import numpy as np


def predict(params: dict, G, N, T=None):
    G = np.asarray(G, np.float64)
    N = np.asarray(N, np.float64)
    flat = params["a"] + params["b"] * G
    if params.get("b2") is not None and T is not None:
        flat = flat + params["b2"] * (np.asarray(T, np.float64) - G)
    return np.maximum(flat, params["c"] + params["beta"] * N)


def _ls(X: np.ndarray, y: np.ndarray):
    if len(y) == 0:
        return None
    if len(np.unique(X, axis=0)) < 2:
        coef = np.zeros(X.shape[1])
        coef[0] = y.mean()
        return coef
    return np.linalg.lstsq(X, y, rcond=None)[0]


def fit(G, N, t, T=None, iters: int = 50, init=None, start: dict | None = None) -> dict:
    """Alternating-assignment fit of Eq. 1 (or Eq. 2 when tile counts T are
    given).  Returns a, b, c, beta, (b2), n_star, err_mean, err_max, sse,
    iterations, flat (boolean assignment).  `start` (a, b, c, beta, [b2])
    is a round-0 iterate: it competes for the lowest SSE and its
    larger-piece assignment starts the alternation."""
    G = np.asarray(G, np.float64)
    N = np.asarray(N, np.float64)
    t = np.asarray(t, np.float64)
    tile = T is not None
    Xf = np.stack([np.ones_like(G), G] + ([np.asarray(T, np.float64) - G] if tile else []), axis=1)
    Xl = np.stack([np.ones_like(N), N], axis=1)
    ratio = N / G
    flat = (ratio <= np.median(ratio)) if init is None else np.asarray(init, bool)
    cf = cl = None
    it = 0
    best = None  # the lowest-SSE iterate: (sse, cf, cl, assignment)
    if start is not None:
        cf = np.array([start["a"], start["b"]] + ([start.get("b2") or 0.0] if tile else []), np.float64)
        cl = np.array([start["c"], start["beta"]], np.float64)
        pf, pl = Xf @ cf, Xl @ cl
        flat = pf >= pl
        best = (float(((np.maximum(pf, pl) - t) ** 2).sum()), cf, cl, flat)
    for it in range(1, iters + 1):
        cf = _ls(Xf[flat], t[flat])
        cl = _ls(Xl[~flat], t[~flat])
        pf = Xf @ cf if cf is not None else np.full_like(t, -np.inf)
        pl = Xl @ cl if cl is not None else np.full_like(t, -np.inf)
        sse = float(((np.maximum(pf, pl) - t) ** 2).sum())
        if best is None or sse < best[0]:
            best = (sse, cf, cl, flat)
        new = pf >= pl
        if np.array_equal(new, flat):
            break
        flat = new
    _, cf, cl, flat = best
    nan = float("nan")
    a, b = (float(cf[0]), float(cf[1])) if cf is not None else (nan, nan)
    c, beta = (float(cl[0]), float(cl[1])) if cl is not None else (nan, nan)
    out = dict(a=a, b=b, c=c, beta=beta, b2=(float(cf[2]) if (tile and cf is not None) else None))
    pred = np.maximum(Xf @ cf if cf is not None else -np.inf, Xl @ cl if cl is not None else -np.inf)
    rel = np.abs(pred - t) / t
    out.update(n_star=(b / beta if (cl is not None and beta != 0) else nan), err_mean=float(rel.mean()),
               err_max=float(rel.max()), sse=float(((pred - t) ** 2).sum()), iterations=it, flat=flat)
    return out


def fit_restarts(G, N, t, T=None, iters: int = 50) -> dict:
    """fit() from the median split and from every single-breakpoint split by
    N/G (flat iff N/G <= tau over the distinct ratios, plus all-flat and
    all-linear); for Eq. 2 also from the Eq. 1 fit's assignment and from the
    Eq. 1 fit with b2 = 0.  The lowest-SSE result (ties: the earliest
    start)."""
    G = np.asarray(G, np.float64)
    N = np.asarray(N, np.float64)
    ratio = N / G
    starts = [(None, None)] + [(ratio <= tau, None) for tau in np.unique(ratio)] + [(np.zeros(len(ratio), bool), None)]
    if T is not None:
        e1 = fit_restarts(G, N, t, None, iters)
        starts += [(e1["flat"], None), (None, dict(e1, b2=0.0))]
    best = None
    for init, start in starts:
        r = fit(G, N, t, T, iters, init, start)
        if best is None or r["sse"] < best["sse"]:
            best = r
    return best


def degenerate(params: dict, eq1: dict | None = None) -> str | None:
    """Why a fit is not a usable profile, or None: a negative or undefined a,
    b, c, beta or b2, or (for Eq. 2, given the Eq. 1 fit) a larger SSE than
    Eq. 1, which it contains (b2 = 0)."""
    bad = [k for k in ("a", "b", "c", "beta", "b2") if params.get(k) is not None and not params[k] >= 0]
    if bad:
        return "negative or undefined " + ", ".join(bad)
    if eq1 is not None and params["sse"] > eq1["sse"] * (1 + 1e-9):
        return "SSE above the Eq. 1 fit it contains"
    return None


def n_star_of_G(params: dict, G):
    """Per-slot tokens at which G equally loaded slots reach the linear piece."""
    G = np.asarray(G, np.float64)
    return (params["a"] - params["c"] + params["b"] * G) / (params["beta"] * G)


def bootstrap_b(G, N, t, T=None, reps: int = 1000, seed: int = 0):
    """(p2.5, p50, p97.5) of the fitted b over point resamples."""
    rng = np.random.default_rng(seed)
    G, N, t = map(lambda a: np.asarray(a, np.float64), (G, N, t))
    T = None if T is None else np.asarray(T, np.float64)
    bs = []
    for _ in range(reps):
        i = rng.integers(0, len(t), len(t))
        r = fit(G[i], N[i], t[i], None if T is None else T[i])
        bs.append(r["b"])
    bs = np.array(bs)
    bs = bs[np.isfinite(bs)]
    return tuple(float(v) for v in np.percentile(bs, [2.5, 50, 97.5]))


def mixed_regime(slot_counts, n_star: float, frac: float = 0.2) -> dict:
    """The paper's classifier: >= frac of activated slots flat and >= frac of
    pairs on linear slots."""
    c = np.asarray(slot_counts)
    c = c[c > 0]
    if len(c) == 0:
        return dict(mixed=False, flat_slots=0.0, linear_pairs=0.0)
    flat_slots = float((c <= n_star).mean())
    linear_pairs = float(c[c > n_star].sum() / c.sum())
    return dict(mixed=bool(flat_slots >= frac and linear_pairs >= frac), flat_slots=flat_slots,
                linear_pairs=linear_pairs)
