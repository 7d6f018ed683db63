"""Stage 4: profiling harness for the per-GPU MoE block on MI355X.

Reproduces the paper's calibration protocol (appendix "Calibration details",
Sec. 2.2): a grid over activated slots G and tokens per slot n, each point
timed as the median of 30 back-to-back executions with the expert weights
rotated between executions so no replay finds them in the 256 MB Infinity
Cache, with the tile configuration fixed; then the max-affine fit of Eq. 1
(and Eq. 2 with the tile term) and the inflection n*.

Workload of a point (G, n): G local slots holding G distinct experts, T = G*n
token rows routed top-1 so that slot s receives exactly n pairs; the plan has
one replica per expert.  Two scopes are timed: "gemm" (stage 2 only: the two
grouped GEMMs) and "block" (stages 1-3).

    python -m paper_2608_13057_amd.profile --dtype bf16 --out sweep.jsonl
    python -m paper_2608_13057_amd.profile --from-jsonl sweep.jsonl --md summary.md --command "..."
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

QWEN = dict(H=4096, I=1536)
SHAPES = {"qwen3": QWEN, "dsv3": dict(H=7168, I=2048),  # expert shapes of the paper's two models
          "tiny": dict(H=256, I=512)}  # the tiny parity shape (harness tests)
DEFAULT_G = tuple(range(1, 33))
DEFAULT_N = (1, 2, 4, 8, 16, 32, 48, 64, 96, 128, 129, 160, 192, 256, 257, 320, 384, 512, 768, 1024, 2048)
POOL_SLOTS = 32


def _log(msg):
    print(f"[profile] {msg}", file=sys.stderr, flush=True)


class Harness:
    """Device state for a sweep: a pool of POOL_SLOTS packed slot weights and
    the timing machinery."""

    def __init__(self, dtype="bf16", H=QWEN["H"], I=QWEN["I"], m_tile=128, seed=0, max_tokens=65536):
        import torch

        from . import moe, synth

        self.torch, self.moe = torch, moe
        self.dtype, self.H, self.I, self.m_tile = dtype, H, I, m_tile
        se = np.arange(POOL_SLOTS, dtype=np.int32)
        t0 = time.perf_counter()
        w13, s13, w2, s2 = synth.slot_weights(se, H, I, seed, dtype)
        td = moe.to_device
        pool_shape = moe.MoEShape(T=1, K=1, E=POOL_SLOTS, S=POOL_SLOTS, H=H, I=I, m_tile=m_tile, dtype=dtype)
        nat = moe.WeightTensors(td(w13), td(w2), None if s13 is None else td(s13), None if s2 is None else td(s2))
        self.pool = moe.pack_weights(pool_shape, nat)
        del nat
        x, xs = synth.activations(max_tokens, H, 1, dtype)
        self.x, self.xs = td(x), (None if xs is None else td(xs))
        self.max_tokens = max_tokens
        torch.cuda.synchronize()
        _log(f"weight pool of {POOL_SLOTS} slots ready in {time.perf_counter() - t0:.1f} s")
        self.spin = self._calibrate_spin()

    def _calibrate_spin(self, target_ms=10.0):
        torch = self.torch
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        n = 1 << 20
        for _ in range(6):
            torch.cuda.synchronize()
            a.record()
            torch.cuda._sleep(n)
            b.record()
            torch.cuda.synchronize()
            ms = a.elapsed_time(b)
            if ms >= 1.0:
                break
            n *= 8
        return int(n * target_ms / max(ms, 1e-3))

    def weights_at(self, off: int, G: int):
        """Slots [off, off+G) of the pool as a G-slot weight set (views)."""
        p = self.pool
        return self.moe.WeightTensors(p.w13[off:off + G], p.w2[off:off + G],
                                      None if p.w13_scale is None else p.w13_scale[off:off + G],
                                      None if p.w2_scale is None else p.w2_scale[off:off + G])

    def point(self, G: int, n: int, reps: int = 30, scopes=("gemm", "block")) -> list[dict]:
        torch, moe = self.torch, self.moe
        T = G * n
        shape = moe.MoEShape(T=T, K=1, E=G, S=G, H=self.H, I=self.I, m_tile=self.m_tile, dtype=self.dtype)
        ids = (np.arange(T, dtype=np.int32) // n).reshape(T, 1)
        td = moe.to_device
        assert T <= self.max_tokens
        d_ids, d_w, d_x = td(ids), td(np.ones((T, 1), np.float32)), self.x[:T]
        d_xs = None if self.xs is None else self.xs[:T]
        plan = moe.PlanTensors(td(np.arange(G, dtype=np.int32)), td(np.ones(G, np.uint32)),
                               td(np.zeros(G, np.uint32)), td(np.zeros(G, np.int32)))
        ws = moe.Workspace(shape)
        disp = moe.DispatchBuffers.allocate(shape, ws.row_cap)
        y = torch.empty(T, self.H, dtype=torch.int16, device="cuda")
        y_perm = torch.empty(ws.row_cap, self.H, dtype=torch.int16, device="cuda")
        offs = list(range(0, POOL_SLOTS - G + 1, max(1, G))) or [0]
        wsets = [self.weights_at(o, G) for o in offs]
        fwd = [moe.PreparedForward(shape, plan, d_ids, d_w, d_x, d_xs, w, disp, y, ws) for w in wsets]
        # stage 1 once so that stage 2 alone has its inputs, with the per-slot
        # spans of its stage 2 (the library's per-slot timings)
        spans = torch.zeros(G, dtype=torch.int64, device="cuda")
        moe.forward(shape, plan, d_ids, d_w, d_x, d_xs, wsets[0], disp, y, ws, slot_time_ns=spans)
        torch.cuda.synchronize()
        sc = disp.slot_counts.cpu().numpy()
        slot_us = (spans.cpu().numpy() / 1e3).round(3).tolist()
        assert int(sc.sum()) == T and int((sc > 0).sum()) == G, "sweep routing did not land as constructed"
        tiles = int(sum(-(-int(c) // self.m_tile) for c in sc))
        rows = []
        for scope in scopes:
            evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
            for e in evs:
                e[0].record()
                e[1].record()
            for i in range(3):  # warm-up
                if scope == "gemm":
                    moe.experts(shape, disp, wsets[i % len(wsets)], y_perm, ws)
                else:
                    fwd[i % len(fwd)]()
            torch.cuda.synchronize()
            torch.cuda._sleep(self.spin)
            for i in range(reps):
                evs[i][0].record()
                if scope == "gemm":
                    moe.experts(shape, disp, wsets[i % len(wsets)], y_perm, ws)
                else:
                    fwd[i % len(fwd)]()
                evs[i][1].record()
            torch.cuda.synchronize()
            ts = np.array([a.elapsed_time(b) * 1e3 for a, b in evs])
            rows.append(dict(dtype=self.dtype, H=self.H, I=self.I, m_tile=self.m_tile, scope=scope, G=G, n=n,
                             N=T, tiles=tiles, t_us=float(np.median(ts)), p10=float(np.percentile(ts, 10)),
                             p90=float(np.percentile(ts, 90)), reps=reps, rotation_sets=len(wsets),
                             slot_counts=sc.tolist(), slot_span_us=slot_us))
        del fwd, wsets, disp, ws, y, y_perm
        return rows


def run_sweep(dtype="bf16", m_tile=128, Gs=DEFAULT_G, ns=DEFAULT_N, single_slot_ns=(), out=None, reps=30, shape="qwen3"):
    h = Harness(dtype=dtype, m_tile=m_tile, max_tokens=max(max(Gs) * max(ns), max(single_slot_ns, default=1)),
                **SHAPES[shape])
    rows = []
    f = open(out, "a") if out else None
    pts = [(G, n) for G in Gs for n in ns] + [(1, n) for n in single_slot_ns]
    t0 = time.perf_counter()
    for k, (G, n) in enumerate(pts):
        r = h.point(G, n, reps=reps if (G, n) not in set((1, m) for m in single_slot_ns) else min(reps, 10))
        rows += r
        if f:
            for x in r:
                f.write(json.dumps(x) + "\n")
            f.flush()
        if k % 20 == 0:
            _log(f"{k + 1}/{len(pts)} G={G} n={n} " + " ".join(f"{x['scope']}={x['t_us']:.1f}us" for x in r)
                 + f" ({time.perf_counter() - t0:.0f} s)")
    if f:
        f.close()
    return rows


def summarize(rows, scope="gemm") -> dict:
    """Fit Eq. 1 and Eq. 2 on the grid rows of one scope."""
    from . import fit as F

    R = [r for r in rows if r["scope"] == scope]
    G = np.array([r["G"] for r in R], np.float64)
    N = np.array([r["N"] for r in R], np.float64)
    T = np.array([r["tiles"] for r in R], np.float64)
    t = np.array([r["t_us"] for r in R], np.float64)
    e1 = F.fit_restarts(G, N, t)
    e2 = F.fit_restarts(G, N, t, T=T)
    ci = F.bootstrap_b(G, N, t, reps=200)
    clean = lambda d: {k: v for k, v in d.items() if k != "flat"}
    # where Eq. 1's error sits: its mean relative error on the points of each
    # piece, beside the spread of the repetitions themselves
    rel = np.abs(F.predict(e1, G, N) - t) / t
    flat = np.asarray(e1["flat"], bool)
    spread = np.array([(r["p90"] - r["p10"]) / r["t_us"] for r in R])
    pieces = dict(flat_points=int(flat.sum()), flat_err=float(rel[flat].mean()) if flat.any() else float("nan"),
                  linear_points=int((~flat).sum()),
                  linear_err=float(rel[~flat].mean()) if (~flat).any() else float("nan"),
                  rep_spread=float(spread.mean()))
    return dict(scope=scope, points=len(R), eq1=clean(e1), eq2=clean(e2), b_ci95=ci, eq1_pieces=pieces,
                degenerate1=F.degenerate(e1), degenerate2=F.degenerate(e2, e1))


def markdown(rows, title: str, command: str, ns=DEFAULT_N) -> str:
    """A summary of a sweep: the fits of Eq. 1 / Eq. 2 per scope, the grid of
    stage-2 times, and the single-slot staircase (every 16th point)."""
    grid = [r for r in rows if not (r["G"] == 1 and r["n"] not in ns)]
    out = [f"# Stage-4 profile: {title}", "", "Commands (repo root, MI355X):", "", "```", command, "```", ""]
    for scope in ("gemm", "block"):
        if not any(r["scope"] == scope for r in grid):
            continue
        sm = summarize(grid, scope)
        out += [f"## Fit, scope `{scope}` ({sm['points']} grid points)", "",
                "| model | a (us) | b (us/slot) | c (us) | beta (us/token) | b2 (us/extra tile) | n* = b/beta | mean rel. err | "
                "max rel. err | rounds |", "|---|---|---|---|---|---|---|---|---|---|"]
        fits = []
        for k, dk, lab in (("eq1", "degenerate1", "Eq. 1"), ("eq2", "degenerate2", "Eq. 2 (tiles)")):
            e = sm[k]
            if sm[dk]:
                out.append(f"| {lab} | degenerate: {sm[dk]} | | | | | | {e['err_mean']:.3f} | {e['err_max']:.3f} | "
                           f"{e['iterations']} |")
                continue
            b2 = "" if e.get("b2") is None else f"{e['b2']:.3f}"
            out.append(f"| {lab} | {e['a']:.2f} | {e['b']:.3f} | {e['c']:.2f} | {e['beta']:.5f} | {b2} | "
                       f"{e['n_star']:.1f} | {e['err_mean']:.3f} | {e['err_max']:.3f} | {e['iterations']} |")
            fits.append(dict(scope=scope, model=lab, **{x: e[x] for x in ("a", "b", "c", "beta", "n_star", "err_mean",
                                                                           "err_max")},
                             **({"b2": e["b2"]} if e.get("b2") is not None else {})))
        lo, med, hi = sm["b_ci95"]
        pc = sm["eq1_pieces"]
        out += ["", f"Bootstrap 95% interval of b: {lo:.3f} .. {hi:.3f} us (median {med:.3f}).", "",
                f"Eq. 1 mean relative error on the {pc['flat_points']} points of its flat piece "
                f"{pc['flat_err']:.3f}, on the {pc['linear_points']} of its linear piece {pc['linear_err']:.3f}; "
                f"mean spread of the repetitions (p90 - p10) / median {pc['rep_spread']:.3f}.", ""]
        out += ["fit_json: " + json.dumps(f) for f in fits] + [""]
    g = sorted({r["G"] for r in grid})
    nn = sorted({r["n"] for r in grid})
    t = {(r["G"], r["n"]): r["t_us"] for r in grid if r["scope"] == "gemm"}
    out += ["## Stage-2 time (us), median of the repetitions", "", "| n \\ G | " + " | ".join(map(str, g)) + " |",
            "|---" * (len(g) + 1) + "|"]
    for n in nn:
        out.append(f"| {n} | " + " | ".join(f"{t[(G, n)]:.1f}" if (G, n) in t else "" for G in g) + " |")
    fine = sorted((r["n"], r["t_us"], r["tiles"]) for r in rows if r["G"] == 1 and r["scope"] == "gemm" and r["n"] not in ns)
    if fine:
        out += ["", "## Single slot, n = 1..2048 (every 16th point; the tile staircase of Eq. 2)", "",
                "| n | tiles | stage-2 us |", "|---|---|---|"]
        out += [f"| {n} | {tl} | {tu:.1f} |" for n, tu, tl in fine[::16]]
    out.append("")
    return "\n".join(out)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--dtype", default="bf16")
    ap.add_argument("--m-tile", type=int, default=128)
    ap.add_argument("--shape", default="qwen3", choices=sorted(SHAPES), help="expert shape (H, I)")
    ap.add_argument("--out", default=None)
    ap.add_argument("--reps", type=int, default=30)
    ap.add_argument("--quick", action="store_true", help="small grid")
    ap.add_argument("--fine", action="store_true", help="add the single-slot sweep n = 1..2048")
    ap.add_argument("--from-jsonl", default=None, help="summarise an earlier sweep instead of running one")
    ap.add_argument("--md", default=None, help="write a markdown summary here (after a sweep or with --from-jsonl)")
    ap.add_argument("--title", default="")
    ap.add_argument("--command", default="")
    args = ap.parse_args()
    if args.from_jsonl:
        with open(args.from_jsonl) as fh:
            rows = [json.loads(l) for l in fh if l.strip()]
        md = markdown(rows, args.title or f"{rows[0]['dtype']}, M-tile {rows[0]['m_tile']}", args.command)
        if args.md:
            with open(args.md, "w") as fh:
                fh.write(md)
        print(md)
        return
    Gs, ns = (DEFAULT_G, DEFAULT_N) if not args.quick else ((1, 4, 16), (1, 64, 128, 129, 512, 2048))
    fine = tuple(range(1, 2049)) if args.fine else ()
    rows = run_sweep(args.dtype, args.m_tile, Gs, ns, fine, args.out, args.reps, args.shape)
    if args.md:
        # the summary carries the exact command that produced it
        cmd = "python -m paper_2608_13057_amd.profile " + " ".join(sys.argv[1:])
        md = markdown(rows, args.title or f"{args.shape} {args.dtype}, M-tile {args.m_tile}", cmd, ns)
        with open(args.md, "w") as fh:
            fh.write(md)
    res = {s: summarize([r for r in rows if not (r["G"] == 1 and r["n"] not in ns)], s) for s in ("gemm", "block")}
    print(json.dumps(dict(dtype=args.dtype, m_tile=args.m_tile, fits=res), default=str))


if __name__ == "__main__":
    main()
