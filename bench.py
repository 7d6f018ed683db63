#!/usr/bin/env python3
"""Benchmark: one GPU's share of the expert-parallel MoE block (TEMPO).

A step is one pass of the whole block -- stage 1 dispatch (counts, plan split,
M-tile padded permute), stage 2 grouped expert FFN (gate/up + SwiGLU, down)
and stage 3 combine -- over one synthetic batch already resident in HBM.
Default workload: the Qwen3-235B-shaped prefill share (18 local slots = 16
home experts of 128 + 2 replicas of the hottest experts homed elsewhere,
H 4096, I 1536, 8192 tokens, top-8, Zipf(1.0) popularity, uniform plan) in
fp8 e4m3 with power-of-two (UE8M0) block scales, the largest configuration;
almost every slot is in the linear (compute-bound) regime of the cost model.
The same share in bf16 is measured beside it (`roofline_bf16`).

Prints ONE JSON line: the block time (us/batch, lower is better), the
roofline of the dominant kernel (the gate/up GEMM: MFMA-bound at prefill,
HBM-bound at decode), the same for the bf16 prefill share and for two
flat-regime decode shares (`roofline_flat`: the Qwen3 share, 512 tokens,
mixed regime; `roofline_flat_dsv3`: the DeepSeek-V3 share, 256 tokens, most
slots weight-streaming), with `--linear` stage 2 at a grid point where every
slot is in the linear regime (`roofline_linear`: 32 slots of 1024 rows,
UE8M0 fp8), the fitted max-affine profile (a, b, c, beta, n*) of each one's
dtype and M-tile, per-stage times, and the CPU oracle timed on the host
cores as a baseline.

    python bench.py [--gpus 1] [--steps 20] [--warmup 20] [--workload NAME] [--no-flat] [--no-bf16]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp8": 5000.0, "fp8mx": 5000.0}  # dense


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="qwen3_prefill_fp8mx")
    ap.add_argument("--bf16-workload", default="qwen3_prefill_bf16",
                    help="the same share in bf16, measured beside the headline for roofline_bf16")
    ap.add_argument("--no-bf16", action="store_true")
    ap.add_argument("--flat-workload", default="qwen3_decode_bf16",
                    help="the weight-streaming (decode) share measured beside the headline for roofline_flat")
    ap.add_argument("--flat2-workload", default="dsv3_decode_fp8",
                    help="a second weight-streaming share (most slots far below n*) for roofline_flat_dsv3")
    ap.add_argument("--no-flat", action="store_true")
    ap.add_argument("--linear", action="store_true",
                    help="add the linear-regime grid point (32 slots of 1024 rows, UE8M0 fp8, 256-row tiles); off by "
                         "default: it runs the headline's gate/up kernel on another workload, which would mix into "
                         "that kernel's average in a kernel trace of the same command")
    ap.add_argument("--plan", default=None)
    ap.add_argument("--m-tile", type=int, default=0, help="0: 64 for decode-sized batches, 128 above, 256 for bf16 beyond 128 rows per expert")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copies", type=int, default=0, help="weight copies rotated per step (0 = auto)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    return ap.parse_args()


def gemm_bytes(wl, dtype, G, N, which):
    """Algorithmic HBM bytes of one launch of a stage-2 GEMM: the weights of
    the G activated slots once, the N real activation rows in, the N real
    output rows out (padding rows and re-reads are not counted)."""
    H, I = wl.H, wl.I
    ew = 2 if dtype == "bf16" else 1
    if which == "gateup":
        w = 2 * I * H * ew + (0 if dtype == "bf16" else (2 * I // 128) * (H // 128) * 4)
        a = H * ew + (0 if dtype == "bf16" else H // 128 * 4)
        o = I * ew + (0 if dtype == "bf16" else I // 128 * 4)
    else:
        w = H * I * ew + (0 if dtype == "bf16" else (H // 128) * (I // 128) * 4)
        a = I * ew + (0 if dtype == "bf16" else I // 128 * 4)
        o = H * 2
    return G * w + N * (a + o)


def gemm_flops(wl, N, which):
    """Useful flops (padding rows excluded): 2 * N * K * Nout."""
    return 2.0 * N * wl.H * (2 * wl.I if which == "gateup" else wl.I)


def calibrate_spin(torch, target_ms=15.0):
    """Argument of torch.cuda._sleep that keeps the GPU busy ~target_ms."""
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


def attainable_copy_gbs(torch, spin, nbytes=2 << 30):
    """HBM bandwidth of a plain device-to-device copy of nbytes (read +
    write counted), the attainable reference next to the 8 TB/s peak."""
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    torch.cuda._sleep(spin)
    a.record()
    for _ in range(5):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    gbs = 2 * nbytes * 5 / (a.elapsed_time(b) * 1e-3) / 1e9
    del src, dst
    return gbs


def cpu_baseline(wl, plan, x, xs, w13, s13, w2, s2, m_tile, budget_s):
    """The oracle as it stands, on the host cores: stage-1 dispatch over the
    whole batch, then the fp64 expert FFN + combine on a bounded sample of
    tokens, scaled to the whole batch's local pairs."""
    import oracle

    t0 = time.perf_counter()
    d = oracle.dispatch(wl.topk_ids, wl.T_valid, wl.E, m_tile, wl.placement.slot_expert, plan.slot_weight,
                        plan.remote_weight, plan.remote_replicas)
    t_disp = time.perf_counter() - t0
    ps = oracle.pair_slot(d)
    npairs = ps >= 0
    loc = np.nonzero(npairs.any(axis=1))[0]
    total_pairs = int(npairs.sum())
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    # calibrate on two small token sets (a call has a fixed cost besides its
    # per-pair work), then size the sample to the budget
    rng = np.random.default_rng(0)
    order = rng.permutation(loc)
    pts = []
    for n in (max(1, threads), 4 * max(1, threads)):
        probe = order[: min(len(order), n)]
        sel = np.zeros(wl.T, np.uint8)
        sel[probe] = 1
        t0 = time.perf_counter()
        oracle.moe(x, wl.topk_w, ps, w13, w2, wl.dtype, "exact", xs, s13, s2, token_sel=sel)
        pts.append((int(npairs[probe].sum()), time.perf_counter() - t0))
    (p1, t1), (p2, t2) = pts
    per_pair = max((t2 - t1) / max(1, p2 - p1), t2 / max(1, p2) * 0.05, 1e-9)
    fixed = max(0.0, t2 - per_pair * p2)
    want_pairs = max(p2, int((budget_s - fixed) / per_pair))
    pairs_per_token = max(1e-9, total_pairs / max(1, len(loc)))
    sample = order[: min(len(order), int(want_pairs / pairs_per_token) + 1)]
    sel = np.zeros(wl.T, np.uint8)
    sel[sample] = 1
    t0 = time.perf_counter()
    oracle.moe(x, wl.topk_w, ps, w13, w2, wl.dtype, "exact", xs, s13, s2, token_sel=sel)
    t_moe = time.perf_counter() - t0
    sample_pairs = int(npairs[sample].sum())
    est = t_disp + t_moe * total_pairs / max(1, sample_pairs)
    return {
        "value": est * 1e6,
        "unit": "us/batch",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"stage-1 oracle on the whole batch ({t_disp * 1e3:.1f} ms) + fp64 expert FFN/combine oracle on "
                   f"{len(sample)} of {len(loc)} tokens with local pairs ({sample_pairs} of {total_pairs} pairs, "
                   f"{t_moe:.1f} s), scaled to all {total_pairs} pairs"),
    }


class Measured:
    """Timings of one workload's block on the GPU (see measure_workload)."""


def measure_workload(torch, name, m_tile, plan_name, steps, warmup, seed, copies_arg, spin):
    """Build a workload's inputs in HBM, then time K back-to-back HIP-graph
    replays of the whole block (the headline) and K eager steps with HIP
    events between the stages and around the two GEMM kernels, recorded on
    the stream the kernels run on."""
    from paper_2608_13057_amd import measure, moe, synth
    from paper_2608_13057_amd.moe import to_device as to_dev

    m = Measured()
    wl = synth.make_workload(name, seed=seed)
    m.wl, m.name = wl, name
    m.m_tile = m_tile or measure.auto_m_tile(wl)
    m.plan_name = plan_name or next(iter(wl.plans))
    plan = m.plan = wl.plans[m.plan_name]
    log(f"workload {name} plan {m.plan_name} T={wl.T} K={wl.K} E={wl.E} S={wl.S} H={wl.H} I={wl.I} M={m.m_tile}")
    t0 = time.perf_counter()
    m.x, m.xs = synth.activations(wl.T, wl.H, wl.seed, wl.dtype)
    m.w13, m.s13, m.w2, m.s2 = synth.slot_weights(wl.placement.slot_expert, wl.H, wl.I, wl.seed, wl.dtype)
    log(f"generated inputs in {time.perf_counter() - t0:.1f} s")

    dev = "cuda"
    shape = moe.MoEShape(T=wl.T, K=wl.K, E=wl.E, S=wl.S, H=wl.H, I=wl.I, m_tile=m.m_tile, dtype=wl.dtype)
    d_ids, d_w, d_x = to_dev(wl.topk_ids), to_dev(wl.topk_w), to_dev(m.x)
    d_xs = None if m.xs is None else to_dev(m.xs)
    d_plan = moe.PlanTensors(to_dev(wl.placement.slot_expert), to_dev(plan.slot_weight),
                             to_dev(plan.remote_weight), to_dev(plan.remote_replicas))
    natural = moe.WeightTensors(to_dev(m.w13), to_dev(m.w2), None if m.s13 is None else to_dev(m.s13),
                                None if m.s2 is None else to_dev(m.s2))
    weights0 = moe.pack_weights(shape, natural)  # one-time re-layout, outside the timed region
    del natural
    wbytes = weights0.w13.numel() * weights0.w13.element_size() + weights0.w2.numel() * weights0.w2.element_size()
    # rotate weight copies so that one cycle streams > 2 x the 256 MB Infinity Cache
    copies = m.copies = copies_arg or max(2, math.ceil(1.0e9 / wbytes))
    wsets = [weights0] + [moe.WeightTensors(*(None if t is None else t.clone() for t in
                                              (weights0.w13, weights0.w2, weights0.w13_scale, weights0.w2_scale)))
                          for _ in range(copies - 1)]
    ws = moe.Workspace(shape, dev)
    disp = moe.DispatchBuffers.allocate(shape, ws.row_cap, dev)
    y = torch.empty(wl.T, wl.H, dtype=torch.int16, device=dev)
    fwd = [moe.PreparedForward(shape, d_plan, d_ids, d_w, d_x, d_xs, wsets[i], disp, y, ws) for i in range(copies)]

    for i in range(warmup):
        fwd[i % copies]()
    torch.cuda.synchronize()
    if moe.device_error(ws) != 0:
        raise RuntimeError("device reported a data error")
    sc = disp.slot_counts.cpu().numpy()
    m.G, m.N = int((sc > 0).sum()), int(sc.sum())
    m.tiles = int(sum(-(-int(c) // m.m_tile) for c in sc))
    log(f"G={m.G} N={m.N} tiles={m.tiles} slot_counts={sc.tolist()}")
    K = steps

    # (1) headline: K back-to-back replays of HIP graphs of the whole block;
    # the host enqueues the whole loop while the GPU spins on a short kernel,
    # so launch overhead never shows up between steps
    graphs = []
    for i in range(copies):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fwd[i]()
        graphs.append(g)
    # warm-up of the graph path itself: W replays, every weight copy at least
    # once (the first replays after capture run a few per cent slower than
    # the steady state that back-to-back blocks see)
    for i in range(max(warmup, copies)):
        graphs[i % copies].replay()
    torch.cuda.synchronize()
    ev_a, ev_b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    torch.cuda._sleep(spin)
    ev_a.record()
    for i in range(K):
        graphs[i % copies].replay()
    ev_b.record()
    torch.cuda.synchronize()
    m.ms_per_step = ev_a.elapsed_time(ev_b) / K
    # the spread of single replays: the same replays with an event between
    # each (reported beside the headline mean, not instead of it)
    evr = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    torch.cuda.synchronize()
    torch.cuda._sleep(spin)
    evr[0].record()
    for i in range(K):
        graphs[i % copies].replay()
        evr[i + 1].record()
    torch.cuda.synchronize()
    per = np.array([evr[i].elapsed_time(evr[i + 1]) for i in range(K)]) * 1e3
    m.replay_us = {"p10": float(np.percentile(per, 10)), "median": float(np.median(per)),
                   "p90": float(np.percentile(per, 90))}

    # (2) per-kernel times: K eager steps with HIP events between the stages
    # and around the two GEMM kernels, all on the stream the kernels run on
    NE = moe.STAGE_EVENTS
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(NE)] for _ in range(K)]
    for e in evs:
        for x_ in e:
            x_.record()
    torch.cuda.synchronize()
    torch.cuda._sleep(spin)
    for i in range(K):
        fwd[i % copies](stage_events=evs[i])
    torch.cuda.synchronize()
    at = np.array([[evs[i][0].elapsed_time(evs[i][j]) for j in range(NE)] for i in range(K)]) * 1e3  # us
    m.eager_ms = evs[0][0].elapsed_time(evs[K - 1][NE - 1]) / K
    m.stage_us = {
        "dispatch": float(np.mean(at[:, 1])),
        "gate_up": float(np.mean(at[:, 4] - at[:, 1])),
        "down": float(np.mean(at[:, 6] - at[:, 4])),
        "combine": float(np.mean(at[:, 7] - at[:, 6])),
    }
    # the gate/up GEMM kernel alone (events right before and after it; the
    # large-tile path packs the activation rows first), and the down GEMM
    m.kernel_us = {"gate_up_gemm": float(np.mean(at[:, 3] - at[:, 2])),
                   "down_gemm": float(np.mean(at[:, 5] - at[:, 4])),
                   "before_gate_up_gemm": float(np.mean(at[:, 2] - at[:, 1]))}
    log(f"{name}: graph ms/step {m.ms_per_step:.4f} eager(events) ms/step {m.eager_ms:.4f} "
        f"stages_us {m.stage_us} kernels_us {m.kernel_us}")
    del graphs, fwd, wsets, weights0, ws, disp, y
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return m


def roofline(m, copy_gbs=None):
    """Roofline of the dominant kernel, the gate/up GEMM launch: MFMA-bound
    (useful flops 2 N H 2I per launch against the dense peak of the dtype)
    when the path runs the large-tile kernel or most pairs sit in slots past
    the MFMA/HBM balance point, otherwise HBM-bound (weights of the G
    activated slots once + the N real activation rows in and h rows out)."""
    from paper_2608_13057_amd import measure

    wl = m.wl
    gu_s = m.kernel_us["gate_up_gemm"] * 1e-6
    kernel = measure.gateup_kernel_name(wl.dtype, m.m_tile, wl.H, wl.I)
    traffic, traffic_current = measure.committed_traffic(m.name, m.m_tile)
    common = {"traffic": traffic if traffic_current else None, "kernel": kernel + " (gate/up)",
              "launch_us": m.kernel_us["gate_up_gemm"], "G": m.G, "N": m.N}
    mf = measure.committed_mfma(m.name, m.m_tile)
    if mf is not None:  # counter evidence (rocprofv3 --pmc) for the same kernel sources
        common["mfma_counters"] = {k: mf[k] for k in ("mfma_busy", "clock_ghz", "executed_tflops", "launch_us")}
    # pairs per activated slot against the ideal balance point e P / (2 BW) ~ 312
    linear = measure.uses_big_kernel(wl.dtype, m.m_tile, wl.H, wl.I) or m.N / max(1, m.G) > 312
    if linear:
        fl = gemm_flops(wl, m.N, "gateup")
        peak = MFMA_PEAK_TFLOPS[wl.dtype]
        ach = fl / gu_s / 1e12
        out = {"bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s", "frac": ach / peak,
               **common, "flops_per_launch": fl}
        if mf is not None:  # against the peak at the shader clock the counters saw under this load
            out["frac_at_counter_clock"] = ach / (peak * mf["clock_ghz"] / 2.4)
        return out
    b = gemm_bytes(wl, wl.dtype, m.G, m.N, "gateup")
    ach = b / gu_s / 1e9
    out = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS,
           **common, "bytes_per_launch": b}
    if copy_gbs:  # against what a plain copy attains on this GPU
        out["frac_of_attainable"] = ach / copy_gbs
    return out


def linear_point(torch, G=32, n=1024):
    """Stage 2 (both GEMMs) where every slot is in the linear regime: G slots
    of the Qwen3-235B shape with n rows each (four full 256-row tiles per
    slot), UE8M0 fp8, timed by the stage-4 harness (median of 30 event-timed
    executions); flops 6HI per pair against the fp8 MFMA peak."""
    from paper_2608_13057_amd import profile

    h = profile.Harness(dtype="fp8mx", m_tile=256, max_tokens=G * n)
    r = h.point(G, n, reps=30, scopes=("gemm",))[0]
    H, I = h.H, h.I
    flops = G * n * 6.0 * H * I
    achieved = flops / (r["t_us"] * 1e-6) / 1e12
    del h
    torch.cuda.empty_cache()
    log(f"linear-regime point G={G} n={n}: stage 2 {r['t_us']:.1f} us, {achieved:.0f} TFLOP/s")
    return {"bound": "mfma", "achieved": achieved, "peak": MFMA_PEAK_TFLOPS["fp8mx"], "unit": "TFLOP/s",
            "frac": achieved / MFMA_PEAK_TFLOPS["fp8mx"], "scope": "stage 2 (gate/up and down GEMMs)",
            "workload": f"{G} slots x {n} rows, Qwen3-235B shape (H {H}, I {I}), fp8 UE8M0, M-tile 256, "
                        "one weight set of 32 slots (604 MB, beyond the Infinity Cache)",
            "G": G, "N": G * n, "stage2_us": r["t_us"], "p10_us": r["p10"], "p90_us": r["p90"],
            "flops_per_launch": flops}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs one GPU's share of the EP MoE block on one GPU only; the library has no multi-GPU "
              "path (dispatch / combine all-to-all over xGMI), so --gpus must be 1.", file=sys.stderr)
        return 2

    import torch

    from paper_2608_13057_amd import measure, synth

    spin = calibrate_spin(torch)
    m = measure_workload(torch, args.workload, args.m_tile, args.plan, args.steps, args.warmup, args.seed,
                         args.copies, spin)
    wl = m.wl
    copy_gbs = attainable_copy_gbs(torch, spin)
    log(f"attainable copy bandwidth {copy_gbs:.0f} GB/s")
    gu_s, dn_s = m.kernel_us["gate_up_gemm"] * 1e-6, m.kernel_us["down_gemm"] * 1e-6
    gu_bytes = gemm_bytes(wl, wl.dtype, m.G, m.N, "gateup")
    dn_bytes = gemm_bytes(wl, wl.dtype, m.G, m.N, "down")
    mfma = {
        "gate_up_tflops": gemm_flops(wl, m.N, "gateup") / gu_s / 1e12,
        "down_tflops": gemm_flops(wl, m.N, "down") / dn_s / 1e12,
        "stage2_tflops": (gemm_flops(wl, m.N, "gateup") + gemm_flops(wl, m.N, "down")) / (gu_s + dn_s) / 1e12,
        "peak_tflops": MFMA_PEAK_TFLOPS[wl.dtype],
    }
    shape_name = "dsv3" if wl.H == 7168 else "qwen3"
    out = {
        "metric": "per-GPU MoE block us/batch",
        "value": m.ms_per_step * 1e3,
        "unit": "us/batch",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": m.ms_per_step,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {
            "workload": args.workload,
            "description": synth.describe(args.workload, m.plan_name),
            "m_tile": m.m_tile,
            "plan": m.plan_name,
            "G": m.G, "N": m.N, "tiles": m.tiles,
            "weight_copies_rotated": m.copies,
        },
        "roofline": roofline(m, copy_gbs),
        "replay_us": m.replay_us,
        "stages_us": m.stage_us,
        "kernels_us": m.kernel_us,
        "eager_ms_per_step": m.eager_ms,
        "attainable_copy_gbs": copy_gbs,
        "stage2_hbm_gbs": (gu_bytes + dn_bytes) / (gu_s + dn_s) / 1e9,
        "mfma": mfma,
        "env": {"device": torch.cuda.get_device_name(0), "hip": torch.version.hip, "torch": torch.__version__,
                "compute_units": torch.cuda.get_device_properties(0).multi_processor_count},
        "fit": measure.committed_fit(shape_name, wl.dtype, m.m_tile),
    }
    if not args.no_bf16 and args.bf16_workload != args.workload:
        o = measure_workload(torch, args.bf16_workload, 0, None, args.steps, args.warmup, args.seed, 0, spin)
        out["roofline_bf16"] = {**roofline(o, copy_gbs), "workload": args.bf16_workload, "m_tile": o.m_tile,
                                "block_us": o.ms_per_step * 1e3, "replay_us": o.replay_us, "stages_us": o.stage_us,
                                "fit": measure.committed_fit(shape_name, o.wl.dtype, o.m_tile)}
        del o
    if not args.no_flat and args.flat_workload != args.workload:
        f = measure_workload(torch, args.flat_workload, 0, None, args.steps, args.warmup, args.seed, 0, spin)
        out["roofline_flat"] = {**roofline(f, copy_gbs), "workload": args.flat_workload, "m_tile": f.m_tile,
                                "block_us": f.ms_per_step * 1e3, "replay_us": f.replay_us, "stages_us": f.stage_us,
                                "fit": measure.committed_fit(shape_name, f.wl.dtype, f.m_tile)}
        del f
    if not args.no_flat and args.flat2_workload not in (args.workload, args.flat_workload):
        f2 = measure_workload(torch, args.flat2_workload, 0, None, args.steps, args.warmup, args.seed, 0, spin)
        sh2 = "dsv3" if f2.wl.H == 7168 else "qwen3"
        out["roofline_flat_dsv3"] = {**roofline(f2, copy_gbs), "workload": args.flat2_workload, "m_tile": f2.m_tile,
                                     "block_us": f2.ms_per_step * 1e3, "replay_us": f2.replay_us,
                                     "stages_us": f2.stage_us,
                                     "fit": measure.committed_fit(sh2, f2.wl.dtype, f2.m_tile)}
        del f2
    if args.linear:
        out["roofline_linear"] = linear_point(torch)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle")
        out["cpu_baseline"] = cpu_baseline(wl, m.plan, m.x, m.xs, m.w13, m.s13, m.w2, m.s2, m.m_tile,
                                           args.cpu_budget_s)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
