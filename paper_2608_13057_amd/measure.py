"""Measurement helpers around rocprofv3 (run on the GPU host, summaries kept
under profiles/).

    python -m paper_2608_13057_amd.measure run --workload W [--m-tile M]
        the program to profile: a few eager calls of the whole block on a
        workload, then a plain elementwise kernel that reads 256 MiB and
        writes 256 MiB (y = 2x in fp32; the calibration of the traffic
        counters)
    python -m paper_2608_13057_amd.measure stats DIR --out MD --command CMD
        kernel-time table from `rocprofv3 --kernel-trace --stats` output
    python -m paper_2608_13057_amd.measure traffic FETCH_DIR WRITE_DIR --out MD ...
        HBM bytes per launch of the gate/up GEMM from two `rocprofv3 --pmc`
        passes (FETCH_SIZE, WRITE_SIZE), each scaled by the reading of the
        same counter for that elementwise kernel
    python -m paper_2608_13057_amd.measure mfma PMC_DIR TRACE_DIR --out MD ...
        MFMA busy fraction, shader clock and executed flops of the gate/up
        GEMM from one `rocprofv3 --pmc` pass and a kernel trace
    python -m paper_2608_13057_amd.measure snap --out MD
        the tile-aware split (TEMPO_PLAN_SNAP_TILES) against the plain one:
        M-tiles, activated slots and block time per workload and batch size
    python -m paper_2608_13057_amd.measure library --out MD
        reference points, not part of the path: the vendor GEMM (hipBLASLt,
        through torch) on dense GEMMs of the prefill shapes, fp8 and bf16
    python -m paper_2608_13057_amd.measure readbw --out MD
        the attainable HBM rates of plain torch kernels: a row-wise max
        (reads), a copy (reads and writes) and a fill (writes)

The traffic summary ends with a `traffic_json:` line that bench.py reads; it
carries a hash of the stage-2 sources, and bench.py reports no traffic once
the sources have changed since the counters were taken.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
COPY_BYTES = 256 << 20
GEMM_SOURCES = ("gemm_stream.h", "gemm_common.h", "gemm_bf16.hip", "gemm_fp8.hip", "gemm_big_agpr.hip", "gemm_big_f8_agpr.hip",
                "pack.hip")


def gemm_source_hash() -> str:
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(HERE, "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def auto_m_tile(wl) -> int:
    """64-row tiles when an expert sees a few dozen rows (decode), 128 up to
    128 rows per expert, and beyond that 256 for bf16 and UE8M0 fp8 (the
    large-tile kernels of the linear regime) or 128 for fp8 with fp32
    scales."""
    per_expert = wl.T * wl.K / wl.E
    if per_expert <= 64:
        return 64
    if per_expert <= 128 or wl.dtype == "fp8":
        return 128
    return 256


def uses_big_kernel(dtype: str, m_tile: int, H: int, I: int = 256) -> bool:
    """Whether stage 2 runs a 256 x 256-item large-tile GEMM (bf16, or UE8M0
    fp8 with I a multiple of 256, with 256-row tiles and H a multiple of 256)
    rather than the stream-K one."""
    return (dtype == "bf16" or (dtype == "fp8mx" and I % 256 == 0)) and m_tile == 256 and H % 256 == 0


def gateup_kernel_name(dtype: str, m_tile: int, H: int, I: int = 256) -> str:
    """Symbol (as rocprofv3 prints it) of the gate/up GEMM kernel a forward
    launches."""
    if uses_big_kernel(dtype, m_tile, H, I):
        return ("tempo::(anonymous namespace)::k_gemm_big<true>" if dtype == "bf16" else
                "tempo::(anonymous namespace)::k_gemm_big_f8<true>")
    fp8 = "false" if dtype == "bf16" else "true"
    mx = "true" if dtype == "fp8mx" else "false"
    return f"tempo::gemm::k_gemm<{fp8}, {m_tile}, true, {mx}>"


def traffic_path(workload: str, m_tile: int) -> str:
    return os.path.join(ROOT, "profiles", f"k_gemm_gateup_{workload}_m{m_tile}_traffic.md")


def fit_path(shape: str, dtype: str, m_tile: int) -> str:
    return os.path.join(ROOT, "profiles", f"stage4_{shape}_{dtype}_m{m_tile}.md")


def committed_fit(shape: str, dtype: str, m_tile: int, scope: str = "gemm"):
    """The Eq. 1 fit (a, b, c, beta, n*) of a committed stage-4 profile for
    one scope, or None: from its `fit_json:` line, else from the Eq. 1 row of
    the scope's table."""
    path = fit_path(shape, dtype, m_tile)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        text = fh.read()
    for line in text.splitlines():
        if line.startswith("fit_json: "):
            d = json.loads(line[len("fit_json: "):])
            if d.get("scope") == scope and d.get("model") == "Eq. 1":
                return dict(d, source=os.path.relpath(path, ROOT))
    sec = text.split(f"scope `{scope}`", 1)
    if len(sec) < 2:
        return None
    for line in sec[1].splitlines():
        if line.startswith("| Eq. 1 |"):
            c = [x.strip() for x in line.strip("|").split("|")]
            return {"scope": scope, "model": "Eq. 1", "a": float(c[1]), "b": float(c[2]), "c": float(c[3]),
                    "beta": float(c[4]), "n_star": float(c[6]), "err_mean": float(c[7]), "err_max": float(c[8]),
                    "source": os.path.relpath(path, ROOT)}
    return None


def committed_traffic(workload: str, m_tile: int):
    """(bytes per launch, source hash matches) from the committed summary, or
    (None, False) if there is none."""
    path = traffic_path(workload, m_tile)
    if not os.path.exists(path):
        return None, False
    with open(path) as fh:
        for line in fh:
            if line.startswith("traffic_json: "):
                d = json.loads(line[len("traffic_json: "):])
                return d["bytes_per_launch"], d.get("source_hash") == gemm_source_hash()
    return None, False


def _run(args):
    import numpy as np
    import torch

    from . import moe, synth
    from .moe import to_device as td

    wl = synth.make_workload(args.workload, seed=args.seed)
    mt = args.m_tile or auto_m_tile(wl)
    plan = wl.plans[args.plan or next(iter(wl.plans))]
    x, xs = synth.activations(wl.T, wl.H, wl.seed, wl.dtype)
    w13, s13, w2, s2 = synth.slot_weights(wl.placement.slot_expert, wl.H, wl.I, wl.seed, wl.dtype)
    shape = moe.MoEShape(T=wl.T, K=wl.K, E=wl.E, S=wl.S, H=wl.H, I=wl.I, m_tile=mt, dtype=wl.dtype)
    d_plan = moe.PlanTensors(td(wl.placement.slot_expert), td(plan.slot_weight), td(plan.remote_weight),
                             td(plan.remote_replicas))
    nat = moe.WeightTensors(td(w13), td(w2), None if s13 is None else td(s13), None if s2 is None else td(s2))
    wpk = moe.pack_weights(shape, nat)
    del nat
    ws = moe.Workspace(shape)
    disp = moe.DispatchBuffers.allocate(shape, ws.row_cap)
    y = torch.empty(wl.T, wl.H, dtype=torch.int16, device="cuda")
    f = moe.PreparedForward(shape, d_plan, td(wl.topk_ids), td(wl.topk_w), td(x), None if xs is None else td(xs), wpk,
                            disp, y, ws)
    for _ in range(args.calls):
        f()
    torch.cuda.synchronize()
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.mul(src, 2.0, out=dst)
    torch.cuda.synchronize()
    sc = disp.slot_counts.cpu().numpy()
    print(f"workload {args.workload} m_tile {mt} G={int((sc > 0).sum())} N={int(sc.sum())} calls {args.calls}; "
          f"copy {COPY_BYTES} bytes x3", flush=True)
    return 0


def _rows(d: str):
    rows = []
    for f in sorted(glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)):
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    if not rows:
        raise SystemExit(f"no counter_collection.csv under {d}")
    return rows


def _mean_counter(rows, counter: str, match):
    v = [float(r["Counter_Value"]) for r in rows if r["Counter_Name"] == counter and match(r["Kernel_Name"])]
    if not v:
        raise SystemExit(f"no {counter} for the kernel")
    return sum(v) / len(v), len(v)


def _is_gateup(name: str) -> bool:
    """The gate/up GEMM: the large-tile kernel k_gemm_big<true>, or the
    stream-K instance with GATEUP (its third template argument)."""
    if "k_gemm_big<true>" in name.replace(" ", "") or "k_gemm_big_f8<true>" in name.replace(" ", ""):
        return True
    if "k_gemm<" not in name:
        return False
    args = name.replace(" ", "").split("k_gemm<", 1)[1].split(">", 1)[0].split(",")
    return len(args) >= 3 and args[2] == "true"


def _is_copy(name: str) -> bool:
    return "elementwise_kernel" in name and "Mul" in name


def _traffic(args):
    fr, wr = _rows(args.fetch_dir), _rows(args.write_dir)
    g_f, n_f = _mean_counter(fr, "FETCH_SIZE", _is_gateup)
    c_f, _ = _mean_counter(fr, "FETCH_SIZE", _is_copy)
    g_w, n_w = _mean_counter(wr, "WRITE_SIZE", _is_gateup)
    c_w, _ = _mean_counter(wr, "WRITE_SIZE", _is_copy)
    kib = COPY_BYTES / 1024
    kf, kw = kib / c_f, kib / c_w  # counter readings -> bytes of the copy
    fetch_b, write_b = g_f * kf * 1024, g_w * kw * 1024
    names = sorted({r["Kernel_Name"] for r in fr if _is_gateup(r["Kernel_Name"])})
    d = {"kernel": names[0] if names else "k_gemm gate/up", "workload": args.workload, "m_tile": args.m_tile,
         "fetch_bytes": fetch_b, "write_bytes": write_b, "bytes_per_launch": fetch_b + write_b,
         "copy_fetch_factor": kf, "copy_write_factor": kw, "source_hash": gemm_source_hash()}
    lines = [
        f"# HBM traffic: gate/up GEMM, {args.workload}, M-tile {args.m_tile}",
        "",
        "Commands (repo root, MI355X), one counter pass each:",
        "",
        "```",
        args.command1,
        args.command2,
        f"python -m paper_2608_13057_amd.measure traffic {args.fetch_dir} {args.write_dir} --workload {args.workload} "
        f"--m-tile {args.m_tile} --out <this file>",
        "```",
        "",
        f"Kernel: `{d['kernel']}` ({n_f} / {n_w} dispatches averaged).",
        "",
        "| | gate/up GEMM (counter, KiB) | 256 MiB y = 2x (counter, KiB) | scale | bytes per launch |",
        "|---|---|---|---|---|",
        f"| FETCH_SIZE | {g_f:.0f} | {c_f:.0f} | {kf:.4f} | {fetch_b / 1e6:.2f} MB |",
        f"| WRITE_SIZE | {g_w:.0f} | {c_w:.0f} | {kw:.4f} | {write_b / 1e6:.2f} MB |",
        "",
        f"Scale = 262144 KiB (what y = 2x over 256 MiB of fp32 reads, and writes) / that kernel's counter reading.  "
        f"Total {d['bytes_per_launch'] / 1e6:.2f} MB per launch.",
        "",
        "traffic_json: " + json.dumps(d),
        "",
    ]
    with open(args.out, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))
    return 0


def mfma_path(workload: str, m_tile: int) -> str:
    return os.path.join(ROOT, "profiles", f"k_gemm_gateup_{workload}_m{m_tile}_mfma.md")


def committed_mfma(workload: str, m_tile: int):
    """The committed MFMA-counter summary of the gate/up kernel (dict), or
    None when there is none or the stage-2 sources changed since."""
    path = mfma_path(workload, m_tile)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        for line in fh:
            if line.startswith("mfma_json: "):
                d = json.loads(line[len("mfma_json: "):])
                return d if d.get("source_hash") == gemm_source_hash() else None
    return None


def _agent(d: str) -> dict:
    for f in sorted(glob.glob(os.path.join(d, "**", "*agent_info.csv"), recursive=True)):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r.get("Name", "").startswith("gfx"):
                    return r
    raise SystemExit(f"no GPU agent in {d}")


def _kernel_avg_ns(d: str, match):
    f = glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True)
    if not f:
        raise SystemExit(f"no kernel_stats.csv under {d}")
    with open(f[0]) as fh:
        for r in csv.DictReader(fh):
            if match(r["Name"]):
                return float(r["AverageNs"]), r["Name"]
    raise SystemExit("kernel not in the trace")


def _mfma(args):
    """MFMA utilisation of the gate/up GEMM from one rocprofv3 --pmc pass
    (SQ_VALU_MFMA_BUSY_CYCLES per SIMD, GRBM_GUI_ACTIVE summed over the XCDs,
    the MFMA op counters) and the kernel's mean duration from a kernel trace
    of the same program."""
    from . import synth

    rows = _rows(args.pmc_dir)
    ag = _agent(args.pmc_dir)
    nxcc, nsimd = int(ag["Num_Xcc"]), int(ag["Simd_Count"])
    busy, n = _mean_counter(rows, "SQ_VALU_MFMA_BUSY_CYCLES", _is_gateup)
    gui, _ = _mean_counter(rows, "GRBM_GUI_ACTIVE", _is_gateup)
    ops = 0.0
    for c in ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU_MFMA_MOPS_F8"):
        try:
            ops += _mean_counter(rows, c, _is_gateup)[0]
        except SystemExit:
            pass
    dur_ns, kname = _kernel_avg_ns(args.trace_dir, _is_gateup)
    cycles = gui / nxcc  # GPU cycles of the dispatch (GRBM_GUI_ACTIVE is per XCD)
    util = busy / (cycles * nsimd)
    clock = cycles / dur_ns  # GHz
    wl = synth.make_workload(args.workload)
    executed = ops * 512
    dt = wl.dtype
    peak = {"bf16": 2500.0, "fp8": 5000.0, "fp8mx": 5000.0}[dt]
    d = {"kernel": kname, "workload": args.workload, "m_tile": args.m_tile, "mfma_busy": util, "clock_ghz": clock,
         "launch_us": dur_ns / 1e3, "executed_tflops": executed / dur_ns / 1e3,
         "executed_frac_of_peak": executed / dur_ns / 1e3 / peak, "dispatches": n, "source_hash": gemm_source_hash()}
    lines = [
        f"# MFMA utilisation: gate/up GEMM, {args.workload}, M-tile {args.m_tile}",
        "",
        "Commands (repo root, MI355X):",
        "",
        "```",
        args.command1,
        args.command2,
        f"python -m paper_2608_13057_amd.measure mfma {args.pmc_dir} {args.trace_dir} --workload {args.workload} "
        f"--m-tile {args.m_tile} --out <this file>",
        "```",
        "",
        f"Kernel: `{kname}` ({n} dispatches averaged; mean duration {dur_ns / 1e3:.1f} us from the kernel trace).",
        "",
        "| quantity | value |",
        "|---|---|",
        f"| SQ_VALU_MFMA_BUSY_CYCLES (sum over {nsimd} SIMDs) | {busy:.4g} |",
        f"| GRBM_GUI_ACTIVE (sum over {nxcc} XCDs) | {gui:.4g} |",
        f"| dispatch cycles = GRBM_GUI_ACTIVE / {nxcc} | {cycles:.4g} |",
        f"| MFMA busy = busy / (cycles x {nsimd}) | **{util:.3f}** |",
        f"| shader clock = cycles / duration | {clock:.2f} GHz (nominal {int(ag['Max_Engine_Clk_Fcompute']) / 1e3:.1f}) |",
        f"| executed MFMA flops (MOPS x 512) | {executed / 1e9:.1f} GFLOP ({executed / dur_ns / 1e3:.0f} TFLOP/s, "
        f"{executed / dur_ns / 1e3 / peak:.3f} of {peak:.0f}) |",
        "",
        "The busy fraction counts MFMA pipe cycles against the cycles of the dispatch at the clock the GPU ran; "
        "executed flops include the padding rows of partly filled M-tiles, which the roofline's useful flops do not.",
        "",
        "mfma_json: " + json.dumps(d),
        "",
    ]
    with open(args.out, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))
    return 0


def _stats(args):
    f = glob.glob(os.path.join(args.dir, "**", "*kernel_stats.csv"), recursive=True)
    if not f:
        raise SystemExit(f"no kernel_stats.csv under {args.dir}")
    with open(f[0]) as fh:
        rows = list(csv.DictReader(fh))
    lines = [f"# Kernel times: {args.title}", "", "Command (repo root, MI355X):", "", "```", args.command, "```", "",
             "| kernel | calls | avg us | min us | max us | % |", "|---|---|---|---|---|---|"]
    for r in rows:
        name = r["Name"].replace("|", "\\|")
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                     f"{float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    if args.note:
        lines += ["", args.note]
    lines.append("")
    with open(args.out, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))
    return 0


def _snap(args):
    """Tile-aware split against the plain one: M-tiles, activated slots and
    block time of the forward, per workload, plan, M-tile and batch size."""
    import numpy as np
    import torch

    from . import moe, synth
    from .moe import to_device as td

    title = ("Tile-aware split (TEMPO_PLAN_SNAP_TILES)" if args.variant == "snap" else
             f"Sampled replicas (TEMPO_PLAN_SAMPLE, generator key {args.key})")
    lines = [f"# {title} against the plain split", "",
             "Command (repo root, MI355X):", "", "```", args.command or "python -m paper_2608_13057_amd.measure snap",
             "```", "",
             "Tiles = sum over slots of ceil(c_s / M) as stage 1 placed them on the GPU; extra = plain / variant - 1.  "
             "Block = one forward (stages 1-3), median of "
             f"{args.calls} event-timed calls, the two splits alternating call by call.", "",
             "| workload | T | plan | M | G plain / variant | N plain / variant | tiles plain / variant | extra tiles | "
             "block plain us | block variant us | block change |", "|---|---|---|---|---|---|---|---|---|---|---|"]
    for spec in args.cases:
        name, T, M, timed = spec.split(":")
        T, M, timed = int(T), int(M), timed == "t"
        wl = synth.make_workload(name, seed=args.seed, T=T)
        x, xs = synth.activations(wl.T, wl.H, wl.seed, wl.dtype)
        shape = moe.MoEShape(T=wl.T, K=wl.K, E=wl.E, S=wl.S, H=wl.H, I=wl.I, m_tile=M, dtype=wl.dtype)
        if timed:
            w13, s13, w2, s2 = synth.slot_weights(wl.placement.slot_expert, wl.H, wl.I, wl.seed, wl.dtype)
            nat = moe.WeightTensors(td(w13), td(w2), None if s13 is None else td(s13), None if s2 is None else td(s2))
            wpk = moe.pack_weights(shape, nat)
            del nat, w13, w2
        for pname, plan in wl.plans.items():
            runs = {}
            for snap in (False, True):
                # (a prepared forward holds device pointers only: every tensor
                # it reads stays referenced here until the timing is done)
                keep = dict(plan=moe.PlanTensors(td(wl.placement.slot_expert), td(plan.slot_weight),
                                                 td(plan.remote_weight), td(plan.remote_replicas),
                                                 snap_tiles=snap and args.variant == "snap",
                                                 sample_seed=args.key if snap and args.variant == "sample" else None),
                            ids=td(wl.topk_ids), w=td(wl.topk_w), x=td(x), xs=None if xs is None else td(xs),
                            ws=moe.Workspace(shape))
                keep["disp"] = moe.DispatchBuffers.allocate(shape, keep["ws"].row_cap)
                f = None
                if timed:
                    keep["y"] = torch.empty(wl.T, wl.H, dtype=torch.int16, device="cuda")
                    f = moe.PreparedForward(shape, keep["plan"], keep["ids"], keep["w"], keep["x"], keep["xs"], wpk,
                                            keep["disp"], keep["y"], keep["ws"])
                    for _ in range(3):
                        f()
                else:
                    moe.dispatch(shape, keep["plan"], keep["ids"], keep["x"], keep["xs"], keep["disp"], keep["ws"])
                runs[snap] = (f, keep["disp"], keep)
            torch.cuda.synchronize()
            # the two splits alternate call by call, so that drifts of clock
            # and cache state hit both alike
            ts = {False: [], True: []}
            for _ in range(args.calls if timed else 0):
                for snap in (False, True):
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record()
                    runs[snap][0]()
                    e1.record()
                    torch.cuda.synchronize()
                    ts[snap].append(e0.elapsed_time(e1) * 1e3)
            row = {}
            for snap in (False, True):
                sc = runs[snap][1].slot_counts.cpu().numpy().astype(np.int64)
                row[snap] = (int((sc > 0).sum()), int((-(-sc // M)).sum()), float(np.median(ts[snap])) if timed else None,
                             int(sc.sum()))
            del runs
            (g0, n0, t0, N0), (g1, n1, t1, N1) = row[False], row[True]
            tb = lambda v: "-" if v is None else f"{v:.1f}"
            ch = "-" if t0 is None else f"{(t1 / t0 - 1) * 100:+.1f}%"
            lines.append(f"| {name} | {T} | {pname} | {M} | {g0} / {g1} | {N0} / {N1} | {n0} / {n1} | "
                         f"{(n0 / max(n1, 1) - 1) * 100:.1f}% "
                         f"| {tb(t0)} | {tb(t1)} | {ch} |")
            print(lines[-1], flush=True)
        if timed:
            del wpk
        torch.cuda.empty_cache()
    with open(args.out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    return 0


def _timed_us(f, n=20):
    """Mean time of f over n calls after three warm-up calls, from events."""
    import torch

    for _ in range(3):
        f()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(n):
        f()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / n * 1e3


def _library(args):
    import torch

    torch.cuda.set_device(0)
    # the padded and unpadded gate/up GEMM of the Qwen3 prefill share at
    # 256-row tiles, its down GEMM, and a large square one
    shapes = [(14336, 3072, 4096), (11486, 3072, 4096), (14336, 4096, 1536), (8192, 8192, 8192)]
    lines = ["# Vendor GEMM on dense GEMMs of the prefill shapes (reference points)", "",
             "Command (repo root, MI355X):", "", "```", args.command, "```", "",
             "torch's `_scaled_mm` (fp8 e4m3fn operands, tensor scales, bf16 out; hipBLASLt on ROCm) and bf16 `@`, "
             "20 timed calls after 3 warm-up calls, random operands; one weight matrix per GEMM (no grouping, no gather).",
             "", "| M x N x K | fp8 us | fp8 TFLOP/s | bf16 us | bf16 TFLOP/s |", "|---|---|---|---|---|"]
    for m, n, k in shapes:
        a = torch.randn(m, k, device="cuda").to(torch.float8_e4m3fn)
        b = torch.randn(n, k, device="cuda").to(torch.float8_e4m3fn)
        one = torch.tensor(1.0, device="cuda")
        t8 = _timed_us(lambda: torch._scaled_mm(a, b.t(), scale_a=one, scale_b=one, out_dtype=torch.bfloat16))
        ab = torch.randn(m, k, device="cuda", dtype=torch.bfloat16)
        bb = torch.randn(k, n, device="cuda", dtype=torch.bfloat16)
        t16 = _timed_us(lambda: ab @ bb)
        fl = 2.0 * m * n * k
        lines.append(f"| {m} x {n} x {k} | {t8:.1f} | {fl / t8 / 1e6:.0f} | {t16:.1f} | {fl / t16 / 1e6:.0f} |")
        print(lines[-1], flush=True)
        del a, b, ab, bb
    lines.append("")
    with open(args.out, "w") as fh:
        fh.write("\n".join(lines))
    return 0


def _readbw(args):
    import torch

    torch.cuda.set_device(0)
    lines = ["# Attainable HBM rates of plain kernels", "", "Command (repo root, MI355X):", "", "```", args.command, "```",
             "", "torch kernels over fp32 tensors, 10 timed calls after 3 warm-up calls; bytes counted once each way.",
             "", "| size | row max (4096 per row) read GB/s | copy read+write GB/s | fill write GB/s |", "|---|---|---|---|"]
    for gib in (1, 4):
        n = gib * (1 << 30) // 4
        x = torch.randn(n, device="cuda")
        y = torch.empty_like(x)
        rd = n * 4 / _timed_us(lambda: torch.amax(x.view(-1, 4096), dim=1), 10) / 1e3
        cp = 2 * n * 4 / _timed_us(lambda: y.copy_(x), 10) / 1e3
        wr = n * 4 / _timed_us(lambda: y.fill_(1.0), 10) / 1e3
        lines.append(f"| {gib} GiB | {rd:.0f} | {cp:.0f} | {wr:.0f} |")
        print(lines[-1], flush=True)
        del x, y
    lines.append("")
    with open(args.out, "w") as fh:
        fh.write("\n".join(lines))
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    r = sub.add_parser("run")
    r.add_argument("--workload", default="qwen3_decode_bf16")
    r.add_argument("--plan", default=None)
    r.add_argument("--m-tile", type=int, default=0)
    r.add_argument("--seed", type=int, default=0)
    r.add_argument("--calls", type=int, default=5)
    t = sub.add_parser("traffic")
    t.add_argument("fetch_dir")
    t.add_argument("write_dir")
    t.add_argument("--workload", required=True)
    t.add_argument("--m-tile", type=int, required=True)
    t.add_argument("--out", required=True)
    t.add_argument("--command1", default="")
    t.add_argument("--command2", default="")
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("--out", required=True)
    s.add_argument("--title", default="")
    s.add_argument("--command", default="")
    s.add_argument("--note", default="")
    mf = sub.add_parser("mfma", help="MFMA utilisation of the gate/up GEMM from a counter pass and a kernel trace")
    mf.add_argument("pmc_dir")
    mf.add_argument("trace_dir")
    mf.add_argument("--workload", required=True)
    mf.add_argument("--m-tile", type=int, required=True)
    mf.add_argument("--out", required=True)
    mf.add_argument("--command1", default="")
    mf.add_argument("--command2", default="")
    n = sub.add_parser("snap", help="the tile-aware split or sampled replicas against the plain split")
    n.add_argument("--variant", choices=("snap", "sample"), default="snap")
    n.add_argument("--key", type=int, default=12345, help="generator key of the sampled variant")
    n.add_argument("--cases", nargs="+", default=[
        "qwen3_decode_fp8:1024:128:t", "qwen3_prefill_bf16:2048:128:n", "qwen3_prefill_bf16:4096:128:n",
        "qwen3_prefill_bf16:8192:128:t", "qwen3_prefill_bf16:8192:256:t", "qwen3_prefill_bf16:16384:128:n",
        "qwen3_prefill_fp8:8192:128:t"], help="workload:T:M-tile:t (timed) or n (tiles only)")
    n.add_argument("--seed", type=int, default=0)
    n.add_argument("--calls", type=int, default=30)
    n.add_argument("--out", required=True)
    n.add_argument("--command", default="")
    lb = sub.add_parser("library", help="vendor GEMM on dense GEMMs of the prefill shapes (reference points)")
    lb.add_argument("--out", required=True)
    lb.add_argument("--command", default="python -m paper_2608_13057_amd.measure library --out <this file>")
    rb = sub.add_parser("readbw", help="attainable HBM rates of plain kernels")
    rb.add_argument("--out", required=True)
    rb.add_argument("--command", default="python -m paper_2608_13057_amd.measure readbw --out <this file>")
    a = ap.parse_args(argv)
    return {"run": _run, "traffic": _traffic, "stats": _stats, "snap": _snap, "mfma": _mfma, "library": _library,
            "readbw": _readbw}[a.cmd](a)


if __name__ == "__main__":
    sys.exit(main())
