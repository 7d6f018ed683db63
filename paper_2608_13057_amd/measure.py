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
GEMM_SOURCES = ("gemm_stream.h", "gemm_common.h", "gemm_bf16.hip", "gemm_fp8.hip", "gemm_big_agpr.hip", "pack.hip")


def gemm_source_hash() -> str:
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(HERE, "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def auto_m_tile(wl) -> int:
    """64-row tiles when an expert sees a few dozen rows (decode), else 128."""
    return 64 if wl.T * wl.K / wl.E <= 64 else 128


def traffic_path(workload: str, m_tile: int) -> str:
    return os.path.join(ROOT, "profiles", f"k_gemm_gateup_{workload}_m{m_tile}_traffic.md")


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
    return "k_gemm<" in name and name.replace(" ", "").split("(")[0].endswith(",true>")


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
    a = ap.parse_args(argv)
    return {"run": _run, "traffic": _traffic, "stats": _stats}[a.cmd](a)


if __name__ == "__main__":
    sys.exit(main())
