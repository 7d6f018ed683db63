"""Python binding of the TEMPO per-GPU MoE block library.

Argument marshalling only: torch tensors supply device memory and
``torch.cuda.current_stream()`` the HIP stream; every step of the path runs in
the HIP kernels of libtempo_moe.so (include/tempo_moe.h has the contract of
each call).  The names follow the C ABI: :func:`query`, :func:`dispatch`,
:func:`experts`, :func:`combine`, :func:`forward`, :func:`device_error`.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass

import torch

from . import _lib
from ._lib import DispatchOut, ExpertWeights, Plan, Shape, check

DTYPES = {"bf16": _lib.TEMPO_BF16, "fp8": _lib.TEMPO_FP8_E4M3, "fp8mx": _lib.TEMPO_FP8_E4M3_UE8M0}


def to_device(a, device="cuda") -> torch.Tensor:
    """numpy array -> contiguous device tensor; uint16 (bf16 bits) travels as
    int16 and uint32 (plan weights) as int32, bit for bit."""
    import numpy as np

    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    elif a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(a).to(device)


def _ptr(t) -> int | None:
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream) -> int | None:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _need(t, dtype, shape, name):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


@dataclass
class MoEShape:
    T: int
    K: int
    E: int
    S: int
    H: int
    I: int
    m_tile: int = 128
    dtype: str = "bf16"
    T_valid: int | None = None

    def c(self) -> Shape:
        return Shape(self.T, self.T if self.T_valid is None else self.T_valid, self.K, self.E, self.S, self.H,
                     self.I, self.m_tile, DTYPES[self.dtype])

    @property
    def elem(self):
        return torch.int16 if self.dtype == "bf16" else torch.uint8


def query(shape: MoEShape) -> tuple[int, int]:
    """(workspace_bytes, row_cap)."""
    ws = ctypes.c_size_t(0)
    cap = ctypes.c_int32(0)
    sh = shape.c()
    check(_lib.load().tempo_moe_query(ctypes.byref(sh), ctypes.byref(ws), ctypes.byref(cap), None),
          "tempo_moe_query")
    return int(ws.value), int(cap.value)


def packed_slot_bytes(shape: MoEShape) -> int:
    """Bytes of one slot's packed weights (tempo_moe_query's
    packed_bytes_per_slot)."""
    n = ctypes.c_size_t(0)
    sh = shape.c()
    check(_lib.load().tempo_moe_query(ctypes.byref(sh), None, None, ctypes.byref(n)), "tempo_moe_query")
    return int(n.value)


class Workspace:
    """A zero-filled device workspace for one shape (one per stream in flight)."""

    def __init__(self, shape: MoEShape, device="cuda"):
        nbytes, cap = query(shape)
        self.nbytes = nbytes
        self.row_cap = cap
        self.buf = torch.zeros(nbytes, dtype=torch.uint8, device=device)

    @property
    def ptr(self):
        return self.buf.data_ptr()


@dataclass
class DispatchBuffers:
    expert_counts: torch.Tensor
    slot_counts: torch.Tensor
    slot_offsets: torch.Tensor
    row_token: torch.Tensor
    pair_row: torch.Tensor
    x_perm: torch.Tensor
    x_perm_scale: torch.Tensor | None = None
    cum_counts: torch.Tensor | None = None

    @staticmethod
    def allocate(shape: MoEShape, row_cap: int, device="cuda", cum_counts: bool = False):
        i32 = dict(dtype=torch.int32, device=device)
        return DispatchBuffers(
            expert_counts=torch.empty(shape.E, **i32),
            slot_counts=torch.empty(shape.S, **i32),
            slot_offsets=torch.empty(shape.S + 1, **i32),
            row_token=torch.empty(row_cap, **i32),
            pair_row=torch.empty(shape.T, shape.K, **i32),
            x_perm=torch.empty(row_cap, shape.H, dtype=shape.elem, device=device),
            x_perm_scale=(torch.empty(shape.H // 128, row_cap, dtype=torch.float32, device=device)
                          if shape.dtype != "bf16" else None),
            cum_counts=torch.zeros(shape.E, dtype=torch.int32, device=device) if cum_counts else None,
        )

    def c(self) -> DispatchOut:
        return DispatchOut(_ptr(self.expert_counts), _ptr(self.slot_counts), _ptr(self.slot_offsets),
                           _ptr(self.row_token), _ptr(self.pair_row), _ptr(self.cum_counts), _ptr(self.x_perm),
                           _ptr(self.x_perm_scale))


@dataclass
class PlanTensors:
    slot_expert: torch.Tensor  # [S] int32
    slot_weight: torch.Tensor  # [S] int32 holding uint32 bit patterns
    remote_weight: torch.Tensor  # [E] int32 (uint32 bits)
    remote_replicas: torch.Tensor  # [E] int32
    snap_tiles: bool = False  # tile-aware split (TEMPO_PLAN_SNAP_TILES)
    sample_seed: int | None = None  # sampled replicas with this generator key (TEMPO_PLAN_SAMPLE)

    def c(self) -> Plan:
        flags = (_lib.TEMPO_PLAN_SNAP_TILES if self.snap_tiles else 0) | (
            0 if self.sample_seed is None else _lib.TEMPO_PLAN_SAMPLE)
        return Plan(_ptr(self.slot_expert), _ptr(self.slot_weight), _ptr(self.remote_weight),
                    _ptr(self.remote_replicas), flags, 0 if self.sample_seed is None else int(self.sample_seed))


@dataclass
class WeightTensors:
    w13: torch.Tensor | None
    w2: torch.Tensor | None
    w13_scale: torch.Tensor | None = None
    w2_scale: torch.Tensor | None = None
    # stage 2: [S, 4] int64 device tensor of per-slot pointers
    # (tempo_slot_weights: w13, w13_scale, w2, w2_scale), see slot_table()
    slot_table: torch.Tensor | None = None
    keep: tuple = ()  # the tensors a slot table points into (kept alive)

    def c(self) -> ExpertWeights:
        return ExpertWeights(_ptr(self.w13), _ptr(self.w13_scale), _ptr(self.w2), _ptr(self.w2_scale),
                             _ptr(self.slot_table))


def slot_table(slots: list, device="cuda") -> WeightTensors:
    """Weights given per slot: slots[s] holds slot s's packed tensors (a
    1-slot pack_weights result) wherever they live; returns a WeightTensors
    whose device table (tempo_slot_weights [S]) points at them."""
    rows = [[_ptr(w.w13) or 0, _ptr(w.w13_scale) or 0, _ptr(w.w2) or 0, _ptr(w.w2_scale) or 0] for w in slots]
    tab = torch.tensor(rows, dtype=torch.int64, device=device)
    return WeightTensors(None, None, slot_table=tab, keep=tuple(slots))


def pack_weights(shape: MoEShape, natural: WeightTensors, stream=None) -> WeightTensors:
    """One-time re-layout (tempo_moe_pack_weights): returns new tensors holding
    w13 / w2 in the packed layout stage 2 reads and, for fp8, the packed
    scales ([S, I/64, H/128, 4] and [S, H/128, I/128, 4] fp32)."""
    _check_weights(shape, natural)
    s13 = s2 = None
    if shape.dtype != "bf16":
        dev = natural.w13.device
        s13 = torch.empty(shape.S, shape.I // 64, shape.H // 128, 4, dtype=torch.float32, device=dev)
        s2 = torch.empty(shape.S, shape.H // 128, shape.I // 128, 4, dtype=torch.float32, device=dev)
    packed = WeightTensors(torch.empty_like(natural.w13), torch.empty_like(natural.w2), s13, s2)
    sh, nat, pk = shape.c(), natural.c(), packed.c()
    check(_lib.load().tempo_moe_pack_weights(ctypes.byref(sh), ctypes.byref(nat), ctypes.byref(pk),
                                             _stream(stream)), "tempo_moe_pack_weights")
    return packed


def _check_inputs(shape, topk_ids, x, x_scale):
    _need(topk_ids, torch.int32, (shape.T, shape.K), "topk_ids")
    _need(x, shape.elem, (shape.T, shape.H), "x")
    if shape.dtype != "bf16":
        _need(x_scale, torch.float32, (shape.T, shape.H // 128), "x_scale")


def _check_plan(shape, plan):
    _need(plan.slot_expert, torch.int32, (shape.S,), "slot_expert")
    _need(plan.slot_weight, torch.int32, (shape.S,), "slot_weight")
    _need(plan.remote_weight, torch.int32, (shape.E,), "remote_weight")
    _need(plan.remote_replicas, torch.int32, (shape.E,), "remote_replicas")


def _check_weights(shape, w, packed=False):
    if packed and w.slot_table is not None:
        _need(w.slot_table, torch.int64, (shape.S, 4), "slot_table")
        return
    _need(w.w13, shape.elem, (shape.S, 2 * shape.I, shape.H), "w13")
    _need(w.w2, shape.elem, (shape.S, shape.H, shape.I), "w2")
    if shape.dtype != "bf16":
        if packed:
            _need(w.w13_scale, torch.float32, (shape.S, shape.I // 64, shape.H // 128, 4), "packed w13_scale")
            _need(w.w2_scale, torch.float32, (shape.S, shape.H // 128, shape.I // 128, 4), "packed w2_scale")
        else:
            _need(w.w13_scale, torch.float32, (shape.S, 2 * shape.I // 128, shape.H // 128), "w13_scale")
            _need(w.w2_scale, torch.float32, (shape.S, shape.H // 128, shape.I // 128), "w2_scale")


def _check_disp(shape, d, row_cap):
    _need(d.slot_counts, torch.int32, (shape.S,), "slot_counts")
    _need(d.slot_offsets, torch.int32, (shape.S + 1,), "slot_offsets")
    _need(d.x_perm, shape.elem, (row_cap, shape.H), "x_perm")
    if d.expert_counts is not None:
        _need(d.expert_counts, torch.int32, (shape.E,), "expert_counts")
    _need(d.row_token, torch.int32, (row_cap,), "row_token")
    if d.pair_row is not None:
        _need(d.pair_row, torch.int32, (shape.T, shape.K), "pair_row")
    if shape.dtype != "bf16":
        _need(d.x_perm_scale, torch.float32, (shape.H // 128, row_cap), "x_perm_scale")
    if d.cum_counts is not None:
        _need(d.cum_counts, torch.int32, (shape.E,), "cum_counts")


def dispatch(shape: MoEShape, plan: PlanTensors, topk_ids, x, x_scale, out: DispatchBuffers, ws: Workspace,
             stream=None) -> DispatchBuffers:
    """Stage 1 (tempo_moe_dispatch)."""
    _check_inputs(shape, topk_ids, x, x_scale)
    _check_plan(shape, plan)
    _check_disp(shape, out, ws.row_cap)
    sh, pl, do = shape.c(), plan.c(), out.c()
    check(_lib.load().tempo_moe_dispatch(ctypes.byref(sh), ctypes.byref(pl), _ptr(topk_ids), _ptr(x), _ptr(x_scale),
                                         ctypes.byref(do), ws.ptr, ws.nbytes, _stream(stream)), "tempo_moe_dispatch")
    return out


def experts(shape: MoEShape, disp: DispatchBuffers, weights: WeightTensors, y_perm, ws: Workspace, stream=None):
    """Stage 2 (tempo_moe_experts): writes y_perm [row_cap, H] bf16.  weights
    must be packed (pack_weights)."""
    _check_disp(shape, disp, ws.row_cap)
    _check_weights(shape, weights, packed=True)
    _need(y_perm, torch.int16, (ws.row_cap, shape.H), "y_perm")
    sh, do, w = shape.c(), disp.c(), weights.c()
    check(_lib.load().tempo_moe_experts(ctypes.byref(sh), ctypes.byref(do), ctypes.byref(w), _ptr(y_perm), ws.ptr,
                                        ws.nbytes, _stream(stream)), "tempo_moe_experts")
    return y_perm


def combine(shape: MoEShape, pair_row, topk_w, y_perm, y, stream=None):
    """Stage 3 (tempo_moe_combine): writes y [T, H] bf16."""
    _need(pair_row, torch.int32, (shape.T, shape.K), "pair_row")
    _need(topk_w, torch.float32, (shape.T, shape.K), "topk_w")
    if y_perm.dtype != torch.int16 or y_perm.dim() != 2 or y_perm.shape[1] != shape.H or not y_perm.is_contiguous():
        raise ValueError("y_perm must be a contiguous [rows, H] int16 (bf16 bits) tensor")
    _need(y, torch.int16, (shape.T, shape.H), "y")
    sh = shape.c()
    check(_lib.load().tempo_moe_combine(ctypes.byref(sh), _ptr(pair_row), _ptr(topk_w), _ptr(y_perm), _ptr(y),
                                        _stream(stream)), "tempo_moe_combine")
    return y


# events of tempo_moe_forward's stage_events (TEMPO_STAGE_EVENTS)
STAGE_EVENTS = 8


def forward(shape: MoEShape, plan: PlanTensors, topk_ids, topk_w, x, x_scale, weights: WeightTensors,
            disp: DispatchBuffers, y, ws: Workspace, slot_time_ns=None, stage_events=None, stream=None):
    """Stages 1-3 (tempo_moe_forward): writes y [T, H] bf16 (int16 bits);
    weights must be packed (pack_weights).
    stage_events: optional list of STAGE_EVENTS (8) torch.cuda.Event (created
    with enable_timing=True) recorded before stage 1, after stage 1, right
    before the gate/up GEMM kernel (after the activation pack of the
    large-tile kernels), after it, after the gate/up step, after the down GEMM
    kernel, after the down step and after stage 3."""
    _check_inputs(shape, topk_ids, x, x_scale)
    _need(topk_w, torch.float32, (shape.T, shape.K), "topk_w")
    _check_plan(shape, plan)
    _check_weights(shape, weights, packed=True)
    _check_disp(shape, disp, ws.row_cap)
    _need(y, torch.int16, (shape.T, shape.H), "y")
    if slot_time_ns is not None:
        _need(slot_time_ns, torch.int64, (shape.S,), "slot_time_ns")
    sh, pl, w, do = shape.c(), plan.c(), weights.c(), disp.c()
    evs = None
    if stage_events is not None:
        if len(stage_events) != STAGE_EVENTS:
            raise ValueError(f"stage_events must hold {STAGE_EVENTS} events")
        evs = (ctypes.c_void_p * STAGE_EVENTS)(*[_event_handle(e) for e in stage_events])
    check(_lib.load().tempo_moe_forward(ctypes.byref(sh), ctypes.byref(pl), _ptr(topk_ids), _ptr(topk_w), _ptr(x),
                                        _ptr(x_scale), ctypes.byref(w), ctypes.byref(do), _ptr(y),
                                        _ptr(slot_time_ns), evs, ws.ptr, ws.nbytes, _stream(stream)),
          "tempo_moe_forward")
    return y


def forward_static(shape: MoEShape, plan: PlanTensors, topk_ids, topk_w, x, x_scale, weights: WeightTensors,
                   disp: DispatchBuffers, y, slot_time_ns=None, stream=None):
    """tempo_moe_forward_static: forward() on the library's static scratch
    array instead of a workspace (allocates nothing; the shape's workspace
    must fit in TEMPO_STATIC_SCRATCH_BYTES).  Calls that overlap on one GPU
    race on the array."""
    _check_inputs(shape, topk_ids, x, x_scale)
    _need(topk_w, torch.float32, (shape.T, shape.K), "topk_w")
    _check_plan(shape, plan)
    _check_weights(shape, weights, packed=True)
    _, row_cap = query(shape)
    _check_disp(shape, disp, row_cap)
    _need(y, torch.int16, (shape.T, shape.H), "y")
    if slot_time_ns is not None:
        _need(slot_time_ns, torch.int64, (shape.S,), "slot_time_ns")
    sh, pl, w, do = shape.c(), plan.c(), weights.c(), disp.c()
    check(_lib.load().tempo_moe_forward_static(ctypes.byref(sh), ctypes.byref(pl), _ptr(topk_ids), _ptr(topk_w),
                                               _ptr(x), _ptr(x_scale), ctypes.byref(w), ctypes.byref(do), _ptr(y),
                                               _ptr(slot_time_ns), None, _stream(stream)),
          "tempo_moe_forward_static")
    return y


class PreparedForward:
    """A validated tempo_moe_forward call whose ctypes arguments are built
    once; calling it re-issues the same launch sequence on the current (or a
    given) stream with no per-call Python checks -- for serving loops and
    graph capture.  The tensors passed in must stay alive and in place."""

    def __init__(self, shape: MoEShape, plan: PlanTensors, topk_ids, topk_w, x, x_scale, weights: WeightTensors,
                 disp: DispatchBuffers, y, ws: Workspace, slot_time_ns=None):
        _check_inputs(shape, topk_ids, x, x_scale)
        _need(topk_w, torch.float32, (shape.T, shape.K), "topk_w")
        _check_plan(shape, plan)
        _check_weights(shape, weights, packed=True)
        _check_disp(shape, disp, ws.row_cap)
        _need(y, torch.int16, (shape.T, shape.H), "y")
        if slot_time_ns is not None:
            _need(slot_time_ns, torch.int64, (shape.S,), "slot_time_ns")
        self._keep = (shape.c(), plan.c(), weights.c(), disp.c())
        sh, pl, w, do = self._keep
        self._args = [ctypes.byref(sh), ctypes.byref(pl), _ptr(topk_ids), _ptr(topk_w), _ptr(x), _ptr(x_scale),
                      ctypes.byref(w), ctypes.byref(do), _ptr(y), _ptr(slot_time_ns)]
        self._tail = [ws.ptr, ws.nbytes]
        self._fn = _lib.load().tempo_moe_forward

    def __call__(self, stage_events=None, stream=None):
        evs = None
        if stage_events is not None:
            if len(stage_events) != STAGE_EVENTS:
                raise ValueError(f"stage_events must hold {STAGE_EVENTS} events")
            evs = (ctypes.c_void_p * STAGE_EVENTS)(*[_event_handle(e) for e in stage_events])
        check(self._fn(*self._args, evs, *self._tail, _stream(stream)), "tempo_moe_forward")


def _event_handle(ev):
    """The hipEvent_t behind a torch.cuda.Event (created on first record);
    None for a null entry (the library skips it)."""
    if ev is None:
        return None
    if ev.cuda_event == 0:
        ev.record()  # materialise the event on the current stream
    return ev.cuda_event


def device_error(ws: Workspace, stream=None) -> int:
    """Synchronise and read + clear the sticky device error word."""
    bits = ctypes.c_uint32(0)
    check(_lib.load().tempo_moe_device_error(ws.ptr, _stream(stream), ctypes.byref(bits)), "tempo_moe_device_error")
    return int(bits.value)


def counter_window(before, after):
    """tempo_moe_counter_window: per-expert pair counts of a window from two
    snapshots of the cumulative counters (cum_counts, wrapping modulo 2^32).
    Accepts numpy arrays or CPU tensors of int32 / uint32 bits; returns
    uint32."""
    import numpy as np

    b = np.ascontiguousarray(np.asarray(before.cpu() if hasattr(before, "cpu") else before).view(np.uint32))
    a = np.ascontiguousarray(np.asarray(after.cpu() if hasattr(after, "cpu") else after).view(np.uint32))
    if a.shape != b.shape or a.ndim != 1:
        raise ValueError("before and after must be 1-D arrays of the same length")
    out = np.empty_like(a)
    u32p = ctypes.POINTER(ctypes.c_uint32)
    check(_lib.load().tempo_moe_counter_window(len(a), b.ctypes.data_as(u32p), a.ctypes.data_as(u32p),
                                               out.ctypes.data_as(u32p)), "tempo_moe_counter_window")
    return out
