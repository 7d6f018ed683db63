"""CPU oracle for one GPU's share of the expert-parallel MoE block (TEMPO).

TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check and the benchmark's
CPU-baseline leg may import this package; the product path never does.  It
shares no code with the HIP library (``paper_2608_13057_amd``) and imports
nothing from it.

* :func:`dispatch` -- stage 1 (per-expert counts, plan split, padded groups,
  stable permutation), Sec. 3.1 problem statement, Sec. 2.2 / Eq. 2 M-tiles,
  Sec. 4.4 integration semantics.  Plain C (``tempo_oracle.c``).
* :func:`gather` -- the permuted activation rows, a plain index copy.
* :func:`moe` -- stages 2+3 (gate/up, SwiGLU, down, routing-weighted sum),
  Sec. 2.1, in fp64.  Plain C.
* :mod:`oracle.fit` -- the two-piece max-affine cost (Eq. 1), its tile-aware
  form (Eq. 2) and the alternating-assignment fit (Appendix "Calibration
  details").
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tempo_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libtempo_oracle.so")
_lib = None

ERR_BAD_ID = 1
ERR_BAD_SLOT_EXPERT = 2
ERR_WEIGHT_OVERFLOW = 4


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (-O2, OpenMP) into oracle/libtempo_oracle.so."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.run(
            ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"],
            check=True,
        )
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i32 = ctypes.c_int
        lib.oracle_dispatch.restype = ctypes.c_uint32
        lib.oracle_dispatch.argtypes = [i32] * 6 + [P] * 11 + [i32, ctypes.c_uint64]
        lib.oracle_philox4x64_10.restype = None
        lib.oracle_philox4x64_10.argtypes = [P, P, P]
        lib.oracle_moe.restype = None
        lib.oracle_moe.argtypes = [i32] * 7 + [P] * 10
        lib.oracle_ffn_rows.restype = None
        lib.oracle_ffn_rows.argtypes = [i32] * 5 + [P] * 9
        lib.oracle_combine.restype = None
        lib.oracle_combine.argtypes = [i32] * 4 + [P] * 4
        for n in ("oracle_bf16_value",):
            getattr(lib, n).restype = ctypes.c_double
            getattr(lib, n).argtypes = [ctypes.c_uint16]
        lib.oracle_e4m3_value.restype = ctypes.c_double
        lib.oracle_e4m3_value.argtypes = [ctypes.c_uint8]
        for n in ("oracle_round_bf16", "oracle_round_e4m3"):
            getattr(lib, n).restype = ctypes.c_double
            getattr(lib, n).argtypes = [ctypes.c_double]
        _lib = lib
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def dispatch(topk_ids, T_valid, E, M, slot_expert, slot_weight, remote_weight, remote_replicas,
             cum_counts=None, snap=False, sample_seed=None) -> dict:
    """Stage 1.  Returns a dict with expert_counts, slot_counts, slot_offsets,
    row_token (length slot_offsets[-1]), pair_row, err and (if given) the
    updated cum_counts.  snap: the tile-aware split (interior boundaries on
    the nearest multiple of M, Sec. 2.2 after Eq. 2).  sample_seed: sampled
    replicas instead of the split (Sec. 4.4), one Philox-4x64-10 draw per
    pair keyed by the seed."""
    lib = _load()
    ids = np.ascontiguousarray(topk_ids, dtype=np.int32)
    T, K = ids.shape
    S = len(slot_expert)
    se = np.ascontiguousarray(slot_expert, dtype=np.int32)
    sw = np.ascontiguousarray(slot_weight, dtype=np.uint32)
    rw = np.ascontiguousarray(remote_weight, dtype=np.uint32)
    rr = np.ascontiguousarray(remote_replicas, dtype=np.int32)
    assert rw.shape == (E,) and rr.shape == (E,) and sw.shape == (S,)
    ec = np.zeros(E, np.int32)
    sc = np.zeros(S, np.int32)
    so = np.zeros(S + 1, np.int32)
    cap = T * K + S * (M - 1)
    rt = np.full(max(cap, 1), -1, np.int32)
    pr = np.full(max(T * K, 1), -1, np.int32)
    cum = None if cum_counts is None else np.array(cum_counts, dtype=np.uint32).copy()
    err = lib.oracle_dispatch(T, T_valid, K, E, S, M, _p(ids), _p(se), _p(sw), _p(rw), _p(rr), _p(ec),
                              _p(sc), _p(so), _p(rt), _p(pr), None if cum is None else _p(cum),
                              (1 if snap else 0) | (0 if sample_seed is None else 2),
                              0 if sample_seed is None else int(sample_seed))
    out = dict(expert_counts=ec, slot_counts=sc, slot_offsets=so, row_token=rt[: so[S]].copy(),
               pair_row=pr[: T * K].reshape(T, K).copy(), err=int(err))
    if cum is not None:
        out["cum_counts"] = cum
    return out


def pair_slot(d: dict) -> np.ndarray:
    """Local slot of each pair (-1 = not local), from a dispatch result."""
    pr = d["pair_row"]
    so = d["slot_offsets"]
    ps = np.full(pr.shape, -1, np.int32)
    m = pr >= 0
    ps[m] = np.searchsorted(so, pr[m], side="right") - 1
    return ps


def gather(x: np.ndarray, row_token: np.ndarray, x_scale=None):
    """Permuted activation rows: X_perm[row] = x[row_token[row]] for
    non-padding rows.  Padding rows are returned as zeros (the library leaves
    them unwritten; tests compare non-padding rows only)."""
    R = len(row_token)
    xp = np.zeros((R,) + x.shape[1:], x.dtype)
    m = row_token >= 0
    xp[m] = x[row_token[m]]
    if x_scale is None:
        return xp
    sp = np.zeros((R,) + x_scale.shape[1:], x_scale.dtype)
    sp[m] = x_scale[row_token[m]]
    return xp, sp


def moe(x, topk_w, pslot, w13, w2, dtype: str, mode: str = "exact", x_scale=None, w13_scale=None,
        w2_scale=None, token_sel=None) -> np.ndarray:
    """Stages 2+3 in fp64.  x: [T,H] uint16 (bf16 bits) or uint8 (e4m3);
    w13: [S,2I,H]; w2: [S,H,I]; pslot: [T,K] local slot per pair (-1 = none).
    Returns y [T,H] float64 (rows not selected by token_sel are zeros)."""
    lib = _load()
    x = np.ascontiguousarray(x)
    T, H = x.shape
    K = pslot.shape[1]
    S, I2, H2 = w13.shape
    I = I2 // 2
    assert H2 == H and w2.shape == (S, H, I)
    dt = {"bf16": 0, "fp8": 1, "fp8mx": 2}[dtype]
    md = {"exact": 0, "mirror": 1}[mode]
    if dt != 0:
        assert x_scale is not None and w13_scale is not None and w2_scale is not None
        xs = np.ascontiguousarray(x_scale, np.float32)
        s13 = np.ascontiguousarray(w13_scale, np.float32)
        s2 = np.ascontiguousarray(w2_scale, np.float32)
    else:
        xs = s13 = s2 = None
    tw = np.ascontiguousarray(topk_w, np.float32)
    ps = np.ascontiguousarray(pslot, np.int32)
    sel = np.ones(T, np.uint8) if token_sel is None else np.ascontiguousarray(token_sel, np.uint8)
    y = np.zeros((T, H), np.float64)
    w13c = np.ascontiguousarray(w13)
    w2c = np.ascontiguousarray(w2)
    lib.oracle_moe(T, K, H, I, S, dt, md, _p(x), None if xs is None else _p(xs), _p(w13c),
                   None if s13 is None else _p(s13), _p(w2c), None if s2 is None else _p(s2), _p(tw), _p(ps),
                   _p(sel), _p(y))
    return y


def ffn_rows(x, tok, slot, w13, w2, dtype: str, mode: str = "exact", x_scale=None, w13_scale=None,
             w2_scale=None) -> np.ndarray:
    """Stage 2 alone, per row: o[r] = FFN of expert slot[r] applied to
    x[tok[r]] (fp64).  Rows with slot < 0 are zero."""
    lib = _load()
    x = np.ascontiguousarray(x)
    T, H = x.shape
    S, I2, _ = w13.shape
    I = I2 // 2
    tok = np.ascontiguousarray(tok, np.int32)
    slot = np.ascontiguousarray(slot, np.int32)
    R = len(tok)
    out = np.zeros((R, H), np.float64)
    dt = {"bf16": 0, "fp8": 1, "fp8mx": 2}[dtype]
    md = {"exact": 0, "mirror": 1}[mode]
    keep = [np.ascontiguousarray(a, np.float32) if a is not None else None for a in (x_scale, w13_scale, w2_scale)]
    w13c, w2c = np.ascontiguousarray(w13), np.ascontiguousarray(w2)
    lib.oracle_ffn_rows(R, H, I, dt, md, _p(x), None if keep[0] is None else _p(keep[0]), _p(tok), _p(slot),
                        _p(w13c), None if keep[1] is None else _p(keep[1]), _p(w2c),
                        None if keep[2] is None else _p(keep[2]), _p(out))
    return out


def combine(pair_row, topk_w, y_perm_bits, T_valid) -> np.ndarray:
    """Stage 3 alone: routing-weighted sum of bf16 rows, fp64."""
    lib = _load()
    pr = np.ascontiguousarray(pair_row, np.int32)
    T, K = pr.shape
    yp = np.ascontiguousarray(y_perm_bits, np.uint16)
    H = yp.shape[1]
    tw = np.ascontiguousarray(topk_w, np.float32)
    y = np.zeros((T, H), np.float64)
    lib.oracle_combine(T, T_valid, K, H, _p(pr), _p(tw), _p(yp), _p(y))
    return y


def bf16_value(b: int) -> float:
    return _load().oracle_bf16_value(b)


def e4m3_value(c: int) -> float:
    return _load().oracle_e4m3_value(c)


def round_bf16(x: float) -> float:
    return _load().oracle_round_bf16(x)


def round_e4m3(x: float) -> float:
    return _load().oracle_round_e4m3(x)


def philox4x64_10(counter, key):
    """One block of Philox-4x64-10 (four uint64 words) at a 4-word counter and
    2-word key (the generator of the sampled dispatch)."""
    lib = _load()
    c = np.ascontiguousarray(counter, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, np.uint64)
    lib.oracle_philox4x64_10(_p(c), _p(k), _p(out))
    return out
