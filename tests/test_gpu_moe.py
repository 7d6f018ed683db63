"""GPU parity of stages 2 and 3 and of the whole forward against the oracle.

Tolerances: outputs are compared per token row as
  err = max_t ||y_t - r_t||_inf / ||r_t||_inf
over rows with at least one local pair; rows without one must be exactly
zero.  Against the fp64 oracle in its exact mode the bar is 1e-2 for bf16
and 5e-2 for fp8.  Against its mirror mode (which rounds h, o and y where
the datapath stores them, with the dot products still in fp64) the residual
comes only from the fp32 accumulation order moving a value across a rounding
boundary, so most elements must be bit-identical and the rest differ by such
flips.  A flip of the final rounding of y is one bf16 ulp of that element
(up to 2^-7 of the row's largest value), so the mirror error counts per
element only what exceeds one ulp (helpers.mirror_err_rows): bf16 at least
99.9% identical and err <= 1e-3 (an h flip is one bf16 ulp of one of I
terms of an output; measured 1e-4 .. 3e-4); fp8 at least 85% identical and
err <= 2e-2 (an e4m3 flip of one h element moves every output of its row by
up to 2^-4 of that term; measured 6e-3 .. 1.3e-2, 92% identical)."""
import numpy as np
import pytest

import oracle
from helpers import (Case, bf16_to_f64, identical_share, mirror_err_rows, mirror_stats, rel_err_rows, tile_sample,
                     to_dev,
                     to_host)

pytestmark = pytest.mark.gpu

TOL_EXACT = {"bf16": 1e-2, "fp8": 5e-2, "fp8mx": 5e-2}
# Tests that compare hundreds of rows: the max over rows reaches further into
# the tail of the rounding the method itself does.  fp8, exact mode: h is
# re-quantised to e4m3 (up to 2^-4 relative per value) before the down GEMM.
# bf16, mirror mode: y passes two bf16 roundings in series (y_perm, then the
# combine's y), and a flip of the first can leave one more ulp of y than the
# one-ulp allowance of mirror_err_rows; 2^-8 of the row's largest value.
TOL_EXACT_FP8_MANY = 8e-2
TOL_MIRROR_BF16_MANY, MIRROR_IDENTICAL_BF16_MANY = 4e-3, 0.995
TOL_MIRROR = {"bf16": 1e-3, "fp8": 2e-2, "fp8mx": 2e-2}
MIRROR_IDENTICAL = {"bf16": 0.999, "fp8": 0.85, "fp8mx": 0.85}


def _run_forward(c, timing=False):
    import torch
    from paper_2608_13057_amd import moe

    y = torch.empty(c.wl.T, c.wl.H, dtype=torch.int16, device="cuda")
    st = torch.zeros(c.wl.S, dtype=torch.int64, device="cuda") if timing else None
    moe.forward(c.shape, c.d_plan, c.d_ids, c.d_w, c.d_x, c.d_xs, c.d_weights, c.disp, y, c.ws, slot_time_ns=st)
    torch.cuda.synchronize()
    return (to_host(y), None if st is None else st.cpu().numpy())


def _oracle_y(c, d_ref, mode="exact", token_sel=None):
    return oracle.moe(c.x, c.wl.topk_w, oracle.pair_slot(d_ref), c.w13, c.w2, c.dtype, mode, c.xs, c.s13, c.s2,
                      token_sel=token_sel)


def _check_many_rows(dtype, err, err_m, same):
    """The bars of a test that compares hundreds of rows (see the constants
    above): the mirror mode, which rounds where the GPU rounds, checks the
    kernel; the exact mode bounds what the method's own rounding does."""
    if dtype == "bf16":
        assert err <= TOL_EXACT[dtype]
        assert err_m <= TOL_MIRROR_BF16_MANY and same >= MIRROR_IDENTICAL_BF16_MANY
    else:
        assert err_m <= TOL_MIRROR[dtype] and same >= MIRROR_IDENTICAL[dtype]
        assert err <= TOL_EXACT_FP8_MANY


def _local_rows(d_ref, T_valid):
    has = (d_ref["pair_row"] >= 0).any(axis=1)
    has[T_valid:] = False
    return np.nonzero(has)[0], np.nonzero(~has)[0]


@pytest.mark.parametrize("fresh_ws", [False, True])
@pytest.mark.parametrize("m_tile", [64, 128, 192, 256])
@pytest.mark.parametrize("name", ["tiny", "tiny_fp8", "tiny_fp8mx"])
def test_experts_stage_tiny(m_tile, name, fresh_ws):
    """Stage 2 alone: y_perm real rows against the oracle's per-row FFN.
    fresh_ws: stage 2 runs on a second, never-used workspace (it takes the
    tile count from slot_offsets, not from anything stage 1 left in the
    workspace)."""
    import torch
    from paper_2608_13057_amd import moe, synth

    wl = synth.make_workload(name)
    c = Case(wl, "uniform", m_tile)
    moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
    y_perm = torch.empty(c.ws.row_cap, wl.H, dtype=torch.int16, device="cuda")
    moe.experts(c.shape, c.disp, c.d_weights, y_perm, moe.Workspace(c.shape) if fresh_ws else c.ws)
    torch.cuda.synchronize()
    d = c.oracle_dispatch()
    rt = d["row_token"]
    real = np.nonzero(rt >= 0)[0]
    slot = np.searchsorted(d["slot_offsets"], real, side="right") - 1
    got = bf16_to_f64(to_host(y_perm)[real])
    for mode, tol in (("exact", TOL_EXACT[wl.dtype]), ("mirror", TOL_MIRROR[wl.dtype])):
        ref = oracle.ffn_rows(c.x, rt[real], slot, c.w13, c.w2, wl.dtype, mode, c.xs, c.s13, c.s2)
        err = (rel_err_rows if mode == "exact" else mirror_err_rows)(got, ref, np.arange(len(real)))
        print(f"[experts {name} M={m_tile}] {mode} err={err:.2e} {mirror_stats(got, ref)}")
        assert err <= tol
        if mode == "mirror":
            assert identical_share(got, ref) >= MIRROR_IDENTICAL[wl.dtype]


def test_combine_stage():
    """Stage 3 alone on generator-made bf16 rows and the oracle's pair_row."""
    import torch
    from paper_2608_13057_amd import moe, synth

    rng = np.random.default_rng(9)
    for T, K, H, Tv in ((96, 2, 256, 96), (300, 8, 4096, 250), (7, 32, 128, 7)):
        R = T * K
        yp = synth.to_bf16_bits(rng.standard_normal((R, H)).astype(np.float32))
        pr = rng.permutation(R).astype(np.int32).reshape(T, K)
        pr[rng.random((T, K)) < 0.3] = -1
        w = rng.random((T, K)).astype(np.float32)
        shape = moe.MoEShape(T=T, K=K, E=max(K, 8), S=1, H=H, I=128, T_valid=Tv)
        y = torch.empty(T, H, dtype=torch.int16, device="cuda")
        moe.combine(shape, to_dev(pr), to_dev(w), to_dev(yp), y)
        torch.cuda.synchronize()
        got = bf16_to_f64(to_host(y))
        ref = oracle.combine(pr, w, yp, Tv)
        # one bf16 rounding of an fp32 sum: within one bf16 ulp of the exact value
        ulp = np.where(ref != 0, 2.0 ** (np.floor(np.log2(np.abs(ref) + 1e-300)) - 7), 2.0 ** -133)
        assert np.all(np.abs(got - ref) <= ulp + 1e-6 * np.abs(ref)), f"T={T} K={K}"
        assert np.all(got[Tv:] == 0)


@pytest.mark.parametrize("m_tile", [64, 128, 192, 256])
@pytest.mark.parametrize("name", ["tiny", "tiny_fp8", "tiny_fp8mx"])
def test_forward_tiny(m_tile, name):
    from paper_2608_13057_amd import synth

    wl = synth.make_workload(name)
    c = Case(wl, "uniform", m_tile)
    y, st = _run_forward(c, timing=True)
    d = c.oracle_dispatch()
    loc, none = _local_rows(d, c.T_valid)
    got = bf16_to_f64(y)
    for mode in ("exact", "mirror"):
        ref = _oracle_y(c, d, mode)
        err = (rel_err_rows if mode == "exact" else mirror_err_rows)(got, ref, loc)
        print(f"[forward {name} M={m_tile}] {mode} err={err:.2e} {mirror_stats(got[loc], ref[loc])}")
        assert err <= (TOL_EXACT if mode == "exact" else TOL_MIRROR)[wl.dtype]
        if mode == "mirror":
            assert identical_share(got[loc], ref[loc]) >= MIRROR_IDENTICAL[wl.dtype]
    assert np.all(y[none] == 0)
    sc = d["slot_counts"]
    assert np.all((st > 0) == (sc > 0))


@pytest.mark.parametrize("dtype", ["fp8mx", "bf16", "fp8"])
def test_forward_256_row_tiles_every_live_block_count(dtype):
    """256-row M-tiles whose slots hold 1, 31, 33, 64, 65, 97, 129, 161, 193,
    225, 255, 256, 257, 300 and 520 rows: every number of live 32-row blocks
    in a tile (1..8), full tiles, a slot one row past a tile, and slots of two
    and three tiles; element by element against the oracle (exact and
    mirror modes).  The UE8M0 large-tile kernel skips the row blocks of
    padding only and deals the items by cost; the bf16 one runs whole tiles;
    fp32-scale fp8 runs the stream-K kernel."""
    from paper_2608_13057_amd import synth

    counts = [1, 31, 33, 64, 65, 97, 129, 161, 193, 225, 255, 256, 257, 300, 520]
    E = len(counts)
    ids = np.repeat(np.arange(E, dtype=np.int32), counts)
    np.random.default_rng(11).shuffle(ids)
    T = ids.size
    pl = synth.placement_local_hot(E, E, 0)  # one slot per expert
    wl = synth.Workload("row_blocks", dtype, T, T, 1, E, 256, 512, 0.0, pl, {"uniform": synth.plan_uniform(pl, E)},
                        ids.reshape(T, 1), np.ones((T, 1), np.float32), 0)
    c = Case(wl, "uniform", 256)
    y, _ = _run_forward(c)
    d = c.oracle_dispatch()
    assert np.array_equal(d["slot_counts"], np.array(counts))
    loc, none = _local_rows(d, c.T_valid)
    got = bf16_to_f64(y)
    for mode in ("exact", "mirror"):
        ref = _oracle_y(c, d, mode)
        err = (rel_err_rows if mode == "exact" else mirror_err_rows)(got, ref, loc)
        print(f"[forward row blocks {dtype}] {mode} err={err:.2e} {mirror_stats(got[loc], ref[loc])}")
        assert err <= (TOL_EXACT if mode == "exact" else TOL_MIRROR)[dtype]
        if mode == "mirror":
            assert identical_share(got[loc], ref[loc]) >= MIRROR_IDENTICAL[dtype]
    assert np.all(y[none] == 0)


@pytest.mark.parametrize("dtype,I", [("fp8mx", 512), ("bf16", 128)])
def test_forward_256_row_tiles_shallow_items(dtype, I):
    """The large-tile kernels with the fewest sub-steps per item and several
    items per workgroup: H 256 (a UE8M0 gate/up item is then four sub-steps,
    as many as its operand ring holds; both GEMMs run the same item cursor)
    and, for bf16, I 128 (a down item of eight sub-steps, one less than its
    ring), 64 experts of 1000..1199 rows in over 300 M-tiles, so the DMA
    cursor of every workgroup is an item or more ahead when an item starts.
    y on a token sample with one row of every M-tile and every slot's last
    row against the fp64 oracle (exact and mirror modes); tokens with no
    local pair exactly zero."""
    from paper_2608_13057_amd import synth

    rng = np.random.default_rng(23)
    E, H = 64, 256
    counts = rng.integers(1000, 1200, E)
    ids = np.repeat(np.arange(E, dtype=np.int32), counts)
    rng.shuffle(ids)
    T = ids.size
    pl = synth.placement_local_hot(E, E, 0)  # one slot per expert
    w = rng.uniform(0.1, 1.0, (T, 1)).astype(np.float32)
    wl = synth.Workload("shallow", dtype, T, T, 1, E, H, I, 0.0, pl, {"uniform": synth.plan_uniform(pl, E)},
                        ids.reshape(T, 1), w, 0)
    c = Case(wl, "uniform", 256)
    print(f"[shallow {dtype} I={I}] running, {T} tokens", flush=True)
    y, _ = _run_forward(c)
    d = c.oracle_dispatch()
    assert np.array_equal(to_host(c.disp.slot_counts), d["slot_counts"])
    ntiles = int(sum(-(-int(n) // 256) for n in d["slot_counts"]))
    assert ntiles > 256  # more items than workgroups in both GEMMs
    loc, none = _local_rows(d, c.T_valid)
    assert np.all(y[none] == 0)
    pick = tile_sample(d, 256, np.random.default_rng(2))
    sel = np.zeros(T, np.uint8)
    sel[pick] = 1
    got = bf16_to_f64(y)
    ref = _oracle_y(c, d, "mirror", sel)
    err_m = mirror_err_rows(got, ref, pick)
    same = identical_share(got[pick], ref[pick])
    ref = _oracle_y(c, d, "exact", sel)
    err = rel_err_rows(got, ref, pick)
    print(f"[shallow {dtype} I={I}] {ntiles} tiles, sampled {len(pick)} tokens exact err={err:.2e} "
          f"mirror err={err_m:.2e} identical={same:.4f}")
    _check_many_rows(dtype, err, err_m, same)


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("dtype", ["fp8mx", "bf16"])
def test_forward_256_row_tiles_random_shapes(dtype, seed):
    """The large-tile kernels on random shapes each accepts: H from 256 to
    1280, I from the smallest multiple each takes (UE8M0: 256, bf16: 128)
    up to 1024, 3..24 experts of 1..900 rows routed top-1 or top-2 over
    uniform or hot placements; stage 1 bit-exact, y on a token sample with
    one row of every M-tile and every slot's last row against the fp64
    oracle in exact and mirror modes; tokens with no local pair exactly
    zero."""
    from paper_2608_13057_amd import synth

    rng = np.random.default_rng(100 + seed + (0 if dtype == "bf16" else 50))
    H = int(rng.choice([256, 512, 768, 1280]))
    I = int(rng.choice([256, 512, 768, 1024] if dtype == "fp8mx" else [128, 384, 640, 1024]))
    E = int(rng.integers(3, 25))
    K = int(rng.integers(1, 3))
    counts = rng.integers(1, 900, E)
    T = int(counts.sum()) // K + 1
    ids = np.empty((T, K), np.int32)
    for t in range(T):
        ids[t] = rng.choice(E, K, replace=False)
    pl = synth.placement_local_hot(E, E, int(rng.integers(1, min(E, 7) + 1)) if seed % 2 == 0 else 0)
    w = rng.uniform(0.1, 1.0, (T, K)).astype(np.float32)
    wl = synth.Workload("random", dtype, T, T - int(rng.integers(0, 3)), K, E, H, I, 0.0, pl,
                        {"uniform": synth.plan_uniform(pl, E)}, ids, w, seed)
    c = Case(wl, "uniform", 256)
    print(f"[random {dtype} seed {seed}] T={T} K={K} E={E} S={pl.slot_expert.size} H={H} I={I}", flush=True)
    y, _ = _run_forward(c)
    d = c.oracle_dispatch()
    assert np.array_equal(to_host(c.disp.slot_counts), d["slot_counts"])
    assert np.array_equal(to_host(c.disp.pair_row), d["pair_row"])
    loc, none = _local_rows(d, c.T_valid)
    assert np.all(y[none] == 0)
    r2 = np.random.default_rng(seed)
    pick = np.union1d(tile_sample(d, 256, r2), r2.choice(loc, min(len(loc), 400), replace=False))
    pick = pick[pick < c.T_valid]
    sel = np.zeros(T, np.uint8)
    sel[pick] = 1
    got = bf16_to_f64(y)
    ref = _oracle_y(c, d, "mirror", sel)
    err_m = mirror_err_rows(got, ref, pick)
    same = identical_share(got[pick], ref[pick])
    ref = _oracle_y(c, d, "exact", sel)
    err = rel_err_rows(got, ref, pick)
    print(f"[random {dtype} seed {seed}] sampled {len(pick)} tokens exact err={err:.2e} mirror err={err_m:.2e} "
          f"identical={same:.4f}")
    _check_many_rows(dtype, err, err_m, same)


@pytest.mark.parametrize("m_tile", [64, 128, 192, 256])
@pytest.mark.parametrize("dtype", ["bf16", "fp8", "fp8mx"])
def test_forward_stream_k_random_shapes(dtype, m_tile):
    """The stream-K kernel on random shapes: H and I multiples of 128 (at
    M 256, H an odd multiple of 128, where the large-tile kernels do not
    apply and stream-K takes the tile), 3..24 experts of 1..700 rows routed
    top-1..top-4, some with a second slot, a few padding tokens; stage 1
    bit-exact, y on a token sample (one row of every M-tile, every slot's
    last row and 400 random tokens) against the fp64 oracle in exact and
    mirror modes; tokens with no local pair exactly zero."""
    from paper_2608_13057_amd import synth

    rng = np.random.default_rng(1000 + 10 * m_tile + ["bf16", "fp8", "fp8mx"].index(dtype))
    H = int(rng.choice([128, 384, 640, 896] if m_tile == 256 else [128, 256, 512, 896]))
    I = int(rng.choice([128, 256, 384, 640]))
    E = int(rng.integers(3, 25))
    K = int(rng.integers(1, min(E, 4) + 1))
    counts = rng.integers(1, 700, E)
    T = int(counts.sum()) // K + 1
    ids = np.empty((T, K), np.int32)
    for t in range(T):
        ids[t] = rng.choice(E, K, replace=False)
    pl = synth.placement_local_hot(E, E, int(rng.integers(0, min(E, 5) + 1)))
    w = rng.uniform(0.1, 1.0, (T, K)).astype(np.float32)
    wl = synth.Workload("random_sk", dtype, T, T - int(rng.integers(0, 3)), K, E, H, I, 0.0, pl,
                        {"uniform": synth.plan_uniform(pl, E)}, ids, w, 7)
    c = Case(wl, "uniform", m_tile)
    print(f"[stream-K {dtype} M={m_tile}] T={T} K={K} E={E} S={pl.slot_expert.size} H={H} I={I}", flush=True)
    y, _ = _run_forward(c)
    d = c.oracle_dispatch()
    assert np.array_equal(to_host(c.disp.slot_counts), d["slot_counts"])
    assert np.array_equal(to_host(c.disp.pair_row), d["pair_row"])
    loc, none = _local_rows(d, c.T_valid)
    assert np.all(y[none] == 0)
    r2 = np.random.default_rng(m_tile)
    pick = np.union1d(tile_sample(d, m_tile, r2), r2.choice(loc, min(len(loc), 400), replace=False))
    pick = pick[pick < c.T_valid]
    sel = np.zeros(T, np.uint8)
    sel[pick] = 1
    got = bf16_to_f64(y)
    ref = _oracle_y(c, d, "mirror", sel)
    err_m = mirror_err_rows(got, ref, pick)
    same = identical_share(got[pick], ref[pick])
    ref = _oracle_y(c, d, "exact", sel)
    err = rel_err_rows(got, ref, pick)
    print(f"[stream-K {dtype} M={m_tile}] sampled {len(pick)} tokens exact err={err:.2e} mirror err={err_m:.2e} "
          f"identical={same:.4f}")
    _check_many_rows(dtype, err, err_m, same)


@pytest.mark.parametrize("name,m_tile", [("tiny", 64), ("tiny", 256), ("tiny_fp8", 128), ("tiny_fp8mx", 256)])
def test_stage_events_in_order(name, m_tile):
    """The eight stage events of the forward are recorded in stream order
    (stage 1, the gate/up GEMM kernel alone, the gate/up step, the down GEMM,
    the down step, stage 3), on the stream-K and the large-tile paths, with a
    null entry skipped; the outputs are those of a forward without events."""
    import torch
    from paper_2608_13057_amd import moe, synth

    wl = synth.make_workload(name)
    c = Case(wl, "uniform", m_tile)
    y0, _ = _run_forward(c)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(moe.STAGE_EVENTS)]
    y = torch.empty(c.wl.T, c.wl.H, dtype=torch.int16, device="cuda")
    moe.forward(c.shape, c.d_plan, c.d_ids, c.d_w, c.d_x, c.d_xs, c.d_weights, c.disp, y, c.ws, stage_events=ev)
    torch.cuda.synchronize()
    t = [ev[0].elapsed_time(e) for e in ev]
    assert all(b >= a for a, b in zip(t, t[1:])), t
    assert t[3] - t[2] > 0  # the gate/up GEMM kernel takes time
    assert np.array_equal(to_host(y), y0)
    ev2 = list(ev)
    ev2[2] = None  # a null entry is skipped
    moe.forward(c.shape, c.d_plan, c.d_ids, c.d_w, c.d_x, c.d_xs, c.d_weights, c.disp, y, c.ws, stage_events=ev2)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(y), y0)


@pytest.mark.parametrize("name", ["tiny", "tiny_fp8", "tiny_fp8mx"])
def test_forward_split_invariance_bit_exact(name):
    """The same batch under different splits of the replicated experts over
    their two local slots gives bit-identical y for every M-tile; across
    M-tiles served by the stream-K kernel (64 / 128 / 192, and 256 for fp8
    with fp32 scales) y is bit-identical too (its chunk boundaries do not
    depend on the tile).  bf16 and UE8M0 fp8 256-row tiles run the large-tile
    kernels, whose summation order is a different fixed one."""
    from paper_2608_13057_amd import synth

    wl = synth.make_workload(name)
    base = wl.plans["uniform"]
    outs = {}
    for m_tile in (64, 128, 192, 256):
        for sw in ([1] * 8, [1, 1, 1, 1, 1, 1, 0, 0], [0, 0, 1, 1, 1, 1, 1, 1], [3, 1, 1, 1, 1, 1, 1, 5]):
            wl.plans["p"] = synth.Plan(np.array(sw, np.uint32), base.remote_weight, base.remote_replicas, "p")
            c = Case(wl, "p", m_tile)
            outs.setdefault(m_tile, []).append(_run_forward(c)[0])
    for m_tile, os_ in outs.items():
        for o in os_[1:]:
            assert np.array_equal(o, os_[0]), f"plan changed y at M={m_tile}"
    same = (64, 128, 192, 256) if wl.dtype == "fp8" else (64, 128, 192)
    for m_tile in same[1:]:
        assert np.array_equal(outs[m_tile][0], outs[same[0]][0]), f"M={m_tile} differs from M={same[0]}"


@pytest.mark.parametrize("name,m_tile", [("tiny", 64), ("tiny", 256), ("tiny_fp8", 128), ("tiny_fp8mx", 64),
                                         ("tiny_fp8mx", 256)])
def test_forward_padding_rows_and_empty_batch(name, m_tile):
    """Graph-padding rows (t >= T_valid) and the empty batch, on the stream-K
    kernel and both large-tile kernels: padding rows and tokens without a
    local pair are exactly zero, the rest within tolerance; T_valid = 0
    leaves no tile and y all zero."""
    from paper_2608_13057_amd import synth

    wl = synth.make_workload(name)
    wl.topk_ids[60:] = 0  # degenerate routing on graph-padding rows
    print(f"[padding {name} M={m_tile}]", flush=True)
    c = Case(wl, "uniform", m_tile, T_valid=60)
    y, _ = _run_forward(c)
    d = c.oracle_dispatch()
    loc, none = _local_rows(d, 60)
    assert np.all(y[60:] == 0) and np.all(y[none] == 0)
    ref = _oracle_y(c, d)
    assert rel_err_rows(bf16_to_f64(y), ref, loc) <= TOL_EXACT[wl.dtype]
    c0 = Case(wl, "uniform", m_tile, T_valid=0)
    y0, _ = _run_forward(c0)
    assert np.all(y0 == 0)


@pytest.mark.parametrize("name,plan,m_tile", [("qwen3_decode_bf16", "token_balancing", 0),
                                              ("qwen3_decode_bf16", "token_balancing", 192),
                                              ("qwen3_decode_bf16", "token_balancing", 256),
                                              ("qwen3_decode_fp8", "uniform", 0), ("qwen3_decode_fp8", "replica_min", 0),
                                              ("dsv3_decode_fp8", "uniform", 0), ("dsv3_decode_fp8", "uniform", 128),
                                              ("qwen3_decode_fp8mx", "uniform", 0), ("qwen3_decode_fp8mx", "uniform", 256)])
def test_forward_full_size_sampled(name, plan, m_tile):
    """The full-size workload in the benchmark's launch configuration (M-tile
    0: the one bench.py picks); y is checked on a seeded sample of tokens (the
    oracle computes each one)."""
    from paper_2608_13057_amd import measure, synth

    wl = synth.make_workload(name)
    c = Case(wl, plan, m_tile or measure.auto_m_tile(wl))
    print(f"[forward {name} M={c.m_tile}] running", flush=True)
    y, st = _run_forward(c, timing=True)
    d = c.oracle_dispatch()
    loc, none = _local_rows(d, c.T_valid)
    rng = np.random.default_rng(0)
    pick = np.sort(rng.choice(loc, size=min(24, len(loc)), replace=False))
    sel = np.zeros(wl.T, np.uint8)
    sel[pick] = 1
    ref = _oracle_y(c, d, "exact", sel)
    err = rel_err_rows(bf16_to_f64(y), ref, pick)
    print(f"[forward {name}] sampled {len(pick)} tokens err={err:.2e}")
    assert err <= TOL_EXACT[wl.dtype]
    assert np.all(y[none] == 0)
    assert np.all((st > 0) == (d["slot_counts"] > 0))


@pytest.mark.parametrize("name,m_tile", [("qwen3_prefill_bf16", 256), ("qwen3_prefill_fp8", 128),
                                         ("qwen3_prefill_fp8mx", 256), ("qwen3_prefill_fp8mx", 128),
                                         ("qwen3_prefill_fp8", 256), ("qwen3_prefill_bf16", 128)])
def test_forward_prefill_tile_sampled(name, m_tile):
    """The prefill share (8192 tokens, top-8 of 128, 18 slots) at full size:
    stage 1 bit-exact inside the forward, and y on a token sample stratified
    by M-tile -- one random row of every M-tile of every activated slot (the
    second and later tiles of multi-tile slots included) plus each slot's
    last real row (its ragged tail) -- against the fp64 oracle; tokens with
    no local pair exactly zero."""
    from paper_2608_13057_amd import synth

    wl = synth.make_workload(name)
    c = Case(wl, "uniform", m_tile)
    print(f"[prefill {name} M={m_tile}] running", flush=True)
    y, st = _run_forward(c, timing=True)
    d = c.oracle_dispatch()
    assert np.array_equal(to_host(c.disp.slot_counts), d["slot_counts"])
    assert np.array_equal(to_host(c.disp.slot_offsets), d["slot_offsets"])
    assert np.array_equal(to_host(c.disp.pair_row), d["pair_row"])
    assert np.array_equal(to_host(c.disp.row_token)[: d["slot_offsets"][-1]], d["row_token"])
    loc, none = _local_rows(d, c.T_valid)
    assert np.all(y[none] == 0)
    pick = tile_sample(d, m_tile, np.random.default_rng(1))
    ntiles = int(sum(-(-int(n) // m_tile) for n in d["slot_counts"]))
    assert int((d["slot_counts"] > m_tile).sum()) >= 2  # slots spanning several tiles are covered
    sel = np.zeros(wl.T, np.uint8)
    sel[pick] = 1
    ref = _oracle_y(c, d, "exact", sel)
    err = rel_err_rows(bf16_to_f64(y), ref, pick)
    print(f"[prefill {name} M={m_tile}] {ntiles} tiles, sampled {len(pick)} tokens err={err:.2e}")
    assert err <= TOL_EXACT[wl.dtype]
    assert np.all((st > 0) == (d["slot_counts"] > 0))


@pytest.mark.parametrize("name,m_tile", [("tiny", 64), ("tiny", 256), ("tiny_fp8", 128), ("tiny_fp8mx", 64),
                                         ("tiny_fp8mx", 256)])
def test_forward_slot_table_bit_exact(name, m_tile):
    """Weights given per slot: each slot packed on its own (a 1-slot shape)
    into separately allocated tensors, reached through the slot table; y is
    bit-identical to the forward on the contiguous [S] weights (the stream-K
    and both large-tile kernels)."""
    import dataclasses

    import torch
    from paper_2608_13057_amd import moe, synth

    wl = synth.make_workload(name)
    c = Case(wl, "uniform", m_tile)
    y_ref, _ = _run_forward(c)
    one = dataclasses.replace(c.shape, S=1)
    slots, pad = [], []
    for s_ in range(wl.S):
        nat = moe.WeightTensors(to_dev(c.w13[s_:s_ + 1]), to_dev(c.w2[s_:s_ + 1]),
                                None if c.s13 is None else to_dev(c.s13[s_:s_ + 1]),
                                None if c.s2 is None else to_dev(c.s2[s_:s_ + 1]))
        slots.append(moe.pack_weights(one, nat))
        pad.append(torch.empty(4099, dtype=torch.uint8, device="cuda"))  # slots not adjacent in memory
    tab = moe.slot_table(slots)
    y = torch.empty(wl.T, wl.H, dtype=torch.int16, device="cuda")
    moe.forward(c.shape, c.d_plan, c.d_ids, c.d_w, c.d_x, c.d_xs, tab, c.disp, y, c.ws)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(y), y_ref)
    # replicas of one expert sharing a single packed copy (the use the table
    # is for): every slot points at the copy of the first slot of its expert
    se = wl.placement.slot_expert.tolist()
    first = {e: se.index(e) for e in se}
    assert len(first) < wl.S  # the workload has replicated experts
    shared = moe.slot_table([slots[first[e]] for e in se])
    y.fill_(0)
    moe.forward(c.shape, c.d_plan, c.d_ids, c.d_w, c.d_x, c.d_xs, shared, c.disp, y, c.ws)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(y), y_ref)


def _expect_packed(w, rows_of_block, nblk, fp8):
    """Packed layout: per slot, output block by output block, contraction
    step by step (128 bytes of every row), four 4 KB pieces (wavefront w:
    rows 32w..32w+31), each four 1 KB loads; load j, lane l holds 16-byte
    chunk c(j, l) of row 32w + (l % 32): bf16 c = 2j + l // 32, fp8
    c = 4 (j // 2) + 2 (l // 32) + j % 2."""
    S_, R, C = w.shape
    per = 16 // w.itemsize
    ch = w.reshape(S_, R, C // per, per)  # 16-byte chunks
    KT = C // (128 // w.itemsize)
    out = np.empty((S_, nblk, KT, 4, 4, 64, per), w.dtype)
    for nb in range(nblk):
        rows = rows_of_block(nb)
        for kt in range(KT):
            for wv in range(4):
                for j in range(4):
                    for l in range(64):
                        c = 4 * (j // 2) + 2 * (l // 32) + j % 2 if fp8 else 2 * j + l // 32
                        out[:, nb, kt, wv, j, l] = ch[:, rows[32 * wv + l % 32], kt * 8 + c]
    return out.reshape(S_, -1)


def _gu_rows(I):
    def rows(nb):  # 16-row groups alternate gate and the matching up rows
        return [(I if (r // 16) % 2 else 0) + nb * 64 + (r // 32) * 16 + r % 16 for r in range(128)]
    return rows


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_pack_layout(dtype):
    """The packed weight layout (MFMA operand order, one wavefront's 32 rows
    per 4 KB piece); gate/up blocks pair gate rows n..n+63 with up rows
    I+n..I+n+63, interleaved in groups of 16."""
    import torch
    from paper_2608_13057_amd import moe

    rng = np.random.default_rng(3)
    S, H, I = 2, 256, 384
    fp8 = dtype == "fp8"
    shape = moe.MoEShape(T=4, K=1, E=2, S=S, H=H, I=I, dtype=dtype)
    if fp8:
        w13 = rng.integers(0, 256, size=(S, 2 * I, H), dtype=np.uint8)
        w2 = rng.integers(0, 256, size=(S, H, I), dtype=np.uint8)
        s13 = np.ones((S, 2 * I // 128, H // 128), np.float32)
        s2 = np.ones((S, H // 128, I // 128), np.float32)
        nat = moe.WeightTensors(to_dev(w13), to_dev(w2), to_dev(s13), to_dev(s2))
    else:
        w13 = rng.integers(0, 2**16, size=(S, 2 * I, H), dtype=np.uint16)
        w2 = rng.integers(0, 2**16, size=(S, H, I), dtype=np.uint16)
        nat = moe.WeightTensors(to_dev(w13), to_dev(w2))
    pk = moe.pack_weights(shape, nat)
    torch.cuda.synchronize()
    e13 = _expect_packed(w13, _gu_rows(I), I // 64, fp8)
    e2 = _expect_packed(w2, lambda nb: list(range(nb * 128, nb * 128 + 128)), H // 128, fp8)
    assert np.array_equal(to_host(pk.w13).reshape(S, -1).view(w13.dtype), e13)
    assert np.array_equal(to_host(pk.w2).reshape(S, -1).view(w2.dtype), e2)


def test_pack_fp8_scales():
    """Packed fp8 weight scales: 4 words per (output block, contraction step);
    gate/up {gate-row block scale, up-row block scale, 0, 0} for the block
    pairing gate rows 64n.. with up rows I+64n..; down {block scale, 0, 0, 0}."""
    import torch
    from paper_2608_13057_amd import moe

    rng = np.random.default_rng(4)
    S, H, I = 3, 384, 640
    shape = moe.MoEShape(T=4, K=1, E=3, S=S, H=H, I=I, dtype="fp8")
    w13 = rng.integers(0, 256, size=(S, 2 * I, H), dtype=np.uint8)
    w2 = rng.integers(0, 256, size=(S, H, I), dtype=np.uint8)
    s13 = rng.random((S, 2 * I // 128, H // 128)).astype(np.float32)
    s2 = rng.random((S, H // 128, I // 128)).astype(np.float32)
    pk = moe.pack_weights(shape, moe.WeightTensors(to_dev(w13), to_dev(w2), to_dev(s13), to_dev(s2)))
    torch.cuda.synchronize()
    e13 = np.zeros((S, I // 64, H // 128, 4), np.float32)
    for nb in range(I // 64):
        e13[:, nb, :, 0] = s13[:, nb // 2, :]
        e13[:, nb, :, 1] = s13[:, I // 128 + nb // 2, :]
    e2 = np.zeros((S, H // 128, I // 128, 4), np.float32)
    e2[..., 0] = s2
    assert np.array_equal(to_host(pk.w13_scale), e13)
    assert np.array_equal(to_host(pk.w2_scale), e2)
