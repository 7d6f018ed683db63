"""GPU parity of stage 1 (tempo_moe_dispatch) against the oracle: bit-exact
counts, offsets, permutation and gathered rows.  Runs through the C ABI."""
import numpy as np
import pytest

from helpers import Case, to_dev, to_host

pytestmark = pytest.mark.gpu


def _compare(case, d_ref, check_rows=True, check_scales=None):
    """Bit-exact stage-1 outputs; check_rows: the permuted rows (and fp8
    scales); check_scales (default: with check_rows): the permuted fp8 scales
    alone."""
    import torch

    torch.cuda.synchronize()
    D = case.disp
    used = int(d_ref["slot_offsets"][-1])
    assert np.array_equal(to_host(D.expert_counts), d_ref["expert_counts"])
    assert np.array_equal(to_host(D.slot_counts), d_ref["slot_counts"])
    assert np.array_equal(to_host(D.slot_offsets), d_ref["slot_offsets"])
    assert np.array_equal(to_host(D.row_token)[:used], d_ref["row_token"])
    assert np.array_equal(to_host(D.pair_row), d_ref["pair_row"])
    rt = d_ref["row_token"]
    real = np.nonzero(rt >= 0)[0]
    if check_rows:
        xp = to_host(D.x_perm)
        x = case.x
        assert np.array_equal(xp[real], x[rt[real]])
    if (check_rows if check_scales is None else check_scales) and case.dtype == "fp8":
        xps = to_host(D.x_perm_scale)  # block-major [H/128, row_cap]
        assert np.array_equal(xps[:, real].T, case.xs[rt[real]])


@pytest.mark.parametrize("name", ["tiny", "qwen3_decode_bf16", "qwen3_decode_fp8", "dsv3_decode_fp8",
                                  "qwen3_prefill_bf16", "qwen3_prefill_fp8"])
@pytest.mark.parametrize("m_tile", [64, 128, 192, 256])
def test_dispatch_workloads_bit_exact(name, m_tile):
    from paper_2608_13057_amd import moe, synth

    wl = synth.make_workload(name)
    for plan in wl.plans:
        print(f"[dispatch] {name} plan={plan} m_tile={m_tile}", flush=True)
        c = Case(wl, plan, m_tile, weights=False)
        moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
        _compare(c, c.oracle_dispatch())
        assert moe.device_error(c.ws) == 0


def _random_workload(rng, T, K, E, S, dtype="bf16", H=128):
    from paper_2608_13057_amd import synth

    ids = rng.integers(0, E, size=(T, K)).astype(np.int32)
    ids[rng.random((T, K)) < 0.1] = -1
    se = rng.integers(0, E, size=S).astype(np.int32)
    sw = rng.integers(0, 4, size=S).astype(np.uint32)
    rw = (rng.integers(0, 3, size=E) * (rng.random(E) < 0.5)).astype(np.uint32)
    rr = np.where(rw > 0, rng.integers(1, 3, size=E), (rng.random(E) < 0.2).astype(np.int64)).astype(np.int32)
    pl = synth.Placement(se, np.zeros(E, np.int32), [[0] for _ in range(E)])
    plan = synth.Plan(sw, rw, rr, "rand")
    w = rng.random((T, K)).astype(np.float32)
    return synth.Workload("rand", dtype, T, T, K, E, H, 128, 1.0, pl, {"rand": plan}, ids, w, int(rng.integers(1 << 30)))


@pytest.mark.parametrize("seed", range(16))
def test_dispatch_random_bit_exact(seed):
    """Random small shapes: ragged block tails, several blocks of 1024 pairs,
    padding rows (T_valid < T), zero-weight rows, remote shares, repeated ids."""
    from paper_2608_13057_amd import moe

    rng = np.random.default_rng(100 + seed)
    T = int(rng.choice([1, 3, 37, 300, 700, 2100, 2500]))
    K = int(rng.integers(1, 9))
    E = int(rng.integers(max(K, 1), 300))
    S = int(rng.integers(1, 40))
    wl = _random_workload(rng, T, K, E, S, "bf16" if seed % 2 == 0 else "fp8")
    T_valid = int(rng.integers(0, T + 1))
    m_tile = (64, 128, 192, 256)[seed % 4]
    print(f"[dispatch-rand] seed={seed} T={T} K={K} E={E} S={S} Tv={T_valid} M={m_tile}", flush=True)
    c = Case(wl, "rand", m_tile, weights=False, T_valid=T_valid)
    moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
    _compare(c, c.oracle_dispatch())


def test_dispatch_bad_ids_flagged_and_dropped():
    from paper_2608_13057_amd import moe

    rng = np.random.default_rng(5)
    wl = _random_workload(rng, 200, 4, 20, 8)
    wl.topk_ids[3, 1] = 20
    wl.topk_ids[50, 0] = -5
    c = Case(wl, "rand", 64, weights=False)
    moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
    ref = c.oracle_dispatch()
    _compare(c, ref)
    assert ref["err"] == moe._lib.TEMPO_DERR_BAD_ID
    assert moe.device_error(c.ws) == moe._lib.TEMPO_DERR_BAD_ID
    assert moe.device_error(c.ws) == 0  # read clears


def test_dispatch_bad_slot_and_overflow_flags():
    from paper_2608_13057_amd import moe

    rng = np.random.default_rng(6)
    wl = _random_workload(rng, 64, 2, 10, 4)
    wl.placement.slot_expert[:] = [0, 0, 12, 3]
    wl.plans["rand"].slot_weight[:] = [2**31, 2**31, 1, 1]
    wl.plans["rand"].remote_weight[0] = 0
    c = Case(wl, "rand", 64, weights=False)
    moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
    ref = c.oracle_dispatch()
    _compare(c, ref)
    bits = moe.device_error(c.ws)
    assert bits == ref["err"] == (moe._lib.TEMPO_DERR_BAD_SLOT_EXPERT | moe._lib.TEMPO_DERR_WEIGHT_OVERFLOW)


def test_dispatch_empty_batch_and_cumulative_counter():
    import torch
    from paper_2608_13057_amd import moe, synth

    wl = synth.make_workload("tiny")
    c = Case(wl, "uniform", 64, weights=False, T_valid=0)
    moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
    _compare(c, c.oracle_dispatch())
    # cumulative counter wraps modulo 2^32
    c2 = Case(wl, "uniform", 64, weights=False)
    c2.disp.cum_counts = to_dev(np.array([2**32 - 5, 7, 0, 1, 2**31, 3], np.uint32))
    before = to_host(c2.disp.cum_counts).view(np.uint32).copy()
    moe.dispatch(c2.shape, c2.d_plan, c2.d_ids, c2.d_x, c2.d_xs, c2.disp, c2.ws)
    torch.cuda.synchronize()
    after = to_host(c2.disp.cum_counts).view(np.uint32)
    ref = c2.oracle_dispatch()
    assert np.array_equal((after - before).astype(np.uint32), ref["expert_counts"].astype(np.uint32))


def _forward(c):
    import torch
    from paper_2608_13057_amd import moe

    y = torch.empty(c.wl.T, c.wl.H, dtype=torch.int16, device="cuda")
    moe.forward(c.shape, c.d_plan, c.d_ids, c.d_w, c.d_x, c.d_xs, c.d_weights, c.disp, y, c.ws)
    torch.cuda.synchronize()


@pytest.mark.parametrize("seed", range(12))
def test_forward_stage1_bit_exact(seed):
    """Stage 1 as the forward runs it: for decode-sized bf16 batches one
    workgroup does all of it (x_perm stays unwritten, the gate/up GEMM
    gathers the rows).  Bit-exact counts, offsets and permutation across one
    to eight rounds of 1024 pairs and beyond, more than 64 slots (the
    block-wide plan), padding tokens, bad ids and every M-tile; the
    cumulative counter advances by n_e."""
    from paper_2608_13057_amd import moe

    rng = np.random.default_rng(700 + seed)
    T = int(rng.choice([1, 37, 300, 1024, 1500]))
    K = int(rng.integers(1, 9))
    E = int(rng.integers(K, 300))
    S = int(rng.choice([5, 40, 90]))
    wl = _random_workload(rng, T, K, E, S, "bf16")
    if seed % 3 == 0:
        wl.topk_ids[0, 0] = E  # out of range: flagged and dropped
    T_valid = int(rng.integers(0, T + 1)) if seed % 2 else T
    m_tile = (64, 128, 192, 256)[seed % 4]
    print(f"[forward-stage1] seed={seed} T={T} K={K} E={E} S={S} Tv={T_valid} M={m_tile}", flush=True)
    c = Case(wl, "rand", m_tile, T_valid=T_valid)
    c.disp.cum_counts = to_dev(rng.integers(0, 2**32, size=E, dtype=np.uint64).astype(np.uint32))
    before = to_host(c.disp.cum_counts).view(np.uint32).copy()
    _forward(c)
    ref = c.oracle_dispatch()
    _compare(c, ref, check_rows=False)
    after = to_host(c.disp.cum_counts).view(np.uint32)
    assert np.array_equal((after - before).astype(np.uint32), ref["expert_counts"].astype(np.uint32))
    assert moe.device_error(c.ws) == ref["err"]


@pytest.mark.parametrize("name", ["tiny", "qwen3_decode_bf16", "dsv3_decode_fp8", "qwen3_decode_fp8"])
def test_forward_stage1_workloads_bit_exact(name):
    """Stage 1 as the forward runs it on the decode shares.  fp8 with fp32
    scales: the GEMM gathers the rows and reads the scales permuted, which
    stage 1 copies (2048 pairs of the DeepSeek-V3 share through the single
    workgroup and a scale-copy launch; 8192 pairs of the Qwen3 share through
    count + place)."""
    from paper_2608_13057_amd import measure, synth

    wl = synth.make_workload(name)
    for plan in wl.plans:
        print(f"[forward-stage1] {name} plan={plan}", flush=True)
        c = Case(wl, plan, measure.auto_m_tile(wl))
        _forward(c)
        _compare(c, c.oracle_dispatch(), check_rows=False, check_scales=True)


@pytest.mark.parametrize("seed", range(10))
def test_snap_split_bit_exact(seed):
    """The tile-aware split (TEMPO_PLAN_SNAP_TILES) against the oracle's
    snapped mode, through both stage-1 paths: the dispatch entry point (two
    launches, rows gathered into x_perm) and the forward (one workgroup for
    decode-sized bf16 batches)."""
    from paper_2608_13057_amd import moe

    rng = np.random.default_rng(900 + seed)
    T = int(rng.choice([5, 100, 700, 1500, 3000]))
    K = int(rng.integers(1, 9))
    E = int(rng.integers(K, 40))  # few experts: many pairs per expert, several tiles
    S = int(rng.choice([4, 20, 70]))
    wl = _random_workload(rng, T, K, E, S, "bf16" if seed % 3 else "fp8")
    T_valid = int(rng.integers(0, T + 1)) if seed % 2 else T
    m_tile = (64, 128, 192, 256)[seed % 4]
    print(f"[snap] seed={seed} T={T} K={K} E={E} S={S} Tv={T_valid} M={m_tile} {wl.dtype}", flush=True)
    c = Case(wl, "rand", m_tile, T_valid=T_valid, snap=True)
    ref = c.oracle_dispatch()
    moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
    _compare(c, ref)
    _forward(c)
    _compare(c, ref, check_rows=False)


def test_snap_flag_validated():
    from paper_2608_13057_amd import _lib, moe, synth

    wl = synth.make_workload("tiny")
    c = Case(wl, "uniform", 64, weights=False)
    pl = c.d_plan.c()
    pl.flags = 4  # no such flag
    sh, do = c.shape.c(), c.disp.c()
    rc = _lib.load().tempo_moe_dispatch(moe.ctypes.byref(sh), moe.ctypes.byref(pl), moe._ptr(c.d_ids), moe._ptr(c.d_x),
                                        None, moe.ctypes.byref(do), c.ws.ptr, c.ws.nbytes, None)
    assert rc == _lib.TEMPO_EINVAL  # refused on the host, nothing launched


@pytest.mark.parametrize("seed", range(10))
def test_sampled_dispatch_bit_exact(seed):
    """Sampled replicas (TEMPO_PLAN_SAMPLE, the deployed semantics) against
    the oracle's sampled mode: the dispatch entry point (rows gathered into
    x_perm by the row-copy launch) and the forward; bf16 and fp8; ragged
    batches, padding tokens, zero-weight rows, remote shares."""
    from paper_2608_13057_amd import moe

    rng = np.random.default_rng(1100 + seed)
    T = int(rng.choice([1, 37, 300, 1024]))
    K = int(rng.integers(1, 9))
    E = int(rng.integers(K, 200))
    S = int(rng.choice([3, 30, 90]))
    wl = _random_workload(rng, T, K, E, S, "bf16" if seed % 2 == 0 else "fp8")
    T_valid = int(rng.integers(0, T + 1)) if seed % 3 else T
    m_tile = (64, 128, 192, 256)[seed % 4]
    key = int(rng.integers(0, 2**63))
    print(f"[sample] seed={seed} T={T} K={K} E={E} S={S} Tv={T_valid} M={m_tile} {wl.dtype} key={key}", flush=True)
    c = Case(wl, "rand", m_tile, T_valid=T_valid, sample_seed=key)
    ref = c.oracle_dispatch()
    moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
    _compare(c, ref)
    assert moe.device_error(c.ws) == ref["err"]
    _forward(c)
    _compare(c, ref, check_rows=False)


def test_sampled_dispatch_limits():
    """Sampling is offered up to 8192 pairs and 256 experts; beyond that the
    call is refused on the host; snapping and sampling together are invalid."""
    from paper_2608_13057_amd import _lib, moe

    rng = np.random.default_rng(7)
    wl = _random_workload(rng, 2048, 8, 64, 8)  # 16384 pairs
    c = Case(wl, "rand", 64, weights=False, sample_seed=1)
    with pytest.raises(_lib.TempoError) as ex:
        moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
    assert ex.value.code == _lib.TEMPO_EUNSUPPORTED
    c2 = Case(_random_workload(rng, 64, 2, 10, 4), "rand", 64, weights=False, sample_seed=1)
    pl = c2.d_plan.c()
    pl.flags = _lib.TEMPO_PLAN_SAMPLE | _lib.TEMPO_PLAN_SNAP_TILES
    sh, do = c2.shape.c(), c2.disp.c()
    rc = _lib.load().tempo_moe_dispatch(moe.ctypes.byref(sh), moe.ctypes.byref(pl), moe._ptr(c2.d_ids),
                                        moe._ptr(c2.d_x), None, moe.ctypes.byref(do), c2.ws.ptr, c2.ws.nbytes, None)
    assert rc == _lib.TEMPO_EINVAL


@pytest.mark.parametrize("name", ["qwen3_decode_bf16", "dsv3_decode_fp8"])
def test_counts_solver_plan_loop(name):
    """counts -> plan -> kernel: stage 1 on the GPU collects n_e; the
    tempo_fast solver splits them over an 8-GPU placement in which GPU 0
    holds this workload's slots; the plan it emits for GPU 0, run through
    stage 1 on the GPU again, places exactly the solver's shares."""
    import torch
    from paper_2608_13057_amd import moe, solver, synth

    wl = synth.make_workload(name)
    c = Case(wl, next(iter(wl.plans)), 64, weights=False)
    moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
    n = to_host(c.disp.expert_counts).astype(np.int64)
    se = wl.placement.slot_expert
    R = np.zeros((wl.E, 8), bool)
    R[se, 0] = True
    R[np.arange(wl.E), 1 + np.arange(wl.E) % 7] = True
    x = solver.tempo_fast(n, R, solver.CostModel(41.6, 5.61, 14.1, 0.1122))
    sw, rw, rr = solver.plan_for_gpu(x, se, 0)
    c.d_plan = moe.PlanTensors(to_dev(se), to_dev(sw), to_dev(rw), to_dev(rr))
    moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
    torch.cuda.synchronize()
    sc = to_host(c.disp.slot_counts)
    for e in np.unique(se):
        assert sc[se == e].sum() == x[e, 0], e
    assert sc.sum() == x[:, 0].sum()


def test_dispatch_at_the_limits():
    """The kernels' size limits: 1024 experts, 256 slots and top-32 routing
    through the multi-block stage 1 (scanned prefixes, the block-wide plan);
    exactly 8192 pairs with 256 experts and 256 slots through the single
    workgroup, in the split and the sampled modes, via the dispatch entry
    point and the forward."""
    from paper_2608_13057_amd import moe

    rng = np.random.default_rng(2024)
    wl = _random_workload(rng, 300, 32, 1024, 256)
    c = Case(wl, "rand", 256, weights=False)
    print("[limits] E=1024 S=256 K=32 T=300 M=256", flush=True)
    moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
    _compare(c, c.oracle_dispatch())
    wl = _random_workload(rng, 256, 32, 256, 256)
    for key in (None, 77):
        print(f"[limits] E=256 S=256 K=32 T=256 M=64 sample={key}", flush=True)
        c = Case(wl, "rand", 64, sample_seed=key)
        ref = c.oracle_dispatch()
        moe.dispatch(c.shape, c.d_plan, c.d_ids, c.d_x, c.d_xs, c.disp, c.ws)
        _compare(c, ref)
        _forward(c)
        _compare(c, ref, check_rows=False)
