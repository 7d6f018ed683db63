"""Pins for the stage-1 oracle (per-expert counts, plan split, padded groups,
stable permutation).  The definition follows the fixed-charge problem of
Sec. 3.1 (n_e, R(e), shares x_{e,g}, activations z_{e,g}), the M-tiles of
Sec. 2.2 / Eq. 2 and the integration semantics of Sec. 4.4 (padding rows
masked, rows renormalised at use, zero-sum rows uniform over replicas).

Nothing here re-types the oracle's formulas: the checks are invariants the
definition implies, a special case that reduces to numpy's stable argsort,
proportional-share bounds, and hand-worked tiny cases."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle


def _rand_case(rng, T, K, E, S, M, p_bad=0.0, p_neg=0.1, remote=True, zero_w=0.1):
    ids = rng.integers(0, E, size=(T, K)).astype(np.int32)
    ids[rng.random((T, K)) < p_neg] = -1
    if p_bad:
        bad = rng.random((T, K)) < p_bad
        ids[bad] = rng.choice([E, E + 3, -2, -7], size=bad.sum())
    se = rng.integers(0, E, size=S).astype(np.int32)
    sw = rng.integers(0, 4, size=S).astype(np.uint32)
    sw[rng.random(S) < zero_w] = 0
    rw = (rng.integers(0, 3, size=E) * (rng.random(E) < 0.5)).astype(np.uint32) if remote else np.zeros(E, np.uint32)
    rr = np.where(rw > 0, rng.integers(1, 3, size=E), (rng.random(E) < 0.2).astype(np.int64)).astype(np.int32)
    if not remote:
        rr[:] = 0
    T_valid = int(rng.integers(0, T + 1))
    return ids, T_valid, se, sw, rw, rr


def _check_invariants(ids, T_valid, E, M, se, sw, rw, rr, d):
    T, K = ids.shape
    S = len(se)
    ec, sc, so, rt, pr = d["expert_counts"], d["slot_counts"], d["slot_offsets"], d["row_token"], d["pair_row"]
    valid = np.zeros((T, K), bool)
    valid[:T_valid] = (ids[:T_valid] >= 0) & (ids[:T_valid] < E)
    # counts over valid pairs only (padding rows and bad ids excluded)
    assert np.array_equal(ec, np.bincount(ids[valid], minlength=E))
    # padded sizes and offsets
    P = so[1:] - so[:-1]
    assert so[0] == 0
    assert np.all(P % M == 0) and np.all(P >= sc) and np.all(P - sc < M)
    assert np.all((P == 0) == (sc == 0))
    # rows: inverse maps; rows of a slot in ascending pair index
    assert len(rt) == so[-1]
    placed = pr.reshape(-1) >= 0
    assert np.all(valid.reshape(-1)[placed]), "an invalid pair was placed"
    rows = pr.reshape(-1)[placed]
    assert len(np.unique(rows)) == len(rows), "two pairs share a row"
    pidx = np.nonzero(placed)[0]
    assert np.array_equal(rt[rows], pidx // K)
    assert (rt >= 0).sum() == len(rows)
    for s in range(S):
        lo, c = so[s], sc[s]
        seg = rt[lo:so[s + 1]]
        assert np.all(seg[:c] >= 0) and np.all(seg[c:] == -1)
        # pair indices of the slot's rows, ascending
        inv = {r: p for r, p in zip(rows.tolist(), pidx.tolist())}
        ps = [inv[r] for r in range(lo, lo + c)]
        assert ps == sorted(ps)
        assert all(ids.reshape(-1)[p] == se[s] for p in ps)
    # per expert: local counts + remote remainder = n_e; within one of the
    # proportional share; only experts with a remote entry leave pairs unplaced
    for e in range(E):
        loc = [s for s in range(S) if se[s] == e]
        has_remote = rw[e] > 0 or rr[e] > 0
        n = ec[e]
        placed_e = sum(int(sc[s]) for s in loc)
        if not loc:
            assert placed_e == 0
            continue
        if not has_remote:
            assert placed_e == n
        w = [int(sw[s]) for s in loc] + ([int(rw[e])] if has_remote else [])
        W = sum(w)
        if W == 0:
            w = [1] * len(loc) + ([int(rr[e])] if has_remote else [])
            W = sum(w)
        for j, s in enumerate(loc):
            assert abs(int(sc[s]) - n * w[j] / W) < 1.0 + 1e-12
        assert placed_e <= n


@settings(max_examples=300, deadline=None)
@given(st.integers(0, 2**31 - 1), st.integers(1, 40), st.integers(1, 4), st.integers(1, 9), st.integers(1, 10),
       st.sampled_from([1, 2, 4, 16, 32, 128]))
def test_invariants_random(seed, T, K, E, S, M):
    rng = np.random.default_rng(seed)
    ids, T_valid, se, sw, rw, rr = _rand_case(rng, T, K, E, S, M)
    d = oracle.dispatch(ids, T_valid, E, M, se, sw, rw, rr)
    assert d["err"] == 0
    _check_invariants(ids, T_valid, E, M, se, sw, rw, rr, d)


@settings(max_examples=100, deadline=None)
@given(st.integers(0, 2**31 - 1), st.integers(1, 30), st.integers(1, 3), st.integers(1, 6), st.integers(1, 6))
def test_bad_ids_dropped_and_flagged(seed, T, K, E, S):
    rng = np.random.default_rng(seed)
    ids, T_valid, se, sw, rw, rr = _rand_case(rng, T, K, E, S, 4, p_bad=0.2)
    d = oracle.dispatch(ids, T_valid, E, 4, se, sw, rw, rr)
    bad = ((ids[:T_valid] < -1) | (ids[:T_valid] >= E)).any()
    assert bool(d["err"] & oracle.ERR_BAD_ID) == bool(bad)
    _check_invariants(ids, T_valid, E, 4, se, sw, rw, rr, d)


def test_single_replica_is_stable_argsort():
    """One local slot per expert, nothing remote: the non-padding rows in
    slot order are numpy's stable argsort of the pairs by expert."""
    rng = np.random.default_rng(7)
    for trial in range(50):
        E = int(rng.integers(1, 12))
        T, K, M = int(rng.integers(1, 60)), int(rng.integers(1, 5)), int(rng.choice([1, 8, 64]))
        ids = rng.integers(0, E, size=(T, K)).astype(np.int32)
        ids[rng.random((T, K)) < 0.1] = -1
        se = rng.permutation(E).astype(np.int32)  # slot order != expert order
        d = oracle.dispatch(ids, T, E, M, se, np.ones(E, np.uint32), np.zeros(E, np.uint32), np.zeros(E, np.int32))
        flat = ids.reshape(-1)
        key = np.array([np.nonzero(se == e)[0][0] if e >= 0 else 10**9 for e in flat])
        order = np.argsort(key, kind="stable")
        order = order[key[order] < 10**9]
        rt = d["row_token"]
        inv = {r: p for p, r in enumerate(d["pair_row"].reshape(-1).tolist()) if r >= 0}
        got = [inv[r] for r in range(len(rt)) if rt[r] >= 0]
        assert got == order.tolist()


def test_even_halves_and_uniform_fallback():
    ids = np.zeros((10, 1), np.int32)  # expert 0 gets 10 pairs
    se = np.array([0, 0], np.int32)
    z = np.zeros(1, np.uint32)
    d = oracle.dispatch(ids, 10, 1, 4, se, np.array([1, 1], np.uint32), z, np.zeros(1, np.int32))
    assert d["slot_counts"].tolist() == [5, 5]
    # first half of the pairs (ascending index) on the first slot
    assert d["pair_row"].reshape(-1).tolist() == [0, 1, 2, 3, 4, 8, 9, 10, 11, 12]
    assert d["slot_offsets"].tolist() == [0, 8, 16]
    # a row that sums to zero is renormalised to uniform over its replicas
    d0 = oracle.dispatch(ids, 10, 1, 4, se, np.array([0, 0], np.uint32), z, np.zeros(1, np.int32))
    assert d0["slot_counts"].tolist() == [5, 5] and d0["err"] == 0
    # zero row with a remote replica: uniform over 2 local + 2 remote replicas
    d1 = oracle.dispatch(ids, 10, 1, 4, se, np.array([0, 0], np.uint32), z, np.array([2], np.int32))
    assert d1["slot_counts"].tolist() == [2, 3]
    # weights are renormalised at use: scaling a row changes nothing
    d2 = oracle.dispatch(ids, 10, 1, 4, se, np.array([7, 7], np.uint32), z, np.zeros(1, np.int32))
    assert np.array_equal(d2["pair_row"], d["pair_row"])


def test_hand_worked_three_way_split():
    """n = 7 pairs of expert 1 over local slots with weights 1, 2 and a remote
    share of 4 (W = 7): shares are exactly 1, 2, 4.  Remote pairs are the
    last four by pair index."""
    ids = np.array([[1, 0], [1, 1], [0, 1], [1, 1], [1, 2]], np.int32)  # expert-1 pairs p = 0,2,3,5,6,7,8
    se = np.array([1, 0, 1], np.int32)
    d = oracle.dispatch(ids, 5, 3, 2, se, np.array([1, 5, 2], np.uint32), np.array([0, 4, 0], np.uint32),
                        np.array([0, 1, 0], np.int32))
    assert d["expert_counts"].tolist() == [2, 7, 1]
    assert d["slot_counts"].tolist() == [1, 2, 2]
    assert d["slot_offsets"].tolist() == [0, 2, 4, 6]
    pr = d["pair_row"].reshape(-1).tolist()
    assert pr[0] == 0  # rank 0 -> slot 0
    assert pr[2] == 4 and pr[3] == 5  # ranks 1,2 -> slot 2 (rows 4, 5)
    assert pr[5] == pr[6] == pr[7] == pr[8] == -1  # ranks 3..6 -> remote
    assert pr[1] == 2 and pr[4] == 3  # expert 0 pairs on slot 1
    assert pr[9] == -1  # expert 2 has no slot
    assert d["row_token"].tolist() == [0, -1, 0, 2, 1, 1]


def test_padding_rows_masked_and_cumulative_counter_wraps():
    rng = np.random.default_rng(3)
    ids = rng.integers(0, 4, size=(12, 2)).astype(np.int32)
    ids2 = ids.copy()
    ids2[8:] = 0  # degenerate routing on graph-padding rows ("phantom hot expert")
    se = np.arange(4, dtype=np.int32)
    args = (np.ones(4, np.uint32), np.zeros(4, np.uint32), np.zeros(4, np.int32))
    a = oracle.dispatch(ids, 8, 4, 16, se, *args)
    b = oracle.dispatch(ids2, 8, 4, 16, se, *args)
    for k in ("expert_counts", "slot_counts", "slot_offsets", "row_token", "pair_row"):
        assert np.array_equal(a[k], b[k])
    cum = np.array([2**32 - 3, 0, 5, 2**32 - 1], np.uint32)
    c = oracle.dispatch(ids, 8, 4, 16, se, *args, cum_counts=cum)
    expect = (cum.astype(np.uint64) + a["expert_counts"].astype(np.uint64)) % 2**32
    assert np.array_equal(c["cum_counts"], expect.astype(np.uint32))
    # wrap-safe window difference recovers the window's counts
    assert np.array_equal((c["cum_counts"] - cum).astype(np.uint32), a["expert_counts"].astype(np.uint32))


def test_empty_and_degenerate():
    se = np.array([0, 1], np.int32)
    args = (np.ones(2, np.uint32), np.zeros(2, np.uint32), np.zeros(2, np.int32))
    d = oracle.dispatch(np.zeros((5, 2), np.int32), 0, 2, 8, se, *args)  # T_valid = 0
    assert d["slot_counts"].tolist() == [0, 0] and d["slot_offsets"].tolist() == [0, 0, 0]
    assert np.all(d["pair_row"] == -1) and len(d["row_token"]) == 0
    d = oracle.dispatch(np.full((5, 2), -1, np.int32), 5, 2, 8, se, *args)  # all dropped
    assert d["expert_counts"].tolist() == [0, 0] and d["err"] == 0
    # a bad slot_expert is flagged and that slot receives nothing
    d = oracle.dispatch(np.zeros((5, 1), np.int32), 5, 2, 8, np.array([0, 9], np.int32), *args)
    assert d["err"] & oracle.ERR_BAD_SLOT_EXPERT and d["slot_counts"].tolist() == [5, 0]
    # plan weights that overflow 32 bits: flagged, split uniformly
    d = oracle.dispatch(np.zeros((6, 1), np.int32), 6, 2, 8, np.array([0, 0], np.int32),
                        np.array([2**31, 2**31], np.uint32), np.zeros(2, np.uint32), np.zeros(2, np.int32))
    assert d["err"] & oracle.ERR_WEIGHT_OVERFLOW and d["slot_counts"].tolist() == [3, 3]


def test_tile_count_matches_paper_staircase():
    """Eq. 2: T = sum ceil(n/128); 1..128 tokens take one tile, 129 two."""
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))["tile_count"]
    for n, tiles in g["cases"]:
        d = oracle.dispatch(np.zeros((n, 1), np.int32), n, 1, g["m_tile"], np.array([0], np.int32),
                            np.ones(1, np.uint32), np.zeros(1, np.uint32), np.zeros(1, np.int32))
        assert d["slot_offsets"][-1] // g["m_tile"] == tiles


def test_synthetic_workloads_dispatch_invariants():
    from paper_2608_13057_amd import synth
    for name in synth.WORKLOADS:
        wl = synth.make_workload(name, T=256 if "prefill" in name else None)
        for plan in wl.plans.values():
            for M in (32, 128):
                d = oracle.dispatch(wl.topk_ids, wl.T_valid, wl.E, M, wl.placement.slot_expert, plan.slot_weight,
                                    plan.remote_weight, plan.remote_replicas)
                assert d["err"] == 0
                _check_invariants(wl.topk_ids, wl.T_valid, wl.E, M, wl.placement.slot_expert, plan.slot_weight,
                                  plan.remote_weight, plan.remote_replicas, d)


# ---- tile-aware split (Sec. 2.2 after Eq. 2: partial splits snapped to
# tile boundaries).  Reading: every boundary other than n_e moves to the
# nearest multiple of M (halves up), capped at n_e. ----

@settings(max_examples=200, deadline=None)
@given(st.integers(0, 2**31 - 1), st.integers(1, 60), st.integers(1, 4), st.integers(1, 9), st.integers(1, 10))
def test_snap_is_plain_split_at_tile_one(seed, T, K, E, S):
    """With M = 1 every integer is a tile boundary: snapping changes nothing."""
    rng = np.random.default_rng(seed)
    ids, T_valid, se, sw, rw, rr = _rand_case(rng, T, K, E, S, 1)
    a = oracle.dispatch(ids, T_valid, E, 1, se, sw, rw, rr)
    b = oracle.dispatch(ids, T_valid, E, 1, se, sw, rw, rr, snap=True)
    for k in ("expert_counts", "slot_counts", "slot_offsets", "row_token", "pair_row"):
        assert np.array_equal(a[k], b[k]), k


@settings(max_examples=300, deadline=None)
@given(st.integers(0, 2**31 - 1), st.integers(1, 80), st.integers(1, 8), st.integers(1, 6), st.integers(1, 10),
       st.sampled_from([2, 4, 8, 16, 64]))
def test_snap_invariants_random(seed, T, K, E, S, M):
    """Snapped splits: the same placement invariants as the plain split; the
    local boundaries of an expert (cumulative counts over its slots in slot
    order) are multiples of M unless they reach n_e; each lies within M / 2
    of the plain split's boundary; an expert without a remote share fills
    exactly ceil(n_e / M) tiles."""
    rng = np.random.default_rng(seed)
    ids, T_valid, se, sw, rw, rr = _rand_case(rng, T, K, E, S, M)
    plain = oracle.dispatch(ids, T_valid, E, M, se, sw, rw, rr)
    d = oracle.dispatch(ids, T_valid, E, M, se, sw, rw, rr, snap=True)
    assert np.array_equal(d["expert_counts"], plain["expert_counts"])
    assert d["err"] == plain["err"]
    # placement invariants (the proportional-share bound of the plain split
    # does not apply: shares move by up to M / 2)
    sc, so, rt, pr = d["slot_counts"], d["slot_offsets"], d["row_token"], d["pair_row"]
    Pz = so[1:] - so[:-1]
    assert np.all(Pz % M == 0) and np.all(Pz >= sc) and np.all(Pz - sc < M)
    placed = pr.reshape(-1) >= 0
    rows = pr.reshape(-1)[placed]
    assert len(np.unique(rows)) == len(rows)
    assert np.array_equal(rt[rows], np.nonzero(placed)[0] // ids.shape[1])
    for e in range(E):
        loc = [s for s in range(S) if se[s] == e]
        if not loc:
            continue
        n = int(d["expert_counts"][e])
        has_remote = rw[e] > 0 or rr[e] > 0
        b = np.cumsum([int(sc[s]) for s in loc])
        b0 = np.cumsum([int(plain["slot_counts"][s]) for s in loc])
        for x, x0 in zip(b.tolist(), b0.tolist()):
            assert x == n or x % M == 0, (e, b, n)
            assert abs(x - x0) <= M // 2
        if not has_remote:
            assert b[-1] == n
            assert sum(-(-int(sc[s]) // M) for s in loc) == -(-n // M)
        # ranks on each slot are a contiguous run in slot order: the slot's
        # first pair is the (b_{j-1})-th pair of the expert by pair index
        p_e = np.nonzero((ids.reshape(-1) == e) & np.repeat(np.arange(ids.shape[0]) < T_valid, ids.shape[1]))[0]
        lo = 0
        for s, hi in zip(loc, b.tolist()):
            want = [i for i in range(len(p_e)) if so[s] <= pr.reshape(-1)[p_e[i]] < so[s] + sc[s]]
            assert want == list(range(lo, hi)), (e, s)
            lo = hi


def test_snap_hand_worked():
    """Hand-worked snapped splits (M = 128):
    * 300 pairs, two local slots of equal weight: the plain boundary 150
      moves to 128 -> 128 + 172 rows (3 tiles instead of 2 + 2);
    * 200 pairs, one local slot and a remote share of equal weight: the
      boundary 100 moves to 128 -> 128 local rows, 72 pairs stay remote;
    * 128 pairs over two equal slots: the boundary 64 is a half and rounds
      up -> 128 + 0 (one tile, one slot left empty);
    * 300 pairs over slots of weights 1, 1, 2 (boundaries 75, 150, 300):
      128, 128, 300 -> 128 + 0 + 172."""
    z1 = np.zeros(1, np.uint32)
    zr = np.zeros(1, np.int32)

    def run(n, se, sw, rw=z1, rr=zr):
        ids = np.zeros((n, 1), np.int32)
        return oracle.dispatch(ids, n, 1, 128, np.array(se, np.int32), np.array(sw, np.uint32), rw, rr, snap=True)

    d = run(300, [0, 0], [1, 1])
    assert d["slot_counts"].tolist() == [128, 172] and d["slot_offsets"].tolist() == [0, 128, 384]
    assert d["pair_row"].reshape(-1)[:130].tolist() == list(range(128)) + [128, 129]
    d = run(200, [0], [1], np.array([1], np.uint32), np.array([1], np.int32))
    assert d["slot_counts"].tolist() == [128]
    assert (d["pair_row"].reshape(-1) >= 0).sum() == 128 and d["pair_row"].reshape(-1)[127] == 127
    d = run(128, [0, 0], [1, 1])
    assert d["slot_counts"].tolist() == [128, 0] and d["slot_offsets"].tolist() == [0, 128, 128]
    d = run(300, [0, 0, 0], [1, 1, 2])
    assert d["slot_counts"].tolist() == [128, 0, 172]


# ---- sampled replicas (Sec. 4.4: the deployed kernel samples a replica per
# pair from the renormalised row).  Draw of pair p: word 0 of Philox-4x64-10
# at counter (p, 0, 0, 0), key (seed, 0); u = floor(hi32 * W / 2^32); first
# entry j with u < C_j. ----

def _np_philox_word0(p, seed):
    """numpy's Philox-4x64-10 (an independent implementation) at counter p:
    numpy advances its counter before each block, so it starts from p - 1."""
    c = np.array([(p - 1) % 2**64, 0 if p > 0 else 2**64 - 1, 0 if p > 0 else 2**64 - 1, 0 if p > 0 else 2**64 - 1],
                 dtype=np.uint64)
    bg = np.random.Philox(key=np.array([seed, 0], dtype=np.uint64), counter=c)
    return int(bg.random_raw(4)[0])


def test_philox_matches_numpy():
    rng = np.random.default_rng(3)
    for seed in (0, 1, 2**63 + 5, int(rng.integers(0, 2**63))):
        for p in (0, 1, 2, 77, 4095, 123456789):
            got = int(oracle.philox4x64_10([p, 0, 0, 0], [seed, 0])[0])
            assert got == _np_philox_word0(p, seed), (seed, p)
    # all four words, against numpy's block sequence from counter 0
    bg = np.random.Philox(key=np.array([9, 0], dtype=np.uint64), counter=np.zeros(4, np.uint64))
    raw = bg.random_raw(12).reshape(3, 4)
    for i in range(3):
        assert np.array_equal(oracle.philox4x64_10([i + 1, 0, 0, 0], [9, 0]), raw[i])


@settings(max_examples=100, deadline=None)
@given(st.integers(0, 2**31 - 1), st.integers(1, 60), st.integers(1, 4), st.integers(1, 9), st.integers(0, 2**40),
       st.sampled_from([1, 4, 64]))
def test_sample_with_one_replica_is_the_split(seed, T, K, E, wseed, M):
    """Every expert on at most one local slot and no remote share: there is
    nothing to sample, so the result equals the (pinned) split."""
    rng = np.random.default_rng(seed)
    ids, T_valid, _, _, _, _ = _rand_case(rng, T, K, E, 1, M)
    S = int(rng.integers(1, E + 1))
    se = rng.permutation(E)[:S].astype(np.int32)
    sw = rng.integers(0, 5, size=S).astype(np.uint32)
    z = np.zeros(E, np.uint32)
    zr = np.zeros(E, np.int32)
    a = oracle.dispatch(ids, T_valid, E, M, se, sw, z, zr)
    b = oracle.dispatch(ids, T_valid, E, M, se, sw, z, zr, sample_seed=wseed)
    for k in ("expert_counts", "slot_counts", "slot_offsets", "row_token", "pair_row"):
        assert np.array_equal(a[k], b[k]), k


def test_sample_frequencies_and_zero_sum_row():
    """200000 pairs of one expert over three local slots (weights 1, 2, 5) and
    a remote share of weight 2: each share within 5 sigma of w_j / W; with an
    all-zero row the draw is uniform over the 3 local + 2 remote replicas."""
    n = 200000
    ids = np.zeros((n, 1), np.int32)
    se = np.array([0, 0, 0], np.int32)
    for sw, rw, rr, probs in (([1, 2, 5], [2], [1], [0.1, 0.2, 0.5]), ([0, 0, 0], [0], [2], [0.2, 0.2, 0.2])):
        d = oracle.dispatch(ids, n, 1, 64, se, np.array(sw, np.uint32), np.array(rw, np.uint32),
                            np.array(rr, np.int32), sample_seed=2024)
        for c, pr_ in zip(d["slot_counts"].tolist(), probs):
            sd = np.sqrt(n * pr_ * (1 - pr_))
            assert abs(c - n * pr_) < 5 * sd, (c, n * pr_)
        assert (d["pair_row"] >= 0).sum() == d["slot_counts"].sum()


@settings(max_examples=60, deadline=None)
@given(st.integers(0, 2**31 - 1), st.integers(1, 40), st.integers(1, 4), st.integers(1, 6), st.integers(1, 8),
       st.sampled_from([1, 4, 64]), st.integers(0, 2**62))
def test_sample_assignment_from_numpy_draws(seed, T, K, E, S, M, wseed):
    """Each pair's slot recomputed from numpy's Philox draw and the entry
    weights; rows of a slot in ascending pair index; padding rows -1."""
    rng = np.random.default_rng(seed)
    ids, T_valid, se, sw, rw, rr = _rand_case(rng, T, K, E, S, M)
    d = oracle.dispatch(ids, T_valid, E, M, se, sw, rw, rr, sample_seed=wseed)
    flat = ids.reshape(-1)
    want = np.full(flat.size, -1)
    for p in range(T_valid * K):
        e = int(flat[p])
        if e < 0 or e >= E:
            continue
        loc = [s for s in range(S) if se[s] == e]
        has_remote = rw[e] > 0 or rr[e] > 0
        w = [int(sw[s]) for s in loc] + ([int(rw[e])] if has_remote else [])
        if not loc and not has_remote:
            continue
        if sum(w) == 0:
            w = [1] * len(loc) + ([int(rr[e])] if has_remote else [])
        u = ((_np_philox_word0(p, wseed) >> 32) * sum(w)) >> 32
        j = int(np.searchsorted(np.cumsum(w), u, side="right"))
        if j < len(loc):
            want[p] = loc[j]
    so = d["slot_offsets"]
    got = np.full(flat.size, -1)
    for p, row in enumerate(d["pair_row"].reshape(-1).tolist()):
        if row >= 0:
            got[p] = int(np.searchsorted(so, row, side="right") - 1)
    assert np.array_equal(got, want)
    assert np.array_equal(d["slot_counts"], np.bincount(want[want >= 0], minlength=S))
    for s in range(S):
        ps = np.nonzero(want == s)[0]
        assert np.array_equal(d["pair_row"].reshape(-1)[ps], so[s] + np.arange(len(ps)))
        assert np.all(d["row_token"][so[s] + len(ps):so[s + 1]] == -1)
