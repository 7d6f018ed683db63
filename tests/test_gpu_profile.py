"""The stage-4 profiling harness on the GPU at the tiny expert shape: every
logged point's G, N, M-tiles and per-slot counts are those of its
constructed routing and plan as the oracle's stage 1 places them, the
per-slot stage-2 spans are nonzero on exactly its activated slots, and the
timings are positive; then the fit of a small grid runs end to end."""
import numpy as np
import pytest

import oracle

pytestmark = pytest.mark.gpu


def test_harness_points_match_the_constructed_plan():
    from paper_2608_13057_amd import profile

    M = 64
    h = profile.Harness(dtype="bf16", H=256, I=512, m_tile=M, max_tokens=3 * 70)
    for G in (1, 3):
        for n in (5, 70):
            rows = h.point(G, n, reps=3)
            T = G * n
            ids = (np.arange(T, dtype=np.int32) // n).reshape(T, 1)
            d = oracle.dispatch(ids, T, G, M, np.arange(G, dtype=np.int32), np.ones(G, np.uint32),
                                np.zeros(G, np.uint32), np.zeros(G, np.int32))
            sc = d["slot_counts"]
            assert {r["scope"] for r in rows} == {"gemm", "block"}
            for r in rows:
                print(f"[harness] G={G} n={n} {r['scope']} {r['t_us']:.1f} us spans {r['slot_span_us']}")
                assert r["G"] == int((sc > 0).sum()) == G
                assert r["N"] == int(sc.sum()) == T
                assert r["tiles"] == int(sum(-(-int(c) // M) for c in sc))
                assert r["slot_counts"] == sc.tolist()
                assert len(r["slot_span_us"]) == G and all((s > 0) == (c > 0) for s, c in zip(r["slot_span_us"], sc))
                assert r["t_us"] > 0 and r["p10"] <= r["t_us"] <= r["p90"]


def test_sweep_and_fit_end_to_end():
    from paper_2608_13057_amd import profile

    rows = profile.run_sweep("bf16", 64, Gs=(1, 2, 4), ns=(1, 16, 64, 65, 128), reps=3, shape="tiny")
    assert len(rows) == 2 * 3 * 5
    md = profile.markdown(rows, "tiny", "test", ns=(1, 16, 64, 65, 128))
    assert "Fit, scope `gemm`" in md and "Fit, scope `block`" in md
