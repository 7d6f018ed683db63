"""The allocation-free forward (tempo_moe_forward_static, whose workspace is
the library's static scratch array) against tempo_moe_forward with a
caller workspace: two calls in a row on one GPU, the second with a smaller
batch, each bit-identical to the workspace entry point (same kernels, same
arithmetic) and within the oracle tolerance."""
import numpy as np
import pytest

from helpers import Case, bf16_to_f64, rel_err_rows, to_host

pytestmark = pytest.mark.gpu

TOL = {"bf16": 1e-2, "fp8": 5e-2}


def _both(c):
    import torch
    from paper_2608_13057_amd import moe

    y_ref = torch.empty(c.wl.T, c.wl.H, dtype=torch.int16, device="cuda")
    moe.forward(c.shape, c.d_plan, c.d_ids, c.d_w, c.d_x, c.d_xs, c.d_weights, c.disp, y_ref, c.ws)
    disp2 = moe.DispatchBuffers.allocate(c.shape, c.ws.row_cap)
    y = torch.full((c.wl.T, c.wl.H), 0x7FFF, dtype=torch.int16, device="cuda")
    moe.forward_static(c.shape, c.d_plan, c.d_ids, c.d_w, c.d_x, c.d_xs, c.d_weights, disp2, y)
    torch.cuda.synchronize()
    return to_host(y_ref), to_host(y), disp2


def test_forward_static_two_calls_match_forward():
    import oracle
    from paper_2608_13057_amd import synth

    for name, T in (("tiny", 96), ("tiny_fp8", 40)):
        wl = synth.make_workload(name, T=T)
        c = Case(wl, "uniform", 64)
        print(f"[static] {name} T={T}", flush=True)
        y_ref, y, disp2 = _both(c)
        assert np.array_equal(y, y_ref), f"{name} T={T}: static scratch result differs from the workspace result"
        for f in ("slot_counts", "slot_offsets", "pair_row", "expert_counts"):
            assert np.array_equal(to_host(getattr(disp2, f)), to_host(getattr(c.disp, f))), f
        d = c.oracle_dispatch()
        has = (d["pair_row"] >= 0).any(axis=1)
        ref = oracle.moe(c.x, wl.topk_w, oracle.pair_slot(d), c.w13, c.w2, wl.dtype, "exact", c.xs, c.s13, c.s2)
        err = rel_err_rows(bf16_to_f64(y), ref, np.nonzero(has)[0])
        print(f"[static] {name} T={T} err={err:.2e}")
        assert err <= TOL[wl.dtype]
        assert np.all(y[~has] == 0)
