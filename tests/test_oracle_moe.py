"""Pins for the stage-2/3 oracle (gate/up, SwiGLU, down, routing-weighted
combine; Sec. 2.1) and its number formats.

* bf16 and OCP e4m3 decoding and rounding are checked against torch's own
  bfloat16 / float8_e4m3fn conversions on the CPU (library routines);
* the whole forward is checked against a dense numpy formulation (matmul,
  scipy's expit) on small shapes -- a library computation of the same
  definition, written independently;
* the dense-FFN reduction (K = 1, w = 1, one expert), linearity in the routing
  weights and independence from how an expert's tokens are split across local
  replicas (split invariance) are checked as properties."""
import numpy as np
import pytest
import torch
from scipy.special import expit

import oracle
from paper_2608_13057_amd import synth


def test_bf16_decode_matches_torch():
    codes = np.arange(0, 65536, 97, dtype=np.uint16)
    ref = torch.from_numpy(codes.view(np.int16)).view(torch.bfloat16).float().numpy()
    got = np.array([oracle.bf16_value(int(c)) for c in codes])
    fin = np.isfinite(ref)
    assert np.array_equal(got[fin], ref[fin].astype(np.float64))


def test_e4m3_decode_matches_torch_all_codes():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
    got = np.array([oracle.e4m3_value(int(c)) for c in codes])
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    m = ~np.isnan(ref)
    assert np.array_equal(got[m], ref[m])
    assert got[0x7E] == 448.0 and np.isnan(got[0x7F])


def test_rounding_matches_torch():
    rng = np.random.default_rng(0)
    # exact midpoints between neighbouring e4m3 values and between bf16
    # values: the tie-to-even rule decides these
    e4 = np.sort(torch.arange(0, 127, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).double().numpy())
    mid_e4 = (e4[1:] + e4[:-1]) / 2
    bf = torch.from_numpy(np.arange(0x3F00, 0x4100, dtype=np.int16)).view(torch.bfloat16).double().numpy()
    mid_bf = (bf[1:] + bf[:-1]) / 2
    v = np.concatenate([rng.standard_normal(3000) * 10.0 ** rng.integers(-3, 3, 3000),
                        rng.uniform(-448, 448, 2000), mid_e4, -mid_e4, mid_bf, -mid_bf]).astype(np.float32)
    rb = torch.from_numpy(v).to(torch.bfloat16).float().numpy()
    re = torch.from_numpy(v).to(torch.float8_e4m3fn).float().numpy()
    for i in range(len(v)):
        assert oracle.round_bf16(float(v[i])) == float(rb[i])
        assert oracle.round_e4m3(float(v[i])) == float(re[i])
    # the generator's encoder agrees with the same library conversion
    codes = synth.to_e4m3_codes(v)
    ref_codes = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codes[np.abs(v) > 0], ref_codes[np.abs(v) > 0])


def _small_problem(dtype, T=24, K=2, E=3, S=4, H=256, I=256, seed=5):
    rng = np.random.default_rng(seed)
    ids = rng.integers(0, E, size=(T, K)).astype(np.int32)
    for t in range(T):  # distinct experts per token, as a router emits
        ids[t] = rng.permutation(E)[:K]
    w = rng.random((T, K)).astype(np.float32)
    se = np.array([0, 1, 2, 0][:S], np.int32)
    x, xs = synth.activations(T, H, seed, dtype)
    w13, s13, w2, s2 = synth.slot_weights(se, H, I, seed, dtype)
    return ids, w, se, x, xs, w13, s13, w2, s2


def _dense_numpy(x, xs, w13, s13, w2, s2, ids_slot, w, dtype):
    """Independent dense formulation with numpy matmul and scipy expit."""
    T, K = ids_slot.shape
    S, I2, H = w13.shape
    I = I2 // 2
    if dtype == "bf16":
        X = synth.bf16_bits_to_f32(x).astype(np.float64)
        W13 = synth.bf16_bits_to_f32(w13).astype(np.float64)
        W2 = synth.bf16_bits_to_f32(w2).astype(np.float64)
    else:
        dec = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).double().numpy()
        X = dec[x] * np.repeat(xs.astype(np.float64), 128, axis=1)
        W13 = dec[w13] * np.kron(s13.astype(np.float64), np.ones((1, 128, 128)))
        W2 = dec[w2] * np.kron(s2.astype(np.float64), np.ones((1, 128, 128)))
    y = np.zeros((T, H))
    for s in range(S):
        U = X @ W13[s].T
        g, u = U[:, :I], U[:, I:]
        h = g * expit(g) * u
        O = h @ W2[s].T
        for k in range(K):
            m = ids_slot[:, k] == s
            y[m] += w[m, k:k + 1].astype(np.float64) * O[m]
    return y


@pytest.mark.parametrize("dtype", ["bf16", "fp8", "fp8mx"])
def test_moe_matches_dense_numpy(dtype):
    ids, w, se, x, xs, w13, s13, w2, s2 = _small_problem(dtype)
    E, S = 3, len(se)
    # plan: expert 0 split over slots 0 and 3
    d = oracle.dispatch(ids, ids.shape[0], E, 16, se, np.ones(S, np.uint32), np.zeros(E, np.uint32),
                        np.zeros(E, np.int32))
    ps = oracle.pair_slot(d)
    y = oracle.moe(x, w, ps, w13, w2, dtype, x_scale=xs, w13_scale=s13, w2_scale=s2)
    ref = _dense_numpy(x, xs, w13, s13, w2, s2, ps, w, dtype)
    assert np.max(np.abs(y - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))


def test_dense_ffn_reduction():
    """K = 1, weight 1, one expert: y is the plain SwiGLU FFN of x."""
    T, H, I = 8, 128, 256
    x, _ = synth.activations(T, H, 11, "bf16")
    w13, _, w2, _ = synth.slot_weights(np.array([0], np.int32), H, I, 11, "bf16")
    ps = np.zeros((T, 1), np.int32)
    y = oracle.moe(x, np.ones((T, 1), np.float32), ps, w13, w2, "bf16")
    X = torch.from_numpy(synth.bf16_bits_to_f32(x)).double()
    A = torch.from_numpy(synth.bf16_bits_to_f32(w13[0])).double()
    B = torch.from_numpy(synth.bf16_bits_to_f32(w2[0])).double()
    ref = (torch.nn.functional.silu(X @ A[:I].T) * (X @ A[I:].T)) @ B.T
    assert np.max(np.abs(y - ref.numpy())) < 1e-12


def test_linearity_in_routing_weights():
    ids, w, se, x, xs, w13, s13, w2, s2 = _small_problem("bf16", T=10)
    d = oracle.dispatch(ids, 10, 3, 8, se, np.ones(4, np.uint32), np.zeros(3, np.uint32), np.zeros(3, np.int32))
    ps = oracle.pair_slot(d)
    y1 = oracle.moe(x, w, ps, w13, w2, "bf16")
    y2 = oracle.moe(x, (w * np.float32(0.25)), ps, w13, w2, "bf16")  # exact power-of-two scaling
    assert np.array_equal(y2, y1 * 0.25)


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_split_invariance(dtype):
    """y does not depend on how expert 0's tokens are split over its two
    local slots (both hold copies of the same weights)."""
    ids, w, se, x, xs, w13, s13, w2, s2 = _small_problem(dtype)
    outs = []
    for sw in ([1, 1, 1, 1], [1, 1, 1, 0], [0, 1, 1, 1], [3, 1, 1, 1]):
        d = oracle.dispatch(ids, ids.shape[0], 3, 16, se, np.array(sw, np.uint32), np.zeros(3, np.uint32),
                            np.zeros(3, np.int32))
        outs.append(oracle.moe(x, w, oracle.pair_slot(d), w13, w2, dtype, x_scale=xs, w13_scale=s13,
                               w2_scale=s2))
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])


def test_mirror_mode_rounds_output_and_stays_close():
    ids, w, se, x, xs, w13, s13, w2, s2 = _small_problem("fp8")
    d = oracle.dispatch(ids, ids.shape[0], 3, 16, se, np.ones(4, np.uint32), np.zeros(3, np.uint32),
                        np.zeros(3, np.int32))
    ps = oracle.pair_slot(d)
    ye = oracle.moe(x, w, ps, w13, w2, "fp8", "exact", xs, s13, s2)
    ym = oracle.moe(x, w, ps, w13, w2, "fp8", "mirror", xs, s13, s2)
    # mirror-mode y values are bf16-representable
    yb = torch.from_numpy(ym.astype(np.float32)).to(torch.bfloat16).double().numpy()
    assert np.array_equal(yb, ym)
    rel = np.max(np.abs(ym - ye)) / np.max(np.abs(ye))
    assert 0 < rel < 0.1


def test_nonlocal_and_padding_tokens_are_zero():
    ids, w, se, x, xs, w13, s13, w2, s2 = _small_problem("bf16", T=12)
    d = oracle.dispatch(ids, 6, 3, 8, se, np.ones(4, np.uint32), np.zeros(3, np.uint32), np.zeros(3, np.int32))
    y = oracle.moe(x, w, oracle.pair_slot(d), w13, w2, "bf16")
    assert np.all(y[6:] == 0)


def test_pow2_scales_are_minimal_powers_of_two():
    """fp8mx inputs: every scale is a power of two, the block's amax / scale
    is within e4m3's range and halving the scale would leave it."""
    x = np.random.default_rng(1).standard_normal((40, 512)).astype(np.float32) * 3
    x[3, :128] = 0
    q, sc = synth.quant_rows_1x128(x, pow2=True)
    m, _ = np.frexp(sc.astype(np.float64))
    assert np.all(m == 0.5)
    amax = np.abs(x.reshape(40, 4, 128)).max(axis=2)
    nz = amax > 0
    assert np.all(amax[nz] / sc[nz] <= 448.0) and np.all(amax[nz] / (sc[nz] / 2) > 448.0)
    assert sc[3, 0] == 1.0


def test_mirror_mode_pow2_h_quantisation():
    """fp8mx mirror mode: h re-quantised with power-of-two block scales; the
    output stays close to the exact mode and differs from fp8's mirror mode
    (different h scales) while the exact modes agree (same codes, same
    scales read the same way)."""
    ids, w, se, x, xs, w13, s13, w2, s2 = _small_problem("fp8mx")
    d = oracle.dispatch(ids, ids.shape[0], 3, 16, se, np.ones(4, np.uint32), np.zeros(3, np.uint32),
                        np.zeros(3, np.int32))
    ps = oracle.pair_slot(d)
    ye = oracle.moe(x, w, ps, w13, w2, "fp8mx", "exact", xs, s13, s2)
    ye8 = oracle.moe(x, w, ps, w13, w2, "fp8", "exact", xs, s13, s2)
    assert np.array_equal(ye, ye8)
    ym = oracle.moe(x, w, ps, w13, w2, "fp8mx", "mirror", xs, s13, s2)
    ym8 = oracle.moe(x, w, ps, w13, w2, "fp8", "mirror", xs, s13, s2)
    assert not np.array_equal(ym, ym8)
    assert 0 < np.max(np.abs(ym - ye)) / np.max(np.abs(ye)) < 0.1


# ---- stage 3 alone: oracle.combine (Sec. 2.1, routing-weighted combine) ----

def _combine_problem(T=37, K=5, H=128, R=120, T_valid=31, seed=11):
    rng = np.random.default_rng(seed)
    yp = synth.to_bf16_bits(rng.standard_normal((R, H)).astype(np.float32))
    pr = rng.integers(-1, R, size=(T, K)).astype(np.int32)
    w = rng.random((T, K)).astype(np.float32)
    return pr, w, yp, T_valid


def test_combine_matches_gathered_einsum():
    """y = sum_k w[t,k] * Y_perm[pair_row[t,k]] over pairs with a row, for
    t < T_valid, as one numpy gather + einsum over a 0/1 mask (torch's bf16
    decoding for the rows): an independent vectorised statement of the same
    definition."""
    pr, w, yp, Tv = _combine_problem()
    rows = torch.from_numpy(yp.view(np.int16)).view(torch.bfloat16).double().numpy()
    mask = (pr >= 0).astype(np.float64)
    mask[Tv:] = 0.0
    g = rows[np.maximum(pr, 0)]  # [T, K, H]
    ref = np.einsum("tk,tk,tkh->th", w.astype(np.float64), mask, g)
    got = oracle.combine(pr, w, yp, Tv)
    assert np.allclose(got, ref, rtol=1e-13, atol=1e-13)
    assert np.all(got[Tv:] == 0)


def test_combine_one_hot_is_row_copy():
    """K = 1, w = 1: each token's output is exactly its row's bf16 value
    (a permutation of the rows); a token whose pair has no row is zero."""
    rng = np.random.default_rng(3)
    T, H = 50, 256
    yp = synth.to_bf16_bits(rng.standard_normal((T, H)).astype(np.float32))
    perm = rng.permutation(T).astype(np.int32)
    pr = perm.reshape(T, 1).copy()
    pr[7, 0] = -1
    got = oracle.combine(pr, np.ones((T, 1), np.float32), yp, T)
    vals = synth.bf16_bits_to_f32(yp).astype(np.float64)
    for t in range(T):
        if t == 7:
            assert np.all(got[t] == 0)
        else:
            assert np.array_equal(got[t], vals[perm[t]])


def test_combine_linear_and_order_free():
    """Linear in the routing weights (scaling w by a power of two scales y
    exactly), and permuting a token's k-columns together with their rows
    leaves y unchanged up to fp64 summation order."""
    pr, w, yp, Tv = _combine_problem(seed=12)
    y1 = oracle.combine(pr, w, yp, Tv)
    y2 = oracle.combine(pr, (w * 4.0).astype(np.float32), yp, Tv)
    assert np.array_equal(y2, 4.0 * y1)
    perm = np.random.default_rng(0).permutation(pr.shape[1])
    y3 = oracle.combine(pr[:, perm], w[:, perm], yp, Tv)
    assert np.allclose(y3, y1, rtol=1e-14, atol=1e-14)


def test_combine_hand_worked():
    """Two tokens, K = 2, rows of exactly representable values."""
    vals = np.array([[1.0, -2.0], [0.5, 4.0], [3.0, 0.25]], np.float32)
    yp = synth.to_bf16_bits(vals)
    pr = np.array([[2, 0], [-1, 1]], np.int32)
    w = np.array([[0.5, 0.25], [0.75, 2.0]], np.float32)
    got = oracle.combine(pr, w, yp, 2)
    assert np.array_equal(got, np.array([[0.5 * 3.0 + 0.25 * 1.0, 0.5 * 0.25 + 0.25 * -2.0], [1.0, 8.0]]))
    assert np.all(oracle.combine(pr, w, yp, 1)[1] == 0)  # the second token is graph padding
