"""Exactness of two shortcuts the single-workgroup stage-1 kernel takes in
place of integer division (CPU: numpy's float32 / float64 arithmetic rounds
to nearest even, as the GPU's does).

* token of a pair: p / K as (int)((p + 0.5) * fl(1/K)) in fp32, for every
  p < 8192 and K <= 32 (the kernel's limits);
* the plan's split floor(n_e C / W) in fp64 when n_e < 2^20 (C <= W < 2^32)."""
import numpy as np


def test_token_division_fp32_exhaustive():
    p = np.arange(8192, dtype=np.int64)
    for K in range(1, 33):
        inv = np.float32(1.0) / np.float32(K)
        t = ((p.astype(np.float32) + np.float32(0.5)) * inv).astype(np.int64)
        assert np.array_equal(t, p // K), K


def test_split_floor_fp64():
    rng = np.random.default_rng(0)
    n = np.concatenate([rng.integers(0, 1 << 20, 200000), [0, 1, (1 << 20) - 1] * 100]).astype(np.uint64)
    W = np.concatenate([rng.integers(1, 1 << 32, 200000), [1, (1 << 32) - 1, 3] * 100]).astype(np.uint64)
    C = (rng.random(n.size) * (W.astype(np.float64) + 1)).astype(np.uint64)
    C = np.minimum(C, W)
    C[:300] = W[:300]  # C = W: the last entry of a row
    a = n * C  # < 2^52: exact in uint64 and in float64
    got = np.floor(a.astype(np.float64) / W.astype(np.float64)).astype(np.uint64)
    assert np.array_equal(got, a // W)
    # quotients just below an integer: a = q W - 1
    q = rng.integers(1, 1 << 20, 1000).astype(np.uint64)
    W2 = rng.integers(1 << 31, 1 << 32, 1000).astype(np.uint64)
    a2 = q * W2 - np.uint64(1)
    assert np.array_equal(np.floor(a2.astype(np.float64) / W2.astype(np.float64)).astype(np.uint64), q - np.uint64(1))
