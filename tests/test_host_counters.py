"""Host logic of the library (tempo_moe_counter_window, no GPU): windows of
the cumulative per-expert counters (Sec. 4.4: cumulative counting, windows
recovered by wrap-safe differencing)."""
import numpy as np

from paper_2608_13057_amd import moe


def test_counter_window_wraps():
    rng = np.random.default_rng(0)
    before = rng.integers(0, 2**32, size=1000, dtype=np.uint64).astype(np.uint32)
    adds = rng.integers(0, 2**31, size=1000, dtype=np.uint64)
    after = ((before.astype(np.uint64) + adds) % 2**32).astype(np.uint32)
    assert np.array_equal(moe.counter_window(before, after), adds)
    # int32 bit patterns (how the device buffer is held) give the same window
    assert np.array_equal(moe.counter_window(before.view(np.int32), after.view(np.int32)), adds)
    # a counter that wrapped: 2^32 - 5 -> 7 is a window of 12
    assert moe.counter_window(np.array([2**32 - 5], np.uint32), np.array([7], np.uint32)).tolist() == [12]


def test_counter_window_of_successive_batches_adds_up():
    """Windows over consecutive snapshots add up to the window over the whole
    span, whatever wraps happened in between."""
    rng = np.random.default_rng(1)
    snaps = [rng.integers(0, 2**32, size=16, dtype=np.uint64)]
    for _ in range(20):
        snaps.append((snaps[-1] + rng.integers(0, 2**30, size=16, dtype=np.uint64)) % 2**32)
    snaps = [s.astype(np.uint32) for s in snaps]
    total = sum(moe.counter_window(a, b).astype(np.uint64) for a, b in zip(snaps[:-1], snaps[1:]))
    assert np.array_equal(total % 2**32, moe.counter_window(snaps[0], snaps[-1]))


def test_counter_window_rejects_bad_arguments():
    import ctypes

    from paper_2608_13057_amd import _lib

    lib = _lib.load()
    buf = (ctypes.c_uint32 * 4)()
    assert lib.tempo_moe_counter_window(0, buf, buf, buf) == _lib.TEMPO_EINVAL
    assert lib.tempo_moe_counter_window(4, None, buf, buf) == _lib.TEMPO_EINVAL
