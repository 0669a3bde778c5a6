"""Pins of the state-copy oracle (oracle/state_copy.py).

A range copy has a plain definition, so the pins are that definition checked against things
other than the numpy version itself: the byte-by-byte loop, Python's own bytes slicing, the
bytes outside every range staying untouched, and the round trip offload -> resume restoring the
packed batch exactly (what suspending and resuming a session must do, paper Sec. 3.1).
"""
import numpy as np
import pytest

from oracle import state_copy as SC


def rand_bytes(n, seed):
    return np.random.default_rng(seed).integers(0, 256, size=n, dtype=np.uint8)


def test_numpy_copy_matches_bytewise_loop_and_python_slicing():
    src, dst = rand_bytes(300, 1), rand_bytes(200, 2)
    ranges = [(0, 16, 32), (100, 64, 48), (250, 150, 50), (7, 0, 0)]
    a = SC.copy_ranges(src, dst, ranges)
    b = SC.copy_ranges_bytewise(bytes(src), bytes(dst), ranges)
    assert a.tobytes() == bytes(b)
    expect = bytearray(dst.tobytes())
    for so, do, n in ranges:
        expect[do:do + n] = src.tobytes()[so:so + n]
    assert a.tobytes() == bytes(expect)


def test_bytes_outside_ranges_untouched():
    src, dst = rand_bytes(4096, 3), rand_bytes(4096, 4)
    ranges = [(16, 1024, 512), (2048, 0, 256), (0, 3000, 16)]
    out = SC.copy_ranges(src, dst, ranges)
    mask = np.zeros(4096, bool)
    for _, do, n in ranges:
        mask[do:do + n] = True
    assert np.array_equal(out[~mask], dst[~mask])
    assert not np.array_equal(out[mask], dst[mask])


def test_session_ranges_and_round_trip():
    # a packed batch of 4 sessions, 5 heads x 8 channels of bf16 per token row (80 bytes)
    row = 5 * 8 * 2
    cu = np.array([0, 7, 7, 19, 30], np.int32)
    batch = rand_bytes(int(cu[-1]) * row, 5)
    ranges, end = SC.session_ranges(cu, [3, 0], row)
    assert end == (11 + 7) * row
    assert ranges[0] == (19 * row, 0, 11 * row) and ranges[1] == (0, 11 * row, 7 * row)
    host = SC.copy_ranges(batch, np.zeros(end, np.uint8), ranges)
    # resume into a cleared batch: swap src/dst offsets
    back = [(do, so, n) for so, do, n in ranges]
    restored = SC.copy_ranges(host, np.zeros_like(batch), back)
    for s in (3, 0):
        a, b = cu[s] * row, cu[s + 1] * row
        assert np.array_equal(restored[a:b], batch[a:b])
    assert np.all(restored[7 * row:19 * row] == 0)  # sessions 1 (empty) and 2 were not copied


@pytest.mark.parametrize("n", [0, 1, 17])
def test_zero_and_odd_lengths(n):
    src, dst = rand_bytes(64, 6), rand_bytes(64, 7)
    out = SC.copy_ranges(src, dst, [(3, 40, n)])
    assert out[40:40 + n].tobytes() == src[3:3 + n].tobytes()
    assert np.array_equal(out[:40], dst[:40]) and np.array_equal(out[40 + n:], dst[40 + n:])
