"""Pins the oracle's cache-flush fill (Section 2.1: a flush between timed
iterations; Section 4.2 step 5: a memset over a cache-sized buffer).

The fill's definition is plain: every 32-bit word of the buffer holds the
pattern afterwards. The pin is numpy's own fill of a uint32 array
(``np.full``), compared word for word, on sizes from one word to 64 MiB plus
a ragged tail, with guard words on both sides that must stay untouched, and
the rejection of a byte count that is not a whole number of words.
"""
import ctypes

import numpy as np
import pytest

import oracle

GUARD = 64   # words on each side of the filled range


def _fill_in_guarded(nbytes, pattern):
    """ko_flush over the middle of a buffer with GUARD sentinel words on each
    side; returns (whole buffer as uint32 words, status)."""
    nwords = nbytes // 4
    buf = np.empty(nwords + 2 * GUARD, dtype=np.uint32)
    buf[:] = np.uint32(0xA5A5A5A5)
    ptr = buf.ctypes.data + 4 * GUARD
    st = oracle.lib().ko_flush(ctypes.c_void_p(ptr), nbytes, pattern)
    return buf, st


@pytest.mark.parametrize("nbytes", [4, 16, 4096 + 4, (64 << 20) + 12])
@pytest.mark.parametrize("pattern", [0x00000000, 0x9E3779B9, 0xFFFFFFFF, 0x0000FF01])
def test_every_word_holds_the_pattern(nbytes, pattern):
    buf, st = _fill_in_guarded(nbytes, pattern)
    assert st == 0
    n = nbytes // 4
    body = buf[GUARD:GUARD + n]
    assert np.array_equal(body, np.full(n, pattern, dtype=np.uint32))
    # nothing outside [0, nbytes) is written
    assert np.all(buf[:GUARD] == 0xA5A5A5A5)
    assert np.all(buf[GUARD + n:] == 0xA5A5A5A5)


def test_rep_patterns_of_the_timed_loop_differ():
    # The timed loop's rep r writes 0x9E3779B9 (r + 1) mod 2^32: consecutive
    # reps write different words, so no rep's flush repeats the previous data.
    pats = [(0x9E3779B9 * (r + 1)) & 0xFFFFFFFF for r in range(1000)]
    assert all(pats[r] != pats[r + 1] for r in range(999))
    buf = np.zeros(1024, dtype=np.uint32)
    for p in pats[:3]:
        oracle.flush_fill(buf, p)
        assert np.array_equal(buf, np.full(1024, p, dtype=np.uint32))


@pytest.mark.parametrize("nbytes", [1, 2, 3, 4097, 4098, 4099])
def test_partial_words_rejected(nbytes):
    buf = np.full(4096, 0xA5A5A5A5, dtype=np.uint32)
    st = oracle.lib().ko_flush(ctypes.c_void_p(buf.ctypes.data), nbytes, 0x12345678)
    assert st != 0
    assert np.all(buf == 0xA5A5A5A5), "a rejected call must write nothing"


def test_zero_bytes_writes_nothing():
    buf, st = _fill_in_guarded(0, 0x12345678)
    assert st == 0
    assert np.all(buf == 0xA5A5A5A5)
