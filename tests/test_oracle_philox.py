"""Pins of the oracle's counter-based uniforms (CPU only).

Stochastic drafting (Section 2.2: k candidates sampled per level; Section 3
reports temperature 1) draws its uniforms from a Philox4x64-10 stream (Salmon
et al., SC 2011) keyed by a seed, with the offset in the counter.  Pinned
against numpy's independent Philox4x64-10 bit generator (numpy advances its
256-bit counter before each block, so a generator started at counter c - 1
yields the block of counter c first), including counter wrap-around, and
against the stated map of the top 23 bits to (j + 1/2) / 2^23."""
import numpy as np
import pytest
from scipy import stats


def _numpy_block(counter, key):
    c = [int(x) for x in counter]
    v = (c[0] | (c[1] << 64) | (c[2] << 128) | (c[3] << 192)) - 1
    v %= 1 << 256
    start = [(v >> (64 * i)) & ((1 << 64) - 1) for i in range(4)]
    # uint64 arrays: a list of Python ints above 2^63 would pass through float64
    return np.random.Philox(counter=np.array(start, dtype=np.uint64),
                            key=np.array([int(k) for k in key], dtype=np.uint64)).random_raw(4)


@pytest.mark.parametrize("counter,key", [
    ([0, 0, 0, 0], [0, 0]),
    ([1, 0, 0, 0], [0x1234, 0x5678]),
    ([2**64 - 1, 2**64 - 1, 2**64 - 1, 2**64 - 1], [2**64 - 1, 2**64 - 1]),
    ([0x243F6A8885A308D3, 0x13198A2E03707344, 0xA4093822299F31D0, 0x082EFA98EC4E6C89],
     [0x452821E638D01377, 0xBE5466CF34E90C6C]),
    ([12345, 7, 0, 0], [99, 0]),
])
def test_philox_blocks_match_numpy(feo, counter, key):
    got = feo.philox4x64_10(np.array(counter, dtype=np.uint64), np.array(key, dtype=np.uint64))
    np.testing.assert_array_equal(got, _numpy_block(counter, key))


def test_uniforms_follow_the_stated_map(feo):
    seed, offset, first, n = 0xFEEDFACE12345, 3, 1021, 37
    got = feo.philox_uniforms(seed, offset, first, n)
    want = np.empty(n, np.float32)
    for i in range(n):
        e = first + i
        x = int(_numpy_block([e >> 2, offset, 0, 0], [seed, 0])[e & 3])
        want[i] = np.float32(((x >> 41) + 0.5) / 2.0**23)
    np.testing.assert_array_equal(got, want)
    assert ((got > 0) & (got < 1)).all()


def test_streams_differ_and_are_uniform(feo):
    a = feo.philox_uniforms(1, 0, 0, 200_000)
    b = feo.philox_uniforms(1, 1, 0, 200_000)     # next offset: another stream
    c = feo.philox_uniforms(2, 0, 0, 200_000)     # another seed
    assert (a != b).mean() > 0.999 and (a != c).mean() > 0.999
    for u in (a, b, c):
        assert stats.kstest(u.astype(np.float64), "uniform").pvalue > 1e-4
    # a window of the stream equals the same positions of a longer draw
    np.testing.assert_array_equal(feo.philox_uniforms(1, 0, 1234, 99), a[1234:1333])
