"""The seeded input generators: bf16 rounding pinned by hand-derived bit
patterns, and the chunked (threaded) path equal to the single-chunk path."""
import numpy as np

import workloads as W


def _bits(u32):
    return np.array(u32, dtype=np.uint32).view(np.float32)


def test_bf16_rounding_hand_values():
    cases = {
        0x3F800000: 0x3F80,  # 1.0
        0x3F808000: 0x3F80,  # 1 + 2^-8: a tie, the even neighbour is 1.0
        0x3F818000: 0x3F82,  # 1 + 3*2^-8: a tie, the even neighbour rounds up
        0x3F808001: 0x3F81,  # just above the tie
        0x3F807FFF: 0x3F80,  # just below the tie
        0x7F7F8000: 0x7F80,  # the largest bf16 below the float max, then a tie: rounds to +inf
        0xFF800000: 0xFF80,  # -inf passes through
        0x7F800001: 0x7FC0,  # signalling NaN -> quiet NaN with the same sign
        0xFFFFFFFF: 0xFFFF,  # NaN with every payload bit set stays NaN
        0x00008000: 0x0000,  # subnormal tie to even (zero)
        0x00018000: 0x0002,  # subnormal tie rounds up to even
        0x80000000: 0x8000,  # -0
    }
    got = W.f32_to_bf16_bits(_bits(list(cases)))
    np.testing.assert_array_equal(got, np.array(list(cases.values()), dtype=np.uint16))


def test_bf16_chunked_equals_single_chunk():
    rng = np.random.default_rng(3)
    u = rng.integers(0, 2 ** 32, size=(3, (1 << 22) + 123), dtype=np.uint64).astype(np.uint32)
    x = u.view(np.float32)
    big = W.f32_to_bf16_bits(x)               # more than one chunk: thread pool
    assert big.shape == x.shape and big.dtype == np.uint16
    for r in range(x.shape[0]):               # slices of at most one chunk each
        for lo in range(0, x.shape[1], 1 << 21):
            np.testing.assert_array_equal(big[r, lo:lo + (1 << 21)], W.f32_to_bf16_bits(x[r, lo:lo + (1 << 21)]))
    # widening back is exact on every non-NaN pattern
    back = W.bf16_bits_to_f32(big)
    ok = ~np.isnan(back)
    np.testing.assert_array_equal(W.f32_to_bf16_bits(back[ok]), big[ok])
