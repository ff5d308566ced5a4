"""Pins of the oracle's head-wise mixed-precision rule (Sec. 3.2):
priority = gap x std of the channel-wise gaps, and the n_h lowest-priority
heads stored in 2 bits."""
import math

import numpy as np


def test_worked_example(orc):
    # Two tokens of a 4-channel head:
    #   t0 = [0, 1, 2, -1], t1 = [1, 4, 2, 3]
    # channel gaps (max - min over tokens): [1, 3, 0, 4], mean 2,
    # squared deviations [1, 1, 4, 4] -> variance 10/4 = 2.5;
    # head gap = max over all (4) - min over all (-1) = 5;
    # priority = 5 * sqrt(2.5).
    k = np.zeros((1, 1, 2, 4), np.float32)
    k[0, 0, 0] = [0, 1, 2, -1]
    k[0, 0, 1] = [1, 4, 2, 3]
    assert orc.head_priority(k)[0] == 5 * math.sqrt(2.5)


def test_constant_channels_have_zero_priority(orc):
    k = np.tile(np.arange(8, dtype=np.float32), (2, 3, 5, 1))  # each channel constant
    assert np.all(orc.head_priority(k) == 0.0)


def test_invariances(orc):
    rng = np.random.default_rng(0)
    k = rng.standard_normal((2, 3, 40, 16)).astype(np.float16).astype(np.float32)
    p = orc.head_priority(k)
    # token order and sequence order do not matter
    perm = rng.permutation(40)
    assert np.array_equal(orc.head_priority(k[:, :, perm]), p)
    assert np.array_equal(orc.head_priority(k[::-1]), p)
    # channel order does not matter (up to the order of the std sums)
    cperm = rng.permutation(16)
    np.testing.assert_allclose(orc.head_priority(k[..., cperm]), p, rtol=1e-14)
    # a shift leaves every gap alone; a scale by 2 multiplies gap and std by 2
    np.testing.assert_allclose(orc.head_priority(k + 8.0), p, rtol=1e-12)
    assert np.array_equal(orc.head_priority(2 * k), 4 * p)
    # heads are independent
    assert orc.head_priority(k[:, 1:2])[0] == p[1]


def test_outlier_heads_keep_four_bits(orc):
    """Heads with a few large-magnitude channels (Fig. 3) get the highest
    priority and stay 4-bit; the others go to 2 bits."""
    rng = np.random.default_rng(1)
    k = rng.standard_normal((2, 8, 64, 128)).astype(np.float32)
    outlier_heads = [1, 4, 6, 7]
    for h in outlier_heads:
        k[:, h, :, rng.choice(128, 4, replace=False)] *= 10
    k = k.astype(np.float16).astype(np.float32)
    p = orc.head_priority(k)
    bits = orc.int2_heads(p, 4)
    assert [int(b) for b in bits] == [4 if h in outlier_heads else 2 for h in range(8)]


def test_rank_rule_and_ties(orc):
    assert list(orc.int2_heads([3.0, 1.0, 1.0, 5.0], 2)) == [4, 2, 2, 4]
    assert list(orc.int2_heads([1.0, 1.0, 1.0, 1.0], 2)) == [2, 2, 4, 4]   # ties: lower index first
    assert list(orc.int2_heads([2.0, 0.5, 7.0], 0)) == [4, 4, 4]
    assert list(orc.int2_heads([2.0, 0.5, 7.0], 3)) == [2, 2, 2]
