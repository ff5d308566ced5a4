"""Pins of the oracle's FlashQ steps (Sec. 2.3; Sec. 3.1 eq. step1bpq / step2bpq;
the quantization lines of Algorithms 1 and 2) by invariants and brute force."""
import numpy as np
import pytest


@pytest.mark.parametrize("seed", range(4))
def test_block_quant_invariants(orc, seed):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((50, 64 * 128)) * rng.uniform(0.01, 30, (50, 1))).astype(np.float16)
    x = x.astype(np.float32)
    q, s = orc.block_quant(x)
    amax = np.abs(x).max(axis=1)
    assert np.all(s == (amax / np.float32(119)).astype(np.float32))
    assert np.all(np.abs(q.astype(np.int32)) <= 119)
    # the element of largest magnitude maps to +-119
    i = np.abs(x).argmax(axis=1)
    assert np.all(np.abs(q[np.arange(50), i]) == 119)
    # round-to-nearest: |x - q s| <= s/2 up to the rounding of 119/amax
    err = np.abs(x.astype(np.float64) - q.astype(np.float64) * s[:, None].astype(np.float64))
    assert np.all(err <= s[:, None].astype(np.float64) * (0.5 + 1e-5))
    # sign preserved, zero maps to zero
    assert np.all(np.sign(q) == np.sign(np.where(np.abs(x) * 119 / amax[:, None] < 0.5, 0, x)))


def test_block_quant_zero_block_and_ties(orc):
    q, s = orc.block_quant(np.zeros((1, 300), np.float32))
    assert s[0] == 0 and not q.any()
    # amax = 119 -> 119/amax = 1 exactly: x.5 values are exact ties -> even
    x = np.float32([[119.0, 2.5, 3.5, -2.5, -3.5, 0.5, 1.5, -0.5, 118.5]])
    q, s = orc.block_quant(x)
    assert s[0] == 1.0
    assert q[0].tolist() == [119, 2, 4, -2, -4, 0, 2, 0, 118]


def _brute_groups():
    """One 64-value group for every (min, max) pair in [-119, 119]^2 with
    min <= max: both ends plus 62 values spread between them."""
    mn, mx = np.meshgrid(np.arange(-119, 120), np.arange(-119, 120), indexing="ij")
    keep = mn <= mx
    mn, mx = mn[keep], mx[keep]
    t = np.linspace(0, 1, 62)[:, None]
    mid = np.round(mn[None, :] + t * (mx - mn)[None, :]).astype(np.int64)
    g = np.concatenate([mn[None, :], mid, mx[None, :]], axis=0).astype(np.int8)
    return g, mn, mx


@pytest.mark.parametrize("bits", [4, 2])
def test_step2_brute_force_all_ranges(orc, bits):
    g, mn, mx = _brute_groups()
    s, z, code = orc.step2(g, bits)
    levels = (1 << bits) - 1
    s = s.astype(np.int64)
    assert np.array_equal(z.astype(np.int64), mn)
    assert np.array_equal(s, np.maximum(1, -((mn - mx) // levels)))   # ceil(range/levels), >= 1
    assert code.max() <= levels
    deq = code.astype(np.int64) * s[None, :] + z.astype(np.int64)[None, :]
    # the dequantized value stays inside int8 and within half a step
    assert deq.min() >= -119 and deq.max() <= 127
    assert np.all(np.abs(deq - g.astype(np.int64)) * 2 <= s[None, :])
    # the nearest level is chosen (ties rounded up)
    lo = (g.astype(np.int64) - mn[None, :]) // s[None, :]
    rem = (g.astype(np.int64) - mn[None, :]) - lo * s[None, :]
    want = lo + (2 * rem >= s[None, :])
    assert np.array_equal(code.astype(np.int64), want)


def test_step2_tie_rounds_up(orc):
    # min 0, max 30 with 4 bits -> s = 2; (q - z)/s = 0.5, 1.5, 14.5 -> 1, 2, 15
    col = np.zeros((64, 1), np.int8)
    col[1, 0], col[2, 0], col[3, 0], col[4, 0] = 30, 1, 3, 29
    s, z, code = orc.step2(col, 4)
    assert s[0] == 2 and z[0] == 0
    assert code[1:5, 0].tolist() == [15, 1, 2, 15]


def test_quantize_kv_matches_pieces(orc):
    """Whole-cache FlashQ equals block_quant per 64-token block and step 2 per
    (group, channel); the partial tail block gets step 1 only."""
    rng = np.random.default_rng(9)
    B, H, N, d = 2, 3, 64 * 3 + 17, 128
    k = rng.standard_normal((B, H, N, d)).astype(np.float16)
    v = rng.standard_normal((B, H, N, d)).astype(np.float16)
    k[:, :, :, 5] *= 10
    bits = np.array([4, 2, 4])
    c = orc.quantize_kv(k, v, bits)
    for b in range(B):
        for h in range(H):
            for j in range(4):
                r0, r1 = 64 * j, min(N, 64 * j + 64)
                qk, sk = orc.block_quant(k[b, h, r0:r1].astype(np.float32).reshape(1, -1))
                assert sk[0] == c["sk"][b, h, j]
                assert np.array_equal(qk.reshape(r1 - r0, d), c["k8"][b, h, r0:r1])
            for g in range(3):
                s, z, code = orc.step2(c["v8"][b, h, 64 * g:64 * g + 64], int(bits[h]))
                assert np.array_equal(s, c["vs"][b, h, g]) and np.array_equal(z, c["vz"][b, h, g])
                assert np.array_equal(code, c["vc"][b, h, 64 * g:64 * g + 64])
    assert c["kc"].shape[2] == 192


def test_compression_ratio_closed_form():
    """Bytes per token and KV head: fp16 K+V = 512; int4 = 128 codes + 8 B of
    s/z per channel amortized over 64 tokens + 2 fp32 scales / 64 tokens."""
    d = 128
    fp16 = 2 * d * 2
    def per_token(bits):
        return 2 * d * bits / 8 + 4 * d / 64 + 8 / 64
    assert per_token(4) == 136.125 and per_token(2) == 72.125
    mixed = fp16 / ((per_token(4) + per_token(2)) / 2)
    # the paper reports a KV-cache reduction above 4.4x for half int2 heads
    assert mixed > 4.4
