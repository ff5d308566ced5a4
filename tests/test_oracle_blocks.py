"""Pins of the oracle's block-size variants of Algorithm 1 (Table 3 varies the
query block B_r; key blocks stay 64): the partition the Q scale and the P
scale are taken over, the reduction to the 64-row result where quantization
is off, and the rows of a 128-row block that see no key of a tile being left
untouched."""
import numpy as np
import pytest

SM = 1 / np.sqrt(128)


def _qkv(seed, B, Hq, Hkv, N, kscale=1.0):
    rng = np.random.default_rng(seed)
    f = lambda *s: rng.standard_normal(s).astype(np.float16).astype(np.float32)
    k = f(B, Hkv, N, 128)
    k[..., 3] *= 10 * kscale
    return f(B, Hq, N, 128), k, f(B, Hkv, N, 128)


@pytest.mark.parametrize("causal", [True, False])
def test_one_block_is_the_same_for_every_block_size(orc, causal):
    q, k, v = _qkv(0, 1, 2, 1, 29)
    ref = orc.attn_prefill(q, k, v, SM, causal)
    for br in (32, 128):
        o, lse = orc.attn_prefill(q, k, v, SM, causal, block_rows=br)
        assert np.array_equal(o, ref[0]) and np.array_equal(lse, ref[1])


@pytest.mark.parametrize("br", [32, 128])
@pytest.mark.parametrize("causal", [True, False])
def test_without_quantization_the_block_size_does_not_matter(orc, br, causal):
    """With FlashQ off no scale depends on the block partition; SAS stays on,
    so a row of a 128-row block that were processed with a tile it sees no
    key of would pick up a factor SAS(0) in l (its L would move by ln 0.9996)."""
    q, k, v = _qkv(1, 2, 4, 2, 64 * 3 + 41)
    o64, l64 = orc.attn_prefill(q, k, v, SM, causal, quant=False)
    o, lse = orc.attn_prefill(q, k, v, SM, causal, quant=False, block_rows=br)
    np.testing.assert_allclose(o, o64, rtol=0, atol=1e-14)
    np.testing.assert_allclose(lse, l64, rtol=0, atol=1e-13)


@pytest.mark.parametrize("br", [32, 128])
def test_exact_attention_with_everything_off(orc, br):
    q, k, v = _qkv(2, 1, 2, 2, 200)
    o, lse = orc.attn_prefill(q, k, v, SM, True, quant=False, sas=False, block_rows=br)
    ex, lex = orc.attn_exact(q, k, v, float(np.float32(SM)), True)
    np.testing.assert_allclose(o, ex, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lex, rtol=0, atol=1e-12)


def test_scales_follow_the_block_partition(orc):
    """Scaling Q rows 32..63 by 4 leaves rows 0..31 untouched when B_r = 32
    (their Q scale and P scale cover rows 0..31 only) but not when B_r = 64."""
    q, k, v = _qkv(3, 1, 1, 1, 64)
    q2 = q.copy()
    q2[:, :, 32:] *= 4
    a32, _ = orc.attn_prefill(q, k, v, SM, False, block_rows=32)
    b32, _ = orc.attn_prefill(q2, k, v, SM, False, block_rows=32)
    assert np.array_equal(a32[:, :, :32], b32[:, :, :32])
    a64, _ = orc.attn_prefill(q, k, v, SM, False)
    b64, _ = orc.attn_prefill(q2, k, v, SM, False)
    assert not np.array_equal(a64[:, :, :32], b64[:, :, :32])
    # the same one level up: rows 64..127 against rows 0..63 for B_r = 128 / 64
    q, k, v = _qkv(4, 1, 1, 1, 128)
    q2 = q.copy()
    q2[:, :, 64:] *= 4
    a64, _ = orc.attn_prefill(q, k, v, SM, False)
    b64, _ = orc.attn_prefill(q2, k, v, SM, False)
    assert np.array_equal(a64[:, :, :64], b64[:, :, :64])
    a128, _ = orc.attn_prefill(q, k, v, SM, False, block_rows=128)
    b128, _ = orc.attn_prefill(q2, k, v, SM, False, block_rows=128)
    assert not np.array_equal(a128[:, :, :64], b128[:, :, :64])
