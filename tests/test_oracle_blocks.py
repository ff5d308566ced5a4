"""Pins of the oracle's block-size variants of Algorithm 1 (Table 3 varies the
query block B_r and the key block B_c over {32, 64, 128}): the partitions the
Q, K, V and P scales are taken over, the reduction to the 64 x 64 result or
to exact attention where quantization (and SAS) are off, and the rows of a
block that see no key of a tile being left untouched."""
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
    """With FlashQ off no scale depends on the block partition (SAS stays on),
    so the query block size changes nothing but the summation order."""
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


# ---- key blocks B_c (Table 3) ---------------------------------------------

@pytest.mark.parametrize("bc", [32, 128])
def test_step1_blocks_nest(orc, bc):
    """Step 1 over bc-token blocks: the scale of a 64-token block is the
    larger of its two 32-token scales, and a 128-token scale the larger of its
    two 64-token scales (the rounding of amax/119 is monotone); codes agree
    wherever the scales agree."""
    q, k, v = _qkv(5, 2, 1, 2, 64 * 4 + 50)
    v[:, :, 64 * 2:64 * 2 + 40] *= 3
    fine, coarse = (32, 64) if bc == 32 else (64, 128)
    a = orc.quantize_kv_blocks(k, v, fine)
    c = orc.quantize_kv_blocks(k, v, coarse)
    ref = orc.quantize_kv(k, v, [4, 4])
    b64 = a if fine == 64 else c
    for key in ("k8", "v8", "sk", "sv"):
        assert np.array_equal(b64[key], ref[key]), key
    N = k.shape[2]
    for s, x8 in (("sk", "k8"), ("sv", "v8")):
        nf = a[s].shape[-1]
        pad = np.zeros(a[s].shape[:-1] + (2 * c[s].shape[-1] - nf,), np.float32)
        pairs = np.concatenate([a[s], pad], -1).reshape(a[s].shape[:-1] + (-1, 2))
        assert np.array_equal(pairs.max(-1), c[s]), s
        # codes equal in every fine block whose scale equals the coarse one
        for j in range(nf):
            rows = slice(fine * j, min(N, fine * j + fine))
            same = a[s][..., j] == c[s][..., j // 2]
            assert np.array_equal(a[x8][:, :, rows][same], c[x8][:, :, rows][same])
    # a direct check of one block against the definition
    blk = k[0, 1, bc:2 * bc] if 2 * bc <= N else k[0, 1, :bc]
    j = 1 if 2 * bc <= N else 0
    e = orc.quantize_kv_blocks(k, v, bc)
    assert e["sk"][0, 1, j] == np.float32(np.abs(blk).max()) / np.float32(119)


@pytest.mark.parametrize("br,bc", [(32, 32), (64, 32), (64, 128), (128, 128), (32, 128)])
@pytest.mark.parametrize("causal", [True, False])
def test_key_blocks_reduce_to_exact_attention(orc, br, bc, causal):
    q, k, v = _qkv(6, 1, 4, 2, 64 * 3 + 45)
    o, lse = orc.attn_prefill(q, k, v, SM, causal, quant=False, sas=False, block_rows=br,
                              block_cols=bc)
    ex, lex = orc.attn_exact(q, k, v, float(np.float32(SM)), causal)
    np.testing.assert_allclose(o, ex, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lex, rtol=0, atol=1e-12)


def _split_v(v, lo, hi):
    va, vb = v.copy(), v.copy()
    va[:, :, lo:hi] = 0
    vb[:, :, :lo] = 0
    vb[:, :, hi:] = 0
    return va, vb


@pytest.mark.parametrize("bc,split", [(32, 32), (64, 64)])
def test_v_scales_follow_the_key_blocks(orc, bc, split):
    """P~ and its codes do not depend on V, and a V block that is all zero has
    scale 0: so O(V) = O(V_a) + O(V_b) exactly (up to double rounding) when
    V_a, V_b split V along a boundary of the V blocks, and not otherwise
    (the block scales of V_a differ from V's)."""
    q, k, v = _qkv(7, 1, 2, 1, 2 * split)
    v[:, :, split:] *= 3                    # the block maximum lies after the split
    kw = dict(block_cols=bc)
    o, _ = orc.attn_prefill(q, k, v, SM, False, **kw)
    va, vb = _split_v(v, split, 2 * split)
    oa, _ = orc.attn_prefill(q, k, va, SM, False, **kw)
    ob, _ = orc.attn_prefill(q, k, vb, SM, False, **kw)
    np.testing.assert_allclose(oa + ob, o, rtol=0, atol=1e-12)
    coarse = 64 if bc == 32 else 128
    o2, _ = orc.attn_prefill(q, k, v, SM, False, block_cols=coarse)
    oa2, _ = orc.attn_prefill(q, k, va, SM, False, block_cols=coarse)
    ob2, _ = orc.attn_prefill(q, k, vb, SM, False, block_cols=coarse)
    assert np.abs(oa2 + ob2 - o2).max() > 1e-4


@pytest.mark.parametrize("fine,coarse", [(32, 64), (64, 128)])
def test_kv_scales_follow_the_key_blocks(orc, fine, coarse):
    """Causal rows before key `fine` see only the first key block.  Scaling K
    and V after it by 8 leaves those rows bit-identical when B_c = fine (their
    block's scales are its own) and changes them when B_c = coarse (the block
    scale now covers the scaled keys)."""
    q, k, v = _qkv(8, 1, 2, 1, 2 * fine)
    k2, v2 = k.copy(), v.copy()
    k2[:, :, fine:] *= 8
    v2[:, :, fine:] *= 8
    rows = slice(0, fine)
    for bc, same in ((fine, True), (coarse, False)):
        a, la = orc.attn_prefill(q, k, v, SM, True, block_rows=32, block_cols=bc)
        b, lb = orc.attn_prefill(q, k2, v2, SM, True, block_rows=32, block_cols=bc)
        eq = np.array_equal(a[:, :, rows], b[:, :, rows]) and np.array_equal(la[:, :, rows],
                                                                             lb[:, :, rows])
        assert eq == same, (bc, same)


@pytest.mark.parametrize("br,bc", [(32, 32), (128, 64), (64, 128), (128, 128), (32, 128)])
def test_traced_tile_integers_for_other_block_sizes(orc, br, bc):
    """The trace of a (B_r-row, B_c-key) tile: the Q block codes are step 1 of
    its B_r rows, the accumulators are integer matrix products over the
    visible pairs, Q(P~) is 0 where masked and 119 somewhere, and PV is Q(P~)
    times the B_c-key V block."""
    N = 300
    q, k, v = _qkv(9, 1, 2, 1, N)
    kb = orc.quantize_kv_blocks(k, v, bc)
    nbq, nbc = -(-N // br), -(-N // bc)
    for i, j in [(nbq - 1, (nbq - 1) * br // bc), (nbq - 1, 0), (1, (br + br - 1) // bc)]:
        if j >= nbc or j * bc > i * br + br - 1:
            continue
        _, _, tr = orc.attn_prefill(q, k, v, SM, True, trace=(0, 1, i, j), block_rows=br,
                                    block_cols=bc)
        assert tr["hit"]
        r0, k0 = i * br, j * bc
        nq, nk = min(br, N - r0), min(bc, N - k0)
        q8, s = orc.block_quant(q[0, 1, r0:r0 + nq].reshape(1, -1))
        assert np.array_equal(tr["q8"][:nq], q8.reshape(nq, 128)) and tr["sq"] == s[0]
        assert not tr["q8"][nq:].any()
        vis = (np.arange(nk)[None, :] + k0) <= (np.arange(nq)[:, None] + r0)
        k8 = kb["k8"][0, 0, k0:k0 + nk].astype(np.int64)
        v8 = kb["v8"][0, 0, k0:k0 + nk].astype(np.int64)
        sacc = tr["q8"][:nq].astype(np.int64) @ k8.T
        assert np.array_equal(tr["sacc"][:nq, :nk][vis], sacc[vis])
        qp = tr["qp"][:nq, :nk].astype(np.int64)
        assert qp.min() >= 0 and qp.max() == 119 and not qp[~vis].any()
        assert np.array_equal(tr["pvacc"][:nq], qp @ v8)
