"""Pins of the oracle's QKV projection + FlashQ (Sec. 5.2 fusion; Sec. 3.1):
output features are routed to query, key and value heads in that order, the
projection is rounded to fp16 (ties to even) before quantization, and the
codes equal those of the stand-alone quantizers on the same fp16 values."""
import numpy as np


def _select_weights(D, F, cols):
    """W [F][D] whose feature f copies input channel cols[f]."""
    w = np.zeros((F, D), np.float32)
    w[np.arange(F), cols] = 1.0
    return w


def test_routing_to_heads_and_agreement_with_the_quantizers(orc):
    rng = np.random.default_rng(0)
    B, N, Hq, Hkv, d = 2, 64 + 21, 2, 1, 128
    F = (Hq + 2 * Hkv) * d
    D = F
    x = rng.standard_normal((B, N, D)).astype(np.float16).astype(np.float32)
    perm = rng.permutation(D)
    out = orc.qkv_project(x, _select_weights(D, F, perm), Hq, Hkv, [2])
    y = x[:, :, perm]                                   # the exact projection
    for h in range(Hq):
        assert np.array_equal(out["q"][:, h], y[:, :, h * d:(h + 1) * d])
    assert np.array_equal(out["k"][:, 0], y[:, :, Hq * d:(Hq + 1) * d])
    assert np.array_equal(out["v"][:, 0], y[:, :, (Hq + 1) * d:])
    ref = orc.quantize_kv(out["k"], out["v"], [2])
    for key in ("k8", "v8", "sk", "sv", "kc", "vc", "ks", "kz", "vs", "vz"):
        assert np.array_equal(out[key], ref[key]), key
    # Q: one symmetric block per 64 rows of a head
    for blk in range(2):
        rows = slice(64 * blk, min(N, 64 * blk + 64))
        qb, sb = orc.block_quant(out["q"][:, :, rows].reshape(B, Hq, -1))
        assert np.array_equal(out["q8"][:, :, rows].reshape(B, Hq, -1), qb)
        assert np.array_equal(out["sq"][:, :, blk], sb)


def test_fp16_rounding_of_the_projection(orc):
    """x . w = 1 + 2^-11 lies halfway between the fp16 neighbours 1 and
    1 + 2^-10: it rounds to the even one, 1; 1 + 3 * 2^-11 rounds up."""
    d, Hq, Hkv = 128, 1, 1
    F = (Hq + 2 * Hkv) * d
    D = 2
    w = np.zeros((F, D), np.float32)
    w[:, 0] = 1.0
    w[:, 1] = 2.0 ** -11
    x = np.zeros((1, 2, D), np.float32)
    x[0, 0] = [1.0, 1.0]       # 1 + 2^-11
    x[0, 1] = [1.0, 3.0]       # 1 + 3 * 2^-11
    out = orc.qkv_project(x, w, Hq, Hkv, [4])
    assert out["q"][0, 0, 0, 0] == 1.0
    assert out["q"][0, 0, 1, 0] == np.float32(1.0 + 2.0 ** -9)


def test_scaled_weights_scale_the_block_scales(orc):
    """Doubling W doubles every fp16 output exactly, hence every block scale,
    and leaves the codes unchanged."""
    rng = np.random.default_rng(1)
    B, N, D, Hq, Hkv = 1, 70, 64, 2, 1
    F = (Hq + 2 * Hkv) * 128
    x = rng.standard_normal((B, N, D)).astype(np.float16).astype(np.float32)
    w = (rng.standard_normal((F, D)) / 8).astype(np.float16).astype(np.float32)
    a = orc.qkv_project(x, w, Hq, Hkv, [4])
    b = orc.qkv_project(x, 2 * w, Hq, Hkv, [4])
    for key in ("q8", "k8", "v8"):
        assert np.array_equal(a[key], b[key])
    for key in ("sq", "sk", "sv"):
        assert np.array_equal(2 * a[key], b[key])


def test_project_exact_against_integer_products(orc):
    """The exact projection and its absolute-value sum against integer
    arithmetic (inputs i/8 and j/64 make every product a multiple of 2^-9)."""
    rng = np.random.default_rng(3)
    x = rng.integers(-8, 9, (5, 7, 96))
    w = rng.integers(-8, 9, (40, 96))
    y, yabs = orc.project_exact(x / 8.0, w / 64.0)
    ii = np.einsum("bnd,fd->bnf", x, w)
    ia = np.einsum("bnd,fd->bnf", np.abs(x), np.abs(w))
    assert np.array_equal(y * 512, ii.astype(np.float64))
    assert np.array_equal(yabs * 512, ia.astype(np.float64))
