"""Pins of the oracle's int8 KV-cache buffer (Sec. 3.3): buffer start after a
prefill, one-token appends with a universal scale and clamping, the flush of
a full buffer into a step-2 group, and decode over groups plus the buffer."""
import numpy as np
import pytest

SM = 1 / np.sqrt(128)


def _f16(rng, shape, scale=1.0):
    return (rng.standard_normal(shape) * scale).astype(np.float16).astype(np.float32)


def _dequant(cache, b, h, ng):
    """K^{q1} s_K and V^{q1} s_V of the first ng groups (Sec. 2.3: code*s + z)."""
    d = cache["kc"].shape[3]
    K, V = [], []
    for g in range(ng):
        sl = slice(64 * g, 64 * g + 64)
        k1 = cache["kc"][b, h, sl].astype(np.int32) * cache["ks"][b, h, g] + cache["kz"][b, h, g]
        v1 = cache["vc"][b, h, sl].astype(np.int32) * cache["vs"][b, h, g] + cache["vz"][b, h, g]
        K.append(k1 * np.float64(cache["sk"][b, h, g]))
        V.append(v1 * np.float64(cache["sv"][b, h, g]))
    return (np.concatenate(K) if K else np.zeros((0, d)), np.concatenate(V) if V else np.zeros((0, d)))


def test_tail_init_scale_and_codes(orc):
    rng = np.random.default_rng(0)
    B, H, N = 2, 3, 64 * 2 + 21
    k, v = _f16(rng, (B, H, N, 128)), _f16(rng, (B, H, N, 128), 3.0)
    qkv = orc.quantize_kv(k, v, [4] * H)
    t = orc.tail_init(k, v, qkv)
    # the universal scale is the largest block scale; the 21 trailing tokens are
    # inside its range, so their codes are within half a step of x / s
    assert np.array_equal(t["tsk"], qkv["sk"].max(axis=2))
    assert np.array_equal(t["tsv"], qkv["sv"].max(axis=2))
    for b in range(B):
        for h in range(H):
            tail_k, tail_v = k[b, h, 128:], v[b, h, 128:]
            ek = np.abs(t["tk"][b, h, :21] * np.float64(t["tsk"][b, h]) - tail_k)
            ev = np.abs(t["tv"][b, h, :, :21].T * np.float64(t["tsv"][b, h]) - tail_v)
            # half a step, plus the effect of inv = 1/s rounded to binary32
            # (at most 119 * 2^-23 of a step for codes up to 119)
            assert ek.max() <= (0.5 + 119 * 2.0**-23) * t["tsk"][b, h]
            assert ev.max() <= (0.5 + 119 * 2.0**-23) * t["tsv"][b, h]
            assert not t["tk"][b, h, 21:].any() and not t["tv"][b, h, :, 21:].any()


def test_append_clamps_to_the_universal_range(orc):
    rng = np.random.default_rng(1)
    B, H, N = 1, 2, 64
    k, v = _f16(rng, (B, H, N, 128)), _f16(rng, (B, H, N, 128))
    qkv = orc.quantize_kv(k, v, [4, 4])
    cache = orc.cache_from_prefill(qkv, 64 * 3)
    t = orc.tail_init(k, v, qkv)
    kn, vn = _f16(rng, (B, H, 128)), _f16(rng, (B, H, 128))
    kn[0, 0, 5] = 1000.0 * t["tsk"][0, 0]
    kn[0, 0, 6] = -1000.0 * t["tsk"][0, 0]
    orc.append_kv(cache, t, kn, vn, [N])
    assert t["tk"][0, 0, 0, 5] == 119 and t["tk"][0, 0, 0, 6] == -119
    err = np.abs(t["tk"][0, 1, 0] * np.float64(t["tsk"][0, 1]) - kn[0, 1])
    assert err.max() <= (0.5 + 119 * 2.0**-23) * t["tsk"][0, 1]


@pytest.mark.parametrize("bits", [[4, 2], [2, 4]])
def test_flush_is_step2_of_the_buffer(orc, bits):
    """64 appends after a 64-token prefill fill the buffer; the 64th writes
    group 1 as step 2 of the buffered codes, with the universal scales."""
    rng = np.random.default_rng(2)
    B, H = 2, 2
    k, v = _f16(rng, (B, H, 64, 128)), _f16(rng, (B, H, 64, 128))
    qkv = orc.quantize_kv(k, v, bits)
    cache = orc.cache_from_prefill(qkv, 64 * 3)
    t = orc.tail_init(k, v, qkv)
    before = {key: cache[key].copy() for key in ("kc", "vc", "ks", "kz", "vs", "vz")}
    new_k, new_v = _f16(rng, (64, B, H, 128), 0.5), _f16(rng, (64, B, H, 128), 0.5)
    for i in range(64):
        orc.append_kv(cache, t, new_k[i], new_v[i], [64 + i] * B)
        if i < 63:  # nothing is compressed before the buffer is full
            assert all(np.array_equal(cache[key], before[key]) for key in before)
    for b in range(B):
        for h in range(H):
            ks, kz, kc = orc.step2(t["tk"][b, h], bits[h])
            vs, vz, vc = orc.step2(np.ascontiguousarray(t["tv"][b, h].T), bits[h])
            assert np.array_equal(cache["ks"][b, h, 1], ks) and np.array_equal(cache["kz"][b, h, 1], kz)
            assert np.array_equal(cache["kc"][b, h, 64:128], kc)
            assert np.array_equal(cache["vs"][b, h, 1], vs) and np.array_equal(cache["vz"][b, h, 1], vz)
            assert np.array_equal(cache["vc"][b, h, 64:128], vc)
            assert cache["sk"][b, h, 1] == t["tsk"][b, h] and cache["sv"][b, h, 1] == t["tsv"][b, h]
            # the compressed group stays within the two quantization steps' error
            kd, _ = _dequant(cache, b, h, 2)
            s = np.float64(t["tsk"][b, h])
            bound = s * (0.5 + 119 * 2.0**-23 + 0.5 * cache["ks"][b, h, 1].astype(np.float64))
            assert np.all(np.abs(kd[64:] - new_k[:, b, h]) <= bound)
    assert not cache["kc"][:, :, 128:].any()  # group 2 untouched


@pytest.mark.parametrize("split", [1, 2, 100])
def test_decode_with_buffer_reduces_to_exact_attention(orc, split):
    """FlashQ and SAS off: decode over the groups and the buffer is exact
    softmax attention over their dequantized keys and values, whatever the
    chunking (the merge of chunks is then exact too)."""
    rng = np.random.default_rng(3)
    B, Hq, H, N = 2, 4, 2, 64 * 3 + 29
    k, v = _f16(rng, (B, H, N, 128)), _f16(rng, (B, H, N, 128))
    qkv = orc.quantize_kv(k, v, [4, 2])
    cache = orc.cache_from_prefill(qkv, 64 * 5)
    t = orc.tail_init(k, v, qkv)
    kn, vn = _f16(rng, (B, H, 128)), _f16(rng, (B, H, 128))
    orc.append_kv(cache, t, kn, vn, [N, N])          # one decoding step
    sl = [N + 1, 40]  # sequence 1 attends no group, only 40 buffered tokens
    q = _f16(rng, (B, Hq, 128))
    o, lse = orc.attn_decode(q, cache, sl, SM, split=split, quant=False, sas=False, tail=t)
    for b in range(B):
        ng, nt = sl[b] // 64, sl[b] % 64
        for h in range(Hq):
            kh = h // (Hq // H)
            kd, vd = _dequant(cache, b, kh, ng)
            kt = t["tk"][b, kh, :nt] * np.float64(t["tsk"][b, kh])
            vt = t["tv"][b, kh, :, :nt].T * np.float64(t["tsv"][b, kh])
            K, V = np.concatenate([kd, kt]), np.concatenate([vd, vt])
            s = K @ q[b, h].astype(np.float64) * np.float64(np.float32(SM))
            w = np.exp(s - s.max())
            ref = w @ V / w.sum()
            # the oracle holds the unquantized V rows in binary32 (vf), hence 1e-6
            assert np.abs(o[b, h] - ref).max() <= 1e-6 * np.abs(ref).max()
            np.testing.assert_allclose(lse[b, h], s.max() + np.log(w.sum()), rtol=1e-12)


def test_empty_buffer_changes_nothing(orc):
    rng = np.random.default_rng(4)
    B, Hq, H, N = 1, 2, 1, 128
    k, v = _f16(rng, (B, H, N, 128)), _f16(rng, (B, H, N, 128))
    qkv = orc.quantize_kv(k, v, [4])
    t = orc.tail_init(k, v, qkv)
    q = _f16(rng, (B, Hq, 128))
    for split in (1, 3):
        a = orc.attn_decode(q, qkv, [N], SM, split=split)
        b = orc.attn_decode(q, qkv, [N], SM, split=split, tail=t)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_buffer_trace_is_brute_force(orc):
    rng = np.random.default_rng(5)
    B, Hq, H, N = 1, 2, 1, 64 + 37
    k, v = _f16(rng, (B, H, N, 128)), _f16(rng, (B, H, N, 128))
    qkv = orc.quantize_kv(k, v, [2])
    t = orc.tail_init(k, v, qkv)
    q = _f16(rng, (B, Hq, 128))
    _, _, tr = orc.attn_decode(q, qkv, [N], SM, split=1, tail=t, trace=(0, 1, 1))
    assert tr["hit"] == 1
    q8 = tr["q8"][0].astype(np.int64)
    want = t["tk"][0, 0, :37].astype(np.int64) @ q8
    assert np.array_equal(tr["sacc"][0, :37], want)
    assert not tr["qp"][0, 37:].any()
    pv = tr["qp"][0, :37].astype(np.int64) @ t["tv"][0, 0, :, :37].T.astype(np.int64)
    assert np.array_equal(tr["pvacc"][0], pv)
