"""GPU parity of the method's integers, bit for bit: through the *_trace test
hooks of the C ABI, the gfx950 kernels store the int8 Q block, the int32 QK^T
accumulators, the Q(P~) codes, the int32 PV accumulators, s_Q and the P~
maximum of one selected tile (prefill) or group (decode); the oracle's trace
of the same tile is computed from the same seeded inputs.  The trace instance
is the production kernel with stores added, so its output is also compared,
bit for bit, with the plain call's.
"""
import sys

import numpy as np
import pytest
import torch

from tests.decode_split import split_of

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def ta(dev):
    import paper_2412_08585_amd as ta
    ta.lib()
    return ta


def _rand(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(*shape, generator=g) * scale).half()


def _same_f32(a, b):
    return np.float32(a).view(np.int32) == np.float32(b).view(np.int32)


PREFILL_TRACE_CASES = [
    # B, Hq, Hkv, N, causal, tiles (b, h, i, j)
    (1, 4, 4, 512, True, [(0, 0, 7, 7), (0, 1, 5, 2), (0, 3, 0, 0)]),
    (2, 8, 2, 64 * 3 + 40, True, [(1, 5, 3, 3), (0, 2, 3, 1), (1, 7, 2, 0)]),
    (1, 3, 3, 64 * 2 + 63, False, [(0, 1, 0, 2), (0, 2, 2, 1)]),
    (1, 16, 1, 200, True, [(0, 9, 3, 2)]),
]


@pytest.mark.parametrize("B,Hq,Hkv,N,causal,tiles", PREFILL_TRACE_CASES)
def test_prefill_tile_integers_bit_exact(orc, ta, dev, B, Hq, Hkv, N, causal, tiles):
    q = _rand((B, Hq, N, 128), 1300 + N)
    k = _rand((B, Hkv, N, 128), 1400 + N)
    v = _rand((B, Hkv, N, 128), 1500 + N)
    k[..., 5] *= 10
    sm = 1 / np.sqrt(128)
    k8, v8, sk, sv = ta.turbo_quantize_kv(k.to(dev), v.to(dev))
    o_plain = ta.turbo_attn_prefill(q.to(dev), k8, v8, sk, sv, sm, causal)
    torch.cuda.synchronize()
    for (b, h, i, j) in tiles:
        _log(f"prefill trace B={B} Hq={Hq} Hkv={Hkv} N={N} causal={causal} tile={(b, h, i, j)}")
        o, g = ta.turbo_attn_prefill_trace(q.to(dev), k8, v8, sk, sv, (b, h, i, j), sm, causal)
        assert torch.equal(o.view(torch.int16), o_plain.view(torch.int16))
        _, _, r = orc.attn_prefill(q, k, v, sm, causal, trace=(b, h, i, j), qblocks=(i, i + 1))
        assert r["hit"] == 1
        nq, nk = min(64, N - 64 * i), min(64, N - 64 * j)
        rows = np.arange(64)[:, None]
        keys = np.arange(64)[None, :]
        vis = (rows < nq) & (keys < nk)
        if causal:
            vis &= 64 * j + keys <= 64 * i + rows
        assert np.array_equal(g["q8"], r["q8"]), "Q8"
        assert np.array_equal(g["sacc"][vis], r["sacc"][vis]), "QK^T accumulators"
        assert np.array_equal(g["qp"], r["qp"]), "Q(P~)"
        assert not g["qp"][~vis].any()
        assert np.array_equal(g["pvacc"], r["pvacc"]), "PV accumulators"
        assert _same_f32(g["sq"], r["sq"]) and _same_f32(g["pmax"], r["pmax"])
        # the masked entries of the GPU's S are still the plain integer products
        qi = g["q8"].astype(np.int64)
        kj = k8.cpu().numpy()[b, h // (Hq // Hkv), 64 * j:64 * j + 64].astype(np.int64)
        assert np.array_equal(g["sacc"], qi @ kj.T)


# Table 3's block sizes (and the two other pairs the kernels take): tiles
# (b, h, i, j) count B_r-row query blocks and B_c-key key blocks.  Chosen to
# cover diagonal tiles (for B_r > B_c also the tile whose first rows see no
# key), off-diagonal tiles, ragged last blocks and GQA.
BLOCK_TRACE_CASES = [
    # B_r, B_c, B, Hq, Hkv, N, causal, tiles
    (32, 32, 1, 4, 2, 64 * 4 + 20, True, [(0, 1, 8, 8), (0, 3, 5, 2), (0, 0, 8, 0)]),
    (32, 64, 2, 4, 1, 200, True, [(1, 2, 6, 3), (0, 1, 3, 1), (1, 0, 0, 0)]),
    (64, 32, 1, 2, 2, 64 * 3 + 33, True, [(0, 1, 2, 5), (0, 0, 3, 6), (0, 1, 1, 1), (0, 0, 3, 0)]),
    (64, 128, 1, 4, 2, 64 * 5 + 7, True, [(0, 3, 5, 2), (0, 1, 2, 1), (0, 2, 4, 0)]),
    (128, 64, 2, 4, 2, 64 * 5 + 9, True, [(1, 3, 2, 5), (0, 0, 1, 3), (1, 1, 2, 4), (0, 2, 1, 0)]),
    (128, 128, 1, 2, 1, 64 * 6 + 50, True, [(0, 1, 3, 3), (0, 0, 2, 1), (0, 1, 1, 1)]),
    (32, 128, 1, 2, 2, 64 * 4 + 12, True, [(0, 0, 8, 2), (0, 1, 5, 1)]),
    (128, 32, 1, 2, 1, 64 * 4 + 12, True, [(0, 1, 2, 8), (0, 1, 1, 7), (0, 0, 1, 4), (0, 1, 2, 0)]),
    (64, 64, 1, 2, 2, 64 * 3 + 10, False, [(0, 1, 1, 3)]),
    (128, 64, 1, 2, 1, 64 * 3 + 10, False, [(0, 0, 0, 3), (0, 1, 1, 0)]),
    (32, 128, 1, 2, 1, 64 * 3 + 10, False, [(0, 1, 2, 1)]),
]


@pytest.mark.parametrize("br,bc,B,Hq,Hkv,N,causal,tiles", BLOCK_TRACE_CASES)
def test_prefill_block_size_tile_integers_bit_exact(orc, ta, dev, br, bc, B, Hq, Hkv, N, causal,
                                                    tiles):
    q = _rand((B, Hq, N, 128), 2300 + N + br)
    k = _rand((B, Hkv, N, 128), 2400 + N + bc)
    v = _rand((B, Hkv, N, 128), 2500 + N)
    k[..., 6] *= 10
    sm = 1 / np.sqrt(128)
    k8, v8, sk, sv = ta.turbo_quantize_kv(k.to(dev), v.to(dev), block_cols=bc)
    o_plain = ta.turbo_attn_prefill(q.to(dev), k8, v8, sk, sv, sm, causal, block_rows=br,
                                    block_cols=bc)
    torch.cuda.synchronize()
    k8h = k8.cpu().numpy()
    nkeys = k8h.shape[2]  # key rows held (64 ceil(N / 64))
    for (b, h, i, j) in tiles:
        _log(f"prefill trace B_r={br} B_c={bc} B={B} Hq={Hq} Hkv={Hkv} N={N} causal={causal} "
             f"tile={(b, h, i, j)}")
        o, g = ta.turbo_attn_prefill_trace(q.to(dev), k8, v8, sk, sv, (b, h, i, j), sm, causal,
                                           block_rows=br, block_cols=bc)
        assert torch.equal(o.view(torch.int16), o_plain.view(torch.int16))
        _, _, r = orc.attn_prefill(q, k, v, sm, causal, trace=(b, h, i, j), qblocks=(i, i + 1),
                                   block_rows=br, block_cols=bc)
        assert r["hit"] == 1
        nq, nk = min(br, N - br * i), min(bc, N - bc * j)
        rows = np.arange(br)[:, None]
        keys = np.arange(bc)[None, :]
        vis = (rows < nq) & (keys < nk)
        if causal:
            vis &= bc * j + keys <= br * i + rows
        assert np.array_equal(g["q8"], r["q8"]), "Q8"
        assert np.array_equal(g["sacc"][vis], r["sacc"][vis]), "QK^T accumulators"
        assert np.array_equal(g["qp"], r["qp"]), "Q(P~)"
        assert not g["qp"][~vis].any()
        assert np.array_equal(g["pvacc"], r["pvacc"]), "PV accumulators"
        assert _same_f32(g["sq"], r["sq"]) and _same_f32(g["pmax"], r["pmax"])
        # the GPU's S of every key it holds is the plain product (masked ones too)
        held = min(bc, nkeys - bc * j)
        qi = g["q8"].astype(np.int64)
        kj = k8h[b, h // (Hq // Hkv), bc * j:bc * j + held].astype(np.int64)
        assert np.array_equal(g["sacc"][:, :held], qi @ kj.T)


def test_prefill_trace_of_an_unprocessed_tile_writes_nothing(ta, dev):
    N = 64 * 3
    q, k, v = _rand((1, 2, N, 128), 1), _rand((1, 2, N, 128), 2), _rand((1, 2, N, 128), 3)
    k8, v8, sk, sv = ta.turbo_quantize_kv(k.to(dev), v.to(dev))
    _, g = ta.turbo_attn_prefill_trace(q.to(dev), k8, v8, sk, sv, (0, 1, 0, 2))  # j > i, causal
    assert not any(np.asarray(x).any() for x in g.values())


DECODE_TRACE_CASES = [
    # B, Hq, Hkv, Nc, bits, seq_lens, split, (b, h, g) groups
    (3, 8, 2, 64 * 6, [4, 2], [384, 200, 0], 2, [(0, 1, 0), (0, 5, 4), (1, 6, 2), (1, 2, 3)]),
    (2, 4, 4, 64 * 4, [2, 4, 4, 2], [256, 256], 1, [(1, 0, 3), (0, 2, 1)]),
    (1, 16, 1, 64 * 8, [4], [512], 3, [(0, 13, 5), (0, 0, 7)]),
    # two and eight query heads per KV head (the GP = 2 and GP = 8 instances)
    (2, 4, 2, 64 * 5, [2, 4], [320, 192], 2, [(0, 1, 4), (1, 2, 2), (0, 3, 0)]),
    (2, 16, 2, 64 * 5, [4, 2], [320, 256], 0, [(0, 7, 3), (1, 12, 1), (1, 9, 3)]),
    # the default chunking with one sequence long enough for several chunks
    (1, 8, 2, 64 * 40, [4, 2], [64 * 40], 0, [(0, 2, 35), (0, 6, 3)]),
]


@pytest.mark.parametrize("B,Hq,Hkv,Nc,bits,sl,split,groups", DECODE_TRACE_CASES)
def test_decode_group_integers_bit_exact(orc, ta, dev, B, Hq, Hkv, Nc, bits, sl, split, groups):
    k = _rand((B, Hkv, Nc, 128), 1600 + Nc)
    v = _rand((B, Hkv, Nc, 128), 1700 + Nc)
    k[..., 9] *= 10
    q = _rand((B, Hq, 128), 1800 + Nc)
    sm = 1 / np.sqrt(128)
    mg = Nc // 64
    rng = np.random.default_rng(Nc)
    bt = rng.permutation(B * 4 * mg).astype(np.int32).reshape(B, 4 * mg)
    gt = rng.permutation(B * mg).astype(np.int32).reshape(B, mg)
    cache = ta.PagedKVCache(bt.size, gt.size, bits, dev)
    btd, gtd = torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)
    ta.turbo_quantize_kv(k.to(dev), v.to(dev), cache, btd, gtd)
    sld = torch.tensor(sl, dtype=torch.int32, device=dev)
    o_plain = ta.turbo_attn_decode(q.to(dev), cache, sld, btd, gtd, sm, split)
    torch.cuda.synchronize()
    ref = orc.quantize_kv(k, v, bits)
    for (b, h, gi) in groups:
        _log(f"decode trace B={B} Hq={Hq} Hkv={Hkv} bits={bits} split={split} group={(b, h, gi)}")
        o, g = ta.turbo_attn_decode_trace(q.to(dev), cache, sld, btd, gtd, (b, h, gi), sm, split)
        assert torch.equal(o.view(torch.int16), o_plain.view(torch.int16))
        _, _, r = orc.attn_decode(q, ref, sl, sm, split=split_of(sl[b], split, mg),
                                  trace=(b, h, gi))
        if not r["hit"]:  # group beyond the sequence: nothing traced on either side
            assert not any(np.asarray(x).any() for x in g.values())
            continue
        assert np.array_equal(g["q8"][0], r["q8"][0]), "Q8"
        assert np.array_equal(g["sacc"][0], r["sacc"][0]), "QK^T accumulators"
        assert np.array_equal(g["qp"][0], r["qp"][0]), "Q(P~)"
        assert np.array_equal(g["pvacc"][0], r["pvacc"][0]), "PV accumulators"
        assert _same_f32(g["sq"], r["sq"]) and _same_f32(g["pmax"], r["pmax"])
        assert not g["sacc"][1:].any() and not g["pvacc"][1:].any()
