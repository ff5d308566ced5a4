"""GPU parity of the fused QKV projection + FlashQ (turbo_qkv_project) and of
the prefill on pre-quantized Q (turbo_attn_prefill_q8), against the oracle.

Bar.  With small-integer inputs (x = i/8, w = j/64, |i|, |j| <= 8) every
partial sum of X W^T is a multiple of 2^-9 below 2^15, so the fp32 MFMA sums
and the oracle's float64 sums are the same exact number whatever their order,
and every byte the kernel writes is compared bit for bit: Q8/K8/V8 codes, the
block scales, and the int4/int2 cache groups.  With N(0,1) inputs the fp32
and float64 sums round to fp16 differently now and then; there each block
scale is within one fp16 step of the oracle's and each code within 1.
"""
import sys

import numpy as np
import pytest
import torch

from tests import cache_layout

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


def _inputs(B, N, D, Hq, Hkv, seed, exact=True):
    F = (Hq + 2 * Hkv) * 128
    rng = np.random.default_rng(seed)
    if exact:
        x = rng.integers(-8, 9, (B, N, D)).astype(np.float32) / 8
        w = rng.integers(-8, 9, (F, D)).astype(np.float32) / 64
        scale = 8.0
    else:
        x = rng.standard_normal((B, N, D)).astype(np.float32)
        w = (rng.standard_normal((F, D)) / np.sqrt(D)).astype(np.float32)
        scale = 10.0
    # 4 outlier channels per key head (Fig. 3)
    for h in range(Hkv):
        ch = (Hq + h) * 128 + rng.choice(128, 4, replace=False)
        w[ch] *= scale
    return x.astype(np.float16), w.astype(np.float16)


def _tables(B, mg, seed):
    rng = np.random.default_rng(seed)
    bt = rng.permutation(B * 4 * mg).astype(np.int32).reshape(B, 4 * mg)
    gt = rng.permutation(B * mg).astype(np.int32).reshape(B, mg)
    return bt, gt


def _run(ta, dev, x, w, Hq, Hkv, bits, seed):
    B, N, _ = x.shape
    mg = max(1, N // 64)
    bt, gt = _tables(B, mg, seed)
    cache = ta.PagedKVCache(bt.size, gt.size, bits, dev)
    btd, gtd = torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)
    outs = ta.turbo_qkv_project(torch.from_numpy(x).to(dev), torch.from_numpy(w).to(dev), Hq, Hkv,
                                cache, btd, gtd)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in outs], cache, bt, gt


def _same_bits(a, b):
    return np.array_equal(np.asarray(a, np.float32).view(np.int32),
                          np.asarray(b, np.float32).view(np.int32))


EXACT_CASES = [
    # B, N, D, Hq, Hkv, bits
    (1, 64, 64, 1, 1, [4]),
    (2, 64 * 3 + 37, 256, 4, 2, [4, 2]),
    (2, 1024, 128, 2, 1, [2]),        # 8 token tiles: the XCD-grouped order
    (1, 300, 5120, 2, 1, [4]),        # the Phi-3-medium hidden width
    (1, 17, 64, 1, 1, [4]),           # no full group
    (3, 64 * 5, 192, 3, 3, [2, 4, 4]),
]


@pytest.mark.parametrize("B,N,D,Hq,Hkv,bits", EXACT_CASES)
def test_qkv_project_bit_exact(orc, ta, dev, B, N, D, Hq, Hkv, bits):
    _log(f"qkv_project exact B={B} N={N} D={D} Hq={Hq} Hkv={Hkv} bits={bits}")
    x, w = _inputs(B, N, D, Hq, Hkv, seed=N + D)
    (q8, sq, k8, v8, sk, sv), cache, bt, gt = _run(ta, dev, x, w, Hq, Hkv, bits, seed=N)
    ref = orc.qkv_project(x.astype(np.float32), w.astype(np.float32), Hq, Hkv, bits)
    nb = (N + 63) // 64
    assert np.array_equal(q8[:, :, :N], ref["q8"]) and not q8[:, :, N:].any(), "Q8"
    assert _same_bits(sq, ref["sq"]), "s_Q"
    assert np.array_equal(k8[:, :, :N], ref["k8"]) and not k8[:, :, N:].any(), "K8"
    v8t = v8.transpose(0, 1, 2, 4, 3).reshape(B, Hkv, nb * 64, 128)
    assert np.array_equal(v8t[:, :, :N], ref["v8"]) and not v8t[:, :, N:].any(), "V8"
    assert _same_bits(sk, ref["sk"]) and _same_bits(sv, ref["sv"]), "s_K, s_V"
    ng = N // 64
    if ng:
        pages = cache.pages.cpu().numpy()
        gmeta = cache.group_meta.cpu().numpy()
        gscale = cache.group_scale.cpu().numpy()
        for b in range(B):
            for h in range(Hkv):
                u = cache_layout.read_unit(pages, gmeta, gscale, bits, bt, gt, b, h, ng)
                for key in ("kc", "vc", "ks", "kz", "vs", "vz"):
                    assert np.array_equal(u[key], ref[key][b, h]), (b, h, key)
                assert _same_bits(u["sk"], ref["sk"][b, h, :ng])
                assert _same_bits(u["sv"], ref["sv"][b, h, :ng])


def test_projection_then_prefill_q8(orc, ta, dev):
    """Fused projection -> prefill on its Q8: bit-identical to the fp16-Q
    prefill on the oracle's fp16 Q, and within the O/L bar of the oracle's
    Algorithm 1 on the oracle's fp16 Q, K, V."""
    B, N, D, Hq, Hkv = 2, 64 * 3 + 20, 512, 4, 2
    _log("projection -> prefill_q8")
    x, w = _inputs(B, N, D, Hq, Hkv, seed=11)
    xd, wd = torch.from_numpy(x).to(dev), torch.from_numpy(w).to(dev)
    q8, sq, k8, v8, sk, sv = ta.turbo_qkv_project(xd, wd, Hq, Hkv)
    o8, l8 = ta.turbo_attn_prefill_q8(q8, sq, k8, v8, sk, sv, N, return_lse=True)
    ref = orc.qkv_project(x.astype(np.float32), w.astype(np.float32), Hq, Hkv, [4] * Hkv)
    q16 = torch.from_numpy(ref["q"]).half().to(dev)
    o16, l16 = ta.turbo_attn_prefill(q16, k8, v8, sk, sv, return_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(o8.view(torch.int16), o16.view(torch.int16))
    assert torch.equal(l8, l16)
    ro, rl = orc.attn_prefill(ref["q"], ref["k"], ref["v"], 1 / np.sqrt(128), True)
    g = o8.float().cpu().numpy()
    rowmax = np.maximum(np.abs(ro).max(axis=-1, keepdims=True), 1e-30)
    assert np.max(np.abs(g - ro) / rowmax) < 1e-3
    assert np.max(np.abs(l8.cpu().numpy() - rl)) < 1e-4


def _check_close(got_codes, got_s, ref_codes, ref_s, what):
    """Blocks of 64 rows x 128 (codes [..., rows, 128], scales [..., blocks]):
    every code within 1 and every block scale within one fp16 step (2^-10
    relative) of the oracle's; where the scales agree bit for bit, fewer
    than 1 % of the block's codes differ."""
    got_s = np.asarray(got_s, np.float32)
    ref_s = np.asarray(ref_s, np.float32)
    rel = np.abs(got_s.astype(np.float64) - ref_s) / np.maximum(ref_s, 1e-30)
    assert np.all(rel <= 2.0 ** -10 + 1e-7), f"{what}: scale off by {rel.max():.3e}"
    d = np.abs(got_codes.astype(np.int32) - ref_codes.astype(np.int32))
    assert d.max() <= 1, f"{what}: code off by {d.max()}"
    rows = d.shape[-2]
    for idx in np.ndindex(*got_s.shape):
        blk = d[idx[:-1]][64 * idx[-1]:min(rows, 64 * idx[-1] + 64)]
        if got_s[idx].view(np.int32) == ref_s[idx].view(np.int32):
            assert (blk != 0).mean() < 0.01, f"{what}: block {idx}: {(blk != 0).mean():.4f}"


def test_qkv_project_gaussian_inputs(orc, ta, dev):
    B, N, D, Hq, Hkv = 1, 256 + 40, 1024, 4, 2
    _log("qkv_project gaussian")
    x, w = _inputs(B, N, D, Hq, Hkv, seed=5, exact=False)
    (q8, sq, k8, v8, sk, sv), _, _, _ = _run(ta, dev, x, w, Hq, Hkv, [4, 4], seed=5)
    ref = orc.qkv_project(x.astype(np.float32), w.astype(np.float32), Hq, Hkv, [4, 4])
    _check_close(q8[:, :, :N], sq, ref["q8"], ref["sq"], "Q")
    _check_close(k8[:, :, :N], sk, ref["k8"], ref["sk"], "K")
    nb = (N + 63) // 64
    v8t = v8.transpose(0, 1, 2, 4, 3).reshape(B, Hkv, nb * 64, 128)[:, :, :N]
    _check_close(v8t, sv, ref["v8"], ref["sv"], "V")


def test_qkv_project_full_size_sampled(orc, ta, dev):
    """The benchmark's Phi-3-medium projection (4 x 4096 tokens, hidden 5120,
    40 + 2 x 10 heads) run in full; 12 (sequence, head, 64-token block) blocks
    recomputed by the oracle from their rows and features."""
    from paper_2412_08585_amd import workloads as W
    w_ = W.WORKLOADS["phi3m-qkv-4k"]
    x, wt = W.projection_inputs(w_, device=dev)
    Hq, Hkv = w_.Hq, w_.Hkv
    q8, sq, k8, v8, sk, sv = ta.turbo_qkv_project(x, wt, Hq, Hkv)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    for _ in range(12):
        b = int(rng.integers(w_.B))
        head = int(rng.integers(Hq + 2 * Hkv))
        j = int(rng.integers(w_.N // 64))
        rows = x[b, 64 * j:64 * j + 64].float().cpu().numpy().astype(np.float64)
        feats = wt[head * 128:(head + 1) * 128].float().cpu().numpy().astype(np.float64)
        y = (rows @ feats.T).astype(np.float16).astype(np.float32)
        codes, s = orc.block_quant(y.reshape(1, -1))
        if head < Hq:
            got, gs = q8[b, head, 64 * j:64 * j + 64], sq[b, head, j]
        elif head < Hq + Hkv:
            got, gs = k8[b, head - Hq, 64 * j:64 * j + 64], sk[b, head - Hq, j]
        else:
            got, gs = v8[b, head - Hq - Hkv, j].T, sv[b, head - Hq - Hkv, j]
        _check_close(got.cpu().numpy(), np.array([gs.item()]), codes.reshape(64, 128), s,
                     f"block b={b} head={head} j={j}")
    del x, wt
    torch.cuda.empty_cache()
