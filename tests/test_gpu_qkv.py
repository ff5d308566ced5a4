"""GPU parity of the fused QKV projection + FlashQ (turbo_qkv_project) and of
the prefill on pre-quantized Q (turbo_attn_prefill_q8), against the oracle.

Bar.  Every byte the kernel writes is checked bit for bit:
  * with small-integer inputs (x = i/8, w = j/64, |i|, |j| <= 8) every partial
    sum of X W^T is a multiple of 2^-9 below 2^15, so the fp32 MFMA sums and
    the oracle's sums are the same exact number whatever their order, and the
    codes, block scales and cache bytes equal the oracle's from x and w;
  * with N(0,1) inputs the fp32 sum may round to another fp16 value than the
    exact sum (several fp16 projections are correct), so the test hook
    turbo_qkv_project_trace also returns the kernel's fp16 projection Y, and
      - each Y is within the fp32 summation bound of the exact sum plus half
        an fp16 ulp: |Y - S| <= gamma_D sum|x||w| + ulp16(Y)/2 with
        gamma_D = D u / (1 - D u), u = 2^-23 (twice the unit roundoff, which
        covers accumulation with truncation as well as rounding);
      - the codes, block scales and cache bytes equal the oracle's FlashQ of
        that Y, bit for bit.
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
    _flashq_matches(q8, sq, k8, v8, sk, sv, ref, N, cache, bits, bt, gt)
    # the hook's projection is the exact sum rounded to fp16, and the hook
    # instance writes the same codes
    y = torch.empty(B, N, (Hq + 2 * Hkv) * 128, dtype=torch.float16, device=dev)
    outs = ta.turbo_qkv_project(torch.from_numpy(x).to(dev), torch.from_numpy(w).to(dev), Hq, Hkv,
                                y=y)
    torch.cuda.synchronize()
    ye, _ = orc.project_exact(x.astype(np.float32), w.astype(np.float32))
    assert np.array_equal(y.cpu().numpy(), ye.astype(np.float16)), "Y"
    for a_, b_ in zip(outs, (q8, sq, k8, v8, sk, sv)):
        assert np.array_equal(a_.cpu().numpy().view(np.uint8), b_.view(np.uint8))


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


def _flashq_matches(q8, sq, k8, v8, sk, sv, ref, N, cache=None, bits=None, bt=None, gt=None):
    """Every code, scale and cache byte of the kernel against the oracle's
    FlashQ `ref` (flashq_of_projection / qkv_project), bit for bit."""
    B, Hkv, nb = k8.shape[0], k8.shape[1], sk.shape[2]
    assert np.array_equal(q8[:, :, :N], ref["q8"]) and not q8[:, :, N:].any(), "Q8"
    assert _same_bits(sq, ref["sq"]), "s_Q"
    assert np.array_equal(k8[:, :, :N], ref["k8"]) and not k8[:, :, N:].any(), "K8"
    v8t = v8.transpose(0, 1, 2, 4, 3).reshape(B, Hkv, nb * 64, 128)
    assert np.array_equal(v8t[:, :, :N], ref["v8"]) and not v8t[:, :, N:].any(), "V8"
    assert _same_bits(sk, ref["sk"]) and _same_bits(sv, ref["sv"]), "s_K, s_V"
    ng = N // 64
    if cache is not None and ng:
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


def _within_fp32_sum_bound(y_gpu, y_exact, y_abs, D, what):
    """|Y - S| <= gamma_D sum|x||w| + half an fp16 ulp of Y (see the header)."""
    u = 2.0 ** -23
    gamma = D * u / (1 - D * u)
    y = np.asarray(y_gpu, np.float64)
    ulp = np.spacing(np.abs(y_gpu).astype(np.float16)).astype(np.float64)
    bound = gamma * y_abs + 0.5 * ulp
    err = np.abs(y - y_exact)
    assert np.all(err <= bound), f"{what}: |Y - S| / bound up to {np.max(err / bound):.3f}"
    # how close the kernel runs to the worst case (for the log)
    return float(np.max(err / bound))


@pytest.mark.parametrize("B,N,D,Hq,Hkv,bits,seed", [
    (1, 256 + 40, 1024, 4, 2, [4, 4], 5),
    (2, 64 * 5 + 3, 5120, 2, 1, [2], 6),
    (1, 1024, 256, 3, 3, [4, 2, 4], 7),
])
def test_qkv_project_gaussian_is_flashq_of_its_projection(orc, ta, dev, B, N, D, Hq, Hkv, bits,
                                                          seed):
    _log(f"qkv_project gaussian B={B} N={N} D={D} Hq={Hq} Hkv={Hkv} bits={bits}")
    x, w = _inputs(B, N, D, Hq, Hkv, seed=seed, exact=False)
    F = (Hq + 2 * Hkv) * 128
    mg = max(1, N // 64)
    bt, gt = _tables(B, mg, seed)
    cache = ta.PagedKVCache(bt.size, gt.size, bits, dev)
    btd, gtd = torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)
    y = torch.empty(B, N, F, dtype=torch.float16, device=dev)
    outs = ta.turbo_qkv_project(torch.from_numpy(x).to(dev), torch.from_numpy(w).to(dev), Hq, Hkv,
                                cache, btd, gtd, y=y)
    torch.cuda.synchronize()
    q8, sq, k8, v8, sk, sv = [t.cpu().numpy() for t in outs]
    yg = y.float().cpu().numpy()
    ye, ya = orc.project_exact(x.astype(np.float32), w.astype(np.float32))
    r = _within_fp32_sum_bound(yg, ye, ya, D, "projection")
    _log(f"  |Y - S| at most {r:.3f} of the bound; fp16 values differing from the exact "
         f"sum's rounding: {(yg != ye.astype(np.float16).astype(np.float32)).mean():.2e}")
    ref = orc.flashq_of_projection(yg, Hq, Hkv, bits)
    _flashq_matches(q8, sq, k8, v8, sk, sv, ref, N, cache, bits, bt, gt)


def test_qkv_project_full_size_sampled(orc, ta, dev):
    """The benchmark's Phi-3-medium projection (4 x 4096 tokens, hidden 5120,
    40 + 2 x 10 heads) run in full through the test hook; for 12 sampled
    (sequence, head, 64-token block) blocks the fp16 projection is within the
    fp32 summation bound of the oracle's exact sum, and the codes and scale
    are the oracle's FlashQ of the kernel's projection, bit for bit; for the
    sampled key and value heads the whole sequence's cache groups too."""
    from paper_2412_08585_amd import workloads as W
    w_ = W.WORKLOADS["phi3m-qkv-4k"]
    x, wt = W.projection_inputs(w_, device=dev)
    Hq, Hkv, D = w_.Hq, w_.Hkv, w_.hidden
    F = (Hq + 2 * Hkv) * 128
    bits = W.head_bits(w_)
    bt, gt = W.tables(w_)
    cache = ta.PagedKVCache(bt.size, gt.size, bits, dev)
    btd, gtd = torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)
    y = torch.empty(w_.B, w_.N, F, dtype=torch.float16, device=dev)
    q8, sq, k8, v8, sk, sv = ta.turbo_qkv_project(x, wt, Hq, Hkv, cache, btd, gtd, y=y)
    torch.cuda.synchronize()
    pages = cache.pages.cpu().numpy()
    gmeta = cache.group_meta.cpu().numpy()
    gscale = cache.group_scale.cpu().numpy()
    rng = np.random.default_rng(0)
    worst = 0.0
    for i in range(12):
        b = int(rng.integers(w_.B))
        head = [int(rng.integers(Hq)), Hq + int(rng.integers(Hkv)),
                Hq + Hkv + int(rng.integers(Hkv))][i % 3]
        j = int(rng.integers(w_.N // 64))
        rows = x[b, 64 * j:64 * j + 64].float().cpu().numpy()
        feats = wt[head * 128:(head + 1) * 128].float().cpu().numpy()
        ye, ya = orc.project_exact(rows, feats)
        yb = y[b, 64 * j:64 * j + 64, head * 128:(head + 1) * 128].float().cpu().numpy()
        worst = max(worst, _within_fp32_sum_bound(yb, ye, ya, D, f"block {b},{head},{j}"))
        codes, s = orc.block_quant(yb.reshape(1, -1))
        if head < Hq:
            got, gs = q8[b, head, 64 * j:64 * j + 64], sq[b, head, j]
        elif head < Hq + Hkv:
            got, gs = k8[b, head - Hq, 64 * j:64 * j + 64], sk[b, head - Hq, j]
        else:
            got, gs = v8[b, head - Hq - Hkv, j].T, sv[b, head - Hq - Hkv, j]
        assert np.array_equal(got.cpu().numpy(), codes.reshape(64, 128)), (b, head, j)
        assert _same_bits(np.array([gs.item()]), s), (b, head, j)
        if head >= Hq:  # the whole sequence of this KV head: codes and cache groups
            h = (head - Hq) % Hkv
            ys = y[b, :, (Hq + h) * 128:(Hq + h + 1) * 128].float().cpu().numpy()
            yv = y[b, :, (Hq + Hkv + h) * 128:(Hq + Hkv + h + 1) * 128].float().cpu().numpy()
            ref = orc.quantize_kv(ys[None, None], yv[None, None], [int(bits[h])])
            u = cache_layout.read_unit(pages, gmeta, gscale, bits, bt, gt, b, h, w_.N // 64)
            for key in ("kc", "vc", "ks", "kz", "vs", "vz"):
                assert np.array_equal(u[key], ref[key][0, 0]), (b, h, key)
            assert _same_bits(u["sk"], ref["sk"][0, 0]) and _same_bits(u["sv"], ref["sv"][0, 0])
    _log(f"  full size: |Y - S| at most {worst:.3f} of the bound")
    del x, wt, y, cache
    torch.cuda.empty_cache()
