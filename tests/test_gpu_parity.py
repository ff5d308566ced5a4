"""GPU parity: the gfx950 kernels (called through the C ABI) against the CPU
oracle on the same seeded inputs.

Bar (fixed by the method's integer steps and the fp16 output):
  * bit-exact: int8 K/V codes, block scales (bits), int4/int2 codes, integer
    step-2 scales and zero points, group scales;
  * fp16 O within 1e-3 of the row's largest |O| (the GPU's fp32 l and O sums
    round in another order than the oracle's double ones; every integer of
    the path, including Q(P~), is decided by the same binary32 operations);
  * L = m + ln l within 1e-4 absolute.
Full-size workloads run on the GPU in full, in the launch configuration the
benchmark times, and are compared on sampled (sequence, KV head) units.
"""
import os
import sys

import numpy as np
import pytest
import torch

from tests import cache_layout
from tests.decode_split import oracle_decode, split_of

pytestmark = pytest.mark.gpu

O_TOL = 1e-3
LSE_TOL = 1e-4


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


def _cmp_o(got: torch.Tensor, want: np.ndarray, what: str):
    g = got.float().cpu().numpy()
    rowmax = np.maximum(np.abs(want).max(axis=-1, keepdims=True), 1e-30)
    err = np.abs(g - want) / rowmax
    worst = float(np.nanmax(err))
    assert np.all(np.isfinite(g)), what
    assert worst < O_TOL, f"{what}: max rel-to-row-max error {worst:.3e}"
    return worst


def _cmp_lse(got: torch.Tensor, want: np.ndarray, what: str):
    g = got.cpu().numpy().astype(np.float64)
    fin = np.isfinite(want)
    assert np.array_equal(np.isfinite(g), fin), what
    if fin.any():
        worst = float(np.max(np.abs(g[fin] - want[fin])))
        assert worst < LSE_TOL, f"{what}: lse error {worst:.3e}"


def _tables(B, mg, seed):
    rng = np.random.default_rng(seed)
    bt = rng.permutation(B * 4 * mg).astype(np.int32).reshape(B, 4 * mg)
    gt = rng.permutation(B * mg).astype(np.int32).reshape(B, mg)
    return bt, gt


def _quantize(ta, dev, k, v, bits, seed=0):
    B, H, N, _ = k.shape
    mg = max(1, N // 64)
    bt, gt = _tables(B, mg, seed)
    cache = ta.PagedKVCache(bt.size, gt.size, bits, dev)
    btd, gtd = torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)
    outs = ta.turbo_quantize_kv(k.to(dev), v.to(dev), cache, btd, gtd)
    torch.cuda.synchronize()
    return outs, cache, bt, gt, btd, gtd


def _rand(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(*shape, generator=g) * scale).half()


QUANT_CASES = [
    # B, Hkv, N, bits
    (1, 4, 512, [4, 4, 4, 4]),
    (2, 3, 64 * 5 + 17, [4, 2, 4]),
    (1, 2, 64, [2, 2]),
    (1, 1, 17, [4]),
    (2, 2, 64 * 3, [2, 4]),
]


@pytest.mark.parametrize("B,H,N,bits", QUANT_CASES)
def test_quantize_kv_bit_exact(orc, ta, dev, B, H, N, bits):
    _log(f"quantize_kv B={B} H={H} N={N} bits={bits}")
    k = _rand((B, H, N, 128), 100 + N)
    v = _rand((B, H, N, 128), 200 + N)
    k[..., 7] *= 10
    if N >= 128:
        k[:, 0, 64:128] = 0  # an all-zero block: s = 0, codes 0
    (k8, v8, sk, sv), cache, bt, gt, _, _ = _quantize(ta, dev, k, v, bits)
    ref = orc.quantize_kv(k, v, bits)
    nb = (N + 63) // 64
    k8 = k8.cpu().numpy()
    v8 = v8.cpu().numpy().transpose(0, 1, 2, 4, 3).reshape(B, H, nb * 64, 128)
    assert np.array_equal(k8[:, :, :N], ref["k8"])
    assert np.array_equal(v8[:, :, :N], ref["v8"])
    assert not k8[:, :, N:].any() and not v8[:, :, N:].any()
    assert np.array_equal(sk.cpu().numpy().view(np.int32), ref["sk"].view(np.int32))
    assert np.array_equal(sv.cpu().numpy().view(np.int32), ref["sv"].view(np.int32))
    ng = N // 64
    pages = cache.pages.cpu().numpy()
    gmeta = cache.group_meta.cpu().numpy()
    gscale = cache.group_scale.cpu().numpy()
    for b in range(B):
        for h in range(H):
            if ng == 0:
                continue
            u = cache_layout.read_unit(pages, gmeta, gscale, bits, bt, gt, b, h, ng)
            for key in ("kc", "vc", "ks", "kz", "vs", "vz"):
                assert np.array_equal(u[key], ref[key][b, h]), (b, h, key)
            assert np.array_equal(u["sk"].view(np.int32), ref["sk"][b, h, :ng].view(np.int32))
            assert np.array_equal(u["sv"].view(np.int32), ref["sv"][b, h, :ng].view(np.int32))


PREFILL_CASES = [
    # B, Hq, Hkv, N, causal
    (1, 4, 4, 512, True),
    (2, 8, 2, 64 * 3 + 40, True),
    (1, 2, 1, 130, False),
    (1, 2, 2, 1, True),
    (1, 2, 2, 64, True),
    (1, 16, 1, 200, True),
    (1, 3, 3, 64 * 2 + 63, False),
]


@pytest.mark.parametrize("B,Hq,Hkv,N,causal", PREFILL_CASES)
def test_prefill_parity(orc, ta, dev, B, Hq, Hkv, N, causal):
    _log(f"prefill B={B} Hq={Hq} Hkv={Hkv} N={N} causal={causal}")
    q = _rand((B, Hq, N, 128), 300 + N)
    k = _rand((B, Hkv, N, 128), 400 + N)
    v = _rand((B, Hkv, N, 128), 500 + N)
    k[..., 3] *= 10
    (k8, v8, sk, sv) = ta.turbo_quantize_kv(k.to(dev), v.to(dev))
    o, lse = ta.turbo_attn_prefill(q.to(dev), k8, v8, sk, sv, 1 / np.sqrt(128), causal,
                                   return_lse=True)
    torch.cuda.synchronize()
    ro, rl = orc.attn_prefill(q, k, v, 1 / np.sqrt(128), causal)
    err = _cmp_o(o, ro, "prefill O")
    _cmp_lse(lse, rl, "prefill lse")
    ex, _ = orc.attn_exact(q, k, v, float(np.float32(1 / np.sqrt(128))), causal)
    g = o.float().cpu().numpy()
    _log(f"  vs oracle {err:.2e}; rel-L2 vs exact fp64: gpu "
         f"{np.linalg.norm(g - ex) / np.linalg.norm(ex):.3e} oracle "
         f"{np.linalg.norm(ro - ex) / np.linalg.norm(ex):.3e}")


BLOCK_CASES = [
    # B, Hq, Hkv, N, causal, (B_r, B_c)
    (2, 8, 2, 64 * 3 + 40, True, (32, 64)),
    (2, 8, 2, 64 * 3 + 40, True, (128, 64)),
    (1, 2, 1, 130, False, (32, 64)),
    (1, 2, 1, 130, False, (128, 64)),
    (1, 4, 4, 512, True, (128, 64)),
    (1, 16, 1, 200, True, (128, 64)),
    (1, 3, 3, 64 * 2 + 63, False, (128, 64)),
    (1, 2, 2, 1, True, (32, 64)),
    (1, 2, 2, 97, True, (128, 64)),
    # B_c = 32 and 128 (Table 3 pairs, plus (128, 32) and (32, 128))
    (2, 8, 2, 64 * 3 + 40, True, (32, 32)),
    (2, 8, 2, 64 * 3 + 40, True, (64, 32)),
    (2, 8, 2, 64 * 3 + 40, True, (64, 128)),
    (2, 8, 2, 64 * 3 + 40, True, (128, 128)),
    (1, 4, 2, 64 * 5, True, (128, 32)),
    (1, 4, 2, 64 * 5, True, (32, 128)),
    (1, 4, 2, 64 * 5, True, (64, 128)),
    (1, 2, 1, 130, False, (64, 32)),
    (1, 2, 1, 130, False, (64, 128)),
    (1, 3, 3, 64 * 2 + 63, False, (128, 128)),
    (1, 16, 1, 200, True, (64, 32)),
    (1, 2, 2, 17, True, (64, 128)),
    (1, 2, 2, 33, True, (32, 32)),
]


@pytest.mark.parametrize("B,Hq,Hkv,N,causal,blocks", BLOCK_CASES)
def test_prefill_block_sizes(orc, ta, dev, B, Hq, Hkv, N, causal, blocks):
    """Table 3's block sizes: B_r = 32 / 64 / 128 (one, two or four waves
    sharing the Q scale and the P scale of the block) and B_c = 32 / 64 / 128
    (the K/V step-1 blocks, the keys of each online step)."""
    br, bc = blocks
    _log(f"prefill B_r={br} B_c={bc} B={B} Hq={Hq} Hkv={Hkv} N={N} causal={causal}")
    q = _rand((B, Hq, N, 128), 310 + N)
    k = _rand((B, Hkv, N, 128), 410 + N)
    v = _rand((B, Hkv, N, 128), 510 + N)
    k[..., 3] *= 10
    (k8, v8, sk, sv) = ta.turbo_quantize_kv(k.to(dev), v.to(dev), block_cols=bc)
    o, lse = ta.turbo_attn_prefill(q.to(dev), k8, v8, sk, sv, 1 / np.sqrt(128), causal,
                                   return_lse=True, block_rows=br, block_cols=bc)
    torch.cuda.synchronize()
    ro, rl = orc.attn_prefill(q, k, v, 1 / np.sqrt(128), causal, block_rows=br, block_cols=bc)
    err = _cmp_o(o, ro, f"prefill ({br},{bc}) O")
    _cmp_lse(lse, rl, f"prefill ({br},{bc}) lse")
    _log(f"  vs oracle {err:.2e}")


@pytest.mark.parametrize("bc", [32, 128])
@pytest.mark.parametrize("B,H,N", [(1, 2, 64 * 3 + 40), (2, 3, 64 * 5), (1, 1, 17), (1, 2, 96),
                                   (1, 1, 1), (2, 2, 64 * 8)])
def test_quantize_kv_blocks_bit_exact(orc, ta, dev, B, H, N, bc):
    _log(f"quantize_kv B_c={bc} B={B} H={H} N={N}")
    k = _rand((B, H, N, 128), 120 + N)
    v = _rand((B, H, N, 128), 220 + N)
    k[..., 7] *= 10
    if N >= 64:
        v[:, 0, 32:40] *= 4   # scales that differ between the 32-token halves
    nb = (N + 63) // 64
    k8, v8, sk, sv = ta.turbo_quantize_kv(k.to(dev), v.to(dev), block_cols=bc)
    torch.cuda.synchronize()
    ref = orc.quantize_kv_blocks(k, v, bc)
    k8 = k8.cpu().numpy()
    v8 = v8.cpu().numpy().transpose(0, 1, 2, 4, 3).reshape(B, H, nb * 64, 128)
    assert np.array_equal(k8[:, :, :N], ref["k8"])
    assert np.array_equal(v8[:, :, :N], ref["v8"])
    assert not k8[:, :, N:].any() and not v8[:, :, N:].any()
    assert np.array_equal(sk.cpu().numpy().view(np.int32), ref["sk"].view(np.int32))
    assert np.array_equal(sv.cpu().numpy().view(np.int32), ref["sv"].view(np.int32))


def test_prefill_zero_query_block(orc, ta, dev):
    """An all-zero query block has s_Q = 0: every score is 0 (closed form)."""
    N = 64 * 3
    q = _rand((1, 2, N, 128), 1)
    q[:, :, 64:128] = 0
    k, v = _rand((1, 2, N, 128), 2), _rand((1, 2, N, 128), 3)
    k8, v8, sk, sv = ta.turbo_quantize_kv(k.to(dev), v.to(dev))
    o, lse = ta.turbo_attn_prefill(q.to(dev), k8, v8, sk, sv, 1 / np.sqrt(128), True,
                                   return_lse=True)
    ro, rl = orc.attn_prefill(q, k, v, 1 / np.sqrt(128), True)
    _cmp_o(o, ro, "zero block O")
    _cmp_lse(lse, rl, "zero block lse")


DECODE_CASES = [
    # B, Hq, Hkv, Nc, bits, seq_lens, split
    (3, 8, 2, 64 * 6, [4, 2], [384, 200, 0], 2),
    (3, 8, 2, 64 * 6, [4, 2], [384, 200, 63], 0),
    (2, 4, 4, 64 * 4, [2, 4, 4, 2], [256, 256], 1),
    (1, 16, 1, 64 * 8, [4], [512], 3),
    (2, 16, 2, 64 * 6, [2, 4], [384, 250], 2),   # 8 query heads per KV head
    (2, 2, 1, 64 * 5, [2], [320, 128], 100),
    # default chunking: 4 chunks of 35 groups and 2 chunks of 32 (merged in
    # the decode launch); many chunks of one group
    (2, 8, 2, 64 * 140, [4, 2], [64 * 140, 64 * 50 + 10], 0),
    (1, 4, 1, 64 * 12, [4], [64 * 12], 1),
]


@pytest.mark.parametrize("B,Hq,Hkv,Nc,bits,sl,split", DECODE_CASES)
def test_decode_parity(orc, ta, dev, B, Hq, Hkv, Nc, bits, sl, split):
    _log(f"decode B={B} Hq={Hq} Hkv={Hkv} Nc={Nc} bits={bits} seq={sl} split={split}")
    k = _rand((B, Hkv, Nc, 128), 600 + Nc)
    v = _rand((B, Hkv, Nc, 128), 700 + Nc)
    k[..., 11] *= 10
    q = _rand((B, Hq, 128), 800 + Nc)
    _, cache, bt, gt, btd, gtd = _quantize(ta, dev, k, v, bits, seed=Nc)
    sld = torch.tensor(sl, dtype=torch.int32, device=dev)
    o, lse = ta.turbo_attn_decode(q.to(dev), cache, sld, btd, gtd, 1 / np.sqrt(128), split,
                                  return_lse=True)
    torch.cuda.synchronize()
    ref = orc.quantize_kv(k, v, bits)
    ro, rl = oracle_decode(orc, q, ref, sl, 1 / np.sqrt(128), split, Nc // 64)
    _cmp_o(o, ro, "decode O")
    _cmp_lse(lse, rl, "decode lse")


def test_decode_result_does_not_depend_on_the_batch(orc, ta, dev):
    """With kv_split_groups = 0 the chunking follows each sequence's own group
    count, so a sequence decoded on its own (with tables cut to its groups,
    hence another grid) gives the same O and L bit for bit as inside a batch
    of 64 sequences of other lengths; and both equal the oracle with that
    sequence's chunk length."""
    B, Hq, Hkv, mg = 64, 8, 2, 40
    rng = np.random.default_rng(77)
    sl = [int(x) for x in rng.integers(64 * 3, 64 * mg + 1, size=B)]
    sl[5], sl[6], sl[7] = 64 * mg, 64 * 33, 64 * 32 + 63   # 2, 2 and 1 chunks
    _log(f"decode batch independence B={B} Hq={Hq} Hkv={Hkv} seq={sl[:8]}...")
    k = _rand((B, Hkv, 64 * mg, 128), 1901)
    v = _rand((B, Hkv, 64 * mg, 128), 1902)
    k[..., 5] *= 10
    q = _rand((B, Hq, 128), 1903)
    bits = [4, 2]
    _, cache, bt, gt, btd, gtd = _quantize(ta, dev, k, v, bits, seed=19)
    sld = torch.tensor(sl, dtype=torch.int32, device=dev)
    o, lse = ta.turbo_attn_decode(q.to(dev), cache, sld, btd, gtd, 1 / np.sqrt(128), 0,
                                  return_lse=True)
    torch.cuda.synchronize()
    for b in (5, 6, 7, 11, 40):
        ng = sl[b] // 64
        o1, l1 = ta.turbo_attn_decode(q[b:b + 1].to(dev), cache, sld[b:b + 1],
                                      btd[b:b + 1, :4 * ng].contiguous(),
                                      gtd[b:b + 1, :ng].contiguous(), 1 / np.sqrt(128), 0,
                                      return_lse=True)
        torch.cuda.synchronize()
        assert torch.equal(o1.view(torch.int16), o[b:b + 1].view(torch.int16)), b
        assert torch.equal(l1.view(torch.int32), lse[b:b + 1].view(torch.int32)), b
    ref = orc.quantize_kv(k[[5, 6, 7]], v[[5, 6, 7]], bits)
    ro, rl = oracle_decode(orc, q[[5, 6, 7]], ref, [sl[5], sl[6], sl[7]], 1 / np.sqrt(128), 0)
    _cmp_o(o[[5, 6, 7]], ro, "decode O (default chunking)")
    _cmp_lse(lse[[5, 6, 7]], rl, "decode lse (default chunking)")


def test_decode_rows_with_empty_groups(orc, ta, dev):
    """Rows of one wave whose later groups all fall more than 6 below their
    running maximum (P~ = 0 for a whole group, P scale 0) next to rows for
    which they do not: the quantized P of the former must add nothing."""
    B, Hq, Hkv, Nc = 1, 4, 1, 64 * 4
    k = _rand((B, Hkv, Nc, 128), 901, 0.1)
    k[:, :, :64] = 3.0          # group 0 aligned with +1 queries
    v = _rand((B, Hkv, Nc, 128), 902)
    q = torch.ones(B, Hq, 128, dtype=torch.float16)
    q[:, 1] = -1.0              # row 1: group 0 far below the others
    q[:, 2] = _rand((Hq, 128), 903)[2]
    _, cache, bt, gt, btd, gtd = _quantize(ta, dev, k, v, [4], seed=5)
    sld = torch.tensor([Nc], dtype=torch.int32, device=dev)
    ref = orc.quantize_kv(k, v, [4])
    for split in (1, 2):
        o, lse = ta.turbo_attn_decode(q.to(dev), cache, sld, btd, gtd, 1 / np.sqrt(128), split,
                                      return_lse=True)
        torch.cuda.synchronize()
        ro, rl = orc.attn_decode(q, ref, [Nc], 1 / np.sqrt(128), split=split)
        _cmp_o(o, ro, f"decode empty groups split={split}")
        _cmp_lse(lse, rl, "decode empty groups lse")


def test_prefill_tiles_with_empty_p(orc, ta, dev):
    """Key blocks whose every score lies more than 6 below the running
    maximum: the tile's P scale is 0 and its PV is skipped."""
    N = 64 * 4
    q = torch.ones(1, 2, N, 128, dtype=torch.float16)
    q[:, 1] = _rand((N, 128), 911)
    k = _rand((1, 1, N, 128), 912, 0.1)
    k[:, :, :64] = 3.0
    v = _rand((1, 1, N, 128), 913)
    k8, v8, sk, sv = ta.turbo_quantize_kv(k.to(dev), v.to(dev))
    o, lse = ta.turbo_attn_prefill(q.to(dev), k8, v8, sk, sv, 1 / np.sqrt(128), True,
                                   return_lse=True)
    ro, rl = orc.attn_prefill(q, k, v, 1 / np.sqrt(128), True)
    _cmp_o(o, ro, "prefill empty tiles O")
    _cmp_lse(lse, rl, "prefill empty tiles lse")


def _rowmax_path(q, k, sm, causal):
    """fp64 running maxima of the scaled scores per 64-key tile (no
    quantization): the per-tile drops m_old - m_new and the product of
    e^(m_old - m_new) over the tiles, per row."""
    s = np.einsum("bhnd,bktd->bhnt", q.double().numpy(), k.double().numpy()) * sm
    N = s.shape[-1]
    if causal:
        s = np.where(np.tril(np.ones((N, N), bool)), s, -np.inf)
    m = np.full(s.shape[:-1], -np.inf)
    logbeta = np.zeros(s.shape[:-1])
    jump = np.zeros(s.shape[:-1])
    for j in range(0, N, 64):
        mn = np.maximum(m, s[..., j:j + 64].max(-1))
        d = np.where(np.isfinite(m), mn - m, 0.0)
        jump = np.maximum(jump, d)
        logbeta -= d
        m = mn
    return jump, logbeta


@pytest.mark.parametrize("case", ["jump", "decay"])
@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("br", [64, 128])
def test_prefill_rescale_paths(orc, ta, dev, case, causal, br):
    """The accumulator rescale of Algorithm 1 at its extremes.  "jump": one
    key block whose scores exceed everything before by more than 6, so the
    factor SAS(m_old - m_new) is 0 and the kernel renormalizes its kept
    accumulator (O = beta * Ost with beta = 0).  "decay": scores that rise
    steadily along the keys, so the per-tile factors multiply beta below
    2^-64 and the renormalization runs mid-sequence."""
    sm = 1 / np.sqrt(128)
    g = torch.Generator().manual_seed(77)
    u = torch.randn(128, generator=g, dtype=torch.float64)
    u /= u.norm()
    if case == "jump":
        N = 64 * 5
        q = (torch.randn(1, 2, N, 128, generator=g, dtype=torch.float64) + 3.0 * u).half()
        k = (torch.randn(1, 1, N, 128, generator=g, dtype=torch.float64) * 0.2).half()
        k[0, 0, 200] = (40.0 * u).half()
    else:
        N = 64 * 64
        q = (torch.randn(1, 2, N, 128, generator=g, dtype=torch.float64) + 3.0 * u).half()
        t = torch.arange(N, dtype=torch.float64)[:, None] / 64.0
        k = (torch.randn(1, 1, N, 128, generator=g, dtype=torch.float64) * 0.1
             + 5.0 * t * u).half()
    v = _rand((1, 1, N, 128), 931)
    jump, logbeta = _rowmax_path(q, k, sm, causal)
    if case == "jump":
        assert (jump > 8.0).sum() > 100, "the planted key must raise many rows' maximum by > 6"
    else:
        assert (logbeta < -80.0).sum() > 100, "beta must underflow 2^-64 in many rows"
    _log(f"prefill rescale {case} causal={causal} B_r={br}: max jump {jump.max():.1f}, "
         f"min log beta {logbeta.min():.1f}")
    k8, v8, sk, sv = ta.turbo_quantize_kv(k.to(dev), v.to(dev))
    o, lse = ta.turbo_attn_prefill(q.to(dev), k8, v8, sk, sv, sm, causal, return_lse=True,
                                   block_rows=br)
    ro, rl = orc.attn_prefill(q, k, v, sm, causal, block_rows=br)
    _cmp_o(o, ro, f"prefill rescale {case} O")
    _cmp_lse(lse, rl, f"prefill rescale {case} lse")


def _bits_of(t):
    return t.detach().contiguous().view(torch.uint8).cpu()


def test_determinism(ta, dev):
    """Two runs of the whole path on the same inputs give the same bytes:
    quantization and cache, prefill (and its Table 3 variant), decode (split
    and unsplit, with and without the int8 buffer, also the allocation-free
    entry point), buffer appends with a flush, the fused projection, the
    head priority and the SAS softmax."""
    N, B, Hq, Hkv = 64 * 4 + 9, 2, 4, 2
    q, k, v = _rand((B, Hq, N, 128), 1), _rand((B, Hkv, N, 128), 2), _rand((B, Hkv, N, 128), 3)
    qd = _rand((B, Hq, 128), 4).to(dev)
    kn, vn = _rand((B, Hkv, 128), 5).to(dev), _rand((B, Hkv, 128), 6).to(dev)
    x = _rand((B, N, 128), 7).to(dev)
    w = (_rand(((Hq + 2 * Hkv) * 128, 128), 8).float() / 11).half().to(dev)
    sx = (torch.randn(33, 5000, generator=torch.Generator().manual_seed(9)) * 2).to(dev)
    mg = N // 64 + 1
    bt, gt = _tables(B, mg, 10)
    btd, gtd = torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)
    runs = []
    for _ in range(2):
        out = []
        cache = ta.PagedKVCache(bt.size, gt.size, [4, 2], dev)
        k8, v8, sk, sv = ta.turbo_quantize_kv(k.to(dev), v.to(dev), cache, btd, gtd)
        out += [k8, v8, sk, sv, cache.pages, cache.group_meta, cache.group_scale]
        out.append(ta.turbo_attn_prefill(q.to(dev), k8, v8, sk, sv))
        k8b, v8b, skb, svb = ta.turbo_quantize_kv(k.to(dev), v.to(dev), block_cols=32)
        out.append(ta.turbo_attn_prefill(q.to(dev), k8b, v8b, skb, svb, block_rows=128,
                                         block_cols=32))
        tail = ta.KVTail(B, Hkv, dev)
        ta.turbo_tail_init(k.to(dev), v.to(dev), sk, sv, tail)
        sl = torch.tensor([N, 64 * 3 + 1], dtype=torch.int32, device=dev)
        for split in (0, 1):
            out += list(ta.turbo_attn_decode(qd, cache, sl, btd, gtd, None, split,
                                             return_lse=True))
            out += list(ta.turbo_attn_decode(qd, cache, sl, btd, gtd, None, split,
                                             return_lse=True, tail=tail))
            out += list(ta.turbo_attn_decode_noalloc(qd, cache, sl, btd, gtd, None, split,
                                                     return_lse=True, tail=tail))
        for _step in range(60):  # crosses a flush of both sequences
            ta.turbo_append_kv(kn, vn, sl, cache, tail, btd, gtd)
            sl += 1
        out += [cache.pages, cache.group_meta, cache.group_scale, tail.k, tail.v, tail.scale]
        out += list(ta.turbo_attn_decode(qd, cache, sl, btd, gtd, None, 0, return_lse=True,
                                         tail=tail))
        out += list(ta.turbo_qkv_project(x, w, Hq, Hkv))
        out.append(ta.turbo_head_priority(k.to(dev)))
        out.append(ta.turbo_sas_softmax(sx))
        torch.cuda.synchronize()
        runs.append([_bits_of(t) for t in out])
    for i, (a, b) in enumerate(zip(*runs)):
        assert torch.equal(a, b), f"output {i} differs between runs"


# ---- full-size workloads (launch configuration of the benchmark) -----------

def _sample_units(w, n, seed=0):
    rng = np.random.default_rng(seed)
    return sorted({(int(rng.integers(w.B)), int(rng.integers(w.Hkv))) for _ in range(n)})


@pytest.mark.parametrize("name,qblocks", [("phi3m-prefill-4k", None),
                                          ("llama3-8b-prefill-16k", (0, 2)),
                                          ("llama3-8b-prefill-16k", (255, 256))])
def test_full_size_prefill(orc, ta, dev, name, qblocks):
    from paper_2412_08585_amd import workloads as W
    w = W.WORKLOADS[name]
    _log(f"full-size prefill {name} qblocks={qblocks}")
    q, k, v = W.prefill_inputs(w, device=dev)
    k8, v8, sk, sv = ta.turbo_quantize_kv(k, v)
    o, lse = ta.turbo_attn_prefill(q, k8, v8, sk, sv, w.sm_scale, True, return_lse=True)
    torch.cuda.synchronize()
    for (b, h) in _sample_units(w, 2 if qblocks is None else 1, seed=len(name)):
        qs = q[b:b + 1, h * w.G:(h + 1) * w.G].cpu()
        ro, rl = orc.attn_prefill(qs, k[b:b + 1, h:h + 1].cpu(), v[b:b + 1, h:h + 1].cpu(),
                                  w.sm_scale, True, qblocks=qblocks)
        rows = slice(None) if qblocks is None else slice(64 * qblocks[0], 64 * qblocks[1])
        _cmp_o(o[b:b + 1, h * w.G:(h + 1) * w.G, rows], ro[:, :, rows], f"{name} O unit {b},{h}")
        _cmp_lse(lse[b:b + 1, h * w.G:(h + 1) * w.G, rows], rl[:, :, rows], f"{name} lse")
        _log(f"  unit ({b},{h}) ok")
    del q, k, v, k8, v8, o
    torch.cuda.empty_cache()


@pytest.mark.parametrize("br,bc,qblocks", [(32, 64, (126, 128)), (128, 64, (30, 32)),
                                           (128, 64, (0, 1)), (64, 32, (62, 64)),
                                           (64, 128, (62, 64)), (128, 128, (31, 32))])
def test_full_size_prefill_block_sizes(orc, ta, dev, br, bc, qblocks):
    """The Phi-3-medium prefill (4 x 4096, 40 / 10 heads) at other block sizes
    (B_r, B_c), run in full; one (sequence, KV head) unit's last or first
    query blocks recomputed by the oracle."""
    from paper_2412_08585_amd import workloads as W
    w = W.WORKLOADS["phi3m-prefill-4k"]
    _log(f"full-size prefill B_r={br} B_c={bc} qblocks={qblocks}")
    q, k, v = W.prefill_inputs(w, device=dev)
    k8, v8, sk, sv = ta.turbo_quantize_kv(k, v, block_cols=bc)
    o, lse = ta.turbo_attn_prefill(q, k8, v8, sk, sv, w.sm_scale, True, return_lse=True,
                                   block_rows=br, block_cols=bc)
    torch.cuda.synchronize()
    (b, h), = _sample_units(w, 1, seed=br + bc + qblocks[0])
    qs = q[b:b + 1, h * w.G:(h + 1) * w.G].cpu()
    ro, rl = orc.attn_prefill(qs, k[b:b + 1, h:h + 1].cpu(), v[b:b + 1, h:h + 1].cpu(),
                              w.sm_scale, True, qblocks=qblocks, block_rows=br, block_cols=bc)
    rows = slice(br * qblocks[0], br * qblocks[1])
    _cmp_o(o[b:b + 1, h * w.G:(h + 1) * w.G, rows], ro[:, :, rows], f"({br},{bc}) O unit {b},{h}")
    _cmp_lse(lse[b:b + 1, h * w.G:(h + 1) * w.G, rows], rl[:, :, rows], f"({br},{bc}) lse")
    del q, k, v, k8, v8, o
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["phi3m-decode-8k", "long-decode-32k"])
def test_full_size_decode(orc, ta, dev, name):
    from paper_2412_08585_amd import workloads as W
    w = W.WORKLOADS[name]
    _log(f"full-size decode {name}")
    bits = W.head_bits(w)
    bt, gt = W.tables(w)
    cache = ta.PagedKVCache(bt.size, gt.size, bits, dev)
    btd, gtd = torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)
    chunk = 16
    units = {}
    samples = _sample_units(w, 3, seed=7)
    for b0 in range(0, w.B, chunk):
        nbat = min(chunk, w.B - b0)
        k = torch.empty(nbat, w.Hkv, w.N, 128, dtype=torch.float16, device=dev)
        v = torch.empty_like(k)
        for bb in range(nbat):
            for h in range(w.Hkv):
                k[bb, h], v[bb, h] = W.unit_kv(w, b0 + bb, h, device=dev)
                if (b0 + bb, h) in samples:
                    units[b0 + bb, h] = (k[bb, h].cpu(), v[bb, h].cpu())
        ta.turbo_quantize_kv(k, v, cache, btd[b0:b0 + nbat], gtd[b0:b0 + nbat])
        del k, v
    torch.cuda.synchronize()
    _log("  cache built")
    q = W.decode_query(w, device=dev)
    sl = torch.full((w.B,), w.N, dtype=torch.int32, device=dev)
    o, lse = ta.turbo_attn_decode(q, cache, sl, btd, gtd, w.sm_scale, 0, return_lse=True)
    torch.cuda.synchronize()
    split = split_of(w.N, 0, w.max_groups)
    pages = cache.pages.cpu().numpy()
    gmeta = cache.group_meta.cpu().numpy()
    gscale = cache.group_scale.cpu().numpy()
    for (b, h), (ku, vu) in units.items():
        ref = orc.quantize_kv(ku[None, None], vu[None, None], [int(bits[h])])
        u = cache_layout.read_unit(pages, gmeta, gscale, bits, bt, gt, b, h, w.max_groups)
        for key in ("kc", "vc", "ks", "kz", "vs", "vz"):
            assert np.array_equal(u[key], ref[key][0, 0]), (b, h, key)
        assert np.array_equal(u["sk"].view(np.int32), ref["sk"][0, 0].view(np.int32))
        qs = q[b:b + 1, h * w.G:(h + 1) * w.G].cpu()
        ro, rl = orc.attn_decode(qs, ref, [w.N], w.sm_scale, split=split)
        _cmp_o(o[b:b + 1, h * w.G:(h + 1) * w.G], ro, f"{name} O unit {b},{h}")
        _cmp_lse(lse[b:b + 1, h * w.G:(h + 1) * w.G], rl, f"{name} lse unit {b},{h}")
        _log(f"  unit ({b},{h}) ok")
    del cache
    torch.cuda.empty_cache()


# ---- head-wise mixed precision (Sec. 3.2) ------------------------------------

PRIORITY_CASES = [
    # B, Hkv, N, outlier heads
    (2, 8, 200, [1, 4, 6, 7]),
    (1, 3, 1, [2]),
    (3, 10, 64 * 5 + 13, [0, 3, 5, 8, 9]),
    (2, 2, 257, [1]),         # one row past a 256-token slab
    (1, 4, 256 * 3, [0, 2]),  # whole slabs only
    (1, 3, 700, [2]),         # a slab ending inside a batch of rows
]


@pytest.mark.parametrize("B,Hkv,N,outliers", PRIORITY_CASES)
def test_head_priority_parity(orc, ta, dev, B, Hkv, N, outliers):
    _log(f"head priority B={B} Hkv={Hkv} N={N}")
    k = _rand((B, Hkv, N, 128), 1900 + N)
    rng = np.random.default_rng(N)
    for h in outliers:
        k[:, h, :, torch.from_numpy(rng.choice(128, 4, replace=False))] *= 10
    p = ta.turbo_head_priority(k.to(dev)).cpu().numpy()
    ref = orc.head_priority(k)
    np.testing.assert_allclose(p, ref, rtol=1e-5, atol=0)
    n2 = Hkv - len(outliers)
    bits = ta.turbo_int2_heads(p, n2)
    assert np.array_equal(bits, orc.int2_heads(ref, n2))
    if N > 1:
        assert [int(b) for b in bits] == [4 if h in outliers else 2 for h in range(Hkv)]


def test_head_priority_full_size(orc, ta, dev):
    """The Phi-3-medium prefill keys (4 x 4096 tokens per KV head)."""
    from paper_2412_08585_amd import workloads as W
    w = W.WORKLOADS["phi3m-prefill-4k"]
    _, k, _ = W.prefill_inputs(w, device=dev)
    p = ta.turbo_head_priority(k).cpu().numpy()
    ref = orc.head_priority(k.cpu())
    np.testing.assert_allclose(p, ref, rtol=1e-5, atol=0)
    assert np.array_equal(ta.turbo_int2_heads(p, w.Hkv // 2), orc.int2_heads(ref, w.Hkv // 2))
    del k
    torch.cuda.empty_cache()
