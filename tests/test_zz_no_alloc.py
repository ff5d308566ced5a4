"""turbo_attn_decode_noalloc (the decode for callers that cannot allocate)
against turbo_attn_decode with a caller workspace: the same kernels on the
same inputs, so O and L must agree bit for bit, over two calls in a row on
the shared per-GPU scratch, the second with a smaller input; both within the
parity bar of the oracle; and sizes beyond the scratch rejected before any
launch."""
import ctypes
import sys

import numpy as np
import pytest
import torch

from tests.decode_split import oracle_decode

SM = 1 / np.sqrt(128)


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
    return ta


def _rand(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(*shape, generator=g) * scale).half()


def _case(ta, dev, B, Hq, Hkv, N, bits, seed):
    k = _rand((B, Hkv, N, 128), seed)
    v = _rand((B, Hkv, N, 128), seed + 1)
    k[..., 7] *= 10
    q = _rand((B, Hq, 128), seed + 2)
    mg = N // 64
    rng = np.random.default_rng(seed)
    bt = rng.permutation(B * 4 * mg).astype(np.int32).reshape(B, 4 * mg)
    gt = rng.permutation(B * mg).astype(np.int32).reshape(B, mg)
    cache = ta.PagedKVCache(bt.size, gt.size, bits, dev)
    btd, gtd = torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)
    ta.turbo_quantize_kv(k.to(dev), v.to(dev), cache, btd, gtd)
    return k, v, q, cache, btd, gtd


@pytest.mark.gpu
def test_noalloc_decode_matches_workspace_decode(orc, ta, dev):
    # (B, Hq, Hkv, N, bits, seq_lens, kv_split_groups): the second call is
    # smaller (fewer sequences, shorter cache, fewer chunk states)
    calls = [(3, 8, 2, 64 * 140, [4, 2], [64 * 140, 64 * 77 + 5, 64 * 20], 0),
             (2, 4, 1, 64 * 40, [2], [64 * 40, 64 * 9], 4)]
    for i, (B, Hq, Hkv, N, bits, sl, split) in enumerate(calls):
        _log(f"noalloc decode call {i}: B={B} Hq={Hq} Hkv={Hkv} N={N} seq={sl} split={split}")
        k, v, q, cache, btd, gtd = _case(ta, dev, B, Hq, Hkv, N, bits, 300 + 10 * i)
        sld = torch.tensor(sl, dtype=torch.int32, device=dev)
        qd = q.to(dev)
        o_ws, l_ws = ta.turbo_attn_decode(qd, cache, sld, btd, gtd, SM, split, return_lse=True)
        o_na = torch.empty_like(qd)
        l_na = torch.empty(B, Hq, dtype=torch.float32, device=dev)
        ta.turbo_attn_decode_noalloc(qd, cache, sld, btd, gtd, SM, split, out=o_na, lse_out=l_na)
        torch.cuda.synchronize()
        assert torch.equal(o_na.view(torch.int16), o_ws.view(torch.int16)), i
        assert torch.equal(l_na.view(torch.int32), l_ws.view(torch.int32)), i
        ref = orc.quantize_kv(k, v, bits)
        ro, rl = oracle_decode(orc, q, ref, sl, SM, split, N // 64)
        g = o_na.float().cpu().numpy()
        err = np.max(np.abs(g - ro) / np.maximum(np.abs(ro).max(axis=-1, keepdims=True), 1e-30))
        assert err < 1e-3, err
        assert np.max(np.abs(l_na.cpu().numpy() - rl)) < 1e-4


@pytest.mark.gpu
def test_noalloc_decode_rejects_sizes_beyond_the_scratch(ta, dev):
    L = ta.lib()
    cs = ta.TurboKVCacheStruct()
    cs.pages = cs.group_meta = cs.group_scale = ctypes.c_void_p(256)
    cs.num_pages = cs.num_group_slots = 1
    cs.num_kv_heads, cs.head_dim = 8, 128
    for h in range(8):
        cs.head_bits[h] = 4
    p = ctypes.c_void_p(256)
    # 4096 sequences x 32 query heads x 4 chunk states x 528 bytes > 32 MiB
    assert L.turbo_decode_workspace_bytes(4096, 32, 8, 512, 0, 0) > (32 << 20)
    st = L.turbo_attn_decode_noalloc(p, ctypes.byref(cs), None, p, p, p, 512, 4096, 32,
                                     ctypes.c_float(SM), 0, p, None, None)
    assert st == -3 and b"workspace" in L.turbo_strerror(st)
