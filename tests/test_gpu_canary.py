"""Every entry point writes inside its outputs only: each output (and each
workspace, cache and buffer the call writes) is placed inside a device buffer
whose 4 KiB before and after hold a byte pattern, and the pattern must
survive the call.  Shapes are ragged (partial blocks, short last groups) so
that the kernels' edge paths run."""
import ctypes
import sys

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

PAD = 4096
PAT = 0xA5
SM = float(1 / np.sqrt(128))


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


class Guarded:
    def __init__(self, dev):
        self.dev, self.bufs = dev, []

    def __call__(self, shape, dtype):
        n = int(np.prod(shape)) * torch.empty(0, dtype=dtype).element_size()
        buf = torch.full((n + 2 * PAD,), PAT, dtype=torch.uint8, device=self.dev)
        self.bufs.append((buf, n))
        return buf[PAD:PAD + n].view(dtype).view(*shape)

    def check(self, what):
        torch.cuda.synchronize()
        for i, (buf, n) in enumerate(self.bufs):
            h = buf.cpu().numpy()
            assert (h[:PAD] == PAT).all(), f"{what}: write before output {i}"
            assert (h[PAD + n:] == PAT).all(), f"{what}: write after output {i}"


def _rand(shape, seed, dev):
    g = torch.Generator().manual_seed(seed)
    return torch.randn(*shape, generator=g).half().to(dev)


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _tables(B, mg, seed, dev):
    rng = np.random.default_rng(seed)
    bt = rng.permutation(B * 4 * mg).astype(np.int32).reshape(B, 4 * mg)
    gt = rng.permutation(B * mg).astype(np.int32).reshape(B, mg)
    return torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)


def _cache(ta, g, npages, nslots, bits):
    c = ta.PagedKVCache(1, 1, bits, g.dev)
    c.pages = g((npages, c.page_bytes), torch.uint8)
    c.group_meta = g((nslots, len(bits), 4, 128), torch.int8)
    c.group_scale = g((nslots, len(bits), 2), torch.float32)
    for t in (c.pages, c.group_meta, c.group_scale):
        t.zero_()
    return c


def test_quantize_prefill_decode_stay_inside_outputs(ta, dev):
    L = ta.lib()
    s = ta.binding._stream(dev)
    B, Hq, Hkv, N = 2, 6, 3, 64 * 3 + 17
    bits = [4, 2, 4]
    nb, mg = (N + 63) // 64, N // 64 + 1
    q, k, v = _rand((B, Hq, N, 128), 1, dev), _rand((B, Hkv, N, 128), 2, dev), \
        _rand((B, Hkv, N, 128), 3, dev)
    btd, gtd = _tables(B, mg, 4, dev)
    g = Guarded(dev)
    cache = _cache(ta, g, B * 4 * mg, B * mg, bits)
    k8, v8 = g((B, Hkv, nb * 64, 128), torch.int8), g((B, Hkv, nb, 128, 64), torch.int8)
    sk, sv = g((B, Hkv, nb), torch.float32), g((B, Hkv, nb), torch.float32)
    _log("canary quantize_kv")
    ta.turbo_quantize_kv(k, v, cache, btd, gtd, out=(k8, v8, sk, sv))
    g.check("turbo_quantize_kv")
    for bc in (32, 128):
        nbc = (N + bc - 1) // bc
        gb = Guarded(dev)
        out = (gb((B, Hkv, nb * 64, 128), torch.int8), gb((B, Hkv, nb, 128, 64), torch.int8),
               gb((B, Hkv, nbc), torch.float32), gb((B, Hkv, nbc), torch.float32))
        ta.turbo_quantize_kv(k, v, out=out, block_cols=bc)
        gb.check(f"turbo_quantize_kv_blocks {bc}")
    _log("canary prefill")
    o, lse = g((B, Hq, N, 128), torch.float16), g((B, Hq, N), torch.float32)
    assert L.turbo_attn_prefill(_p(q), _p(k8), _p(v8), _p(sk), _p(sv), B, Hq, Hkv, N, 128, SM, 1,
                                _p(o), _p(lse), s) == 0
    g.check("turbo_attn_prefill")
    for br, bc in [(32, 32), (128, 64), (64, 128), (128, 128)]:
        gb = Guarded(dev)
        k8b, v8b, skb, svb = ta.turbo_quantize_kv(k, v, block_cols=bc)
        ob, lb = gb((B, Hq, N, 128), torch.float16), gb((B, Hq, N), torch.float32)
        assert L.turbo_attn_prefill_blocks(_p(q), _p(k8b), _p(v8b), _p(skb), _p(svb), B, Hq, Hkv,
                                           N, 128, SM, 1, br, bc, _p(ob), _p(lb), s) == 0
        tr = gb((ta.binding.TRACE_BYTES,), torch.uint8)
        assert L.turbo_attn_prefill_blocks_trace(_p(q), _p(k8b), _p(v8b), _p(skb), _p(svb), B,
                                                 Hq, Hkv, N, 128, SM, 1, br, bc, _p(ob), _p(lb),
                                                 1, 4, (N - 1) // br, 0, _p(tr), s) == 0
        gb.check(f"turbo_attn_prefill_blocks ({br}, {bc})")
    _log("canary decode")
    qd = _rand((B, Hq, 128), 5, dev)
    sld = torch.tensor([N, 64 * 2 + 5], dtype=torch.int32, device=dev)
    tail = ta.KVTail(B, Hkv, dev)
    tail.k, tail.v = g((B, Hkv, 64, 128), torch.int8), g((B, Hkv, 128, 64), torch.int8)
    tail.scale = g((B, Hkv, 2), torch.float32)
    ta.turbo_tail_init(k, v, sk, sv, tail)
    g.check("turbo_tail_init")
    for split in (0, 1, 2):
        for with_tail in (False, True):
            n = int(L.turbo_decode_workspace_bytes(B, Hq, Hkv, mg, split, int(with_tail)))
            ws = g((max(n, 4),), torch.uint8)
            od, ld = g((B, Hq, 128), torch.float16), g((B, Hq), torch.float32)
            cs = cache.struct()
            ts = tail.struct() if with_tail else None
            assert L.turbo_attn_decode(_p(qd), ctypes.byref(cs), ctypes.byref(ts) if ts else None,
                                       _p(sld), _p(btd), _p(gtd), mg, B, Hq, SM, split, _p(ws), n,
                                       _p(od), _p(ld), s) == 0
            g.check(f"turbo_attn_decode split={split} tail={with_tail}")
            assert L.turbo_attn_decode_noalloc(_p(qd), ctypes.byref(cs),
                                               ctypes.byref(ts) if ts else None, _p(sld), _p(btd),
                                               _p(gtd), mg, B, Hq, SM, split, _p(od), _p(ld),
                                               s) == 0
            g.check(f"turbo_attn_decode_noalloc split={split} tail={with_tail}")
            tr = g((ta.binding.TRACE_BYTES,), torch.uint8)
            assert L.turbo_attn_decode_trace(_p(qd), ctypes.byref(cs),
                                             ctypes.byref(ts) if ts else None, _p(sld), _p(btd),
                                             _p(gtd), mg, B, Hq, SM, split, _p(ws), n, _p(od),
                                             _p(ld), 1, 5, 2, _p(tr), s) == 0
            g.check(f"turbo_attn_decode_trace split={split} tail={with_tail}")
    _log("canary append")
    for step in range(3):
        kn, vn = _rand((B, Hkv, 128), 10 + step, dev), _rand((B, Hkv, 128), 20 + step, dev)
        ta.turbo_append_kv(kn, vn, sld, cache, tail, btd, gtd)
        sld += 1
        g.check(f"turbo_append_kv step {step}")
    # appends up to the flush of sequence 1's buffer into its next group
    for step in range(64):
        kn, vn = _rand((B, Hkv, 128), 30 + step, dev), _rand((B, Hkv, 128), 40 + step, dev)
        ta.turbo_append_kv(kn, vn, sld, cache, tail, btd, gtd)
        sld += 1
    g.check("turbo_append_kv with flushes")


def test_projection_priority_softmax_probes_stay_inside_outputs(ta, dev):
    L = ta.lib()
    s = ta.binding._stream(dev)
    B, N, D, Hq, Hkv = 2, 64 * 2 + 29, 192, 2, 1
    bits = [2]
    F = (Hq + 2 * Hkv) * 128
    nb, mg = (N + 63) // 64, N // 64
    g = Guarded(dev)
    x = _rand((B, N, D), 50, dev)
    w = (_rand((F, D), 51, dev).float() / 14).half()
    btd, gtd = _tables(B, mg, 52, dev)
    cache = _cache(ta, g, B * 4 * mg, B * mg, bits)
    out = (g((B, Hq, nb * 64, 128), torch.int8), g((B, Hq, nb), torch.float32),
           g((B, Hkv, nb * 64, 128), torch.int8), g((B, Hkv, nb, 128, 64), torch.int8),
           g((B, Hkv, nb), torch.float32), g((B, Hkv, nb), torch.float32))
    _log("canary qkv_project")
    ta.turbo_qkv_project(x, w, Hq, Hkv, cache, btd, gtd, out=out)
    g.check("turbo_qkv_project")
    y = g((B, N, F), torch.float16)
    ta.turbo_qkv_project(x, w, Hq, Hkv, cache, btd, gtd, out=out, y=y)
    g.check("turbo_qkv_project_trace")
    o = g((B, Hq, N, 128), torch.float16)
    ta.turbo_attn_prefill_q8(out[0], out[1], out[2], out[3], out[4], out[5], N, out=o)
    g.check("turbo_attn_prefill_q8")
    _log("canary head_priority")
    k = _rand((3, 5, 300, 128), 53, dev)
    n = int(L.turbo_head_priority_workspace_bytes(3, 5, 300))
    ws, pr = g((n,), torch.uint8), g((5,), torch.float32)
    assert L.turbo_head_priority(_p(k), 3, 5, 300, 128, _p(ws), n, _p(pr), s) == 0
    g.check("turbo_head_priority")
    _log("canary sas_softmax")
    for rows, cols in [(37, 4096), (5, 3000), (9, 21), (3, 20000)]:
        xs = torch.randn(rows, cols, device=dev) * 2
        ys = g((rows, cols), torch.float32)
        assert L.turbo_sas_softmax(_p(xs), _p(ys), rows, cols, s) == 0
        g.check(f"turbo_sas_softmax {rows}x{cols}")
    _log("canary probes")
    sink = g((512,), torch.int32)
    ops = ctypes.c_int64(0)
    assert L.turbo_probe_mfma_i8(4, _p(sink), ctypes.byref(ops), s) == 0
    src = torch.ones(1 << 18, dtype=torch.float32, device=dev)
    sink1 = g((1,), torch.int32)
    assert L.turbo_probe_read(_p(src), src.numel() * 4, _p(sink1), s) == 0
    sink2 = g((1024,), torch.float32)
    insts = ctypes.c_int64(0)
    assert L.turbo_probe_valu(4, _p(sink2), ctypes.byref(insts), s) == 0
    assert insts.value == 1024 * 4 * 8 * 4
    g.check("probes")
