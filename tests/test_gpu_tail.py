"""GPU parity of the int8 KV-cache buffer (Sec. 3.3): its start after a
prefill, one-token appends with the flush of a full buffer into a step-2
group, and decode over the groups plus the buffer, against the oracle.

Bar: the buffer's codes and universal scales, and every byte, code, scale
and zero point a flush writes into the paged cache, bit-exact; decode O
within 1e-3 of the row's largest |O| and L within 1e-4 (as for the decode
without a buffer); the integers of the buffer's chunk bit-exact through the
trace hook.
"""
import sys

import numpy as np
import pytest
import torch

from tests import cache_layout
from tests.decode_split import oracle_decode, split_of

pytestmark = pytest.mark.gpu

SM = 1 / np.sqrt(128)
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


def _rand(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(*shape, generator=g) * scale).half()


def _bits_equal(a, b):
    return np.array_equal(np.asarray(a, np.float32).view(np.int32),
                          np.asarray(b, np.float32).view(np.int32))


def _cmp_o(got, want, what):
    g = got.float().cpu().numpy()
    rowmax = np.maximum(np.abs(want).max(axis=-1, keepdims=True), 1e-30)
    worst = float(np.max(np.abs(g - want) / rowmax))
    assert np.all(np.isfinite(g)), what
    assert worst < O_TOL, f"{what}: max rel-to-row-max error {worst:.3e}"


def _cmp_lse(got, want, what):
    g = got.cpu().numpy().astype(np.float64)
    fin = np.isfinite(want)
    assert np.array_equal(np.isfinite(g), fin), what
    if fin.any():
        worst = float(np.max(np.abs(g[fin] - want[fin])))
        assert worst < LSE_TOL, f"{what}: lse error {worst:.3e}"


class Session:
    """One prefill of B sequences of N tokens into a paged cache of mg groups
    per sequence and the buffer after it, on the GPU and in the oracle."""

    def __init__(self, orc, ta, dev, B, Hkv, N, mg, bits, seed):
        self.orc, self.ta, self.dev = orc, ta, dev
        self.B, self.Hkv, self.N, self.mg, self.bits = B, Hkv, N, mg, list(bits)
        k = _rand((B, Hkv, N, 128), seed)
        v = _rand((B, Hkv, N, 128), seed + 1, 2.0)
        k[..., 3] *= 8
        rng = np.random.default_rng(seed)
        self.bt = rng.permutation(B * 4 * mg).astype(np.int32).reshape(B, 4 * mg)
        self.gt = rng.permutation(B * mg).astype(np.int32).reshape(B, mg)
        self.btd, self.gtd = torch.from_numpy(self.bt).to(dev), torch.from_numpy(self.gt).to(dev)
        self.cache = ta.PagedKVCache(self.bt.size, self.gt.size, bits, dev)
        kd, vd = k.to(dev), v.to(dev)
        _, _, sk, sv = ta.turbo_quantize_kv(kd, vd, self.cache, self.btd, self.gtd)
        self.tail = ta.KVTail(B, Hkv, dev)
        ta.turbo_tail_init(kd, vd, sk, sv, self.tail)
        torch.cuda.synchronize()
        qkv = orc.quantize_kv(k, v, bits)
        self.rcache = orc.cache_from_prefill(qkv, 64 * mg)
        self.rtail = orc.tail_init(k, v, qkv)
        self.pos = N

    def append(self, kn, vn):
        sl = torch.full((self.B,), self.pos, dtype=torch.int32, device=self.dev)
        self.ta.turbo_append_kv(kn.to(self.dev), vn.to(self.dev), sl, self.cache, self.tail,
                                self.btd, self.gtd)
        self.orc.append_kv(self.rcache, self.rtail, kn, vn, [self.pos] * self.B)
        self.pos += 1

    def check_tail(self):
        torch.cuda.synchronize()
        assert np.array_equal(self.tail.k.cpu().numpy(), self.rtail["tk"]), "buffer K codes"
        assert np.array_equal(self.tail.v.cpu().numpy(), self.rtail["tv"]), "buffer V codes"
        sc = self.tail.scale.cpu().numpy()
        assert _bits_equal(sc[..., 0], self.rtail["tsk"]) and _bits_equal(sc[..., 1], self.rtail["tsv"])

    def check_cache(self, ng):
        torch.cuda.synchronize()
        pages = self.cache.pages.cpu().numpy()
        gmeta = self.cache.group_meta.cpu().numpy()
        gscale = self.cache.group_scale.cpu().numpy()
        for b in range(self.B):
            for h in range(self.Hkv):
                u = cache_layout.read_unit(pages, gmeta, gscale, self.bits, self.bt, self.gt, b, h, ng)
                for key in ("kc", "vc"):
                    assert np.array_equal(u[key], self.rcache[key][b, h, :64 * ng]), (b, h, key)
                for key in ("ks", "kz", "vs", "vz"):
                    assert np.array_equal(u[key], self.rcache[key][b, h, :ng]), (b, h, key)
                assert _bits_equal(u["sk"], self.rcache["sk"][b, h, :ng]), (b, h, "sk")
                assert _bits_equal(u["sv"], self.rcache["sv"][b, h, :ng]), (b, h, "sv")


TAIL_INIT_CASES = [
    # B, Hkv, N, bits
    (2, 3, 64 * 2 + 21, [4, 2, 4]),
    (1, 2, 64 * 3, [2, 4]),     # no trailing token: an empty buffer
    (2, 1, 17, [4]),            # no full group: everything in the buffer
    (1, 4, 64 + 63, [4, 4, 2, 2]),
]


@pytest.mark.parametrize("B,Hkv,N,bits", TAIL_INIT_CASES)
def test_tail_init_bit_exact(orc, ta, dev, B, Hkv, N, bits):
    _log(f"tail_init B={B} Hkv={Hkv} N={N} bits={bits}")
    s = Session(orc, ta, dev, B, Hkv, N, max(1, N // 64 + 1), bits, 2000 + N)
    s.check_tail()


@pytest.mark.parametrize("bits", [[4, 2], [2, 4, 4]])
def test_append_and_flush_bit_exact(orc, ta, dev, bits):
    """Appends from a 124-token prefill: the 4th fills the buffer and flushes
    it into group 1, the 68th into group 2; new tokens far outside the
    universal range clamp to +-119."""
    Hkv = len(bits)
    B, N, mg = 2, 64 + 60, 4
    _log(f"append B={B} Hkv={Hkv} N={N} bits={bits}")
    s = Session(orc, ta, dev, B, Hkv, N, mg, bits, 2100 + Hkv)
    for i in range(70):
        kn = _rand((B, Hkv, 128), 3000 + i, 0.7)
        vn = _rand((B, Hkv, 128), 4000 + i, 1.5)
        if i % 9 == 0:
            kn[0, 0, 17] = 60000.0
            vn[B - 1, Hkv - 1, 5] = -60000.0
        s.append(kn, vn)
        if i in (2, 3, 4, 67, 69):
            _log(f"  after append {i}: position {s.pos}")
            s.check_tail()
            s.check_cache(s.pos // 64)
    assert s.pos // 64 == 3


def test_append_beyond_the_table_keeps_the_buffer(orc, ta, dev):
    """A buffer that fills past the last group of the tables is not flushed
    (no table entry to write); the cache stays as it was."""
    B, Hkv, N, mg = 1, 2, 64 + 62, 1
    _log("append beyond the tables")
    s = Session(orc, ta, dev, B, Hkv, N, mg, [4, 2], 2200)
    before = s.cache.pages.clone(), s.cache.group_meta.clone(), s.cache.group_scale.clone()
    for i in range(2):
        s.append(_rand((B, Hkv, 128), 5000 + i), _rand((B, Hkv, 128), 5100 + i))
    s.check_tail()
    torch.cuda.synchronize()
    assert torch.equal(s.cache.pages, before[0]) and torch.equal(s.cache.group_meta, before[1])
    assert torch.equal(s.cache.group_scale, before[2])


DECODE_TAIL_CASES = [
    # B, Hq, Hkv, N, mg, bits, extra appends, per-sequence seq_lens (None: the
    # session's position), split
    (2, 8, 2, 64 * 3 + 29, 5, [4, 2], 1, None, 1),
    (2, 8, 2, 64 * 3 + 29, 5, [4, 2], 1, None, 2),
    (2, 8, 2, 64 * 3 + 29, 5, [4, 2], 1, None, 0),
    (2, 10, 2, 64 * 2 + 5, 4, [2, 4], 3, [40, 128], 1),     # G = 5; no group / no buffer
    (2, 10, 2, 64 * 2 + 5, 4, [2, 4], 3, [0, 64 * 2 + 8], 100),
    (1, 16, 1, 64 * 6 + 50, 7, [4], 26, None, 3),  # flush at 447; 12 more past the tables
    (3, 4, 4, 64 + 1, 3, [4, 2, 2, 4], 0, None, 0),
]


@pytest.mark.parametrize("B,Hq,Hkv,N,mg,bits,extra,sl,split", DECODE_TAIL_CASES)
def test_decode_with_buffer_parity(orc, ta, dev, B, Hq, Hkv, N, mg, bits, extra, sl, split):
    _log(f"decode+buffer B={B} Hq={Hq} Hkv={Hkv} N={N} mg={mg} bits={bits} extra={extra} "
         f"seq={sl} split={split}")
    s = Session(orc, ta, dev, B, Hkv, N, mg, bits, 2300 + N + extra)
    for i in range(extra):
        s.append(_rand((B, Hkv, 128), 6000 + i), _rand((B, Hkv, 128), 6100 + i))
    seq = [s.pos] * B if sl is None else sl
    q = _rand((B, Hq, 128), 2400 + N)
    sld = torch.tensor(seq, dtype=torch.int32, device=dev)
    o, lse = ta.turbo_attn_decode(q.to(dev), s.cache, sld, s.btd, s.gtd, SM, split,
                                  return_lse=True, tail=s.tail)
    torch.cuda.synchronize()
    ro, rl = oracle_decode(orc, q, s.rcache, seq, SM, split, mg, tail=s.rtail)
    _cmp_o(o, ro, "decode+buffer O")
    _cmp_lse(lse, rl, "decode+buffer lse")
    # the buffer's chunk, bit for bit, for one query row of each sequence
    for b in range(B):
        ng = min(seq[b] // 64, mg)
        h = (3 * b + 1) % Hq
        o2, g = ta.turbo_attn_decode_trace(q.to(dev), s.cache, sld, s.btd, s.gtd, (b, h, ng), SM,
                                           split, tail=s.tail)
        assert torch.equal(o2.view(torch.int16), o.view(torch.int16))
        _, _, r = orc.attn_decode(q, s.rcache, seq, SM, split=split_of(seq[b], split, mg),
                                  tail=s.rtail,
                                  trace=(b, h, ng))
        if not r["hit"]:  # empty buffer: nothing traced on either side
            assert not any(np.asarray(x).any() for x in g.values())
            continue
        nt = seq[b] - 64 * ng
        assert np.array_equal(g["q8"][0], r["q8"][0]), "Q8"
        assert np.array_equal(g["sacc"][0, :nt], r["sacc"][0, :nt]), "QK^T of the buffer"
        assert np.array_equal(g["qp"][0], r["qp"][0]), "Q(P~) of the buffer"
        assert np.array_equal(g["pvacc"][0], r["pvacc"][0]), "PV of the buffer"
        assert _bits_equal(g["sq"], r["sq"]) and _bits_equal(g["pmax"], r["pmax"])


def test_decode_with_empty_buffer_matches_plain_decode(orc, ta, dev):
    """With no buffered token the buffer adds nothing: the same O and L as the
    decode without it (bit for bit when both go through the chunk merge; with
    one chunk the plain decode writes O directly, in another rounding order)."""
    B, Hq, Hkv, N, mg = 2, 8, 2, 64 * 4, 4
    _log("decode with an empty buffer")
    s = Session(orc, ta, dev, B, Hkv, N, mg, [4, 2], 2500)
    q = _rand((B, Hq, 128), 2501).to(dev)
    sld = torch.tensor([N, 128], dtype=torch.int32, device=dev)
    for split in (1, 2, 3):
        a, la = ta.turbo_attn_decode(q, s.cache, sld, s.btd, s.gtd, SM, split, return_lse=True)
        b, lb = ta.turbo_attn_decode(q, s.cache, sld, s.btd, s.gtd, SM, split, return_lse=True,
                                     tail=s.tail)
        torch.cuda.synchronize()
        if split == 1:
            _cmp_o(b, a.float().cpu().numpy(), "one chunk, merged vs direct")
            _cmp_lse(lb, la.cpu().numpy().astype(np.float64), "one chunk lse")
        else:
            assert torch.equal(a.view(torch.int16), b.view(torch.int16))
            assert torch.equal(la, lb)


def test_tail_init_on_views_of_one_buffer(ta, dev):
    """KVTail.narrow: starting the buffers of a batch in two parts (as a caller
    that builds the cache sequence by sequence does) gives the same buffer as
    one call over the whole batch."""
    B, Hkv, N = 4, 2, 64 + 30
    k, v = _rand((B, Hkv, N, 128), 2600).to(dev), _rand((B, Hkv, N, 128), 2601).to(dev)
    whole = ta.KVTail(B, Hkv, dev)
    _, _, sk, sv = ta.turbo_quantize_kv(k, v)
    ta.turbo_tail_init(k, v, sk, sv, whole)
    parts = ta.KVTail(B, Hkv, dev)
    for b0, n in ((0, 1), (1, 3)):
        _, _, skp, svp = ta.turbo_quantize_kv(k[b0:b0 + n], v[b0:b0 + n])
        ta.turbo_tail_init(k[b0:b0 + n], v[b0:b0 + n], skp, svp, parts.narrow(b0, n))
    torch.cuda.synchronize()
    assert torch.equal(whole.k, parts.k) and torch.equal(whole.v, parts.v)
    assert torch.equal(whole.scale, parts.scale)
