"""Host-side checks of the C ABI library (no GPU): it loads, exports every
function declared in include/*.h, rejects bad arguments before any launch,
and its sizing helpers follow the documented formulas.  Also host checks of
the integer tricks the kernels rely on and of the cache format reader."""
import ctypes
import glob
import os
import re

import numpy as np
import pytest

from tests import cache_layout

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def ta():
    import paper_2412_08585_amd as ta
    if not os.path.exists(ta.binding.LIB_PATH):
        from paper_2412_08585_amd import build
        build.build()
    return ta


def _declared_functions():
    names = []
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        src = open(h).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names += re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(turbo_\w+)\s*\(", src, flags=re.M)
    return sorted(set(names))


def test_exports_every_declared_function(ta):
    names = _declared_functions()
    assert {"turbo_quantize_kv", "turbo_attn_prefill", "turbo_attn_decode"} <= set(names)
    L = ctypes.CDLL(ta.binding.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n


def test_version_and_strerror(ta):
    L = ta.lib()
    assert L.turbo_abi_version() == 4
    for st in (0, -1, -2, -3, -4, 7):
        assert L.turbo_strerror(st)


def test_page_bytes(ta):
    assert ta.page_bytes([4] * 10) == 10 * 2048
    assert ta.page_bytes([4, 2, 2, 4]) == 2048 * 2 + 1024 * 2
    assert ta.page_bytes([3]) == 0
    assert ta.page_bytes([]) == 0
    assert ta.page_bytes([4] * 65) == 0


def test_invalid_arguments_rejected_before_launch(ta):
    L = ta.lib()
    P = ctypes.c_void_p
    dummy = P(16)
    # d != 128
    assert L.turbo_quantize_kv(dummy, dummy, 1, 1, 64, 64, dummy, dummy, dummy, dummy, None, None,
                               None, 0, None) == -1
    # Hq % Hkv != 0
    assert L.turbo_attn_prefill(dummy, dummy, dummy, dummy, dummy, 1, 6, 4, 64, 128, 0.1, 1, dummy,
                                None, None) == -1
    # GQA ratio above 16
    assert L.turbo_attn_prefill(dummy, dummy, dummy, dummy, dummy, 1, 34, 2, 64, 128, 0.1, 1, dummy,
                                None, None) == -1
    # null output
    assert L.turbo_attn_prefill(dummy, dummy, dummy, dummy, dummy, 1, 4, 4, 64, 128, 0.1, 1, None,
                                None, None) == -1
    # non-positive / NaN scale
    for sm in (0.0, -1.0, float("nan")):
        assert L.turbo_attn_prefill(dummy, dummy, dummy, dummy, dummy, 1, 4, 4, 64, 128, sm, 1,
                                    dummy, None, None) == -1
    # empty problem is a no-op success (no device touched)
    assert L.turbo_attn_prefill(None, None, None, None, None, 0, 4, 4, 64, 128, 0.1, 1, None, None,
                                None) == 0
    assert L.turbo_quantize_kv(None, None, 1, 1, 0, 128, None, None, None, None, None, None, None, 0,
                               None) == 0
    # cache with a bad bit width
    c = ta.TurboKVCacheStruct()
    c.pages, c.group_meta, c.group_scale = 16, 16, 16
    c.num_pages, c.num_group_slots, c.num_kv_heads, c.head_dim = 4, 1, 1, 128
    c.head_bits[0] = 3
    assert L.turbo_attn_decode(dummy, ctypes.byref(c), None, dummy, dummy, dummy, 1, 1, 1, 0.1, 1,
                               None, 0, dummy, None, None) == -1
    c.head_bits[0] = 4
    # workspace required for 2 chunks of 1 group each but not given
    assert L.turbo_attn_decode(dummy, ctypes.byref(c), None, dummy, dummy, dummy, 2, 1, 1, 0.1, 1,
                               None, 0, dummy, None, None) == -3
    # quantize with a cache whose head count differs from Hkv
    assert L.turbo_quantize_kv(dummy, dummy, 1, 2, 64, 128, dummy, dummy, dummy, dummy,
                               ctypes.byref(c), dummy, dummy, 1, None) == -1
    # max_groups too small for N
    assert L.turbo_quantize_kv(dummy, dummy, 1, 1, 192, 128, dummy, dummy, dummy, dummy,
                               ctypes.byref(c), dummy, dummy, 2, None) == -1
    # block sizes outside {32, 64, 128}
    for br, bc in ((0, 64), (16, 64), (96, 64), (256, 64), (64, 0), (64, 16), (32, 256)):
        assert L.turbo_attn_prefill_blocks(dummy, dummy, dummy, dummy, dummy, 1, 4, 4, 64, 128,
                                           0.1, 1, br, bc, dummy, None, None) == -1
    for bc in (0, 16, 48, 256):
        assert L.turbo_quantize_kv_blocks(dummy, dummy, 1, 1, 64, 128, bc, dummy, dummy, dummy,
                                          dummy, None) == -1
    assert L.turbo_quantize_kv_blocks(None, None, 0, 1, 64, 128, 32, None, None, None, None,
                                      None) == 0
    # SAS softmax: bad sizes and null pointers; zero rows is a no-op
    assert L.turbo_sas_softmax(dummy, dummy, -1, 8, None) == -1
    assert L.turbo_sas_softmax(dummy, dummy, 4, 0, None) == -1
    assert L.turbo_sas_softmax(dummy, dummy, 1 << 31, 8, None) == -1
    assert L.turbo_sas_softmax(None, dummy, 4, 8, None) == -1
    assert L.turbo_sas_softmax(None, None, 0, 8, None) == 0


def test_trace_hooks_reject_bad_arguments(ta):
    """The *_trace test hooks check the trace buffer and the selected tile or
    group before any launch."""
    L = ta.lib()
    P = ctypes.c_void_p
    dummy = P(16)
    pre = (dummy, dummy, dummy, dummy, dummy, 1, 4, 4, 130, 128, 0.1, 1, dummy, None)
    assert L.turbo_attn_prefill_trace(*pre, 0, 0, 0, 0, None, None) == -1     # no buffer
    for tile in [(1, 0, 0, 0), (0, 4, 0, 0), (0, 0, 3, 0), (0, 0, 0, 3), (-1, 0, 0, 0)]:
        assert L.turbo_attn_prefill_trace(*pre, *tile, dummy, None) == -1
    bad = (dummy, dummy, dummy, dummy, dummy, 1, 6, 4, 130, 128, 0.1, 1, dummy, None)
    assert L.turbo_attn_prefill_trace(*bad, 0, 0, 0, 0, dummy, None) == -1     # Hq % Hkv
    c = ta.TurboKVCacheStruct()
    c.pages, c.group_meta, c.group_scale = 16, 16, 16
    c.num_pages, c.num_group_slots, c.num_kv_heads, c.head_dim = 4, 1, 1, 128
    c.head_bits[0] = 4
    dec = (dummy, ctypes.byref(c), None, dummy, dummy, dummy, 2, 1, 1, 0.1, 1, None, 0, dummy, None)
    assert L.turbo_attn_decode_trace(*dec, 0, 0, 0, None, None) == -1
    for sel in [(1, 0, 0), (0, 1, 0), (0, 0, 3), (0, 0, -1)]:
        assert L.turbo_attn_decode_trace(*dec, *sel, dummy, None) == -1


def test_trace_layout_matches_header(ta):
    src = open(os.path.join(ROOT, "include", "turbo_attn.h")).read()
    vals = {m[0]: int(m[1]) for m in re.findall(r"#define (TURBO_TRACE_\w+) (\d+)", src)}
    b = ta.binding
    assert (vals["TURBO_TRACE_Q8"], vals["TURBO_TRACE_S"], vals["TURBO_TRACE_P"],
            vals["TURBO_TRACE_PV"], vals["TURBO_TRACE_SQ"], vals["TURBO_TRACE_PMAX"],
            vals["TURBO_TRACE_BYTES"]) == (b.TRACE_Q8, b.TRACE_S, b.TRACE_P, b.TRACE_PV,
                                           b.TRACE_SQ, b.TRACE_PMAX, b.TRACE_BYTES)
    # contiguous, sized for the largest tile (B_r = B_c = 128): int8 128x128,
    # int32 128x128, int8 128x128, int32 128x128, two floats
    assert b.TRACE_S == 128 * 128 and b.TRACE_P == b.TRACE_S + 4 * 128 * 128
    assert b.TRACE_PV == b.TRACE_P + 128 * 128 and b.TRACE_SQ == b.TRACE_PV + 4 * 128 * 128
    assert b.TRACE_BYTES == b.TRACE_SQ + 8


def test_decode_load_addresses_stay_in_their_regions():
    """Host replica of the decode prefetch addresses (load_group in
    attn_decode.hip): every byte a lane reads lies in its KV head's region of a
    16-token page (K codes in the first half, V codes in the second) or in the
    group's 512-byte metadata, and the lanes together cover each region once."""
    for bits in (4, 2):
        kbytes, vbytes = (16, 8) if bits == 4 else (8, 4)
        kstep, vstep = 4 * 16 * bits, 2 * bits
        kseen, vseen = set(), set()
        for lane in range(64):
            n, g4, m = lane & 15, lane >> 4, lane & 15
            for mb in range(4):
                o = (m & 3) * 16 * bits + 4 * bits * g4 + mb * kstep
                assert 0 <= o and o + kbytes <= 256 * bits
                kseen |= set(range(o, o + kbytes))
            for cb in range(8):
                o = 256 * bits + (16 * cb + n) * vstep
                assert o + vbytes <= 512 * bits
                vseen |= set(range(o, o + vbytes))
            for o, w in [(32 * g4, 16), (32 * g4 + 16, 16), (128 + 32 * g4, 16),
                         (144 + 32 * g4, 16), (256 + 4 * (lane >> 1), 4), (384 + 4 * (lane >> 1), 4)]:
                assert o + w <= 512 and o % w == 0
        assert kseen == set(range(256 * bits))
        assert vseen == set(range(256 * bits, 512 * bits))


def test_int2_heads_rule_matches_the_oracle(ta, orc):
    rng = np.random.default_rng(3)
    for Hkv in (1, 2, 8, 10, 64):
        p = rng.random(Hkv).astype(np.float32)
        p[rng.integers(Hkv)] = p[0]                        # a tie
        for n in sorted({0, Hkv // 2, Hkv}):
            assert np.array_equal(ta.turbo_int2_heads(p, n), orc.int2_heads(p.astype(np.float64), n))
    L = ta.lib()
    P = ctypes.c_void_p
    out = np.empty(4, np.uint8)
    nan = np.array([1.0, np.nan, 2.0, 3.0], np.float32)
    assert L.turbo_int2_heads(nan.ctypes.data_as(P), 4, 2, out.ctypes.data_as(P)) == -1
    ok = np.ones(4, np.float32)
    assert L.turbo_int2_heads(ok.ctypes.data_as(P), 4, 5, out.ctypes.data_as(P)) == -1
    assert L.turbo_int2_heads(None, 4, 2, out.ctypes.data_as(P)) == -1
    # head priority: empty input and bad shapes are rejected before any launch
    dummy = P(16)
    assert L.turbo_head_priority(dummy, 0, 4, 64, 128, dummy, 1 << 20, dummy, None) == -1
    assert L.turbo_head_priority(dummy, 1, 4, 64, 64, dummy, 1 << 20, dummy, None) == -1
    assert L.turbo_head_priority(None, 1, 4, 64, 128, dummy, 1 << 20, dummy, None) == -1
    # workspace: [Hkv][B * ceil(N / 256)][256] fp32
    assert L.turbo_head_priority_workspace_bytes(4, 10, 4096) == 10 * 4 * 16 * 256 * 4
    assert L.turbo_head_priority_workspace_bytes(2, 3, 257) == 3 * 2 * 2 * 256 * 4
    assert L.turbo_head_priority(dummy, 2, 3, 257, 128, dummy, 3 * 2 * 2 * 256 * 4 - 1, dummy,
                                 None) == -3


def test_decode_split_and_workspace(ta):
    L = ta.lib()
    # fewest (evenly filled) chunks whose waves fill two thirds of the
    # resident slots: 3072 (3 waves per SIMD) for up to 8 query heads per KV
    # head, else 2048
    assert L.turbo_decode_auto_split(64, 40, 10, 128) == 32   # 4 chunks: 2560 waves >= 2048
    assert L.turbo_decode_auto_split(256, 32, 8, 512) == 512  # 2048 waves unsplit
    assert L.turbo_decode_auto_split(4096, 32, 8, 4) == 4     # one chunk
    assert L.turbo_decode_auto_split(4, 40, 10, 64) == 2      # at least 2 groups a chunk
    assert L.turbo_decode_auto_split(16, 128, 8, 64) == 6     # G = 16: 11 chunks, 1408 >= 1366
    assert L.turbo_decode_auto_split(16, 64, 8, 64) == 4      # G = 8: 16 chunks, 2048 >= 2048
    assert L.turbo_decode_auto_split(1, 1, 1, 1) == 1
    assert L.turbo_decode_auto_split(1, 1, 1, 5) == 2
    assert L.turbo_decode_auto_split(0, 1, 1, 1) == 1

    def brute(B, Hq, Hkv, G):
        want = -(-2 * 1024 * (3 if Hq // Hkv <= 8 else 2) // 3)
        for n in range(1, G + 1):
            split = -(-G // n)
            if B * Hkv * -(-G // split) >= want:
                return max(split, min(2, G))
        return min(2, G)
    for B, Hq, Hkv, G in [(1, 8, 8, 256), (8, 32, 8, 128), (32, 16, 4, 300), (128, 16, 16, 64),
                          (3, 10, 5, 7), (2, 64, 4, 1000)]:
        assert L.turbo_decode_auto_split(B, Hq, Hkv, G) == brute(B, Hq, Hkv, G)
    cnt = 0
    assert L.turbo_decode_workspace_bytes(4, 8, 2, 10, 10, 0) == 0
    assert L.turbo_decode_workspace_bytes(4, 8, 2, 10, 3, 0) == cnt + 4 * 8 * 4 * 132 * 4
    assert L.turbo_decode_workspace_bytes(4, 8, 2, 10, 10, 1) == cnt + 4 * 8 * 2 * 132 * 4
    assert L.turbo_decode_workspace_bytes(4, 8, 2, 10, 3, 1) == cnt + 4 * 8 * 5 * 132 * 4
    assert L.turbo_decode_workspace_bytes(100, 8, 2, 10, 3, 0) == 100 * 8 * 4 * 132 * 4
    # the default chunking (kv_split_groups = 0) follows each sequence's own
    # group count: at most one chunk up to 32 groups, 4 chunks beyond 128
    assert L.turbo_decode_workspace_bytes(4, 8, 2, 32, 0, 0) == 0
    assert L.turbo_decode_workspace_bytes(4, 8, 2, 32, 0, 1) == cnt + 4 * 8 * 2 * 132 * 4
    assert L.turbo_decode_workspace_bytes(4, 8, 2, 100, 0, 0) == cnt + 4 * 8 * 4 * 132 * 4
    assert L.turbo_decode_workspace_bytes(4, 8, 2, 5000, 0, 1) == cnt + 4 * 8 * 5 * 132 * 4


def test_default_decode_split_depends_on_the_sequence_only(ta):
    from tests.decode_split import default_split
    L = ta.lib()
    for ng in list(range(0, 300)) + [511, 512, 513, 4096, 100000]:
        assert L.turbo_decode_default_split(ng) == default_split(ng), ng
        n = -(-max(ng, 1) // default_split(ng))
        assert n <= 4 and (ng > 32 or n == 1)


def test_step2_reciprocal_division_is_exact():
    """The step-2 kernel divides by 2s as (num * (2^20 // (2s) + 1)) >> 20;
    exact for every integer scale s in 1..80 and numerator up to 2*238 + s."""
    for s in range(1, 81):
        M = (1 << 20) // (2 * s) + 1
        num = np.arange(0, 2 * 238 + s + 1, dtype=np.int64)
        assert np.array_equal((num * M) >> 20, num // (2 * s)), s


def test_rne_magic_constant():
    """fma(a, b, 1.5*2^23) leaves round-half-even(a*b) in the low mantissa
    bits for |a*b| < 2^22 (binary32)."""
    magic = np.float32(12582912.0)
    assert magic.view(np.int32) == 0x4B400000
    x = np.array([-119.0, -2.5, -0.5, 0.5, 1.5, 2.5, 118.5, 119.0, 3.4999998], np.float64)
    got = ((x + np.float64(magic)).astype(np.float32).view(np.int32) - 0x4B400000)
    assert got.tolist() == np.rint(x).astype(int).tolist()


@pytest.mark.parametrize("bits", [[4, 2, 4], [2, 2], [4]])
def test_cache_format_round_trip(bits):
    rng = np.random.default_rng(1)
    H, ng, B = len(bits), 3, 2
    off, pb = cache_layout.head_offsets(bits)
    pages = np.zeros((B * ng * 4, pb), np.uint8)
    gmeta = np.zeros((B * ng, H, 4, 128), np.int8)
    gscale = np.zeros((B * ng, H, 2), np.float32)
    bt = rng.permutation(B * ng * 4).reshape(B, ng * 4)
    gt = rng.permutation(B * ng).reshape(B, ng)
    units = {}
    for b in range(B):
        for h in range(H):
            lv = (1 << bits[h]) - 1
            u = dict(kc=rng.integers(0, lv + 1, (ng * 64, 128)).astype(np.uint8),
                     vc=rng.integers(0, lv + 1, (ng * 64, 128)).astype(np.uint8),
                     ks=rng.integers(1, 80, (ng, 128)).astype(np.uint8),
                     kz=rng.integers(-119, 120, (ng, 128)).astype(np.int8),
                     vs=rng.integers(1, 80, (ng, 128)).astype(np.uint8),
                     vz=rng.integers(-119, 120, (ng, 128)).astype(np.int8),
                     sk=rng.random(ng).astype(np.float32), sv=rng.random(ng).astype(np.float32))
            units[b, h] = u
            cache_layout.write_unit(pages, gmeta, gscale, bits, bt, gt, b, h, u)
    for (b, h), u in units.items():
        r = cache_layout.read_unit(pages, gmeta, gscale, bits, bt, gt, b, h, ng)
        for key in u:
            assert np.array_equal(r[key], u[key]), (b, h, key)
    # documented byte order: int4 K byte 0 = channel 0 (low nibble), channel 1 (high)
    u = units[0, 0]
    first = pages[bt[0, 0], off[0]]
    if bits[0] == 4:
        assert first == (u["kc"][0, 0] | (u["kc"][0, 1] << 4))
    else:
        assert first == (u["kc"][0, 0] | (u["kc"][0, 1] << 2) | (u["kc"][0, 2] << 4)
                         | (u["kc"][0, 3] << 6))


def _qkv_tile(x, ntiles, nheads):
    """Host replica of the work-group order of k_qkv_project (qkv_tile)."""
    if ntiles % 8:
        return x // nheads, x % nheads
    k, i = x % 8, x // 8
    ntk, full = ntiles // 8, nheads // 8
    if i < full * ntk * 8:
        hg, rem = divmod(i, ntk * 8)
        tl, head = rem // 8, 8 * hg + rem % 8
    else:
        r = nheads - 8 * full
        rem = i - full * ntk * 8
        tl, head = rem // r, 8 * full + rem % r
    return tl * 8 + k, head


@pytest.mark.parametrize("ntiles,nheads", [(64, 60), (8, 3), (16, 8), (8, 17), (24, 60), (3, 5),
                                           (8, 1), (64, 48), (1, 1)])
def test_projection_work_order_is_a_bijection(ntiles, nheads):
    """Every (token tile, head) unit gets exactly one work-group; with 8 | ntiles,
    XCD k (work-groups x = k mod 8) runs only tiles = k mod 8, in blocks of
    consecutive work-groups that cover all of its tiles and at most 8 heads."""
    got = [_qkv_tile(x, ntiles, nheads) for x in range(ntiles * nheads)]
    assert sorted(got) == [(t, h) for t in range(ntiles) for h in range(nheads)]
    if ntiles % 8 == 0:
        ntk = ntiles // 8
        for k in range(8):
            seq = [got[x] for x in range(k, ntiles * nheads, 8)]
            assert all(t % 8 == k for t, _ in seq)
            for b0 in range(0, len(seq), 8 * ntk):
                blk = seq[b0:b0 + 8 * ntk]
                assert len({h for _, h in blk}) <= 8
                assert {t for t, _ in blk} == set(range(k, ntiles, 8))
