"""Test-side reader/writer of the paged cache format documented in
include/turbo_attn.h (turbo_kv_cache).  Test infrastructure only: it lets the
tests turn the GPU's pages back into logical step-2 codes, and build pages
from logical codes for host-side round trips."""
import numpy as np

D = 128


def head_offsets(head_bits):
    hb = np.asarray(head_bits, dtype=np.int64)
    off = np.concatenate([[0], np.cumsum(512 * hb)[:-1]])
    return off, int((512 * hb).sum())


def _unpack_bits(byts: np.ndarray, bits: int) -> np.ndarray:
    """uint8 [..., n] -> codes [..., n*8/bits], little-endian within a byte."""
    per = 8 // bits
    mask = (1 << bits) - 1
    out = np.stack([(byts >> (bits * i)) & mask for i in range(per)], axis=-1)
    return out.reshape(*byts.shape[:-1], byts.shape[-1] * per).astype(np.uint8)


def _pack_bits(codes: np.ndarray, bits: int) -> np.ndarray:
    per = 8 // bits
    c = codes.reshape(*codes.shape[:-1], codes.shape[-1] // per, per).astype(np.uint16)
    out = np.zeros(c.shape[:-1], np.uint16)
    for i in range(per):
        out |= c[..., i] << (bits * i)
    return out.astype(np.uint8)


def read_unit(pages, gmeta, gscale, head_bits, block_table, group_table, b, h, ng):
    """Logical cache of sequence b, KV head h, groups 0..ng-1:
    kc, vc uint8 [ng*64][128]; ks, vs uint8 [ng][128]; kz, vz int8 [ng][128];
    sk, sv float32 [ng]."""
    off, pb = head_offsets(head_bits)
    bits = int(head_bits[h])
    assert pages.shape[1] == pb
    kc = np.zeros((ng * 64, D), np.uint8)
    vc = np.zeros((ng * 64, D), np.uint8)
    for g in range(ng):
        for p in range(4):
            page = pages[block_table[b, 4 * g + p]]
            reg = page[off[h]: off[h] + 512 * bits]
            kbytes = reg[: 256 * bits].reshape(16, 16 * bits)          # token-major
            vbytes = reg[256 * bits:].reshape(D, 2 * bits)             # channel-major
            t0 = 64 * g + 16 * p
            kc[t0:t0 + 16] = _unpack_bits(kbytes, bits)
            vc[t0:t0 + 16] = _unpack_bits(vbytes, bits).T
    slots = group_table[b, :ng]
    meta = gmeta[slots, h]                       # [ng][4][128] int8
    sc = gscale[slots, h]                        # [ng][2]
    return dict(kc=kc, vc=vc, ks=meta[:, 0].view(np.uint8), kz=meta[:, 1],
                vs=meta[:, 2].view(np.uint8), vz=meta[:, 3], sk=sc[:, 0], sv=sc[:, 1])


def write_unit(pages, gmeta, gscale, head_bits, block_table, group_table, b, h, unit):
    """Inverse of read_unit (host-side packing of logical codes)."""
    off, pb = head_offsets(head_bits)
    bits = int(head_bits[h])
    ng = unit["kc"].shape[0] // 64
    for g in range(ng):
        for p in range(4):
            t0 = 64 * g + 16 * p
            page = pages[block_table[b, 4 * g + p]]
            page[off[h]: off[h] + 256 * bits] = _pack_bits(unit["kc"][t0:t0 + 16], bits).ravel()
            page[off[h] + 256 * bits: off[h] + 512 * bits] = \
                _pack_bits(np.ascontiguousarray(unit["vc"][t0:t0 + 16].T), bits).ravel()
        s = group_table[b, g]
        gmeta[s, h, 0] = unit["ks"][g].view(np.int8)
        gmeta[s, h, 1] = unit["kz"][g]
        gmeta[s, h, 2] = unit["vs"][g].view(np.int8)
        gmeta[s, h, 3] = unit["vz"][g]
        gscale[s, h, 0] = unit["sk"][g]
        gscale[s, h, 1] = unit["sv"][g]
