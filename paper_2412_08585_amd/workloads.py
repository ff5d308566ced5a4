"""Seeded synthetic workloads for the TurboAttention hot path.

This module only draws inputs; it holds none of the method's arithmetic, so the
oracle tests and the HIP path can both take their inputs from it.

The paper measures on Phi3-medium attention shapes with contexts of 1k-32k
tokens (Sec. 5.3) and motivates FlashQ's channel-wise step by outlier channels
in Q and K (Sec. 3.2, Fig. 3).  No model weights or datasets are used here:
activations are stood in for by N(0,1) fp16 tensors in which four channels of
K per (sequence, KV head) are scaled by 10.

Recipe (per unit = one sequence b and one KV head h of a named workload):
  * a torch.Generator on the requested device, seeded with
    seed_of(workload_id, b, h, stream) (stream 0 = prefill Q/K/V, 1 = decode
    query);
  * draws in this order: the 4 outlier channels (randperm(128)[:4]), K, V
    ~ N(0,1) fp32 [N][128], the G query heads ~ N(0,1) fp32 [G][N][128];
  * K[:, outliers] *= 10, then round-to-nearest-even to fp16.
A CPU generator and a CUDA generator give different (equally valid) values
for the same seed; every test compares both sides on one draw.

Head bit widths (Sec. 3.2, Sec. 5.2: half of the heads at 2 bits): for the
"mixed" workloads each KV head gets a priority u ~ U(0,1) from seed
seed_of(workload_id, 0, 0, 2); the Hkv/2 lowest priorities (ties to the lower
index) are stored with 2 bits, the others with 4.

Block/group tables: physical pages and group slots are a seeded random
permutation (seed_of(workload_id, 0, 0, 3)), so that logically adjacent
pages are not adjacent in memory.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np
import torch

HEAD_DIM = 128
BLOCK = 64
PAGE_TOKENS = 16
N_OUTLIER = 4
OUTLIER_GAIN = 10.0


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    wid: int          # numeric id used in seeds
    kind: str         # "prefill" or "decode"
    B: int
    Hq: int
    Hkv: int
    N: int            # sequence length (prefill) or cached KV length (decode)
    bits: str         # "int4" or "mixed"
    causal: bool = True
    hidden: int = 0   # model width D of the QKV projection (projection workloads)

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def sm_scale(self) -> float:
        return 1.0 / float(np.sqrt(HEAD_DIM))

    @property
    def max_groups(self) -> int:
        return (self.N + BLOCK - 1) // BLOCK

    def scaled(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads of the build: a tiny causal prefill, a Phi-3-medium-shaped
# prefill, a Phi-3-medium-shaped decode with mixed int4/int2 heads, a
# Llama-3-8B-shaped 16k prefill and a long-context batched decode.
WORKLOADS = {
    "tiny-prefill": Workload("tiny-prefill", 0, "prefill", 1, 4, 4, 512, "int4"),
    "phi3m-prefill-4k": Workload("phi3m-prefill-4k", 1, "prefill", 4, 40, 10, 4096, "int4"),
    "phi3m-decode-8k": Workload("phi3m-decode-8k", 2, "decode", 64, 40, 10, 8192, "mixed"),
    "llama3-8b-prefill-16k": Workload("llama3-8b-prefill-16k", 3, "prefill", 1, 32, 8, 16384, "int4"),
    "long-decode-32k": Workload("long-decode-32k", 4, "decode", 256, 32, 8, 32768, "int4"),
    # Algorithm 3 on its own: the score rows of one Phi-3-medium-shaped
    # sequence (40 query heads x 4096 queries, 4096 keys each).
    "phi3m-sas-softmax-4k": Workload("phi3m-sas-softmax-4k", 5, "softmax", 1, 40, 10, 4096, "int4"),
    # The QKV projection with FlashQ fused (Sec. 5.2) for the Phi-3-medium
    # prefill: hidden width 5120 -> 40 query + 10 key + 10 value heads.
    "phi3m-qkv-4k": Workload("phi3m-qkv-4k", 6, "projection", 4, 40, 10, 4096, "int4",
                             hidden=5120),
}

# Standard deviation of the score stand-in: q.k / sqrt(128) for N(0,1) q and
# k with 4 of 128 channels of k scaled by 10 has variance (124 + 4*100)/128.
SCORE_STD = float(np.sqrt((HEAD_DIM - N_OUTLIER + N_OUTLIER * OUTLIER_GAIN ** 2) / HEAD_DIM))


def seed_of(wid: int, b: int, h: int, stream: int) -> int:
    return ((wid * 65536 + b) * 1024 + h) * 8 + stream + 0x5EED


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def unit_qkv(w: Workload, b: int, h: int, device="cpu", N: Optional[int] = None,
             outliers: bool = True):
    """fp16 (q [G][N][128], k [N][128], v [N][128]) for sequence b, KV head h."""
    N = w.N if N is None else N
    g = _gen(device, seed_of(w.wid, b, h, 0))
    ch = torch.randperm(HEAD_DIM, generator=g, device=device)[:N_OUTLIER]
    k = torch.randn(N, HEAD_DIM, generator=g, device=device, dtype=torch.float32)
    v = torch.randn(N, HEAD_DIM, generator=g, device=device, dtype=torch.float32)
    q = torch.randn(w.G, N, HEAD_DIM, generator=g, device=device, dtype=torch.float32)
    if outliers:
        k[:, ch] *= OUTLIER_GAIN
    return q.half(), k.half(), v.half()


def unit_kv(w: Workload, b: int, h: int, device="cpu", N: Optional[int] = None,
            outliers: bool = True):
    """fp16 (k [N][128], v [N][128]) of sequence b, KV head h: the same draws
    as unit_qkv (K and V come before Q in the stream)."""
    N = w.N if N is None else N
    g = _gen(device, seed_of(w.wid, b, h, 0))
    ch = torch.randperm(HEAD_DIM, generator=g, device=device)[:N_OUTLIER]
    k = torch.randn(N, HEAD_DIM, generator=g, device=device, dtype=torch.float32)
    v = torch.randn(N, HEAD_DIM, generator=g, device=device, dtype=torch.float32)
    if outliers:
        k[:, ch] *= OUTLIER_GAIN
    return k.half(), v.half()


def prefill_inputs(w: Workload, device="cpu", N: Optional[int] = None, B: Optional[int] = None):
    """fp16 Q [B][Hq][N][128], K, V [B][Hkv][N][128] built unit by unit."""
    N = w.N if N is None else N
    B = w.B if B is None else B
    q = torch.empty(B, w.Hq, N, HEAD_DIM, dtype=torch.float16, device=device)
    k = torch.empty(B, w.Hkv, N, HEAD_DIM, dtype=torch.float16, device=device)
    v = torch.empty_like(k)
    for b in range(B):
        for h in range(w.Hkv):
            qu, ku, vu = unit_qkv(w, b, h, device, N)
            q[b, h * w.G:(h + 1) * w.G] = qu
            k[b, h] = ku
            v[b, h] = vu
    return q, k, v


def decode_query(w: Workload, device="cpu", B: Optional[int] = None):
    """fp16 q [B][Hq][128] ~ N(0,1), one seed per (b, KV head)."""
    B = w.B if B is None else B
    q = torch.empty(B, w.Hq, HEAD_DIM, dtype=torch.float16, device=device)
    for b in range(B):
        for h in range(w.Hkv):
            g = _gen(device, seed_of(w.wid, b, h, 1))
            q[b, h * w.G:(h + 1) * w.G] = torch.randn(
                w.G, HEAD_DIM, generator=g, device=device, dtype=torch.float32).half()
    return q


def head_bits(w: Workload, Hkv: Optional[int] = None) -> np.ndarray:
    """uint8 [Hkv] of 4/2: all 4 for "int4"; for "mixed" the lowest-priority half gets 2."""
    Hkv = w.Hkv if Hkv is None else Hkv
    bits = np.full(Hkv, 4, dtype=np.uint8)
    if w.bits == "mixed":
        rng = np.random.default_rng(seed_of(w.wid, 0, 0, 2))
        prio = rng.random(Hkv)
        order = sorted(range(Hkv), key=lambda i: (prio[i], i))
        for i in order[: Hkv // 2]:
            bits[i] = 2
    return bits


def tables(w: Workload, B: Optional[int] = None, max_groups: Optional[int] = None):
    """int32 block_table [B][4*max_groups] and group_table [B][max_groups] as seeded
    random permutations of page ids 0..B*4*max_groups-1 and slot ids 0..B*max_groups-1."""
    B = w.B if B is None else B
    mg = w.max_groups if max_groups is None else max_groups
    rng = np.random.default_rng(seed_of(w.wid, 0, 0, 3))
    pages = rng.permutation(B * 4 * mg).astype(np.int32).reshape(B, 4 * mg)
    slots = rng.permutation(B * mg).astype(np.int32).reshape(B, mg)
    return pages, slots


def softmax_scores(w: Workload, device="cpu", rows: Optional[int] = None, row0: int = 0):
    """fp32 score rows [rows][N] for Algorithm 3: N(0, SCORE_STD^2), drawn in
    blocks of 1024 rows, block i from seed_of(workload_id, i, 0, 4), so that
    any block can be drawn alone (row0 must be a multiple of 1024)."""
    total = w.B * w.Hq * w.N
    rows = total - row0 if rows is None else rows
    assert row0 % 1024 == 0 and row0 + rows <= total
    out = torch.empty(rows, w.N, dtype=torch.float32, device=device)
    for r in range(0, rows, 1024):
        n = min(1024, rows - r)
        g = _gen(device, seed_of(w.wid, (row0 + r) // 1024, 0, 4))
        out[r:r + n] = torch.randn(n, w.N, generator=g, device=device) * SCORE_STD
    return out


def projection_inputs(w: Workload, device="cpu"):
    """fp16 hidden states X [B][N][D] ~ N(0,1) and weights W [(Hq+2Hkv)128][D]
    ~ N(0, 1/D), with 4 channels of every key head scaled by 10 (the outlier
    channels of Fig. 3 come from the projection); X from seed_of(wid, b, 0, 5)
    per sequence, W from seed_of(wid, 0, 0, 6)."""
    D = w.hidden
    F = (w.Hq + 2 * w.Hkv) * HEAD_DIM
    x = torch.empty(w.B, w.N, D, dtype=torch.float16, device=device)
    for b in range(w.B):
        g = _gen(device, seed_of(w.wid, b, 0, 5))
        x[b] = torch.randn(w.N, D, generator=g, device=device).half()
    g = _gen(device, seed_of(w.wid, 0, 0, 6))
    wt = torch.randn(F, D, generator=g, device=device) / float(np.sqrt(D))
    for h in range(w.Hkv):
        ch = torch.randperm(HEAD_DIM, generator=g, device=device)[:N_OUTLIER]
        wt[(w.Hq + h) * HEAD_DIM + ch] *= OUTLIER_GAIN
    return x, wt.half()
