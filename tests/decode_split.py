"""Chunking of the decode's split-KV extension, restated for the tests.

With kv_split_groups = 0 the decode cuts each sequence by its own group count
(the rule the C ABI documents for turbo_decode_default_split): one chunk up to
32 groups, chunks of 32 groups up to 128 groups, four equal chunks beyond.
The oracle takes one chunk length per call, so a batch whose sequences get
different lengths is run once per distinct length.
"""
import numpy as np


def default_split(ng: int) -> int:
    if ng <= 32:
        return max(ng, 1)
    if ng <= 128:
        return 32
    return (ng + 3) // 4


def split_of(seq_len: int, split: int, max_groups: int = None) -> int:
    ng = seq_len // 64
    if max_groups is not None:
        ng = min(ng, max_groups)
    return split if split > 0 else default_split(max(ng, 0))


def oracle_decode(orc, q, cache, seq, sm, split, max_groups=None, **kw):
    """orc.attn_decode with the chunk length the decode uses for each sequence
    (split > 0: that length for all).  Returns (o, lse) like the oracle."""
    used = [split_of(s, split, max_groups) for s in seq]
    o = lse = None
    for u in sorted(set(used)):
        ro, rl = orc.attn_decode(q, cache, seq, sm, split=u, **kw)
        if o is None:
            o, lse = np.empty_like(ro), np.empty_like(rl)
        for b, ub in enumerate(used):
            if ub == u:
                o[b], lse[b] = ro[b], rl[b]
    return o, lse
