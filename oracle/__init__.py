"""CPU oracle of TurboAttention (FlashQ + SAS) — TEST INFRASTRUCTURE ONLY.

Only tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It wraps ``turbo_oracle.c`` (plain C,
written from the paper, sharing nothing with the GPU library) with numpy.

Each wrapper names the paper passage its C function follows; the arithmetic
and its readings are documented in ``turbo_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "turbo_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

# -O2 without fast-math and without FMA contraction: every binary32 operation
# of the C source is one IEEE operation.  Generic x86-64 code (no -march).
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
          "-fno-fast-math", "-Wall", "-Wno-unused-function"]


def build(force: bool = True) -> str:
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Opts(ctypes.Structure):
    _fields_ = [("quant", ctypes.c_int), ("sas", ctypes.c_int)]


class Trace(ctypes.Structure):
    _fields_ = [("b", ctypes.c_int), ("h", ctypes.c_int), ("i", ctypes.c_int), ("j", ctypes.c_int),
                ("hit", ctypes.c_int),
                ("q8", ctypes.c_void_p), ("sacc", ctypes.c_void_p), ("qp", ctypes.c_void_p),
                ("pvacc", ctypes.c_void_p), ("sq", ctypes.c_float), ("pmax", ctypes.c_float)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I, F, L, D = ctypes.c_int, ctypes.c_float, ctypes.c_long, ctypes.c_double
        sig = {
            "or_num_threads": ([], I),
            "or_head_priority": ([P, I, I, I, I, P], None),
            "or_int2_heads": ([P, I, I, P], None),
            "or_lut": ([I], F),
            "or_poly": ([F], F),
            "or_sas_y": ([F], F),
            "or_sas": ([F], F),
            "or_sas_y_vec": ([P, L, P], None),
            "or_poly_vec": ([P, L, P], None),
            "or_block_quant_vec": ([P, L, L, P, P], None),
            "or_step2_vec": ([P, I, I, I, P, P, P], None),
            "or_sas_softmax_rows": ([P, I, I, P], None),
            "or_quantize_kv": ([P, P, I, I, I, I, P, P, P, P, P, P, P, P, P, P, P], None),
            "or_attn_prefill": ([P, P, P, I, I, I, I, I, F, I, _Opts, P, P, P, I, I], None),
            "or_attn_prefill_blocks": ([P, P, P, I, I, I, I, I, F, I, _Opts, I, I, P, P, P, I,
                                        I], None),
            "or_quantize_kv_blocks": ([P, P, I, I, I, I, I, P, P, P, P], None),
            "or_tail_init": ([P, P, I, I, I, I, P, P, P, P, P, P], None),
            "or_append_kv": ([P, P, I, I, I, P, P, I, P, P, P, P, P, P, P, P, P, P, P, P], None),
            "or_attn_decode": ([P, P, P, P, P, P, P, P, P, P, I, I, I, I, I, F, I, _Opts, P, P, P,
                                P, P, P, P],
                               None),
            "or_attn_exact": ([P, P, P, I, I, I, I, I, I, D, I, P, P], None),
        }
        for name, (args, res) in sig.items():
            fn = getattr(_lib, name)
            fn.argtypes = args
            fn.restype = res
    return _lib


def _p(a):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _f32(x) -> np.ndarray:
    """fp16 (numpy or torch) -> contiguous float32 numpy (exact)."""
    if hasattr(x, "detach"):
        x = x.detach().cpu().float().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.float32))


def num_threads() -> int:
    return lib().or_num_threads()


# ---- SAS (Sec. 4; Algorithm 3) -------------------------------------------
def lut(k: int) -> float:
    return lib().or_lut(k)


def sas_y(y) -> np.ndarray:
    """SAS of x = -y for y >= 0 (binary32), elementwise."""
    y = np.ascontiguousarray(np.asarray(y, dtype=np.float32))
    out = np.empty_like(y)
    lib().or_sas_y_vec(_p(y), y.size, _p(out))
    return out


def sas(x) -> np.ndarray:
    """SAS(x) in the paper's sign convention (x <= 0)."""
    return sas_y(-np.asarray(x, dtype=np.float32))


def poly(f) -> np.ndarray:
    f = np.ascontiguousarray(np.asarray(f, dtype=np.float32))
    out = np.empty_like(f)
    lib().or_poly_vec(_p(f), f.size, _p(out))
    return out


def sas_softmax_rows(x) -> np.ndarray:
    """Algorithm 3 on the rows of a 2-D array."""
    x = _f32(x)
    out = np.empty(x.shape, dtype=np.float64)
    lib().or_sas_softmax_rows(_p(x), x.shape[0], x.shape[1], _p(out))
    return out


# ---- FlashQ (eq. step1bpq, step2bpq) ---------------------------------------
def block_quant(x) -> tuple:
    """Symmetric int8 of blocks: x [..., n] -> (q int8 [..., n], s float32 [...])."""
    x = _f32(x)
    n = x.shape[-1]
    nblk = x.size // n if n else 0
    q = np.empty(x.shape, dtype=np.int8)
    s = np.empty(x.shape[:-1], dtype=np.float32)
    lib().or_block_quant_vec(_p(x), nblk, n, _p(q), _p(s))
    return q, s


def step2(q1, bits: int) -> tuple:
    """Asymmetric step 2 of groups along axis 0: q1 int8 [n][ncol] ->
    (s uint8 [ncol], z int8 [ncol], code uint8 [n][ncol])."""
    q1 = np.ascontiguousarray(np.asarray(q1, dtype=np.int8))
    n, ncol = q1.shape
    s = np.empty(ncol, np.uint8)
    z = np.empty(ncol, np.int8)
    code = np.empty((n, ncol), np.uint8)
    lib().or_step2_vec(_p(q1), n, ncol, bits, _p(s), _p(z), _p(code))
    return s, z, code


def quantize_kv(k, v, bits) -> dict:
    """FlashQ of K/V [B][Hkv][N][d] (fp16 values) with per-head bits."""
    k, v = _f32(k), _f32(v)
    B, Hkv, N, d = k.shape
    nb, ng = (N + 63) // 64, N // 64
    bits = np.ascontiguousarray(np.asarray(bits, dtype=np.int32))
    out = dict(
        k8=np.empty((B, Hkv, N, d), np.int8), v8=np.empty((B, Hkv, N, d), np.int8),
        sk=np.empty((B, Hkv, nb), np.float32), sv=np.empty((B, Hkv, nb), np.float32),
        kc=np.empty((B, Hkv, ng * 64, d), np.uint8), vc=np.empty((B, Hkv, ng * 64, d), np.uint8),
        ks=np.empty((B, Hkv, ng, d), np.uint8), kz=np.empty((B, Hkv, ng, d), np.int8),
        vs=np.empty((B, Hkv, ng, d), np.uint8), vz=np.empty((B, Hkv, ng, d), np.int8))
    o = out
    lib().or_quantize_kv(_p(k), _p(v), B, Hkv, N, d, _p(bits), _p(o["k8"]), _p(o["v8"]),
                         _p(o["sk"]), _p(o["sv"]), _p(o["kc"]), _p(o["vc"]), _p(o["ks"]),
                         _p(o["kz"]), _p(o["vs"]), _p(o["vz"]))
    out["bits"] = bits
    return out


def quantize_kv_blocks(k, v, block_cols: int) -> dict:
    """FlashQ step 1 of K/V [B][Hkv][N][d] (fp16 values) with blocks of
    block_cols = B_c tokens (Table 3): k8, v8 [B][Hkv][N][d] and sk, sv
    [B][Hkv][ceil(N / B_c)].  No step 2: the cache keeps its 64-token groups."""
    k, v = _f32(k), _f32(v)
    B, Hkv, N, d = k.shape
    assert block_cols in (32, 64, 128)
    nbc = (N + block_cols - 1) // block_cols
    out = dict(k8=np.empty((B, Hkv, N, d), np.int8), v8=np.empty((B, Hkv, N, d), np.int8),
               sk=np.empty((B, Hkv, nbc), np.float32), sv=np.empty((B, Hkv, nbc), np.float32))
    lib().or_quantize_kv_blocks(_p(k), _p(v), B, Hkv, N, d, int(block_cols), _p(out["k8"]),
                                _p(out["v8"]), _p(out["sk"]), _p(out["sv"]))
    return out


def project_exact(x, w):
    """The QKV projection X W^T of fp16 values before any rounding, and
    sum_i |x_i| |w_i| of every output (the scale of its summation error).
    x [..., D], w [F][D]; float64 matmuls (a library primitive), whose own
    error (below D 2^-53 of sum |x||w|) is negligible next to any fp32 sum.
    Returns (y, yabs), float64 [..., F]."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    return x @ w.T, np.abs(x) @ np.abs(w).T


def flashq_of_projection(y, Hq: int, Hkv: int, bits, d: int = 128) -> dict:
    """FlashQ applied to a projection y [B][N][(Hq + 2 Hkv) d] of fp16 values
    (Sec. 5.2 folds the quantization into the projection; Sec. 3.1 steps 1
    and 2): y splits into the query heads, key heads and value heads; Q gets
    the prefill's rule (one int8 block per 64 rows of a head), K and V
    quantize_kv(k, v, bits).  Returns q [B][Hq][N][d], k, v [B][Hkv][N][d]
    (the fp16 values), q8 [B][Hq][N][d], sq [B][Hq][ceil(N/64)] and the
    entries of quantize_kv."""
    y = np.asarray(y, dtype=np.float32)
    B, N, F = y.shape
    y = y.reshape(B, N, Hq + 2 * Hkv, d).transpose(0, 2, 1, 3)
    q = np.ascontiguousarray(y[:, :Hq])
    k = np.ascontiguousarray(y[:, Hq:Hq + Hkv])
    v = np.ascontiguousarray(y[:, Hq + Hkv:])
    nb = (N + 63) // 64
    qp = np.zeros((B, Hq, nb * 64, d), np.float32)
    qp[:, :, :N] = q
    q8, sq = block_quant(qp.reshape(B, Hq, nb, 64 * d))
    out = quantize_kv(k, v, bits)
    out.update(q=q, k=k, v=v, q8=q8.reshape(B, Hq, nb * 64, d)[:, :, :N].copy(), sq=sq)
    return out


def qkv_project(x, w, Hq: int, Hkv: int, bits, d: int = 128) -> dict:
    """The QKV projection followed by FlashQ (Sec. 5.2 folds the quantization
    into this projection; Sec. 3.1 step 1 and step 2).

    x: [B][N][D] hidden states, w: [(Hq + 2 Hkv) d][D] weights (fp16 values;
    query heads, then key heads, then value heads).  Reading: each projection
    output is the exact sum X W^T rounded to fp16 (the precision of the
    unfused path's Q, K, V) before FlashQ.  The sum is a float64 matmul, exact
    for the small-integer test inputs whose partial sums fit in 53 bits.
    Returns flashq_of_projection of that fp16 projection."""
    x = np.asarray(x, dtype=np.float64)
    B, N, D = x.shape
    y, _ = project_exact(x.reshape(B * N, D), w)
    y = y.astype(np.float16).astype(np.float32).reshape(B, N, -1)
    return flashq_of_projection(y, Hq, Hkv, bits, d)


def _trace(d: int, sel, br: int = 64, bc: int = 64):
    if sel is None:
        return None, None
    bufs = dict(q8=np.zeros((br, d), np.int8), sacc=np.zeros((br, bc), np.int32),
                qp=np.zeros((br, bc), np.int8), pvacc=np.zeros((br, d), np.int32))
    b, h, i, j = sel
    tr = Trace(b, h, i, j, 0, _p(bufs["q8"]).value, _p(bufs["sacc"]).value, _p(bufs["qp"]).value,
               _p(bufs["pvacc"]).value, 0.0, 0.0)
    return tr, bufs


def attn_prefill(q, k, v, sm_scale: float, causal: bool = True, quant: bool = True,
                 sas: bool = True, trace=None, qblocks=None, block_rows: int = 64,
                 block_cols: int = 64):
    """Algorithm 1.  q [B][Hq][N][d], k, v [B][Hkv][N][d] (fp16 values).
    Returns (o float64 [B][Hq][N][d] = O/l before fp16 rounding, lse float64
    [B][Hq][N]) and, with trace=(b, h, i, j) (query block i of B_r rows, key
    block j of B_c keys), a dict of that tile's integers.
    qblocks=(i0, i1) restricts the work to query blocks i0..i1-1 (other rows NaN).
    block_rows = B_r, block_cols = B_c (Table 3): the query block of the Q
    scale, the key block of the K/V scales and of each online step, and the
    B_r x B_c tile of the P scale."""
    q, k, v = _f32(q), _f32(k), _f32(v)
    B, Hq, N, d = q.shape
    Hkv = k.shape[1]
    o = np.full((B, Hq, N, d), np.nan, np.float64)
    lse = np.full((B, Hq, N), np.nan, np.float64)
    assert block_rows in (32, 64, 128) and block_cols in (32, 64, 128)
    tr, bufs = _trace(d, trace, block_rows, block_cols)
    i0, i1 = (-1, -1) if qblocks is None else qblocks
    lib().or_attn_prefill_blocks(_p(q), _p(k), _p(v), B, Hq, Hkv, N, d,
                                 float(np.float32(sm_scale)), int(causal),
                                 _Opts(int(quant), int(sas)), int(block_rows), int(block_cols),
                                 _p(o), _p(lse),
                                 ctypes.byref(tr) if tr is not None else None, int(i0), int(i1))
    if tr is None:
        return o, lse
    bufs.update(hit=tr.hit, sq=np.float32(tr.sq), pmax=np.float32(tr.pmax))
    return o, lse, bufs


def attn_decode(q, qkv: dict, seq_lens, sm_scale: float, split: int, quant: bool = True,
                sas: bool = True, trace=None, tail: dict = None):
    """Algorithm 2 (+ split-KV merge).  q [B][Hq][d] fp16 values; qkv is the
    dict of quantize_kv (or empty_cache); seq_lens int [B].  trace=(b, h, group)
    (group ng = seq_len // 64 selects the buffer).  tail: the Sec. 3.3 int8
    buffer of tail_init / append_kv, attended as one more chunk."""
    q = _f32(q)
    B, Hq, d = q.shape
    Hkv = qkv["kc"].shape[1]
    Nc = qkv["kc"].shape[2]
    ng = Nc // 64
    sk = np.ascontiguousarray(qkv["sk"][:, :, :ng])
    sv = np.ascontiguousarray(qkv["sv"][:, :, :ng])
    sl = np.ascontiguousarray(np.asarray(seq_lens, dtype=np.int32))
    o = np.empty((B, Hq, d), np.float64)
    lse = np.empty((B, Hq), np.float64)
    tr, bufs = _trace(d, None if trace is None else (trace[0], trace[1], 0, trace[2]))
    c = {n: np.ascontiguousarray(qkv[n]) for n in ("kc", "vc", "ks", "kz", "vs", "vz")}
    t = {n: None for n in ("tk", "tv", "tsk", "tsv")} if tail is None else tail
    lib().or_attn_decode(_p(q), _p(c["kc"]), _p(c["vc"]), _p(c["ks"]), _p(c["kz"]), _p(c["vs"]),
                         _p(c["vz"]), _p(sk), _p(sv), _p(sl), B, Hq, Hkv, Nc, d,
                         float(np.float32(sm_scale)), int(split), _Opts(int(quant), int(sas)),
                         _p(o), _p(lse), ctypes.byref(tr) if tr is not None else None,
                         _p(t["tk"]), _p(t["tv"]), _p(t["tsk"]), _p(t["tsv"]))
    if tr is None:
        return o, lse
    bufs.update(hit=tr.hit, sq=np.float32(tr.sq), pmax=np.float32(tr.pmax))
    return o, lse, bufs


def attn_exact(q, k, v, sm_scale: float, causal: bool = True):
    """Exact softmax attention in double (eq. stdattn).  q [B][Hq][Nq][d],
    k, v [B][Hkv][Nk][d]; query r sits at position r + Nk - Nq."""
    q, k, v = _f32(q), _f32(k), _f32(v)
    B, Hq, Nq, d = q.shape
    Hkv, Nk = k.shape[1], k.shape[2]
    o = np.empty((B, Hq, Nq, d), np.float64)
    lse = np.empty((B, Hq, Nq), np.float64)
    lib().or_attn_exact(_p(q), _p(k), _p(v), B, Hq, Hkv, Nq, Nk, d, float(sm_scale), int(causal),
                        _p(o), _p(lse))
    return o, lse


def head_priority(k):
    """Sec. 3.2 priority gap x std of each KV head; k [B][Hkv][N][d] (fp16
    values).  Returns float64 [Hkv]."""
    k = _f32(k)
    B, Hkv, N, d = k.shape
    out = np.empty(Hkv, np.float64)
    lib().or_head_priority(_p(k), B, Hkv, N, d, _p(out))
    return out


def int2_heads(prio, n_int2: int):
    """Sec. 3.2 strategy: uint8 [Hkv] of 2 for the n_int2 lowest priorities
    (ties by head index), 4 otherwise."""
    p = np.ascontiguousarray(np.asarray(prio, dtype=np.float64))
    bits = np.empty(p.size, np.uint8)
    lib().or_int2_heads(_p(p), p.size, int(n_int2), _p(bits))
    return bits


def empty_cache(B: int, Hkv: int, Nc: int, d: int = 128, bits=None) -> dict:
    """A compressed cache of capacity Nc tokens (Nc/64 groups) in the layout of
    quantize_kv, all zero; sk, sv [B][Hkv][Nc/64]."""
    ng = Nc // 64
    return dict(kc=np.zeros((B, Hkv, Nc, d), np.uint8), vc=np.zeros((B, Hkv, Nc, d), np.uint8),
                ks=np.zeros((B, Hkv, ng, d), np.uint8), kz=np.zeros((B, Hkv, ng, d), np.int8),
                vs=np.zeros((B, Hkv, ng, d), np.uint8), vz=np.zeros((B, Hkv, ng, d), np.int8),
                sk=np.zeros((B, Hkv, ng), np.float32), sv=np.zeros((B, Hkv, ng), np.float32),
                bits=np.ascontiguousarray(np.asarray(bits if bits is not None else [4] * Hkv,
                                                     dtype=np.int32)))


def cache_from_prefill(qkv: dict, Nc: int) -> dict:
    """The groups of quantize_kv placed in an empty cache of capacity Nc."""
    B, Hkv, _, d = qkv["k8"].shape
    c = empty_cache(B, Hkv, Nc, d, qkv["bits"])
    n = qkv["kc"].shape[2]
    ng = n // 64
    for key in ("kc", "vc"):
        c[key][:, :, :n] = qkv[key]
    for key in ("ks", "kz", "vs", "vz"):
        c[key][:, :, :ng] = qkv[key]
    c["sk"][:, :, :ng] = qkv["sk"][:, :, :ng]
    c["sv"][:, :, :ng] = qkv["sv"][:, :, :ng]
    return c


def tail_init(k, v, qkv: dict) -> dict:
    """Sec. 3.3 buffer after a prefill: universal scales (largest block scale
    of each (b, kv-head)) and the N mod 64 trailing tokens as int8.
    Returns dict tk [B][Hkv][64][d], tv [B][Hkv][d][64], tsk, tsv [B][Hkv]."""
    k, v = _f32(k), _f32(v)
    B, Hkv, N, d = k.shape
    t = dict(tk=np.zeros((B, Hkv, 64, d), np.int8), tv=np.zeros((B, Hkv, d, 64), np.int8),
             tsk=np.zeros((B, Hkv), np.float32), tsv=np.zeros((B, Hkv), np.float32))
    sk, sv = np.ascontiguousarray(qkv["sk"]), np.ascontiguousarray(qkv["sv"])
    lib().or_tail_init(_p(k), _p(v), B, Hkv, N, d, _p(sk), _p(sv), _p(t["tk"]), _p(t["tv"]),
                       _p(t["tsk"]), _p(t["tsv"]))
    return t


def append_kv(cache: dict, tail: dict, knew, vnew, seq_lens):
    """Sec. 3.3 decoding step: the new key/value [B][Hkv][d] of each sequence
    into its buffer at row seq_len % 64; a full buffer is compressed (step 2)
    into group seq_len // 64 of `cache` (from empty_cache / cache_from_prefill).
    Updates cache and tail in place; seq_lens are the lengths before the step."""
    knew, vnew = _f32(knew), _f32(vnew)
    B, Hkv, d = knew.shape
    Nc = cache["kc"].shape[2]
    sl = np.ascontiguousarray(np.asarray(seq_lens, dtype=np.int32))
    c = cache
    lib().or_append_kv(_p(knew), _p(vnew), B, Hkv, d, _p(sl), _p(c["bits"]), Nc, _p(c["kc"]),
                       _p(c["vc"]), _p(c["ks"]), _p(c["kz"]), _p(c["vs"]), _p(c["vz"]),
                       _p(c["sk"]), _p(c["sv"]), _p(tail["tk"]), _p(tail["tv"]), _p(tail["tsk"]),
                       _p(tail["tsv"]))

