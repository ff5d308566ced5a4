"""Thin Python binding of libturboattn.so (argument marshalling only).

The functions carry the C ABI's names and forward torch tensors as raw device
pointers together with torch's current HIP stream.  Every computation runs in
the library's gfx950 kernels; if the library is missing or the device is not
gfx950 the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch

HEAD_DIM = 128
BLOCK = 64
PAGE_TOKENS = 16
MAX_KV_HEADS = 64
# tile trace layout of the *_trace test hooks (include/turbo_attn.h)
TRACE_Q8, TRACE_S, TRACE_P, TRACE_PV, TRACE_SQ, TRACE_PMAX, TRACE_BYTES = (
    0, 16384, 81920, 98304, 163840, 163844, 163848)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libturboattn.so")


class TurboKVCacheStruct(ctypes.Structure):
    """Mirror of turbo_kv_cache (include/turbo_attn.h)."""
    _fields_ = [("pages", ctypes.c_void_p), ("group_meta", ctypes.c_void_p),
                ("group_scale", ctypes.c_void_p), ("num_pages", ctypes.c_int64),
                ("num_group_slots", ctypes.c_int64), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("head_bits", ctypes.c_uint8 * MAX_KV_HEADS)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load the in-tree HIP library; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2412_08585_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I, F, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
        sig = {
            "turbo_abi_version": ([], I),
            "turbo_strerror": ([I], ctypes.c_char_p),
            "turbo_page_bytes": ([P, I], Z),
            "turbo_quantize_kv": ([P, P, I, I, I, I, P, P, P, P, P, P, P, I, P], I),
            "turbo_attn_prefill": ([P, P, P, P, P, I, I, I, I, I, F, I, P, P, P], I),
            "turbo_attn_decode": ([P, P, P, P, P, P, I, I, I, F, I, P, Z, P, P, P], I),
            "turbo_attn_decode_noalloc": ([P, P, P, P, P, P, I, I, I, F, I, P, P, P], I),
            "turbo_attn_prefill_trace": ([P, P, P, P, P, I, I, I, I, I, F, I, P, P, I, I, I, I, P,
                                          P], I),
            "turbo_attn_prefill_blocks_trace": ([P, P, P, P, P, I, I, I, I, I, F, I, I, I, P, P, I,
                                                 I, I, I, P, P], I),
            "turbo_attn_decode_trace": ([P, P, P, P, P, P, I, I, I, F, I, P, Z, P, P, I, I, I, P,
                                         P], I),
            "turbo_tail_init": ([P, P, I, I, I, I, P, P, P, P], I),
            "turbo_append_kv": ([P, P, I, I, I, P, P, P, P, P, I, P], I),
            "turbo_head_priority": ([P, I, I, I, I, P, Z, P, P], I),
            "turbo_head_priority_workspace_bytes": ([I, I, I], Z),
            "turbo_int2_heads": ([P, I, I, P], I),
            "turbo_sas_softmax": ([P, P, ctypes.c_int64, I, P], I),
            "turbo_attn_prefill_q8": ([P, P, P, P, P, P, I, I, I, I, I, F, I, P, P, P], I),
            "turbo_attn_prefill_blocks": ([P, P, P, P, P, I, I, I, I, I, F, I, I, I, P, P, P],
                                          I),
            "turbo_quantize_kv_blocks": ([P, P, I, I, I, I, I, P, P, P, P, P], I),
            "turbo_qkv_project": ([P, P, I, I, I, I, I, I, P, P, P, P, P, P, P, P, P, I, P], I),
            "turbo_qkv_project_trace": ([P, P, I, I, I, I, I, I, P, P, P, P, P, P, P, P, P, I, P,
                                         P], I),
            "turbo_decode_auto_split": ([I, I, I, I], I),
            "turbo_decode_default_split": ([I], I),
            "turbo_probe_mfma_i8": ([I, P, P, P], I),
            "turbo_probe_read": ([P, Z, P, P], I),
            "turbo_probe_valu": ([I, P, P, P], I),
            "turbo_decode_workspace_bytes": ([I, I, I, I, I, I], Z),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check(status: int, what: str):
    if status != 0:
        msg = lib().turbo_strerror(status).decode()
        raise RuntimeError(f"{what} failed: {msg} ({status})")


def page_bytes(head_bits) -> int:
    hb = np.ascontiguousarray(np.asarray(head_bits, dtype=np.uint8))
    return int(lib().turbo_page_bytes(hb.ctypes.data_as(ctypes.c_void_p), hb.size))


class PagedKVCache:
    """Device storage of the compressed cache (pages, group metadata, group
    scales) plus the host copy of the per-head bit widths."""

    def __init__(self, num_pages: int, num_group_slots: int, head_bits, device="cuda"):
        self.head_bits = np.ascontiguousarray(np.asarray(head_bits, dtype=np.uint8))
        self.num_kv_heads = int(self.head_bits.size)
        self.page_bytes = page_bytes(self.head_bits)
        if self.page_bytes == 0:
            raise ValueError("head_bits must hold 1..64 entries of 2 or 4")
        self.pages = torch.zeros(num_pages, self.page_bytes, dtype=torch.uint8, device=device)
        self.group_meta = torch.zeros(num_group_slots, self.num_kv_heads, 4, HEAD_DIM,
                                      dtype=torch.int8, device=device)
        self.group_scale = torch.zeros(num_group_slots, self.num_kv_heads, 2,
                                       dtype=torch.float32, device=device)

    def struct(self) -> TurboKVCacheStruct:
        s = TurboKVCacheStruct()
        s.pages = self.pages.data_ptr()
        s.group_meta = self.group_meta.data_ptr()
        s.group_scale = self.group_scale.data_ptr()
        s.num_pages = self.pages.shape[0]
        s.num_group_slots = self.group_meta.shape[0]
        s.num_kv_heads = self.num_kv_heads
        s.head_dim = HEAD_DIM
        for i, b in enumerate(self.head_bits):
            s.head_bits[i] = int(b)
        return s


class TurboKVTailStruct(ctypes.Structure):
    """Mirror of turbo_kv_tail (include/turbo_attn.h)."""
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("scale", ctypes.c_void_p),
                ("batch", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32)]


class KVTail:
    """Device storage of the Sec. 3.3 int8 buffer: k [batch][Hkv][64][128]
    (token-major), v [batch][Hkv][128][64] (channel-major), universal scales
    [batch][Hkv][2]."""

    def __init__(self, batch: int, num_kv_heads: int, device="cuda"):
        self.batch, self.num_kv_heads = batch, num_kv_heads
        self.k = torch.zeros(batch, num_kv_heads, BLOCK, HEAD_DIM, dtype=torch.int8, device=device)
        self.v = torch.zeros(batch, num_kv_heads, HEAD_DIM, BLOCK, dtype=torch.int8, device=device)
        self.scale = torch.zeros(batch, num_kv_heads, 2, dtype=torch.float32, device=device)

    def struct(self) -> TurboKVTailStruct:
        s = TurboKVTailStruct()
        s.k, s.v, s.scale = self.k.data_ptr(), self.v.data_ptr(), self.scale.data_ptr()
        s.batch, s.num_kv_heads = self.batch, self.num_kv_heads
        return s

    def narrow(self, b0: int, n: int) -> "KVTail":
        """The buffers of sequences b0 .. b0+n-1 (a view sharing the storage)."""
        if not (0 <= b0 and n >= 1 and b0 + n <= self.batch):
            raise ValueError("sequence range outside the buffer")
        t = KVTail.__new__(KVTail)
        t.batch, t.num_kv_heads = n, self.num_kv_heads
        t.k, t.v, t.scale = self.k[b0:b0 + n], self.v[b0:b0 + n], self.scale[b0:b0 + n]
        return t


def turbo_tail_init(k: torch.Tensor, v: torch.Tensor, s_k, s_v, tail: KVTail):
    """Sec. 3.3 buffer after a prefill of k, v fp16 [B][Hkv][N][128] with the
    block scales s_k, s_v of turbo_quantize_kv."""
    B, Hkv, N, d = k.shape
    ts = tail.struct()
    _check(lib().turbo_tail_init(_ptr(k), _ptr(v), B, Hkv, N, d, _ptr(s_k), _ptr(s_v),
                                 ctypes.byref(ts), _stream(k.device)), "turbo_tail_init")


def turbo_append_kv(k_new: torch.Tensor, v_new: torch.Tensor, seq_lens: torch.Tensor,
                    cache: PagedKVCache, tail: KVTail, block_table: torch.Tensor,
                    group_table: torch.Tensor):
    """Sec. 3.3 decoding step: k_new, v_new fp16 [B][Hkv][128] at positions
    seq_lens (lengths before the step, device int32 [B])."""
    B, Hkv, d = k_new.shape
    cs, ts = cache.struct(), tail.struct()
    _check(lib().turbo_append_kv(_ptr(k_new), _ptr(v_new), B, Hkv, d, _ptr(seq_lens),
                                 ctypes.byref(cs), ctypes.byref(ts), _ptr(block_table),
                                 _ptr(group_table), group_table.shape[1], _stream(k_new.device)),
           "turbo_append_kv")


def turbo_quantize_kv(k: torch.Tensor, v: torch.Tensor, cache: Optional[PagedKVCache] = None,
                      block_table: Optional[torch.Tensor] = None,
                      group_table: Optional[torch.Tensor] = None, out=None,
                      block_cols: int = 64):
    """FlashQ of K, V fp16 [B][Hkv][N][128].  Returns (k8, v8, s_k, s_v) in the
    layouts of include/turbo_attn.h; writes the full groups into `cache`.
    block_cols = B_c in {32, 64, 128} (Table 3): the step-1 block of K and V
    (s_k, s_v [B][Hkv][ceil(N / B_c)]); the cache needs B_c = 64."""
    B, Hkv, N, d = k.shape
    nb = (N + BLOCK - 1) // BLOCK
    nbc = (N + block_cols - 1) // block_cols
    dev = k.device
    if out is None:
        k8 = torch.empty(B, Hkv, nb * BLOCK, d, dtype=torch.int8, device=dev)
        v8 = torch.empty(B, Hkv, nb, d, BLOCK, dtype=torch.int8, device=dev)
        s_k = torch.empty(B, Hkv, nbc, dtype=torch.float32, device=dev)
        s_v = torch.empty(B, Hkv, nbc, dtype=torch.float32, device=dev)
    else:
        k8, v8, s_k, s_v = out
    if block_cols != BLOCK:
        if cache is not None:
            raise ValueError("the cache is written with 64-token blocks only")
        st = lib().turbo_quantize_kv_blocks(_ptr(k), _ptr(v), B, Hkv, N, d, int(block_cols),
                                            _ptr(k8), _ptr(v8), _ptr(s_k), _ptr(s_v),
                                            _stream(dev))
        _check(st, "turbo_quantize_kv_blocks")
        return k8, v8, s_k, s_v
    cs = cache.struct() if cache is not None else None
    mg = group_table.shape[1] if group_table is not None else 0
    st = lib().turbo_quantize_kv(_ptr(k), _ptr(v), B, Hkv, N, d, _ptr(k8), _ptr(v8), _ptr(s_k),
                                 _ptr(s_v), ctypes.byref(cs) if cs is not None else None,
                                 _ptr(block_table), _ptr(group_table), mg, _stream(dev))
    _check(st, "turbo_quantize_kv")
    return k8, v8, s_k, s_v


def turbo_attn_prefill(q: torch.Tensor, k8, v8, s_k, s_v, sm_scale: Optional[float] = None,
                       causal: bool = True, return_lse: bool = False, out=None,
                       block_rows: int = 64, block_cols: int = 64):
    """Algorithm 1 prefill.  q fp16 [B][Hq][N][128]; k8/v8/s_k/s_v from
    turbo_quantize_kv (with the same block_cols).  Returns o fp16
    [B][Hq][N][128] (and lse fp32).  block_rows = B_r, block_cols = B_c in
    {32, 64, 128} (Table 3); (64, 64) is the default path."""
    B, Hq, N, d = q.shape
    Hkv = s_k.shape[1]
    sm = float(1.0 / np.sqrt(d)) if sm_scale is None else float(sm_scale)
    o = torch.empty_like(q) if out is None else out
    lse = torch.empty(B, Hq, N, dtype=torch.float32, device=q.device) if return_lse else None
    if s_k.shape[-1] != (N + block_cols - 1) // block_cols:
        raise ValueError(f"s_k holds {s_k.shape[-1]} blocks, not those of B_c = {block_cols}")
    if block_rows == 64 and block_cols == 64:
        st = lib().turbo_attn_prefill(_ptr(q), _ptr(k8), _ptr(v8), _ptr(s_k), _ptr(s_v), B, Hq,
                                      Hkv, N, d, sm, int(bool(causal)), _ptr(o), _ptr(lse),
                                      _stream(q.device))
    else:
        st = lib().turbo_attn_prefill_blocks(_ptr(q), _ptr(k8), _ptr(v8), _ptr(s_k), _ptr(s_v), B,
                                             Hq, Hkv, N, d, sm, int(bool(causal)),
                                             int(block_rows), int(block_cols), _ptr(o),
                                             _ptr(lse), _stream(q.device))
    _check(st, "turbo_attn_prefill")
    return (o, lse) if return_lse else o


def _trace_buffer(device) -> torch.Tensor:
    return torch.zeros(TRACE_BYTES, dtype=torch.uint8, device=device)


def _trace_dict(buf: torch.Tensor, br: int = 64, bc: int = 64) -> dict:
    """The trace of a B_r x B_c tile (layout TURBO_TRACE_* of the header)."""
    h = buf.cpu().numpy()
    return dict(q8=h[TRACE_Q8:TRACE_Q8 + br * HEAD_DIM].view(np.int8).reshape(br, HEAD_DIM).copy(),
                sacc=h[TRACE_S:TRACE_S + 4 * br * bc].view(np.int32).reshape(br, bc).copy(),
                qp=h[TRACE_P:TRACE_P + br * bc].view(np.int8).reshape(br, bc).copy(),
                pvacc=h[TRACE_PV:TRACE_PV + 4 * br * HEAD_DIM].view(np.int32)
                .reshape(br, HEAD_DIM).copy(),
                sq=h[TRACE_SQ:TRACE_PMAX].view(np.float32)[0],
                pmax=h[TRACE_PMAX:TRACE_BYTES].view(np.float32)[0])


def turbo_attn_prefill_trace(q: torch.Tensor, k8, v8, s_k, s_v, tile, sm_scale=None,
                             causal: bool = True, block_rows: int = 64, block_cols: int = 64):
    """Test hook: turbo_attn_prefill (turbo_attn_prefill_blocks for other
    block sizes) that also returns the integers of tile (b, h, i, j) -- query
    block i of block_rows rows, key block j of block_cols keys -- as a dict of
    numpy arrays (q8, sacc, qp, pvacc, sq, pmax)."""
    B, Hq, N, d = q.shape
    Hkv = s_k.shape[1]
    sm = float(1.0 / np.sqrt(d)) if sm_scale is None else float(sm_scale)
    o = torch.empty_like(q)
    buf = _trace_buffer(q.device)
    b, h, i, j = tile
    st = lib().turbo_attn_prefill_blocks_trace(_ptr(q), _ptr(k8), _ptr(v8), _ptr(s_k), _ptr(s_v),
                                               B, Hq, Hkv, N, d, sm, int(bool(causal)),
                                               int(block_rows), int(block_cols), _ptr(o), None,
                                               b, h, i, j, _ptr(buf), _stream(q.device))
    _check(st, "turbo_attn_prefill_blocks_trace")
    torch.cuda.synchronize(q.device)
    return o, _trace_dict(buf, block_rows, block_cols)


def decode_split(seq_len: int, kv_split_groups: int = 0) -> int:
    """Chunk length turbo_attn_decode uses for a sequence of seq_len tokens."""
    return kv_split_groups or int(lib().turbo_decode_default_split(int(seq_len) // 64))


def decode_auto_split(B: int, Hq: int, Hkv: int, max_groups: int) -> int:
    """Chunk length fitted to a batch's occupancy (turbo_decode_auto_split)."""
    return int(lib().turbo_decode_auto_split(B, Hq, Hkv, max_groups))


def decode_workspace(B: int, Hq: int, Hkv: int, max_groups: int, kv_split_groups: int = 0,
                     device="cuda", with_tail: bool = False) -> Optional[torch.Tensor]:
    n = int(lib().turbo_decode_workspace_bytes(B, Hq, Hkv, max_groups, kv_split_groups,
                                               int(bool(with_tail))))
    if n == 0:
        return None
    return torch.empty(n // 4, dtype=torch.float32, device=device)


def turbo_attn_decode(q: torch.Tensor, cache: PagedKVCache, seq_lens: torch.Tensor,
                      block_table: torch.Tensor, group_table: torch.Tensor,
                      sm_scale: Optional[float] = None, kv_split_groups: int = 0,
                      workspace: Optional[torch.Tensor] = None, return_lse: bool = False,
                      out=None, tail: Optional[KVTail] = None):
    """Algorithm 2 decode over the paged cache (and the Sec. 3.3 buffer when
    tail is given).  q fp16 [B][Hq][128]."""
    B, Hq, d = q.shape
    mg = group_table.shape[1]
    sm = float(1.0 / np.sqrt(d)) if sm_scale is None else float(sm_scale)
    if workspace is None:
        workspace = decode_workspace(B, Hq, cache.num_kv_heads, mg, kv_split_groups, q.device,
                                     with_tail=tail is not None)
    wbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    o = torch.empty_like(q) if out is None else out
    lse = torch.empty(B, Hq, dtype=torch.float32, device=q.device) if return_lse else None
    cs = cache.struct()
    ts = tail.struct() if tail is not None else None
    st = lib().turbo_attn_decode(_ptr(q), ctypes.byref(cs),
                                 ctypes.byref(ts) if ts is not None else None, _ptr(seq_lens),
                                 _ptr(block_table), _ptr(group_table), mg, B, Hq, sm,
                                 int(kv_split_groups), _ptr(workspace), wbytes, _ptr(o),
                                 _ptr(lse), _stream(q.device))
    _check(st, "turbo_attn_decode")
    return (o, lse) if return_lse else o


def turbo_attn_decode_noalloc(q: torch.Tensor, cache: PagedKVCache, seq_lens: torch.Tensor,
                              block_table: torch.Tensor, group_table: torch.Tensor,
                              sm_scale: Optional[float] = None, kv_split_groups: int = 0,
                              return_lse: bool = False, out=None,
                              tail: Optional[KVTail] = None, lse_out=None):
    """turbo_attn_decode without a workspace: the library's fixed per-GPU
    scratch holds the chunk states (no device allocation by the library;
    pass `out` and `lse_out` to allocate nothing here either)."""
    B, Hq, d = q.shape
    mg = group_table.shape[1]
    sm = float(1.0 / np.sqrt(d)) if sm_scale is None else float(sm_scale)
    o = torch.empty_like(q) if out is None else out
    lse = lse_out
    if return_lse and lse is None:
        lse = torch.empty(B, Hq, dtype=torch.float32, device=q.device)
    cs = cache.struct()
    ts = tail.struct() if tail is not None else None
    st = lib().turbo_attn_decode_noalloc(_ptr(q), ctypes.byref(cs),
                                         ctypes.byref(ts) if ts is not None else None,
                                         _ptr(seq_lens), _ptr(block_table), _ptr(group_table),
                                         mg, B, Hq, sm, int(kv_split_groups), _ptr(o), _ptr(lse),
                                         _stream(q.device))
    _check(st, "turbo_attn_decode_noalloc")
    return (o, lse) if (return_lse or lse_out is not None) else o


def turbo_attn_decode_trace(q: torch.Tensor, cache: PagedKVCache, seq_lens: torch.Tensor,
                            block_table: torch.Tensor, group_table: torch.Tensor, sel,
                            sm_scale: Optional[float] = None, kv_split_groups: int = 0,
                            tail: Optional[KVTail] = None):
    """Test hook: turbo_attn_decode that also returns the integers of group g
    of (sequence b, query head h), sel = (b, h, g); row 0 of each array."""
    B, Hq, d = q.shape
    mg = group_table.shape[1]
    sm = float(1.0 / np.sqrt(d)) if sm_scale is None else float(sm_scale)
    workspace = decode_workspace(B, Hq, cache.num_kv_heads, mg, kv_split_groups, q.device,
                                 with_tail=tail is not None)
    wbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    o = torch.empty_like(q)
    buf = _trace_buffer(q.device)
    cs = cache.struct()
    ts = tail.struct() if tail is not None else None
    b, h, g = sel
    st = lib().turbo_attn_decode_trace(_ptr(q), ctypes.byref(cs),
                                       ctypes.byref(ts) if ts is not None else None, _ptr(seq_lens),
                                       _ptr(block_table), _ptr(group_table), mg, B, Hq, sm,
                                       int(kv_split_groups), _ptr(workspace), wbytes, _ptr(o),
                                       None, b, h, g, _ptr(buf), _stream(q.device))
    _check(st, "turbo_attn_decode_trace")
    torch.cuda.synchronize(q.device)
    return o, _trace_dict(buf)


def turbo_head_priority(k: torch.Tensor) -> torch.Tensor:
    """Sec. 3.2 priority (gap x std) of each KV head of the prefill keys
    k fp16 [B][Hkv][N][128]; returns fp32 [Hkv] on k's device."""
    B, Hkv, N, d = k.shape
    out = torch.empty(Hkv, dtype=torch.float32, device=k.device)
    n = int(lib().turbo_head_priority_workspace_bytes(B, Hkv, N))
    ws = torch.empty(max(n, 4) // 4, dtype=torch.float32, device=k.device)
    _check(lib().turbo_head_priority(_ptr(k), B, Hkv, N, d, _ptr(ws), n, _ptr(out),
                                     _stream(k.device)), "turbo_head_priority")
    return out


def turbo_int2_heads(priority, n_int2: int) -> np.ndarray:
    """Sec. 3.2 strategy: uint8 [Hkv] bit widths, 2 for the n_int2 lowest
    priorities (host)."""
    p = np.ascontiguousarray(np.asarray(priority, dtype=np.float32))
    bits = np.empty(p.size, np.uint8)
    _check(lib().turbo_int2_heads(p.ctypes.data_as(ctypes.c_void_p), p.size, int(n_int2),
                                  bits.ctypes.data_as(ctypes.c_void_p)), "turbo_int2_heads")
    return bits


def turbo_sas_softmax(x: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Algorithm 3: SAS softmax of the rows of x (fp32, contiguous, last dim =
    columns).  out may be x itself."""
    if x.dtype != torch.float32 or not x.is_contiguous() or x.dim() < 1:
        raise ValueError("x must be a contiguous float32 tensor")
    cols = x.shape[-1]
    rows = x.numel() // max(cols, 1)
    y = torch.empty_like(x) if out is None else out
    _check(lib().turbo_sas_softmax(_ptr(x), _ptr(y), rows, cols, _stream(x.device)),
           "turbo_sas_softmax")
    return y


def turbo_qkv_project(x: torch.Tensor, w: torch.Tensor, Hq: int, Hkv: int,
                      cache: Optional[PagedKVCache] = None,
                      block_table: Optional[torch.Tensor] = None,
                      group_table: Optional[torch.Tensor] = None, out=None, y=None):
    """QKV projection with FlashQ fused (Sec. 5.2): x fp16 [B][N][D], w fp16
    [(Hq + 2 Hkv) 128][D].  Returns (q8, s_q, k8, v8, s_k, s_v) in the layouts
    of include/turbo_attn.h; writes the full K/V groups into `cache`.  With y
    (fp16 [B][N][(Hq + 2 Hkv) 128]) the test hook turbo_qkv_project_trace runs
    and also stores the fp16 projection there."""
    B, N, D = x.shape
    nb = (N + BLOCK - 1) // BLOCK
    dev = x.device
    if out is None:
        q8 = torch.empty(B, Hq, nb * BLOCK, HEAD_DIM, dtype=torch.int8, device=dev)
        s_q = torch.empty(B, Hq, nb, dtype=torch.float32, device=dev)
        k8 = torch.empty(B, Hkv, nb * BLOCK, HEAD_DIM, dtype=torch.int8, device=dev)
        v8 = torch.empty(B, Hkv, nb, HEAD_DIM, BLOCK, dtype=torch.int8, device=dev)
        s_k = torch.empty(B, Hkv, nb, dtype=torch.float32, device=dev)
        s_v = torch.empty_like(s_k)
    else:
        q8, s_q, k8, v8, s_k, s_v = out
    cs = cache.struct() if cache is not None else None
    mg = group_table.shape[1] if group_table is not None else 0
    args = [_ptr(x), _ptr(w), B, N, D, Hq, Hkv, HEAD_DIM, _ptr(q8), _ptr(s_q), _ptr(k8), _ptr(v8),
            _ptr(s_k), _ptr(s_v), ctypes.byref(cs) if cs is not None else None,
            _ptr(block_table), _ptr(group_table), mg]
    if y is None:
        _check(lib().turbo_qkv_project(*args, _stream(dev)), "turbo_qkv_project")
    else:
        _check(lib().turbo_qkv_project_trace(*args, _ptr(y), _stream(dev)),
               "turbo_qkv_project_trace")
    return q8, s_q, k8, v8, s_k, s_v


def turbo_attn_prefill_q8(q8: torch.Tensor, s_q: torch.Tensor, k8, v8, s_k, s_v, N: int,
                          sm_scale: Optional[float] = None, causal: bool = True,
                          return_lse: bool = False, out=None):
    """Algorithm 1 prefill on pre-quantized Q (q8 [B][Hq][64 nb][128], s_q)."""
    B, Hq = q8.shape[0], q8.shape[1]
    Hkv = k8.shape[1]
    sm = float(1.0 / np.sqrt(HEAD_DIM)) if sm_scale is None else float(sm_scale)
    o = torch.empty(B, Hq, N, HEAD_DIM, dtype=torch.float16, device=q8.device) if out is None else out
    lse = torch.empty(B, Hq, N, dtype=torch.float32, device=q8.device) if return_lse else None
    _check(lib().turbo_attn_prefill_q8(_ptr(q8), _ptr(s_q), _ptr(k8), _ptr(v8), _ptr(s_k),
                                       _ptr(s_v), B, Hq, Hkv, N, HEAD_DIM, sm, int(causal),
                                       _ptr(o), _ptr(lse), _stream(q8.device)),
           "turbo_attn_prefill_q8")
    return (o, lse) if return_lse else o


def probe_mfma_i8(iters: int, device="cuda") -> int:
    """Queues the int8 MFMA ceiling probe; returns the int8 ops it performs."""
    sink = torch.empty(512, dtype=torch.int32, device=device)
    ops = ctypes.c_int64(0)
    _check(lib().turbo_probe_mfma_i8(int(iters), _ptr(sink), ctypes.byref(ops),
                                     _stream(torch.device(device))), "turbo_probe_mfma_i8")
    return int(ops.value)


def probe_valu(iters: int, device="cuda") -> int:
    """Queues the vector-ALU issue probe; returns the wave instructions it issues."""
    sink = torch.empty(1024, dtype=torch.float32, device=device)
    n = ctypes.c_int64(0)
    _check(lib().turbo_probe_valu(int(iters), _ptr(sink), ctypes.byref(n),
                                  _stream(torch.device(device))), "turbo_probe_valu")
    return int(n.value)


def probe_read(buf: torch.Tensor) -> int:
    """Queues the streaming-read probe over buf; returns the bytes it reads."""
    sink = torch.empty(1, dtype=torch.int32, device=buf.device)
    n = buf.numel() * buf.element_size()
    _check(lib().turbo_probe_read(_ptr(buf), n, _ptr(sink), _stream(buf.device)),
           "turbo_probe_read")
    return n
