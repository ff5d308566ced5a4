"""Benchmark of the TurboAttention hot path on one MI355X.

A step is one pass of the whole path over one batch of synthetic input:
  turbo_quantize_kv  (FlashQ step 1 + step 2, K/V -> int8 blocks + int4/int2 cache)
  turbo_attn_prefill (Algorithm 1: causal FlashQ + SAS attention)
  turbo_attn_decode  (Algorithm 2: one new query per sequence over the cache)
on the Phi-3-medium-shaped prefill workload (batch 4, 40 query / 10 KV heads,
head_dim 128, 4096 tokens, int4 cache) unless --workload says otherwise.
Inputs are resident in HBM before the timed region.

The JSON line reports the attention int-op rate of the step (dense causal
count: 4*d ops per visible (query, key) pair of prefill plus 4*d per cached
key and query head of decode), per-kernel times, the roofline of the dominant
kernel (HIP-event timed on the stream its launches go to), and the CPU oracle
timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_INT8_TOPS = 5000.0   # MI355X dense int8 MFMA, 5.0 POP/s
PEAK_HBM_GBS = 8000.0     # MI355X HBM3E, 8 TB/s
PEAK_FP16_TFLOPS = 2500.0  # MI355X dense fp16 MFMA, 2.5 PFLOP/s


def source_digest(paths) -> str:
    """First 16 hex digits of the sha256 of the given source files with their
    comments, leading/trailing blanks and empty lines removed, so that an edit
    of the prose alone keeps the digest (and the counters taken under it)."""
    import hashlib
    import re
    m = hashlib.sha256()
    for f in paths:
        with open(os.path.join(ROOT, f), encoding="utf-8") as fh:
            text = fh.read()
        if f.endswith(".py"):
            text = re.sub(r"(?m)^\s*#.*$", "", text)
        else:
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            text = re.sub(r"//[^\n]*", "", text)
        lines = [ln.strip() for ln in text.splitlines()]
        m.update("\n".join(ln for ln in lines if ln).encode())
    return m.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    summary (profiles/traffic.txt), or None if the kernel's sources changed
    since the counters were taken."""
    srcs = {"k_attn_prefill16": ["paper_2412_08585_amd/csrc/attn_prefill.hip",
                                 "paper_2412_08585_amd/csrc/turbo_common.h",
                                 "paper_2412_08585_amd/build.py"],
            "k_attn_decode": ["paper_2412_08585_amd/csrc/attn_decode.hip",
                              "paper_2412_08585_amd/csrc/kv_tail.hip",
                              "paper_2412_08585_amd/csrc/turbo_common.h",
                              "paper_2412_08585_amd/csrc/stream_loads.h",
                              "paper_2412_08585_amd/build.py"]}.get(kernel)
    path = os.path.join(ROOT, "profiles", "traffic.txt")
    if not srcs or not os.path.exists(path):
        return None
    digest = source_digest(srcs)
    for line in open(path):
        parts = line.split()
        if len(parts) == 4 and parts[0] == kernel and parts[1] == workload and parts[2] == digest:
            return float(parts[3])
    return None


# Vector ALU issue peak of the MI355X in G wave64 instructions/s: the fp32
# vector peak of 157.3 TFLOP/s is one 64-lane FMA (2 flops a lane) per 2
# clocks per SIMD (1,024 SIMDs at 2.4 GHz).
PEAK_VALU_GINST = 157.3e3 / (64 * 2)


def measured_valu(kernel: str, workload: str):
    """Non-MFMA vector ALU instructions per launch from the committed rocprofv3
    SQ_INSTS_VALU - SQ_INSTS_MFMA summary (profiles/valu.txt), or None if the
    kernel's sources changed since the counters were taken."""
    srcs = {"k_attn_prefill16": ["paper_2412_08585_amd/csrc/attn_prefill.hip",
                                 "paper_2412_08585_amd/csrc/turbo_common.h",
                                 "paper_2412_08585_amd/build.py"]}.get(kernel)
    path = os.path.join(ROOT, "profiles", "valu.txt")
    if not srcs or not os.path.exists(path):
        return None
    digest = source_digest(srcs)
    for line in open(path):
        parts = line.split()
        if len(parts) == 4 and parts[0] == kernel and parts[1] == workload and parts[2] == digest:
            return float(parts[3])
    return None


def decode_bytes_per_token(bits: int) -> float:
    """Compressed K+V bytes read per cached token and KV head: codes plus the
    per-channel integer scale/zero (4 x 128 B per 64-token group) plus the
    two fp32 block scales per group."""
    return 2 * 128 * bits / 8 + 4 * 128 / 64 + 8 / 64


def ramp_clocks(fn, seconds: float = 0.2):
    """Untimed launches of the step until `seconds` of wall time have passed:
    the GPU idles during input generation and its clocks fall; the warmup
    steps proper (--warmup) and the timed steps (--steps) follow."""
    import torch
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(4):
            fn()
        torch.cuda.synchronize()


def launch_times(fn, iters: int, prev=None):
    """GPU time (ms) of each of `iters` launches of fn, from a HIP event pair
    around each launch on the stream the library launches on (torch's current
    stream).  prev (optional) is launched untimed before each timed launch:
    it hides the host's launch overhead of fn when fn is shorter than it."""
    import torch
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(iters)]
    fn()
    torch.cuda.synchronize()
    for a, b in ev:
        if prev is not None:
            prev()
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in ev]


def stats(ts):
    """Median and mean of per-launch times (ms)."""
    return float(np.median(ts)), float(np.mean(ts))


CPU_SAMPLE_SECONDS = 10.0


def cpu_sample(run_chunk, n_total: int, chunk: int, seconds: float = CPU_SAMPLE_SECONDS):
    """Runs the oracle over consecutive chunks of the workload, run_chunk(lo,
    hi), until `seconds` of oracle time have passed or the whole workload is
    done; returns (items done, oracle seconds).  Copies to the host are not
    timed."""
    done, dt = 0, 0.0
    while done < n_total and dt < seconds:
        hi = min(n_total, done + chunk)
        dt += run_chunk(done, hi)
        done = hi
    return done, dt


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


# The paper's own efficiency result, quoted as context (other hardware, other
# baseline): TurboAttention's attention speedup over FP16 FlashAttention.
PAPER_CONTEXT = {
    "attention_speedup_vs_fp16_flashattention": "1.2-1.8x (prefill up to 1.8x, decode up to 1.7x)",
    "hardware": "NVIDIA A100-80GB-SXM, Triton kernels",
    "workload": "Phi3-medium attention, batch 1-64 at 1k context and 4k-32k context at batch 4",
    "source": "Abstract; Sec. 5.3, Fig. 5",
    "comparable_here": False,
}


def fp16_attention_here(q, k, v, causal: bool, iters: int, ms_turbo: float, label: str):
    """The paper's comparison measured on this GPU: torch's fp16
    scaled_dot_product_attention (its flash or memory-efficient backend, a
    library kernel; never the math path) on the same q, k, v, against the
    TurboAttention time ms_turbo.  None when neither backend takes the shapes."""
    import torch
    from torch.nn.attention import SDPBackend, sdpa_kernel
    G = q.shape[1] // k.shape[1]
    for name, backend in (("flash", SDPBackend.FLASH_ATTENTION),
                          ("memory-efficient", SDPBackend.EFFICIENT_ATTENTION)):
        for gqa in (True, False):
            try:
                kk, vv = (k, v) if gqa else (k.repeat_interleave(G, dim=1).contiguous(),
                                             v.repeat_interleave(G, dim=1).contiguous())
                kw = {"enable_gqa": True} if gqa and G > 1 else {}
                with sdpa_kernel([backend]):
                    fn = lambda: torch.nn.functional.scaled_dot_product_attention(
                        q, kk, vv, is_causal=causal, **kw)
                    ramp_clocks(fn, 0.1)
                    ms, _ = stats(launch_times(fn, iters))
            except Exception:  # this backend does not take these shapes
                continue
            return {"library": f"torch {torch.__version__} scaled_dot_product_attention, fp16, "
                               f"{name} backend" + (", GQA in the kernel" if gqa and G > 1 else
                                                    ", K/V expanded to the query heads"),
                    "workload": label, "ms": round(ms, 4),
                    "turbo_ms": round(ms_turbo, 4), "turbo_speedup": round(ms / ms_turbo, 3)}
    return None


def measured_ceilings(dev):
    """The int8 MFMA rate and the HBM streaming-read rate of this GPU, from the
    library's probe kernels (median of 5 launches each)."""
    import torch

    import paper_2412_08585_amd as ta
    ops = [0]

    def mfma():
        ops[0] = ta.binding.probe_mfma_i8(4096, dev)

    insts = [0]

    def valu():
        insts[0] = ta.binding.probe_valu(4096, dev)

    buf = torch.ones(1 << 28, dtype=torch.float32, device=dev)  # 1 GiB
    ramp_clocks(mfma, 0.1)
    t_m, _ = stats(launch_times(mfma, 5))
    t_v, _ = stats(launch_times(valu, 5))
    t_r, _ = stats(launch_times(lambda: ta.binding.probe_read(buf), 5))
    nbytes = buf.numel() * 4
    del buf
    return {"int8_mfma_TOPS": round(ops[0] / (t_m * 1e-3) / 1e12, 1),
            "hbm_read_GBs": round(nbytes / (t_r * 1e-3) / 1e9, 1),
            "valu_Ginst_per_s": round(insts[0] / (t_v * 1e-3) / 1e9, 1),
            "probes": "turbo_probe_mfma_i8 (8 chains of v_mfma_i32_16x16x64_i8 per wave, 2048 "
                      "waves), turbo_probe_valu (8 chains of v_fma_f32 per wave, 4096 waves) "
                      "and turbo_probe_read (1 GiB nontemporal streaming read, one 32 KiB "
                      "chunk per work-group), median of 5"}


def valu_roofline(kernel: str, workload: str, ms: float, ceil: dict):
    """The vector ALU roofline of a kernel: its committed non-MFMA VALU
    instruction count per launch over its measured time, against the issue
    peak and the probe's measured rate (None without a current count)."""
    n = measured_valu(kernel, workload)
    if n is None:
        return None
    rate = n / (ms * 1e-3) / 1e9
    return {"kernel": kernel, "bound": "alu", "achieved": round(rate, 1),
            "peak": PEAK_VALU_GINST, "unit": "G wave-instructions/s",
            "frac": round(rate / PEAK_VALU_GINST, 4),
            "frac_of_measured_ceiling": round(rate / ceil["valu_Ginst_per_s"], 4),
            "instructions_per_launch": n,
            "derivation": "fp32 vector peak 157.3 TFLOP/s / (64 lanes x 2 flops per FMA) = one "
                          "wave64 instruction per 2 clocks per SIMD (1,024 SIMDs, 2.4 GHz); "
                          "instructions = SQ_INSTS_VALU - SQ_INSTS_MFMA from profiles/valu.txt",
            "note": "on gfx950 the issue cost of a wave64 VALU instruction depends on the opcode "
                    "and its operands: 2.6-3.2 clocks for VOP2 add/sub/mul/fmac with VGPR operands, "
                    "4.3-4.8 for VOP3, SGPR operands, compares, selects, conversions, shifts and "
                    "maxima (none at 2); the measured ceiling is the FMA-chain probe "
                    "(turbo_probe_valu, about 3.1 clocks)"}


def rel_l2(a, ref) -> float:
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.linalg.norm(a - ref) / np.linalg.norm(ref))


def error_decomposition(run_oracle, exact, got):
    """rel-L2 against exact fp64 softmax attention of the GPU output and of the
    oracle with FlashQ and SAS on (the method), FlashQ alone (exact exp, no
    threshold) and SAS alone (unquantized operands): the operator-level
    analogue of the paper's Table 4 ablation."""
    both = run_oracle(True, True)
    return {"gpu": rel_l2(got, exact), "oracle_flashq_and_sas": rel_l2(both, exact),
            "oracle_flashq_only": rel_l2(run_oracle(True, False), exact),
            "oracle_sas_only": rel_l2(run_oracle(False, True), exact),
            "gpu_vs_oracle_max_rel_rowmax": float(
                np.max(np.abs(np.asarray(got, np.float64) - both)
                       / np.maximum(np.abs(both).max(axis=-1, keepdims=True), 1e-30)))}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="phi3m-prefill-4k")
    ap.add_argument("--kernel-iters", type=int, default=30)
    ap.add_argument("--kv-split-groups", type=int, default=0,
                    help="decode workloads: chunk length of the split-KV decode (0: the "
                         "library's default, each sequence by its own length; -1: the "
                         "occupancy-fitted turbo_decode_auto_split)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode-half", action="store_true",
                    help="prefill workloads: skip the Phi-3-medium decode half of the line")
    ap.add_argument("--no-error", action="store_true",
                    help="skip the error decomposition against exact fp64 attention")
    ap.add_argument("--only", choices=["quantize", "prefill", "decode", "copy", "mfma-ceiling",
                                       "read-ceiling"], default=None,
                    help="launch only this kernel --steps times (for profiler passes); "
                         "'copy' runs a plain 1 GiB device copy (calibration of the HBM "
                         "byte counters); the ceilings run the library's probe kernels")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only (--gpus 1); the "
                          "library has no multi-GPU sharding"}))
        sys.exit(2)
    import torch

    import paper_2412_08585_amd as ta
    from paper_2412_08585_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.only in ("copy", "mfma-ceiling", "read-ceiling"):
        n = args.warmup + args.steps
        if args.only == "copy":
            src = torch.ones(1 << 28, dtype=torch.float32, device=dev)  # 1 GiB
            dst = torch.empty_like(src)
            for _ in range(n):
                dst.copy_(src)
            info = {"bytes_read": src.numel() * 4, "bytes_written": dst.numel() * 4}
        elif args.only == "mfma-ceiling":
            for _ in range(n):
                ops = ta.binding.probe_mfma_i8(4096, dev)
            info = {"int8_ops_per_launch": ops}
        else:
            buf = torch.ones(1 << 28, dtype=torch.float32, device=dev)
            for _ in range(n):
                nb_ = ta.binding.probe_read(buf)
            info = {"bytes_read_per_launch": nb_}
        torch.cuda.synchronize()
        print(json.dumps({"only": args.only, "launches": n, **info}))
        return
    w = W.WORKLOADS[args.workload]
    if w.kind == "decode":
        return bench_decode(args, w)
    if w.kind == "softmax":
        return bench_softmax(args, w)
    if w.kind == "projection":
        return bench_projection(args, w)
    B, Hq, Hkv, N, G = w.B, w.Hq, w.Hkv, w.N, w.G
    d = 128

    # ---- inputs (resident in HBM) -------------------------------------------
    q, k, v = W.prefill_inputs(w, device=dev)
    qd = W.decode_query(w, device=dev)
    bits = W.head_bits(w)
    bt, gt = W.tables(w)
    btd, gtd = torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)
    cache = ta.PagedKVCache(bt.size, gt.size, bits, dev)
    nb = (N + 63) // 64
    k8 = torch.empty(B, Hkv, nb * 64, d, dtype=torch.int8, device=dev)
    v8 = torch.empty(B, Hkv, nb, d, 64, dtype=torch.int8, device=dev)
    sk = torch.empty(B, Hkv, nb, dtype=torch.float32, device=dev)
    sv = torch.empty_like(sk)
    o = torch.empty_like(q)
    od = torch.empty_like(qd)
    sl = torch.full((B,), N, dtype=torch.int32, device=dev)
    # the decode of this batch (B * Hkv = 40 units of 64 groups) takes the
    # occupancy-fitted chunk length; the decode half below uses the default
    split = ta.decode_auto_split(B, Hq, Hkv, w.max_groups)
    ws = ta.decode_workspace(B, Hq, Hkv, w.max_groups, split, dev)

    def run_quant():
        ta.turbo_quantize_kv(k, v, cache, btd, gtd, out=(k8, v8, sk, sv))

    def run_prefill():
        ta.turbo_attn_prefill(q, k8, v8, sk, sv, w.sm_scale, True, out=o)

    def run_decode():
        ta.turbo_attn_decode(qd, cache, sl, btd, gtd, w.sm_scale, split, workspace=ws, out=od)

    def step():
        run_quant()
        run_prefill()
        run_decode()

    if args.only:
        fn = {"quantize": run_quant, "prefill": run_prefill, "decode": run_decode}[args.only]
        run_quant()
        for _ in range(args.warmup + args.steps):
            fn()
        torch.cuda.synchronize()
        print(json.dumps({"only": args.only, "launches": args.warmup + args.steps}))
        return

    # ---- whole-step timing ----------------------------------------------------
    ramp_clocks(step)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    mk = lambda: torch.cuda.Event(enable_timing=True)
    e0, e1 = mk(), mk()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps

    # ---- per-kernel timing: the same steps again, with an event pair around
    # every kernel on the library's stream; medians over the steps ------------
    evs = [[mk() for _ in range(4)] for _ in range(args.steps)]
    for ev in evs:
        ev[0].record(stream)
        run_quant()
        ev[1].record(stream)
        run_prefill()
        ev[2].record(stream)
        run_decode()
        ev[3].record(stream)
    torch.cuda.synchronize()
    ms_q, mean_q = stats([ev[0].elapsed_time(ev[1]) for ev in evs])
    ms_p, mean_p = stats([ev[1].elapsed_time(ev[2]) for ev in evs])
    ms_d, mean_d = stats([ev[2].elapsed_time(ev[3]) for ev in evs])
    prio = torch.empty(Hkv, dtype=torch.float32, device=dev)
    nws_h = int(ta.binding.lib().turbo_head_priority_workspace_bytes(B, Hkv, N))
    ws_h = torch.empty(nws_h // 4, dtype=torch.float32, device=dev)
    ms_h, _ = stats(launch_times(lambda: ta.binding.lib().turbo_head_priority(
        ta.binding._ptr(k), B, Hkv, N, d, ta.binding._ptr(ws_h), nws_h, ta.binding._ptr(prio),
        ta.binding._stream(dev)), args.kernel_iters))

    # ---- algorithmic work -------------------------------------------------------
    prefill_ops = 2.0 * d * N * (N + 1) * B * Hq          # QK^T + PV over causal pairs
    decode_ops = 4.0 * d * (N // 64 * 64) * B * Hq
    step_ops = prefill_ops + decode_ops
    quant_bytes = B * Hkv * N * d * 2 * 2                 # fp16 K, V in
    quant_bytes += B * Hkv * nb * 64 * d * 2 + B * Hkv * nb * 8   # int8 K8/V8 + scales out
    quant_bytes += sum(decode_bytes_per_token(int(bits[h])) for h in range(Hkv)) * B * (N // 64 * 64)
    decode_bytes = sum(decode_bytes_per_token(int(bits[h])) for h in range(Hkv)) * B * (N // 64 * 64)
    decode_bytes += B * Hq * d * 2 * 2                    # q in, o out (fp16)
    prefill_tops = prefill_ops / (ms_p * 1e-3) / 1e12
    ceil = measured_ceilings(dev)

    result = {
        "metric": "attention TOPS (prefill) & HBM GB/s (decode), % of MI355X roofline",
        "value": round(step_ops / (ms_step * 1e-3) / 1e12, 3),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic (seeded N(0,1) fp16 with 4 K outlier channels x10; no weights)",
        "config": {"workload": w.name, "batch": B, "q_heads": Hq, "kv_heads": Hkv, "seq_len": N,
                   "head_dim": d, "causal": True, "kv_cache": w.bits, "block_rows": 64,
                   "block_cols": 64, "decode_tokens": 1, "decode_kv_split_groups": split,
                   "decode_half": "phi3m-decode-8k"},
        "kernels": {
            "timing": "median over the timed steps of HIP events around each kernel (mean in "
                      "brackets)",
            "quantize_kv": {"ms": round(ms_q, 4), "mean_ms": round(mean_q, 4),
                            "GB/s": round(quant_bytes / ms_q / 1e6, 1),
                            "frac_hbm": round(quant_bytes / ms_q / 1e6 / PEAK_HBM_GBS, 4)},
            "head_priority": {"ms": round(ms_h, 4), "GB/s": round(B * Hkv * N * d * 2 / ms_h / 1e6, 1),
                              "frac_hbm": round(B * Hkv * N * d * 2 / ms_h / 1e6 / PEAK_HBM_GBS, 4),
                              "note": "Sec. 3.2 bit choice from the prefill K; not in the step; "
                                      "K (B*Hkv*N*128 fp16) may stay in the 256 MB MALL across "
                                      "the repeated launches"},
            "attn_prefill": {"ms": round(ms_p, 4), "mean_ms": round(mean_p, 4),
                             "TOPS": round(prefill_tops, 2),
                             "frac_int8_mfma": round(prefill_tops / PEAK_INT8_TOPS, 4)},
            "attn_decode": {"ms": round(ms_d, 4), "mean_ms": round(mean_d, 4),
                            "GB/s": round(decode_bytes / ms_d / 1e6, 1),
                            "frac_hbm": round(decode_bytes / ms_d / 1e6 / PEAK_HBM_GBS, 4),
                            "note": "this workload's 22 MB cache may sit in the 256 MB MALL; "
                                    "the decode roofline is roofline_decode"},
        },
        "roofline": {"kernel": "k_attn_prefill16", "bound": "mfma",
                     "achieved": round(prefill_tops, 2), "peak": PEAK_INT8_TOPS,
                     "unit": "TOP/s", "frac": round(prefill_tops / PEAK_INT8_TOPS, 4),
                     "traffic": measured_traffic("k_attn_prefill16", w.name),
                     "per_launch_ops": prefill_ops,
                     "frac_of_measured_ceiling": round(prefill_tops / ceil["int8_mfma_TOPS"], 4),
                     "valu_note": "issue-bound on the VALU (SAS + P quantization + accumulator "
                                  "update); see profiles/k_attn_prefill16_phi3m-prefill-4k.md"},
        "roofline_valu": valu_roofline("k_attn_prefill16", w.name, ms_p, ceil),
        "ceilings_measured": ceil,
        "paper_context": PAPER_CONTEXT,
    }
    # the paper's comparison (fp16 attention) measured here: the quantization
    # of K and V counts on TurboAttention's side
    fp16_here = fp16_attention_here(q, k, v, True, args.kernel_iters, ms_q + ms_p,
                                    f"{w.name} prefill (quantize_kv + attn_prefill)")
    if fp16_here is not None:
        result["paper_context"] = dict(PAPER_CONTEXT, fp16_attention_here=fp16_here)

    # ---- the decode half of the headline: Phi-3-medium decode ---------------
    if not args.no_decode_half:
        wd = W.WORKLOADS["phi3m-decode-8k"]
        dec = decode_measure(args, wd, dev, 0)
        result["roofline_decode"] = dict(dec["roofline"],
                                         frac_of_measured_ceiling=round(
                                             dec["roofline"]["achieved"] / ceil["hbm_read_GBs"], 4),
                                         workload=wd.name, ms=dec["ms"], mean_ms=dec["mean_ms"],
                                         kv_split_groups=dec["split"])
        if dec["fp16_here"] is not None:
            result["paper_context"] = dict(result["paper_context"],
                                           fp16_decode_here=dec["fp16_here"])
        if not args.no_error:
            result["error_vs_fp64"] = {"decode": decode_error(wd, dec, dev)}
        del dec
        torch.cuda.empty_cache()

    # ---- error of GPU and oracle against exact fp64 attention (one unit) -----
    if not args.no_error:
        import oracle
        b0, h0 = 0, 0
        qs = q[b0, h0 * G:(h0 + 1) * G][None].cpu()
        ks, vs = k[b0, h0][None, None].cpu(), v[b0, h0][None, None].cpu()
        got = o[b0, h0 * G:(h0 + 1) * G][None].float().cpu().numpy()
        ex, _ = oracle.attn_exact(qs, ks, vs, float(np.float32(w.sm_scale)), True)
        dec_err = result.get("error_vs_fp64", {}).get("decode")
        result["error_vs_fp64"] = {
            "metric": "rel-L2 over the unit's query heads, rows and channels",
            "prefill": dict(error_decomposition(
                lambda qu, sa: oracle.attn_prefill(qs, ks, vs, w.sm_scale, True, quant=qu,
                                                   sas=sa)[0], ex, got),
                sample=f"sequence {b0}, KV head {h0} with its {G} query heads, {N} causal rows")}
        if dec_err is not None:
            result["error_vs_fp64"]["decode"] = dec_err

    # ---- CPU oracle on a bounded sample -----------------------------------------
    if not args.no_cpu_baseline:
        import oracle
        threads = oracle.num_threads()
        rng = np.random.default_rng(0)
        order = [divmod(int(u), Hkv) for u in rng.permutation(B * Hkv)]
        ros = []

        def run_units(lo, hi):
            # one unit = one sequence with one KV head and its G query heads
            us, n = order[lo:hi], hi - lo
            qs = torch.stack([q[b, h * G:(h + 1) * G] for b, h in us]).cpu()
            ks = torch.stack([k[b, h] for b, h in us])[:, None].cpu()
            vs = torch.stack([v[b, h] for b, h in us])[:, None].cpu()
            qds = torch.stack([qd[b, h * G:(h + 1) * G] for b, h in us]).cpu()
            t0 = time.perf_counter()
            ref = oracle.quantize_kv(ks, vs, [4])
            ro, _ = oracle.attn_prefill(qs, ks, vs, w.sm_scale, True)
            oracle.attn_decode(qds, ref, [N] * n, w.sm_scale, split=split)
            t = time.perf_counter() - t0
            ros.append(ro)
            return t

        n_units, dt = cpu_sample(run_units, B * Hkv, max(1, math.ceil(threads / G)))
        units, ro = order[:n_units], np.concatenate(ros)
        sample_ops = (prefill_ops + decode_ops) * n_units / (B * Hkv)
        result["cpu_baseline"] = {
            "value": round(sample_ops / dt / 1e12, 6), "unit": "TOPS",
            "cores": min(threads, n_units * G), "kind": "oracle",
            "cpu_model": cpu_model(), "host_threads": os.cpu_count(),
            "sample": f"{n_units} of {B * Hkv} (sequence, KV head) units, full length "
                      f"(quantize + prefill + decode), {dt:.1f} s"}
        got = torch.stack([o[b, h * G:(h + 1) * G] for b, h in units]).float().cpu().numpy()
        rowmax = np.abs(ro).max(axis=-1, keepdims=True)
        result["parity"] = {
            "max_err_vs_oracle_rel_rowmax": float(np.max(np.abs(got - ro) / rowmax)),
            "sample_units": n_units}
    print(json.dumps(result), flush=True)


def build_decode_caches(w, dev, ncopy: int):
    """The compressed cache of a decode workload (and its Sec. 3.3 buffer),
    built untimed, `ncopy` times with the same contents so that timed calls
    can alternate between copies and stream from HBM rather than the MALL."""
    import torch

    import paper_2412_08585_amd as ta
    from paper_2412_08585_amd import workloads as W
    B, Hkv, N = w.B, w.Hkv, w.N
    bits = W.head_bits(w)
    bt, gt = W.tables(w)
    caches, tails = [], []
    for c in range(ncopy):
        cache = ta.PagedKVCache(bt.size, gt.size, bits, dev)
        tail = ta.KVTail(B, Hkv, dev)
        btd, gtd = torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)
        chunk = 16
        for b0 in range(0, B, chunk):
            nbat = min(chunk, B - b0)
            k = torch.empty(nbat, Hkv, N, 128, dtype=torch.float16, device=dev)
            v = torch.empty_like(k)
            for bb in range(nbat):
                for h in range(Hkv):
                    k[bb, h], v[bb, h] = W.unit_kv(w, b0 + bb, h, device=dev)
            _, _, sk, sv = ta.turbo_quantize_kv(k, v, cache, btd[b0:b0 + nbat], gtd[b0:b0 + nbat])
            ta.turbo_tail_init(k, v, sk, sv, tail.narrow(b0, nbat))
            del k, v, sk, sv
        caches.append((cache, btd, gtd))
        tails.append(tail)
    torch.cuda.synchronize()
    return caches, tails, bits


def decode_measure(args, w, dev, split: int, buffer_step: bool = False):
    """Times turbo_attn_decode on a decode workload (two cache copies used
    alternately); returns the timing, the roofline and the output."""
    import torch

    import paper_2412_08585_amd as ta
    from paper_2412_08585_amd import workloads as W
    B, Hq, Hkv, N = w.B, w.Hq, w.Hkv, w.N
    ncopy = 2
    caches, tails, bits = build_decode_caches(w, dev, ncopy)
    q = W.decode_query(w, device=dev)
    sl = torch.full((B,), N, dtype=torch.int32, device=dev)
    if split < 0:
        split = ta.decode_auto_split(B, Hq, Hkv, w.max_groups)
    ws = ta.decode_workspace(B, Hq, Hkv, w.max_groups, split, dev)
    o = torch.empty_like(q)
    it = [0]

    def run():
        cache, btd, gtd = caches[it[0] % ncopy]
        it[0] += 1
        ta.turbo_attn_decode(q, cache, sl, btd, gtd, w.sm_scale, split, workspace=ws, out=o)

    out = {"run": run, "q": q, "o": o, "split": ta.decode_split(N, split), "bits": bits}
    if args.only:
        return out
    ramp_clocks(run)
    for _ in range(args.warmup):
        run()
    ts = launch_times(run, max(args.steps, 20))
    ms, mean = stats(ts)
    kv_bytes = sum(decode_bytes_per_token(int(bits[h])) for h in range(Hkv)) * B * N
    qo_bytes = B * Hq * 128 * 2 * 2
    gbs = (kv_bytes + qo_bytes) / (ms * 1e-3) / 1e9
    out.update(ms=ms, mean_ms=mean, kv_bytes=kv_bytes, qo_bytes=qo_bytes, gbs=gbs,
               roofline={"kernel": "k_attn_decode", "bound": "hbm", "achieved": round(gbs, 1),
                         "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(gbs / PEAK_HBM_GBS, 4),
                         "traffic": measured_traffic("k_attn_decode", w.name),
                         "per_launch_bytes": kv_bytes + qo_bytes})
    run()  # o of the first copy (both copies hold the same cache)
    torch.cuda.synchronize()
    # the paper's comparison measured here: fp16 attention of the same query
    # over an fp16 cache of the same shape (random values: only time is taken)
    kf = torch.randn(B, Hkv, N, 128, dtype=torch.float16, device=dev)
    vf = torch.randn_like(kf)
    here = fp16_attention_here(q[:, :, None], kf, vf, False, max(args.steps, 20), ms,
                               f"{w.name} decode (attn_decode + merge)")
    del kf, vf
    if here is not None:
        # a decode reads its cache once: the fp16 cache at the HBM peak bounds
        # any fp16 decode kernel, the library's included
        fp16_bytes = 2 * B * Hkv * N * 128 * 2 + qo_bytes
        bound_ms = fp16_bytes / (PEAK_HBM_GBS * 1e9) * 1e3
        here.update(library_GBs=round(fp16_bytes / (here["ms"] * 1e-3) / 1e9, 1),
                    fp16_bytes=fp16_bytes, fp16_hbm_bound_ms=round(bound_ms, 4),
                    turbo_speedup_vs_fp16_hbm_bound=round(bound_ms / ms, 3),
                    note="the library's kernel is not a split-KV decode kernel; the fp16 bound "
                         "(the fp16 cache read once at 8 TB/s) is the fair comparison")
    out["fp16_here"] = here
    if buffer_step:
        # the Sec. 3.3 decoding step: append the new token's K/V to the int8
        # buffer, then attend the cache plus the buffer (not the headline)
        g = torch.Generator(device="cpu").manual_seed(7)
        knew = torch.randn(B, Hkv, 128, generator=g).half().to(dev)
        vnew = torch.randn(B, Hkv, 128, generator=g).half().to(dev)
        sl1 = torch.full((B,), N + 1, dtype=torch.int32, device=dev)
        ws1 = ta.decode_workspace(B, Hq, Hkv, w.max_groups, split, dev, with_tail=True)
        o1 = torch.empty_like(q)
        it1 = [0]

        def run_append():
            cache, btd, gtd = caches[it1[0] % ncopy]
            ta.turbo_append_kv(knew, vnew, sl, cache, tails[it1[0] % ncopy], btd, gtd)

        def run_decode_buf():
            cache, btd, gtd = caches[it1[0] % ncopy]
            ta.turbo_attn_decode(q, cache, sl1, btd, gtd, w.sm_scale, split, workspace=ws1,
                                 out=o1, tail=tails[it1[0] % ncopy])
            it1[0] += 1

        ms_app, _ = stats(launch_times(run_append, args.steps))
        ms_buf, _ = stats(launch_times(lambda: (run_append(), run_decode_buf()), args.steps))
        out["buffer_step"] = {
            "note": "Sec. 3.3 decoding step: turbo_append_kv of the new token, then "
                    "turbo_attn_decode over the cache plus the int8 buffer (seq_len N+1)",
            "append_ms": round(ms_app, 4), "step_ms": round(ms_buf, 4),
            "GB/s": round((kv_bytes + qo_bytes) / (ms_buf * 1e-3) / 1e9, 1)}
    del caches, tails, ws
    return out


def decode_error(w, dec, dev):
    """rel-L2 against exact fp64 attention of the decode output of one
    sequence over all its cached tokens, for one int4 and (mixed caches) one
    int2 KV head, with the oracle's decomposition."""
    import oracle
    import torch

    from paper_2412_08585_amd import workloads as W
    bits = dec["bits"]
    heads = [int(np.argmax(bits == 4))] + ([int(np.argmax(bits == 2))] if (bits == 2).any() else [])
    res = {"metric": "rel-L2 over the query heads of the KV head and channels"}
    for h in heads:
        ku, vu = W.unit_kv(w, 0, h, device=dev)
        ks, vs = ku[None, None].cpu(), vu[None, None].cpu()
        qs = dec["q"][0:1, h * w.G:(h + 1) * w.G].cpu()
        got = dec["o"][0:1, h * w.G:(h + 1) * w.G].float().cpu().numpy()
        ref = oracle.quantize_kv(ks, vs, [int(bits[h])])
        ex, _ = oracle.attn_exact(qs[:, :, None], ks, vs, float(np.float32(w.sm_scale)), False)
        res[f"kv_head_{h}_int{int(bits[h])}"] = error_decomposition(
            lambda qu, sa: oracle.attn_decode(qs, ref, [w.N], w.sm_scale, split=dec["split"],
                                              quant=qu, sas=sa)[0], ex[:, :, 0], got)
    res["sample"] = f"sequence 0, {w.N} cached tokens, chunks of {dec['split']} groups"
    return res


def bench_decode(args, w):
    """Decode-only workload: the compressed cache (built once, untimed) is read
    by turbo_attn_decode for one new query per sequence.  Two cache copies
    with their own page/group tables are used alternately so that timed calls
    stream from HBM rather than from the 256 MB MALL."""
    import torch
    dev = torch.device("cuda:0")
    B, Hq, Hkv, N = w.B, w.Hq, w.Hkv, w.N
    dec = decode_measure(args, w, dev, args.kv_split_groups, buffer_step=True)
    if args.only:
        for _ in range(args.warmup + args.steps):
            dec["run"]()
        torch.cuda.synchronize()
        print(json.dumps({"only": "decode", "launches": args.warmup + args.steps}))
        return
    ceil = measured_ceilings(dev)
    ops = 4.0 * 128 * N * B * Hq
    result = {
        "metric": "attention TOPS (prefill) & HBM GB/s (decode), % of MI355X roofline",
        "value": round(dec["gbs"], 1), "unit": "GB/s", "n_gpus": 1, "steps": max(args.steps, 20),
        "warmup": args.warmup, "ms_per_step": round(dec["ms"], 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int8",
        "data": "synthetic (seeded N(0,1) fp16 K/V with 4 K outlier channels x10, "
                "compressed before timing; no weights)",
        "config": {"workload": w.name, "batch": B, "q_heads": Hq, "kv_heads": Hkv, "kv_len": N,
                   "head_dim": 128, "kv_cache": w.bits,
                   "head_bits": [int(x) for x in dec["bits"]], "page_tokens": 16,
                   "kv_split_groups": dec["split"], "cache_copies": 2,
                   "timing": "median of per-launch HIP events"},
        "attention_TOPS": round(ops / (dec["ms"] * 1e-3) / 1e12, 3),
        "roofline": dict(dec["roofline"], frac_of_measured_ceiling=round(
            dec["gbs"] / ceil["hbm_read_GBs"], 4), mean_ms=round(dec["mean_ms"], 4)),
        "ceilings_measured": ceil,
        "buffer_step": dec["buffer_step"],
        "paper_context": (PAPER_CONTEXT if dec["fp16_here"] is None
                          else dict(PAPER_CONTEXT, fp16_decode_here=dec["fp16_here"])),
    }
    if not args.no_error:
        result["error_vs_fp64"] = {"decode": decode_error(w, dec, dev)}

    # ---- CPU oracle: the oracle's caches of the first sequences (built
    # untimed, like the GPU cache), attended until the sample time is spent ----
    if not args.no_cpu_baseline:
        import oracle

        from paper_2412_08585_amd import workloads as W
        qc = dec["q"].cpu()
        got = dec["o"].float().cpu().numpy()
        bits = dec["bits"]
        refs, t0 = [], time.perf_counter()
        while len(refs) < B and time.perf_counter() - t0 < 15.0:
            b = len(refs)
            kv = [W.unit_kv(w, b, h, device=dev) for h in range(Hkv)]
            ref = oracle.quantize_kv(torch.stack([a for a, _ in kv])[None].cpu(),
                                     torch.stack([c for _, c in kv])[None].cpu(), bits)
            del ref["k8"], ref["v8"], kv
            refs.append(ref)
        passes, dt, err = 0, 0.0, 0.0
        while passes == 0 or dt < CPU_SAMPLE_SECONDS:
            for b, ref in enumerate(refs):
                t1 = time.perf_counter()
                ro, _ = oracle.attn_decode(qc[b:b + 1], ref, [N], w.sm_scale, split=dec["split"])
                dt += time.perf_counter() - t1
                rowmax = np.abs(ro[0]).max(axis=-1, keepdims=True)
                err = max(err, float(np.max(np.abs(got[b] - ro[0]) / rowmax)))
            passes += 1
        nseq = len(refs) * passes
        result["cpu_baseline"] = {
            "value": round((dec["kv_bytes"] + dec["qo_bytes"]) * nseq / B / dt / 1e9, 3),
            "unit": "GB/s", "cores": min(oracle.num_threads(), Hq), "kind": "oracle",
            "cpu_model": cpu_model(), "host_threads": os.cpu_count(),
            "sample": f"{len(refs)} of {B} sequences (oracle cache built untimed), each attended "
                      f"{passes} times, {dt:.1f} s"}
        result["parity"] = {"max_err_vs_oracle_rel_rowmax": err, "sample_sequences": len(refs)}
    print(json.dumps(result), flush=True)


def bench_softmax(args, w):
    """Algorithm 3 on its own: turbo_sas_softmax over the B*Hq*N score rows
    of N keys (fp32 in, fp32 out, resident in HBM)."""
    import torch

    import paper_2412_08585_amd as ta
    from paper_2412_08585_amd import workloads as W

    dev = torch.device("cuda:0")
    x = W.softmax_scores(w, device=dev)
    y = torch.empty_like(x)
    rows, cols = x.shape
    run = lambda: ta.turbo_sas_softmax(x, out=y)
    ramp_clocks(run)
    for _ in range(args.warmup):
        run()
    ms, _ = stats(launch_times(run, args.steps))
    nbytes = rows * cols * 4 * 2               # fp32 read once, written once
    gbs = nbytes / (ms * 1e-3) / 1e9
    result = {
        "metric": "attention TOPS (prefill) & HBM GB/s (decode), % of MI355X roofline",
        "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": f"synthetic (seeded N(0, {W.SCORE_STD:.3f}^2) fp32 score rows)",
        "config": {"workload": w.name, "rows": rows, "cols": cols},
        "roofline": {"kernel": "k_sas_softmax_block<4>", "bound": "hbm", "achieved": round(gbs, 1),
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "traffic": None, "per_launch_bytes": nbytes},
    }
    if not args.no_cpu_baseline:
        import oracle

        def run_rows(lo, hi):
            xs = x[lo:hi].cpu().numpy()
            t0 = time.perf_counter()
            oracle.sas_softmax_rows(xs)
            return time.perf_counter() - t0

        n, dt = cpu_sample(run_rows, rows, 4096)
        result["cpu_baseline"] = {"value": round(n * cols * 8 / dt / 1e9, 3), "unit": "GB/s",
                                  "cores": 1, "kind": "oracle",
                                  "sample": f"{n} of {rows} rows, {dt:.1f} s"}
    print(json.dumps(result), flush=True)


def bench_projection(args, w):
    """The QKV projection with FlashQ fused (turbo_qkv_project: fp16 GEMM on
    the MFMA, FlashQ step 1 of Q/K/V and step 2 + cache write of K/V in the
    epilogue), inputs resident in HBM."""
    import torch

    import paper_2412_08585_amd as ta
    from paper_2412_08585_amd import workloads as W

    dev = torch.device("cuda:0")
    B, N, D, Hq, Hkv = w.B, w.N, w.hidden, w.Hq, w.Hkv
    F = (Hq + 2 * Hkv) * 128
    x, wt = W.projection_inputs(w, device=dev)
    bits = W.head_bits(w)
    bt, gt = W.tables(w)
    cache = ta.PagedKVCache(bt.size, gt.size, bits, dev)
    btd, gtd = torch.from_numpy(bt).to(dev), torch.from_numpy(gt).to(dev)
    outs = ta.turbo_qkv_project(x, wt, Hq, Hkv, cache, btd, gtd)
    run = lambda: ta.turbo_qkv_project(x, wt, Hq, Hkv, cache, btd, gtd, out=outs)
    stream = torch.cuda.current_stream()

    def time_loop(fn, iters):
        ramp_clocks(fn)
        for _ in range(args.warmup):
            fn()
        return stats(launch_times(fn, iters))[0]

    ms = time_loop(run, args.steps)
    # context: the library fp16 GEMM alone (no quantization, fp16 output)
    y = torch.empty(B * N, F, dtype=torch.float16, device=dev)
    x2 = x.view(B * N, D)
    ms_lib = time_loop(lambda: torch.matmul(x2, wt.t(), out=y), args.steps)
    flops = 2.0 * B * N * D * F
    tflops = flops / (ms * 1e-3) / 1e12
    result = {
        "metric": "attention TOPS (prefill) & HBM GB/s (decode), % of MI355X roofline",
        "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f16",
        "data": "synthetic (seeded N(0,1) fp16 hidden states, N(0,1/D) fp16 weights with 4 "
                "outlier channels per key head x10)",
        "config": {"workload": w.name, "batch": B, "seq_len": N, "hidden": D, "q_heads": Hq,
                   "kv_heads": Hkv, "head_dim": 128, "kv_cache": w.bits},
        "library_gemm_fp16_out": {"ms": round(ms_lib, 4),
                                  "TFLOP/s": round(flops / (ms_lib * 1e-3) / 1e12, 2),
                                  "note": "torch.matmul X W^T alone, fp16 output, no FlashQ"},
        "roofline": {"kernel": "k_qkv_project", "bound": "mfma", "achieved": round(tflops, 2),
                     "peak": PEAK_FP16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tflops / PEAK_FP16_TFLOPS, 4), "traffic": None,
                     "per_launch_flops": flops},
    }
    if not args.no_cpu_baseline:
        import oracle
        ws = wt.float().cpu().numpy()
        xt = x.reshape(B * N, D)

        def run_tokens(lo, hi):
            xs = xt[lo:hi].float().cpu().numpy()[None]
            t0 = time.perf_counter()
            oracle.qkv_project(xs, ws, Hq, Hkv, bits)
            return time.perf_counter() - t0

        n, dt = cpu_sample(run_tokens, B * N, 1024)
        result["cpu_baseline"] = {"value": round(2.0 * n * D * F / dt / 1e12, 5), "unit": "TFLOP/s",
                                  "cores": oracle.num_threads(), "kind": "oracle",
                                  "sample": f"{n} of {B * N} tokens, {dt:.1f} s"}
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
