"""Decode-attention throughput of the D-Quant hot path on one MI355X.

    python bench.py [--gpus 1] [--steps 100] [--warmup 10] [--workload b16_t32k]
                    [--variant paper|literal] [--bpe 2.26] [--precision 12] [--no-cpu-baseline]

A step is one decode-attention pass over the whole compressed cache of the
workload: batch 16 x 32768 tokens x 8 KV heads (32 query heads, head_dim 128)
with 36-byte key and value records (2.25 bits per element).  The cache is
filled once by the encoder, one prefill append of all B x T tokens per tensor
(timed separately and reported under "encode"), the raw K/V are freed, and
the timed region holds only the decode-attention steps with the compressed
cache resident in HBM.  Prints one JSON line.

--workload b16_t32k_tok runs the paper's default grouping instead: one stream
of 1024 values per token over the 8 KV heads (331 + 4 and 231 + 4 byte
records, 8 / 6 levels), decoded by the per-token kernel.

Other modes (for the profiles under profiles/):
    --copy-calibration BYTES   time a plain device copy of BYTES bytes
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "KV tokens/s + achieved HBM GB/s, D-Quant decode attention at 2.26 bits/elem"
HBM_PEAK_GBS = 8000.0
# VALU issue peak: 256 CUs x 4 SIMDs, a wave64 instruction occupies a 16-lane
# SIMD for 4 cycles, 2.4 GHz
VALU_PEAK_GINST = 256 * 4 / 4 * 2.4
# GPU time of the untimed decode steps run between the warmup and the timed region
SETTLE_MS = 50.0
# committed counter summaries: (workload, variant) -> (summary, kernel sources it was taken from)
_CSRC = os.path.join(ROOT, "paper_2609_19880_amd", "csrc")
COUNTER_SUMMARIES = {
    ("b16_t32k", "paper"): (os.path.join(ROOT, "profiles", "attn_partial_b16_t32k_pmc.md"),
                            [os.path.join(_CSRC, f) for f in ("dq_decode.hip", "dq_attn.h", "dq_common.h", "dq_internal.h")]),
    ("b16_t32k_tok", "paper"): (os.path.join(ROOT, "profiles", "attn_token_b16_t32k_tok_pmc.md"),
                                [os.path.join(_CSRC, f)
                                 for f in ("dq_token.hip", "dq_attn.h", "dq_common.h", "dq_internal.h")]),
}

# encoder counters: summary, sources, streams per dispatch they were taken over
ENCODE_SUMMARY = (os.path.join(ROOT, "profiles", "encode_kernel_b16_t32k_pmc.md"),
                  [os.path.join(_CSRC, f) for f in ("dq_encode.hip", "dq_common.h", "dq_internal.h")],
                  16 * 32768 * 8)


# The paper's own system figures (Sec. 5.3 and its efficiency figure; setup
# of Sec. 5.1), quoted with the hardware they were measured on.  They are
# end-to-end serving figures of a whole model; the paper gives no kernel
# time or bandwidth, so nothing here is a baseline for "value".
PAPER_CONTEXT = {
    "source": "Sec. 5.3 (efficiency figure and text); operating point of Sec. 5.1",
    "hardware": "one NVIDIA H20 96 GB",
    "model": "Qwen3-8B",
    "kv_format": "2.26 bits per value: per token one 1024-value stream, K 331 B / V 231 B containers, "
                 "8 / 6 levels, alpha 1.4, newest 128 tokens kept in BF16",
    "decode_tokens_per_s": {"d_quant": 563.6, "bf16": 159.5,
                            "setting": "8K prompt, each format at its largest batch that fits "
                                       "(D-Quant 128; BF16 runs out of memory at 64)"},
    "throughput_gain": 3.5,
    "peak_memory_gib": {"d_quant_batch_128_8k_prompt": 49.4},
    "kv_memory_reduction": {"factor": 7, "setting": "1K prompt decoded to 64K tokens at batch 1"},
    "small_batch": "D-Quant decodes slower than BF16 at small batch (entropy decoding costs compute)",
}


def _args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="b16_t32k")
    ap.add_argument("--variant", default="paper", choices=["paper", "literal"])
    ap.add_argument("--bpe", type=float, default=None)
    ap.add_argument("--precision", type=int, default=None, help="rANS precision p of both tables (default 12)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of a HIP graph captured from one step instead of eager launches")
    ap.add_argument("--copy-calibration", type=int, default=0)
    ap.add_argument("--compare-bf16", action="store_true",
                    help="also time the BF16 comparator (uncompressed cache of the same shape)")
    ap.add_argument("--compare-fixed", action="store_true",
                    help="also time the fixed-width comparator (App. B: 36-byte INT2 records of the same workload)")
    ap.add_argument("--residual", type=int, default=0,
                    help="also attend over this many raw BF16 tokens per sequence (residual window, <= 255)")
    ap.add_argument("--residual-two-call", action="store_true",
                    help="with --residual: the window as its own launch before the merge, instead of the "
                         "one-launch window + merge")
    return ap.parse_args()


def time_steps(calls, steps: int, warmup: int, graph: bool = False):
    """Time `steps` decode steps, each the launches in `calls` in order on the
    current stream (graph: one replay of a HIP graph captured from them).  The
    timed region holds only the steps, bracketed by a synchronize and one HIP
    event on each side (no events between kernels).  A second pass, eager,
    with an event pair around every launch gives each launch's mean duration.
    Returns (ms per step, [mean ms per call], wall seconds of the timed
    region, settle steps run after the warmup)."""
    import torch

    def step():
        for c in calls:
            c()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    # Settle: a decode launch right after an idle spell runs about 9 % slower
    # until the GPU has been kept busy for some 20 ms (b16_t32k: 0.366 ms per
    # partial launch after 5 warmup steps, 0.338 after 50, 0.335 after 200).
    # Untimed steps, eight at a time, continue after the warmup until they
    # have filled SETTLE_MS of GPU time, so that the timed steps see the
    # steady state of a serving loop; the count is reported beside `warmup`.
    settle = 0
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    busy = 0.0
    while busy < SETTLE_MS and settle < 100000:
        n = 8
        s0.record()
        for _ in range(n):
            step()
        s1.record()
        s1.synchronize()
        busy += s0.elapsed_time(s1)
        settle += n
    if graph:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        step = g.replay
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    step_ms = e0.elapsed_time(e1) / steps
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in calls]
          for _ in range(steps)]
    for i in range(steps):
        for j, c in enumerate(calls):
            ev[i][j][0].record()
            c()
            ev[i][j][1].record()
    torch.cuda.synchronize()
    per_call = [sum(ev[i][j][0].elapsed_time(ev[i][j][1]) for i in range(steps)) / steps
                for j in range(len(calls))]
    return step_ms, per_call, wall, settle


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor()


def copy_calibration(nbytes: int, steps: int):
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    print(json.dumps({"mode": "copy_calibration", "bytes": nbytes, "ms_per_copy": ms,
                      "gbs_read_plus_write": 2 * nbytes / ms / 1e6}))


def _summary_text(summary: str, sources):
    """The text of a committed rocprofv3 counter summary if the kernel sources
    still hash to the value it records (else None)."""
    import hashlib
    import re
    if not os.path.exists(summary):
        return None
    text = open(summary).read()
    h = hashlib.sha256()
    for f in sources:
        h.update(open(f, "rb").read())
    m_sha = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text)
    return text if m_sha and m_sha.group(1) == h.hexdigest() else None


def counter_figures(workload: str, variant: str):
    """HBM bytes and VALU instructions per partial launch from the committed
    rocprofv3 counter summary, if it was taken on this workload from the
    kernel sources as they are now (else None)."""
    import re
    if (workload, variant) not in COUNTER_SUMMARIES:
        return None
    text = _summary_text(*COUNTER_SUMMARIES[(workload, variant)])
    if text is None:
        return None
    m_tr = re.search(r"traffic_bytes_per_launch:\s*(\d+)", text)
    m_valu = re.search(r"\|\s*SQ_INSTS_VALU\s*\|\s*([\d,]+)", text)
    if not (m_tr and m_valu):
        return None
    return int(m_tr.group(1)), int(m_valu.group(1).replace(",", ""))


def encode_valu_per_stream(wl, variant: str):
    """VALU instructions per encoded stream from the committed encoder counter
    summary (taken on 36-byte, 6-level, p 12 per-(token, KV head) records),
    for workloads that encode with that coding (else None)."""
    import re
    summary, sources, streams = ENCODE_SUMMARY
    c = wl.k
    if (wl.streams != "head" or variant != "paper" or wl.v != c or wl.head_dim != 128
            or (c.record_bytes, c.levels, c.precision, c.alpha) != (36, 6, 12, 1.4)):
        return None
    text = _summary_text(summary, sources)
    m = None if text is None else re.search(r"\|\s*SQ_INSTS_VALU\s*\|\s*([\d,]+)\s*\|", text)
    return None if m is None else int(m.group(1).replace(",", "")) / streams


CPU_SECONDS = 10.0          # wall time each CPU worker spends in the timed oracle loop


def _pool_size() -> int:
    """Host cores the CPU baseline uses: the cores this process may run on,
    at most 16 (the host share of one GPU)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _oracle_tables(wl):
    from oracle import tables
    c = [(wl.k.n, wl.k.levels, wl.k.precision, wl.k.alpha, wl.k.record_bytes),
         (wl.v.n, wl.v.levels, wl.v.precision, wl.v.alpha, wl.v.record_bytes)]
    return [tables.build_tables(*x) for x in c]


def _cpu_encode_part(args):
    """Worker: the oracle's records of tokens [t0, t0 + n) of the sample (one
    KV head, or every head for per-token streams)."""
    wl, seed, T, t0, n = args
    from threadpoolctl import threadpool_limits
    import dq_workloads as wlmod
    from oracle import kv
    otk, otv = _oracle_tables(wl)
    one = wl.with_context(T, batch=1)
    tok = wl.streams == "token"
    with threadpool_limits(limits=1):
        k = wlmod.bf16_bits(wlmod.make_k(one, seed + 100))[:, t0:t0 + n]
        v = wlmod.bf16_bits(wlmod.make_v(one, seed + 100))[:, t0:t0 + n]
        if tok:
            krec, mq, ms, _ = kv.encode_keys_tokenwise(k, otk)
            vrec, _ = kv.encode_values_tokenwise(v, otv)
        else:
            krec, mq, ms, _ = kv.encode_keys(k[:, :, :1], otk)
            vrec, _ = kv.encode_values(v[:, :, :1], otv)
    return krec, mq, ms, vrec


def _cpu_attend_loop(args):
    """Worker: the oracle's decode attention over the sample (rANS decode of
    every key and value record, fp64 folded attention), repeated for `secs`
    seconds on one thread.  Returns (repetitions, seconds)."""
    wl, krec, mq, ms, vrec, q, T, secs = args
    import numpy as np
    from threadpoolctl import threadpool_limits
    from oracle import attention, kmean, kv
    otk, otv = _oracle_tables(wl)
    H = wl.kv_heads
    reps, t0 = 0, time.perf_counter()
    with threadpool_limits(limits=1):
        while True:
            ksym, ks, ko, _ = kv.decode_records(krec, otk, wl.k.n)
            vsym, vs, vo, _ = kv.decode_records(vrec, otv, wl.v.n)
            if wl.streams == "token":
                ksym, ks, ko = kv.tokenwise_as_heads(ksym, ks, ko, H)
                vsym, vs, vo = kv.tokenwise_as_heads(vsym, vs, vo, H)
            attention.attention_folded(kv.bf16_to_f64(q), ksym, ks, ko, kmean.dequantize_mean(mq, ms),
                                       vsym, vs, vo, [T], wl.gqa, 1 / np.sqrt(wl.head_dim))
            reps += 1
            el = time.perf_counter() - t0
            if el > secs:
                return reps, el


def cpu_baseline(wl, seed: int):
    """The CPU oracle's decode attention, on a pool of one process per host
    core (at most 16), every process single-threaded.  The sample is one
    (sequence, KV head) slice at full context (per-token streams: the first
    4096 tokens of one sequence, every head), encoded by the oracle across the
    pool; each process then decodes and attends over it for CPU_SECONDS and
    the aggregate rate is scaled to a whole step."""
    import multiprocessing as mp
    import numpy as np
    import dq_workloads as wlmod

    tok = wl.streams == "token"
    T = min(4096, wl.context) if tok else wl.context
    n = _pool_size()
    parts = max(1, min(n, T // 128))
    step = -(-T // parts // 128) * 128
    spans = [(t0, min(step, T - t0)) for t0 in range(0, T, step)]
    one = wl.with_context(T, batch=1)
    q = wlmod.bf16_bits(wlmod.make_q(one, seed + 100))
    if not tok:
        q = q[:, : wl.gqa]
    with mp.get_context("spawn").Pool(n) as pool:
        enc = pool.map(_cpu_encode_part, [(wl, seed, T, t0, m) for t0, m in spans])
        krec = np.concatenate([e[0] for e in enc], axis=1 if tok else 2)
        mq = np.concatenate([e[1] for e in enc], axis=2)
        ms = np.concatenate([e[2] for e in enc], axis=2)
        vrec = np.concatenate([e[3] for e in enc], axis=1 if tok else 2)
        w0 = time.perf_counter()
        runs = pool.map(_cpu_attend_loop, [(wl, krec, mq, ms, vrec, q, T, CPU_SECONDS)] * n, chunksize=1)
        wall = time.perf_counter() - w0
    samples_per_s = sum(r / el for r, el in runs)
    reps = sum(r for r, _ in runs)
    if tok:
        scale = wl.batch * wl.context / T
        what = (f"oracle rANS decode of the per-token K and V records plus fp64 folded attention for "
                f"{T} tokens of one sequence (all {wl.kv_heads} KV heads, {wl.q_heads} query heads)")
    else:
        scale = wl.batch * wl.kv_heads
        what = (f"oracle rANS decode of the K and V records plus fp64 folded attention for one "
                f"(sequence, KV head) slice: {T} tokens, {wl.gqa} query heads")
    step_s = scale / samples_per_s
    return {"value": wl.batch * wl.context / step_s, "unit": "tokens/s", "cores": n, "kind": "oracle",
            "sample": f"{what}; {n} single-threaded processes, {reps} repetitions in {wall:.1f} s "
                      f"({samples_per_s:.2f} samples/s together), scaled x{scale:.0f} to a step; numpy on "
                      f"{_cpu_model()} ({os.cpu_count()} host cores visible)"}


def fill_cache(wl, seed: int, dev):
    """Tables and a compressed cache holding the whole workload, filled by one
    prefill append per tensor: dq_encode_kv (or its per-token form) over all
    B x T tokens at once, timed with HIP events.  Sequence b's inputs come
    from the seeded generators with seed 1000 seed + b on the device.
    Returns (tk, tv, cache, encode_ms)."""
    import torch
    import dq_workloads as wlmod
    import paper_2609_19880_amd as dq

    B, T, Hq, Hkv, d = wl.batch, wl.context, wl.q_heads, wl.kv_heads, wl.head_dim
    tok = wl.streams == "token"
    tk = dq.Tables(wl.k.n, wl.k.levels, wl.k.precision, wl.k.record_bytes, wl.k.alpha)
    tv = dq.Tables(wl.v.n, wl.v.levels, wl.v.precision, wl.v.record_bytes, wl.v.alpha)
    cache = (dq.TokenKVCache if tok else dq.KVCache)(B, Hkv, Hq, T, tk, tv, device=dev)
    enc = dq.dq_encode_kv_token if tok else dq.dq_encode_kv
    k = torch.cat([wlmod.make_k(wl, seed * 1000 + b, device=dev, batch=1) for b in range(B)])
    v = torch.cat([wlmod.make_v(wl, seed * 1000 + b, device=dev, batch=1) for b in range(B)])
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    enc(tk, k, 0, T, cache.k_records, cache.k_mean_q, cache.k_mean_scale, cache.status)
    enc(tv, v, 0, T, cache.v_records, None, None, cache.status)
    e1.record()
    torch.cuda.synchronize()
    del k, v
    return tk, tv, cache, e0.elapsed_time(e1)


def step_inputs(wl, seed: int, dev):
    """Query (seeded), full-length sequence lengths and the output buffer."""
    import torch
    import dq_workloads as wlmod
    q = wlmod.make_q(wl, seed, device=dev)
    seq = torch.full((wl.batch,), wl.context, dtype=torch.int32, device=dev)
    out = torch.empty((wl.batch, wl.q_heads, wl.head_dim), dtype=torch.float32, device=dev)
    return q, seq, out


def decode_step(tk, tv, cache, q, seq, out, ring=None):
    """One step: split-K partials over the whole cache (and the residual
    window's partial, if a ring is given), then the merge."""
    import paper_2609_19880_amd as dq
    cache.partial(q, seq)
    if ring is not None:
        dq.dq_decode_attention_residual(q, ring[0], ring[1], seq, ring[2], cache.t_cap, cache.workspace)
    cache.merge(seq, out)


def bf16_comparator(wl, a, q, seq, out, ws, alg_bytes):
    """The same decode step over an uncompressed BF16 cache of the same shape
    (random contents), timed like the compressed one."""
    import torch
    import paper_2609_19880_amd as dq
    B, T, Hq, Hkv, d = wl.batch, wl.context, wl.q_heads, wl.kv_heads, wl.head_dim
    g = torch.Generator(device="cuda")
    g.manual_seed(a.seed * 7 + 11)
    k = torch.randn((B, Hkv, T, d), generator=g, device="cuda").to(torch.bfloat16)
    v = torch.randn((B, Hkv, T, d), generator=g, device="cuda").to(torch.bfloat16)
    sms, (pms, _), _, _ = time_steps([lambda: dq.dq_bf16_decode_attention_partial(q, k, v, seq, ws),
                                   lambda: dq.dq_decode_attention_merge(B, Hq, Hkv, seq, T, ws, out)],
                                  a.steps, a.warmup)
    nbytes = 2 * B * Hkv * T * d * 2
    del k, v
    torch.cuda.empty_cache()
    return {"ms_per_step": sms, "tokens_per_s": B * T / (sms * 1e-3), "partial_ms": pms,
            "bytes_per_step": nbytes, "gbs": nbytes / (pms * 1e-3) / 1e9,
            "hbm_frac": nbytes / (pms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "kv_bytes_ratio": nbytes / alg_bytes}


def fixed_comparator(wl, a, q, seq, out, ws):
    """The same decode step over fixed-width records of the same size (App. B
    comparator: 36-byte records of 2-bit levels), encoded from the same seeded
    inputs and timed like the compressed path."""
    import torch
    import dq_workloads as wlmod
    import paper_2609_19880_amd as dq
    B, T, Hq, Hkv, d = wl.batch, wl.context, wl.q_heads, wl.kv_heads, wl.head_dim
    C = 36
    kr = torch.empty((B, Hkv, T, C), dtype=torch.uint8, device="cuda")
    vr = torch.empty_like(kr)
    mq = torch.empty((B, Hkv, T // 128, d), dtype=torch.int8, device="cuda")
    ms = torch.empty((B, Hkv, T // 128), dtype=torch.int16, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    for b in range(B):
        k = wlmod.make_k(wl, a.seed * 1000 + b, device="cuda", batch=1)
        v = wlmod.make_v(wl, a.seed * 1000 + b, device="cuda", batch=1)
        dq.dq_encode_kv_fixed(d, C, k, 0, T, kr[b:b + 1], mq[b:b + 1], ms[b:b + 1], status)
        dq.dq_encode_kv_fixed(d, C, v, 0, T, vr[b:b + 1], None, None, status)
        del k, v
    torch.cuda.synchronize()
    if int(status.item()):
        raise RuntimeError(f"fixed-width encoder status {int(status.item())}")
    sms, (pms, _), _, _ = time_steps([lambda: dq.dq_decode_attention_fixed_partial(q, kr, mq, ms, vr, seq, ws),
                                   lambda: dq.dq_decode_attention_merge(B, Hq, Hkv, seq, T, ws, out)],
                                  a.steps, a.warmup)
    nbytes = B * Hkv * T * (2 * C + (d + 2) / 128)
    del kr, vr, mq, ms
    torch.cuda.empty_cache()
    return {"record_bytes": C, "bits_per_symbol": 2, "ms_per_step": sms, "tokens_per_s": B * T / (sms * 1e-3),
            "partial_ms": pms, "bytes_per_step": nbytes, "gbs": nbytes / (pms * 1e-3) / 1e9,
            "hbm_frac": nbytes / (pms * 1e-3) / 1e9 / HBM_PEAK_GBS}


def main():
    a = _args()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only: the decode-attention path has no multi-GPU leg "
              f"(asked for --gpus {a.gpus})", file=sys.stderr)
        sys.exit(2)
    import torch

    if a.copy_calibration:
        copy_calibration(a.copy_calibration, a.steps)
        return

    import dq_workloads as wlmod
    import paper_2609_19880_amd as dq

    wl = wlmod.workload(a.workload, a.variant, a.bpe) if a.workload == "b1_t128k" else \
        wlmod.workload(a.workload, a.variant)
    # the committed counter summaries hold for the workload's own precision
    own_precision = a.precision is None or (a.precision == wl.k.precision and a.precision == wl.v.precision)
    if a.precision is not None:
        from dataclasses import replace
        wl = replace(wl, k=replace(wl.k, precision=a.precision), v=replace(wl.v, precision=a.precision))
    tok = wl.streams == "token"
    dev = torch.device("cuda")
    B, T, Hq, Hkv, d = wl.batch, wl.context, wl.q_heads, wl.kv_heads, wl.head_dim
    tk, tv, cache, enc_ms = fill_cache(wl, a.seed, dev)
    status = int(cache.status.item())
    if status:
        raise RuntimeError(f"encoder status {status}")
    torch.cuda.empty_cache()
    q, seq, out = step_inputs(wl, a.seed, dev)

    ring = None
    if a.residual:
        if not 0 < a.residual < 256:
            raise SystemExit("--residual must be in 1..255")
        # the newest tokens of every sequence, raw, in the ring slots that follow
        # the compressed ones
        g = torch.Generator(device=dev)
        g.manual_seed(a.seed * 7 + 5)
        rk = torch.randn((B, Hkv, 256, d), generator=g, device=dev).to(torch.bfloat16)
        rv = torch.randn((B, Hkv, 256, d), generator=g, device=dev).to(torch.bfloat16)
        rl = torch.full((B,), a.residual, dtype=torch.int32, device=dev)
        ring = (rk, rv, rl)

    calls = [lambda: cache.partial(q, seq)]
    if ring is not None and a.residual_two_call:
        calls.append(lambda: dq.dq_decode_attention_residual(q, ring[0], ring[1], seq, ring[2], T, cache.workspace))
        calls.append(lambda: cache.merge(seq, out))
    elif ring is not None:
        calls.append(lambda: dq.dq_decode_attention_merge_residual(q, ring[0], ring[1], seq, ring[2], T,
                                                                   cache.workspace, out))
    else:
        calls.append(lambda: cache.merge(seq, out))
    step_ms, per_call, wall, settle = time_steps(calls, a.steps, a.warmup, graph=a.graph)
    if int(cache.status.item()):
        raise RuntimeError(f"decode status {int(cache.status.item())}")
    partial_ms, merge_ms = per_call[0], per_call[-1]
    residual_ms = per_call[1] if ring is not None and a.residual_two_call else 0.0

    # algorithmic bytes of one partial launch: per (token, KV head) the two
    # records plus the amortized INT8 key mean and its fp16 scale (per token
    # for per-token streams: the two records plus the means of every head)
    if tok:
        per_unit = wl.k.record_bytes + wl.v.record_bytes + Hkv * (d + 2) / 128.0
        units = B * T
    else:
        per_unit = wl.k.record_bytes + wl.v.record_bytes + (d + 2) / 128.0
        units = B * T * Hkv
    alg_bytes = per_unit * units
    n_symbols = 2 * B * T * Hkv * d
    achieved = alg_bytes / (partial_ms * 1e-3) / 1e9
    tokens_s = B * (T + a.residual) / (step_ms * 1e-3)
    counters = counter_figures(wl.name, a.variant) if own_precision else None
    traffic = counters[0] if counters else None
    n_streams = 2 * B * T if tok else 2 * B * T * Hkv
    enc_vps = encode_valu_per_stream(wl, a.variant) if own_precision else None

    rec = {
        "metric": METRIC,
        "value": tokens_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "settle": {"steps": settle, "min_gpu_ms": SETTLE_MS,
                   "why": "untimed steps after the warmup until the GPU has been busy SETTLE_MS: "
                          "launches right after an idle spell run ~9 % slower"},
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "arithmetic": "rANS decode in 32-bit integers; q.k and p.v as int8 x int8 -> int32 MFMA on "
                      "three 8-bit digits of 22-bit fixed-point query / weight values (levels exact); "
                      "softmax, scales and merge in fp32; records stored as u8",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: batch {B} x context {T}, {Hq} query / {Hkv} KV heads, "
                               f"head_dim {d}, "
                               + (f"one stream of {wl.k.n} values per token, " if tok else "")
                               + f"K {wl.k.record_bytes} B / V {wl.v.record_bytes} B records "
                               f"({wl.k.bits_per_elem:.2f}/{wl.v.bits_per_elem:.2f} bits/elem), "
                               f"{wl.k.levels}/{wl.v.levels} levels, alpha {wl.k.alpha}/{wl.v.alpha}, "
                               f"p {wl.k.precision}",
                   "streams": "per token" if tok else "per (token, KV head)",
                   "variant": a.variant, "batch": B, "context": T, "q_heads": Hq, "kv_heads": Hkv,
                   "head_dim": d, "k_record_bytes": wl.k.record_bytes, "v_record_bytes": wl.v.record_bytes,
                   "k_levels": wl.k.levels, "v_levels": wl.v.levels, "residual_tokens": a.residual},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "traffic_unit": "HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "kernel": "attn_token_kernel" if tok else "attn_partial_kernel",
                     "alg_bytes_per_launch": alg_bytes,
                     "kernel_ms": partial_ms},
        "valu_issue": None if counters is None else {
            "bound": "alu", "achieved": counters[1] / (partial_ms * 1e-3) / 1e9,
            "peak": VALU_PEAK_GINST, "unit": "G wave64 VALU instructions/s",
            "frac": counters[1] / (partial_ms * 1e-3) / 1e9 / VALU_PEAK_GINST,
            "valu_insts_per_launch": counters[1],
            "valu_lane_ops_per_symbol": counters[1] * 64 / n_symbols},
        "merge_ms": merge_ms,
        "residual": None if ring is None else (
            {"tokens_per_sequence": a.residual, "form": "own launch, then the merge", "ms": residual_ms,
             "gbs": B * Hkv * a.residual * d * 2 * 2 / (residual_ms * 1e-3) / 1e9}
            if a.residual_two_call else
            {"tokens_per_sequence": a.residual, "form": "one launch with the merge (merge_ms)",
             "window_bytes": B * Hkv * a.residual * d * 2 * 2}),
        "wall_ms_per_step": wall * 1e3 / a.steps,
        "step_launch": "graph replay" if a.graph else "eager",
        "symbols_per_s": n_symbols / (step_ms * 1e-3),
        "encode": {"what": f"prefill append of {B} x {T} tokens, K and V, one encode call per tensor",
                   "ms": enc_ms, "tokens_per_s": B * T / (enc_ms * 1e-3),
                   "streams_per_s": n_streams / (enc_ms * 1e-3),
                   "input_gbs": 2 * B * T * Hkv * d * 2 / (enc_ms * 1e-3) / 1e9,
                   "valu_issue": None if enc_vps is None else {
                       "bound": "alu", "valu_insts_per_stream": enc_vps,
                       "achieved": enc_vps * n_streams / (enc_ms * 1e-3) / 1e9,
                       "peak": VALU_PEAK_GINST, "unit": "G wave64 VALU instructions/s",
                       "frac": enc_vps * n_streams / (enc_ms * 1e-3) / 1e9 / VALU_PEAK_GINST,
                       "note": "encode_kernel instructions over the whole append time (key means included)"}},
    }
    if a.compare_fixed:
        if tok or d != 128 or wl.gqa > 4:
            raise SystemExit("--compare-fixed runs on the per-(token, KV head) workloads with head_dim 128, G <= 4")
        rec["fixed_width_decode"] = fixed_comparator(wl, a, q, seq, out, cache.workspace)
    if a.compare_bf16:
        rec["bf16_decode"] = bf16_comparator(wl, a, q, seq, out, cache.workspace, alg_bytes)
    rec["paper_context"] = PAPER_CONTEXT
    if not a.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(wl, a.seed)
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
