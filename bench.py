#!/usr/bin/env python3
"""Encoder-forward benchmark on one MI355X.

Workload: the MiniLM-L6-shaped encoder (hidden 384, 12 heads x 32, FFN 1536,
6 post-LN layers), batch 32 x sequence 128, bf16 storage with fp32
accumulation, seeded synthetic ids and N(0, 0.02) weights, valid lengths
U[16, 128] -- the paper's inference measurement (p50 of the encoder forward
at seq 128, batch up to 32) restated on this GPU.  One step is one whole
forward (embedding, 6 layers, pooling) with the inputs resident in HBM,
enqueued by rlx_encoder_forward in the encoder's default launch mode
(--graph: replayed from its recorded HIP graph instead).

Prints one JSON line: sequences/s, p50 ms, the roofline of the dominant
kernel (algorithmic flops per launch / its event-timed average duration) and
the CPU oracle timed on this host as a reported baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def gemm_flops_per_token(sp):
    H, F = sp.hidden, sp.ffn
    return {"gemm_qkv": 2 * H * 3 * H, "gemm_attn_out": 2 * H * H, "gemm_ffn_up": 2 * H * F, "gemm_ffn_down": 2 * F * H}


def attention_flops(sp, lengths):
    # QK^T and PV over real queries x real keys, per layer: 2 * 2 * d * L^2 per head
    return sum(4 * sp.head_dim * sp.heads * int(L) ** 2 for L in lengths)


# the sources of each measured kernel class (with the shared device headers)
_SHARED = ("common.hpp", "kernels.hpp")
KERNEL_SOURCES = {
    "qkv_attention": ("attention.hip", "qkv_attention.hpp"),
    "attention": ("attention.hip", "qkv_attention.hpp"),
    "mx_gemm": ("mx_gemm.hip",),
    "gemv": ("gemv.hip",),
    "encoder_pipe": ("pipe.hip", "gemm_tile.hpp", "qkv_attention.hpp"),
    # every kernel of an encoder forward (the counter summaries of a whole forward)
    "encoder": ("attention.hip", "qkv_attention.hpp", "gemm.hip", "gemm_tile.hpp", "rowops.hip", "pipe.hip"),
}


def kernel_source_digest(kernel_class="gemm"):
    """Digest of the sources of one kernel class (its .hip files and the shared
    device headers): counter figures taken before a change to them are no
    longer reported."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_37916_amd", "csrc")
    for f in sorted(set(KERNEL_SOURCES.get(kernel_class, ("gemm.hip", "gemm_tile.hpp"))) | set(_SHARED)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def _committed_summary(kernel_class, workload, digest_class=None):
    path = os.path.join(ROOT, "profiles", f"{kernel_class}_{workload}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_h = re.search(r"^kernel_source_digest:\s*([0-9a-f]+)", text, re.M)
    if not m_h or m_h.group(1) != kernel_source_digest(digest_class or kernel_class):
        return None
    return text


def committed_traffic(kernel_class, workload, digest_class=None):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when no summary exists or the kernel's sources changed since it was taken."""
    text = _committed_summary(kernel_class, workload, digest_class)
    m_b = re.search(r"^hbm_bytes_per_launch:\s*([0-9.eE+]+)", text, re.M) if text else None
    return float(m_b.group(1)) if m_b else None


def committed_forward_counters(workload):
    """Per kernel class of a forward, from the committed counter summary of that
    forward: calibrated HBM bytes per launch (FETCH_SIZE, WRITE_SIZE) and
    executed matrix flops per launch (SQ_INSTS_VALU_MFMA_MOPS_* x 512); None
    when no summary exists or the encoder's kernel sources changed since."""
    text = _committed_summary("encoder_forward", workload, "encoder")
    if text is None:
        return None
    out = {}
    for key in ("hbm_bytes_per_launch", "mfma_flops_per_launch"):
        m = re.search(r"^%s:\s*(\{.*\})\s*$" % key, text, re.M)
        out[key] = json.loads(m.group(1)) if m else {}
    return out


def cpu_baseline(workload_name, target_s):
    """The float64 oracle on this host's cores, on a bounded sample of the workload."""
    import numpy as np

    import oracle
    import workloads
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:
        threads = None
    wl = workloads.make(workload_name)
    B = wl.spec.batch
    probe = workloads.select_rows(wl, np.arange(min(2, B)))
    t0 = time.perf_counter()
    oracle.encoder_forward(probe)
    per_seq = (time.perf_counter() - t0) / probe.spec.batch
    # the first n sequences, or the whole batch `reps` times when it takes less than the target
    want = max(1, round(target_s / max(per_seq, 1e-6)))
    n = int(min(B, want))
    reps = int(max(1, want // B)) if want > B else 1
    sample = workloads.select_rows(wl, np.arange(n))
    t0 = time.perf_counter()
    for _ in range(reps):
        oracle.encoder_forward(sample)
    dt = time.perf_counter() - t0
    what = f"first {n} of {B} sequences" if reps == 1 else f"all {B} sequences, {reps} times"
    # cores: the threads the oracle used (its BLAS pool; the rest of NumPy runs on one);
    # the host's CPU count and the CPUs this process may run on, beside it
    try:
        affinity = len(os.sched_getaffinity(0))
    except Exception:
        affinity = None
    rec = {"value": n * reps / dt, "unit": "sequences/s", "cores": threads, "kind": "oracle",
           "blas_threads": threads, "host_cpu_count": os.cpu_count(), "affinity_cpus": affinity,
           "sample": f"{what} of {workload_name}, float64 NumPy oracle, {dt:.1f} s"}
    # the same oracle on one thread, over a quarter of the time
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            n1 = max(1, min(B, round(target_s / 4 / max(per_seq, 1e-6))))
            one = workloads.select_rows(wl, np.arange(n1))
            t0 = time.perf_counter()
            oracle.encoder_forward(one)
            d1 = time.perf_counter() - t0
        rec["one_thread"] = {"value": n1 / d1, "sample": f"first {n1} sequences, {d1:.1f} s"}
    except Exception:
        rec["one_thread"] = None
    return rec


def gpu_state():
    """Shader clock and temperatures from rocm-smi after the timed region (run as a
    child process), or None where it is unavailable."""
    import shutil
    import subprocess
    exe = shutil.which("rocm-smi") or ("/opt/rocm/bin/rocm-smi" if os.path.exists("/opt/rocm/bin/rocm-smi") else None)
    if exe is None:
        return None
    # Under a profiler its preloaded library would follow the child (and
    # initialise the GPU there); not needed for a profile.
    if "rocprof" in os.environ.get("LD_PRELOAD", ""):
        return {"skipped": "run under a profiler"}
    try:
        # a Python script runs under this interpreter directly: no '/usr/bin/env python3' hop
        with open(exe, "rb") as fh:
            first = fh.readline()
        cmd = [sys.executable, exe] if first.startswith(b"#!") and b"python" in first else [exe]
        r = subprocess.run(cmd + ["--showclocks", "--showtemp", "--json"], capture_output=True, text=True, timeout=30)
        card = next(iter(json.loads(r.stdout[r.stdout.index("{"):]).values()))
    except Exception:
        return None
    keep = {k: v for k, v in card.items() if "sclk" in k.lower() or "mclk" in k.lower() or "emperature" in k}
    return keep or None


MX_PEAK_TFLOPS = {"e4m3": 5000.0, "e5m2": 5000.0, "e2m3": 10100.0, "e3m2": 10100.0, "e2m1": 10100.0}


def bench_scaled_matmul(args):
    """Block-scaled minifloat matmul (rlx_scaled_matmul) on one shape: the
    encoder's FFN-down at batch 256 x 128 by default (18048 real tokens)."""
    import numpy as np
    import torch

    import paper_2609_37916_amd as rlx
    from workloads import mx as wmx

    M, N, K = args.mx_shape
    fx = fw = args.mx_format
    x, w = wmx.matmul_inputs(1, M, N, K, fx, fw)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
    xp, xs, wp, ws = dev(x.packed), dev(x.scales), dev(w.packed), dev(w.scales)
    y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        rlx.scaled_matmul(xp, xs, fx, wp, ws, fw, K=K, out=y)
    torch.cuda.synchronize()
    # K back-to-back launches between two events on the launch stream (per-launch
    # event pairs would add the enqueue gap to every launch)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(args.steps):
        rlx.scaled_matmul(xp, xs, fx, wp, ws, fw, K=K, out=y)
    e1.record(stream)
    torch.cuda.synchronize()
    us = 1e3 * e0.elapsed_time(e1) / args.steps
    launch_us = [us]
    flops = 2.0 * M * N * K
    tf = flops / (us * 1e-6) / 1e12
    peak = MX_PEAK_TFLOPS[fx]
    name = f"mx_{fx}_m{M}_n{N}_k{K}"
    # algorithmic bytes: both operands' codes and scales once, the fp32 output once
    nbytes = (M * K * wmx.BITS[fx] + N * K * wmx.BITS[fw]) // 8 + (M + N) * (K // 32) + 4 * M * N
    gbs = nbytes / (us * 1e-6) / 1e9
    # the binding roofline: below the ridge point (peak flops / peak bandwidth) it is HBM
    hbm_bound = flops / nbytes < peak * 1e12 / (PEAK_HBM_GBS * 1e9)
    rec = {
        "metric": f"scaled matmul TFLOP/s (MX {fx} x {fw}, {M}x{N}x{K}, 1 MI355X)",
        "value": round(tf, 1), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(us / 1e3, 5), "p50_ms": round(statistics.median(launch_us) / 1e3, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": fx,
        "data": "synthetic (seeded finite codes, E8M0 scales 2^-7 .. 2^7)",
        "config": {"workload": name, "M": M, "N": N, "K": K, "format_x": fx, "format_w": fw,
                   "parallelism": "single GPU"},
        "roofline": ({"bound": "hbm", "kernel": "mx_gemm_kernel", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                      "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4)} if hbm_bound else
                     {"bound": "mfma", "kernel": "mx_gemm_kernel", "achieved": round(tf, 2), "peak": peak,
                      "unit": "TFLOP/s", "frac": round(tf / peak, 4)}) | {
                     "traffic": committed_traffic("mx_gemm", name), "flops_per_launch": flops,
                     "bytes_per_launch": nbytes, "mfma_frac": round(tf / peak, 4),
                     "hbm_frac": round(gbs / PEAK_HBM_GBS, 4), "avg_launch_us": round(us, 3)},
    }
    if not args.no_cpu_baseline:
        import oracle
        rows = min(M, 2048)
        t0 = time.perf_counter()
        reps = 0
        while True:
            oracle.mx.scaled_matmul(x.packed[:rows], x.scales[:rows], fx, w.packed, w.scales, fw, K)
            reps += 1
            dt = time.perf_counter() - t0
            if dt >= args.cpu_seconds or reps >= 1000:
                break
        try:
            from threadpoolctl import threadpool_info
            threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
        except Exception:
            threads = os.cpu_count() or 1
        rec["cpu_baseline"] = {"value": round(2.0 * rows * N * K * reps / dt / 1e12, 4), "unit": "TFLOP/s",
                               "cores": threads, "kind": "oracle",
                               "sample": f"first {rows} rows of X, {reps} times, float64 NumPy oracle, {dt:.1f} s"}
    print(json.dumps(rec), flush=True)


# Chip-wide rate of the bare exp2 instruction (v_exp_f32), measured on one MI355X
# with independent exp2 chains against fma chains: ~17.0 T/s, a quarter of the
# measured fp32 fma rate (63 T/s).
EXP2_PEAK_G = 17000.0


def attention_pairs(kind, S, lens, window):
    """Visible (query, key) pairs per head summed over the batch (every query row is computed)."""
    if kind == "custom":
        return sum(S * int(L) for L in lens)
    if kind == "none":
        return len(lens) * S * S
    if kind == "causal":
        return len(lens) * S * (S + 1) // 2
    return len(lens) * sum(min(window, i + 1) for i in range(S))


def bench_attention(args):
    """rlx_masked_attention on the long-sequence shape: batch 8 x 512, 12 heads
    x 32, bf16, Q / K / V as column views of one fused [B*S, 3H] buffer; key
    lengths half U[64, 512], half 512 (custom mask) or the mask kind's own
    visibility (none, causal, sliding window)."""
    import numpy as np
    import torch

    import paper_2609_37916_amd as rlx

    B, S, heads, d = 8, 512, 12, 32
    H = heads * d
    kind = args.attn_kind
    code = {"none": rlx.MASK_NONE, "causal": rlx.MASK_CAUSAL, "sliding": rlx.MASK_SLIDING_WINDOW,
            "custom": rlx.MASK_CUSTOM}[kind]
    rng = np.random.default_rng(11)
    lens = np.concatenate([rng.integers(64, S + 1, B // 2), np.full(B - B // 2, S)])
    mask = (np.arange(S)[None, :] < lens[:, None]).astype(np.uint8)
    qkv = torch.from_numpy(rng.normal(0, 1, (B * S, 3 * H)).astype(np.float32)).to("cuda", torch.bfloat16)
    km = torch.from_numpy(mask).cuda() if kind == "custom" else None
    out = torch.empty((B * S, H), dtype=torch.bfloat16, device="cuda")
    window = args.attn_window

    def launch():
        rlx.masked_attention(qkv[:, :H], qkv[:, H:2 * H], qkv[:, 2 * H:], B=B, S=S, heads=heads, kind=code,
                             key_mask=km, window=window, row_stride=3 * H, out=out)

    for _ in range(args.warmup):
        launch()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        launch()
    e1.record(stream)
    torch.cuda.synchronize()
    us = 1e3 * e0.elapsed_time(e1) / args.steps
    pairs = attention_pairs(kind, S, lens, window) * heads
    flops = 4.0 * d * pairs  # Q K^T and P V over the visible pairs
    tf = flops / (us * 1e-6) / 1e12
    name = f"attention_{kind}_b{B}_s{S}"
    rec = {
        "metric": f"masked attention TFLOP/s ({kind} mask, batch {B} x {S}, {heads} heads x {d}, bf16, 1 MI355X)",
        "value": round(tf, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(us / 1e3, 5), "p50_ms": round(us / 1e3, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (N(0,1) Q / K / V; key lengths half U[64,512], half 512)",
        "config": {"workload": name, "batch": B, "seq_len": S, "heads": heads, "head_dim": d, "mask": kind,
                   "window": window if kind == "sliding" else None, "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "kernel": "attn_bf16_kernel", "achieved": round(tf, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(tf / PEAK_BF16_TFLOPS, 4),
                     "traffic": committed_traffic("attention", f"{kind}_b{B}_s{S}"),
                     "flops_per_launch": flops, "avg_launch_us": round(us, 3),
                     # at head_dim 32 every score costs one exp2 against 64 MFMA flops: the exp pipe's
                     # ceiling in visible scores per second (measured rate of the bare exp2 instruction)
                     "exp_ceiling": {"achieved_g_per_s": round(pairs / us / 1e3, 1), "peak_g_per_s": EXP2_PEAK_G,
                                     "frac": round(pairs / us / 1e3 / EXP2_PEAK_G, 4)}},
    }
    if not args.no_cpu_baseline:
        import oracle
        q4 = qkv.float().cpu().numpy().reshape(B, S, 3, heads, d)
        okind = {"none": oracle.MASK_NONE, "causal": oracle.MASK_CAUSAL, "sliding": oracle.MASK_SLIDING_WINDOW,
                 "custom": oracle.MASK_CUSTOM}[kind]
        t0 = time.perf_counter()
        reps = 0
        while True:
            b = reps % B
            oracle.masked_attention(q4[b:b + 1, :, 0], q4[b:b + 1, :, 1], q4[b:b + 1, :, 2], kind=okind,
                                    key_mask=mask[b:b + 1] if kind == "custom" else None, window=window)
            reps += 1
            dt = time.perf_counter() - t0
            if dt >= args.cpu_seconds or reps >= 1000:
                break
        done = sum(attention_pairs(kind, S, lens[[r % B]], window) for r in range(reps)) * heads * 4.0 * d
        try:
            from threadpoolctl import threadpool_info
            threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
        except Exception:
            threads = os.cpu_count() or 1
        rec["cpu_baseline"] = {"value": round(done / dt / 1e12, 6), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
                               "sample": f"{reps} single-sequence calls (all heads), float64 NumPy oracle, {dt:.1f} s"}
    print(json.dumps(rec), flush=True)


def gemv_bytes(scheme, M, N, K, epi_bias=True):
    """Algorithmic HBM bytes of one few-row dequantising matmul: every weight
    code, scale and zero-point (or min) once, the activations, the bias and the
    output.  GGUF schemes count their repacked layout (Q4_0 and Q4_1: int4
    codes, f16 scales and f16 zeros / mins; Q8_0: int8 codes and f16 scales;
    Q4_K: as Q4_1, a composed f16 scale and min per 32 weights; Q6_K: int8
    codes and a composed f16 scale per 16 weights)."""
    four = scheme in ("int4", "q4_0", "q4_1", "q4_k")
    codes = N * K // 2 if four else N * K
    if four:
        meta = 2 * N * (K // 32) * 2
    else:
        meta = {"q8_0": 2 * N * (K // 32), "q6_k": 2 * N * (K // 16)}.get(scheme, 2 * N)
    return codes + meta + 2 * M * K + 2 * M * N + (4 * N if epi_bias else 0)


def bench_dequant_gemv(args):
    """Few-row dequantising matmul (rlx_dequant_matmul with M <= 16 rows, the
    GEMV regime): a decode-sized product, N 14336 x K 4096 by default.  The
    launches cycle through enough weight copies (> 512 MB) that every launch
    streams its weights from HBM rather than from the 256 MB last-level cache."""
    import numpy as np
    import torch

    import paper_2609_37916_amd as rlx
    import workloads

    M, N, K = args.gemv_shape
    scheme = args.gemv_scheme
    rng = np.random.default_rng(7)
    x = workloads.round_to_bf16(rng.normal(0, 1, (M, K)).astype(np.float32))
    wf = rng.normal(0, 0.02, (N, K)).astype(np.float32)
    b = rng.normal(0, 0.5, N).astype(np.float32)
    dev = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dt)
    if scheme in ("q4_0", "q4_1", "q8_0", "q4_k", "q6_k"):
        from workloads import gguf as wg
        if scheme in ("q4_k", "q6_k"):
            # no K-quant quantiser here: random super-blocks stream the same bytes
            blocks = wg.random_kquant_blocks(rng, N, K, scheme)
        else:
            blocks = wg.quantize(wf, scheme)
        sch, codes, scl, zr = rlx.gguf_repack(dev(blocks, torch.uint8), scheme, N=N, K=K)
        one = (codes, scl, zr)
        kw = dict(scheme=sch, group_size=16 if scheme == "q6_k" else 32)
    elif scheme == "int8":
        q, s = workloads.quantize_int8_per_channel(wf)
        one = (dev(q, torch.int8), dev(s, torch.float16), None)
        kw = dict(scheme=rlx.Q_INT8_PER_CHANNEL)
    else:
        q, s, z = workloads.quantize_int4_grouped(wf, 32)
        one = (dev(q, torch.uint8), dev(s, torch.float16), dev(z, torch.float16))
        kw = dict(scheme=rlx.Q_INT4_GROUP_ZP, group_size=32)
    nbytes = gemv_bytes(scheme, M, N, K)
    copies = max(1, -(-512 * 2 ** 20 // nbytes))
    ws = [one] + [tuple(None if t is None else t.clone() for t in one) for _ in range(copies - 1)]
    xd, bd = dev(x, torch.bfloat16), dev(b, torch.float32)
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()

    def launch(i):
        w, sc, zr = ws[i % copies]
        rlx.dequant_matmul(xd, w, scales=sc, zeros=zr, N=N, bias=bd, epi=rlx.EPI_BIAS, out=y, **kw)

    for i in range(args.warmup):
        launch(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(args.steps):
        launch(i)
    e1.record(stream)
    torch.cuda.synchronize()
    us = 1e3 * e0.elapsed_time(e1) / args.steps
    gbs = nbytes / (us * 1e-6) / 1e9
    name = f"gemv_{scheme}_m{M}_n{N}_k{K}"
    rec = {
        "metric": f"dequant GEMV GB/s ({scheme} weights, bf16 x, {M}x{N}x{K}, 1 MI355X)",
        "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(us / 1e3, 5), "p50_ms": round(us / 1e3, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": (f"synthetic (random {scheme} super-blocks: uniform codes, scales and mins, repacked"
                 if scheme in ("q4_k", "q6_k") else
                 f"synthetic (N(0,0.02) weights quantised {scheme}{' (GGUF blocks, repacked)' if scheme.startswith('q') else ''}")
                + f", N(0,1) bf16 activations), {copies} weight copies",
        "config": {"workload": name, "M": M, "N": N, "K": K, "scheme": scheme, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "kernel": "gemv_q_kernel", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "traffic": committed_traffic("gemv", f"{scheme}_m{M}_n{N}_k{K}"),
                     "bytes_per_launch": nbytes, "avg_launch_us": round(us, 3)},
    }
    if not args.no_cpu_baseline:
        import oracle
        cols = min(N, 1024)
        t0 = time.perf_counter()
        reps = 0
        while True:
            if scheme in ("q4_k", "q6_k"):
                wd = oracle.gguf.dequant_k(blocks[:cols], scheme, K)
            elif scheme in ("q4_0", "q4_1", "q8_0"):
                wd = oracle.gguf.dequant(blocks[:cols], scheme, K)
            elif scheme == "int8":
                wd = oracle.dequant_int8(q[:cols], s[:cols])
            else:
                wd = oracle.dequant_int4(q[:cols], s[:cols], z[:cols], 32)
            oracle.linear(x, wd, b[:cols])
            reps += 1
            dt = time.perf_counter() - t0
            if dt >= args.cpu_seconds or reps >= 1000:
                break
        try:
            from threadpoolctl import threadpool_info
            threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
        except Exception:
            threads = os.cpu_count() or 1
        rec["cpu_baseline"] = {"value": round(gemv_bytes(scheme, M, cols, K) * reps / dt / 1e9, 4), "unit": "GB/s",
                               "cores": threads, "kind": "oracle",
                               "sample": f"first {cols} weight rows, {reps} times, float64 NumPy oracle, {dt:.1f} s"}
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="minilm_b32_s128_bf16")
    ap.add_argument("--profile-steps", type=int, default=20, help="profiled forwards (per-kernel event times)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target length of the CPU-oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="time the encoder forward replayed from its HIP graph instead of launched kernel by kernel")
    ap.add_argument("--op", choices=("encoder", "scaled_matmul", "dequant_gemv", "attention"), default="encoder",
                    help="encoder: the encoder forward (default); scaled_matmul: the block-scaled minifloat matmul; "
                         "dequant_gemv: the few-row dequantising matmul; attention: rlx_masked_attention")
    ap.add_argument("--attn-kind", default="causal", choices=("none", "causal", "sliding", "custom"))
    ap.add_argument("--attn-window", type=int, default=128)
    ap.add_argument("--gemv-scheme", default="int4", choices=("int4", "int8", "q4_0", "q4_1", "q8_0", "q4_k", "q6_k"))
    ap.add_argument("--gemv-shape", type=int, nargs=3, default=(1, 14336, 4096), metavar=("M", "N", "K"))
    ap.add_argument("--mx-format", default="e4m3", choices=sorted(MX_PEAK_TFLOPS))
    ap.add_argument("--mx-shape", type=int, nargs=3, default=(18048, 384, 1536), metavar=("M", "N", "K"))
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy (counter calibration for FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} (WORLD_SIZE {world}) is not supported; the encoder "
              f"forward is data-parallel over sequences and this library runs it on a single MI355X.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_37916_amd as rlx
    import workloads
    from workloads.device import encoder_kwargs, to_device

    if not os.path.exists(rlx.LIB_PATH):
        from paper_2609_37916_amd import _build
        _build.build_library()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)

    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "device copy", "bytes_read": src.numel() * 4, "bytes_written": dst.numel() * 4,
                          "launches": 3}), flush=True)
        return

    if args.op == "scaled_matmul":
        bench_scaled_matmul(args)
        return
    if args.op == "dequant_gemv":
        bench_dequant_gemv(args)
        return
    if args.op == "attention":
        bench_attention(args)
        return

    sp = workloads.spec(args.workload)
    wl = workloads.make(sp)
    weights, inputs = to_device(wl)
    enc = rlx.Encoder(**encoder_kwargs(sp, use_graph=args.graph), weights=weights)
    persistent = enc.persistent
    out = torch.empty((sp.batch, sp.hidden), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        enc.forward(inputs["input"], inputs["mask"], out=out)
    torch.cuda.synchronize()

    # timed region: K back-to-back forwards, an event before each and after the last
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t_host = time.perf_counter()
    evs[0].record(stream)
    for i in range(args.steps):
        enc.forward(inputs["input"], inputs["mask"], out=out)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    t_host = time.perf_counter() - t_host
    enc.check()  # the persistent forward's bounded waits never gave up
    total_ms = evs[0].elapsed_time(evs[-1])
    step_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    ms_per_step = total_ms / args.steps
    p50 = statistics.median(step_ms)
    p10, p90 = np.percentile(step_ms, [10, 90]).tolist()
    seq_per_s = sp.batch * args.steps / (total_ms / 1e3)

    # per-kernel times: the same forward replayed from a graph with an event pair around every kernel
    enc.set_profiling(True)
    for _ in range(args.profile_steps):
        enc.forward(inputs["input"], inputs["mask"], out=out)
    prof = enc.profile_read()
    enc.set_profiling(False)
    per_launch_us = {k: 1e3 * ms / n for k, (n, ms) in prof.items()}
    per_fwd_us = {k: 1e3 * ms / args.profile_steps for k, (n, ms) in prof.items()}

    tokens = int(wl.mask.sum())  # real tokens: every row-local step runs on these after compaction
    fpt = gemm_flops_per_token(sp)
    flops_launch = {k: v * tokens for k, v in fpt.items()}
    flops_launch["attention"] = attention_flops(sp, wl.mask.sum(axis=1))
    # sequences of <= 128 tokens run the QKV projection inside the attention kernel
    flops_launch["qkv_attention"] = flops_launch["gemm_qkv"] + flops_launch["attention"]
    # the persistent forward: every layer's products and attention in one launch
    flops_launch["encoder_pipe"] = sp.layers * (sum(fpt.values()) * tokens + flops_launch["attention"])
    per_layer = {k for k in flops_launch if k != "encoder_pipe"}
    matrix_classes = [k for k in flops_launch if k in per_fwd_us]
    dominant = max(matrix_classes, key=lambda k: per_fwd_us.get(k, 0.0))
    counters = committed_forward_counters(args.workload)
    traffic = counters["hbm_bytes_per_launch"].get(dominant) if counters else None
    peak = PEAK_BF16_TFLOPS if sp.dtype == "bf16" else PEAK_F32_TFLOPS  # quantised weights: bf16 products
    achieved = flops_launch[dominant] / (per_launch_us[dominant] * 1e-6) / 1e12
    mm_flops = sum(flops_launch[k] * (sp.layers if k in per_layer else 1) for k in matrix_classes)
    mm_us = sum(per_fwd_us.get(k, 0.0) for k in matrix_classes)
    mfma_util = mm_flops / (mm_us * 1e-6) / (peak * 1e12)
    # the same from the matrix cores' own count: executed flops per launch (counter summary of this
    # workload's forward, padding included) over this run's per-launch times
    mfma_counter = None
    executed = counters["mfma_flops_per_launch"] if counters else {}
    if executed and all(k in executed for k in matrix_classes):
        launches = {k: per_fwd_us[k] / per_launch_us[k] for k in matrix_classes}
        mfma_counter = {
            "per_kernel": {k: round(executed[k] / (per_launch_us[k] * 1e-6) / (peak * 1e12), 4) for k in matrix_classes},
            "aggregate": round(sum(executed[k] * launches[k] for k in matrix_classes) / (mm_us * 1e-6) / (peak * 1e12), 4),
            "source": f"profiles/encoder_forward_{args.workload}_counters.md",
        }

    rec = {
        "metric": f"encoder fwd sequences/sec (b{sp.batch}, s{sp.seq}, "
                  f"{sp.quant if sp.quant != 'none' else sp.dtype}, 1 MI355X)",
        "value": round(seq_per_s, 1),
        "unit": "sequences/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "p50_ms": round(p50, 5),
        "p10_ms": round(p10, 5),
        "p90_ms": round(p90, 5),
        "host_wall_ms_per_step": round(1e3 * t_host / args.steps, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if sp.dtype == "bf16" else "f32",
        "data": "synthetic (seeded ids, N(0,0.02) weights, lengths U[%d,%d])" % (sp.len_lo, sp.len_hi),
        "config": {"workload": sp.name, "batch": sp.batch, "seq_len": sp.seq, "layers": sp.layers,
                   "hidden": sp.hidden, "heads": sp.heads, "ffn": sp.ffn, "real_tokens": tokens,
                   "quant": sp.quant, "parallelism": "single GPU", "graph_replay": args.graph,
                   "persistent_forward": persistent,
                   # quantised weights: dequantised to bf16 by the forward's first kernel (large calls)
                   # or inside the GEMMs
                   "dequant_prologue": "dequant_weights" in per_fwd_us},
        "mfma_util_pct": round(100 * mfma_util, 2),
        "mfma_util_counter": mfma_counter,
        "roofline": {"bound": "mfma", "kernel": dominant, "achieved": round(achieved, 2), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                     "traffic": traffic, "flops_per_launch": flops_launch[dominant],
                     "avg_launch_us": round(per_launch_us[dominant], 3)},
        "kernel_us_per_forward": {k: round(v, 2) for k, v in sorted(per_fwd_us.items(), key=lambda kv: -kv[1])},
    }
    enc.close()

    # the same forward in the other launch mode (HIP graph replay or kernel by kernel), a shorter sample
    eager = rlx.Encoder(**encoder_kwargs(sp, use_graph=not args.graph), weights=weights)
    for _ in range(5):
        eager.forward(inputs["input"], inputs["mask"], out=out)
    n_eager = max(10, args.steps // 4)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_eager + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for i in range(n_eager):
        eager.forward(inputs["input"], inputs["mask"], out=out)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    eager_p50 = statistics.median([evs[i].elapsed_time(evs[i + 1]) for i in range(n_eager)])
    eager.close()
    rec["other_mode"] = {"graph_replay": not args.graph, "p50_ms": round(eager_p50, 5),
                         "sequences_per_s": round(sp.batch / (eager_p50 / 1e3), 1), "steps": n_eager}
    rec["gpu_state"] = gpu_state()
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(args.workload, args.cpu_seconds)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
