#!/usr/bin/env python3
"""Throughput of the MixFP4 hot path on one MI355X.

One step = one pass of the whole path over the large prefill workload (seed
4): compute the tensor scale of and quantize the activations A [16384, 8192]
(block mixture: 90% of 16-blocks N(0, 0.1), 10% Laplace(0, 1) with one x40
spike), then C = A W^T [16384, 8192] in fp32 on the matrix cores.  The weight
W [8192, 8192] (N(0, 0.02)) is quantized once before timing, as weights are
quantized offline.  Inputs are resident in HBM before timing starts.

Prints ONE JSON line:
  value         GEMM FLOPs of the step / step time (TFLOP/s; the activation
                quantizer is inside the step time), from K steps timed
                wall-clock between device synchronizations, after W warmup
                steps and a time-based spin-up to loaded clocks
  roofline      the dominant kernel, the GEMM C = A W^T of the step, against
                the dense fp16 MFMA peak (its operands are exact fp16 values):
                its FLOPs per launch over its mean launch time, timed with HIP
                events on the stream it runs on during a second pass of the
                same K steps
  quantize      the quantizer kernel on the standalone 2^28-element tensor
                (seed 4 block mixture) against HBM, with the tensor scale given
                (algorithmic 2.5625 B / element), plus the end-to-end time with
                the tensor scale computed on the device, and the other
                encodings / roundings / rotation on the same tensor
  quantize_step the activation quantizer inside the step
  prefill_7b    the 7B-class prefill step (seed 1): quantize A [2048, 4096],
                C1 = A W1^T [2048, 11008], C2 = A W2^T [2048, 4096]
  rotated       the rotated-operand step (seed 2): quantize A [4096, 4096],
                C = A W^T [4096, 14336]
  decode_shape  the memory-bound m = 16 step (seed 3) against HBM
  train_step    one training step of a 7B-class linear layer (FPROP, DGRAD,
                WGRAD with 2D weight blocks, stochastic rounding and the
                16-row Hadamard rotation of the WGRAD inputs; seed 5)
  cpu_baseline  the CPU oracle on a bounded sample of the headline step
Usage: python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
                       [--only large,quantize,prefill_7b,rotated,decode,train]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MixFP4 quantize GB/s + MixFP4 GEMM TFLOP/s (% of roofline), 1x MI355X"
PEAK_F16_TFLOPS = 2500.0           # MI355X dense fp16 / bf16 MFMA
PEAK_HBM_GBPS = 8000.0             # MI355X HBM3E
QUANT_BYTES_PER_ELEM = 2 + 0.5 + 1 / 16   # read bf16, write codes + scales
AMAX_BYTES_PER_ELEM = 2                   # the tensor-scale pass re-reads X

# HBM traffic of one launch of the dominant GEMM (C = A W^T of the large
# workload, 16384 x 8192 x 8192), from two rocprofv3 --pmc runs of this script
# (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch; summary and commands in
# profiles/), scaled by what the same counters read for a 512 MiB elementwise
# copy (--calibrate-copy).  Valid only for the GEMM source it was measured on
# (first 16 hex digits of its SHA-256); reported as null otherwise, and null
# until it has been measured.
GEMM_TRAFFIC = {
    "gemm_src_sha256_16": "654483a34ab9f56c",    # csrc/gemm_f16.hip as measured
    "fetch_kib": 1584598, "write_kib": 611848,  # KiB per dispatch, gemm_f16_kernel
    "fetch_scale": 2.0, "write_scale": 1.0,     # 512 MiB copy: 262168 KiB fetched, 524288 written
}


def gemm_traffic_bytes():
    import hashlib
    t = GEMM_TRAFFIC
    if t is None:
        return None
    with open(os.path.join(ROOT, "paper_2605_31035_amd", "csrc", "gemm_f16.hip"), "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()[:16]
    if sha != t["gemm_src_sha256_16"]:
        return None
    return round((t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"]) * 1024)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def _oracle_quantize_rows(args):
    from oracle import quant as Q
    bits, s32 = args
    q = Q.quantize(bits, s32)
    return q.codes, q.scales


def _blas_threads() -> int | None:
    try:
        from threadpoolctl import threadpool_info
        n = [i["num_threads"] for i in threadpool_info() if i.get("user_api") == "blas"]
        return max(n) if n else None
    except Exception:
        return None


# The sample of the headline step that the oracle runs: the first SAMPLE_ROWS
# rows of A against the first SAMPLE_COLS rows of W (all of K), with the
# tensor scales of the full tensors, as in the GPU step.
SAMPLE_ROWS, SAMPLE_COLS = 512, 2048


def cpu_baseline(wl, budget_s: float = 12.0, max_reps: int = 200) -> dict:
    """The CPU oracle on a bounded sample of the headline step: the oracle
    quantize of A's first SAMPLE_ROWS rows (row chunks in a process pool; the
    tensor scale is the oracle's max over all of A) and the oracle GEMM of
    those rows against W's first SAMPLE_COLS rows (fp64 matmul of exactly
    dequantized operands plus its bound matmul, multithreaded BLAS).  W's
    sample is quantized by the oracle once, outside the timed sample, as W is
    in the GPU step.  Samples repeat until `budget_s` has elapsed; the rate is
    the sample's GEMM FLOPs over its time.  The pool takes every core of this
    process's affinity mask up to 16, the CPU share one GPU of the box has."""
    from concurrent.futures import ProcessPoolExecutor

    from oracle import gemm as G
    from oracle import quant as Q

    affinity = len(os.sched_getaffinity(0))
    cores = max(1, min(16, affinity))
    a_bits, w_bits = wl.tensors["A"], wl.tensors["W"]
    sa, sw = Q.tensor_scale(a_bits), Q.tensor_scale(w_bits)
    a_s, w_s = a_bits[:SAMPLE_ROWS], w_bits[:SAMPLE_COLS]
    k = a_bits.shape[1]
    flops = 2.0 * a_s.shape[0] * w_s.shape[0] * k

    def quantize(ex, bits, s32):
        parts = list(ex.map(_oracle_quantize_rows,
                            [(c, s32) for c in np.array_split(bits, 4 * cores)]))
        return Q.Quantized(codes=np.concatenate([p[0] for p in parts]),
                           scales=np.concatenate([p[1] for p in parts]),
                           s32=s32, t=None, sf_code=None, si_code=None, delta=None)

    times = []
    with ProcessPoolExecutor(cores) as ex:
        qw = quantize(ex, w_s, sw)
        while len(times) < max_reps and sum(times) < budget_s:
            t0 = time.perf_counter()
            qa = quantize(ex, a_s, sa)
            G.gemm(*G.operands(qa, qw))
            times.append(time.perf_counter() - t0)
    t = float(np.mean(times))
    blas = _blas_threads()
    return {
        "value": flops / t / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
        "blas_threads": blas, "affinity_cores": affinity,
        "sample": (f"{len(times)} sample(s) of the headline step: oracle quantize of "
                   f"A[:{SAMPLE_ROWS}] of [16384,8192] ({cores} processes, s32 of all of A) + "
                   f"oracle fp64 GEMM of those rows against W[:{SAMPLE_COLS}] with its bound "
                   f"matmul ({blas} BLAS threads); W's rows quantized by the oracle "
                   f"beforehand; {t:.2f} s per sample of {flops / 1e9:.1f} GFLOP"),
    }


def spin_up(torch, fn, seconds: float = 0.2) -> None:
    """Call fn back to back for about `seconds` before a timed region.  The
    GPU lowers its clocks when idle (the workloads are generated on the host
    between measurements) and takes tens of milliseconds of load to raise
    them again; measured on MI355X, a 2^28-element quantize takes ~170 us
    from idle and ~147 us at speed, and the prefill step 0.367 against
    0.333 ms.  Untimed, like every warmup."""
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(8):
            fn()
        torch.cuda.synchronize()


def measure_quantize(M, torch, dev, iters: int = 20) -> dict:
    """Quantize-only throughput on the standalone tensor Q [16384, 16384]
    (2^28 elements, seed 4 block mixture).  The kernel alone: tensor scale
    given (computed once beforehand on the device); end to end: tensor scale
    computed on the device in the same call (one extra read of Q)."""
    import workloads as W
    log("generating the 2^28-element quantize-only tensor (seed 4)")
    bits = W.large(tensors=("Q",)).tensors["Q"]
    xq = torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)
    del bits
    r, k = xq.shape
    codes = torch.empty((r, k // 2), dtype=torch.uint8, device=dev)
    scales = torch.empty((r, k // 16), dtype=torch.uint8, device=dev)
    s32 = torch.empty(1, dtype=torch.float32, device=dev)
    M.mixfp4_quantize(xq, None, codes, scales, scale_out=s32)     # s32 for the given mode

    signs = torch.tensor(np.where(np.random.default_rng(4).random(128) < 0.5, -1, 1)
                         .astype(np.int8), device=dev)

    def time_calls(fn) -> float:
        # `iters` back-to-back calls between two HIP events (an event between
        # calls would add its own ~3.5 us to every span)
        spin_up(torch, fn, 0.15)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters

    def timed(given: bool, mode: str = "mixfp4", **kw) -> float:
        return time_calls(lambda: M.mixfp4_quantize(xq, s32 if given else None, codes, scales,
                                                    scale_out=s32, mode=mode, **kw))

    ms_given = timed(True)
    ms_compute = timed(False)
    ms_nvfp4 = timed(True, "e2m1")
    ms_46 = timed(True, "four_six")
    ms_sr = timed(True, rounding="stochastic", seed=1, offset=0)
    ms_rht = timed(True, hadamard_block=128, hadamard_signs=signs)
    ms_rht_sr = timed(True, rounding="stochastic", seed=1, hadamard_block=128,
                      hadamard_signs=signs)
    n = xq.numel()
    del codes, scales
    torch.cuda.empty_cache()
    yq = torch.empty_like(xq)
    ms_had = time_calls(lambda: M.mixfp4_hadamard(xq, 128, signs, out=yq))
    del yq
    torch.cuda.empty_cache()
    variants = measure_variants(M, torch, xq, time_calls)
    del xq
    torch.cuda.empty_cache()
    gbps = n * QUANT_BYTES_PER_ELEM / (ms_given * 1e-3) / 1e9

    def rate(ms, bpe=QUANT_BYTES_PER_ELEM):
        return round(n * bpe / (ms * 1e-3) / 1e9, 1)
    return {
        "workload": "quantize-only Q[16384,16384] bf16 (2^28 elements), seed 4 block mixture: "
                    "90% of 16-blocks N(0,0.1), 10% Laplace(0,1) with one x40 spike",
        "bound": "hbm", "kernel": "quantize_kernel (tensor scale given)",
        "achieved": round(gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
        "frac": round(gbps / PEAK_HBM_GBPS, 4), "us": round(ms_given * 1e3, 2),
        "bytes_per_elem": QUANT_BYTES_PER_ELEM,
        "compute_mode_us": round(ms_compute * 1e3, 2),
        "compute_mode_GBps": round(n * QUANT_BYTES_PER_ELEM / (ms_compute * 1e-3) / 1e9, 1),
        "compute_mode_note": "tensor scale computed on the device (amax pass + quantize); "
                             "GB/s counts the same 2.5625 B/element",
        "e2m1_only_us": round(ms_nvfp4 * 1e3, 2),
        "e2m1_only_GBps": round(n * QUANT_BYTES_PER_ELEM / (ms_nvfp4 * 1e-3) / 1e9, 1),
        "e2m1_only_note": "the same kernel forced to the E2M1 branch (NVFP4 encoding), s32 given",
        "four_six_us": round(ms_46 * 1e3, 2), "four_six_GBps": rate(ms_46),
        "four_six_note": "the 4/6 candidate set (E2M1 under max/6 or max/4), s32 given",
        "stochastic_us": round(ms_sr * 1e3, 2), "stochastic_GBps": rate(ms_sr),
        "stochastic_note": "MixFP4 selection with stochastic rounding of the codes (App. D), "
                           "Philox4x32-10 draws per block, s32 given",
        "rht128_quantize_us": round(ms_rht * 1e3, 2), "rht128_quantize_GBps": rate(ms_rht),
        "rht128_sr_quantize_us": round(ms_rht_sr * 1e3, 2),
        "rht128_sr_quantize_GBps": rate(ms_rht_sr),
        "rht_note": "random Hadamard rotation with 128-blocks fused before the quantizer "
                    "(exact fp64 transform, rounded to bf16), s32 given; with and without "
                    "stochastic rounding",
        "hadamard128_us": round(ms_had * 1e3, 2), "hadamard128_GBps": rate(ms_had, 4.0),
        "hadamard_note": "standalone mixfp4_hadamard, 128-blocks with signs: 2 B read + 2 B "
                         "written per element",
        "variants": variants,
    }


VARIANT_SETS = (("e2m1",), ("e2m1", "e1m2"), ("e2m1", "e3m0"), ("e2m1", "e1m2", "e3m0"))


def measure_variants(M, torch, xq, time_calls) -> dict:
    """Algorithm 1's selection over the candidate sets and block sizes of the
    paper's ablation (Table 5: FP4-E2, +FP4-E1, +FP4-E3, +E1+E3 at block
    sizes 8, 16, 32, 64) on the same 2^28-element tensor: the kernel's rate
    (tensor scale given; 2 B read, 0.5 B of codes and two bytes per block
    written) and the relative squared error sum (X - dequant)^2 / sum X^2 of
    the result (tensor scale computed), summed in fp64 on the device."""
    n = xq.numel()
    x64 = None
    out = {}
    for block in (8, 16, 32, 64):
        for cands in VARIANT_SETS:
            q = M.mixfp4_quantize_variant(xq, block, cands)
            ms = time_calls(lambda: M.mixfp4_quantize_variant(xq, block, cands, q.s32))
            d = M.mixfp4_dequantize_variant(q)
            if x64 is None:
                x64 = xq.to(torch.float64)
                den = float((x64 * x64).sum())
            err = float(((x64 - d.to(torch.float64)) ** 2).sum()) / den
            frac = [round(float((q.fmt == i).sum()) / q.fmt.numel(), 4) for i in range(len(cands))]
            del d, q
            bpe = 2.0 + 0.5 + 2.0 / block
            out[f"g{block}_" + "+".join(cands)] = {
                "us": round(ms * 1e3, 2), "GBps": round(n * bpe / (ms * 1e-3) / 1e9, 1),
                "bytes_per_elem": round(bpe, 4), "rel_sse": float(f"{err:.6g}"),
                "chosen_fraction": frac}
    del x64
    torch.cuda.empty_cache()
    return out


def measure_decode(M, torch, dev, iters: int = 50) -> dict:
    """Decode-shape step (seed 3): online tensor scale + quantize of A[16,8192],
    then C = A W^T [16, 28672] against W[28672,8192] quantized once before
    timing.  HBM-bound: algorithmic bytes = W codes + W scales + A (bf16 in,
    codes + scales) + C."""
    import workloads as W
    wl = W.decode()
    xa = torch.from_numpy(wl.tensors["A"].view(np.int16)).to(dev).view(torch.bfloat16)
    xw = torch.from_numpy(wl.tensors["W"].view(np.int16)).to(dev).view(torch.bfloat16)
    qw = M.mixfp4_quantize(xw)
    del xw
    r, k = xa.shape
    qa = (torch.empty((r, k // 2), dtype=torch.uint8, device=dev),
          torch.empty((r, k // 16), dtype=torch.uint8, device=dev),
          torch.empty(1, dtype=torch.float32, device=dev))
    out = torch.empty((r, qw[0].shape[0]), dtype=torch.float32, device=dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(iters)]

    def decode_step():
        M.mixfp4_quantize(xa, None, qa[0], qa[1], scale_out=qa[2])
        M.mixfp4_gemm(qa, qw, out=out)

    spin_up(torch, decode_step)
    for i in range(5 + iters):
        e = ev[i - 5] if i >= 5 else None
        if e:
            e[0].record()
        M.mixfp4_quantize(xa, None, qa[0], qa[1], scale_out=qa[2])
        if e:
            e[1].record()
        M.mixfp4_gemm(qa, qw, out=out)
        if e:
            e[2].record()
    torch.cuda.synchronize()
    q_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    step_g_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    # the GEMM kernel alone: launches back to back, so no dispatch gap after
    # the quantizer is counted
    b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    b0.record()
    for _ in range(iters):
        M.mixfp4_gemm(qa, qw, out=out)
    b1.record()
    torch.cuda.synchronize()
    g_ms = b0.elapsed_time(b1) / iters
    # the whole decode step (quantize A, then the GEMM), steps back to back
    b0.record()
    for _ in range(iters):
        decode_step()
    b1.record()
    torch.cuda.synchronize()
    st_ms = b0.elapsed_time(b1) / iters
    # the same step as one launch (mixfp4_decode_step: A quantized by the
    # first workgroups and handed to the GEMM inside the launch), steps back
    # to back on the same buffers
    sync = torch.zeros(4, dtype=torch.int32, device=dev)

    def fused_step():
        M.mixfp4_decode_step(xa, qw, out=out, a_out=qa, sync=sync)

    spin_up(torch, fused_step)
    b0.record()
    for _ in range(iters):
        fused_step()
    b1.record()
    torch.cuda.synchronize()
    fs_ms = b0.elapsed_time(b1) / iters
    n = qw[0].shape[0]
    gemm_bytes = n * k / 2 + n * k / 16 + r * k / 2 + r * k / 16 + r * n * 4
    step_bytes = gemm_bytes + r * k * 2          # plus reading A in bf16
    return {
        "workload": "decode: A[16,8192] N(0,1) with 4 outlier channels x30 quantized online; "
                    "W[28672,8192] N(0,0.02) with 0.5% outliers, quantized before timing",
        "gemm_us": round(g_ms * 1e3, 2), "quantize_a_us": round(q_ms * 1e3, 2),
        "gemm_bound": "hbm", "gemm_bytes": gemm_bytes,
        "gemm_GBps": round(gemm_bytes / (g_ms * 1e-3) / 1e9, 1),
        "gemm_hbm_frac": round(gemm_bytes / (g_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
        "gemm_TFLOPs": round(2.0 * r * n * k / (g_ms * 1e-3) / 1e12, 2),
        "gemm_in_step_us": round(step_g_ms * 1e3, 2),
        "step_us": round(st_ms * 1e3, 2),
        "fused_step_us": round(fs_ms * 1e3, 2),
        "fused_step_GBps": round(step_bytes / (fs_ms * 1e-3) / 1e9, 1),
        "fused_step_hbm_frac": round(step_bytes / (fs_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
        "fused_step": "mixfp4_decode_step: tensor scale, quantization of A and the GEMM in one "
                      "launch (A's codes, scales and s32 written as outputs)",
        "timing": "gemm_us: back-to-back GEMM launches; step_us: back-to-back steps of quantize "
                  "A then GEMM (dispatch gaps included); fused_step_us: back-to-back one-launch "
                  "steps; quantize_a_us and gemm_in_step_us: HIP event spans around each launch "
                  "of a separate pass of steps",
    }


def measure_train(M, torch, dev, iters: int = 10) -> dict:
    """One training step of a 7B-class linear layer in the flow of the paper's
    Fig. 7 (workload train_7b, seed 5): every quantization with its tensor
    scale computed on the device, inside the timed region.
      FPROP  quantize X; 2D-quantize W (16x16 tiles, W and W^T layouts);
             Y = X W^T                      [2048 x 11008 x 4096]
      DGRAD  quantize dY (stochastic rounding); dX = dY W   [2048 x 4096 x 11008]
      WGRAD  quantize dY^T (stochastic rounding) and X^T, both after a 16-row
             random Hadamard rotation; dW = dY^T X          [11008 x 4096 x 2048]"""
    import workloads as W
    log("generating train_7b workload (seed 5)")
    wl = W.train_7b()
    t = {n: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
         for n, b in wl.tensors.items()}
    del wl
    X, Wt, dY = t["X"], t["W"], t["dY"]
    tok, d_in = X.shape
    d_out = Wt.shape[0]
    signs = torch.tensor(np.where(np.random.default_rng(5).random(16) < 0.5, -1, 1)
                         .astype(np.int8), device=dev)
    names = ["quantize X", "quantize_2d W", "fprop gemm", "quantize dY (SR)", "dgrad gemm",
             "quantize dY^T (RHT16, SR)", "quantize X^T (RHT16)", "wgrad gemm"]
    # every GEMM on its preferred route (gemm_two_pass_preferred), the
    # two-pass workspace allocated once before timing
    shapes = {"fprop": (tok, d_out, d_in), "dgrad": (tok, d_in, d_out), "wgrad": (d_out, d_in, tok)}
    two = {g: M.gemm_two_pass_preferred(*mnk) for g, mnk in shapes.items()}
    ws_bytes = max([M.mixfp4_gemm_workspace_size(*shapes[g]) for g in shapes if two[g]] + [1])
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    wsp = {g: (ws if two[g] else None) for g in shapes}

    def step(e=None, it=0):
        def mark(i):
            if e is not None:
                e[i].record()
        mark(0)
        qx = M.mixfp4_quantize(X)
        mark(1)
        qw, qwt = M.mixfp4_quantize_2d(Wt)
        mark(2)
        M.mixfp4_gemm(qx, qw, workspace=wsp["fprop"])
        mark(3)
        qg = M.mixfp4_quantize(dY, rounding="stochastic", seed=it)
        mark(4)
        M.mixfp4_gemm(qg, qwt, workspace=wsp["dgrad"])
        mark(5)
        qgt = M.mixfp4_quantize(dY, rounding="stochastic", seed=it, offset=1, hadamard_block=16,
                                hadamard_signs=signs, transpose=True)
        mark(6)
        qxt = M.mixfp4_quantize(X, hadamard_block=16, hadamard_signs=signs, transpose=True)
        mark(7)
        M.mixfp4_gemm(qgt, qxt, workspace=wsp["wgrad"])
        mark(8)

    spin_up(torch, step, 0.3)
    # step time without events, then the per-launch spans in a second pass
    t0 = time.perf_counter()
    for i in range(iters):
        step(None, i)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / iters
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(9)] for _ in range(iters)]
    for i in range(iters):
        step(ev[i], i)
    torch.cuda.synchronize()
    spans = [float(np.mean([e[j].elapsed_time(e[j + 1]) for e in ev])) for j in range(8)]
    flops = 2.0 * tok * d_in * d_out
    # The 2D weight quantizer on its own, back to back, W's tensor scale given:
    # 2 B read, both layouts' codes and scales written (3.125 B/element).  In
    # the step it runs right after the GEMMs, at the clock they leave.
    w_ts = M.mixfp4_quantize_2d(Wt)[0][2].clone()
    q2d = lambda: M.mixfp4_quantize_2d(Wt, tensor_scale=w_ts)
    spin_up(torch, q2d, 0.2)
    b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    b0.record()
    for _ in range(20):
        q2d()
    b1.record()
    torch.cuda.synchronize()
    q2d_us = b0.elapsed_time(b1) / 20 * 1e3
    q2d_gbps = d_out * d_in * 3.125 / (q2d_us * 1e-6) / 1e9
    out = {
        "workload": "train_7b: X[2048,4096] Student-t nu=4 (8 channels x50), W[11008,4096] "
                    "N(0,0.02), dY[2048,11008] 1e-4 Student-t nu=3 (16 channels x20)",
        "ms_per_step": round(ms, 4),
        "gemm_TFLOPs_per_step": round(3 * flops / (ms * 1e-3) / 1e12, 2),
        "us": {n: round(v * 1e3, 2) for n, v in zip(names, spans)},
        "gemm_TFLOPs": {n: round(flops / (spans[j] * 1e-3) / 1e12, 1)
                        for n, j in (("fprop", 2), ("dgrad", 4), ("wgrad", 7))},
        "gemm_path": {g: ("two-pass (both operands decoded in the call)" if two[g] else "fused")
                      for g in shapes},
        "quantize_GBps": {n: round(el * QUANT_BYTES_PER_ELEM / (spans[j] * 1e-3) / 1e9, 1)
                          for n, j, el in (("quantize_2d W (COMPUTE)", 1, d_out * d_in),
                                           ("quantize dY^T (COMPUTE, RHT16, SR)", 5, tok * d_out),
                                           ("quantize X^T (COMPUTE, RHT16)", 6, tok * d_in))},
        "quantize_2d_standalone": {
            "what": "mixfp4_quantize_2d of W[11008,4096] (both layouts) back to back, s32 given",
            "us": round(q2d_us, 2), "GBps": round(q2d_gbps, 1), "bytes_per_elem": 3.125,
            "hbm_frac": round(q2d_gbps / 8000.0, 4)},
    }
    del X, Wt, dY, t, ws
    torch.cuda.empty_cache()
    return out


def gemm_decoded_bytes(m: int, n: int, k: int) -> float:
    """Algorithmic HBM bytes of one GEMM launch on decoded operands: the 16-bit
    A and W read once and the fp32 C written."""
    return (m + n) * k * 2.0 + 4.0 * m * n


def measure_prefill(M, torch, dev, wl, steps: int, warmup: int, spin_s: float) -> dict:
    """One prefill step of a workload: quantize A (tensor scale computed on the
    device), then every GEMM of the workload on the path the library's rule
    picks for its shape (gemm_two_pass_preferred): two passes (A decoded once
    into exact 16-bit values for all of the step's two-pass GEMMs, the weight
    decoded, then the GEMM on the decoded operands; the passes of
    mixfp4_gemm_ws, called separately so that A is decoded once and every
    kernel has its own span) or the fused kernel (mixfp4_gemm, which decodes
    inside its MFMA loop).  The weights are quantized before timing; their
    decode is inside the step.  The step time comes from `steps` steps with
    nothing else on the stream, timed wall-clock between device
    synchronizations, after `warmup` untimed steps and `spin_s` seconds of
    untimed steps that bring the clocks to their loaded level.  The
    per-launch spans come from a second pass of the same steps with HIP
    events recorded on the launching stream around each launch (an event
    adds ~3.5 us of GPU time between launches, so the step time is taken
    without them).  Both paths are also timed back to back on the same
    operands for every GEMM, whichever the step uses."""
    x = {n: torch.from_numpy(b.view(np.int16)).to(dev).view(torch.bfloat16)
         for n, b in wl.tensors.items()}
    wnames = [w for _, w in wl.gemms]
    qw = {w: M.mixfp4_quantize(x[w]) for w in wnames}
    for w in wnames:
        del x[w]
    ra, ka = x["A"].shape
    qa = (torch.empty((ra, ka // 2), dtype=torch.uint8, device=dev),
          torch.empty((ra, ka // 16), dtype=torch.uint8, device=dev),
          torch.empty(1, dtype=torch.float32, device=dev))
    outs = {w: torch.empty((ra, qw[w][0].shape[0]), dtype=torch.float32, device=dev)
            for w in wnames}
    two = {w: M.gemm_two_pass_preferred(ra, qw[w][0].shape[0], ka) for w in wnames}
    # decoded-operand buffers, allocated once (the step writes them every time)
    da = M.mixfp4_decode_operand(qa)
    dws = {w: M.mixfp4_decode_operand(qw[w]) for w in wnames}
    torch.cuda.synchronize()
    nspan = 2 + 2 * len(wnames)

    fused_a = any(two.values())

    def step(e=None):
        if e is not None:
            e[0].record()
        if fused_a:
            # A quantized and decoded for the two-pass GEMMs in one pass
            M.mixfp4_quantize_decode(x["A"], None, out=da.buf, codes=qa[0], scales=qa[1],
                                     scale_out=qa[2])
        else:
            M.mixfp4_quantize(x["A"], None, qa[0], qa[1], scale_out=qa[2])
        if e is not None:
            e[1].record()
        for i, w in enumerate(wnames):
            if e is not None:
                e[2 + 2 * i].record()
            if two[w]:
                M.mixfp4_decode_operand(qw[w], out=dws[w].buf)
            if e is not None:
                e[3 + 2 * i].record()
            if two[w]:
                M.mixfp4_gemm_decoded(da, dws[w], out=outs[w])
            else:
                M.mixfp4_gemm(qa, qw[w], out=outs[w])
        if e is not None:
            e[nspan].record()

    for _ in range(warmup):
        step()
    spin_up(torch, step, spin_s)
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / steps
    marks = [[torch.cuda.Event(enable_timing=True) for _ in range(nspan + 1)]
             for _ in range(steps)]
    for i in range(steps):
        step(marks[i])
    torch.cuda.synchronize()
    span = lambda a, b: float(np.mean([m[a].elapsed_time(m[b]) for m in marks]))  # noqa: E731
    q_ms = span(0, 1)
    gemms = {}
    total_flops = 0.0

    def back_to_back(f) -> float:
        spin_up(torch, f, 0.1)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            f()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    for i, w in enumerate(wnames):
        n = qw[w][0].shape[0]
        fl = 2.0 * ra * n * ka
        total_flops += fl
        dw_ms = span(2 + 2 * i, 3 + 2 * i)
        g_ms = span(3 + 2 * i, 4 + 2 * i)
        tf = fl / (g_ms * 1e-3) / 1e12
        dec_bytes = n * ka * (0.5 + 1 / 16 + 2)
        gemms[w] = {"shape": [ra, n, ka], "flops": fl,
                    "path": "two-pass" if two[w] else "fused",
                    "kernel": "gemm_f16_kernel (decoded operands)" if two[w]
                    else "gemm_kernel (decode inside the MFMA loop)",
                    "us_per_launch": round(g_ms * 1e3, 2),
                    "achieved": round(tf, 2), "unit": "TFLOP/s",
                    "frac": round(tf / PEAK_F16_TFLOPS, 4),
                    "gemm_call_us": round((dw_ms + g_ms) * 1e3, 2),
                    "gemm_call_TFLOPs": round(fl / ((dw_ms + g_ms) * 1e-3) / 1e12, 2)}
        if two[w]:
            gemms[w]["decode_w_us"] = round(dw_ms * 1e3, 2)
            gemms[w]["decode_w_GBps"] = round(dec_bytes / (dw_ms * 1e-3) / 1e9, 1)
        # both paths back to back on the same operands (A decoded beforehand
        # for the two-pass one, as the step does once for all its GEMMs)
        f_ms = back_to_back(lambda: M.mixfp4_gemm(qa, qw[w], out=outs[w]))
        M.mixfp4_decode_operand(qa, out=da.buf)

        def two_pass_call():
            M.mixfp4_decode_operand(qw[w], out=dws[w].buf)
            M.mixfp4_gemm_decoded(da, dws[w], out=outs[w])
        t_ms = back_to_back(two_pass_call)
        gemms[w]["fused_call"] = {"kernel": "gemm_kernel", "us": round(f_ms * 1e3, 2),
                                  "TFLOPs": round(fl / (f_ms * 1e-3) / 1e12, 2),
                                  "frac": round(fl / (f_ms * 1e-3) / 1e12 / PEAK_F16_TFLOPS, 4)}
        gemms[w]["two_pass_call"] = {"kernels": "decode_blocked_kernel (W) + gemm_f16_kernel",
                                     "us": round(t_ms * 1e3, 2),
                                     "TFLOPs": round(fl / (t_ms * 1e-3) / 1e12, 2)}
    out = {"ms_per_step": round(ms_step, 4), "steps": steps, "warmup": warmup,
           "spin_up_s": spin_s,
           "step_TFLOPs": round(total_flops / (ms_step * 1e-3) / 1e12, 3),
           "gemm_flops_per_step": total_flops,
           "path_rule": "two passes where m n / (m + n) >= 1280 (gemm_two_pass_preferred), "
                        "else the fused kernel",
           "quantize_a": ({"what": f"A[{ra},{ka}] quantized and decoded for the two-pass GEMM "
                                   "in one pass (mixfp4_quantize_decode: amax pass + reduction + "
                                   "quantize_decode_kernel), tensor scale computed on the device",
                           "us": round(q_ms * 1e3, 2),
                           "GBps": round(ra * ka * (QUANT_BYTES_PER_ELEM + 2.0) / (q_ms * 1e-3)
                                         / 1e9, 1),
                           "bytes_per_elem": QUANT_BYTES_PER_ELEM + 2.0,
                           "bytes_note": "2 B read + 0.5625 B of codes and scales + 2 B of "
                                         "decoded operand written (the amax pass's read of A "
                                         "is not counted)"}
                          if fused_a else
                          {"what": f"A[{ra},{ka}] with the tensor scale computed on the device "
                                   "(amax pass + reduction + quantize kernel)",
                           "us": round(q_ms * 1e3, 2),
                           "GBps": round(ra * ka * QUANT_BYTES_PER_ELEM / (q_ms * 1e-3) / 1e9, 1),
                           "bytes_per_elem": QUANT_BYTES_PER_ELEM}),
           "gemms": gemms}
    del x, qw, qa, outs, da, dws
    torch.cuda.empty_cache()
    return out


SECTIONS = ("large", "quantize", "prefill_7b", "rotated", "decode", "train")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--spin-up", type=float, default=0.5,
                    help="seconds of untimed steps before the timed ones (loaded clocks)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only", default=",".join(SECTIONS),
                    help="comma-separated sections to run (profiling runs isolate one)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run one elementwise copy of 512 MiB (read + write of known "
                         "size) so hardware byte counters can be scaled")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the MixFP4 path here runs on a single MI355X "
              "(--gpus 1).", file=sys.stderr)
        sys.exit(2)
    only = set(args.only.split(","))
    unknown = only - set(SECTIONS)
    if unknown:
        print(f"unknown sections {sorted(unknown)}; choose from {SECTIONS}", file=sys.stderr)
        sys.exit(2)

    import workloads as W
    wl5 = None
    cpu = None
    if "large" in only:
        log("generating the large workload (seed 4): A[16384,8192], W[8192,8192]")
        wl5 = W.large(tensors=("A", "W"))
        if not args.no_cpu_baseline:
            cpu = cpu_baseline(wl5)
            log(f"cpu baseline: {cpu['value']:.4g} TFLOP/s ({cpu['sample']})")

    import torch

    import paper_2605_31035_amd as M
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.calibrate_copy:
        src = torch.ones(128 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    out = {"metric": METRIC, "value": None, "unit": "TFLOP/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": None,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "fp16", "data": "synthetic"}
    if wl5 is not None:
        log("large step: quantize A[16384,8192] + GEMM 16384x8192x8192")
        r = measure_prefill(M, torch, dev, wl5, args.steps, args.warmup, args.spin_up)
        del wl5
        g = r["gemms"]["W"]
        out["value"] = r["step_TFLOPs"]
        out["ms_per_step"] = r["ms_per_step"]
        out["config"] = {
            "workload": "large (seed 4): quantize A[16384,8192] (block mixture: 90% of "
                        "16-blocks N(0,0.1), 10% Laplace(0,1) with one x40 spike; tensor scale "
                        "computed on the device) and decode it to exact 16-bit values in the "
                        "same pass, decode W, then C = A W^T [16384,8192] fp32; W[8192,8192] "
                        "N(0,0.02) quantized before timing (its decode is inside the step)",
            "seed": 4, "gemm_flops_per_step": r["gemm_flops_per_step"],
            "quantized_elements_per_step": 16384 * 8192, "spin_up_s": args.spin_up,
            "timing": "value: K steps back to back, wall clock between device "
                      "synchronizations, after W warmup steps and spin_up_s seconds of "
                      "untimed steps (loaded clocks)"}
        out["roofline"] = {"bound": "mfma",
                           "kernel": "gemm_f16_kernel on decoded operands, C = A W^T "
                                     "16384x8192x8192, 256x256 tiles (2048 tiles: 8 whole rounds "
                                     "of 256 CUs, one launch)",
                           "achieved": g["achieved"], "peak": PEAK_F16_TFLOPS,
                           "unit": "TFLOP/s", "frac": g["frac"],
                           "traffic": gemm_traffic_bytes(),
                           "algorithmic_bytes": gemm_decoded_bytes(16384, 8192, 8192),
                           "flops_per_launch": g["flops"],
                           "us_per_launch": g["us_per_launch"]}
        out["quantize_step"] = r["quantize_a"]
        out["decode_w"] = {"kernel": "decode_blocked_kernel", "us": g["decode_w_us"],
                           "GBps": g["decode_w_GBps"], "bound": "hbm",
                           "bytes_per_elem": 0.5 + 1 / 16 + 2}
        out["gemm_call"] = {"what": "decode W + GEMM (the mixfp4_gemm_ws work for an operand "
                                    "decoded once) in the step, and both paths back to back",
                            "path": g["path"], "us": g["gemm_call_us"],
                            "TFLOPs": g["gemm_call_TFLOPs"],
                            "two_pass_call": g["two_pass_call"], "fused_call": g["fused_call"]}
    if "quantize" in only:
        out["quantize"] = measure_quantize(M, torch, dev)
    if "prefill_7b" in only:
        log("generating prefill_7b workload (seed 1)")
        r = measure_prefill(M, torch, dev, W.prefill_7b(), args.steps, min(args.warmup, 20), 0.3)
        r["workload"] = ("prefill_7b (seed 1): quantize A[2048,4096] (Student-t nu=4, 8 outlier "
                         "channels x50), C1 = A W1^T [2048,11008], C2 = A W2^T [2048,4096]; "
                         "W1, W2 N(0,0.02) quantized before timing")
        out["prefill_7b"] = r
    if "rotated" in only:
        log("generating rotated workload (seed 2)")
        r = measure_prefill(M, torch, dev, W.rotated(), args.steps, min(args.warmup, 20), 0.3)
        r["workload"] = ("rotated (seed 2): quantize A[4096,4096] (Student-t nu=3 times "
                         "blockdiag(H128/sqrt(128)) along K), C = A W^T [4096,14336]; W rotated "
                         "the same way, quantized before timing")
        out["rotated"] = r
    if "decode" in only:
        out["decode_shape"] = measure_decode(M, torch, dev)
    if "train" in only:
        out["train_step"] = measure_train(M, torch, dev)
    out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
