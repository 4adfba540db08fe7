"""Cached-context action decoding throughput on one MI355X.

Workload (default): the 12-layer d=1024 decoder (16 heads of 64, FFN 4096,
256 action bins), 8 episodes, each with a cached prefix of 256 patch
embeddings + 24 instruction tokens, 7 greedy action tokens per step.  The
timed region is one episode window: ctx_build of the 8 prefixes followed by
K ctx_steps (K = 500 by default), inputs resident in HBM beforehand.
Each step = 7 bin-logit evaluations and 6 decode passes over all layers.

Prints one JSON line: action steps/s (rows x steps / s), the roofline of the
dominant kernel (timed live with HIP events on its own stream), and the fp64
CPU reference timed on a bounded sample on this host.
"""
from __future__ import annotations

import argparse
import ctypes as C
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, GB/s
MFMA_F16_PEAK_TFLOPS = 2500.0  # dense fp16/bf16


def step_bytes(spec, lens, n_actions, es=2):
    """Algorithmic bytes of one ctx_step with no new tokens: every decode pass
    reads all matmul weights once and each row's K/V up to its current
    position, writes the new token's K/V; every action reads the bin head."""
    d, L = spec.d_model, spec.n_layers
    w = spec.matmul_params * es
    kv_tok = L * 2 * d * es
    total = 0
    for j in range(1, n_actions):
        total += w
        total += sum(int(l) + j for l in lens) * kv_tok  # keys 0..L_b+j-1 incl. the new one
        total += len(lens) * kv_tok  # append
    total += n_actions * spec.n_bins * d * es
    return total


def build_flops(spec, lens):
    """Matmul + attention FLOPs of ctx_build."""
    d, L = spec.d_model, spec.n_layers
    m = sum(int(l) for l in lens)
    pairs = sum(int(l) * (int(l) + 1) // 2 for l in lens)
    return 2 * spec.matmul_params * m + 4 * d * L * pairs


def gu_launch_bytes(spec, B, es=2):
    """Decode gate|up projection: weights [2F, d] once, the input rows and the [B, F] gated
    out, both as fp16 pairs (hi + lo, 4 bytes a value); from 9 to 64 rows the wide kernel
    leaves the out to its split-K reduction."""
    w = 2 * spec.d_ffn * spec.d_model * es + B * spec.d_model * 4
    return w + (B * spec.d_ffn * 4 if B <= 8 or B > 64 else 0)


def time_gate_up_kernel(model, B, iters=240):
    """Average duration of the decode gate|up kernel (RMSNorm + gate|up GEMV + SiLU gate,
    the largest weight stream of a decode pass) in the decode step's launch shape, timed with
    HIP events on its own stream.  Each launch reads a different copy of a layer's packed
    weights out of a buffer of at least 1 GiB, four times the 256 MB memory-side cache, so
    that every launch streams its weights from HBM as it does inside a decode pass."""
    import torch
    from paper_2508_10259_amd.build import PROBE_LIB
    lib = C.CDLL(PROBE_LIB)
    spec = model.spec
    d, F, es = spec.d_model, spec.d_ffn, 2
    # packed layout of the model workspace: [wqkv | wo | wgu | ...], each region 256-byte aligned
    align = lambda x: (x + 255) // 256 * 256
    off_gu = align(3 * d * d * es * spec.n_layers) + align(d * d * es * spec.n_layers)
    slice_b = 2 * F * d * es
    n_copy = max(4, -(-(1 << 30) // slice_b))
    wbuf = torch.empty((n_copy, slice_b), dtype=torch.uint8, device="cuda")
    for i in range(n_copy):
        l = i % spec.n_layers
        wbuf[i].copy_(model.ws[off_gu + l * slice_b: off_gu + (l + 1) * slice_b])
    # the decode pass's form: inputs and SwiGLU output as fp16 pairs (hi + rounding error)
    h = torch.randn((B, d), device="cuda") * 30.0
    hhi = h.half()
    hlo = (h - hhi.float()).half()
    u = torch.randn((B, d), device="cuda")
    uhi = u.half()
    ulo = (u - uhi.float()).half()
    a = torch.empty((B, F), device="cuda", dtype=torch.float16)
    alo = torch.empty((B, F), device="cuda", dtype=torch.float16)
    # split count of the wide kernel over its 128-row tiles (the library's rule: the smallest
    # S <= min(16, chunks / 4) within 5% of the minimum of ceil(tiles * S / 256) / S)
    tiles, smax = max(2 * F // 128, 1), max(1, min(16, d // 128 // 4))
    model = {s_: -(-tiles * s_ // 256) / s_ for s_ in range(1, smax + 1)}
    wsplit = min(s_ for s_, t_ in model.items() if t_ <= 1.05 * min(model.values()))
    part = torch.empty((wsplit, B, 2 * F) if 8 < B <= 64 else (1,), device="cuda", dtype=torch.float32)
    s = torch.cuda.Stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def launch(l):
        w = C.c_void_p(wbuf[l % n_copy].data_ptr())
        if B <= 8:  # the decode pass fuses the RMSNorm up to 8 rows
            lib.ams_probe_gemv_rmsnorm(2, 2, C.c_void_p(hhi.data_ptr()), C.c_void_p(hlo.data_ptr()),
                                       C.c_float(spec.rms_eps), w, B, 2 * F, d, C.c_void_p(a.data_ptr()), F,
                                       C.c_void_p(None), C.c_void_p(alo.data_ptr()), C.c_void_p(s.cuda_stream))
        elif B <= 64:  # the wide kernel writes split-K partial sums; the reduction is timed apart
            lib.ams_probe_gemm_wide(C.c_void_p(uhi.data_ptr()), C.c_void_p(ulo.data_ptr()), w, B, 2 * F, d,
                                    wsplit, C.c_void_p(part.data_ptr()), C.c_void_p(s.cuda_stream))
        else:
            lib.ams_probe_gemm(2, 2, C.c_void_p(uhi.data_ptr()), C.c_void_p(ulo.data_ptr()), w, B, 2 * F, d,
                               C.c_void_p(a.data_ptr()), F, C.c_void_p(None), C.c_void_p(alo.data_ptr()),
                               C.c_void_p(s.cuda_stream))
    torch.cuda.synchronize()
    iters = max(iters, 2 * n_copy)
    with torch.cuda.stream(s):
        for l in range(n_copy):
            launch(l)
        ev0.record(s)
        for l in range(iters):
            launch(l)
        ev1.record(s)
    s.synchronize()
    del wbuf
    return ev0.elapsed_time(ev1) / iters * 1e-3  # seconds per launch


def profiled_traffic(workload, kernel):
    """HBM bytes per launch of the roofline kernel from a committed PMC summary
    (profiles/*_pmc.txt) of this workload and kernel, or None when there is none or
    the kernel's source has changed since the counters were taken."""
    import glob
    import hashlib
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*_pmc.txt"))):
        try:
            kv = dict(l.strip().split("=", 1) for l in open(path) if "=" in l and not l.startswith("#"))
            if kv.get("workload") != workload or kv.get("kernel") != kernel:
                continue
            src = open(os.path.join(ROOT, kv["kernel_source"]), "rb").read()
            if hashlib.sha256(src).hexdigest() != kv["kernel_source_sha256"]:
                return None
            return int(kv["traffic_bytes"])
        except (OSError, KeyError, ValueError):
            continue
    return None


def time_persistent_step(ctx, n_actions, iters=40):
    """Average duration of a decode-only ctx_step when the decode is one persistent
    launch (that launch plus the small kernel that clears its barrier words), timed
    with HIP events on torch's current stream, where the step's graph runs."""
    import torch
    B, nb = ctx.batch, ctx.model.spec.n_bins
    tokens = torch.empty((B, n_actions), dtype=torch.int32, device="cuda")
    logits = torch.empty((B, n_actions, nb), dtype=torch.float32, device="cuda")
    for _ in range(3):
        ctx.step(n_actions, tokens=tokens, logits=logits)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(iters):
        ctx.step(n_actions, tokens=tokens, logits=logits)
    ev1.record()
    torch.cuda.synchronize()
    return ev0.elapsed_time(ev1) / iters * 1e-3


def measured_peaks(nbytes=1 << 30, iters=10):
    """The two roofs measured on this GPU (the library's peak kernels): HBM stream copy and
    read of 1 GiB buffers (four times the 256 MB memory-side cache; best of three grid sizes,
    copy counted as read + write bytes) and the dense fp16 MFMA rate of register-only MFMA
    chains on every SIMD."""
    import torch
    from paper_2508_10259_amd.build import PROBE_LIB
    lib = C.CDLL(PROBE_LIB)
    lib.ams_probe_mfma_loop_flops.restype = C.c_double
    s = torch.cuda.current_stream()
    sp = C.c_void_p(s.cuda_stream)
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    red = torch.empty(8192 * 256, dtype=torch.float32, device="cuda")
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def rate(launch, nbytes_moved):
        for _ in range(2):
            assert launch() == 0
        ev0.record(s)
        for _ in range(iters):
            launch()
        ev1.record(s)
        torch.cuda.synchronize()
        return nbytes_moved / (ev0.elapsed_time(ev1) / iters * 1e-3) / 1e9

    copy = max(rate(lambda g=g: lib.ams_probe_stream_copy(C.c_void_p(src.data_ptr()), C.c_void_p(dst.data_ptr()),
                                                          C.c_size_t(nbytes), g, sp), 2 * nbytes)
               for g in (2048, 4096, 8192))
    read = max(rate(lambda g=g: lib.ams_probe_stream_read(C.c_void_p(src.data_ptr()), C.c_size_t(nbytes),
                                                          C.c_void_p(red.data_ptr()), g, sp), nbytes)
               for g in (2048, 4096, 8192))
    grid, mi = 2048, 4000
    fl = lib.ams_probe_mfma_loop_flops(mi, grid)
    by_shape = [rate(lambda sh=sh: lib.ams_probe_mfma_loop(sh, C.c_float(1.0), mi, C.c_void_p(red.data_ptr()), grid,
                                                         sp), fl) / 1e3 for sh in (0, 1)]
    tflops = max(by_shape)
    del src, dst, red
    return {"hbm_copy_GBps": round(copy, 1), "hbm_read_GBps": round(read, 1), "mfma_f16_TFLOPs": round(tflops, 1),
            "mfma_f16_TFLOPs_16x16x32": round(by_shape[0], 1), "mfma_f16_TFLOPs_32x32x16": round(by_shape[1], 1),
            "how": "stream copy (read + write bytes) and read of 1 GiB; fp16 MFMA 16x16x32 / 32x32x16 register chains, best"}


def copy_calibration(nbytes=256 << 20):
    """A device-to-device copy of known size, for scaling the FETCH_SIZE/WRITE_SIZE counters."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    return nbytes


def cpu_baseline(wl, w, seed, sample_steps, window_steps):
    """fp64 reference on row 0 (same weights `w` as the GPU run): build its prefix, then
    `sample_steps` steps; row-steps/s with the build amortised over the workload's window."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle.decoder as D
    from ref_bridge import oracle_params, prefix_f64
    from paper_2508_10259_amd import workload as W
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    p = oracle_params(w)
    x = prefix_f64(p, wl.spec, W.make_prefix(wl, seed, 0, 0))
    new = [W.to_f32(W.make_observation(wl.spec, seed, 0, 0, wl.new_per_step), wl.spec.dtype).astype(np.float64)] \
        if wl.new_per_step else None
    for l in range(wl.spec.n_layers):  # decode every weight once before timing
        for n in W.MATRICES:
            p.layer(n, l)
    ctx = D.ActionContext(p, 1)
    t0 = time.perf_counter()
    ctx.build([x])
    t1 = time.perf_counter()
    for _ in range(sample_steps):
        ctx.step(new, wl.n_actions)
    t2 = time.perf_counter()
    per_step = (t2 - t1) / sample_steps + (t1 - t0) / window_steps
    return {"value": 1.0 / per_step, "unit": "action-steps/s", "cores": int(cores), "kind": "oracle",
            "sample": f"row 0 of {wl.name}: build of its {x.shape[0]}-token prefix ({t1 - t0:.2f} s) + "
                      f"{sample_steps} steps ({t2 - t1:.2f} s), fp64 NumPy; build amortised over "
                      f"{window_steps} steps as in the timed GPU window"}


def make_inputs(model, wl, seed, steps, device_draws):
    """Every input of the timed window, resident in HBM: one packed prefix set per build
    epoch and a pool of per-step observation tokens (one invalidation window's worth)."""
    import torch
    from paper_2508_10259_amd import workload as W
    inv = wl.invalidate_every
    n_epochs = 1 + (steps - 1) // inv if inv else 1
    epochs = []
    for e in range(n_epochs):
        lens = W.prefix_lengths(wl, seed, e)
        if device_draws:
            pre = [W.make_prefix_device(wl, seed, e, b, int(lens[b])) for b in range(wl.batch)]
        else:
            pre = [W.make_prefix(wl, seed, e, b, int(lens[b])) for b in range(wl.batch)]
        epochs.append(model.pack_prefixes(pre))
    pool = []
    if wl.new_per_step:
        for s in range(min(steps, inv or steps)):
            pool.append(W.make_observation_device(wl.spec, seed, s, wl.batch, wl.new_per_step))
    torch.cuda.synchronize()
    return epochs, pool


def roofline_kernel_name(spec, A, B, persistent):
    """The dominant decode kernel of a workload, as its roofline entry and profiles name it."""
    if persistent:
        return f"k_decode_fused<{spec.head_dim}> (persistent decode: head, feed and {A - 1} passes of every layer)"
    return ("k_gemm_skinny<2,1,SWIGLU,NRM> (decode RMSNorm + gate|up projection + SiLU gate)" if B <= 8
            else f"k_gemm_wide<{(B + 15) // 16},2> (decode gate|up projection, split-K partial sums)"
            if B <= 64 else "k_gemm_tiled or k_gemm_big (decode gate|up projection + SiLU gate)")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="default: the workload's step count")
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="mid-b8")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-steps", type=int, default=100)
    ap.add_argument("--recompute", action="store_true",
                    help="invalidate + rebuild the prefix before every step (the no-reuse comparison)")
    ap.add_argument("--roofline-only", action="store_true",
                    help="time only the roofline kernel (and the calibration copy), print one JSON line and exit: "
                         "the command the profiles' counter runs use")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the decoder shards by episode, "
              "one process per GPU, with no communication on the hot path", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2508_10259_amd import workload as W
    from paper_2508_10259_amd.runtime import DeviceContext, DeviceModel

    wl = W.WORKLOADS[args.workload]
    spec = wl.spec
    steps = args.steps if args.steps is not None else wl.steps
    big = spec.matmul_params > 1e9
    torch.cuda.set_device(0)
    print(f"[bench] {wl.name}: weights", file=sys.stderr, flush=True)
    weights = W.make_device_weights(spec, args.seed) if big else W.make_weights(spec, args.seed)
    model = DeviceModel(weights, "cuda:0")
    cap = wl.derived_capacity()
    ctx = DeviceContext(model, wl.batch, cap)
    persistent = ctx.persistent_decode
    print(f"[bench] inputs (capacity {cap}, persistent decode {persistent})", file=sys.stderr, flush=True)
    epochs, pool = make_inputs(model, wl, args.seed, steps, big)
    B, A = wl.batch, wl.n_actions
    if args.roofline_only:
        if persistent:
            ctx.build(*epochs[0])
            t_k = time_persistent_step(ctx, A)
        else:
            t_k = time_gate_up_kernel(model, B)
        copy_calibration()
        print(json.dumps({"workload": wl.name, "kernel": roofline_kernel_name(spec, A, B, persistent),
                          "avg_launch_us": round(t_k * 1e6, 3)}), flush=True)
        ctx.close()
        model.close()
        return
    tokens = torch.empty((B, A), dtype=torch.int32, device="cuda")
    logits = torch.empty((B, A, spec.n_bins), dtype=torch.float32, device="cuda")
    new_lens = [wl.new_per_step] * B if wl.new_per_step else None
    inv = wl.invalidate_every

    def window(n_steps):
        """One build then n_steps steps, with the workload's rebuilds; returns (t_build, t_steps)."""
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev[0].record()
        ctx.build(*epochs[0])
        ev[1].record()
        for s_ in range(n_steps):
            if inv and s_ and s_ % inv == 0:
                ctx.invalidate()
                ctx.build(*epochs[(s_ // inv) % len(epochs)])
            if args.recompute and s_:
                ctx.invalidate()
                ctx.build(*epochs[0])
            new = pool[s_ % len(pool)] if pool else None
            ctx.step(A, new, new_lens, tokens=tokens, logits=logits)
        ev[2].record()
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) * 1e-3, ev[1].elapsed_time(ev[2]) * 1e-3

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    window(min(args.warmup, inv or args.warmup))
    t_build, t_steps = window(steps)
    total = t_build + t_steps
    value = B * steps / total
    lens = epochs[0][1]
    sb = step_bytes(spec, lens, A)
    print(f"[bench] build {t_build * 1e3:.3f} ms, {steps} steps {t_steps * 1e3:.1f} ms", file=sys.stderr,
          flush=True)

    kname = roofline_kernel_name(spec, A, B, persistent)
    if persistent:
        # the step's whole decode is one launch: its algorithmic bytes are the step's
        t_k = time_persistent_step(ctx, A)
        kb = sb
    else:
        t_k = time_gate_up_kernel(model, B)
        kb = gu_launch_bytes(spec, B)
    achieved = kb / t_k / 1e9
    copy_calibration()
    peaks = measured_peaks()
    hbm_meas = max(peaks["hbm_copy_GBps"], peaks["hbm_read_GBps"])
    roof = {"kernel": kname, "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": profiled_traffic(wl.name, kname.split(" ")[0]),
            "bytes_per_launch": kb, "avg_launch_us": round(t_k * 1e6, 3),
            "frac_vs_measured": round(achieved / hbm_meas, 4)}

    out = {
        "metric": "action steps/s per GPU (cached-context decode)",
        "value": round(value, 2), "unit": "action-steps/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": round(total / steps * 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "fp16",
        "data": "synthetic (seeded N(0,0.02) weights stored bf16, N(0,1) patch embeddings, uniform ids)",
        "config": {"workload": wl.name, "n_layers": spec.n_layers, "d_model": spec.d_model,
                   "n_heads": spec.n_heads, "head_dim": spec.head_dim, "d_ffn": spec.d_ffn,
                   "vocab": spec.vocab, "n_bins": spec.n_bins, "batch": B, "prefix_tokens": int(lens[0]),
                   "n_actions": A, "capacity": cap, "new_tokens_per_step": wl.new_per_step,
                   "invalidate_every": inv, "recompute_each_step": bool(args.recompute),
                   "timed": f"1 build + {steps} steps" + (f" (rebuild every {inv})" if inv else "")
                            + (" (rebuild before every step)" if args.recompute else "")},
        "roofline": roof,
        "step": {"ms": round(t_steps / steps * 1e3, 4), "algorithmic_bytes_no_new_tokens": sb,
                 "hbm_frac": round(sb / (t_steps / steps) / (HBM_PEAK_GBS * 1e9), 4),
                 "hbm_frac_vs_measured": round(sb / (t_steps / steps) / (hbm_meas * 1e9), 4)},
        "build": {"ms": round(t_build * 1e3, 4), "flops": build_flops(spec, lens),
                  "mfma_frac": round(build_flops(spec, lens) / t_build / (MFMA_F16_PEAK_TFLOPS * 1e12), 4),
                  "mfma_frac_vs_measured": round(build_flops(spec, lens) / t_build / (peaks["mfma_f16_TFLOPs"] * 1e12),
                                                 4)},
        "measured_peaks": peaks,
    }
    ctx.close()
    model.close()
    del epochs, pool
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, weights, args.seed, args.cpu_sample_steps if not big else 1, steps)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
