"""Cached-context action decoding throughput on one MI355X.

Workload (default): the 7B Llama-style decoder (32 layers, d=4096, 32 heads of
128, FFN 11008, vocab 32000 with the last 256 ids as action bins), 64 parallel
episodes with ragged cached prefixes U{200..400} (patches + 32 instruction
tokens); per step every row commits 16 fresh observation tokens and decodes 7
greedy action tokens; every row is invalidated and rebuilt every 20 steps.  The
timed region is K steps (K = 20 by default) of that window -- one build of the
64 prefixes, then per step the 1,024-token extension (ams_ctx_append) and the
action decode (ams_ctx_step) -- with every input resident in HBM beforehand.

Each phase is timed live with HIP events on the stream the library enqueues on:
the decode against the HBM roofline (its algorithmic bytes: weights once per
pass, each row's K/V, the bin head), the extension and the rebuild against the
fp16 MFMA roofline; the whole step against the sum of the three rooflines.
Extra keys time the other workloads (7B one row, 7B 56-token action chunks with
and without reuse, the 12-layer model, and the batch-64 workload with row-level
rebuilds staggered over the steps), and the fp64 CPU reference is timed on a
bounded sample on this host.  One JSON line.
"""
from __future__ import annotations

import argparse
import ctypes as C
import json
import os
import subprocess
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


def build_flops(spec, lens, starts=None):
    """Matmul + attention FLOPs of ctx_build; starts[b]: the first position row b computes
    (the positions before it sit in prefix pages it shares with an earlier row)."""
    d, L = spec.d_model, spec.n_layers
    starts = starts if starts is not None else [0] * len(lens)
    m = sum(int(l) - int(s) for l, s in zip(lens, starts))
    pairs = sum(int(l) * (int(l) + 1) // 2 - int(s) * (int(s) + 1) // 2 for l, s in zip(lens, starts))
    return 2 * spec.matmul_params * m + 4 * d * L * pairs


def shared_starts(pt, lens, page=64):
    """First computed position of every row of a build that shares prefix pages: row b attaches
    the leading run of its pages that an earlier row of the same build holds."""
    seen, starts = set(), []
    for b, l in enumerate(lens):
        k = 0
        while k < (int(l) - 1) // page and int(pt[b, k]) in seen:
            k += 1
        starts.append(k * page)
        seen.update(int(x) for x in pt[b, :(int(l) + page - 1) // page])
    return starts


def extension_flops(spec, lens_before, n_new):
    """Matmul + attention FLOPs of appending n_new[b] tokens to rows of committed lengths
    lens_before[b]: new token i of row b attends to lens_before[b] + i + 1 keys."""
    d, L = spec.d_model, spec.n_layers
    m = sum(int(n) for n in n_new)
    pairs = sum(int(n) * int(l) + int(n) * (int(n) + 1) // 2 for l, n in zip(lens_before, n_new))
    return 2 * spec.matmul_params * m + 4 * d * L * pairs


def profiled_traffic(workload, kernel):
    """HBM bytes per launch (per step, for a whole phase) from a committed PMC summary
    (profiles/*_pmc.txt) of this workload and kernel, or None when there is none or a kernel
    source it covers has changed since the counters were taken."""
    import glob
    import hashlib
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*_pmc.txt"))):
        try:
            kv = dict(l.strip().split("=", 1) for l in open(path) if "=" in l and not l.startswith("#"))
            if kv.get("workload") != workload or kv.get("kernel") != kernel:
                continue
            srcs = kv.get("kernel_sources", kv.get("kernel_source", "")).split(",")
            shas = kv.get("kernel_sources_sha256", kv.get("kernel_source_sha256", "")).split(",")
            for src, sha in zip(srcs, shas):
                if hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest() != sha:
                    return None
            return int(kv["traffic_bytes"]), int(kv.get("algorithmic_bytes", 0)) or None
        except (OSError, KeyError, ValueError):
            continue
    return None


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


def lscpu_model():
    try:
        out = subprocess.run(["lscpu"], stdout=subprocess.PIPE, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except Exception:
        pass
    return "unknown"


def blas_info():
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                return {"vendor": i.get("internal_api"), "version": i.get("version"),
                        "threads": int(i.get("num_threads", 1))}
    except Exception:
        pass
    return {"vendor": "unknown", "version": None, "threads": len(os.sched_getaffinity(0))}


def _oracle_sample(wl, p, seed, n_steps, window_steps, n_layers=None):
    """fp64 reference on row 0 of `wl` (epoch 0): build of its prefix, then `n_steps` steps with
    the workload's per-step observation tokens.  With `n_layers` the reference runs the first
    n_layers layers of the model only and both times are scaled to all layers (the head's and
    the embedding gather's share is below 0.1%).  Returns (row-steps/s, build s, step s, text)."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle.decoder as D
    from ref_bridge import prefix_f64
    from paper_2508_10259_amd import workload as W
    spec = wl.spec
    if n_layers is not None:
        c = p.cfg
        p = D.Params(D.Config(n_layers, c.d_model, c.n_heads, c.head_dim, c.d_ffn, c.vocab, c.n_bins, c.rms_eps,
                              c.rope_theta), **p.arrays)
    L = p.cfg.n_layers
    for l in range(L):  # decode the sampled layers' weights before timing
        for n in W.MATRICES:
            p.layer(n, l)
    x = prefix_f64(p, spec, W.make_prefix(wl, seed, 0, 0))
    ctx = D.ActionContext(p, 1)
    t0 = time.perf_counter()
    ctx.build([x])
    t1 = time.perf_counter()
    for s_ in range(n_steps):
        new = [W.to_f32(W.make_observation(spec, seed, s_, 0, wl.new_per_step), spec.dtype).astype(np.float64)] \
            if wl.new_per_step else None
        ctx.step(new, wl.n_actions)
    t2 = time.perf_counter()
    scale = spec.n_layers / L
    t_build, t_step = (t1 - t0) * scale, (t2 - t1) / n_steps * scale
    per_step = t_step + t_build / window_steps
    what = (f"row 0 of {wl.name}: build of its {x.shape[0]}-token prefix ({t1 - t0:.2f} s) + {n_steps} step(s) "
            f"({t2 - t1:.2f} s)" + (f" through the first {L} of {spec.n_layers} layers, both scaled x{scale:g} "
                                    "to all layers" if n_layers is not None else "") +
            f"; fp64 NumPy; build amortised over {window_steps} steps as in the timed GPU window")
    return 1.0 / per_step, t_build, t_step, what


def cpu_baseline(wl, weights, seed, window_steps, others=True):
    """The fp64 reference as it stands, timed on this host's cores on a bounded sample of the
    timed workload (row 0; for the 7B model 4 of its 32 layers, scaled), plus the 2-layer and
    12-layer workloads with all BLAS threads and with one."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from ref_bridge import oracle_params
    from paper_2508_10259_amd import workload as W
    blas = blas_info()
    big = wl.spec.matmul_params > 1e9
    p = oracle_params(weights)
    v, tb, ts, what = _oracle_sample(wl, p, seed, 1 if big else 20, window_steps, n_layers=4 if big else None)
    del p
    out = {"value": v, "unit": "action-steps/s", "cores": blas["threads"], "kind": "oracle", "sample": what,
           "host_cpu": lscpu_model(), "blas": blas}
    if not others:
        return out
    from threadpoolctl import threadpool_limits
    extra, one = {}, {}
    for name, n in (("tiny-b1", 100), ("mid-b8", 10)):
        ow = W.WORKLOADS[name]
        if ow.name == wl.name:
            continue
        po = oracle_params(W.make_weights(ow.spec, seed))
        vo, _, _, wo = _oracle_sample(ow, po, seed, n, ow.invalidate_every or 20)
        extra[name] = {"value": vo, "cores": blas["threads"], "sample": wo}
        with threadpool_limits(limits=1, user_api="blas"):
            v1, _, _, w1 = _oracle_sample(ow, po, seed, max(2, n // 5), ow.invalidate_every or 20)
        one[name] = {"value": v1, "cores": 1, "sample": w1}
    out["other_workloads"] = extra
    out["one_thread"] = one
    return out


def make_inputs(model, wl, seed, steps, device_draws, stagger=False):
    """Every input of the timed window, resident in HBM: one packed prefix set per build
    epoch, a pool of per-step observation tokens (one invalidation window's worth) and, for
    staggered row rebuilds, the fresh prefixes of the rows rebuilt before each step."""
    import torch
    from paper_2508_10259_amd import workload as W
    inv = wl.invalidate_every
    n_epochs = 1 if stagger else (1 + (steps - 1) // inv if inv else 1)
    draw = W.make_prefix_device if device_draws else W.make_prefix
    epochs = []
    for e in range(n_epochs):
        lens = W.prefix_lengths(wl, seed, e)
        epochs.append(model.pack_prefixes([draw(wl, seed, e, b, int(lens[b])) for b in range(wl.batch)]))
    pool = []
    if wl.new_per_step:
        for s_ in range(min(steps, inv or steps)):
            pool.append(W.make_observation_device(wl.spec, seed, s_, wl.batch, wl.new_per_step))
    rebuild = {}
    if stagger:  # before step s the rows b with (s + b) % inv == 0: one residue class of s per entry
        for r in range(inv):
            rows = [b for b in range(wl.batch) if (r + b) % inv == 0]
            lens = W.prefix_lengths(wl, seed, 100 + r)
            packed, plens = model.pack_prefixes([draw(wl, seed, 100 + r, b, int(lens[b])) for b in rows])
            rebuild[r] = (rows, packed, plens)
    torch.cuda.synchronize()
    return epochs, pool, rebuild


def run_window(ctx, wl, epochs, pool, rebuild, steps, A, tokens, logits, mode):
    """One build then `steps` steps with the workload's rebuilds (mode "cached"), a rebuild
    before every step ("recompute"), or row-level rebuilds of the rows b with
    (step + b) % invalidate_every == 0 before each step ("staggered").  New observation
    tokens go in through ams_ctx_append, the action decode through ams_ctx_step (no new
    tokens), so each phase is bracketed by its own HIP events on the library's stream.
    Returns the window's duration and per-phase (seconds, algorithmic work) lists."""
    import torch
    spec = wl.spec
    inv = wl.invalidate_every
    new_lens = [wl.new_per_step] * wl.batch if wl.new_per_step else None
    marks = []  # (phase, ev0, ev1, work)

    def timed(phase, work, fn):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        marks.append((phase, e0, e1, work))

    def build_work(lens):
        # a build that shares prefix pages computes only the pages no earlier row holds (the
        # page table is the library's host copy: reading it does not wait for the GPU)
        if not ctx.share_prefix:
            return build_flops(spec, lens)
        return build_flops(spec, lens, shared_starts(ctx.pages()[0], lens))

    w0, w1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0.record()
    timed("build", 0, lambda: ctx.build(*epochs[0]))
    marks[-1] = marks[-1][:3] + (build_work(epochs[0][1]),)
    for s_ in range(steps):
        if mode == "cached" and inv and s_ and s_ % inv == 0:
            ctx.invalidate()
            e = epochs[(s_ // inv) % len(epochs)]
            timed("build", 0, lambda e=e: ctx.build(*e))
            marks[-1] = marks[-1][:3] + (build_work(e[1]),)
        elif mode == "recompute" and s_:
            ctx.invalidate()
            timed("build", 0, lambda: ctx.build(*epochs[0]))
            marks[-1] = marks[-1][:3] + (build_work(epochs[0][1]),)
        elif mode == "staggered" and s_:
            rows, packed, plens = rebuild[s_ % inv]
            ctx.invalidate_rows(rows)
            timed("build", build_flops(spec, plens), lambda: ctx.build_rows(rows, packed, plens))
        if new_lens:
            before = ctx.lengths()
            new = pool[s_ % len(pool)]
            timed("extension", extension_flops(spec, before, new_lens), lambda: ctx.append(new, new_lens))
        lens = ctx.lengths()
        timed("decode", step_bytes(spec, lens, A), lambda: ctx.step(A, tokens=tokens, logits=logits))
    w1.record()
    torch.cuda.synchronize()
    ph = {"build": [], "extension": [], "decode": []}
    for phase, e0, e1, work in marks:
        ph[phase].append((e0.elapsed_time(e1) * 1e-3, work))
    return w0.elapsed_time(w1) * 1e-3, ph


def phase_summary(entries, bound, peak):
    """Achieved rate of a phase over the window: its algorithmic work / its measured time."""
    if not entries:
        return None
    t = sum(e[0] for e in entries)
    w = sum(e[1] for e in entries)
    if bound == "hbm":
        return {"bound": "hbm", "achieved": round(w / t / 1e9, 1), "peak": peak, "unit": "GB/s",
                "frac": round(w / t / 1e9 / peak, 4), "bytes_per_launch": int(w / len(entries)),
                "avg_launch_us": round(t / len(entries) * 1e6, 1), "launches": len(entries)}
    return {"bound": "mfma", "achieved": round(w / t / 1e12, 1), "peak": peak, "unit": "TFLOP/s",
            "frac": round(w / t / 1e12 / peak, 4), "flops_per_launch": int(w / len(entries)),
            "avg_launch_us": round(t / len(entries) * 1e6, 1), "launches": len(entries)}


def measure(model, wl, seed, steps, warmup, mode, device_draws, share=False):
    """Warm-up window, then the timed window; returns the workload's figures.  share: a paged
    context whose rows share prefix pages (the build computes only unshared pages)."""
    import torch
    from paper_2508_10259_amd.runtime import DeviceContext
    spec = wl.spec
    cap = wl.derived_capacity()
    ctx = DeviceContext(model, wl.batch, cap, share_prefix=share)
    epochs, pool, rebuild = make_inputs(model, wl, seed, max(steps, warmup), device_draws,
                                        stagger=(mode == "staggered"))
    B, A = wl.batch, wl.n_actions
    tokens = torch.empty((B, A), dtype=torch.int32, device="cuda")
    logits = torch.empty((B, A, spec.n_bins), dtype=torch.float32, device="cuda")
    run_window(ctx, wl, epochs, pool, rebuild, warmup, A, tokens, logits, mode)
    t_win, ph = run_window(ctx, wl, epochs, pool, rebuild, steps, A, tokens, logits, mode)
    persistent = ctx.persistent_decode
    pages_in_use = ctx.pages()[2] if share else None
    ctx.close()
    del epochs, pool, rebuild
    dec = phase_summary(ph["decode"], "hbm", HBM_PEAK_GBS)
    ext = phase_summary(ph["extension"], "mfma", MFMA_F16_PEAK_TFLOPS)
    bld = phase_summary(ph["build"], "mfma", MFMA_F16_PEAK_TFLOPS)
    roof_s = (sum(w for _, w in ph["decode"]) / (HBM_PEAK_GBS * 1e9) +
              sum(w for _, w in ph["extension"] + ph["build"]) / (MFMA_F16_PEAK_TFLOPS * 1e12))
    return {"workload": wl.name, "mode": mode, "batch": B, "steps": steps, "capacity": cap,
            "persistent_decode": bool(persistent), "window_s": t_win, "value": B * steps / t_win,
            "ms_per_step": t_win / steps * 1e3, "decode": dec, "extension": ext, "build": bld,
            "pages_in_use": pages_in_use, "pages_total": wl.batch * (cap // 64),
            "step": {"ms": round(t_win / steps * 1e3, 4), "roofline_ms": round(roof_s / steps * 1e3, 4),
                     "frac": round(roof_s / t_win, 4),
                     "phases_ms": {k: round(sum(e[0] for e in v) / steps * 1e3, 4) for k, v in ph.items()}}}


def tier_rates(model, wl, seed, rows=8, device_draws=True):
    """The host tier on the workload's first build: `rows` rows moved to pinned host memory and
    back (library kernels writing / reading the host images), timed with HIP events, against
    dropping the same rows and rebuilding them from their inputs."""
    import torch
    from paper_2508_10259_amd.runtime import DeviceContext
    cap = wl.derived_capacity()
    ctx = DeviceContext(model, wl.batch, cap, n_pages=0)
    epochs, _, _ = make_inputs(model, wl, seed, 1, device_draws)
    ctx.build(*epochs[0])
    sel = list(range(rows))
    lens = ctx.lengths()
    bufs = [torch.empty(ctx.row_host_bytes(lens[r]), dtype=torch.uint8).pin_memory() for r in sel]
    from paper_2508_10259_amd import workload as W
    draw = W.make_prefix_device if device_draws else W.make_prefix
    packed, plens = model.pack_prefixes([draw(wl, seed, 0, b, int(lens[b])) for b in sel])
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    for rep in range(2):  # the second round is timed
        ev[0].record()
        ctx.offload_rows(sel, bufs)
        ev[1].record()
        ctx.reload_rows(sel, bufs)
        ev[2].record()
        ctx.invalidate_rows(sel)
        ev[3].record()
        ctx.build_rows(sel, packed, plens)
        ev[4].record()
        torch.cuda.synchronize()
    nbytes = sum(b.numel() for b in bufs)
    t_off, t_re, t_build = (ev[0].elapsed_time(ev[1]) * 1e-3, ev[1].elapsed_time(ev[2]) * 1e-3,
                            ev[3].elapsed_time(ev[4]) * 1e-3)
    ctx.close()
    return {"rows": rows, "tokens": int(sum(lens[r] for r in sel)), "host_bytes": int(nbytes),
            "offload_ms": round(t_off * 1e3, 3), "offload_GBps": round(nbytes / t_off / 1e9, 2),
            "reload_ms": round(t_re * 1e3, 3), "reload_GBps": round(nbytes / t_re / 1e9, 2),
            "rebuild_ms": round(t_build * 1e3, 3),
            "what": "rows moved to pinned host memory and back by the library's kernels vs dropped and rebuilt"}


def flow_rates(model, wl, seed, a=7, n_tokens=8, cold_steps=10, warm_steps=4, warm_tau=0.6, device_draws=True):
    """Flow-matching action head on the workload's rows (an 8 x 7 action chunk per row): a cold
    start from noise (cold_steps Euler steps from tau 0) against a warm start from a stored latent
    (warm_steps steps from warm_tau), timed with HIP events."""
    import torch
    from paper_2508_10259_amd import workload as W
    from paper_2508_10259_amd.runtime import DeviceContext, DeviceFlowHead
    ctx = DeviceContext(model, wl.batch, wl.derived_capacity())
    epochs, _, _ = make_inputs(model, wl, seed, 1, device_draws)
    ctx.build(*epochs[0])
    head = DeviceFlowHead(wl.spec, *W.make_flow_head(wl.spec, a, seed), n_tokens=n_tokens)
    x = torch.from_numpy(W.make_latent(seed, 0, wl.batch, n_tokens, a)).cuda()
    out = {}
    for name, tau0, k in (("cold", 0.0, cold_steps), ("warm", warm_tau, warm_steps)):
        ctx.flow(head, x, tau0, k)  # warm-up
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(3):
            ctx.flow(head, x, tau0, k)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 3
        out[name] = {"tau0": tau0, "euler_steps": k, "ms_per_chunk": round(ms, 3),
                     "row_chunks_per_s": round(wl.batch / (ms * 1e-3), 2)}
    out["warm_speedup"] = round(out["cold"]["ms_per_chunk"] / out["warm"]["ms_per_chunk"], 3)
    out["what"] = (f"{wl.batch} rows x {sum(wl.prefix) if wl.prefix else wl.ragged[1]} cached tokens, "
                   f"chunk of {n_tokens} action tokens x {a} values per row")
    ctx.close()
    return out


def decode_kernel_name(spec, B, A, persistent):
    if persistent:
        return (f"k_decode_fused<{spec.head_dim}> (persistent decode: head, feed and {A - 1} passes of every layer, "
                "+ the barrier-clearing kernel)")
    return (f"decode phase of a step: {A - 1} passes x {spec.n_layers} layers of k_gemm_wide<{(B + 15) // 16},2> "
            "(QKV, O, gate|up, down) + the O, gate|up and down split-K reductions + k_attn_decode (which adds the "
            f"QKV partial sums), and {A} bin heads")


def compact(r):
    """The figures of an extra workload."""
    out = {"value": round(r["value"], 2), "unit": "action-steps/s", "ms_per_step": round(r["ms_per_step"], 4),
           "batch": r["batch"], "steps": r["steps"], "mode": r["mode"], "step": r["step"]}
    if r.get("pages_in_use") is not None:
        out["pages_in_use"], out["pages_total"] = r["pages_in_use"], r["pages_total"]
    for k in ("decode", "extension", "build"):
        if r[k]:
            out[k] = {kk: r[k][kk] for kk in ("frac", "achieved", "unit", "avg_launch_us")}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="7b-b64-ragged")
    ap.add_argument("--mode", default="cached", choices=("cached", "recompute", "staggered"))
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true")
    ap.add_argument("--counters", action="store_true",
                    help="for counter runs: build, one append, the calibration copy, then --steps decode-only "
                         "steps; prints the per-step decode time")
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
    big = spec.matmul_params > 1e9
    torch.cuda.set_device(0)
    print(f"[bench] {wl.name}: weights", file=sys.stderr, flush=True)
    weights = W.make_device_weights(spec, args.seed) if big else W.make_weights(spec, args.seed)
    model = DeviceModel(weights, "cuda:0")
    B, A = wl.batch, wl.n_actions

    if args.counters:
        ctx = DeviceContext(model, B, wl.derived_capacity())
        epochs, pool, _ = make_inputs(model, wl, args.seed, 1, big)
        ctx.build(*epochs[0])
        if pool:
            ctx.append(pool[0], [wl.new_per_step] * B)
        tokens = torch.empty((B, A), dtype=torch.int32, device="cuda")
        torch.cuda.synchronize()
        copy_calibration()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            ctx.step(A, tokens=tokens, want_logits=False)
        e1.record()
        torch.cuda.synchronize()
        print(json.dumps({"workload": wl.name, "decode_steps": args.steps,
                          "avg_decode_us": round(e0.elapsed_time(e1) / args.steps * 1e3, 1),
                          "bytes_per_step": step_bytes(spec, ctx.lengths(), A)}), flush=True)
        ctx.close()
        model.close()
        return

    print(f"[bench] {wl.name}: warmup {args.warmup}, timed {args.steps} steps ({args.mode})", file=sys.stderr,
          flush=True)
    r = measure(model, wl, args.seed, args.steps, args.warmup, args.mode, big)
    print(f"[bench] {wl.name}: {r['value']:.1f} row-steps/s, {r['ms_per_step']:.3f} ms/step", file=sys.stderr,
          flush=True)
    extras = {}
    if not args.no_extras:
        plan = []
        if spec.name == "7b":
            plan = [("7b-b1", "cached", 20, False), ("7b-chunk56-b16", "cached", 8, False),
                    ("7b-chunk56-b16", "recompute", 8, False), ("7b-b64-ragged", "staggered", 20, False),
                    ("7b-b64-shared", "cached", 20, False), ("7b-b64-shared", "cached", 20, True)]
        for name, mode, n, share in plan:
            if name == wl.name and mode == args.mode:
                continue
            print(f"[bench] extra {name} ({mode}, {n} steps{', shared prefix pages' if share else ''})",
                  file=sys.stderr, flush=True)
            x = measure(model, W.WORKLOADS[name], args.seed, n, 2, mode, big, share=share)
            key = (f"{name}/{mode}" if mode != "cached" else name) + ("/shared-pages" if share else "")
            extras[key] = compact(x)
        if spec.name == "7b":
            print("[bench] host tier: 8 rows of 7b-b64-ragged to host memory and back", file=sys.stderr, flush=True)
            extras["host-tier/7b-b64-ragged"] = tier_rates(model, W.WORKLOADS["7b-b64-ragged"], args.seed)
            print("[bench] flow head: cold vs warm start on 7b-chunk56-b16 rows", file=sys.stderr, flush=True)
            extras["flow-head/7b-chunk56-b16"] = flow_rates(model, W.WORKLOADS["7b-chunk56-b16"], args.seed)
        if spec.name != "mid":
            model.close()
            print("[bench] extra mid-b8 (cached, 100 steps)", file=sys.stderr, flush=True)
            mw = DeviceModel(W.make_weights(W.MODELS["mid"], args.seed), "cuda:0")
            extras["mid-b8"] = compact(measure(mw, W.WORKLOADS["mid-b8"], args.seed, 100, 10, "cached", False))
            mw.close()
        c5, c5r = extras.get("7b-chunk56-b16"), extras.get("7b-chunk56-b16/recompute")
        if c5 and c5r:
            c5["speedup_vs_recompute"] = round(c5["value"] / c5r["value"], 3)
            c5["actions_per_s"] = round(c5["value"] * 8, 2)  # 56 tokens = 8 actions of 7 tokens
    copy_calibration()
    peaks = measured_peaks()
    hbm_meas = max(peaks["hbm_copy_GBps"], peaks["hbm_read_GBps"])

    dec = dict(r["decode"])
    kname = decode_kernel_name(spec, B, A, r["persistent_decode"])
    tr = profiled_traffic(wl.name, "decode-phase")
    roof = {"kernel": kname, **dec, "traffic": tr[0] if tr else None,
            "frac_vs_measured": round(dec["achieved"] / hbm_meas, 4)}
    if tr and tr[1]:  # HBM bytes over algorithmic bytes of the counted step (profiles/*_pmc.txt)
        roof["traffic_vs_algorithmic"] = round(tr[0] / tr[1], 3)
    if r["build"]:
        roof["rebuild"] = {"kernel": "ams_ctx_build: k_gemm_big GEMMs + k_attn_prefill_mfma + row kernels",
                           **r["build"], "frac_vs_measured": round(r["build"]["achieved"] / peaks["mfma_f16_TFLOPs"], 4)}
    if r["extension"]:
        roof["extension"] = {"kernel": "ams_ctx_append: k_gemm_big GEMMs (split-K O/down) + k_attn_extend + row kernels",
                             **r["extension"],
                             "frac_vs_measured": round(r["extension"]["achieved"] / peaks["mfma_f16_TFLOPs"], 4)}
    out = {
        "metric": "action steps/s per GPU (cached-context decode)",
        "value": round(r["value"], 2), "unit": "action-steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(r["ms_per_step"], 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "fp16",
        "data": "synthetic (seeded N(0,0.02) weights stored bf16, N(0,1) patch/observation embeddings, uniform ids)",
        "config": {"workload": wl.name, "n_layers": spec.n_layers, "d_model": spec.d_model,
                   "n_heads": spec.n_heads, "head_dim": spec.head_dim, "d_ffn": spec.d_ffn,
                   "vocab": spec.vocab, "n_bins": spec.n_bins, "batch": B,
                   "prefix_tokens": (f"U{{{wl.ragged[0]}..{wl.ragged[1]}}}" if wl.ragged else sum(wl.prefix)),
                   "n_actions": A, "capacity": r["capacity"], "new_tokens_per_step": wl.new_per_step,
                   "invalidate_every": wl.invalidate_every, "mode": args.mode,
                   "timed": f"1 build + {args.steps} steps" + (f" (rebuild every {wl.invalidate_every})"
                                                                if wl.invalidate_every else "")},
        "roofline": roof,
        "step": {**r["step"], "what": "whole timed window per step against the sum of the decode (HBM), extension "
                                      "and rebuild (MFMA) rooflines"},
        "measured_peaks": peaks,
    }
    if extras:
        out["extra_workloads"] = extras
    del model
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, weights, args.seed, wl.invalidate_every or args.steps)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
