#!/usr/bin/env python3
"""Benchmark of the LegoLink link step on one MI355X.

Default workload: the long-context link step -- 64 cached chunks x 2048 tokens
(131 072 linked tokens) + 256 suffix tokens, LegoLink-32 (the first 32 tokens
of chunks 1..63 and the suffix are recomputed: |S| = 2272 rows), GQA 32 query /
8 KV heads, head_dim 128, bf16 KV in 16-token paged blocks.  One step = one
call of epic_link_attention: build the private blocks (copy-on-write + write of
the recomputed K/V), scattered-query causal attention over the linked cache,
split-KV combine.  Inputs are resident in HBM before the timed region.

Prints ONE JSON line on stdout.  value = recomputed tokens / s (|S| / step
time); ms_per_step = link-step time (TTFT of this layer); roofline = the
attention kernel's algorithmic TFLOP/s (4 Hq D sum(p+1) per launch) against the
bf16 dense MFMA peak, timed with HIP events recorded around that kernel on its
stream inside the timed region; cpu_baseline = the float64 CPU oracle on a
sample of S rows, scaled by algorithmic flops.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "link-step TTFT (ms) + recomputed tokens/s; attention TFLOP/s vs MFMA peak"
PEAK_BF16_TFLOPS = 2500.0          # MI355X dense bf16 MFMA, published
PEAK_HBM_GBS = 8000.0
WORKLOADS = {
    "c5k32": ("c5", {"k": 32}),
    "c5k4": ("c5", {"k": 4}),
    "c5k0": ("c5", {"k": 0}),
    "c5all": ("c5", {"k": -1}),
    # the same long-context link step with cached K re-rotated to its linked positions
    "c5k32rr": ("c5", {"k": 32}),
    "c4": ("c4", {}),
    "c2": ("c2", {}),
    "c1": ("c1", {}),
    "c3": ("c3", {}),
    # compile step of the same 20 chunks with LegoLink-0's 4 dummy tokens, and the
    # link step (k = 0) over those caches
    "c3compile": ("c3", {}),
    "c3lego0": ("c3", {"k": 0}),
    # TTFT against context length at 512-token chunks: recompute-all (FR) vs LegoLink-16
    "sweep512": ("c3", {"chunk_len": 512, "k": 16}),
    # decode after the link step (one new token per request), not the default line
    "c5k32dec": ("c5", {"k": 32}),
    "c4dec": ("c4", {}),
}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def mfma_probe_tflops(iters: int = 200000, blocks: int = 512, reps: int = 3, varied: bool = False):
    """bf16 MFMA rate this chip sustains: a probe kernel whose wavefronts issue only
    independent 32x32x16 MFMAs (paper_2410_15332_amd/probe), best of `reps` launches.
    varied: operands with hashed signs and mantissas that change from one MFMA to the
    next (the datapath toggles as with real data) instead of one fixed operand pair."""
    import ctypes
    import torch

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2410_15332_amd", "probe", "libepic_probe.so"))
    fn = lib.epic_probe_mfma_bf16_varied if varied else lib.epic_probe_mfma_bf16
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
    lib.epic_probe_mfma_bf16_flops.restype = ctypes.c_double
    lib.epic_probe_mfma_bf16_flops.argtypes = [ctypes.c_int, ctypes.c_int]
    out = torch.empty(blocks * 512, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    best = 0.0
    for i in range(reps + 1):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        rc = fn(out.data_ptr(), blocks, iters, stream)
        b.record()
        torch.cuda.synchronize()
        if rc != 0:
            raise RuntimeError(f"MFMA probe launch failed: HIP error {rc}")
        if i > 0:                                   # the first launch warms the clock up
            best = max(best, lib.epic_probe_mfma_bf16_flops(blocks, iters) / (a.elapsed_time(b) * 1e-3) / 1e12)
    return best


def hbm_copy_probe_gbs(mib: int = 2048, reps: int = 5):
    """HBM rate of a plain device-to-device copy of `mib` MiB (torch's copy kernel),
    counting bytes read plus bytes written; best of `reps` after a warm-up."""
    import torch

    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    best = 0.0
    for i in range(reps + 1):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src)
        b.record()
        torch.cuda.synchronize()
        if i > 0:
            best = max(best, 2.0 * n * 4 / (a.elapsed_time(b) * 1e-3) / 1e9)
    del src, dst
    return best


def hbm_read_probe_gbs(mib: int = 2048, reps: int = 5, blocks: int = 4096):
    """HBM read rate of a streaming-read probe kernel (paper_2410_15332_amd/probe)
    over a `mib` MiB buffer read once per launch; best of `reps` after a warm-up."""
    import ctypes
    import torch

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2410_15332_amd", "probe", "libepic_probe.so"))
    fn = lib.epic_probe_hbm_read
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    nbytes = mib * (1 << 20)
    src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
    out = torch.empty(blocks, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    best = 0.0
    for i in range(reps + 1):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        rc = fn(src.data_ptr(), nbytes, out.data_ptr(), blocks, stream)
        b.record()
        torch.cuda.synchronize()
        if rc != 0:
            raise RuntimeError(f"HBM read probe launch failed: HIP error {rc}")
        if i > 0:
            best = max(best, nbytes / (a.elapsed_time(b) * 1e-3) / 1e9)
    del src, out
    return best


def graph_step_ms(run, reps: int):
    """Mean step time of `reps` back-to-back replays of the step captured in a HIP
    graph (the same kernels; the launch gaps between them are gone)."""
    import torch

    from paper_2410_15332_amd import harness

    g = harness.capture_graph(run)
    g.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    del g
    return ms


def ttft_medians(run, reps: int, evict_mib: int = 1024):
    """Median link-step time of `reps` single runs (HIP events around each): warm
    (back to back) and cold (each run after a write of evict_mib MiB on the same
    stream, more than L2 plus the 256 MB MALL, so caches and operands start in HBM).
    Taken after the timed region; the timed region itself is the K-step mean."""
    import numpy as np
    import torch

    evict = torch.empty(evict_mib * (1 << 20) // 4, dtype=torch.float32, device="cuda")
    out = {}
    for kind in ("warm", "cold"):
        times = []
        for _ in range(reps):
            if kind == "cold":
                evict.fill_(1.0)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            run()
            b.record()
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b))
        out[kind] = float(np.median(times))
    del evict
    return out


def code_without_comments(text: str) -> str:
    """C/C++ source with comments removed and whitespace runs collapsed (string
    literals are kept as they are; these sources put no comment markers in them)."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return re.sub(r"\s+", " ", text).strip()


ATTENTION_SOURCES = ("attention.hip", "device_common.h", "kernels.h", "plan.cpp", "plan_internal.h")
DECODE_SOURCES = ("decode_attention.hip", "decode_attention.h", "device_common.h", "kernels.h", "plan.cpp",
                  "plan_internal.h")


def kernel_source_hash(sources=None, files=ATTENTION_SOURCES) -> str:
    """Hash of what decides a kernel launch's memory traffic: the kernel sources and
    the planner that picks the kernel instance, tiles and split (code only, so an edit
    of comments keeps a profile valid).  sources: {file name: text} to hash instead of
    the files in the tree."""
    h = hashlib.sha256()
    for f in files:
        if sources is not None:
            text = sources[f]
        else:
            with open(os.path.join(ROOT, "paper_2410_15332_amd", "csrc", f)) as fh:
                text = fh.read()
        h.update(code_without_comments(text).encode())
    return h.hexdigest()[:16]


def traffic_from_profile(workload: str, kernel: str = "link_attention", files=ATTENTION_SOURCES):
    """HBM bytes per launch of `kernel` from a committed rocprofv3 --pmc summary, if it
    was taken on the current code; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    s = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    if not m or not s or s.group(1) != kernel_source_hash(files=files):
        return None
    return float(m.group(1))


def calibration_copy(mib: int):
    """A plain device-to-device copy of `mib` MiB before the timed region: the known
    bytes that scale the FETCH_SIZE / WRITE_SIZE counters of a --pmc run."""
    import torch

    if mib <= 0:
        return
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    log(f"calibration copy of {mib} MiB done")


def cpu_baseline(st, n_rows: int, seed: int = 1):
    """Time the float64 oracle on a seeded sample of S rows; scale to tokens/s by flops."""
    import numpy as np

    import oracle
    import synth
    from threadpoolctl import threadpool_info

    wl = st.wl
    r = 0
    lens = [wl.chunk_lens[c] for c in wl.requests[r]]
    a, b = int(st.views["s_off"][r]), int(st.views["s_off"][r + 1])
    s_pos = st.views["s_pos"][a:b].astype(np.int64)
    rows = np.sort(np.random.default_rng(seed).choice(len(s_pos), size=min(n_rows, len(s_pos)), replace=False))
    f = lambda x: synth.bf16_bits_to_f32(x).astype(np.float64)  # noqa: E731
    ck, cv = [], []
    for c in wl.requests[r]:
        kb, vb = synth.chunk_cache(wl.seed, c, wl.chunk_lens[c], wl.num_kv_heads, wl.head_dim, wl.value_scale,
                                   qk_scale=wl.qk_scale)
        ck.append(f(kb))
        cv.append(f(vb))
    q, k, v = (f(x) for x in synth.row_qkv(wl.seed, r, s_pos, wl.num_q_heads, wl.num_kv_heads, wl.head_dim,
                                            wl.value_scale, wl.qk_scale))
    t0 = time.perf_counter()
    oracle.link_attention(lens, wl.suffix_lens[r], wl.k, ck, cv, q, k, v, rows=rows)
    dt = time.perf_counter() - t0
    all_pos = st.views["s_pos"].astype(np.int64)
    f_total = float(np.sum(all_pos + 1))
    f_sample = float(np.sum(s_pos[rows] + 1))
    est_total_s = dt * f_total / f_sample
    cores = max([x.get("num_threads", 1) for x in threadpool_info() if x.get("user_api") == "blas"] or [1])
    return {
        "value": round(len(all_pos) / est_total_s, 3),
        "unit": "recomputed tokens/s",
        "cores": int(cores),
        "kind": "oracle",
        "sample": (f"{len(rows)} of {len(all_pos)} S rows of request 0 (seeded uniform), float64 NumPy oracle "
                   f"incl. K/V expansion, {dt:.1f} s; tokens/s scaled by algorithmic flops sum(p+1) "
                   f"({f_sample:.3e} of {f_total:.3e})"),
        "sample_seconds": round(dt, 2),
    }


def cpu_baseline_model(wl, n_rows: int):
    """Time one decoder layer of the float64 oracle on all S rows (layers run one after
    another, so the link step is n_layers times this); synthetic caches for that layer."""
    import numpy as np

    import oracle
    import synth
    from threadpoolctl import threadpool_info

    s_pos = oracle.legolink_positions(wl.chunk_lens, wl.suffix_len, wl.k)
    w = [synth.model_weights(wl.seed, 0, wl.hidden, wl.ffn, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, threads=8)]
    fn = synth.final_norm_weight(wl.seed, wl.hidden)
    f = lambda x: synth.bf16_bits_to_f32(x).astype(np.float64)  # noqa: E731
    ck, cv = [], []
    for j, L in enumerate(wl.chunk_lens):
        kb, vb = synth.chunk_cache(wl.seed, j, L, wl.num_kv_heads, wl.head_dim, 0.5, layer=0)
        ck.append(f(kb))
        cv.append(f(vb))
    emb = np.random.default_rng(0).standard_normal((len(s_pos), wl.hidden))
    t0 = time.perf_counter()
    oracle.link_model(emb, wl.chunk_lens, wl.suffix_len, wl.k, w, fn, [(ck, cv)], wl.hidden, wl.ffn,
                      wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.rope_theta, wl.rms_eps)
    dt = time.perf_counter() - t0
    cores = max([x.get("num_threads", 1) for x in threadpool_info() if x.get("user_api") == "blas"] or [1])
    return {
        "value": round(len(s_pos) / (dt * wl.n_layers), 4),
        "unit": "recomputed tokens/s",
        "cores": int(cores),
        "kind": "oracle",
        "sample": (f"1 of {wl.n_layers} decoder layers on all {len(s_pos)} S rows, float64 NumPy oracle, "
                   f"{dt:.1f} s; link-step time = {wl.n_layers} x that"),
        "sample_seconds": round(dt, 2),
    }


def cpu_baseline_compile(wl, n_dummy: int, budget_s: float = 10.0):
    """Time the float64 oracle's compile of one decoder layer, chunk after chunk
    (each after the dummy tokens) until about budget_s seconds have passed; the
    compile step is n_layers x that per compiled token."""
    import numpy as np

    import oracle
    import synth
    from threadpoolctl import threadpool_info

    w = [synth.model_weights(wl.seed, 0, wl.hidden, wl.ffn, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, threads=8)]
    fn = synth.final_norm_weight(wl.seed, wl.hidden)
    dummy = synth.dummy_embeddings(wl.seed, n_dummy, wl.hidden).astype(np.float64) if n_dummy else None
    dt, n_tok, n_chunks = 0.0, 0, 0
    for j, L in enumerate(wl.chunk_lens):
        emb = synth.token_embeddings(wl.seed, 0, j, range(L), wl.hidden).astype(np.float64)
        t0 = time.perf_counter()
        oracle.compile_chunk(emb, w, fn, wl.hidden, wl.ffn, wl.num_q_heads, wl.num_kv_heads, wl.head_dim,
                             wl.rope_theta, wl.rms_eps, dummy_emb=dummy)
        dt += time.perf_counter() - t0
        n_tok += L
        n_chunks += 1
        if dt >= budget_s:
            break
    cores = max([x.get("num_threads", 1) for x in threadpool_info() if x.get("user_api") == "blas"] or [1])
    return {
        "value": round(n_tok / (dt * wl.n_layers), 4),
        "unit": "compiled chunk tokens/s",
        "cores": int(cores),
        "kind": "oracle",
        "sample": (f"1 of {wl.n_layers} decoder layers of {n_chunks} chunks x ({n_dummy} dummy + "
                   f"{wl.chunk_lens[0]} tokens), float64 NumPy oracle, {dt:.1f} s; compile time = "
                   f"{wl.n_layers} layers x that per token"),
        "sample_seconds": round(dt, 2),
    }


def bench_compile(args, wl, n_dummy: int):
    """Compile step of the 32-layer configuration: all chunks prefilled alone (each
    after n_dummy dummy tokens, whose K/V are dropped), K/V stored per layer."""
    import numpy as np
    import torch

    from paper_2410_15332_amd import epic_link as el
    from paper_2410_15332_amd import harness

    t0 = time.time()
    st = harness.stage_model(wl, caches="compile", weights_on_device=True, n_dummy=n_dummy, keep_compile=True)
    cst = st.compile_stage
    torch.cuda.synchronize()
    log(f"staged {wl.name}: compile n_s={cst.sizes.n_s} ({len(wl.chunk_lens)} chunks x ({n_dummy} + "
        f"{wl.chunk_lens[0]})), {wl.n_layers} layers, in {time.time() - t0:.1f}s")
    for _ in range(args.warmup):
        cst.run(st.k_caches, st.v_caches)
    torch.cuda.synchronize()
    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    for e in (x for row in ev for x in row):
        e.record()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(K):
        el.epic_set_profile_events(ev[i])
        cst.run(st.k_caches, st.v_caches)
    end.record()
    el.epic_set_profile_events(None)
    torch.cuda.synchronize()
    step_ms = start.elapsed_time(end) / K
    attn_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    n_s = cst.sizes.n_s
    n_tok = sum(wl.chunk_lens)
    attn_flops = harness.attention_flops(cst.views, wl.num_q_heads, wl.head_dim)
    total = wl.n_layers * (attn_flops + harness.gemm_flops_per_layer(wl, n_s))
    achieved = total / (step_ms * 1e-3) / 1e12
    log(f"compile {step_ms:.3f} ms; layer attention {attn_ms:.4f} ms; all layers {achieved:.1f} TFLOP/s")
    result = {
        "metric": "compile step (ms) + compiled chunk tokens/s; whole-step TFLOP/s vs MFMA peak",
        "value": round(n_tok / (step_ms * 1e-3), 1), "unit": "compiled chunk tokens/s", "n_gpus": 1,
        "steps": K, "warmup": args.warmup, "ms_per_step": round(step_ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (random-init weights, seeded N(0,1) token embeddings, one seeded dummy token)",
        "config": {"workload": f"compile of {len(wl.chunk_lens)} x {wl.chunk_lens[0]} tokens + {n_dummy} dummy "
                               f"tokens per chunk, {wl.n_layers}-layer Llama-3-8B shape",
                   "layers": wl.n_layers, "hidden": wl.hidden, "ffn": wl.ffn, "num_q_heads": wl.num_q_heads,
                   "num_kv_heads": wl.num_kv_heads, "head_dim": wl.head_dim, "chunks": len(wl.chunk_lens),
                   "chunk_len": wl.chunk_lens[0], "dummy_tokens": n_dummy, "rows": n_s,
                   "parallelism": "single GPU"},
        "attention_tflops": round(attn_flops / attn_ms / 1e9, 2),
        "roofline": {"bound": "mfma", "kernel": "whole compile step (GEMMs + attention)",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "algorithmic_flops_per_launch": total,
                     "traffic": None},
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on one decoder layer of one chunk ...")
        result["cpu_baseline"] = cpu_baseline_compile(wl, n_dummy)
    print(json.dumps(result), flush=True)


def bench_sweep(args, wl, contexts=(2048, 4096, 8192, 16384, 32768, 65536)):
    """TTFT against context length with 512-token chunks and a 128-token suffix, on
    the 32-layer Llama-3-8B shape: FR prefills all N + 128 tokens (no chunk caches are
    compiled, as for FR in the paper's long-context experiment), LegoLink-16 links
    caches compiled beforehand by the library (untimed) and recomputes 16 tokens of
    every chunk but the first plus the suffix.  Weights are drawn once, reused."""
    import dataclasses

    import numpy as np
    import torch

    from paper_2410_15332_amd import harness

    weights = None
    points = []
    for n_ctx in contexts:
        m = n_ctx // wl.chunk_lens[0]
        row = {"context_tokens": n_ctx, "chunks": m}
        for method, k in (("legolink16", 16), ("fr", -1)):
            w2 = dataclasses.replace(wl, name=f"sweep_{method}_{n_ctx}", chunk_lens=[wl.chunk_lens[0]] * m, k=k)
            t0 = time.time()
            st = harness.stage_model(w2, caches="compile" if k >= 0 else "none", weights_on_device=True,
                                     weights=weights)
            weights = st.weights
            st.run()
            torch.cuda.synchronize()
            reps = max(1, min(args.steps, 10 if k >= 0 else 3))
            times = []
            for _ in range(reps):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                st.run()
                b.record()
                torch.cuda.synchronize()
                times.append(a.elapsed_time(b))
            ms = float(np.median(times))
            row[f"{method}_ms"] = round(ms, 3)
            row[f"{method}_rows"] = st.sizes.n_s
            log(f"N={n_ctx} {method}: {st.sizes.n_s} rows, TTFT {ms:.3f} ms (median of {reps}; staged in "
                f"{time.time() - t0:.1f}s)")
            del st
            torch.cuda.empty_cache()
        row["speedup"] = round(row["fr_ms"] / row["legolink16_ms"], 2)
        points.append(row)
    last = points[-1]
    result = {
        "metric": "TTFT (ms) against context length, 512-token chunks: FR vs LegoLink-16",
        "value": last["legolink16_ms"], "unit": "ms (LegoLink-16 TTFT at the longest context)", "n_gpus": 1,
        "steps": args.steps, "warmup": 1, "ms_per_step": last["legolink16_ms"], "higher_is_better": False,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (random-init weights, seeded N(0,1) token embeddings)",
        "config": {"workload": f"long-context sweep, {wl.n_layers}-layer Llama-3-8B shape, 512-token chunks, "
                               f"{wl.suffix_len}-token suffix", "parallelism": "single GPU"},
        "points": points,
    }
    print(json.dumps(result), flush=True)


def bench_model(args, wl, n_dummy: int = 0):
    """Full-model link step (all decoder layers + final norm) on the 32-layer configuration."""
    import numpy as np
    import torch

    from paper_2410_15332_amd import epic_link as el
    from paper_2410_15332_amd import harness

    t0 = time.time()
    st = harness.stage_model(wl, caches="compile", weights_on_device=True, n_dummy=n_dummy, tile_rows=args.tile_rows,
                             split_blocks=args.split_blocks)
    torch.cuda.synchronize()
    calibration_copy(args.calibrate_copy_mib)
    log(f"staged {wl.name}: n_s={st.sizes.n_s}, {wl.n_layers} layers, chunks compiled on the GPU "
        f"({n_dummy} dummy tokens) in {time.time() - t0:.1f}s")
    for _ in range(args.warmup):
        st.run()
    torch.cuda.synchronize()
    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    for e in (x for row in ev for x in row):
        e.record()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(K):
        el.epic_set_profile_events(ev[i])      # records the last layer's attention kernels
        st.run()
    end.record()
    el.epic_set_profile_events(None)
    torch.cuda.synchronize()
    step_ms = start.elapsed_time(end) / K
    attn_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    n_s = st.sizes.n_s
    attn_flops = harness.attention_flops(st.views, wl.num_q_heads, wl.head_dim)
    gemm_flops = harness.gemm_flops_per_layer(wl, n_s)
    total = wl.n_layers * (attn_flops + gemm_flops)
    achieved = total / (step_ms * 1e-3) / 1e12
    log(f"step {step_ms:.3f} ms; layer attention {attn_ms:.4f} ms ({attn_flops / attn_ms / 1e9:.1f} TFLOP/s); "
        f"all layers {achieved:.1f} TFLOP/s")
    med = {"warm": float("nan"), "cold": float("nan")} if args.no_ttft_medians else ttft_medians(st.run, max(K, 20))
    log(f"median of {max(K, 20)} single runs: warm {med['warm']:.3f} ms, cold {med['cold']:.3f} ms")
    gms = None if args.no_ttft_medians else graph_step_ms(st.run, K)
    if gms is not None:
        log(f"the step replayed from a HIP graph: {gms:.3f} ms")
    result = {
        "metric": METRIC, "value": round(n_s / (step_ms * 1e-3), 1), "unit": "recomputed tokens/s", "n_gpus": 1,
        "steps": K, "warmup": args.warmup, "ms_per_step": round(step_ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (random-init weights, seeded N(0,1) token embeddings, chunk caches compiled on the GPU)",
        "config": {"workload": wl.name, "layers": wl.n_layers, "hidden": wl.hidden, "ffn": wl.ffn,
                   "num_q_heads": wl.num_q_heads, "num_kv_heads": wl.num_kv_heads, "head_dim": wl.head_dim,
                   "chunks": len(wl.chunk_lens), "chunk_len": wl.chunk_lens[0], "suffix_len": wl.suffix_len,
                   "k": wl.k, "compile_dummy_tokens": n_dummy, "recomputed_rows": n_s,
                   "linked_tokens": int(st.sizes.max_pos),
                   "parallelism": "single GPU"},
        "ttft_ms": round(step_ms, 4),
        "ttft_warm_median_ms": None if args.no_ttft_medians else round(med["warm"], 4),
        "ttft_cold_median_ms": None if args.no_ttft_medians else round(med["cold"], 4),
        "ttft_graph_ms": None if gms is None else round(gms, 4),
        "attention_tflops": round(attn_flops / attn_ms / 1e9, 2),
        "model_tflops": round(achieved, 2),
        "roofline": {"bound": "mfma", "kernel": "whole link step (GEMMs + attention)", "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "algorithmic_flops_per_launch": total, "traffic": None},
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on one decoder layer ...")
        result["cpu_baseline"] = cpu_baseline_model(wl, args.cpu_rows)
    print(json.dumps(result), flush=True)


def cpu_baseline_decode(wl, st, ds, budget_s: float = 10.0):
    """Time the float64 oracle's decode step (oracle.decode_attention, one new token)
    request after request, cycling back to request 0, until about budget_s seconds
    have passed; tokens/s over the calls timed (each request costs the same at these
    shapes).  Inputs are generated outside the timed calls."""
    import numpy as np

    import oracle
    import synth
    from threadpoolctl import threadpool_info

    f = lambda x: synth.bf16_bits_to_f32(x).astype(np.float64)  # noqa: E731
    dt, n_req, prepared = 0.0, 0, None
    while dt < budget_s:
        r = n_req % wl.batch
        if prepared is None or prepared[0] != r:
            prepared = (r, _decode_inputs(wl, ds, r, f))
        args = prepared[1]
        t0 = time.perf_counter()
        oracle.decode_attention(*args)
        dt += time.perf_counter() - t0
        n_req += 1
    cores = max([x.get("num_threads", 1) for x in threadpool_info() if x.get("user_api") == "blas"] or [1])
    return {"value": round(n_req / dt, 4), "unit": "decoded tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{n_req} decode calls over {min(n_req, wl.batch)} of {wl.batch} requests, one new token "
                      f"each, float64 NumPy oracle incl. K/V expansion, {dt:.1f} s", "sample_seconds": round(dt, 2)}


def _decode_inputs(wl, ds, r, f):
    """oracle.decode_attention's arguments for request r of a one-token decode step."""
    import oracle
    import synth

    hq, hkv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    chunks = wl.requests[r]
    lens = [wl.chunk_lens[c] for c in chunks]
    ck, cv = [], []
    for c in chunks:
        kb, vb = synth.chunk_cache(wl.seed, c, wl.chunk_lens[c], hkv, d, wl.value_scale, qk_scale=wl.qk_scale)
        ck.append(f(kb))
        cv.append(f(vb))
    s_ref = oracle.legolink_positions(lens, wl.suffix_lens[r], wl.k)
    _, k, v = synth.row_qkv(wl.seed, r, s_ref, hq, hkv, d, wl.value_scale, wl.qk_scale)
    pos = ds.views["s_pos"][ds.views["s_off"][r]:ds.views["s_off"][r + 1]]
    qn, kn, vn = (f(x) for x in synth.row_qkv(wl.seed, r, pos, hq, hkv, d, wl.value_scale, wl.qk_scale))
    return (lens, wl.suffix_lens[r], wl.k, ck, cv, f(k), f(v), qn, kn, vn)


def bench_decode(args, wl):
    """Decode after the link step: one new token per request attends over its linked
    sequence (link step run once, untimed; the same decode step is then timed).  The
    attention kernel reads each request's K/V once: roofline against HBM, algorithmic
    bytes = sum over requests of (linked tokens + 1) x Hkv x D x 2 B x 2 (K and V)."""
    import numpy as np
    import torch

    from paper_2410_15332_amd import epic_link as el
    from paper_2410_15332_amd import harness

    st = harness.stage_attention(wl, device="cuda", spare_blocks=4 * wl.batch, split_blocks=args.split_blocks)
    st.run()
    ds = harness.stage_decode(wl, st.cfg, st.sizes, st.dplan.host, st.spare, st.num_blocks, [1] * wl.batch)
    torch.cuda.synchronize()
    calibration_copy(args.calibrate_copy_mib)
    for _ in range(args.warmup):
        ds.run(st.k_cache, st.v_cache)
    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    for e in (x for row in ev for x in row):
        e.record()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(K):
        el.epic_set_profile_events(ev[i])
        ds.run(st.k_cache, st.v_cache)
    end.record()
    el.epic_set_profile_events(None)
    torch.cuda.synchronize()
    step_ms = start.elapsed_time(end) / K
    attn_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    comb_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in ev]))
    linked = ds.views["s_pos"].astype(np.int64) + 1
    kv_bytes = float(linked.sum()) * wl.num_kv_heads * wl.head_dim * 2 * 2
    gbs = kv_bytes / (attn_ms * 1e-3) / 1e9
    log(f"decode step {step_ms:.4f} ms: attention {attn_ms:.4f} ms ({gbs:.0f} GB/s of K/V), combine {comb_ms:.4f}")
    result = {
        "metric": "decode step (ms) + tokens/s; attention K/V GB/s vs HBM peak", "value": round(wl.batch / (step_ms * 1e-3), 1),
        "unit": "decoded tokens/s", "n_gpus": 1, "steps": K, "warmup": args.warmup, "ms_per_step": round(step_ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 chunk caches and q/k/v)",
        "config": {"workload": wl.name + "_decode1", "batch": wl.batch, "k": wl.k, "num_q_heads": wl.num_q_heads,
                   "num_kv_heads": wl.num_kv_heads, "head_dim": wl.head_dim,
                   "linked_tokens_per_request": int(linked.max()), "parallelism": "single GPU"},
        "kernel_ms": {"attention": round(attn_ms, 5), "combine": round(comb_ms, 5)},
        "roofline": {"bound": "hbm",
                     "kernel": (f"link_decode_kernel<{wl.head_dim}>" if ds.sizes.tile_rows == 16
                                else f"link_attention_kernel<{wl.head_dim}, {ds.sizes.tile_rows // 32}>"),
                     "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "algorithmic_bytes_per_launch": kv_bytes,
                     "traffic": (traffic_from_profile(args.workload, "link_decode", DECODE_SOURCES)
                                 if ds.sizes.tile_rows == 16 else None)},
    }
    if not args.no_ttft_medians:
        gms = graph_step_ms(lambda: ds.run(st.k_cache, st.v_cache), K)
        log(f"the decode step replayed from a HIP graph: {gms:.4f} ms")
        result["step_graph_ms"] = round(gms, 5)
        read_gbs = hbm_read_probe_gbs()
        copy_gbs = hbm_copy_probe_gbs()
        log(f"HBM probes: a streaming read of 2 GiB moves {read_gbs:.0f} GB/s, a 2 GiB device-to-device copy "
            f"{copy_gbs:.0f} GB/s (read + write); decode attention at {gbs / read_gbs:.1%} of the read rate")
        result["roofline"]["peak_measured"] = round(read_gbs, 1)
        result["roofline"]["frac_of_measured_peak"] = round(gbs / read_gbs, 4)
        result["roofline"]["peak_measured_by"] = "streaming-read probe kernel over 2 GiB (16-byte loads, grid stride)"
        result["roofline"]["copy_measured"] = round(copy_gbs, 1)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle's decode step ...")
        result["cpu_baseline"] = cpu_baseline_decode(wl, st, ds)
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="c5k32", choices=sorted(WORKLOADS))
    ap.add_argument("--split-blocks", type=int, default=0, help="override the planner's split-KV size")
    ap.add_argument("--tile-rows", type=int, default=0, choices=(0, 128, 256),
                    help="override the planner's attention tile size (rows = S rows x query heads)")
    ap.add_argument("--cpu-rows", type=int, default=1024, help="S rows in the CPU-oracle sample (about 13 s on 16 cores)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ttft-medians", action="store_true",
                    help="skip the warm / cold single-run medians after the timed region (profiling runs, "
                         "so every launch of a kernel belongs to the warm-up or the timed steps)")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="before the timed region, run one device copy of this many MiB (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the link step is built and timed on a single MI355X, and "
              "sharding across GPUs is not built. Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2410_15332_amd import epic_link as el
    from paper_2410_15332_amd import harness
    from synth.configs import get_config

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    name, kw = WORKLOADS[args.workload]
    wl = get_config(name, **kw)
    if args.workload == "sweep512":
        bench_sweep(args, wl)
        return
    if args.workload == "c3compile":
        bench_compile(args, wl, 4)
        return
    if name == "c3":
        bench_model(args, wl, 4 if args.workload == "c3lego0" else 0)
        return
    if args.workload.endswith("dec"):
        bench_decode(args, wl)
        return
    t0 = time.time()
    rr_theta = 500000.0 if args.workload.endswith("rr") else 0.0
    st = harness.stage_attention(wl, device="cuda", split_blocks=args.split_blocks, rerotate_theta=rr_theta,
                                 tile_rows=args.tile_rows)
    torch.cuda.synchronize()
    log(f"staged {wl.name}: n_s={st.sizes.n_s} tiles={st.sizes.n_tiles} work={st.sizes.n_work} "
        f"partials={st.sizes.n_partials} private={st.sizes.n_private} re-rotated={st.sizes.n_rerotated} "
        f"in {time.time() - t0:.1f}s")
    flops = harness.attention_flops(st.views, wl.num_q_heads, wl.head_dim)

    calibration_copy(args.calibrate_copy_mib)

    for _ in range(args.warmup):
        st.run()
    torch.cuda.synchronize()

    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for e in (x for row in ev for x in row):   # torch creates the HIP event on its first record
        e.record()
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    start.record()
    for i in range(K):
        el.epic_set_profile_events(ev[i])
        st.run()
    end.record()
    el.epic_set_profile_events(None)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    step_ms = start.elapsed_time(end) / K
    attn_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    comb_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in ev]))
    write_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    n_s = st.sizes.n_s
    achieved = flops / (attn_ms * 1e-3) / 1e12
    log(f"step {step_ms:.4f} ms (wall {wall / K * 1e3:.4f} ms): write {write_ms:.4f} attn {attn_ms:.4f} "
        f"combine {comb_ms:.4f}; attention {achieved:.1f} TFLOP/s")
    med = {"warm": float("nan"), "cold": float("nan")} if args.no_ttft_medians else ttft_medians(st.run, max(K, 20))
    log(f"median of {max(K, 20)} single runs: warm {med['warm']:.4f} ms, cold {med['cold']:.4f} ms")
    gms = None if args.no_ttft_medians else graph_step_ms(st.run, K)
    if gms is not None:
        log(f"the step replayed from a HIP graph: {gms:.4f} ms")
    probe = None if args.no_ttft_medians else mfma_probe_tflops()
    probe_v = None if args.no_ttft_medians else mfma_probe_tflops(varied=True)
    if probe is not None:
        log(f"MFMA probe: {probe:.1f} TFLOP/s bf16 sustained with fixed operands, {probe_v:.1f} with operands "
            f"that change every MFMA; attention at {achieved / probe:.1%} / {achieved / probe_v:.1%} of them")

    traffic = traffic_from_profile(args.workload)
    result = {
        "metric": METRIC,
        "value": round(n_s / (step_ms * 1e-3), 1),
        "unit": "recomputed tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 chunk caches and recomputed q/k/v)",
        "config": {
            "workload": wl.name,
            "chunks": len(wl.requests[0]) if wl.batch == 1 else [len(r) for r in wl.requests][0],
            "batch": wl.batch,
            "chunk_len": wl.chunk_lens[0],
            "suffix_len": wl.suffix_lens[0],
            "k": wl.k,
            "num_q_heads": wl.num_q_heads,
            "num_kv_heads": wl.num_kv_heads,
            "head_dim": wl.head_dim,
            "block_size": 16,
            "recomputed_rows": n_s,
            "linked_tokens": int(st.sizes.max_pos),
            "rerotate_cached_k": bool(rr_theta),
            "parallelism": "single GPU",
        },
        "ttft_ms": round(step_ms, 5),
        "ttft_warm_median_ms": None if args.no_ttft_medians else round(med["warm"], 5),
        "ttft_cold_median_ms": None if args.no_ttft_medians else round(med["cold"], 5),
        "ttft_graph_ms": None if gms is None else round(gms, 5),
        "attention_tflops": round(achieved, 2),
        "attention_incl_combine_tflops": round(flops / ((attn_ms + comb_ms) * 1e-3) / 1e12, 2),
        "kernel_ms": {"link_write": round(write_ms, 5), "attention": round(attn_ms, 5),
                      "combine": round(comb_ms, 5)},
        "roofline": {
            "bound": "mfma",
            "kernel": f"link_attention_kernel<{wl.head_dim}, {st.sizes.tile_rows // 32}>",
            "achieved": round(achieved, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "algorithmic_flops_per_launch": flops,
            "traffic": traffic,
            "peak_measured": None if probe is None else round(probe, 1),
            "frac_of_measured_peak": None if probe is None else round(achieved / probe, 4),
            "peak_measured_by": "MFMA-only probe kernel (independent v_mfma_f32_32x32x16_bf16 chains on every SIMD)",
            "peak_measured_varied_operands": None if probe_v is None else round(probe_v, 1),
            "frac_of_measured_peak_varied_operands": None if probe_v is None else round(achieved / probe_v, 4),
        },
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample of S rows ...")
        result["cpu_baseline"] = cpu_baseline(st, args.cpu_rows)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
