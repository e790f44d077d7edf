"""Benchmark of the batched text-encoder prefill on one MI355X.

One step = one pass of the whole hot path over one batch: device-side
position build (mte_build_positions) + the 28-layer encoder forward
(mte_encode), inputs resident in HBM. Prints ONE JSON line.

Default workload: 16 frames x 96 tokens (8x8 merged image grid + 32
instruction tokens), 28 layers of the Qwen3-VL-2B-class decoder, bf16
weights, synthetic seeded weights and embeddings. The batch-1 frame
(96 tokens) is timed as well and reported in the same line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gate_up_gemm_b16_traffic.json")
STEP_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "te_prefill_28L_b1_L96_step_traffic.json")
KERNEL_SOURCES = ["paper_2606_05981_amd/csrc/gemm_kernel.h", "paper_2606_05981_amd/csrc/gemm.hip",
                  "paper_2606_05981_amd/csrc/common.h", "paper_2606_05981_amd/csrc/launch.h"]


def kernel_source_hash(files=None):
    import hashlib
    h = hashlib.sha256()
    for f in files or KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def all_kernel_sources():
    """Every source file of the library (a whole step's traffic depends on all of them)."""
    d = os.path.join(ROOT, "paper_2606_05981_amd", "csrc")
    return [os.path.join("paper_2606_05981_amd", "csrc", f) for f in sorted(os.listdir(d))]


def measured_step_traffic():
    """HBM-side bytes of one single-frame step (every kernel of positions + 28 layers +
    final norm) from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE passes, each divided by
    its copy-kernel calibration factor; None when missing or the sources changed since."""
    try:
        with open(STEP_TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_sha256") != kernel_source_hash(all_kernel_sources()):
        return None
    return t["hbm_bytes_per_step"]


def measured_traffic():
    """HBM-side bytes per gate/up GEMM launch from the committed rocprofv3 counter
    summary (FETCH_SIZE and WRITE_SIZE, each divided by its copy-kernel calibration
    factor); None when the summary is missing or the kernel sources changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return (t["fetch_kib_per_launch"] / t["fetch_factor"] +
            t["write_kib_per_launch"] / t["write_factor"]) * 1024.0


def gemm_flops(dims, T):
    """Algorithmic flops of the four projection GEMMs for T tokens, per layer."""
    D, F, d = dims.hidden, dims.ffn, dims.head_dim
    nqkv = (dims.n_q_heads + 2 * dims.n_kv_heads) * d
    return {"qkv": 2 * T * nqkv * D, "o": 2 * T * D * dims.n_q_heads * d,
            "gate_up": 2 * T * 2 * F * D, "down": 2 * T * D * F}


KERNEL_CLASSES = {0: "qkv_gemm", 1: "attention", 2: "o_gemm", 3: "gate_up_gemm", 4: "down_gemm"}


def kernel_work(dims, lens):
    """Algorithmic flops and bytes of one launch of each timed kernel class at these
    sequence lengths (one layer): the projections read their fp16 weights and fp16 input
    once and write their output (QKV: fp16 attention operands; SwiGLU fp16; the residual
    projections read and write the fp32 residual stream); attention reads fp16 q/k/v and
    writes fp16 o.
    With a K split the timed launch is the split GEMM alone (its partial sums are added
    by the next kernel); its bytes are still counted as the finished product's."""
    T = sum(lens)
    D, F, d, hq, hkv = dims.hidden, dims.ffn, dims.head_dim, dims.n_q_heads, dims.n_kv_heads
    nqkv = (hq + 2 * hkv) * d
    g = gemm_flops(dims, T)
    att = sum(4 * hq * d * L * (L + 1) // 2 for L in lens)
    return {
        0: (g["qkv"], 2 * nqkv * D + 2 * T * D + 2 * T * nqkv),
        1: (att, 2 * T * nqkv + 2 * T * hq * d),
        2: (g["o"], 2 * D * hq * d + 2 * T * hq * d + 8 * T * D),
        3: (g["gate_up"], 2 * 2 * F * D + 2 * T * D + 2 * T * F),
        4: (g["down"], 2 * D * F + 2 * T * F + 8 * T * D),
    }


def kernel_table(dims, lens, kern):
    """Per-kernel average launch time (HIP events on the launch stream) and its rates
    against both published peaks."""
    work = kernel_work(dims, lens)
    out = {}
    for cls, (n, ms) in kern.items():
        us = ms * 1e3 / max(n, 1)
        fl, by = work[cls]
        out[KERNEL_CLASSES[cls]] = {
            "avg_launch_us": round(us, 2), "launches": n,
            "tflops": round(fl / (us * 1e-6) / 1e12, 1),
            "frac_bf16_peak": round(fl / (us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "gbs": round(by / (us * 1e-6) / 1e9, 1),
            "frac_hbm_peak": round(by / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
            "flops_per_launch": fl, "algorithmic_bytes_per_launch": by}
    return out


def step_flops(dims, lens):
    g = sum(gemm_flops(dims, sum(lens)).values())
    att = sum(4 * dims.n_q_heads * dims.head_dim * L * (L + 1) // 2 for L in lens)
    return dims.n_layers * (g + att)


def run_workload(torch, name, steps, warmup, timing_classes=(), use_graph=True, weight_format=0):
    from paper_2606_05981_amd import binding as B
    from paper_2606_05981_amd.encoder import TextEncoder, build_positions
    from synth import workloads as W

    wl = W.workload(name)
    dims = wl.dims
    lens = W.seq_lens(wl.layouts)
    T = sum(lens)
    cfg = B.make_config(dims.n_layers, dims.hidden, dims.n_q_heads, dims.n_kv_heads,
                        dims.head_dim, dims.ffn, rms_eps=dims.rms_eps, rope_theta=dims.rope_theta,
                        mrope_section=dims.mrope_section, mrope_layout=dims.mrope_layout,
                        qk_norm=dims.qk_norm, dtype=B.MTE_BF16, out_dtype=B.MTE_F32, max_tokens=T,
                        max_batch=len(lens), max_seq=max(lens), weight_format=weight_format)
    enc = TextEncoder.from_host(cfg, (W.layer_weights(dims, l) for l in range(dims.n_layers)),
                                W.final_norm_gain(dims))
    emb = torch.from_numpy(W.embeddings(dims, wl.layouts)).to("cuda", torch.bfloat16)
    layouts = [(s.n_text_before, s.grid_t, s.grid_h, s.grid_w, s.n_text_after) for s in wl.layouts]
    out = torch.empty((T, dims.hidden), dtype=torch.float32, device="cuda")
    pos = torch.empty((3, T), dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    def step():
        B.mte_build_positions(layouts, pos.data_ptr(), stream.cuda_stream)
        B.mte_encode(enc.handle, emb.data_ptr(), pos.data_ptr(), lens, len(lens), out.data_ptr(),
                     stream.cuda_stream)

    # The whole step is captured once into a HIP graph (mte_encode and
    # mte_build_positions only enqueue work) and replayed: one launch per step.
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    graph = None
    if use_graph:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            stream = side
            with torch.cuda.graph(graph, stream=side):
                step()
        torch.cuda.current_stream().wait_stream(side)
        stream = torch.cuda.current_stream()
        for _ in range(warmup):
            graph.replay()
        torch.cuda.synchronize()
    run_step = graph.replay if graph is not None else step
    # Eager passes over the same steps, one per timed kernel class: the library
    # records HIP events around every launch of that class on the launch stream.
    kern = {}
    torch.cuda.synchronize()
    te = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    eager_s = time.perf_counter() - te
    for cls in timing_classes:
        B.mte_timing_enable(enc.handle, cls, steps * dims.n_layers)
        for _ in range(steps):
            step()
        kern[cls] = B.mte_timing_read(enc.handle)
        B.mte_timing_disable(enc.handle)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        run_step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = wall * 1e3
    # per-step spread: HIP events around each of `steps` further replays
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for e0, e1 in evs:
        e0.record()
        run_step()
        e1.record()
    torch.cuda.synchronize()
    per = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    mean = sum(per) / len(per)
    sd = (sum((x - mean) ** 2 for x in per) / max(len(per) - 1, 1)) ** 0.5
    stats = {"median_ms": round(per[len(per) // 2], 4), "mean_ms": round(mean, 4), "sd_ms": round(sd, 4),
             "steps": len(per)}
    enc.close()
    return dict(name=name, dims=dims, lens=lens, T=T, wall_s=wall, gpu_ms=gpu_ms, kern=kern,
                eager_s=eager_s, graph=graph is not None, stats=stats)


def cpu_baseline():
    """The fp64 oracle on the host cores, once over each of the small and medium
    workloads: the tiny fp32 decoder (32 tokens), one full-width layer (96 tokens)
    and the 28-layer stack at one frame (96 tokens), 8 frames and 16 frames (packed
    batches of 96-token frames). `value` is the 16-frame rate, the benchmark's
    own workload; about 15 s of host time in all."""
    from oracle import te_oracle as O
    from synth import workloads as W
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1

    def rate(name, min_s):
        wl = W.workload(name)
        dims = wl.dims
        lens = W.seq_lens(wl.layouts)
        emb = W.embeddings(dims, wl.layouts)
        pos = O.positions(wl.layouts)
        ws = [W.layer_weights(dims, l) for l in range(dims.n_layers)]
        fin = W.final_norm_gain(dims)
        runs, t0 = 0, time.perf_counter()
        while True:
            O.encode(emb, pos, lens, dims, lambda l: ws[l], fin)
            runs += 1
            dt = time.perf_counter() - t0
            if dt >= min_s:
                break
        T = sum(lens)
        return {"workload": name, "layers": dims.n_layers, "tokens": T, "runs": runs,
                "seconds": round(dt, 2), "tokens_per_s": round(T * runs / dt, 2),
                "frames_per_s": round(len(lens) * runs / dt, 3)}

    cfgs = {"tiny_fp32": rate("tiny_fp32", 1.0), "layer1_b1": rate("layer1_b1", 2.0),
            "stack_b1": rate("stack_b1", 0.0), "stack_b8": rate("stack_b8", 0.0),
            "stack_b16": rate("stack_b16", 0.0)}
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            cpu = next(l.split(":", 1)[1].strip() for l in f if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    main = cfgs["stack_b16"]
    return {"value": main["tokens_per_s"], "unit": "tokens/s", "cores": int(cores),
            "kind": "oracle", "cpu_model": cpu, "host_cpus": os.cpu_count(),
            "sample": f"the 16 x 96-token batch as one packed batch, one whole 28-layer forward "
                      f"({main['tokens']} tokens in {main['seconds']} s, fp64 numpy oracle); the other "
                      "configurations' rates in 'configs'",
            "configs": cfgs}


def run_overlap(torch, name, steps, warmup):
    """Side-stream overlap (the paper's pipelining, Alg. 1: the text encoder on a side stream
    beside the main-stream denoiser): the captured encoder step replays on a side stream while
    the main stream runs a dense fp16 GEMM load standing in for the U-Net, joined by events.
    Returns solo and concurrent wall times and the overlap efficiency
    (solo_te + solo_load - concurrent) / min(solo_te, solo_load)."""
    from paper_2606_05981_amd import binding as B
    from paper_2606_05981_amd.encoder import TextEncoder
    from synth import workloads as W

    wl = W.workload(name)
    dims = wl.dims
    lens = W.seq_lens(wl.layouts)
    T = sum(lens)
    cfg = B.make_config(dims.n_layers, dims.hidden, dims.n_q_heads, dims.n_kv_heads,
                        dims.head_dim, dims.ffn, rms_eps=dims.rms_eps, rope_theta=dims.rope_theta,
                        mrope_section=dims.mrope_section, mrope_layout=dims.mrope_layout,
                        qk_norm=dims.qk_norm, dtype=B.MTE_BF16, out_dtype=B.MTE_F32, max_tokens=T,
                        max_batch=len(lens), max_seq=max(lens))
    enc = TextEncoder.from_host(cfg, (W.layer_weights(dims, l) for l in range(dims.n_layers)),
                                W.final_norm_gain(dims))
    emb = torch.from_numpy(W.embeddings(dims, wl.layouts)).to("cuda", torch.bfloat16)
    layouts = [(s.n_text_before, s.grid_t, s.grid_h, s.grid_w, s.n_text_after) for s in wl.layouts]
    out = torch.empty((T, dims.hidden), dtype=torch.float32, device="cuda")
    pos = torch.empty((3, T), dtype=torch.int32, device="cuda")
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()

    def enc_step(st):
        B.mte_build_positions(layouts, pos.data_ptr(), st.cuda_stream)
        B.mte_encode(enc.handle, emb.data_ptr(), pos.data_ptr(), lens, len(lens), out.data_ptr(),
                     st.cuda_stream)

    side.wait_stream(main)
    with torch.cuda.stream(side):
        for _ in range(warmup):
            enc_step(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            enc_step(side)
    main.wait_stream(side)
    torch.cuda.synchronize()
    a = torch.randn(4096, 4096, device="cuda", dtype=torch.float16)
    b = torch.randn(4096, 4096, device="cuda", dtype=torch.float16)
    c = torch.empty_like(a)

    def timed(fn):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        fn()
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    def te_only():
        with torch.cuda.stream(side):
            for _ in range(steps):
                graph.replay()

    for _ in range(warmup):
        torch.mm(a, b, out=c)
    te_s = timed(te_only)
    t_mm = timed(lambda: [torch.mm(a, b, out=c) for _ in range(20)]) / 20
    n_mm = max(1, int(round(te_s / t_mm)))     # a main-stream load as long as the encoder work

    def load_only():
        for _ in range(n_mm):
            torch.mm(a, b, out=c)

    load_s = timed(load_only)

    def both():
        side.wait_stream(main)
        te_only()
        load_only()
        main.wait_stream(side)

    both_s = timed(both)
    enc.close()
    eff = (te_s + load_s - both_s) / min(te_s, load_s)
    return {"workload": f"{name}: encoder graph x{steps} on a side stream", "main_load":
            f"{n_mm} x fp16 GEMM 4096^3 on the main stream",
            "te_ms": round(te_s * 1e3, 3), "load_ms": round(load_s * 1e3, 3),
            "concurrent_ms": round(both_s * 1e3, 3), "overlap_efficiency": round(eff, 3),
            "te_ms_per_step_alone": round(te_s * 1e3 / steps, 4)}


def run_regimes(torch, steps, warmup, names=("stack_b8", "stack_b32_l320", "stack_mixed32")):
    """The other measured regimes of the same 28-layer encoder: 8 frames of 96 tokens,
    32 sequences of 320 tokens, and 32 sequences of mixed lengths (96..320). One encoder
    sized for the largest serves all three; each step is captured as a HIP graph and
    replayed, timed with HIP events (median, and the model's TFLOP/s against the
    published bf16 peak)."""
    from paper_2606_05981_amd import binding as B
    from paper_2606_05981_amd.encoder import TextEncoder
    from synth import workloads as W
    wls = [W.workload(n) for n in names]
    dims = wls[0].dims
    lens_all = [W.seq_lens(w.layouts) for w in wls]
    cfg = B.make_config(dims.n_layers, dims.hidden, dims.n_q_heads, dims.n_kv_heads,
                        dims.head_dim, dims.ffn, rms_eps=dims.rms_eps, rope_theta=dims.rope_theta,
                        mrope_section=dims.mrope_section, mrope_layout=dims.mrope_layout,
                        qk_norm=dims.qk_norm, dtype=B.MTE_BF16, out_dtype=B.MTE_F32,
                        max_tokens=max(sum(l) for l in lens_all),
                        max_batch=max(len(l) for l in lens_all), max_seq=max(max(l) for l in lens_all))
    enc = TextEncoder.from_host(cfg, (W.layer_weights(dims, l) for l in range(dims.n_layers)),
                                W.final_norm_gain(dims))
    out = {}
    for wl, lens in zip(wls, lens_all):
        T = sum(lens)
        emb = torch.from_numpy(W.embeddings(dims, wl.layouts)).to("cuda", torch.bfloat16)
        layouts = [(q.n_text_before, q.grid_t, q.grid_h, q.grid_w, q.n_text_after) for q in wl.layouts]
        o = torch.empty((T, dims.hidden), dtype=torch.float32, device="cuda")
        pos = torch.empty((3, T), dtype=torch.int32, device="cuda")
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())

        def step(st):
            B.mte_build_positions(layouts, pos.data_ptr(), st.cuda_stream)
            B.mte_encode(enc.handle, emb.data_ptr(), pos.data_ptr(), lens, len(lens), o.data_ptr(), st.cuda_stream)

        with torch.cuda.stream(side):
            for _ in range(warmup):
                step(side)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=side):
                step(side)
        torch.cuda.current_stream().wait_stream(side)
        for _ in range(warmup):
            graph.replay()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        for e0, e1 in evs:
            e0.record()
            graph.replay()
            e1.record()
        torch.cuda.synchronize()
        per = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
        ms = per[len(per) // 2]
        tflops = step_flops(dims, lens) / (ms * 1e-3) / 1e12
        out[wl.name] = {"sequences": len(lens), "tokens_per_step": T, "min_len": min(lens), "max_len": max(lens),
                        "ms_per_step_median": round(ms, 4), "tokens_per_s": round(T / ms * 1e3, 1),
                        "frames_per_s": round(len(lens) / ms * 1e3, 1), "model_tflops": round(tflops, 1),
                        "frac_of_bf16_peak": round(tflops / PEAK_BF16_TFLOPS, 4), "steps": len(per)}
        del graph
    enc.close()
    return out


def run_prefix(torch, prefix, steps, warmup, frames=16):
    """Shared prefix (the paper's system prompt, Sec. V): `frames` frames whose sequences all
    start with the same `prefix` text tokens, then an 8x8 image grid and 32 instruction tokens.
    Times the whole sequences through mte_encode against mte_encode_prefixed (the prefix once,
    then each frame's own 96 tokens attending to its cached keys / values); both captured as
    HIP graphs and replayed."""
    import numpy as np
    from paper_2606_05981_amd import binding as B
    from paper_2606_05981_amd.encoder import TextEncoder, build_positions
    from synth import workloads as W

    dims = W.DIMS_FULL
    full = tuple(W.SeqLayout(prefix, 1, 8, 8, 32) for _ in range(frames))
    L = full[0].length
    T = L * frames
    cfg = B.make_config(dims.n_layers, dims.hidden, dims.n_q_heads, dims.n_kv_heads,
                        dims.head_dim, dims.ffn, rms_eps=dims.rms_eps, rope_theta=dims.rope_theta,
                        mrope_section=dims.mrope_section, mrope_layout=dims.mrope_layout,
                        qk_norm=dims.qk_norm, dtype=B.MTE_BF16, out_dtype=B.MTE_F32, max_tokens=T,
                        max_batch=frames, max_seq=L)
    enc = TextEncoder.from_host(cfg, (W.layer_weights(dims, l) for l in range(dims.n_layers)),
                                W.final_norm_gain(dims))
    enc.reserve_prefix(prefix)
    emb_np = W.embeddings(dims, full)
    own = np.concatenate([np.arange(f * L + prefix, (f + 1) * L) for f in range(frames)])
    dev = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to("cuda", dt)
    emb = dev(emb_np, torch.bfloat16)
    # positions of the full sequences, built on the device (mte_build_positions)
    pos = build_positions([(q.n_text_before, q.grid_t, q.grid_h, q.grid_w, q.n_text_after) for q in full])
    own_g = torch.from_numpy(own).cuda()
    p_emb, p_pos = dev(emb_np[:prefix], torch.bfloat16), pos[:, :prefix].contiguous()
    o_emb, o_pos = dev(emb_np[own], torch.bfloat16), pos[:, own_g].contiguous()
    out = torch.empty((T, dims.hidden), dtype=torch.float32, device="cuda")
    out_p = torch.empty((prefix, dims.hidden), dtype=torch.float32, device="cuda")
    out_o = torch.empty((len(own), dims.hidden), dtype=torch.float32, device="cuda")
    side = torch.cuda.Stream()

    def full_step(st):
        B.mte_encode(enc.handle, emb.data_ptr(), pos.data_ptr(), [L] * frames, frames,
                     out.data_ptr(), st.cuda_stream)

    def prefixed_step(st):
        B.mte_encode_prefixed(enc.handle, p_emb.data_ptr(), p_pos.data_ptr(), prefix,
                              o_emb.data_ptr(), o_pos.data_ptr(), [L - prefix] * frames, frames,
                              out_p.data_ptr(), out_o.data_ptr(), st.cuda_stream)

    res = {}
    for name, fn in (("full_sequences", full_step), ("prefix_once", prefixed_step)):
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for _ in range(warmup):
                fn(side)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                fn(side)
        torch.cuda.current_stream().wait_stream(side)
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            g.replay()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / steps
        res[name] = {"ms_per_step": round(dt * 1e3, 4), "frames_per_s": round(frames / dt, 1)}
    dev_err = float((out[own_g] - out_o).abs().max() / out.pow(2).mean().sqrt())
    enc.close()
    res.update({"workload": f"{frames} frames x ({prefix} shared prefix + 8x8 image + 32 instruction) "
                            "tokens, 28 layers",
                "speedup": round(res["full_sequences"]["ms_per_step"] / res["prefix_once"]["ms_per_step"], 3),
                "max_abs_diff_vs_full_over_rms": dev_err})
    return res


def e4m3_weight_bytes(dims):
    """Bytes the encoder reads per forward with e4m3 weights: one byte per linear
    weight, a float scale per weight row, fp32 norm gains."""
    D, F, d = dims.hidden, dims.ffn, dims.head_dim
    nqkv = (dims.n_q_heads + 2 * dims.n_kv_heads) * d
    rows = nqkv + D + 2 * F + D
    gains = 2 * D + (2 * d if dims.qk_norm else 0)
    return dims.n_layers * (dims.params_per_layer + 4 * rows + 4 * gains)


def run_e4m3(torch, name, steps, warmup, dims, batch1=True):
    """The same steps with MTE_WEIGHTS_E4M3 encoders (weights quantised at creation)."""
    out = {"format": "OCP e4m3 codes, power-of-two scale per weight row; fp16 activations, "
                     "fp16 MFMA after exact widening, fp32 accumulate"}
    m = run_workload(torch, name, steps, warmup, weight_format=1)
    out["main"] = {"workload": name, "ms_per_step": round(m["wall_s"] * 1e3 / steps, 4),
                   "tokens_per_s": round(m["T"] * steps / m["wall_s"], 1)}
    if batch1:
        b1 = run_workload(torch, "stack_b1", steps, warmup, weight_format=1)
        t1 = b1["wall_s"] / steps
        wbytes = e4m3_weight_bytes(dims) + 2 * b1["T"] * dims.hidden * 2
        out["batch1"] = {"workload": "stack_b1: 1 frame x 96 tokens, 28 layers",
                         "ms_per_step": round(t1 * 1e3, 4), "tokens_per_s": round(b1["T"] / t1, 1),
                         "hbm_roofline": {"bound": "hbm", "achieved": round(wbytes / t1 / 1e9, 1),
                                          "peak": PEAK_HBM_GBS, "unit": "GB/s",
                                          "frac": round(wbytes / t1 / 1e9 / PEAK_HBM_GBS, 4),
                                          "bytes_per_step": wbytes}}
    return out


def vision_flops(v, n, h, w):
    """Algorithmic flops of one vision-tower pass over n images of h x w."""
    per = (h // v.patch) * (w // v.patch)
    T, D, F = n * per, v.hidden, v.ffn
    mm = v.merge * v.merge
    kp = v.in_channels * v.patch * v.patch
    blocks = v.depth * (2 * T * (4 * D * D + 2 * F * D) + n * 4 * per * per * D)
    merger = 2 * (T // mm) * (mm * D * mm * D + v.out_hidden * mm * D)
    return 2 * T * D * kp + blocks + merger


def run_vision(torch, steps, warmup, n=16, side=256):
    """The vision tower on n images of side x side: 24 pre-norm ViT blocks of width 1024
    and the 2x2 merger, captured once into a HIP graph and replayed."""
    from paper_2606_05981_amd import binding as B
    from paper_2606_05981_amd.encoder import VisionEncoder
    from synth import vision as SV
    v = SV.VDIMS_FULL
    cfg = B.make_vision_config(v.depth, v.hidden, v.n_heads, v.head_dim, v.ffn, patch=v.patch, merge=v.merge,
                               in_channels=v.in_channels, out_hidden=v.out_hidden, ln_eps=v.ln_eps,
                               rope_theta=v.rope_theta, dtype=B.MTE_BF16, out_dtype=B.MTE_BF16,
                               max_images=n, max_side=side)
    enc = VisionEncoder.from_host(cfg, SV.outer_weights(v), (SV.block_weights(v, l) for l in range(v.depth)))
    px = torch.from_numpy(SV.images(v, n, side, side)).to("cuda", torch.bfloat16)
    out = torch.empty((n * v.tokens_per_image(side, side), v.out_hidden), dtype=torch.bfloat16, device="cuda")
    for _ in range(warmup):
        enc.encode(px, out)
    torch.cuda.synchronize()
    side_s = torch.cuda.Stream()
    side_s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side_s):
        with torch.cuda.graph(graph, stream=side_s):
            enc.encode(px, out, stream=side_s)
    torch.cuda.current_stream().wait_stream(side_s)
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        graph.replay()
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    enc.close()
    fl = vision_flops(v, n, side, side)
    return {"workload": f"{n} images of {side}x{side}, 24 ViT blocks (width 1024, 16 heads of 64, MLP 4096) "
                        "+ 2x2 merger to 2048",
            "ms_per_step": round(dt * 1e3, 4), "images_per_s": round(n / dt, 1),
            "image_tokens_per_s": round(n * v.tokens_per_image(side, side) / dt, 1),
            "model_tflops": round(fl / dt / 1e12, 1), "frac_of_bf16_peak": round(fl / dt / 1e12 / PEAK_BF16_TFLOPS, 4),
            "flops_per_step": fl}


def run_pipeline(torch, steps, warmup, n=16, side=256):
    """Source frames to conditioning hidden states: n 256x256 frames through the vision
    tower, whose image tokens land (strided) in the packed decoder input next to each
    frame's 32 instruction embeddings, then positions and the 28-layer decoder; one
    captured graph per step."""
    from paper_2606_05981_amd import binding as B
    from paper_2606_05981_amd.encoder import TextEncoder, VisionEncoder
    from synth import vision as SV
    from synth import workloads as W
    v = SV.VDIMS_FULL
    wl = W.workload("stack_b16")
    dims = wl.dims
    lens = W.seq_lens(wl.layouts)
    L, T = lens[0], sum(lens)
    tpi = v.tokens_per_image(side, side)
    assert len(lens) == n and all(x == L for x in lens) and all(s.n_text_before == 0 and s.n_image == tpi
                                                                 for s in wl.layouts)
    vcfg = B.make_vision_config(v.depth, v.hidden, v.n_heads, v.head_dim, v.ffn, patch=v.patch, merge=v.merge,
                                in_channels=v.in_channels, out_hidden=dims.hidden, ln_eps=v.ln_eps,
                                rope_theta=v.rope_theta, dtype=B.MTE_BF16, out_dtype=B.MTE_BF16,
                                max_images=n, max_side=side)
    venc = VisionEncoder.from_host(vcfg, SV.outer_weights(v.with_(out_hidden=dims.hidden)),
                                   (SV.block_weights(v, l) for l in range(v.depth)))
    cfg = B.make_config(dims.n_layers, dims.hidden, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.ffn,
                        rms_eps=dims.rms_eps, rope_theta=dims.rope_theta, mrope_section=dims.mrope_section,
                        mrope_layout=dims.mrope_layout, qk_norm=dims.qk_norm, dtype=B.MTE_BF16,
                        out_dtype=B.MTE_F32, max_tokens=T, max_batch=n, max_seq=L)
    tenc = TextEncoder.from_host(cfg, (W.layer_weights(dims, l) for l in range(dims.n_layers)),
                                 W.final_norm_gain(dims))
    px = torch.from_numpy(SV.images(v, n, side, side)).to("cuda", torch.bfloat16)
    # the packed decoder input: the instruction rows are filled once; the image rows by every step
    emb = torch.from_numpy(W.embeddings(dims, wl.layouts)).to("cuda", torch.bfloat16)
    out = torch.empty((T, dims.hidden), dtype=torch.float32, device="cuda")
    pos = torch.empty((3, T), dtype=torch.int32, device="cuda")
    layouts = [(s.n_text_before, s.grid_t, s.grid_h, s.grid_w, s.n_text_after) for s in wl.layouts]

    def step(st):
        venc.encode(px, out=emb, image_stride=L, stream=st)
        B.mte_build_positions(layouts, pos.data_ptr(), st.cuda_stream)
        B.mte_encode(tenc.handle, emb.data_ptr(), pos.data_ptr(), lens, n, out.data_ptr(), st.cuda_stream)

    cur = torch.cuda.current_stream()
    for _ in range(warmup):
        step(cur)
    torch.cuda.synchronize()
    side_s = torch.cuda.Stream()
    side_s.wait_stream(cur)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(side_s):
        with torch.cuda.graph(graph, stream=side_s):
            step(side_s)
    cur.wait_stream(side_s)
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        graph.replay()
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    venc.close()
    tenc.close()
    return {"workload": f"{n} frames: {side}x{side} source through the vision tower ({tpi} image tokens each, "
                        f"written into the packed decoder input) + {L - tpi} instruction tokens, 28-layer decoder",
            "ms_per_step": round(dt * 1e3, 4), "frames_per_s": round(n / dt, 1),
            "ms_per_frame": round(dt * 1e3 / n, 4)}


def copy_bandwidth(torch, mib=1024, reps=10):
    """Achieved HBM bandwidth of a plain device copy (read + write bytes / time): the
    measured counterpart of the published 8 TB/s, for context."""
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    dt = e0.elapsed_time(e1) / 1e3 / reps
    del src, dst
    return round(2 * mib * (1 << 20) / dt / 1e9, 1)


def _probe_lib():
    """The measurement-only probe library (paper_2606_05981_amd/libmte_probe.so), built next
    to libmte by the package's build step; it is not part of the encoder's C ABI."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2606_05981_amd", "libmte_probe.so"))
    lib.mte_probe_mfma.restype = ctypes.c_int
    lib.mte_probe_mfma.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]
    return lib


def mfma_rate(torch, blocks=512, iters=20000):
    """Dense fp16 matrix-core rate the device sustains under load (mte_probe_mfma: independent
    32x32x16 MFMA chains, no memory traffic), TFLOP/s: the measured counterpart of the
    published 2.5 PFLOP/s, which assumes the 2.4 GHz peak clock."""
    lib = _probe_lib()

    class _P:
        @staticmethod
        def mte_probe_mfma(b, i, sink, st):
            if lib.mte_probe_mfma(b, i, sink, st) != 0:
                raise RuntimeError("mte_probe_mfma failed")

    B = _P
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    B.mte_probe_mfma(blocks, iters // 10, sink.data_ptr(), st)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    B.mte_probe_mfma(blocks, iters, sink.data_ptr(), st)
    e1.record()
    torch.cuda.synchronize()
    flops = blocks * 4 * iters * 8 * 32768
    return round(flops / (e0.elapsed_time(e1) / 1e3) / 1e12, 1)


def copy_calibration(torch, mib=512, reps=5):
    """A plain device-to-device copy of `mib` MiB, `reps` times: the known-size kernel
    that calibrates the FETCH_SIZE / WRITE_SIZE counters (each dispatch moves exactly
    mib MiB in and mib MiB out)."""
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_mib": mib, "dispatches": reps}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="stack_b16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-batch1", action="store_true")
    ap.add_argument("--no-regimes", action="store_true",
                    help="skip the 8 x 96, 32 x 320 and mixed 32-sequence regimes")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run the known-size copy used to calibrate HBM byte counters")
    ap.add_argument("--prefix", type=int, default=0,
                    help="also measure frames sharing a prefix of this many text tokens")
    ap.add_argument("--no-e4m3", action="store_true",
                    help="skip the runs with e4m3 weights (batch 1 and the main workload)")
    ap.add_argument("--no-pipeline", action="store_true",
                    help="skip the frames -> vision tower -> decoder run")
    ap.add_argument("--vision-only", action="store_true",
                    help="only run the vision tower and print its figures (for profiling)")
    ap.add_argument("--no-vision", action="store_true",
                    help="skip the vision-tower run (16 images of 256x256)")
    ap.add_argument("--profile-pass", action="store_true",
                    help="only the main workload's warm-up and timed steps (for counter runs under rocprofv3)")
    ap.add_argument("--e4m3-weights", action="store_true",
                    help="with --profile-pass: the encoder holds e4m3 weights")
    ap.add_argument("--no-overlap", action="store_true",
                    help="skip the encoder on a side stream beside a main-stream GEMM load")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); frames are independent, "
              "so more GPUs would each run this same single-GPU path on a share of the batch.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "no GPU"
    if args.copy_calibration:
        copy_calibration(torch)
        return
    if args.vision_only:
        print(json.dumps({"vision_tower": run_vision(torch, args.steps, args.warmup)}), flush=True)
        return

    if args.profile_pass:
        r = run_workload(torch, args.workload, args.steps, args.warmup, weight_format=1 if args.e4m3_weights else 0)
        print(json.dumps({"profile_pass": args.workload, "e4m3_weights": args.e4m3_weights,
                          "ms_per_step": round(r["wall_s"] * 1e3 / args.steps, 4)}), flush=True)
        return
    main_run = run_workload(torch, args.workload, args.steps, args.warmup, timing_classes=(0, 1, 2, 3, 4))
    dims, T = main_run["dims"], main_run["T"]
    K = args.steps
    ms_step = main_run["wall_s"] * 1e3 / K
    tok_s = T * K / main_run["wall_s"]
    frames_s = len(main_run["lens"]) * K / main_run["wall_s"]
    n_launch, kern_ms = main_run["kern"][3]
    gu_flops = gemm_flops(dims, T)["gate_up"]
    # fp16 weights + fp16 normalised input + fp16 SwiGLU output
    gu_bytes = 2 * dims.ffn * dims.hidden * 2 + T * dims.hidden * 2 + T * dims.ffn * 2
    avg_us = kern_ms * 1e3 / max(n_launch, 1)
    achieved = gu_flops / (avg_us * 1e-6) / 1e12
    total_tflops = step_flops(dims, main_run["lens"]) * K / main_run["wall_s"] / 1e12
    res = {
        # value: tokens/s at batch 16 (frames_per_s beside it); batch 1 in "batch1"; the
        # roofline fractions in "roofline" (MFMA, batch 16) and "batch1.hbm_roofline"
        "metric": "encoder prefill tokens/s & frames/s (96 tok/frame, bs 1/16); % MFMA/HBM roofline",
        "value": round(tok_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "precision": ("projections: fp16 MFMA operands (bf16 weights as power-of-two scaled "
                      "fp16, exact for every weight down to 2^-31 of its matrix's largest "
                      "magnitude; activations rounded once to fp16), fp32 "
                      "accumulate; attention: bf16 hi+lo split operands, fp32 softmax; fp32 "
                      "residual stream and norms"),
        "data": "synthetic (seeded random-init weights and embeddings)",
        "config": {"workload": f"{args.workload}: {len(main_run['lens'])} frames x "
                               f"{max(main_run['lens'])} tokens, 28-layer Qwen3-VL-2B-class decoder "
                               "(D 2048, 16q/8kv heads, d 128, FFN 6144), M-RoPE 24/20/20",
                   "batch": len(main_run["lens"]), "tokens_per_step": T},
        "frames_per_s": round(frames_s, 1),
        "step_launch": "HIP graph replay" if main_run["graph"] else "eager",
        "step_ms_stats": main_run["stats"],
        "hbm_copy_gbs_measured": copy_bandwidth(torch),
        "mfma_f16_tflops_measured": None,
        "eager_ms_per_step": round(main_run["eager_s"] * 1e3 / K, 4),
        "model_tflops": round(total_tflops, 1),
        "roofline": {"kernel": "gate/up GEMM + SwiGLU", "bound": "mfma",
                     "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": measured_traffic(),
                     "algorithmic_bytes_per_launch": gu_bytes,
                     "avg_launch_us": round(avg_us, 2), "launches": n_launch,
                     "flops_per_launch": gu_flops,
                     # the whole step (all kernels, algorithmic flops) against the same peak
                     "step_achieved": round(total_tflops, 1),
                     "step_frac": round(total_tflops / PEAK_BF16_TFLOPS, 4),
                     "kernels": kernel_table(dims, main_run["lens"], main_run["kern"])},
    }
    measured = mfma_rate(torch)
    res["mfma_f16_tflops_measured"] = measured
    res["roofline"]["frac_of_measured_peak"] = round(achieved / measured, 4)
    if not args.no_batch1:
        b1 = run_workload(torch, "stack_b1", K, args.warmup, timing_classes=(0, 1, 2, 3, 4))
        t1 = b1["wall_s"] / K
        wbytes = dims.n_layers * dims.params_per_layer * 2 + 2 * b1["T"] * dims.hidden * 2
        res["batch1"] = {"workload": "stack_b1: 1 frame x 96 tokens, 28 layers",
                         "tokens_per_s": round(b1["T"] / t1, 1), "frames_per_s": round(1 / t1, 1),
                         "ms_per_step": round(t1 * 1e3, 4),
                         "step_ms_stats": b1["stats"],
                         "eager_ms_per_step": round(b1["eager_s"] * 1e3 / K, 4),
                         "hbm_roofline": {"bound": "hbm", "achieved": round(wbytes / t1 / 1e9, 1),
                                          "peak": PEAK_HBM_GBS, "unit": "GB/s",
                                          "frac": round(wbytes / t1 / 1e9 / PEAK_HBM_GBS, 4),
                                          "bytes_per_step": wbytes, "traffic": measured_step_traffic(),
                                          "frac_of_measured_copy": round(wbytes / t1 / 1e9 / res["hbm_copy_gbs_measured"], 4),
                                          "kernels": kernel_table(dims, b1["lens"], b1["kern"])}}
    if not args.no_regimes:
        res["other_regimes"] = run_regimes(torch, min(K, 10), args.warmup)
    if not args.no_vision:
        res["vision_tower"] = run_vision(torch, K, args.warmup)
        if not args.no_pipeline:
            res["frames_to_hidden"] = run_pipeline(torch, K, args.warmup)
    if not args.no_e4m3:
        res["e4m3_weights"] = run_e4m3(torch, args.workload, K, args.warmup, dims, not args.no_batch1)
    if not args.no_overlap:
        res["side_stream_overlap"] = {
            "batch16": run_overlap(torch, args.workload, K, args.warmup),
            "batch1": run_overlap(torch, "stack_b1", K, args.warmup)}
    if args.prefix > 0:
        res["shared_prefix"] = run_prefix(torch, args.prefix, K, args.warmup)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
