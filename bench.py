#!/usr/bin/env python3
"""Throughput of the layer-replica hot path on one MI355X.

One step = one pass of the whole path (gather, RMSNorm, QKV, RoPE + cache
append, paged attention, O projection + residual, RMSNorm, SwiGLU MLP +
residual, scatter) over one batch, through the C ABI. The default run measures
both halves of the metric:
  * the headline: the Llama-3-8B-shaped layer, bf16 decode of a 64-request
    batch with lognormal contexts (decode layer-steps/s, HBM roofline);
  * under "prefill": the Qwen-32B-shaped layer, a 2048-token chunked prefill
    over four requests (tokens/s per layer, MFMA roofline).
--workload runs one workload alone. Each workload reports the mean of K hot
back-to-back steps (the value), the median of at least 30 steps each after a
1 GiB cache-flushing write, a HIP-graph replay, per-kernel event timings, and
fractions of the published peaks and of the peaks measured on this GPU.

Prints one JSON line on stdout; per-kernel timings go to stderr. Inputs are
synthetic (seeded) and resident in HBM before the timed region.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode layer-steps/s & prefill tokens/s per layer; % HBM / MFMA peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, TFLOP/s
XGMI_LINK_BPS = 153e9           # one MI355X xGMI link, bytes/s (boundary transfers)
FLUSH_BYTES = 1 << 30           # written between flushed steps: 4x the 256 MB MALL


def parse():
    p = argparse.ArgumentParser(description=__doc__)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default=None,
                   choices=["c2", "c3", "c3full", "c4p", "c4d", "c5"],
                   help="one workload only (default: the 8B batch-64 decode step as the "
                        "headline, plus the 32B 2048-token prefill under \"prefill\")")
    p.add_argument("--batch", type=int, default=64,
                   help="decode rows of the 8B workload (c2): one replica's share of the batch")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="target duration of the oracle CPU baseline (0 = skip)")
    p.add_argument("--no-graph", action="store_true",
                   help="skip the HIP-graph replay measurement of the same step")
    p.add_argument("--no-peaks", action="store_true",
                   help="skip the measured-peak probes (read stream, copy, MFMA loop)")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only time a plain 1 GiB device copy (the reference kernel that "
                        "scales the FETCH_SIZE / WRITE_SIZE counters to bytes)")
    return p.parse_args()


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_sha():
    """Digest of every kernel source without its comments and whitespace: a
    counter summary is only valid for the code it was taken with."""
    csrc = os.path.join(ROOT, "paper_2607_04181_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            with open(os.path.join(csrc, f), encoding="utf-8") as fh:
                code = fh.read()
            code = re.sub(r"/\*.*?\*/", " ", code, flags=re.S)
            code = re.sub(r"//[^\n]*", " ", code)
            code = " ".join(code.split())
            h.update(f.encode() + b"\0" + code.encode())
    return h.hexdigest()[:16]


def copy_calibration():
    """A 1 GiB device-to-device copy (torch's copy kernel): 1 GiB read and
    1 GiB written per launch, the known size the HBM counters are scaled by;
    also the practical copy bandwidth of the part."""
    import torch
    n = 1 << 28  # float32 elements: 1 GiB
    x = torch.empty(n, device="cuda")
    x.normal_()
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 20
    e0.record()
    for _ in range(reps):
        y.copy_(x)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n,
                      "us_per_copy": round(ms * 1e3, 1),
                      "GBps_read_plus_write": round(8 * n / (ms * 1e-3) / 1e9, 1)}), flush=True)


def load_traffic(kernel_kind, workload_name, src_sha):
    """HBM bytes per launch from a committed rocprofv3 counter summary, or
    None when there is none or the kernel sources changed since."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel_kind}_{workload_name}.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    m_sha = re.search(r"kernel_source_sha:\s*(\w+)", txt)
    m_b = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", txt)
    if not m_sha or not m_b or m_sha.group(1) != src_sha:
        return None
    return float(m_b.group(1))


def build_workload(name, batch=64):
    import numpy as np
    import workloads as W
    if name == "c2":
        wl = W.c2_llama8b_decode(batch)
        if batch != 64:
            wl.name = f"llama8b_decode_b{batch}"
        return wl, wl.batch, 1
    if name == "c3":
        wl = W.c3_llama8b_skewed()
        return wl, wl.batch, 1
    if name == "c3full":
        wl = W.c3_llama8b_skewed()
        wl.name = "llama8b_skewed_all256"
        return wl, wl.full_batch, 1
    if name == "c4p":
        wl = W.c4_qwen32b()
        return wl, wl.batch, 1
    if name == "c4d":
        wl = W.c4_qwen32b()
        wl.name = "qwen32b_decode_b128"
        return wl, wl.decode_after, 1
    if name == "c5":
        wl = W.c5_llama70b_span()
        return wl, wl.batch, wl.n_layers
    raise ValueError(name)


def measure_peaks(num_cus):
    """What this GPU sustains, measured here: a read stream over 2 GiB (the
    library's read probe; the best of its load depths and grid sizes), a 1 GiB
    device copy (torch's copy kernel, read + write) and a loop of bf16 MFMAs
    (the library's MFMA probe; the best of its chain counts and waves per
    SIMD), on random operands that change from one instruction to the next
    (the rate the power draw of real data allows: the MFMA ceiling used) and
    on constant ones. Each configuration: the median of 10 timed launches after 2
    warm-ups."""
    import torch
    import paper_2607_04181_amd as coco
    stream = torch.cuda.current_stream()

    def timed(fn, reps=10, warm=2):
        for _ in range(warm):
            fn()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps)]
        for a, b in ev:
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        t = sorted(a.elapsed_time(b) for a, b in ev)
        return t[len(t) // 2]

    nbytes = 2 << 30
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    buf.random_(0, 255)
    out = torch.empty(32 * num_cus, dtype=torch.int32, device="cuda")
    reads = {}
    for variant in (0, 1, 2):
        for per_cu in (4, 8, 16, 32):
            blocks = per_cu * num_cus
            reads[(variant, per_cu)] = timed(
                lambda: coco.coco_probe_read(buf, out, blocks, variant, stream))
    (best_v, best_cu), ms_read = min(reads.items(), key=lambda kv: kv[1])
    x = buf[: nbytes // 2]
    y = torch.empty_like(x)
    ms_copy = timed(lambda: y.copy_(x))
    del buf, x, y
    mout = torch.empty(4 * 4 * num_cus, dtype=torch.float32, device="cuda")
    mfmas = {}
    for operands in (0, 1):  # constant operands; random operands changing per instruction
        for chains in (4, 8):
            for per_cu in (1, 2, 4):  # 4-wave workgroups per CU: waves per SIMD
                blocks = per_cu * num_cus
                flops = [0.0]

                def mfma():
                    flops[0] = coco.coco_probe_mfma_bf16(40000 // chains, mout, blocks, chains,
                                                         operands, stream)
                ms = timed(mfma)
                mfmas[(operands, chains, per_cu)] = flops[0] / (ms * 1e-3) / 1e12
    best = {op: max(((c, w, t) for (o, c, w), t in mfmas.items() if o == op),
                    key=lambda x: x[2]) for op in (0, 1)}
    torch.cuda.empty_cache()
    return {"read_GBps": round(nbytes / (ms_read * 1e-3) / 1e9, 1),
            "copy_GBps": round(nbytes / (ms_copy * 1e-3) / 1e9, 1),
            "mfma_bf16_TFLOPs": round(best[1][2], 1),
            "mfma_bf16_const_operands_TFLOPs": round(best[0][2], 1),
            "method": (f"medians of 10 launches: read probe over 2 GiB (best of 3 load depths "
                       f"x 4 grid sizes: variant {best_v}, {best_cu} workgroups/CU), 1 GiB "
                       f"device copy (bytes read + written), bf16 MFMA probe (best of 4/8 "
                       f"chains x 1/2/4 waves per SIMD) with random operands that change "
                       f"from one instruction to the next ({best[1][0]} chains, {best[1][1]} "
                       f"waves; the rate under a GEMM's power draw, mfma_bf16_TFLOPs) and "
                       f"with constant operands ({best[0][0]} chains, {best[0][1]} waves)"),
            "read_GBps_all": {f"v{v}_{c}": round(nbytes / (ms * 1e-3) / 1e9, 1)
                              for (v, c), ms in reads.items()},
            "mfma_TFLOPs_all": {f"{'rand' if o else 'const'}_c{c}_w{w}": round(t, 1)
                                for (o, c, w), t in mfmas.items()}}


def run_workload(name, batch_rows, args, peaks, flush):
    """One workload: hot K-step timing (the contract's value), a cache-flushed
    median, a HIP-graph replay, per-kernel event timings, rooflines, and the
    oracle's CPU baseline. Frees its device memory before returning."""
    import numpy as np
    import torch

    import paper_2607_04181_amd as coco
    from workloads import device as WD

    wl, batch, n_layers = build_workload(name, batch_rows)
    shape = wl.shape
    t0 = time.time()
    layers = [WD.layer_tensors(shape, wl.tag, l, batch.num_blocks) for l in range(n_layers)]
    cfg = coco.make_config(shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                           shape.d_ffn, n_layers, shape.dtype, batch.n_rows, batch.n_seqs,
                           batch.block_table.shape[1], shape.rope_theta, shape.rms_eps)
    handle = coco.coco_layer_init(cfg, layers)
    hidden = WD.hidden_tensor(shape, wl.tag, batch.hidden_rows)
    bt = WD.batch_tensors(batch)
    torch.cuda.synchronize()
    log(f"setup {time.time() - t0:.1f}s: {wl.name}, {n_layers} layer(s), rows {batch.n_rows}, "
        f"blocks {batch.num_blocks}")

    # Oracle inputs for the CPU baseline, taken before the GPU touches them.
    cpu_inputs = None
    if args.cpu_seconds > 0:
        cpu_inputs = prepare_cpu_inputs(wl, batch, layers[0], hidden)

    stream = torch.cuda.current_stream()

    def step(st=None):
        st = stream if st is None else st
        if n_layers == 1:
            coco.coco_layer_forward(handle, 0, hidden, bt["row_idx"], bt["positions"],
                                    bt["seq_starts"], bt["block_table"], bt["ctx_lens"], st)
        else:
            coco.coco_layer_span_forward(handle, 0, n_layers, hidden, bt["row_idx"],
                                         bt["positions"], bt["seq_starts"], bt["block_table"],
                                         bt["ctx_lens"], st)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps

    # Cache-flushed steps: before each, a kernel writes the 1 GiB flush buffer
    # (four times the 256 MB last-level cache), outside the timed interval.
    # The written lines are dirty, so the step also pays their write-back; a
    # second series flushes with a read of the buffer (clean lines) instead.
    reps = max(30, args.steps)
    num_cus = torch.cuda.get_device_properties(0).multi_processor_count
    probe_out = torch.empty(8 * num_cus, dtype=torch.int32, device="cuda")

    def flushed_series(flush_fn):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        for r, (a, b) in enumerate(evs):
            flush_fn(r)
            a.record(stream)
            step()
            b.record(stream)
        torch.cuda.synchronize()
        return sorted(a.elapsed_time(b) for a, b in evs)

    flushed = flushed_series(lambda r: flush.fill_(float(r)))
    fms = flushed[len(flushed) // 2]
    flushed_rd = flushed_series(
        lambda r: coco.coco_probe_read(flush, probe_out, 8 * num_cus, 0, stream))
    fms_rd = flushed_rd[len(flushed_rd) // 2]

    # The same step captured once as a HIP graph and replayed (the forward
    # only enqueues kernels on fixed buffers, so it is capturable as is).
    graph = None
    if not args.no_graph:
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step(side)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step(torch.cuda.current_stream())
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        gms = e0.elapsed_time(e1) / args.steps
        graph = {"ms_per_step": round(gms, 4)}
        del g

    # Per-kernel durations: every launch carries a pair of HIP events that the
    # runtime timestamps at the kernel's start and end on its stream.
    coco.coco_layer_set_timing(handle, True)
    per_kernel = {}
    for _ in range(args.steps):
        step()
        for k, (t, n) in coco.coco_layer_read_timing(handle).items():
            t0_, n0_ = per_kernel.get(k, (0.0, 0))
            per_kernel[k] = (t0_ + t, n0_ + n)
    coco.coco_layer_set_timing(handle, False)

    M = batch.n_rows
    d, F = shape.d_model, shape.d_ffn
    Hq, Hkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    nqkv = (Hq + 2 * Hkv) * hd
    eb = shape.elem_bytes
    kvb = shape.kv_bytes_per_token()
    gemms = {"gemm_qkv": (nqkv, d), "gemm_o": (d, Hq * hd), "gemm_gate_up": (2 * F, d),
             "gemm_down": (d, F)}
    sum_ctx = int(np.sum(batch.ctx_lens))
    is_decode = batch.is_decode
    # Algorithmic work of one launch of each kernel kind.
    alg_bytes = {k: N * K * eb + M * K * eb + M * N * eb for k, (N, K) in gemms.items()}
    alg_flops = {k: 2.0 * M * N * K for k, (N, K) in gemms.items()}
    if is_decode:
        alg_bytes["attention"] = sum_ctx * kvb + 2 * M * Hq * hd * eb
        alg_flops["attention"] = 4.0 * Hq * hd * sum_ctx
    else:
        pairs = float(np.sum(batch.positions.astype(np.int64) + 1))
        alg_flops["attention"] = 4.0 * Hq * hd * pairs
        alg_bytes["attention"] = sum_ctx * kvb + 2 * M * Hq * hd * eb
    weight_bytes = shape.param_count() * eb * n_layers
    step_bytes = weight_bytes + n_layers * (sum_ctx * kvb + M * kvb) + 2 * M * d * eb
    step_flops = n_layers * (2.0 * M * (shape.param_count() - 2 * d) +
                             alg_flops["attention"])

    rows = []
    for k, (tot, n) in per_kernel.items():
        if n:
            rows.append((k, tot / n, n, tot))
    rows.sort(key=lambda r: -r[3])
    tot_all = sum(r[3] for r in rows)
    log(f"{wl.name}: hot {ms:.4f} ms/step, flushed median {fms:.4f} ms (write flush), "
        f"{fms_rd:.4f} ms (read flush), {reps} reps each")
    log(f"{'kernel':18s} {'avg us':>9s} {'share':>6s} {'GB/s':>8s} {'TFLOP/s':>8s}")
    for k, avg, n, tot in rows:
        gbs = alg_bytes.get(k, 0) / (avg * 1e-3) / 1e9 if k in alg_bytes else float("nan")
        tfs = alg_flops.get(k, 0) / (avg * 1e-3) / 1e12 if k in alg_flops else float("nan")
        log(f"{k:18s} {avg * 1e3:9.1f} {tot / tot_all:6.1%} {gbs:8.0f} {tfs:8.1f}")

    cand = [r for r in rows if r[0] in alg_bytes]
    dom, dom_avg, dom_n, _ = cand[0]
    bound = "hbm" if is_decode else "mfma"
    src_sha = kernel_source_sha()
    whole = {"step_hbm_bytes": step_bytes, "step_flops": step_flops,
             "step_GBps": round(step_bytes / (ms * 1e-3) / 1e9, 1),
             "step_TFLOPs": round(step_flops / (ms * 1e-3) / 1e12, 2)}
    whole["step_frac_hbm"] = round(whole["step_GBps"] / HBM_PEAK_GBS, 4)
    whole["step_frac_mfma"] = round(whole["step_TFLOPs"] / MFMA_BF16_PEAK_TFLOPS, 4)
    if bound == "hbm":
        achieved = alg_bytes[dom] / (dom_avg * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4)}
        step_frac = whole["step_frac_hbm"]
        meas_peak = peaks.get("read_GBps") if peaks else None
        step_meas = whole["step_GBps"]
    else:
        achieved = alg_flops[dom] / (dom_avg * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4)}
        step_frac = whole["step_frac_mfma"]
        meas_peak = peaks.get("mfma_bf16_TFLOPs") if peaks else None
        step_meas = whole["step_TFLOPs"]
    roof["traffic"] = load_traffic(dom, wl.name, src_sha)
    roof["kernel"] = dom
    roof["avg_launch_us"] = round(dom_avg * 1e3, 2)
    roof["algorithmic_per_launch"] = alg_bytes[dom] if bound == "hbm" else alg_flops[dom]
    # The whole step (every kernel and the gaps between them) against the same
    # peak: the layer's own fraction of the roofline.
    roof["step_frac"] = step_frac
    if meas_peak:
        roof["peak_measured"] = meas_peak
        roof["frac_measured"] = round(achieved / meas_peak, 4)
        roof["step_frac_measured"] = round(step_meas / meas_peak, 4)

    per_unit = n_layers * 1000.0 if is_decode else M * 1000.0
    value = per_unit / ms
    unit = "layer-steps/s" if is_decode else "tokens/s per layer"
    if graph is not None:
        graph["value"] = round(per_unit / graph["ms_per_step"], 2)
    def frac(t_ms):
        return round((step_bytes / (t_ms * 1e-3) / 1e9 / HBM_PEAK_GBS) if is_decode else
                     (step_flops / (t_ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS), 4)
    flushed_out = {"median_ms": round(fms, 4), "reps": reps,
                   "min_ms": round(flushed[0], 4), "max_ms": round(flushed[-1], 4),
                   "value": round(per_unit / fms, 2), "flush_bytes": flush.numel() * 4,
                   "flush": "1 GiB written before each step", "step_frac": frac(fms),
                   "read_flush": {"median_ms": round(fms_rd, 4),
                                  "value": round(per_unit / fms_rd, 2),
                                  "flush": "1 GiB read before each step",
                                  "step_frac": frac(fms_rd)}}

    # The paper's speedup model (Sec. 4.2) fed with this measured per-layer
    # time: boundary rows over one xGMI link, bf16 hidden states.
    full_layers = {4096: 32, 5120: 64, 8192: 80}.get(d)
    scaling = None
    if full_layers:
        t_layer = ms * 1e-3 / n_layers
        if is_decode:
            bs_rows, toks = M, 1
        else:
            bs_rows, toks = batch.n_seqs, max(1, M // max(1, batch.n_seqs))
        sm = coco.make_scale_model(full_layers, bs_rows, toks, d, 2.0, t_layer, XGMI_LINK_BPS)
        L = full_layers
        scaling = {"model_layers": L, "t_comp_ms": round(t_layer * 1e3, 4),
                   "link_GBps": XGMI_LINK_BPS / 1e9,
                   "comm_ms_P2": round(coco.coco_comm_time(sm, 2) * 1e3, 5),
                   "S": {f"N={N},P={P}": round(coco.coco_speedup(sm, N, P), 4)
                         for N in (L // 4, L // 2, L) for P in (2, 4)}}

    del handle, layers, hidden, bt
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    cpu = None
    if cpu_inputs is not None:
        cpu = cpu_baseline(wl, batch, cpu_inputs, args.cpu_seconds, n_layers, is_decode)
        del cpu_inputs

    config = {"workload": wl.name, "d_model": d, "n_q_heads": Hq, "n_kv_heads": Hkv,
              "head_dim": hd, "d_ffn": F, "layers": n_layers, "rows": M,
              "hidden_rows": batch.hidden_rows, "sum_ctx": sum_ctx,
              "mode": "decode" if is_decode else "prefill", "kv_block": 16,
              "parallelism": "single GPU (one replica's share)"}
    return {"value": round(value, 2), "unit": unit, "ms_per_step": round(ms, 4),
            "dtype": shape.dtype, "config": config, "roofline": roof, "whole_step": whole,
            "flushed": flushed_out, "graph_replay": graph, "scaling_model": scaling,
            "cpu_baseline": cpu}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "bench.py runs one replica's share on one MI355X; "
                          "sharding the row subsets over several GPUs is not implemented",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration()
        return

    if args.batch != 64 and args.workload not in (None, "c2"):
        print(json.dumps({"error": "--batch applies to the 8B decode workload (c2) only"}))
        sys.exit(2)
    if args.batch < 1:
        print(json.dumps({"error": "--batch must be >= 1"}))
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    num_cus = torch.cuda.get_device_properties(0).multi_processor_count
    peaks = None if args.no_peaks else measure_peaks(num_cus)
    if peaks:
        log(f"measured peaks: {peaks}")
    flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")

    if args.workload is None:
        # The metric's two halves: the 8B decode step (headline value) and the
        # 32B 2048-token chunked prefill (under "prefill").
        dec = run_workload("c2", args.batch, args, peaks, flush)
        pre = None if args.batch != 64 else run_workload("c4p", 64, args, peaks, flush)
    else:
        dec = run_workload(args.workload, args.batch, args, peaks, flush)
        pre = None

    out = {
        "metric": METRIC, "value": dec["value"], "unit": dec["unit"], "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": dec["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dec["dtype"], "data": "synthetic (seeded counter-based generator)",
        "config": dec["config"], "roofline": dec["roofline"], "whole_step": dec["whole_step"],
        "flushed": dec["flushed"], "graph_replay": dec["graph_replay"],
        "peaks_measured": peaks, "scaling_model": dec["scaling_model"],
        "cpu_baseline": dec["cpu_baseline"],
    }
    if pre is not None:
        out["prefill"] = {k: pre[k] for k in ("value", "unit", "ms_per_step", "config",
                                               "roofline", "whole_step", "flushed",
                                               "graph_replay", "cpu_baseline")}
    print(json.dumps(out), flush=True)


def prepare_cpu_inputs(wl, batch, layer0, hidden):
    """Host copies of the generator's tensors for the oracle (same bits as
    the CPU generator would give), taken before any kernel runs."""
    import numpy as np
    import torch
    from oracle.paged import depage_blocks

    def f64(t):
        return t.detach().to("cpu", torch.float32).numpy().astype(np.float64)

    shape = wl.shape
    sample_seqs = list(range(batch.n_seqs)) if batch.is_decode else [0]
    w = {k: f64(layer0[k]) for k in shape.weight_shapes()}
    K, V = [], []
    for s in sample_seqs:
        prior, ctx = int(batch.prior_lens[s]), int(batch.ctx_lens[s])
        nb = -(-prior // 16)
        Kc = np.zeros((ctx, shape.n_kv_heads, shape.head_dim))
        Vc = np.zeros_like(Kc)
        if nb:
            idx = torch.from_numpy(batch.block_table[s, :nb].astype(np.int64)).cuda()
            kb, vb = f64(layer0["k_cache"].index_select(0, idx)), f64(
                layer0["v_cache"].index_select(0, idx))
            Kc[:prior], Vc[:prior] = depage_blocks(kb, vb, prior)
        K.append(Kc)
        V.append(Vc)
    return {"w": w, "K": K, "V": V, "hidden": f64(hidden), "seqs": sample_seqs}


def cpu_baseline(wl, batch, inp, seconds, n_layers, is_decode):
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
    except ImportError:  # pragma: no cover
        threadpool_limits = None
    share = int(os.environ.get("OMP_NUM_THREADS", "0")) or len(os.sched_getaffinity(0))
    cores = min(share, len(os.sched_getaffinity(0)))
    ctx = threadpool_limits(cores) if threadpool_limits else None
    if ctx:
        ctx.__enter__()
    try:
        used = cores
        if threadpool_limits:
            info = threadpool_info()
            if info:
                used = max(i.get("num_threads", 1) for i in info)
        shape = wl.shape
        if is_decode:
            sub = batch
            n_units, unit = 1, "layer-steps/s"
            sample = f"whole {wl.name} decode step ({batch.n_rows} rows), one layer"
            seq_starts = None
        else:
            sub = batch.select_seqs(inp["seqs"])
            unit = "tokens/s per layer"
            sample = (f"request 0 of {wl.name} ({sub.n_rows} of {batch.n_rows} prefill tokens), "
                      "one layer")
            seq_starts = sub.seq_starts
        reps, t_start = 0, time.perf_counter()
        while True:
            cache = oracle.KVCache(inp["K"], inp["V"])
            oracle.layer_forward(inp["w"], shape, inp["hidden"], sub.row_idx, sub.positions,
                                 seq_starts, sub.ctx_lens, cache)
            reps += 1
            el = time.perf_counter() - t_start
            if el >= seconds:
                break
        if is_decode:
            value = reps / el
        else:
            value = reps * sub.n_rows / el
        return {"value": round(value, 4), "unit": unit, "cores": used, "kind": "oracle",
                "sample": f"{sample}, {reps} repetition(s) in {el:.1f}s, fp64 numpy"}
    finally:
        if ctx:
            ctx.__exit__(None, None, None)


if __name__ == "__main__":
    main()
