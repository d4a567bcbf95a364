#!/usr/bin/env python3
"""Benchmark of the SAS hot path on one MI355X.

A step is one decoder-layer forward of the 7B-shape workload (batch 1,
1024 tokens: 576 image tokens then 448 text tokens, bf16, GATED SAS attention
with B = 64, K = 8): RMSNorm, QKV GEMM + RoPE, block summaries, selector and
Top-K, gated block-sparse attention, O-projection + residual, RMSNorm,
gate/up GEMM + SwiGLU, down GEMM + residual -- all HIP kernels of libsas.so.
Inputs are resident in HBM before the timed region.

Prints one JSON line: tokens/s per layer (value), algorithmic TFLOP/s and
its fraction of the bf16 MFMA peak, the roofline of the dominant kernel
(timed with HIP events on its stream over a second pass of the same steps)
and the fp64 CPU oracle timed on the host over one layer forward.
"""
import argparse
import csv
import glob
import hashlib
import json
import os
import sys
import time

BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
HBM_PEAK_GBS = 8000.0

METRIC = "prefill tokens/s per layer + % bf16 MFMA peak; decode % HBM GB/s"

HERE = os.path.dirname(os.path.abspath(__file__))
GEMM_SRC = os.path.join(HERE, "paper_2609_13141_amd", "csrc", "gemm.hip")
TRAFFIC_FILE = os.path.join(HERE, "profiles", "gemm_gate_up_7b_layer_1k_traffic.txt")
# the gate/up GEMM at 1024 rows: one round of 256x256 tiles, then 256x128 tiles
DOM_KERNELS = ("gemm_bf16_lds_kernel<1, 256, 256, 2, 4, 2>", "gemm_bf16_lds_kernel<1, 256, 128, 4, 2, 3>")
COPY_BYTES = 512 * 2**20  # calibration copy: reads and writes this many bytes once


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # about 0.1 s of layer steps timed after 25 ms of warmup: a 20-step region (12 ms) ends
    # before the clocks have settled and measured about 12% slower per step
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="7b_layer_1k")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true", help="skip the decode-step measurement")
    ap.add_argument("--no-long-decode", action="store_true", help="skip the 64K..512K-context decode sweep")
    ap.add_argument("--no-backward", action="store_true", help="skip the training-step backward measurement")
    ap.add_argument("--no-stats", action="store_true", help="skip the selection-statistics measurement")
    ap.add_argument("--cpu-threads", type=int, default=0, help="oracle BLAS threads (0: affinity, max 16)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain device copy of %d MiB (reference for HBM counters)" % (COPY_BYTES >> 20))
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write the gate/up GEMM traffic summary from two rocprofv3 --pmc runs and exit")
    return ap.parse_args()


def source_hash():
    with open(GEMM_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def pmc_per_dispatch(run_dir, counter):
    """Per-call value of `counter` for the dominant GEMM (the sum over its
    launches of each kernel's mean per dispatch) and the mean for the
    calibration copy, from a rocprofv3 --pmc csv run directory."""
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    keys = list(DOM_KERNELS) + ["copy"]
    vals = {k: {} for k in keys}
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            key = next((k for k in DOM_KERNELS if k in name), None)
            if key is None and "copy" in name.lower():
                key = "copy"
            if key:
                d = vals[key]
                d[r["Dispatch_Id"]] = d.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    out = {}
    for k, d in vals.items():
        if not d:
            raise SystemExit(f"{counter}: no {k} dispatch found in {run_dir}")
        v = sorted(d.values())
        if k == "copy":
            v = v[-2:]  # the two calibration copies are by far the largest copy dispatches
        out[k] = sum(v) / len(v)
    out["gemm"] = sum(out[k] for k in DOM_KERNELS)
    return out


def write_traffic_summary(fetch_dir, write_dir):
    """HBM traffic per launch of the gate/up GEMM: FETCH_SIZE and WRITE_SIZE
    (KiB per dispatch) scaled by what they read for a copy of known size."""
    fe = pmc_per_dispatch(fetch_dir, "FETCH_SIZE")
    wr = pmc_per_dispatch(write_dir, "WRITE_SIZE")
    f_fetch = COPY_BYTES / (fe["copy"] * 1024.0)
    f_write = COPY_BYTES / (wr["copy"] * 1024.0)
    fetch_b = fe["gemm"] * 1024.0 * f_fetch
    write_b = wr["gemm"] * 1024.0 * f_write
    lines = [
        "# HBM traffic of the gate/up GEMM (7b_layer_1k, 1024 x 4096 x 2*11008) per launch",
        f"# kernels (summed per call): {', '.join(DOM_KERNELS)}",
        "# rocprofv3 --pmc FETCH_SIZE (then WRITE_SIZE) -- python3 bench.py --no-decode --no-cpu-baseline "
        "--steps 5 --warmup 2 --calibrate-copy",
        f"# calibration: plain copy of {COPY_BYTES} bytes read {fe['copy']:.0f} KiB fetch, {wr['copy']:.0f} KiB write",
        f"source_sha={source_hash()}",
        f"fetch_kib_raw={fe['gemm']:.1f}",
        f"write_kib_raw={wr['gemm']:.1f}",
        f"fetch_factor={f_fetch:.4f}",
        f"write_factor={f_write:.4f}",
        f"fetch_bytes={fetch_b:.0f}",
        f"write_bytes={write_b:.0f}",
        f"traffic_bytes={fetch_b + write_b:.0f}",
    ]
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def measured_traffic():
    """Traffic per launch from the committed counter summary, or None if the
    GEMM source changed since the counters were taken."""
    try:
        kv = dict(l.strip().split("=", 1) for l in open(TRAFFIC_FILE) if "=" in l and not l.startswith("#"))
    except OSError:
        return None
    if kv.get("source_sha") != source_hash():
        return None
    return int(float(kv["traffic_bytes"]))


def main():
    args = parse()
    if args.pmc_summary:
        write_traffic_summary(*args.pmc_summary)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the SAS hot path here is single-GPU "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    cores = args.cpu_threads or min(16, len(os.sched_getaffinity(0)))
    for var in ("OPENBLAS_NUM_THREADS", "OMP_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = str(cores)

    import numpy as np
    import torch

    here = os.path.dirname(os.path.abspath(__file__))
    sys.path.insert(0, here)
    from paper_2609_13141_amd import configs, inputs, sas

    w = configs.BY_NAME[args.workload]
    dev = "cuda:0"
    torch.cuda.set_device(0)
    x_np = inputs.embeddings(w)
    W_np = inputs.layer_weights(w)
    x = sas.to_device(x_np, w.dtype, dev)
    W = sas.weights_to_device(W_np, w.dtype, dev)
    cfg = sas.make_config(w)
    ws = sas.Workspace(dev)

    def step():
        return sas.layer_forward(cfg, x, W, stats=False, ws=ws)["y"]

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / args.steps
    T = w.tokens
    tok_s = T / (ms * 1e-3)
    flops = w.prefill_flops()
    tflops = flops / (ms * 1e-3) / 1e12

    # second pass of the same steps with an event pair around every kernel
    sas.profiler_start(64 * args.steps + 64)
    for _ in range(args.steps):
        step()
    recs = sas.profiler_stop()
    if args.calibrate_copy:
        src = torch.empty(COPY_BYTES // 2, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    fam = {}
    for name, t in recs:
        fam.setdefault(name, []).append(t)
    kern_ms = {k: sum(v) / len(v) for k, v in fam.items()}
    kern_calls = {k: len(v) // args.steps for k, v in fam.items()}
    # dominant kernel: the gate/up GEMM (2 * T * d * 2 * d_ff algorithmic flops per launch)
    dom = "gemm_gate_up"
    dom_flops = 2.0 * T * w.d_model * 2 * w.d_ff
    dom_tf = dom_flops / (kern_ms[dom] * 1e-3) / 1e12

    line = {
        "metric": METRIC,
        "value": round(tok_s, 1),
        "unit": "tokens/s/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1) text / N(0,1)*2 image embeddings, N(0,0.02) weights)",
        "config": {"workload": w.name, "batch": w.batch, "seq_len": w.seq_len, "d_model": w.d_model,
                   "n_heads": w.n_heads, "n_kv_heads": w.n_kv_heads, "head_dim": w.head_dim,
                   "d_ff": w.d_ff, "mode": w.mode, "block_size": w.block_size, "top_k": w.top_k},
        "alg_tflops": round(tflops, 2),
        "mfma_frac": round(tflops / BF16_PEAK_TFLOPS, 4),
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(dom_tf, 2),
                     "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(dom_tf / BF16_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic(), "alg_gflop_per_launch": round(dom_flops / 1e9, 3),
                     "avg_ms": round(kern_ms[dom], 4)},
        "kernels_ms": {k: round(v, 4) for k, v in sorted(kern_ms.items(), key=lambda kv: -kv[1] * kern_calls[kv[0]])},
    }

    if not args.no_decode:
        del x, W, ws
        torch.cuda.empty_cache()
        line["decode"] = decode_bench(DECODE_WARMUP)
        torch.cuda.empty_cache()
    if not args.no_long_decode:
        line["decode_long"] = decode_long_bench()
        torch.cuda.empty_cache()
    if not args.no_backward:
        line["backward"] = backward_bench()
        torch.cuda.empty_cache()
    if not args.no_stats:
        line["stats"] = stats_bench()
        torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, x_np, W_np, cores)
    print(json.dumps(line), flush=True)


# untimed decode steps before the 256 timed ones (fixes the positions 2053..2308)
DECODE_WARMUP = 5


def decode_bench(warmup):
    """The serving workload of the paper's method (Sec. 5.1, Alg. 2): a
    32-layer 7B-shape stack, 8 sequences of 576 image + 1472 text tokens
    prefilled densely into 16-token pages, then greedy SAS decode steps
    (B = 64, K = 16): every step embeds the 8 new tokens, runs the decode step
    of each layer (Top-K blocks per KV group, attention to them plus the
    current block) and the LM head with greedy argmax.  `warmup` untimed
    steps, then the workload's 256 timed steps; weights and inputs resident
    in HBM (13 GB of weights per step defeat the 256 MB last-level cache)."""
    import torch
    from paper_2609_13141_amd import configs, inputs, model, sas
    w = configs.STACK_DECODE
    dev = "cuda:0"
    layers = [inputs.layer_weights_device(w, layer=l, device=dev) for l in range(w.n_layers)]
    ends = inputs.model_ends_device(w, device=dev)
    steps = w.decode_steps
    max_len = w.seq_len + warmup + steps + 8
    st = model.Stack(w, layers, ends, max_len=max_len, device=dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    tok = st.prefill(ends["token_ids"], ends["img_embed"])
    torch.cuda.synchronize()
    prefill_ms = (time.perf_counter() - t0) * 1e3
    pos_all = st.positions(warmup + steps + 4)
    for p in pos_all[:warmup]:
        tok, _, _ = st.step(tok, p)
    torch.cuda.synchronize()
    t_first = st.pos
    t0 = time.perf_counter()
    for p in pos_all[warmup:warmup + steps]:
        tok, _, _ = st.step(tok, p)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    # algorithmic bytes of one step: every layer's weights, kept K/V and
    # summaries read, the new K/V written; the embedding rows and LM head
    B, K, dh, Hkv, b, L = w.block_size, w.top_k, w.head_dim, w.n_kv_heads, w.batch, w.n_layers
    tot = 0.0
    for t in range(t_first, t_first + steps):
        ct = t // B
        kept = B * min(K, ct) + (t % B) + 1
        per_layer = 2.0 * w.linear_params() + b * Hkv * (kept * dh * 2 * 2 + ct * dh * 2 + 2 * dh * 2)
        tot += L * per_layer + 2.0 * w.vocab * w.d_model + b * w.d_model * 2
    nbytes = tot / steps
    # per-kernel view over a few more steps, with an event pair around every launch
    nprof = 3
    sas.profiler_start(64 * L * nprof + 256)
    for p in pos_all[warmup + steps:warmup + steps + nprof]:
        tok, _, _ = st.step(tok, p)
    recs = sas.profiler_stop()
    fam = {}
    for name, v in recs:
        fam.setdefault(name, []).append(v)
    kms = {k: sum(v) / len(v) for k, v in fam.items()}
    gu_bytes = 2.0 * w.d_model * 2 * w.d_ff
    return {"workload": f"{w.name}: {L} layers, batch {b}, prompt {w.seq_len} tokens (576 image + 1472 text), "
                        f"pages of {w.page_size}, B={B}, K={K}, greedy steps at positions {t_first}.."
                        f"{t_first + steps - 1}",
            "steps": steps, "warmup": warmup,
            "ms_per_step": round(ms, 4),
            "tokens_per_s": round(b / (ms * 1e-3), 1),
            "ms_per_layer_step": round(ms / L, 4),
            "bytes_per_step": int(nbytes),
            "hbm_gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "prefill_ms": round(prefill_ms, 2),
            "prefill_tokens_per_s_per_layer": round(w.tokens / (prefill_ms * 1e-3 / L), 1),
            "gate_up_gemv_gbs": round(gu_bytes / (kms["dec_gate_up"] * 1e-3) / 1e9, 1),
            "kernels_ms": {k: round(v, 4) for k, v in sorted(kms.items(), key=lambda kv: -kv[1])}}


def decode_long_bench(steps=60, warmup=20):
    """One 7B-shape layer's SAS decode step at 64K..512K tokens of context,
    batch 1 and 8, K = 32 blocks of 64 (the paper's default budget): the
    selection scores every cached block summary (8192 at 512K) and attends
    to the 32 kept blocks plus the current one.  The caches are filled on
    the GPU with synthetic N(0,1) keys, values and summaries (timing does not
    depend on their values); the steps cycle over the last 20 positions (a
    step at position p attends to positions <= p only, so the later ones
    written before it do not change its work)."""
    import torch
    from paper_2609_13141_amd import configs, inputs, sas
    base = configs.LONG_DECODE
    dev = "cuda:0"
    Wd = inputs.layer_weights_device(base, device=dev)
    out = []
    for b in (1, 8):
        for ctx in (65536, 131072, 262144, 524288):
            w = base.with_(batch=b, seq_len=ctx)
            cfg = sas.make_config(w, "sparse")
            cache = sas.alloc_cache(cfg, b, ctx, page_size=w.page_size, device=dev, seed=b)
            cache.k_pages.normal_()
            cache.v_pages.normal_()
            cache.k_summary.normal_()
            x = torch.randn(b, w.d_model, device=dev).to(torch.bfloat16)
            ws = sas.Workspace(dev)
            p0 = ctx - 20
            poss = [torch.full((b,), p0 + s, dtype=torch.int32, device=dev) for s in range(20)]
            for s in range(warmup):
                sas.decode_step(cfg, x, poss[s % len(poss)], Wd, cache, sel_idx=False, ws=ws)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for s in range(warmup, warmup + steps):
                sas.decode_step(cfg, x, poss[s % len(poss)], Wd, cache, sel_idx=False, ws=ws)
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) * 1e3 / steps
            sas.profiler_start(64 * 3 + 16)
            for s in range(warmup + steps, warmup + steps + 3):
                sas.decode_step(cfg, x, poss[s % len(poss)], Wd, cache, sel_idx=False, ws=ws)
            recs = sas.profiler_stop()
            fam = {}
            for name, v in recs:
                fam.setdefault(name, []).append(v)
            kms = {k: sum(v) / len(v) for k, v in fam.items()}
            B, K, dh, Hkv = w.block_size, w.top_k, w.head_dim, w.n_kv_heads
            tot = 0.0
            for s in range(warmup, warmup + steps):
                t = p0 + s % len(poss)
                ct = t // B
                kept = B * min(K, ct) + (t % B) + 1
                tot += 2.0 * w.linear_params() + b * Hkv * (kept * dh * 2 * 2 + ct * dh * 2 + 2 * dh * 2)
            nbytes = tot / steps
            sel_ms = kms.get("dec_select", 0.0)
            out.append({"context": ctx, "batch": b, "ms_per_layer_step": round(ms, 4),
                        "bytes_per_layer_step": int(nbytes),
                        "hbm_gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
                        "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                        "select_ms": round(sel_ms, 4), "select_share": round(sel_ms / sum(kms.values()), 3),
                        "summary_bytes": b * Hkv * (ctx // B) * dh * 2})
            del cache, ws
            torch.cuda.empty_cache()
    return out


def backward_bench(steps=10, warmup=3):
    """The kernels of the method's training step (Alg. 1; App. E's
    recomputation backward): the attention backward (dQ, dK, dV and the
    selected blocks' log-gate gradient) and the selector backward (score,
    gate-query and summary gradients), after one GATED forward of the same
    inputs.  Q, K, V and dO are N(0,1) drawn on the GPU (seeded); timing
    depends on the inputs only through which blocks are selected.
    Algorithmic FLOPs of the attention backward: 10 dh per attended
    (query, key) pair and head (QK^T and dO V^T recomputed, dQ, dK, dV)."""
    import torch
    from paper_2609_13141_amd import configs, sas
    dev = "cuda:0"
    out = []
    for name in ("7b_layer_4k_b4", "gqa28x4_layer_16k"):
        w = configs.BY_NAME[name]
        g = torch.Generator(device=dev)
        g.manual_seed(1000 + w.index)
        b, n, H, Hkv, dh = w.batch, w.seq_len, w.n_heads, w.n_kv_heads, w.head_dim

        def rnd(*shape):
            return torch.randn(*shape, generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
        q, k, v, d_o = rnd(b, n, H, dh), rnd(b, n, Hkv, dh), rnd(b, n, Hkv, dh), rnd(b, n, H, dh)
        cfg = sas.make_config(w)
        ws_f, ws_b, ws_s = sas.Workspace(dev), sas.Workspace(dev), sas.Workspace(dev)
        fw = sas.attention_prefill(cfg, q, k, v, log_gate=True, ws=ws_f)

        def bwd():
            ab = sas.attention_backward(cfg, q, k, v, fw["o"], d_o, fw["lse"], fw["sel_idx"], fw["log_gate"],
                                        ws=ws_b)
            sas.selector_backward(cfg, q, k, fw["sel_idx"], fw["log_gate"], ab["dlog_gate"], ws=ws_s)
        for _ in range(warmup):
            bwd()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            bwd()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / steps
        sas.profiler_start(64 * steps + 64)
        for _ in range(steps):
            bwd()
            sas.attention_prefill(cfg, q, k, v, log_gate=True, ws=ws_f)
        recs = sas.profiler_stop()
        fam = {}
        for nm, t in recs:
            fam.setdefault(nm, []).append(t)
        kms = {kk: sum(vv) / len(vv) for kk, vv in fam.items()}
        flops = 10.0 * dh * H * b * w.attended_pairs()
        att_ms = kms["attention_bwd"]
        tf = flops / (att_ms * 1e-3) / 1e12
        sel_ms = sum(kms.get(kk, 0.0) for kk in ("sel_bwd_ds", "sel_bwd_gemm"))
        out.append({"workload": f"{w.name}: batch {b}, {n} tokens, {H}/{Hkv} heads, dh {dh}, B={w.block_size}, "
                                f"K={w.top_k}, GATED",
                    "ms_per_backward": round(ms, 4),
                    "attention_bwd_ms": round(att_ms, 4),
                    "attention_bwd_gflop": round(flops / 1e9, 2),
                    "attention_bwd_tflops": round(tf, 1),
                    "mfma_frac": round(tf / BF16_PEAK_TFLOPS, 4),
                    "attention_fwd_ms": round(kms["attention"], 4),
                    "bwd_over_fwd": round(att_ms / kms["attention"], 2),
                    "selector_bwd_ms": round(sel_ms, 4),
                    "kernels_ms": {kk: round(vv, 4) for kk, vv in sorted(kms.items(), key=lambda kv: -kv[1])}})
        del q, k, v, d_o, fw, ws_f, ws_b, ws_s
        torch.cuda.empty_cache()
    return out


def stats_bench(steps=10, warmup=3):
    """The selection statistics of Sec. 6.1 for one layer of 7b_layer_4k_b4
    (4 x 4096 tokens, 32 heads, B = 64, K = 16): mass coverage with both
    weightings and the accumulation of the selected and full-attention
    reference block sets.  A dense causal Q K^T pass: 2 dh flops per
    (query, key <= query) pair and head, plus per-head Top-K and votes."""
    import torch
    from paper_2609_13141_amd import configs, sas
    dev = "cuda:0"
    w = configs.BY_NAME["7b_layer_4k_b4"]
    g = torch.Generator(device=dev)
    g.manual_seed(2000 + w.index)
    b, n, H, Hkv, dh = w.batch, w.seq_len, w.n_heads, w.n_kv_heads, w.head_dim
    q, k, v = (torch.randn(*s, generator=g, device=dev).to(torch.bfloat16)
               for s in ((b, n, H, dh), (b, n, Hkv, dh), (b, n, Hkv, dh)))
    cfg = sas.make_config(w)
    fw = sas.attention_prefill(cfg, q, k, v)
    su, ru = sas.alloc_union(cfg, b, n), sas.alloc_union(cfg, b, n)
    ws = sas.Workspace(dev)

    def run():
        sas.selection_stats(cfg, q, k, v, fw["sel_idx"], sel_union=su, ref_union=ru, ws=ws)
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        run()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    sas.profiler_start(16 * steps + 16)
    for _ in range(steps):
        run()
    recs = sas.profiler_stop()
    fam = {}
    for nm, t in recs:
        fam.setdefault(nm, []).append(t)
    kms = {kk: sum(vv) / len(vv) for kk, vv in fam.items()}
    flops = 2.0 * dh * H * b * n * (n + 1) / 2
    inter, tot, rec = sas.overlap_recall(su, ru)
    return {"workload": f"{w.name}: batch {b}, {n} tokens, {H}/{Hkv} heads, dh {dh}, B={w.block_size}, K={w.top_k}",
            "ms_per_layer": round(ms, 4), "pass_gflop": round(flops / 1e9, 2),
            "pass_tflops": round(flops / (kms["stats"] * 1e-3) / 1e12, 1),
            "recall_random_inputs": round(rec, 4),
            "kernels_ms": {kk: round(vv, 4) for kk, vv in sorted(kms.items(), key=lambda kv: -kv[1])}}


def cpu_baseline(w, x_np, W_np, cores):
    """The fp64 oracle, as it stands, over one full layer forward of the same
    workload on the host cores."""
    import numpy as np

    import oracle
    from oracle.layer import Spec
    try:
        from threadpoolctl import threadpool_info
        used = max([p.get("num_threads", 1) for p in threadpool_info()] or [cores])
    except Exception:
        used = cores
    spec = Spec(w.n_heads, w.n_kv_heads, w.head_dim, w.block_size, w.top_k, w.mode, w.dtype, w.rope_base,
                w.rms_eps)
    x = x_np.astype(np.float64)
    Wd = {k: (None if a is None else a.astype(np.float64)) for k, a in W_np.items()}
    t0 = time.perf_counter()
    oracle.layer_forward(x, Wd, spec)
    dt = time.perf_counter() - t0
    return {"value": round(w.tokens / dt, 2), "unit": "tokens/s/layer", "cores": int(used), "kind": "oracle",
            "sample": f"one full layer forward of {w.name} ({w.tokens} tokens), fp64 NumPy, {dt:.2f} s"}


if __name__ == "__main__":
    main()
