#!/usr/bin/env python3
"""Benchmark of the SAS hot path on one MI355X.

Headline workload: 7b_stack32_prefill2k_decode256_b8, the serving job of the
method (Sec. 5.1, Alg. 2) on a 32-layer 7B-shape stack.  One step is one pass
over one batch:
  * dense prefill of 8 sequences x 2048 tokens (576 image + 1472 text)
    through the 32 layers into 16-token pages: RMSNorm, QKV GEMM + RoPE,
    block summaries, causal attention, O-projection + residual, RMSNorm,
    gate/up GEMM + SwiGLU, down GEMM + residual, K/V and summaries into the
    cache; then the LM head and greedy argmax of the first token;
  * 256 greedy SAS decode steps (B = 64, K = 16): embedding, every layer's
    decode step (RMSNorm, QKV + RoPE + append, Top-K selection over the
    cached block summaries, block-sparse attention, O, MLP), LM head, argmax.
All in the HIP kernels of libsas.so; weights and prompts resident in HBM
before the timed region.

`value` = prefill tokens/s per layer (8 x 2048 tokens / (prefill time / 32));
`decode` carries the decode half of the metric (algorithmic HBM bytes per
step / step time, against 8 TB/s).  Each carries the roofline of its
dominant kernel: the prefill's gate/up GEMM and the decode's gate/up GEMV,
timed with HIP events recorded by the library on the kernels' stream inside
the timed region.  `layers` times the GATED layer forward (the SAS training-
form prefill, Eq. ours_train) of the other bf16 workloads, with the
attention's algorithmic and executed (whole key tiles) FLOPs.
`cpu_baseline`: the fp64 oracle on a bounded sample of the headline prefill.
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
HBM_PEAK_GBS = 8000.0       # MI355X HBM3E

METRIC = "prefill tokens/s per layer + % bf16 MFMA peak; decode % HBM GB/s"
HEADLINE = "7b_stack32_prefill2k_decode256_b8"

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "paper_2609_13141_amd", "csrc")
PROFILES = os.path.join(HERE, "profiles")
COPY_BYTES = 512 * 2**20  # calibration copy: reads and writes this many bytes once
COPY_KERNEL = "__amd_rocclr_copyBuffer"  # the runtime's blit kernel of a device-to-device copy

# Dominant kernels of the headline step and their HBM-traffic summaries
# (written by --pmc-summary from rocprofv3 --pmc runs of --only-headline).
DOMINANT = {
    "prefill": {"family": "gemm_gate_up", "kernel": "gemm_bf16_lds_kernel<1, 256, 256, 2, 4, 2, 64, 16>",
                "source": "gemm.hip", "file": "gemm_gate_up_7b_stack32_prefill2k_traffic.txt"},
    "decode": {"family": "dec_gate_up", "kernel": "gemv_kernel<4, 1>",
               "source": "gemv.hip", "file": "gemv_gate_up_7b_stack32_decode_b8_traffic.txt"},
}
DECODE_SAMPLE = 8   # the decode GEMV is event-timed on every 8th decode step of the timed region


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5, help="timed steps (one step: prefill + 256 decode steps)")
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--only-headline", action="store_true", help="the headline workload only (profiling runs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-layers", action="store_true", help="skip the GATED layer forwards")
    ap.add_argument("--no-long-decode", action="store_true", help="skip the 64K..512K-context decode sweep")
    ap.add_argument("--no-backward", action="store_true", help="skip the training-step backward measurement")
    ap.add_argument("--no-stats", action="store_true", help="skip the selection-statistics measurement")
    ap.add_argument("--cpu-threads", type=int, default=0, help="oracle BLAS threads (0: affinity, max 16)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain device copy of %d MiB (reference for HBM counters)" % (COPY_BYTES >> 20))
    ap.add_argument("--decode-steps", type=int, default=0,
                    help="decode steps per step (profiling runs; default: the workload's 256)")
    ap.add_argument("--only-layer", metavar="NAME", help="time only this workload's GATED layer forward "
                    "(profiling runs)")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write the dominant kernels' traffic summaries from two rocprofv3 --pmc runs and exit")
    ap.add_argument("--trace-summary", nargs=2, metavar=("RUN_DIR", "OUT"),
                    help="write a per-kernel table from a rocprofv3 --kernel-trace --stats run and exit")
    ap.add_argument("--mfma-summary", nargs=2, metavar=("RUN_DIR", "OUT"),
                    help="write per-kernel MFMA busy and clock from a rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES "
                         "GRBM_GUI_ACTIVE SQ_BUSY_CU_CYCLES run and exit")
    ap.add_argument("--hbm-summary", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "OUT"),
                    help="write per-kernel HBM bytes from rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE runs of a "
                         "command with --calibrate-copy and exit")
    ap.add_argument("--cmd", default="", help="the profiled command, recorded in a summary")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# HBM traffic of the dominant kernels from rocprofv3 counters

def source_hash(name):
    with open(os.path.join(CSRC, name), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def pmc_means(run_dir, counter):
    """Per-dispatch mean of `counter` for each dominant kernel and for the
    calibration copy, from a rocprofv3 --pmc csv run directory."""
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    vals = {k: {} for k in list(DOMINANT) + ["copy"]}
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            key = next((k for k, d in DOMINANT.items() if d["kernel"] in name), None)
            if key is None and COPY_KERNEL in name:
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
        out[k] = (sum(v) / len(v), len(v))
    return out


def write_traffic_summaries(fetch_dir, write_dir):
    """HBM bytes per launch of each dominant kernel: FETCH_SIZE and WRITE_SIZE
    (KiB per dispatch) scaled by what they read for a copy of known size."""
    fe = pmc_means(fetch_dir, "FETCH_SIZE")
    wr = pmc_means(write_dir, "WRITE_SIZE")
    f_fetch = COPY_BYTES / (fe["copy"][0] * 1024.0)
    f_write = COPY_BYTES / (wr["copy"][0] * 1024.0)
    for key, d in DOMINANT.items():
        fetch_b = fe[key][0] * 1024.0 * f_fetch
        write_b = wr[key][0] * 1024.0 * f_write
        lines = [
            f"# HBM traffic per launch of the {key} dominant kernel of {HEADLINE} ({d['family']})",
            f"# kernel: {d['kernel']} ({fe[key][1]} dispatches averaged)",
            "# cd /tmp && export TMPDIR=/tmp && cd <repo> && rocprofv3 --pmc FETCH_SIZE (then WRITE_SIZE) -d <dir> "
            "--output-format csv -- python3 bench.py --only-headline --no-cpu-baseline --steps 1 --warmup 0 "
            "--decode-steps 8 --calibrate-copy",
            f"# calibration: a plain copy of {COPY_BYTES} bytes reads {fe['copy'][0]:.0f} KiB FETCH_SIZE and "
            f"{wr['copy'][0]:.0f} KiB WRITE_SIZE",
            f"source={d['source']}",
            f"source_sha={source_hash(d['source'])}",
            f"fetch_kib_raw={fe[key][0]:.1f}",
            f"write_kib_raw={wr[key][0]:.1f}",
            f"fetch_factor={f_fetch:.4f}",
            f"write_factor={f_write:.4f}",
            f"fetch_bytes={fetch_b:.0f}",
            f"write_bytes={write_b:.0f}",
            f"traffic_bytes={fetch_b + write_b:.0f}",
        ]
        with open(os.path.join(PROFILES, d["file"]), "w") as f:
            f.write("\n".join(lines) + "\n")
        print("\n".join(lines))


def short_name(name):
    """Kernel name without the namespace, return type and parameter list."""
    n = name.strip('"')
    for pre in ("void ", "sas::"):
        if n.startswith(pre):
            n = n[len(pre):]
    depth = 0
    for i, ch in enumerate(n):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return n[:i]
    return n


def _csv(run_dir, suffix):
    files = sorted(glob.glob(os.path.join(run_dir, "**", "*" + suffix), recursive=True))
    if not files:
        raise SystemExit(f"no *{suffix} under {run_dir}")
    rows = []
    for f in files:
        rows += list(csv.DictReader(open(f)))
    return rows


def _summary_head(title, cmd):
    return [f"# {title}", "", "Command (from the repository root, after `cd /tmp && export TMPDIR=/tmp`):", "",
            "```", cmd or "(not recorded)", "```", ""]


def write_trace_summary(run_dir, out, cmd, top=40):
    """Per-kernel calls and durations from rocprofv3 --stats (kernel_stats.csv)."""
    rows = _csv(run_dir, "kernel_stats.csv")
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    tot = sum(float(r["TotalDurationNs"]) for r in rows)
    lines = _summary_head("rocprofv3 --kernel-trace --stats: kernel durations", cmd)
    lines += ["| kernel | calls | avg us | min us | max us | total ms | share |", "|---|---:|---:|---:|---:|---:|---:|"]
    for r in rows[:top]:
        lines.append(f"| `{short_name(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.3f} | {float(r['TotalDurationNs']) / tot:.1%} |")
    if len(rows) > top:
        rest = sum(float(r["TotalDurationNs"]) for r in rows[top:])
        lines.append(f"| ({len(rows) - top} more kernels) | | | | | {rest / 1e6:.3f} | {rest / tot:.1%} |")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter_means(run_dir, peak=False):
    """{kernel: {counter: mean per dispatch}} (with peak: the largest
    dispatch's value), dispatch counts and mean durations (ns)."""
    vals, disp, dur = {}, {}, {}
    for r in _csv(run_dir, "counter_collection.csv"):
        k = short_name(r["Kernel_Name"])
        d = vals.setdefault(k, {}).setdefault(r["Counter_Name"], {})
        d[r["Dispatch_Id"]] = d.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
        disp.setdefault(k, set()).add(r["Dispatch_Id"])
        if r.get("Start_Timestamp") and r.get("End_Timestamp"):
            dur.setdefault(k, {})[r["Dispatch_Id"]] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    agg = (lambda d: max(d.values())) if peak else (lambda d: sum(d.values()) / len(d))
    means = {k: {c: agg(d) for c, d in cs.items()} for k, cs in vals.items()}
    return means, {k: len(v) for k, v in disp.items()}, {k: sum(v.values()) / len(v) for k, v in dur.items()}


N_SIMD = 1024   # 256 compute units x 4 SIMDs
N_XCD = 8


def write_mfma_summary(run_dir, out, cmd, min_busy=1e6):
    """MFMA busy fraction and shader clock per kernel.  GRBM_GUI_ACTIVE is
    summed over the 8 XCDs (per-XCD cycles = value / 8) and
    SQ_VALU_MFMA_BUSY_CYCLES over all SIMDs, so busy = MFMA / (1024 x
    GUI / 8); the clock is the per-XCD cycles over the dispatch duration."""
    means, n, dur = _counter_means(run_dir)
    lines = _summary_head("rocprofv3 --pmc: MFMA busy and clock per kernel", cmd)
    lines += ["MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE / 8 XCDs); "
              "clock = (GRBM_GUI_ACTIVE / 8) / duration.", "",
              "| kernel | dispatches | avg us | clock GHz | MFMA busy | CU busy |", "|---|---:|---:|---:|---:|---:|"]
    rows = [(k, m) for k, m in means.items() if m.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) >= min_busy]
    rows.sort(key=lambda km: -km[1].get("SQ_VALU_MFMA_BUSY_CYCLES", 0) * n[km[0]])
    for k, m in rows:
        gui = m.get("GRBM_GUI_ACTIVE", 0.0) / N_XCD
        busy = m["SQ_VALU_MFMA_BUSY_CYCLES"] / (N_SIMD * gui) if gui else float("nan")
        cu = m.get("SQ_BUSY_CU_CYCLES", 0.0) / (256 * gui) if gui else float("nan")
        us = dur.get(k, 0.0) / 1e3
        ghz = gui / (us * 1e3) if us else float("nan")
        lines.append(f"| `{k}` | {n[k]} | {us:.1f} | {ghz:.2f} | {busy:.1%} | {cu:.1%} |")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def write_hbm_summary(fetch_dir, write_dir, out, cmd, min_kib=64.0):
    """HBM bytes per dispatch per kernel: FETCH_SIZE and WRITE_SIZE (KiB)
    scaled by what they read for the plain copy of COPY_BYTES."""
    fe, nf, dur = _counter_means(fetch_dir)
    wr, _, _ = _counter_means(write_dir)
    # the calibration copy: the largest dispatch of a copy kernel
    cpf, cpw = _counter_means(fetch_dir, peak=True)[0], _counter_means(write_dir, peak=True)[0]
    copies = [k for k in fe if COPY_KERNEL in k]
    cf = max((cpf[k]["FETCH_SIZE"] for k in copies), default=0.0)
    cw = max((cpw[k]["WRITE_SIZE"] for k in copies if k in cpw), default=0.0)
    if not cf or not cw:
        raise SystemExit("no calibration copy found (run the command with --calibrate-copy)")
    ff, fw = COPY_BYTES / (cf * 1024.0), COPY_BYTES / (cw * 1024.0)
    lines = _summary_head("rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE: HBM bytes per dispatch", cmd)
    lines += [f"Calibration: a plain copy of {COPY_BYTES} bytes reads FETCH_SIZE {cf:.0f} KiB and WRITE_SIZE "
              f"{cw:.0f} KiB, so the factors are {ff:.4f} (fetch) and {fw:.4f} (write).  The duration is that "
              "of the FETCH_SIZE run (counters serialise the dispatches).", "",
              "| kernel | dispatches | avg us | fetch MB | write MB | HBM MB | GB/s |", "|---|---:|---:|---:|---:|---:|---:|"]
    rows = [k for k in fe if k not in copies and fe[k].get("FETCH_SIZE", 0) >= min_kib]
    rows.sort(key=lambda k: -fe[k]["FETCH_SIZE"] * nf[k])
    for k in rows:
        fb = fe[k]["FETCH_SIZE"] * 1024.0 * ff
        wb = wr.get(k, {}).get("WRITE_SIZE", 0.0) * 1024.0 * fw
        us = dur.get(k, 0.0) / 1e3
        gbs = (fb + wb) / (us * 1e3) if us else float("nan")
        lines.append(f"| `{k}` | {nf[k]} | {us:.1f} | {fb / 1e6:.1f} | {wb / 1e6:.1f} | {(fb + wb) / 1e6:.1f} | "
                     f"{gbs:.0f} |")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def stored_traffic(key):
    """HBM bytes per launch from the committed counter summary, or None when
    the kernel's source changed since the counters were taken."""
    d = DOMINANT[key]
    try:
        kv = dict(l.strip().split("=", 1) for l in open(os.path.join(PROFILES, d["file"]))
                  if "=" in l and not l.startswith("#"))
    except OSError:
        return None
    if kv.get("source_sha") != source_hash(d["source"]):
        return None
    return int(float(kv["traffic_bytes"]))


# ---------------------------------------------------------------------------

def family_means(recs):
    fam = {}
    for name, t in recs:
        fam.setdefault(name, []).append(t)
    return {k: sum(v) / len(v) for k, v in fam.items()}, {k: len(v) for k, v in fam.items()}


def decode_bytes(w, t_first, steps, batch=None):
    """Algorithmic HBM bytes of `steps` decode steps of the stack starting at
    position t_first: every layer's weights, the kept K/V (current block +
    min(K, C_t) blocks), the summaries scored, the appended K/V; the LM head
    and the embedding rows."""
    B, K, dh, Hkv, L = w.block_size, w.top_k, w.head_dim, w.n_kv_heads, w.n_layers
    b = batch or w.batch
    tot = 0.0
    for t in range(t_first, t_first + steps):
        ct = t // B
        kept = B * min(K, ct) + (t % B) + 1
        per_layer = 2.0 * w.linear_params() + b * Hkv * (kept * dh * 2 * 2 + ct * dh * 2 + 2 * dh * 2)
        tot += L * per_layer + 2.0 * w.vocab * w.d_model + b * w.d_model * 2
    return tot


def headline(args):
    """The serving job: timed steps of (prefill + 256 decode steps)."""
    import torch
    from paper_2609_13141_amd import configs, inputs, model, sas
    w = configs.BY_NAME[HEADLINE]
    dev = "cuda:0"
    L, T, nd = w.n_layers, w.tokens, args.decode_steps or w.decode_steps
    layers = [inputs.layer_weights_device(w, layer=l, device=dev) for l in range(L)]
    ends = inputs.model_ends_device(w, device=dev)
    st = model.Stack(w, layers, ends, max_len=w.seq_len + nd + 8, device=dev)
    # the decode positions 2048 .. 2303 of every step
    positions = [torch.full((w.batch,), w.seq_len + s, dtype=torch.int32, device=dev) for s in range(nd)]

    def one_step(dec_sample=0):
        """Prefill then the decode steps; returns the events bracketing the prefill."""
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if dec_sample:
            sas.profiler_select([DOMINANT["prefill"]["family"]])
        e0.record()
        tok = st.prefill(ends["token_ids"], ends["img_embed"])
        e1.record()
        for s, p in enumerate(positions):
            if dec_sample:
                sas.profiler_select([DOMINANT["decode"]["family"]] if s % dec_sample == 0 else [])
            tok, _, _ = st.step(tok, p)
        return e0, e1

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    per_step = L + L * ((nd + DECODE_SAMPLE - 1) // DECODE_SAMPLE) + 8
    sas.profiler_start(per_step * args.steps + 64)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs = [one_step(DECODE_SAMPLE) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    recs = sas.profiler_stop()
    sas.profiler_select(None)
    ms = (t1 - t0) * 1e3 / args.steps
    pre_ms = sum(a.elapsed_time(b) for a, b in evs) / args.steps
    dec_ms = (ms - pre_ms) / nd
    kms, kcnt = family_means(recs)

    # prefill: value and the gate/up GEMM's roofline
    tok_s_layer = T / (pre_ms * 1e-3 / L)
    pre_flops = w.prefill_flops("dense")
    pre_tf = pre_flops / (pre_ms * 1e-3 / L) / 1e12
    gu = DOMINANT["prefill"]["family"]
    gu_flops = 2.0 * T * w.d_model * 2 * w.d_ff
    gu_tf = gu_flops / (kms[gu] * 1e-3) / 1e12
    # decode: HBM bytes and the gate/up GEMV's roofline (weights + activations in, activations out)
    nbytes = decode_bytes(w, w.seq_len, nd) / nd
    dgu = DOMINANT["decode"]["family"]
    dgu_bytes = 2.0 * w.d_model * 2 * w.d_ff + w.batch * (w.d_model + w.d_ff) * 2
    dgu_gbs = dgu_bytes / (kms[dgu] * 1e-3) / 1e9
    att_alg = 4.0 * w.head_dim * w.n_heads * w.batch * w.attended_pairs("dense")
    nq = -(-w.seq_len // 128)
    att_exec = sum(4.0 * w.head_dim * 128 * 64 * min(2 * q + 2, -(-w.seq_len // 64)) for q in range(nq)) \
        * w.n_heads * w.batch

    # per-kernel view: one more step with every launch timed (not part of the timed region)
    sas.profiler_start(64 * L * 4 + 256)
    tok = st.prefill(ends["token_ids"], ends["img_embed"])
    for p in positions[:4]:
        tok, _, _ = st.step(tok, p)
    recs = sas.profiler_stop()
    kall, kall_n = family_means(recs)
    yard = hipblaslt_yardstick(w, dev)
    out = {
        "value": round(tok_s_layer, 1),
        "ms_per_step": round(ms, 3),
        "prefill_ms_per_step": round(pre_ms, 3),
        "prefill_ms_per_layer": round(pre_ms / L, 4),
        "alg_tflops": round(pre_tf, 1),
        "mfma_frac": round(pre_tf / BF16_PEAK_TFLOPS, 4),
        "attention": {"alg_gflop_per_layer": round(att_alg / 1e9, 2), "executed_gflop_per_layer": round(att_exec / 1e9, 2),
                      "ms_per_layer": round(kall.get("attention", 0.0), 4),
                      "alg_tflops": round(att_alg / (kall.get("attention", 1e9) * 1e-3) / 1e12, 1),
                      "executed_tflops": round(att_exec / (kall.get("attention", 1e9) * 1e-3) / 1e12, 1)},
        "roofline": {"bound": "mfma", "kernel": gu, "achieved": round(gu_tf, 1), "peak": BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(gu_tf / BF16_PEAK_TFLOPS, 4), "traffic": stored_traffic("prefill"),
                     "traffic_source": "profiles/" + DOMINANT["prefill"]["file"],
                     "alg_gflop_per_launch": round(gu_flops / 1e9, 1), "avg_ms": round(kms[gu], 4),
                     "launches_timed": kcnt[gu]},
        "decode": {
            "workload": f"{w.name}: {L} layers, batch {w.batch}, positions {w.seq_len}..{w.seq_len + nd - 1} "
                        f"after the prompt, pages of {w.page_size}, B={w.block_size}, K={w.top_k}, greedy",
            "steps_per_step": nd,
            "ms_per_step": round(dec_ms, 4),
            "tokens_per_s": round(w.batch / (dec_ms * 1e-3), 1),
            "ms_per_layer_step": round(dec_ms / L, 4),
            "bytes_per_step": int(nbytes),
            "hbm_gbs": round(nbytes / (dec_ms * 1e-3) / 1e9, 1),
            "hbm_frac": round(nbytes / (dec_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "roofline": {"bound": "hbm", "kernel": dgu, "achieved": round(dgu_gbs, 1), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(dgu_gbs / HBM_PEAK_GBS, 4),
                         "traffic": stored_traffic("decode"),
                         "traffic_source": "profiles/" + DOMINANT["decode"]["file"],
                         "alg_bytes_per_launch": int(dgu_bytes), "avg_ms": round(kms[dgu], 4),
                         "launches_timed": kcnt[dgu]},
        },
        "kernels_ms": {k: round(v, 4) for k, v in sorted(kall.items(), key=lambda kv: -kv[1] * kall_n[kv[0]])},
        "kernel_calls": kall_n,
        "yardstick_hipblaslt_ms": {k: round(v, 4) for k, v in yard.items()},
    }
    del st, layers
    return w, ends, out


def hipblaslt_yardstick(w, dev, reps=10, copies=4):
    """An outside yardstick for the prefill GEMMs: torch's bf16 linear
    (hipBLASLt) at the same shapes (M = the prefill's tokens), plain
    products without the fused epilogues, cycling over `copies` weight
    buffers so that the weights stream from HBM as in a layer."""
    import torch
    T = w.tokens
    shapes = (("gemm_qkv", (w.n_heads + 2 * w.n_kv_heads) * w.head_dim, w.d_model),
              ("gemm_o", w.d_model, w.n_heads * w.head_dim),
              ("gemm_gate_up", 2 * w.d_ff, w.d_model),
              ("gemm_down", w.d_model, w.d_ff))
    out = {}
    for fam, N, K in shapes:
        A = torch.randn(T, K, device=dev).to(torch.bfloat16)
        Ws = [(torch.randn(N, K, device=dev) * 0.02).to(torch.bfloat16) for _ in range(copies)]
        for i in range(3):
            torch.nn.functional.linear(A, Ws[i % copies])
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for i in range(reps):
            torch.nn.functional.linear(A, Ws[i % copies])
        e1.record()
        torch.cuda.synchronize()
        out[fam] = e0.elapsed_time(e1) / reps
        del A, Ws
    torch.cuda.empty_cache()
    return out


def attention_executed_flops(w, sel):
    """MFMA work the attention kernel executes: every job (128 rows: 128 / G
    consecutive positions x the G heads of one kv group) multiplies whole
    64-key tiles, those holding any key one of its rows attends (the selected
    blocks of any of the tile's positions and the current blocks up to the
    tile's last position).  sel [b, Hkv, n, K]."""
    import numpy as np
    b, Hkv, n, K = sel.shape
    B, G, dh = w.block_size, w.n_heads // w.n_kv_heads, w.head_dim
    qpt = 128 // G
    tiles = 0
    for q0 in range(0, n, qpt):
        q1 = min(n, q0 + qpt)
        rows = sel[:, :, q0:q1, :].reshape(b, Hkv, -1)
        for bi in range(b):
            for g in range(Hkv):
                blk = np.unique(rows[bi, g])
                blk = blk[blk >= 0]
                keys = set()
                for m in blk.tolist():
                    keys.update(range(m * B // 64, ((m + 1) * B - 1) // 64 + 1))
                keys.update(range((q0 // B) * B // 64, (q1 - 1) // 64 + 1))   # current blocks (causal)
                tiles += len(keys)
    return 4.0 * dh * 128 * 64 * tiles


def layer_bench(name, steps=30, warmup=10):
    """One GATED layer forward (RMSNorm, QKV + RoPE, summaries, selector and
    Top-K, gated block-sparse attention, O + residual, MLP) of a workload."""
    import numpy as np
    import torch
    from paper_2609_13141_amd import configs, inputs, sas
    w = configs.BY_NAME[name]
    dev = "cuda:0"
    x = sas.to_device(inputs.embeddings(w), "bf16", dev)
    W = inputs.layer_weights_device(w, device=dev)
    cfg = sas.make_config(w)
    ws = sas.Workspace(dev)

    def run():
        return sas.layer_forward(cfg, x, W, stats=False, ws=ws)
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        run()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    sas.profiler_start(64 * 5 + 64)
    for _ in range(5):
        run()
    recs = sas.profiler_stop()
    kms, kn = family_means(recs)
    sel = sas.layer_forward(cfg, x, W, stats=True, lse=False, sel_idx=True, ws=ws)["sel_idx"].cpu().numpy()
    flops = w.prefill_flops()
    att_alg = 4.0 * w.head_dim * w.n_heads * w.batch * w.attended_pairs()
    att_exec = attention_executed_flops(w, sel)
    att_ms = kms["attention"]
    tf = flops / (ms * 1e-3) / 1e12
    del x, W, ws
    return {"workload": f"{w.name}: batch {w.batch}, {w.seq_len} tokens, {w.n_heads}/{w.n_kv_heads} heads, "
                        f"d={w.d_model}, d_ff={w.d_ff}, B={w.block_size}, K={w.top_k}, GATED",
            "ms_per_layer": round(ms, 4), "tokens_per_s": round(w.tokens / (ms * 1e-3), 1),
            "alg_gflop": round(flops / 1e9, 1), "alg_tflops": round(tf, 1),
            "mfma_frac": round(tf / BF16_PEAK_TFLOPS, 4),
            "attention": {"alg_gflop": round(att_alg / 1e9, 2), "executed_gflop": round(att_exec / 1e9, 2),
                          "ms": round(att_ms, 4), "alg_tflops": round(att_alg / (att_ms * 1e-3) / 1e12, 1),
                          "executed_tflops": round(att_exec / (att_ms * 1e-3) / 1e12, 1),
                          "executed_frac": round(att_exec / (att_ms * 1e-3) / 1e12 / BF16_PEAK_TFLOPS, 4)},
            "kernels_ms": {k: round(v, 4) for k, v in sorted(kms.items(), key=lambda kv: -kv[1] * kn[kv[0]])}}


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
            kms, _ = family_means(recs)
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
        kms, _ = family_means(recs)
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
    kms, _ = family_means(recs)
    flops = 2.0 * dh * H * b * n * (n + 1) / 2
    inter, tot, rec = sas.overlap_recall(su, ru)
    return {"workload": f"{w.name}: batch {b}, {n} tokens, {H}/{Hkv} heads, dh {dh}, B={w.block_size}, K={w.top_k}",
            "ms_per_layer": round(ms, 4), "pass_gflop": round(flops / 1e9, 2),
            "pass_tflops": round(flops / (kms["stats"] * 1e-3) / 1e12, 1),
            "recall_random_inputs": round(rec, 4),
            "kernels_ms": {kk: round(vv, 4) for kk, vv in sorted(kms.items(), key=lambda kv: -kv[1])}}


def cpu_baseline(w, ends, cores, n_layers=8):
    """The fp64 oracle, as it stands, on a bounded sample of the headline
    prefill: the first `n_layers` DENSE layers of one 2048-token sequence,
    with the stack's own weights copied to the host."""
    import numpy as np
    import torch

    import oracle
    from oracle.layer import Spec
    from paper_2609_13141_amd import inputs
    try:
        from threadpoolctl import threadpool_info
        used = max([p.get("num_threads", 1) for p in threadpool_info()] or [cores])
    except Exception:
        used = cores
    spec = Spec(w.n_heads, w.n_kv_heads, w.head_dim, w.block_size, w.top_k, "dense", w.dtype, w.rope_base,
                w.rms_eps)
    ids = ends["token_ids"][:1].cpu().numpy()
    n_img = int((ids < 0).sum())
    table = ends["embed"].float().cpu().numpy()
    x = oracle.embed_tokens(ids, table, ends["img_embed"][:1, :n_img].float().cpu().numpy())[0]
    del table
    Ws = []
    for l in range(n_layers):
        Wd = inputs.layer_weights_device(w, layer=l, device="cuda:0")
        Ws.append({k: (None if v is None else v.float().cpu().numpy().astype(np.float64)) for k, v in Wd.items()})
        del Wd
    torch.cuda.empty_cache()
    t0 = time.perf_counter()
    for l in range(n_layers):
        x = oracle.dense_prefill_layer(x, Ws[l], spec)["y"]
    dt = time.perf_counter() - t0
    return {"value": round(w.seq_len * n_layers / dt, 2), "unit": "tokens/s/layer", "cores": int(used),
            "kind": "oracle",
            "sample": f"the first {n_layers} DENSE prefill layers of one {w.seq_len}-token sequence of {w.name} "
                      f"(every row), fp64 NumPy, {dt:.2f} s"}


def main():
    args = parse()
    if args.pmc_summary:
        write_traffic_summaries(*args.pmc_summary)
        return
    if args.trace_summary:
        write_trace_summary(*args.trace_summary, args.cmd)
        return
    if args.mfma_summary:
        write_mfma_summary(*args.mfma_summary, args.cmd)
        return
    if args.hbm_summary:
        write_hbm_summary(*args.hbm_summary, args.cmd)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the SAS hot path here is single-GPU "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    cores = args.cpu_threads or min(16, len(os.sched_getaffinity(0)))
    for var in ("OPENBLAS_NUM_THREADS", "OMP_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = str(cores)

    import torch

    sys.path.insert(0, HERE)
    torch.cuda.set_device(0)
    if args.only_layer:
        print(json.dumps({"layer": layer_bench(args.only_layer)}), flush=True)
        return
    w, ends, head = headline(args)
    line = {
        "metric": METRIC,
        "value": head.pop("value"),
        "unit": "tokens/s/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded prompt ids + N(0,1)*2 image embeddings, N(0,1) embedding table, N(0,0.02) "
                "weights drawn on the GPU)",
        "config": {"workload": w.name, "batch": w.batch, "seq_len": w.seq_len, "n_layers": w.n_layers,
                   "decode_steps": args.decode_steps or w.decode_steps, "d_model": w.d_model, "n_heads": w.n_heads,
                   "n_kv_heads": w.n_kv_heads, "head_dim": w.head_dim, "d_ff": w.d_ff, "vocab": w.vocab,
                   "prefill_mode": "dense", "decode_mode": "sparse", "block_size": w.block_size,
                   "top_k": w.top_k, "page_size": w.page_size},
    }
    line.update(head)
    if args.calibrate_copy:
        # same dtype, contiguous: torch issues a device-to-device copy, which the
        # runtime runs as its blit kernel (the one the counter summaries look for)
        src = torch.empty(COPY_BYTES // 2, dtype=torch.bfloat16, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    torch.cuda.empty_cache()
    if not args.only_headline:
        if not args.no_layers:
            line["layers"] = [layer_bench(nm) for nm in ("7b_layer_1k", "7b_layer_4k_b4", "gqa28x4_layer_16k")]
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
        line["cpu_baseline"] = cpu_baseline(w, ends, cores)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
