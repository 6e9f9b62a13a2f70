"""Benchmark of one speculative-verify step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c2_7b_greedy]

A step is one pass of the whole hot path for one batch of synthetic input:
spade_verify (embedding, every decoder layer, LM head, softmax, accept /
reject, correction draw) + spade_kv_commit, followed by a device-side restore
of the request lengths so every step verifies the same configuration.  The
default workload is the Llama-7B-shaped bf16 verifier (32 layers, d_model
4096, 32 heads x 128, SwiGLU 11008, vocab 32000), batch 1, 1024 cached tokens,
gamma = 5, greedy, weights N(0, 0.02) from a seed.

Printed: one JSON line with verified draft tokens/s (B * gamma / step time),
the step latency, the whole-pass algorithmic bytes and their rate against the
8 TB/s HBM peak, the dominant kernel's roofline (HIP events around that
kernel alone, same launch configuration), and the CPU oracle timed on a
bounded sample of the same workload.
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

HBM_PEAK_GBS = 8000.0


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_bytes(w, lens) -> dict:
    """Bytes one verify pass must move at minimum: every weight matrix and
    gain once, the M gathered embedding rows, the cached K/V of every request
    read once, the new K/V rows written once, the q rows of sampling
    requests (their draft tokens' entries and the residual row)."""
    m = w.model
    elt = 2 if m.weight_dtype == "bf16" else 4
    kvelt = 2 if m.kv_dtype == "bf16" else 4
    d, f, v, L = m.d_model, m.d_ffn, m.vocab, m.n_layers
    dkv = m.kv_heads * m.head_dim  # K/V width (grouped-query attention: fewer K/V heads)
    R = w.gamma + 1
    M = w.batch * R
    weights = L * (2 * d * d + 2 * d * dkv + 3 * d * f) * elt + L * 2 * d * 4 + v * d * elt + d * 4
    embed = M * d * elt
    kv_read = sum(int(l) + R for l in lens) * L * 2 * dkv * kvelt
    kv_write = M * L * 2 * dkv * kvelt
    return {"weights": weights, "embed": embed, "kv_read": kv_read, "kv_write": kv_write,
            "total": weights + embed + kv_read + kv_write}


def cpu_baseline(w, inp, layers: int) -> dict:
    """The oracle, unchanged, on the first `layers` decoder layers of the same
    model (same weights, same cached context, same rows), scaled to all
    layers; the LM head and accept/reject are timed in full."""
    from oracle import Decoder
    from oracle import verify as oracle_verify
    from synth import ModelWeights
    m = w.model
    part = m.__class__(**{**m.__dict__, "n_layers": layers})
    mw = ModelWeights(m, w.seed)
    dec = Decoder(part, mw.get, keep_f64=True)
    b = 0
    cache = dec.new_cache(int(inp.lens[b]) + w.gamma + 2)
    t0 = time.perf_counter()
    dec.prefill(cache, inp.prompts[b][:-1])
    t_prefill = time.perf_counter() - t0
    # warm the converted weights, then time the verify pass
    reps = []
    for _ in range(3):
        c = cache.copy()
        t0 = time.perf_counter()
        oracle_verify(dec, c, inp.pending[b], inp.drafts[b], None, inp.uniforms[b], int(inp.modes[b]))
        reps.append(time.perf_counter() - t0)
    t_part = float(np.median(reps))
    # LM head + accept share: time the last-stage alone (x -> logits -> accept)
    t0 = time.perf_counter()
    lm = dec.w("lm_head")
    h = np.random.default_rng(0).standard_normal((w.gamma + 1, m.d_model))
    for _ in range(3):
        _ = h @ lm.T
    t_lm = (time.perf_counter() - t0) / 3
    t_layers = max(t_part - t_lm, 1e-9)
    t_full = t_layers * m.n_layers / layers + t_lm
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count()
    threads = int(os.environ.get("OMP_NUM_THREADS", cores))
    mw.close()
    return {"value": round(w.batch * w.gamma / t_full, 3), "unit": "draft tokens/s", "cores": min(cores, threads),
            "kind": "oracle",
            "sample": f"float64 NumPy oracle verify of batch 1 over the first {layers} of {m.n_layers} layers "
                      f"(median of 3, prefill of {int(inp.lens[b])} tokens excluded, weights pre-converted), "
                      f"scaled by {m.n_layers}/{layers}, plus the LM head",
            "latency_us": round(t_full * 1e6, 1), "prefill_s_sample": round(t_prefill, 2)}


COUNTER_FILE = os.path.join(ROOT, "profiles", "gu_gemm_hbm_traffic.txt")
COPY_BYTES = 256 << 20  # the calibration copy reads and writes this many bytes


def gemm_source_digest() -> str:
    """Digest of the sources the gate/up GEMM kernel is built from."""
    import hashlib
    h = hashlib.sha256()
    for f in ("device_util.h", "device_gemm.h", "kernels.hip"):
        with open(os.path.join(ROOT, "paper_2608_13076_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def read_traffic():
    """Measured HBM bytes per gate/up launch from the committed counter
    summary, or None if it is missing or the kernel sources changed since."""
    try:
        txt = open(COUNTER_FILE).read()
    except OSError:
        return None
    vals = dict(line.split(":", 1) for line in txt.splitlines() if line.startswith(("traffic_bytes", "source_digest")))
    if vals.get("source_digest", "").strip() != gemm_source_digest():
        return None
    return int(vals["traffic_bytes"].strip())


def summarize_counters(fetch_dir: str, write_dir: str, cmd_fetch: str, cmd_write: str) -> int:
    """FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the calibration copy and of
    the gate/up GEMM launches from two rocprofv3 --pmc runs of --counters; the
    copy's known bytes give the scale of each counter."""
    import csv
    import glob

    def per_kernel(d, counter):
        f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        acc = {}
        for r in csv.DictReader(open(f)):
            if r.get("Counter_Name") != counter:
                continue
            name = r["Kernel_Name"]
            key = "copy" if "neg" in name else ("gu" if "gemm_kernel" in name else None)
            if key:
                acc.setdefault(key, []).append(float(r["Counter_Value"]))
        return {k: (sum(v) / len(v), len(v)) for k, v in acc.items()}

    fe = per_kernel(fetch_dir, "FETCH_SIZE")
    wr = per_kernel(write_dir, "WRITE_SIZE")
    f_fetch = COPY_BYTES / fe["copy"][0]
    f_write = COPY_BYTES / wr["copy"][0]
    traffic = int(round(fe["gu"][0] * f_fetch + wr["gu"][0] * f_write))
    with open(COUNTER_FILE, "w") as f:
        f.write("# HBM traffic of the gate/up GEMM launch (7B, batch 1, gamma 5)\n\n")
        f.write("Two rocprofv3 counter runs of `bench.py --counters` (a calibration copy of a known size,\n"
                "then the gate/up GEMM launches of the measurement hook), from the repository root:\n\n")
        f.write(f"    {cmd_fetch}\n    {cmd_write}\n\n")
        f.write("| kernel | FETCH_SIZE (KiB/dispatch) | WRITE_SIZE (KiB/dispatch) | dispatches |\n|---|---|---|---|\n")
        f.write(f"| calibration copy ({COPY_BYTES} B read, {COPY_BYTES} B written) | {fe['copy'][0]:.1f} | "
                f"{wr['copy'][0]:.1f} | {fe['copy'][1]} |\n")
        f.write(f"| gate/up GEMM | {fe['gu'][0]:.1f} | {wr['gu'][0]:.1f} | {fe['gu'][1]} |\n\n")
        f.write(f"Scale (bytes per counter unit): fetch {f_fetch:.2f}, write {f_write:.2f}.\n\n")
        f.write(f"traffic_bytes: {traffic}\n")
        f.write(f"source_digest: {gemm_source_digest()}\n")
    print(open(COUNTER_FILE).read())
    return 0


STEP_PASSES = (("FETCH_SIZE",), ("WRITE_SIZE",),
               ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE",
                "SQ_LDS_BANK_CONFLICT", "SQ_INSTS_LDS"),
               ("TCC_HIT_sum", "TCC_MISS_sum"))
N_SIMD = 1024  # 256 compute units x 4 SIMDs
MFMA_PEAK_TFLOPS = 2500.0  # dense bf16


def kernel_alg_bytes(name: str, w, lens) -> int:
    """Algorithmic bytes of one launch of a verify-step kernel: a projection
    GEMM's weights once plus its fp32 input and output rows; the attention's
    cached and new K/V rows of one layer."""
    import re
    name = name.replace("void ", "", 1).replace("spade::", "")
    m = w.model
    d, f, v = m.d_model, m.d_ffn, m.vocab
    dkv = m.kv_heads * m.head_dim
    M = w.batch * (w.gamma + 1)
    kind = None
    t = re.search(r"<([^>]*)>", name)
    args = [a.strip() for a in t.group(1).split(",")] if t else []
    if name.startswith("gemm_wide_kernel") and len(args) >= 3:
        kind = int(args[2])
    elif name.startswith("gemm_kernel") and len(args) >= 4:
        kind = int(args[3])
    elif name.startswith("gemm_split_kernel") and len(args) >= 2:
        kind = int(args[1])
    elif name.startswith("gemm_mid_kernel") and len(args) >= 1:
        kind = int(args[0])  # the first pass; its second pass (gemm_mid_finish_kernel) counts nothing
    if kind is not None:
        n_out, k_in = [(d + 2 * dkv, d), (d, d), (2 * f, d), (d, f), (v, d)][kind]
        return n_out * k_in * 2 + M * k_in * 4 + M * (n_out // (2 if kind == 2 else 1)) * 4
    if name.startswith(("attn_lr_kernel", "attn_g_kernel", "attn_kernel")):
        return sum(int(l) + w.gamma + 1 for l in lens) * 2 * dkv * 2
    return 0


def summarize_step_counters(workload_name: str, dirs, cmds) -> int:
    """Per-kernel counters of one verify step (the dispatches after the last
    calibration copy) from the rocprofv3 --pmc passes of --counters-step."""
    import csv
    import glob
    from synth import make_inputs, workload
    w = workload(workload_name)
    inp = make_inputs(w)

    def rows(d):
        f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        return list(csv.DictReader(open(f)))

    per = {}  # kernel -> counter -> [values]
    meta = {}
    copy = {}
    for d in dirs:
        rs = rows(d)
        cut = max(int(r["Dispatch_Id"]) for r in rs if "neg" in r["Kernel_Name"])
        for r in rs:
            did = int(r["Dispatch_Id"])
            name = r["Kernel_Name"]
            val = float(r["Counter_Value"])
            if did == cut:
                copy.setdefault(r["Counter_Name"], []).append(val)
                continue
            if did < cut:
                continue
            per.setdefault(name, {}).setdefault(r["Counter_Name"], {}).setdefault(did, 0.0)
            per[name][r["Counter_Name"]][did] += val
            mm = meta.setdefault(name, {"dur": {}, "vgpr": r["VGPR_Count"], "agpr": r["Accum_VGPR_Count"],
                                        "lds": r["LDS_Block_Size"], "grid": r["Grid_Size"]})
            mm["dur"][did] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3
    f_fetch = COPY_BYTES / (sum(copy["FETCH_SIZE"]) * 1024) * 1024
    f_write = COPY_BYTES / (sum(copy["WRITE_SIZE"]) * 1024) * 1024

    def avg(name, c):
        vals = per.get(name, {}).get(c)
        return sum(vals.values()) / len(vals) if vals else None

    out = os.path.join(ROOT, "profiles", f"{workload_name}_counters.md")
    lines = [f"# Hardware counters of one verify step: {w.description}", "",
             "Four rocprofv3 counter passes of `bench.py --counters-step` (a calibration copy of "
             f"{COPY_BYTES} bytes read and written, then one verify step), from the repository root:", ""]
    lines += [f"    {c}" for c in cmds]
    lines += ["", f"Calibration: FETCH_SIZE counts {f_fetch:.1f} bytes per KiB unit, WRITE_SIZE {f_write:.1f} "
              "(HBM traffic = counter x that).  MFMA TFLOP/s = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 / duration "
              "(the matrix operations executed, both bf16 terms of each activation counted), and its fraction "
              f"of the {MFMA_PEAK_TFLOPS:.0f} TFLOP/s dense bf16 peak.  Durations are those of the counter runs "
              "(kernels serialised).  Averages per launch.", "",
              "| kernel | launches | us | alg. MB | HBM read MB | HBM write MB | traffic / alg. | HBM TB/s | "
              "MFMA TFLOP/s | MFMA frac | L2 hit | LDS bank conflicts / LDS instr | VGPRs |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    order = sorted(per, key=lambda n: -sum(meta[n]["dur"].values()))
    for name in order:
        mm = meta[name]
        n = len(mm["dur"])
        us = sum(mm["dur"].values()) / n
        alg = kernel_alg_bytes(name, w, inp.lens)
        fe = avg(name, "FETCH_SIZE")
        wr = avg(name, "WRITE_SIZE")
        rd_b = fe * f_fetch if fe is not None else None
        wr_b = wr * f_write if wr is not None else None
        mops = avg(name, "SQ_INSTS_VALU_MFMA_MOPS_BF16")
        hit = avg(name, "TCC_HIT_sum")
        miss = avg(name, "TCC_MISS_sum")
        bank = avg(name, "SQ_LDS_BANK_CONFLICT")
        ldsi = avg(name, "SQ_INSTS_LDS")

        def fmt(x, p=1):
            return "-" if x is None else f"{x:.{p}f}"
        tb = (rd_b + wr_b) / (us * 1e-6) / 1e12 if rd_b is not None and wr_b is not None else None
        ratio = (rd_b + wr_b) / alg if alg and rd_b is not None and wr_b is not None else None
        tf = mops * 512 / (us * 1e-6) / 1e12 if mops is not None else None
        mb = f"{tf / MFMA_PEAK_TFLOPS:.3f}" if tf is not None else "-"
        hr = f"{100 * hit / (hit + miss):.1f}%" if hit is not None and miss is not None and hit + miss > 0 else "-"
        lb = f"{bank / ldsi:.2f}" if bank is not None and ldsi else "-"
        short = name.replace("void ", "", 1).replace("spade::", "").split("(")[0]
        lines.append(f"| `{short}` | {n} | {us:.1f} | {fmt(alg / 1e6 if alg else None)} | {fmt(rd_b / 1e6 if rd_b else None)} | "
                     f"{fmt(wr_b / 1e6 if wr_b else None)} | {fmt(ratio, 2)} | {fmt(tb, 2)} | {fmt(tf)} | {mb} | {hr} | "
                     f"{lb} | {mm['vgpr']} |")
    lines += ["", "Kernel names: `gemm_wide_kernel<row tiles, panels per wave, kind, k-splits, non-temporal weight loads>`, "
              "`gemm_kernel<bf16, row tiles, operand in LDS, kind>`, `gemm_split_kernel<k-splits, kind>`, "
              "`gemm_mid_kernel<kind>` (its algorithmic bytes: the whole projection's; the published sums it "
              "writes and `gemm_mid_finish_kernel<kind>` reads back are traffic beyond them) with kind "
              "0 QKV, 1 O, 2 gate/up, 3 down, 4 LM head; attention kernels read one layer's K/V.", ""]
    with open(out, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))
    return 0


def prefill_flops(m, lens) -> float:
    """Dense flops of caching the prompts: 2 per weight and token for the
    projections, and 4 hd per (query, key) pair and head for the causal scores
    and weighted values (a prompt of n tokens has n (n + 1) / 2 pairs)."""
    dkv = m.kv_heads * m.head_dim
    per_tok = m.n_layers * 2 * (m.d_model * (m.d_model + 2 * dkv) + m.d_model * m.d_model + 3 * m.d_model * m.d_ffn)
    pairs = sum(int(n) * (int(n) + 1) // 2 for n in lens)
    return float(per_tok * sum(int(n) for n in lens) + m.n_layers * m.n_heads * 4 * m.head_dim * pairs)


def time_prefill(model, kv, inp, w) -> dict:
    """The same prompts again, into an empty cache (same contents and state
    afterwards), timed around the call (host to device copy of the ids and the
    final synchronisation included)."""
    import torch
    zeros = np.zeros(w.batch, dtype=np.int32)
    kv.set_state(zeros, zeros)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    kv.prefill_batch(inp.prompts)
    t = time.perf_counter() - t0
    tokens = int(sum(len(p) - 1 for p in inp.prompts))
    fl = prefill_flops(w.model, [len(p) - 1 for p in inp.prompts])
    return {"tokens": tokens, "s": round(t, 4), "tokens_per_s": round(tokens / t, 1),
            "tflops": round(fl / t / 1e12, 1), "frac_bf16_peak": round(fl / t / 1e12 / MFMA_PEAK_TFLOPS, 4)}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="c2_7b_greedy")
    ap.add_argument("--cpu-layers", type=int, default=8)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kernel-reps", type=int, default=20)
    ap.add_argument("--all-kernels", action="store_true", help="also time every other projection GEMM")
    ap.add_argument("--graph", action="store_true", help="replay the step as a captured HIP graph")
    ap.add_argument("--prefill-only", action="store_true",
                    help="time the workload's prefill only (a cold run, then a warm one) and print it as JSON")
    ap.add_argument("--counters", action="store_true",
                    help="counter-collection run: a calibration copy, then the gate/up GEMM launches; no timing")
    ap.add_argument("--summarize-counters", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "CMD_FETCH", "CMD_WRITE"),
                    help="write the HBM traffic summary from two rocprofv3 --pmc runs of --counters")
    ap.add_argument("--counters-step", action="store_true",
                    help="counter-collection run: one warm-up step, a calibration copy, one verify step; no timing")
    ap.add_argument("--summarize-step-counters", nargs=8, metavar=("D1", "D2", "D3", "D4", "C1", "C2", "C3", "C4"),
                    help="write profiles/<workload>_counters.md from the four rocprofv3 --pmc passes of "
                         "--counters-step (output dirs, then the commands)")
    args = ap.parse_args()
    if args.summarize_counters:
        return summarize_counters(*args.summarize_counters)
    if args.summarize_step_counters:
        a = args.summarize_step_counters
        return summarize_step_counters(args.workload, a[:4], a[4:])
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark measures one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        print("bench.py: only --gpus 1 is supported (one GPU)", file=sys.stderr)
        return 2

    import torch
    from paper_2608_13076_amd import spade
    from synth import iter_weights, make_inputs, workload
    from tests.golden.drafts import load_drafts

    w = workload(args.workload)
    m = w.model
    inp = make_inputs(w)
    drafts_src = load_drafts(w, inp)
    log(f"workload {w.name}: {w.description}; drafts: {drafts_src}")

    R = w.gamma + 1
    max_len = int(inp.lens.max()) + 2 * R + 8
    model = spade.Model(m, w.batch, w.gamma, max_len)
    t0 = time.perf_counter()
    for kind, layer, arr in iter_weights(m, w.seed):
        model.load_numpy(kind, layer, arr)
    log(f"weights generated + loaded in {time.perf_counter() - t0:.1f}s "
        f"({model.weight_bytes() / 1e9:.2f} GB arena)")
    kv = spade.KVCache(model, w.batch, max_len)
    if args.counters:
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)  # calibration: reads and writes COPY_BYTES
        torch.cuda.synchronize()
        _check = spade._check
        _check(model.lib.spade_profile_gemm(model.handle, kv.handle, spade.GEMM_KINDS["gu"], w.batch, w.gamma,
                                            4, spade._stream()))
        torch.cuda.synchronize()
        log("counter run done: 1 calibration copy, 4 gate/up launches")
        return 0
    if args.prefill_only:
        kv.prefill_batch(inp.prompts)  # cold: first launches, code loading
        pf = time_prefill(model, kv, inp, w)
        log(f"prefill (warm): {pf}")
        if model.device_error() != 0:
            log("device error word set")
            return 1
        print(json.dumps({"workload": w.name, "prefill": pf,
                          "prompt_tokens": [len(p) - 1 for p in inp.prompts]}), flush=True)
        return 0
    t0 = time.perf_counter()
    if args.counters_step:
        # the cache's contents do not change what the counters measure: set the
        # lengths directly (a zero-filled cache) instead of prefilling
        kv.buf.zero_()
        kv.set_state(inp.lens, inp.pending)
    else:
        kv.prefill_batch(inp.prompts)  # all requests' chunks in one forward each
    log(f"prefill of {inp.lens.tolist()} tokens in {time.perf_counter() - t0:.1f}s")
    prefill = None
    if not args.counters_step:
        prefill = time_prefill(model, kv, inp, w)
        log(f"prefill (warm): {prefill}")
    lens0, pend0 = kv.snapshot(w.batch)
    buf = spade.VerifyBuffers(model, inp.drafts, inp.draft_probs, inp.uniforms, inp.modes, want_logits=False)

    def step():
        spade.verify(model, kv, buf, inp.temperature)
        kv.commit(buf.n, buf.corr)
        kv.restore(lens0, pend0)

    if args.counters_step:
        step()
        torch.cuda.synchronize()
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)  # calibration (and the marker before the measured step)
        torch.cuda.synchronize()
        step()
        torch.cuda.synchronize()
        log("counter run done: 1 warm-up step, 1 calibration copy, 1 step")
        return 0
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run = step
    if args.graph:
        # capture one step (all launches are stream-ordered kernels) and replay it
        graph = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            with torch.cuda.graph(graph, stream=s):
                step()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        run = graph.replay
        log("graph captured")
    log("warmup done")
    t0 = time.perf_counter()
    for _ in range(args.steps):
        run()
    torch.cuda.synchronize()
    t = time.perf_counter() - t0
    ms = t / args.steps * 1e3
    n_acc = buf.n.cpu().numpy()
    log(f"{args.steps} steps: {ms:.3f} ms/step; n_accepted {n_acc.tolist()}")
    if model.device_error() != 0:
        log("device error word set")
        return 1

    ab = algorithmic_bytes(w, inp.lens)
    gbs = ab["total"] / (ms * 1e-3) / 1e9

    # Dominant kernel: the gate/up GEMM (45% of the weight bytes at this shape),
    # timed alone with HIP events on the current stream, same launch config.
    roof = spade.gemm_roofline(model, kv, "gu", w.batch, w.gamma, args.kernel_reps, HBM_PEAK_GBS)
    if w.name == "c2_7b_greedy":
        roof["traffic"] = read_traffic()
    log(f"dominant kernel: {roof}")
    if args.all_kernels:
        for kind in ("qkv", "o", "down", "lm"):
            r = spade.gemm_roofline(model, kv, kind, w.batch, w.gamma, args.kernel_reps, HBM_PEAK_GBS)
            log(f"gemm {kind}: {r['avg_launch_us']} us, {r['achieved']} GB/s ({r['frac']:.3f})")
    kv.restore(lens0, pend0)

    out = {
        "metric": "verified draft tokens/sec and verify-pass latency (us); achieved HBM GB/s vs peak",
        "value": round(w.batch * w.gamma / (ms * 1e-3), 2),
        "unit": "draft tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "verify_latency_us": round(ms * 1e3, 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 weights+KV, f32 activations" if m.weight_dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0,0.02) weights, uniform prompt ids; no trained weights)",
        "config": {"workload": w.name, "shape": m.name, "batch": w.batch, "gamma": w.gamma,
                   "cached_tokens": inp.lens.tolist(), "mode": w.mode, "drafts": drafts_src},
        "algorithmic_bytes_per_step": ab["total"],
        "achieved_GBps_whole_pass": round(gbs, 1),
        "hbm_frac_whole_pass": round(gbs / HBM_PEAK_GBS, 4),
        "emitted_tokens_per_call": float(np.mean(n_acc + 1)),
        "roofline": roof,
        "prefill": prefill,
    }
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle on {args.cpu_layers} layers")
        t0 = time.perf_counter()
        out["cpu_baseline"] = cpu_baseline(w, inp, args.cpu_layers)
        log(f"cpu baseline done in {time.perf_counter() - t0:.1f}s")
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
