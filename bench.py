#!/usr/bin/env python
"""Benchmark of the greedy speculative-verification step on one MI355X.

Workload (synthetic stand-in for the paper's code-editing benchmarks): a
7B-class Llama-style decoder with random bf16 weights, a 2048-token Zipf
prompt, and an "original code" c made from the model's own 512-token greedy
continuation G with 5% of its positions replaced in 3-8-token spans.  A
benchmark step is one edit task: the whole Reuse session that re-creates G
from c after the prompt.  Each verify call of it is one pass of the hot path:
the matcher picks where the generated output continues in c (a suffix match
of at least 3 tokens, else the position right after the last verified
draft), K = 32 tokens of c from there are verified in one forward, and the
accepted prefix plus the target's next token are emitted.  Every session is
checked to re-create G exactly (greedy verification is lossless), and every
session makes the same verify calls, so tokens/s does not depend on how many
steps are timed.

Printed: one JSON line.  value = emitted tokens per second over the timed
sessions (the paper's Tokens/s); also the verify-step latency at exactly 2048
committed positions (p50/p90 of 200 calls after 20 warm-up calls), the
whole-step HBM fraction of the 8 TB/s peak and of the streaming-read rate
measured on this GPU, each projection's rate, the dominant kernel's live
roofline and the CPU oracle's rate.

Other modes: --profile-only runs only fixed-context K = 32 verify steps and
the projection timing sequences (for rocprofv3); --rocprof-summary DIR
reduces rocprofv3's CSV output to the tables kept with the profiles.
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
MFMA_BF16_PEAK_TFLOPS = 2500.0   # dense bf16 matrix-core peak
LONG_K = 512                      # longest draft the engine is built for
CTX_SWEEP = (1024, 2048, 4096, 8000)   # committed lengths of the K = 32 step's context sweep (7B; max_ctx <= 8192)
# The Reuse driver resumes at a match of at least this many generated tokens;
# shorter (single-token) matches are frequent by chance and can move the
# cursor past the true position in the original code.
MIN_NGRAM = 3
METRIC = "verified tokens/sec + verify-step latency at K=32, 7B bf16; % peak HBM BW"


def linear_weight_bytes(s) -> int:
    esz = 2 if s.dtype == "bf16" else 4
    per_layer = (s.q_dim + 2 * s.kv_dim) * s.d_model + s.d_model * s.q_dim + 3 * s.ffn * s.d_model
    return esz * (s.n_layers * per_layer + s.vocab * s.d_model)


def step_bytes(s, t: int, n: int) -> dict:
    """Bytes one verify step must move: every weight once, the committed K/V
    once, the block's K/V written, the gathered embedding rows and the logits."""
    esz = 2 if s.dtype == "bf16" else 4
    kv_row = 2 * s.kv_dim * esz * s.n_layers
    parts = dict(weights=linear_weight_bytes(s), kv_read=n * kv_row, kv_write=t * kv_row,
                 embed=t * s.d_model * esz, logits=t * s.vocab * 4)
    parts["total"] = sum(parts.values())
    return parts


def gateup_bytes(s, t: int) -> int:
    """Algorithmic bytes of one fused gate/up + SwiGLU launch: the [2F, d]
    weights, the T normalised input rows it multiplies and the T x F SwiGLU
    outputs it writes."""
    esz = 2 if s.dtype == "bf16" else 4
    return esz * (2 * s.ffn * s.d_model + t * s.d_model + t * s.ffn)


def projection_model(s, cls: str, t: int):
    """(N, K, algorithmic bytes, flops) of one projection launch on t rows:
    the [N, K] weights once, the t input rows, and the t output rows (fp32
    results; the fused gate/up writes its t x F SwiGLU products in the model
    dtype instead)."""
    esz = 2 if s.dtype == "bf16" else 4
    d, qd, kd, f = s.d_model, s.q_dim, s.kv_dim, s.ffn
    n, k = {"qkv": (qd + 2 * kd, d), "oproj": (d, qd), "gateup": (2 * f, d), "down": (d, f),
            "lmhead": (s.vocab, d)}[cls]
    out = t * f * esz if cls == "gateup" else t * n * 4
    return n, k, esz * (n * k + t * k) + out, 2 * t * n * k


def _gemm_source_digest(path):
    """sha256 of the fused gate/up + SwiGLU section of the kernel source (from
    its section banner to the next one): the code the counter figures were
    taken on."""
    import hashlib
    out, on = [], False
    for ln in open(path).read().splitlines(keepends=True):
        if ln.startswith("// ----"):
            if on:
                break
            on = ln.rstrip().endswith(" gate/up + SwiGLU --")
        if on:
            out.append(ln)
    return hashlib.sha256("".join(out).encode()).hexdigest() if out else None


def measured_traffic():
    """Per-launch HBM bytes of the gate/up kernel from the committed counter
    summary, or None if its source has changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "gemm_swiglu_gateup_7b_k32_traffic.md")
    src = os.path.join(ROOT, "paper_2506_02780_amd", "csrc", "kernels.hip")
    try:
        text = open(path).read()
        digest = _gemm_source_digest(src)
    except OSError:
        return None
    fields = dict(ln.split(": ", 1) for ln in text.splitlines() if ": " in ln and ln[:1].isalpha())
    if digest is None or fields.get("gemm_source_sha256", "").strip() != digest:
        return None
    return int(fields["gateup_traffic_bytes_per_launch"])


def measured_gap_fraction():
    """The kernel-gap fraction of the 33-row blocks from the committed
    rocprofv3 kernel trace, or None if kernels.hip has changed since it was
    taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "verify_7b_k32_kernel_trace.md")
    src = os.path.join(ROOT, "paper_2506_02780_amd", "csrc", "kernels.hip")
    try:
        text = open(path).read()
        digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except OSError:
        return None
    fields = dict(ln.split(": ", 1) for ln in text.splitlines() if ": " in ln and ln[:1].isalpha())
    if fields.get("kernels_source_sha256", "").strip() != digest:
        return None
    import re
    m = re.search(r"kernel-gap fraction median ([0-9.]+)", text)
    return float(m.group(1)) if m else None


def cpu_info() -> dict:
    """CPU model and core count of this host."""
    model = "unknown"
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"model": model, "logical_cpus": os.cpu_count()}


def cpu_baseline(shape, weights, k: int, ctx: int, steps: int, emitted_per_verify: float):
    """The oracle (float64 NumPy, as it stands) timed on this host: `steps`
    whole K = k verify steps through all layers over a `ctx`-position
    committed cache, and one K = 0 step.  The committed cache is a seeded
    random bf16 one (the oracle's own 2048-token prefill would take minutes);
    the per-layer widening of the bf16 weights to float64, which the oracle
    does inside its forward, is part of the time."""
    from threadpoolctl import threadpool_info

    from oracle import OracleSession
    from oracle.numerics import to_f64
    from workloads import random_kv_context, zipf_tokens

    kv = random_kv_context(shape.n_layers, ctx, shape.n_kv_heads, shape.head_dim, seed=5, dtype=shape.dtype)
    cache = [(to_f64(a, shape.dtype), to_f64(b, shape.dtype)) for a, b in kv]
    del kv
    pending = int(zipf_tokens(shape.vocab, 1, seed=3)[0])

    def run(draft):
        ref = OracleSession(shape, weights)
        ref.set_cache(cache, pending)
        t0 = time.perf_counter()
        ref.verify(draft)
        return time.perf_counter() - t0

    times = [run(zipf_tokens(shape.vocab, k, seed=10 + i)) for i in range(steps)]
    t_ar = run(np.zeros(0, dtype=np.int32))
    per = float(np.mean(times))
    threads = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    info = cpu_info()
    return {
        "value": round(emitted_per_verify / per, 4), "unit": "tokens/s", "cores": int(threads),
        "kind": "oracle",
        "sample": (f"{steps} whole K={k} verify steps ({shape.n_layers} layers, LM head and acceptance) "
                   f"over a {ctx}-position committed cache of seeded random bf16 values, float64 NumPy, "
                   f"{per:.2f} s per step; tokens/s uses the GPU session's {emitted_per_verify:.2f} emitted "
                   f"tokens per verify call; plus one K=0 step (one plain greedy token) in {t_ar:.2f} s"),
        "verify_step_seconds": [round(t, 3) for t in times],
        "k0_step_seconds": round(t_ar, 3),
        "cpu_model": info["model"], "logical_cpus": info["logical_cpus"], "blas_threads": int(threads),
    }


def other_config(ee, name: str, k: int, ctx: int, reps: int = 60) -> dict:
    """Verify latency of another model shape at a fixed context: drafts are
    the model's own next k tokens (all accepted); the cache is rolled back to
    `ctx` after every step."""
    from workloads import gen_weights, get_shape, zipf_tokens
    shape = get_shape(name)
    weights = gen_weights(shape, seed=1234)
    eng = ee.Engine(shape, weights, max_ctx=ctx + k + 2, k_max=k)
    prompt = zipf_tokens(shape.vocab, ctx, seed=42)
    first = eng.prefill(0, prompt)
    cont = [eng.verify(0, [])[1] for _ in range(k)]
    lat = []
    for i in range(reps):
        eng.rollback(0, ctx, first)
        ts = time.perf_counter()
        a, _, _ = eng.verify(0, cont)
        if i >= 10:
            lat.append(time.perf_counter() - ts)
        assert a == k
    eng.close()
    p50 = float(np.percentile(lat, 50))
    tb = step_bytes(shape, k + 1, ctx)["total"]
    return {"model": f"{name} Llama-style random-init {shape.dtype}", "k": k, "ctx": ctx,
            "p50_ms": round(p50 * 1e3, 4), "p90_ms": round(float(np.percentile(lat, 90)) * 1e3, 4),
            "algorithmic_bytes": tb, "hbm_frac": round(tb / p50 / 1e9 / HBM_PEAK_GBS, 4),
            "tokens_per_s_full_acceptance": round((k + 1) / p50, 1)}


def batch_config(ee, name: str, n_seq: int, k: int, ctx: int, reps: int = 20) -> dict:
    """Latency of one ee_verify_batch block of n_seq sequences with k-token
    drafts, every sequence at `ctx` committed positions (rolled back after
    every step); drafts are each sequence's own next k tokens (all accepted)."""
    from workloads import gen_weights, get_shape, zipf_tokens
    shape = get_shape(name)
    t0 = time.perf_counter()
    weights = gen_weights(shape, seed=1234, eager=False)   # layers drawn while uploading
    eng = ee.Engine(shape, weights, max_ctx=ctx + k + 2, max_seqs=n_seq, k_max=k)
    del weights
    firsts = [eng.prefill(b, zipf_tokens(shape.vocab, ctx, seed=42 + b)) for b in range(n_seq)]
    conts = [[eng.verify(b, [])[1] for _ in range(k)] for b in range(n_seq)]
    setup_s = time.perf_counter() - t0
    lat = []
    for i in range(reps + 5):
        for b in range(n_seq):
            eng.rollback(b, ctx, firsts[b])
        ts = time.perf_counter()
        res = eng.verify_batch(list(range(n_seq)), conts)
        if i >= 5:
            lat.append(time.perf_counter() - ts)
        assert all(a == k for a, _, _ in res)
    eng.close()
    p50 = float(np.percentile(lat, 50))
    one = step_bytes(shape, k + 1, ctx)
    tb = one["weights"] + n_seq * (one["total"] - one["weights"])
    rows = n_seq * (k + 1)
    esz = 2 if shape.dtype == "bf16" else 4
    flops = 2 * rows * linear_weight_bytes(shape) // esz + n_seq * attention_flops(shape, k + 1, ctx)
    return {"model": f"{name} Llama-style random-init {shape.dtype}", "sequences": n_seq, "k": k,
            "ctx": ctx, "rows": rows, "p50_ms": round(p50 * 1e3, 3),
            "p90_ms": round(float(np.percentile(lat, 90)) * 1e3, 3),
            "algorithmic_bytes": tb, "hbm_frac": round(tb / p50 / 1e9 / HBM_PEAK_GBS, 4),
            "flops": flops, "mfma_frac": round(flops / p50 / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
            "emitted_tokens_per_s": round(n_seq * (k + 1) / p50, 1), "setup_s": round(setup_s, 1)}


def edit_sessions(ee, eng, shape, ctx: int, first: int, G, log) -> dict:
    """Whole edit sessions (ee_edit_step) re-creating the model's own greedy
    output G from an edited copy, at several edit densities: plain greedy
    decoding, Reuse with plain greedy steps at edit positions, and Reuse with
    a 1B-class draft model in the Generate phase (gamma = 7; greedy or
    entropy-aware verification, k = 5).  Random-init models: the draft model
    shares no knowledge with the target, so its tokens are rarely accepted;
    the figures show what the phases cost, not the paper's trained speedups."""
    from workloads import gen_weights, get_shape, inject_edits, zipf_tokens
    n = len(G)
    dshape = get_shape("1b")
    t0 = time.perf_counter()
    deng = ee.Engine(dshape, gen_weights(dshape, seed=4321), max_ctx=ctx + n + 80, k_max=64)
    deng.prefill(0, zipf_tokens(shape.vocab, ctx, seed=42))      # the target's prompt
    setup = time.perf_counter() - t0

    def run(original, draft, top_k, k_reuse=32):
        eng.rollback(0, ctx, first)
        if draft is not None:
            draft.rollback(0, ctx, first)
        s = ee.EditSession(eng, 0, original, draft, 0, k_reuse=k_reuse, gamma=7, top_k=top_k, dynamic=True)
        torch_sync()
        ts = time.perf_counter()
        while s.n < n:
            s.step()
        el = time.perf_counter() - ts
        out, st = s.output[:n], s.state
        return {"tokens_per_s": round(n / el, 1), "seconds": round(el, 3),
                "steps_reuse": int(st.steps[0]), "steps_generate": int(st.steps[1]),
                "emitted_reuse": int(st.emitted[0]), "emitted_generate": int(st.emitted[1]),
                "draft_tokens": int(st.draft_tokens), "equals_greedy_output": out == list(G)}

    res = {"tokens": n, "draft_model": "1b Llama-style random-init bf16", "gamma": 7, "k_reuse": 32,
           "draft_setup_s": round(setup, 1)}
    eng.rollback(0, ctx, first)
    torch_sync()
    ts = time.perf_counter()
    for _ in range(n - 1):
        eng.verify(0, [])
    ar = (n - 1) / (time.perf_counter() - ts)
    res["greedy_decoding_tokens_per_s"] = round(ar, 1)
    for frac in (0.05, 0.25, 0.5):
        log(f"[bench] edit sessions at edit density {frac}")
        original, _ = inject_edits(np.asarray(G, dtype=np.int32), shape.vocab, seed=7, frac=frac)
        row = {"reuse_plus_greedy_steps": run(list(original), None, 0),
               "reuse_plus_draft_greedy": run(list(original), deng, 0),
               "reuse_plus_draft_entropy_k5": run(list(original), deng, 5)}
        for v in row.values():
            v["speedup_vs_greedy_decoding"] = round(v["tokens_per_s"] / ar, 2)
        res[f"edit_density_{frac}"] = row
    deng.close()
    eng.rollback(0, ctx, first)
    return res


def torch_sync():
    import torch
    torch.cuda.synchronize()


def attention_flops(s, t: int, n: int) -> int:
    """Score and value products of t rows over n committed keys plus the
    block, in every layer."""
    return s.n_layers * 2 * 2 * s.n_heads * s.head_dim * t * (n + (t + 1) // 2)


def projection_rates(eng, shape, t: int) -> dict:
    """Each projection's GEMM (and the LM head's) on t rows, launched for
    every layer in turn, 3 times, back to back between two HIP events
    (ee_time_gemm): microseconds per launch, algorithmic HBM rate and
    matrix-core rate (t rows, no padding) against the peaks."""
    out = {}
    for cls in ("qkv", "oproj", "gateup", "down", "lmhead"):
        us = eng.time_gemm(cls, t, reps=3)
        n, k, nbytes, flops = projection_model(shape, cls, t)
        out[cls] = {"n": n, "k": k, "us_per_launch": round(us, 2), "algorithmic_bytes": nbytes,
                    "GBps": round(nbytes / us / 1e3, 1), "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4),
                    "TFLOPs": round(flops / us / 1e6, 2),
                    "mfma_frac": round(flops / us / 1e6 / MFMA_BF16_PEAK_TFLOPS, 4)}
    return out


def calibration_copy():
    """A plain 256 MiB device copy, so that hardware byte counters read on
    the same run can be scaled against a transfer of known size."""
    import torch
    cal = torch.empty(64 << 20, dtype=torch.float32, device="cuda")
    cal_dst = torch.empty_like(cal)
    cal_dst.copy_(cal)
    torch.cuda.synchronize()
    del cal, cal_dst


def profile_only(eng, shape, ctx, K, first, args, log):
    """The run rocprofv3 profiles: K = K verify blocks of the model's own
    continuation at exactly ctx committed positions, the projection timing
    sequences of that block shape, and the calibration copy."""
    cont = [eng.verify(0, [])[1] for _ in range(K)]
    for _ in range(args.profile_steps):
        eng.rollback(0, ctx, first)
        a, _, _ = eng.verify(0, cont)
        assert a == K
    gemms = projection_rates(eng, shape, K + 1)
    calibration_copy()
    log(f"[bench] profile run: {args.profile_steps} K={K} verify blocks at n={ctx}")
    print(json.dumps({"profile_only": True, "k": K, "ctx": ctx, "verify_blocks": args.profile_steps,
                      "projections": gemms}), flush=True)


# Kernels of one layer of a T = 33 block, in dispatch order (bf16, head_dim 128,
# d <= 4096): role and kernel name prefix.
LAYER_ROLES = [("QKV projection + rotary + KV append", "gemm_ep_kernel<1, 2, 16, 1>"),
               ("attention", "attn_kernel<1, 128, false>"), ("split merge", "attn_combine_kernel<1, 128>"),
               ("O projection + residual + FFN norm sums", "gemm_ep_kernel<1, 2, 16, 2>"),
               ("gate/up + SwiGLU", "gemm_swiglu_kernel<1, 2, 16, true>"), ("down projection", "gemm_kernel<1, 3"),
               ("residual + norm (after down)", "resid_kernel<1, 1>")]
NORM_ROLE = len(LAYER_ROLES) - 1   # its grid has one row of workgroups per block row: 33 for T = 33


def _short(name: str) -> str:
    return name.split("(")[0].replace("void ", "").replace("ee::", "").strip()


def _layer_starts(names):
    """Indices i where the dispatches of a T = 33 layer (LAYER_ROLES) start."""
    n = len(LAYER_ROLES)
    return [i for i in range(len(names) - n + 1)
            if all(names[i + j].startswith(p) for j, (_, p) in enumerate(LAYER_ROLES))]


def _md_rows(text: str) -> dict:
    """role -> {column: value} from the role tables of a rocprof summary."""
    rows, hdr = {}, None
    for ln in text.splitlines():
        if ln.startswith("| role |"):
            hdr = [c.strip() for c in ln.strip().strip("|").split("|")][1:]
        elif ln.startswith("| ") and hdr and not ln.startswith("|---"):
            cells = [c.strip() for c in ln.strip().strip("|").split("|")]
            try:
                rows[cells[0]] = dict(zip(hdr, [float(x) for x in cells[1:1 + len(hdr)]]))
            except ValueError:
                pass
    return rows


def counter_table(fetch_dir: str, write_dir: str, mfma_dir: str, trace_dir: str, lm_head_us: float):
    """The combined per-role table of profiles/verify_7b_k32_counters.md from
    the four rocprofv3 output directories (FETCH_SIZE, WRITE_SIZE and MFMA
    counter runs, kernel trace): counters scaled by the 256 MiB calibration
    copy, algorithmic bytes of the projection model, matrix-core rate at the
    traced median durations (the LM head's from its ee_time_gemm time) and
    the MFMA-busy fraction.  Prints to stdout."""
    import contextlib
    import io
    import re

    def summary(d):
        buf = io.StringIO()
        with contextlib.redirect_stdout(buf):
            rocprof_summary(d)
        return buf.getvalue()
    ft, wt, mt, tt = (summary(d) for d in (fetch_dir, write_dir, mfma_dir, trace_dir))
    f, w, m = _md_rows(ft), _md_rows(wt), _md_rows(mt)
    fcal = float(re.search(r"FETCH_SIZE ([0-9.]+)", ft.split("calibration copy", 1)[1]).group(1))
    wcal = float(re.search(r"WRITE_SIZE ([0-9.]+)", wt.split("calibration copy", 1)[1]).group(1))
    fs, ws = 262144 / fcal, 262144 / wcal
    traced = {}
    for ln in tt.splitlines():
        cells = [c.strip() for c in ln.strip().strip("|").split("|")]
        if len(cells) == 5 and cells[2].isdigit():
            traced[cells[0]] = float(cells[3])
    s7 = get_shape_for_table()
    alg = {LAYER_ROLES[0][0]: projection_model(s7, "qkv", 33)[2],
           LAYER_ROLES[3][0]: projection_model(s7, "oproj", 33)[2],
           "gate/up + SwiGLU": projection_model(s7, "gateup", 33)[2],
           "down projection": projection_model(s7, "down", 33)[2],
           "LM head (the GEMM before the logits kernel)": projection_model(s7, "lmhead", 33)[2]}
    print(f"FETCH_SIZE scale {fs:.4f} (copy read 262144 KiB, counter {fcal}); "
          f"WRITE_SIZE scale {ws:.4f} (counter {wcal})")
    print("| role | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM bytes (scaled) | algorithmic bytes | ratio | "
          "bf16 MFMA flops | MFMA TFLOP/s at the traced time | MFMA busy |\n|---|---|---|---|---|---|---|---|---|")
    for role in f:
        fe, wr = f[role]["FETCH_SIZE"], w[role]["WRITE_SIZE"]
        hb = (fe * fs + wr * ws) * 1024
        a = alg.get(role)
        mm = m[role]
        fl = mm["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512
        us = lm_head_us if role.startswith("LM head") else traced.get(role)
        busy = mm["SQ_VALU_MFMA_BUSY_CYCLES"] / 1024 / (mm["GRBM_GUI_ACTIVE"] / 8) if mm["GRBM_GUI_ACTIVE"] else 0.0
        tf = f"{fl / us / 1e6:.1f} ({fl / us / 1e6 / MFMA_BF16_PEAK_TFLOPS:.3f} of peak)" if fl and us else ""
        name = "LM head" if role.startswith("LM head") else role
        ab = f"{a / 1e6:.2f} MB | {hb / a:.3f}" if a else " | "
        print(f"| {name} | {fe:.1f} | {wr:.1f} | {hb / 1e6:.2f} MB | {ab} | "
              f"{(f'{fl / 1e9:.3f} G' if fl else '0')} | {tf} | {busy:.3f} |")


def get_shape_for_table():
    sys.path.insert(0, ROOT)
    from workloads import get_shape
    return get_shape("7b")


def rocprof_summary(d: str):
    """Markdown tables from rocprofv3 CSV output under directory d: kernel
    statistics, per-role durations of T = 33 layers, the kernel-gap fraction
    of T = 33 blocks (kernel trace), and per-role counter values (counter
    runs).  Prints to stdout."""
    import csv
    import glob
    import statistics as st

    def rows_of(pat):
        f = sorted(glob.glob(os.path.join(d, "**", pat), recursive=True))
        return list(csv.DictReader(open(f[0]))) if f else None

    stats = rows_of("*kernel_stats.csv")
    if stats:
        print("| kernel | calls | total ms | avg us | % |\n|---|---|---|---|---|")
        for r in stats[:20]:
            print(f"| `{_short(r['Name'])}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
                  f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    tr = rows_of("*kernel_trace.csv")
    if tr:
        tr.sort(key=lambda r: int(r["Start_Timestamp"]))
        names = [_short(r["Kernel_Name"]) for r in tr]
        gy = [int(r["Grid_Size_Y"]) for r in tr]
        t0 = [int(r["Start_Timestamp"]) for r in tr]
        t1 = [int(r["End_Timestamp"]) for r in tr]
        starts = [i for i in _layer_starts(names) if gy[i + NORM_ROLE] == 33]
        print(f"\nT = 33 layers found: {len(starts)}\n")
        print("| role | kernel | dispatches | median us | mean us |\n|---|---|---|---|---|")
        tot = 0.0
        for j, (role, _) in enumerate(LAYER_ROLES):
            v = [(t1[i + j] - t0[i + j]) / 1e3 for i in starts]
            if v:
                tot += st.median(v)
                print(f"| {role} | `{names[starts[0] + j]}` | {len(v)} | {st.median(v):.2f} | {st.mean(v):.2f} |")
        print(f"| one layer (sum of medians) | | | {tot:.2f} | |")
        # blocks of 33 rows: stage_in_kernel .. result_out_kernel; kernels busy
        # = the union of their intervals
        spans, busy = [], []
        i = 0
        while i < len(names):
            if names[i] != "stage_in_kernel":
                i += 1
                continue
            j = i
            while j < len(names) and names[j] != "result_out_kernel":
                j += 1
            if j < len(names) and any(names[x] == "resid_kernel<1, 1>" and gy[x] == 33 for x in range(i, j)):
                b, cur_end = 0, t0[i]
                for x in range(i, j + 1):
                    s0, s1 = max(t0[x], cur_end), t1[x]
                    if s1 > s0:
                        b += s1 - s0
                        cur_end = s1
                spans.append((t1[j] - t0[i]) / 1e3)
                busy.append(b / 1e3)
            i = j + 1
        if spans:
            fr = [1 - b / s for b, s in zip(busy, spans)]
            print(f"\nT = 33 blocks: {len(spans)}; first kernel start to last kernel end: median "
                  f"{st.median(spans):.1f} us, of which kernels run {st.median(busy):.1f} us; "
                  f"kernel-gap fraction median {st.median(fr):.4f}")
    pmc = rows_of("*counter_collection.csv")
    if pmc:
        by = {}
        for r in pmc:
            by.setdefault(int(r["Dispatch_Id"]), []).append(r)
        ids = sorted(by)
        names = [_short(by[i][0]["Kernel_Name"]) for i in ids]
        counters = sorted({r["Counter_Name"] for r in pmc})

        def val(i, c):
            return sum(float(r["Counter_Value"]) for r in by[i] if r["Counter_Name"] == c)
        cal = [i for i in ids if "copyBuffer" in by[i][0]["Kernel_Name"]]
        if cal:
            big = max(cal, key=lambda i: int(by[i][0]["Grid_Size"]))
            print("\ncalibration copy (256 MiB read, 256 MiB written): " +
                  ", ".join(f"{c} {val(big, c):.1f}" for c in counters))
        starts = _layer_starts(names)
        print(f"\nT = 33 layers found: {len(starts)} (mean per dispatch)\n")
        print("| role | " + " | ".join(counters) + " |\n|---|" + "---|" * len(counters))
        for j, (role, _) in enumerate(LAYER_ROLES):
            if starts:
                print(f"| {role} | " + " | ".join(f"{st.mean(val(ids[k + j], c) for k in starts):.1f}"
                                                  for c in counters) + " |")
        # the LM head: the dispatch after a block's last T = 33 layer, when the
        # logits kernel follows it
        nl = len(LAYER_ROLES)
        lm = [s + nl for s in starts if s + nl + 1 < len(names) and names[s + nl + 1].startswith("logits_kernel")]
        if lm:
            print("| LM head (the GEMM before the logits kernel) | " + " | ".join(
                f"{st.mean(val(ids[k], c) for k in lm):.1f}" for c in counters) + " |")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20, help="timed edit tasks (whole Reuse sessions re-creating G)")
    ap.add_argument("--warmup", type=int, default=5, help="untimed edit tasks before them")
    ap.add_argument("--config", default="7b", choices=["tiny", "1b", "7b", "33b"])
    ap.add_argument("--k", type=int, default=32)
    ap.add_argument("--ctx", type=int, default=2048)
    ap.add_argument("--gen", type=int, default=512, help="length of the greedy output re-created")
    ap.add_argument("--cpu-steps", type=int, default=3, help="whole K-token oracle verify steps timed")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-only", action="store_true",
                    help="only fixed-context verify steps and the projection timing sequences (for rocprofv3)")
    ap.add_argument("--profile-steps", type=int, default=20)
    ap.add_argument("--rocprof-summary", metavar="DIR", help="reduce rocprofv3 CSV output in DIR to tables")
    ap.add_argument("--counter-table", nargs=5, metavar=("FETCH", "WRITE", "MFMA", "TRACE", "LMHEAD_US"),
                    help="combine the FETCH_SIZE, WRITE_SIZE and MFMA counter runs and the kernel trace into one "
                         "per-role table (LMHEAD_US: the LM head's ee_time_gemm time)")
    ap.add_argument("--eager", action="store_true", help="launch kernel by kernel (no graph replay)")
    ap.add_argument("--no-33b", action="store_true", help="skip the 33B batch-of-4 measurement")
    ap.add_argument("--no-long", action="store_true", help="skip the long-draft (K = 128..512) measurement")
    ap.add_argument("--no-edit", action="store_true", help="skip the edit sessions with a draft model")
    args = ap.parse_args()
    if args.rocprof_summary:
        rocprof_summary(args.rocprof_summary)
        return
    if args.counter_table:
        counter_table(*args.counter_table[:4], float(args.counter_table[4]))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the verification step of one edit session is "
              "not sharded across GPUs (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2506_02780_amd as ee
    from workloads import gen_weights, get_shape, inject_edits, random_tree, tree_tokens, zipf_tokens

    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    shape = get_shape(args.config)
    K, ctx = args.k, args.ctx
    t0 = time.perf_counter()
    weights = gen_weights(shape, seed=1234)
    log(f"[bench] weights drawn in {time.perf_counter() - t0:.1f}s")
    max_ctx = max(ctx + args.gen + 66, ctx + LONG_K + 2)
    if args.config == "7b" and not args.profile_only:
        max_ctx = max(max_ctx, max(CTX_SWEEP) + K + 2)
    eng = ee.Engine(shape, weights, max_ctx=max_ctx, k_max=LONG_K)
    if args.eager:
        eng.use_graphs(False)
    log(f"[bench] engine ready at {time.perf_counter() - t0:.1f}s")

    prompt = zipf_tokens(shape.vocab, ctx, seed=42)
    first = eng.prefill(0, prompt)
    if args.profile_only:
        profile_only(eng, shape, ctx, K, first, args, log)
        return
    G = [first]
    for _ in range((args.gen if args.no_long else max(args.gen, LONG_K + 1)) - 1):
        G.append(eng.verify(0, [])[1])
    G_long = list(G)             # the continuation long drafts are taken from
    G = G[:args.gen]
    code, _ = inject_edits(np.asarray(G, dtype=np.int32), shape.vocab, seed=7)
    code = code.tolist()
    log(f"[bench] prompt + {args.gen}-token greedy output ready at {time.perf_counter() - t0:.1f}s")

    # the session's token sequences as int32 arrays, handed to the library
    # without a per-call conversion (the output grows in place in gen_buf)
    code_a = np.asarray(code, dtype=np.int32)
    G_a = np.asarray(G, dtype=np.int32)
    gen_buf = np.empty(len(G) + K + 2, dtype=np.int32)

    def edit_task(lat=None):
        """One whole Reuse session re-creating G: (verify calls, emitted tokens)."""
        eng.rollback(0, ctx, first)
        gen_buf[0] = first
        n, cur, calls, emitted = 1, 0, 0, 0
        while n < len(G):
            ds, _ = ee.match_reuse(gen_buf[:n], code_a, cur, MIN_NGRAM, 8)
            start = ds if ds >= 0 else cur
            d = code_a[start:start + K]
            ts = time.perf_counter()
            a, nxt, _ = eng.verify(0, d)
            if lat is not None:
                lat.append(time.perf_counter() - ts)
            gen_buf[n:n + a] = d[:a]
            gen_buf[n + a] = nxt
            m = min(n + a + 1, len(G))
            if not np.array_equal(gen_buf[n:m], G_a[n:m]):
                raise SystemExit(f"lossless check failed at output position {n}")
            n += a + 1
            cur = start + a + 1
            calls += 1
            emitted += a + 1
        return calls, emitted

    for _ in range(args.warmup):
        edit_task()
    torch.cuda.synchronize()
    emitted, calls, sess_lat = 0, 0, []
    t_start = time.perf_counter()
    for _ in range(args.steps):
        c_, e_ = edit_task(sess_lat)
        calls += c_
        emitted += e_
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    log(f"[bench] {args.steps} edit tasks: {calls} verify calls, {emitted} tokens in {elapsed:.3f}s")

    # dominant kernel: after the timed steps, the gate/up GEMM of the block
    # shape the session uses (T rows) is launched for each of the layers in
    # turn, back to back on the library stream, between two HIP events
    # (events around single launches add ~4 us of their own to each)
    T = K + 1
    gu_avg_s = eng.time_gemm("gateup", T, reps=5) * 1e-6
    gu_n = 5 * shape.n_layers
    gu_alg = gateup_bytes(shape, T)

    # verify latency at exactly `ctx` committed positions (rollback after every step)
    def fixed_ctx(draft, parent=None, reps=220, warm=20):
        lat, acc = [], []
        for i in range(reps):
            eng.rollback(0, ctx, first)
            ts = time.perf_counter()
            a, _, _ = eng.verify(0, draft, parent)
            if i >= warm:
                lat.append(time.perf_counter() - ts)
                acc.append(a)
        return float(np.percentile(lat, 50)), float(np.percentile(lat, 90)), float(np.mean(acc))

    d = code[1:1 + K]
    p50, p90, _ = fixed_ctx(d)
    sb = step_bytes(shape, T, ctx)

    # K sweep and a 64-node draft tree at the same context; drafts follow the
    # model's own continuation (G), so every draft token is accepted
    def lat_entry(kk, lat50, lat90, acc):
        tb = step_bytes(shape, kk + 1, ctx)["total"]
        return {"p50_ms": round(lat50 * 1e3, 4), "p90_ms": round(lat90 * 1e3, 4),
                "hbm_frac": round(tb / lat50 / 1e9 / HBM_PEAK_GBS, 4),
                "accepted": round(acc, 2), "tokens_per_s_at_this_acceptance": round((acc + 1) / lat50, 1)}
    k_sweep = {}
    for kk in (0, 8, 16, 32, 64):
        l50, l90, acc = fixed_ctx(list(G[1:1 + kk]))
        k_sweep[str(kk)] = lat_entry(kk, l50, l90, acc)
    parent = random_tree(64, max_depth=8, max_branch=3, seed=11)
    ttoks = tree_tokens(parent, G[1:9], shape.vocab, seed=11)
    l50, l90, acc = fixed_ctx(ttoks, parent)
    tree64 = dict(lat_entry(64, l50, l90, acc), nodes=64, max_depth=8, max_branch=3)

    # long Reuse drafts: one block of K + 1 rows verifies a long span (the
    # model's own continuation, so every draft token is accepted)
    long_drafts = {}
    for kk in (() if args.no_long else (128, 256, LONG_K)):
        l50, l90, acc = fixed_ctx(list(G_long[1:1 + kk]), reps=40, warm=10)
        e = lat_entry(kk, l50, l90, acc)
        fl = 2 * (kk + 1) * linear_weight_bytes(shape) // 2 + attention_flops(shape, kk + 1, ctx)
        e["mfma_frac"] = round(fl / l50 / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)
        long_drafts[str(kk)] = e

    # entropy-aware dynamic and fixed top-k verification (Eq. 9-10) on the
    # same draft as the headline latency, with the per-class time of the
    # kernels that differ from greedy verification (logits epilogue, selection)
    def topk_ctx(draft, k, dynamic, reps=60):
        lat, acc = [], []
        for i in range(reps):
            eng.rollback(0, ctx, first)
            ts = time.perf_counter()
            (a, _, _), = eng.verify_topk([0], [draft], k, dynamic)
            if i >= 10:
                lat.append(time.perf_counter() - ts)
                acc.append(a)
        return float(np.percentile(lat, 50)), float(np.percentile(lat, 90)), float(np.mean(acc))

    def select_ms(fn):
        eng.profile(["finish", "argmax"])
        eng.profile_read(reset=True)
        for _ in range(10):
            eng.rollback(0, ctx, first)
            fn()
        pr = eng.profile_read(reset=True)
        eng.profile([])
        return {c: round(ms / 10, 4) for c, (ms, n) in pr.items() if n}
    d_topk = code[1:1 + K]
    entropy = {"k_draft": K, "draft": "the headline draft (edited copy of the greedy output)"}
    for kk, dyn in ((5, True), (3, True), (5, False)):
        l50, l90, acc = topk_ctx(d_topk, kk, dyn)
        entropy[f"{'dynamic' if dyn else 'fixed'}_top{kk}"] = {
            "p50_ms": round(l50 * 1e3, 4), "p90_ms": round(l90 * 1e3, 4), "accepted": round(acc, 2)}
    entropy["per_step_ms_topk5_dynamic"] = select_ms(lambda: eng.verify_topk([0], [d_topk], 5, True))
    # stochastic verification (Eq. 4) on the same draft: a greedy draft
    # (no distribution) and a draft distribution over the whole vocabulary
    rs = np.random.default_rng(5)
    qd = rs.dirichlet(np.full(shape.vocab, 0.1), size=K).astype(np.float32)
    for i, t in enumerate(d_topk):
        qd[i, t] += 1.0
    qd /= qd.sum(axis=1, keepdims=True)
    sampled = {}
    for name, qq in (("greedy_draft", None), ("draft_distribution", qd)):
        lat, acc = [], []
        for i in range(40):
            eng.rollback(0, ctx, first)
            e_, u_ = rs.random(K), rs.random(K + 1)
            ts = time.perf_counter()
            a, _ = eng.verify_sample(0, d_topk, e_, u_, qq, 1.0, True)
            if i >= 5:
                lat.append(time.perf_counter() - ts)
                acc.append(a)
        sampled[name] = {"p50_ms": round(float(np.percentile(lat, 50)) * 1e3, 4), "accepted": round(float(np.mean(acc)), 2)}
    sampled["note"] = "the draft distribution is uploaded inside each call (a 4.1 MB host-to-device copy)"
    entropy["per_step_ms_greedy"] = select_ms(lambda: eng.verify(0, d_topk))
    eng.rollback(0, ctx, first)

    gemms = projection_rates(eng, shape, T)
    # the streaming-read rate this GPU reaches (a 2 GiB buffer, well past the
    # 256 MB Infinity Cache)
    sbuf = torch.empty(2 << 30, dtype=torch.uint8, device="cuda")
    stream_us = eng.time_stream_read(sbuf, reps=10)
    stream_gbps = sbuf.numel() / stream_us / 1e3
    del sbuf
    calibration_copy()

    # per-class breakdown of one step (separate pass, every class instrumented)
    eng.profile(list(ee.PROF_CLASSES))
    for _ in range(10):
        eng.rollback(0, ctx, first)
        eng.verify(0, d)
    prof = eng.profile_read(reset=True)
    brk = {c: round(ms / 10, 4) for c, (ms, n) in prof.items() if n}
    brk_launches = {c: n // 10 for c, (ms, n) in prof.items() if n}
    eng.profile([])
    eng.rollback(0, ctx, first)

    edit = None if (args.no_edit or args.config != "7b") else edit_sessions(ee, eng, shape, ctx, first, G, log)

    # the step at several committed lengths (attention's share of the bytes
    # grows with n): each prompt is prefilled into the sequence afresh, the
    # draft is K Zipf tokens, the cache is rolled back after every step
    ctx_sweep = {}
    for n_ctx in (CTX_SWEEP if args.config == "7b" else ()):
        eng.rollback(0, 0, -1)
        f_n = eng.prefill(0, zipf_tokens(shape.vocab, n_ctx, seed=42))
        d_n = [int(x) for x in zipf_tokens(shape.vocab, K, seed=43)]
        lat_n = []
        for i in range(120):
            eng.rollback(0, n_ctx, f_n)
            ts = time.perf_counter()
            eng.verify(0, d_n)
            if i >= 20:
                lat_n.append(time.perf_counter() - ts)
        l50 = float(np.percentile(lat_n, 50))
        sb_n = step_bytes(shape, K + 1, n_ctx)
        ctx_sweep[str(n_ctx)] = {"p50_ms": round(l50 * 1e3, 4), "p90_ms": round(float(np.percentile(lat_n, 90)) * 1e3, 4),
                                 "kv_read_bytes": sb_n["kv_read"], "algorithmic_bytes": sb_n["total"],
                                 "hbm_frac": round(sb_n["total"] / l50 / 1e9 / HBM_PEAK_GBS, 4)}

    result = {
        "metric": METRIC,
        "value": round(emitted / elapsed, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": shape.dtype,
        "data": "synthetic",
        "config": {
            "workload": (f"{args.config} Llama-style random-init {shape.dtype}, Reuse session: K={K} "
                         f"drafts from an edited copy (5% in 3-8-token spans) of the model's own "
                         f"{args.gen}-token greedy output, after a {ctx}-token Zipf prompt"),
            "k": K, "prompt_tokens": ctx, "regenerated_tokens": args.gen, "batch": 1,
        },
        "step": "one edit task: the whole Reuse session re-creating the regenerated tokens",
        "emitted_per_step": round(emitted / args.steps, 3),
        "verify_calls_per_step": round(calls / args.steps, 3),
        "emitted_per_verify": round(emitted / calls, 3),
        "ms_per_verify": {"mean": round(elapsed / calls * 1e3, 4),
                          "p50": round(float(np.percentile(sess_lat, 50)) * 1e3, 4),
                          "p90": round(float(np.percentile(sess_lat, 90)) * 1e3, 4)},
        "verify_latency_ms_at_ctx": {"ctx": ctx, "k": K, "calls": 200, "warmup_calls": 20,
                                     "p50": round(p50 * 1e3, 4), "p90": round(p90 * 1e3, 4)},
        "draft_tokens_checked_per_s_at_ctx": round(K / p50, 1),
        "full_acceptance_tokens_per_s_at_ctx": round((K + 1) / p50, 1),
        "step_hbm": {"algorithmic_bytes": sb["total"], "achieved_GBps": round(sb["total"] / p50 / 1e9, 1),
                     "frac_of_peak": round(sb["total"] / p50 / 1e9 / HBM_PEAK_GBS, 4),
                     "streaming_read_GBps": round(stream_gbps, 1),
                     "frac_of_streaming_read": round(sb["total"] / p50 / 1e9 / stream_gbps, 4),
                     "kernel_gap_fraction": measured_gap_fraction(),
                     "kernel_gap_note": ("share of a 33-row block's span in which no kernel of it runs, from the "
                                         "committed rocprofv3 kernel trace of this kernel source (null once "
                                         "kernels.hip has changed since)")},
        "projections": gemms,
        "roofline": {
            "kernel": f"gemm_swiglu_kernel<{shape.dtype}> (gate/up projection + SwiGLU, T={T})",
            "measured": ("HIP events around 5 x 32 gate/up launches (every layer's weights in turn) run back "
                         "to back on the library stream after the timed steps, with the timed block's shape"),
            "bound": "hbm",
            "achieved": round(gu_alg / gu_avg_s / 1e9, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(gu_alg / gu_avg_s / 1e9 / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(),
            "launch_us": round(gu_avg_s * 1e6, 2),
            "launches": int(gu_n),
            "bytes_per_launch": gu_alg,
        },
        "breakdown_ms_per_verify": brk,
        "breakdown_launches_per_verify": brk_launches,
        "breakdown_note": ("one K=32 verify at the fixed context, every launch bracketed by HIP events (each figure "
                           "includes ~3-4 us of event overhead per launch; every launch of the block is counted)"),
        "k_sweep_at_ctx": k_sweep,
        "ctx_sweep_k": ({"k": K, "draft": "K Zipf tokens (the step's cost, not its acceptance)", "by_ctx": ctx_sweep}
                        if ctx_sweep else None),
        "tree64_at_ctx": tree64,
        "long_drafts_at_ctx": long_drafts or None,
        "entropy_verify_at_ctx": entropy,
        "sampled_verify_at_ctx": sampled,
        "edit_sessions": edit,
        "lossless_check": "emitted stream equals the GPU's own greedy output",
    }
    eng.close()
    if args.config == "7b":
        result["other_configs"] = {"1b_k16_ctx1024": other_config(ee, "1b", 16, 1024)}
        if not args.no_33b:
            log("[bench] 33B batch of 4 sequences")
            result["other_configs"]["33b_batch4_k64_ctx4096"] = batch_config(ee, "33b", 4, 64, 4096)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle sample")
        result["cpu_baseline"] = cpu_baseline(shape, weights, K, ctx, args.cpu_steps, emitted / calls)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
