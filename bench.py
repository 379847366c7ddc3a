#!/usr/bin/env python3
"""Benchmark of one OmniQuant block-wise calibration step on one MI355X.

A step is the whole hot path on one batch: LWC fake-quant of the block's
seven linears, the forward matrix products with the residual epilogue, the
loss, the weight-gradient products, the straight-through clipping gradients
(plus, for LET workloads, the activation-side products and LET gradients) and
the AdamW update.  Inputs are synthetic (seeded, drawn on the GPU), resident
in HBM before the timed region; the full-precision targets are produced once
before timing, as Algorithm 1 does once per block.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--tokens T]
    python bench.py --decode [--decode-bits B] [--decode-tokens N]   (deployment workload)

Prints one JSON line.  ``roofline`` describes the dominant kernel kind,
timed with HIP events on the launching stream during the timed steps;
``cpu_baseline`` times the CPU oracle on a bounded sample of the same
workload (rank 0, one GPU only).
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK = {"mfma_bf16_tflops": 2500.0, "fp32_tflops": 157.3, "hbm_gbs": 8000.0}
GEMM_KINDS = ("gemm_fwd", "gemm_wgrad", "gemm_dgrad")
# sources whose text defines the forward-product kernel; a traffic summary
# taken on other sources no longer describes it
GEMM_SOURCES = ("paper_2308_13137_amd/csrc/gemm.hip", "paper_2308_13137_amd/csrc/common.h",
                "paper_2308_13137_amd/csrc/oq_internal.h")
COPY_BYTES = 1 << 30          # calibration copy: 1 GiB read, 1 GiB written


# sources whose text defines the packed linear's kernel
PACKED_SOURCES = ("paper_2308_13137_amd/csrc/packed.hip", "paper_2308_13137_amd/csrc/packed.h",
                  "paper_2308_13137_amd/csrc/common.h")
# per dominant kernel: its sources, the key of their hash in the summary, the
# dispatches the counters are read from, and what they are called
TRAFFIC_KINDS = {
    "gemm_fwd": (GEMM_SOURCES, "gemm source hash",
                 lambda n: "gemm_bf16_w8_kernel" in n and "EpiResid" in n, "the forward product"),
    "packed_linear": (PACKED_SOURCES, "packed source hash", lambda n: "packed_linear_kernel" in n,
                      "the packed-weight linear"),
}


def source_hash(kind="gemm_fwd"):
    import hashlib
    h = hashlib.sha256()
    for rel in TRAFFIC_KINDS[kind][0]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def gemm_source_hash():
    return source_hash("gemm_fwd")


def traffic_file(workload, kind="gemm_fwd"):
    return os.path.join(ROOT, "profiles", f"{kind}_{workload}_hbm_traffic.md")


def read_traffic(workload, kind="gemm_fwd"):
    """HBM bytes per launch of the kind's kernel from the committed counter
    summary, or None when there is none or it was taken on other sources."""
    path = traffic_file(workload, kind)
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and line.startswith("- "):
                k, v = line[2:].split(":", 1)
                vals[k.strip()] = v.strip().strip("`")
    if vals.get(TRAFFIC_KINDS[kind][1]) != source_hash(kind):
        return None
    try:
        return float(vals["HBM bytes per launch"])
    except (KeyError, ValueError):
        return None


def summarize_traffic(fetch_dir, write_dir, workload, cmd_fetch, cmd_write, kind="gemm_fwd"):
    """Counter passes (FETCH_SIZE, WRITE_SIZE, KiB per dispatch) -> summary:
    the kind's dispatches averaged, each counter scaled by what it reads for
    the calibration copy of COPY_BYTES."""
    import glob
    import sqlite3

    def per_kernel(d, counter):
        out = {}
        for db in glob.glob(os.path.join(d, "**", "*.db"), recursive=True):
            con = sqlite3.connect(db)
            for name, cn, v in con.execute(
                    "select kernel_name, counter_name, value from counters_collection"):
                if cn == counter:
                    out.setdefault(name, []).append(v)
        return out

    def pick(d, pred):
        return [v for n, vs in d.items() if pred(n) for v in vs]

    fwd = TRAFFIC_KINDS[kind][2]
    copy = lambda n: "neg" in n
    f = per_kernel(fetch_dir, "FETCH_SIZE")
    w = per_kernel(write_dir, "WRITE_SIZE")
    ff, ww, fc, wc = pick(f, fwd), pick(w, fwd), pick(f, copy), pick(w, copy)
    if not (ff and ww and fc and wc):
        raise SystemExit(f"counter databases lack the {kind} or copy dispatches")
    k_fetch = COPY_BYTES / 1024 / (sum(fc) / len(fc))
    k_write = COPY_BYTES / 1024 / (sum(wc) / len(wc))
    fetch_kib = sum(ff) / len(ff)
    write_kib = sum(ww) / len(ww)
    total = (fetch_kib * k_fetch + write_kib * k_write) * 1024
    lines = [
        f"# HBM traffic of {TRAFFIC_KINDS[kind][3]} ({workload}), rocprofv3 counters",
        "",
        f"FETCH_SIZE pass: `{cmd_fetch}`",
        "",
        f"WRITE_SIZE pass: `{cmd_write}`",
        "",
        "Each counter is scaled by what it reads for a plain copy kernel of "
        f"{COPY_BYTES >> 20} MiB read and {COPY_BYTES >> 20} MiB written (`--copy-calibration`).",
        "",
        f"- {'forward' if kind == 'gemm_fwd' else kind} dispatches: {len(ff)}",
        f"- FETCH_SIZE KiB per dispatch: {fetch_kib:.1f}",
        f"- WRITE_SIZE KiB per dispatch: {write_kib:.1f}",
        f"- copy FETCH_SIZE KiB: {sum(fc) / len(fc):.1f} (factor {k_fetch:.4f})",
        f"- copy WRITE_SIZE KiB: {sum(wc) / len(wc):.1f} (factor {k_write:.4f})",
        f"- HBM bytes per launch: {total:.6e}",
        f"- {TRAFFIC_KINDS[kind][1]}: `{source_hash(kind)}`",
    ]
    with open(traffic_file(workload, kind), "w") as fo:
        fo.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_trace(db_path, steps, title, cmd):
    """Markdown summary of a rocprofv3 kernel trace (its rocpd database),
    restricted to the timed steps: every step launches the same kernels, so
    the step's length is the smallest window whose kernel multiset repeats
    over the last ``steps`` windows of the trace, and those windows are the
    timed steps."""
    import sqlite3
    con = sqlite3.connect(db_path)
    rows = con.execute("select name, start, end from kernels order by start").fetchall()
    period, drop = None, 0
    # trailing dispatches after the steps (the runtime's copy of the loss to
    # the host) are not part of the period
    from collections import Counter
    for drop in range(0, 16):
        names = [r[0] for r in rows[:len(rows) - drop]]
        for L in range(1, len(names) // (steps + 1) + 1):
            # the same kernels in each of the last `steps` windows (their order
            # may differ where a step forks work onto side streams)
            last = Counter(names[len(names) - L:])
            if all(Counter(names[len(names) - (i + 1) * L:len(names) - i * L]) == last
                   for i in range(1, steps)):
                period = L
                break
        if period:
            break
    if period is None:
        raise SystemExit("no repeating step found at the end of the trace")
    end = len(rows) - drop
    timed = rows[end - steps * period:end]
    agg = {}
    for name, t0, t1 in timed:
        a = agg.setdefault(name, [0, 0.0, float("inf"), 0.0])
        d = (t1 - t0) / 1e6
        a[0] += 1
        a[1] += d
        a[2] = min(a[2], d)
        a[3] = max(a[3], d)
    total = sum(a[1] for a in agg.values())
    span = (timed[-1][2] - timed[0][1]) / 1e6
    out = [f"# rocprofv3 kernel trace: {title}", "",
           f"Command: `{cmd}`", "",
           f"Table: the last {steps} steps of that run ({period} dispatches per step, "
           f"{steps * period} dispatches), grouped by kernel; warmup, input setup and "
           f"{drop} trailing dispatch(es) after the steps excluded.  "
           f"Kernel time per step {total / steps:.3f} ms; first-dispatch-start to "
           f"last-dispatch-end per step {span / steps:.3f} ms.", "",
           "| kernel | calls/step | ms/step | avg ms | min ms | max ms | % |",
           "|---|---|---|---|---|---|---|"]
    for name, (n, tot, mn, mx) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        short = name.replace("oq::(anonymous namespace)::", "").replace("unsigned short", "u16")
        short = short.split("(")[0] if "(" in short else short
        out.append(f"| {short[:110]} | {n / steps:g} | {tot / steps:.4f} | {tot / n:.4f} | "
                   f"{mn:.4f} | {mx:.4f} | {100 * tot / total:.1f} |")
    print("\n".join(out))


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def make_inputs(w, device="cuda"):
    import torch

    from paper_2308_13137_amd import inputs, oq
    dt = torch.bfloat16 if w.bf16 else torch.float32
    gen = torch.Generator(device=device)
    gen.manual_seed(inputs.SEED)
    X = []
    for s in w.sites:
        if w.x_recipe == "small":
            x = torch.randn((w.T, s.width), generator=gen, device=device)
        else:
            x = inputs.torch_activations(gen, w.T, s.width, dtype=dt, device=device)
        X.append(x.to(dt).contiguous())
    W = [inputs.torch_weights(gen, l.c_out, w.c_in(i), w.w_sigma, w.w_outlier, dtype=dt,
                              device=device).contiguous() for i, l in enumerate(w.linears)]
    Y = [oq.fp_target(X[l.site], W[i]) for i, l in enumerate(w.linears)]
    gl = [torch.full((l.c_out, w.c_in(i) // l.group), 4.0, device=device)
          for i, l in enumerate(w.linears)]
    bl = [g.clone() for g in gl]
    s, d = [], []
    for k, site in enumerate(w.sites):
        if site.let:
            Ws = [W[i] for i, l in enumerate(w.linears) if l.site == k]
            sk, dk = oq.let_init(X[k], Ws)
            s.append(sk)
            d.append(dk)
        else:
            s.append(None)
            d.append(None)
    return X, W, Y, gl, bl, s, d


def cpu_facts():
    """The host the CPU baseline ran on, and the threads it used: the fp64
    products run on BLAS threads, the oracle's elementwise numpy on one."""
    from threadpoolctl import threadpool_info
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    return {"cores": threads, "cores_note": "BLAS threads of the fp64 products; the "
            "oracle's elementwise code runs on one core", "nproc": os.cpu_count(),
            "affinity": len(os.sched_getaffinity(0)), "cpu_model": model}


def cpu_baseline(w, tokens):
    """Time the oracle's step on the same block at ``tokens`` tokens, then on
    an eighth of them with one BLAS thread (the one-core figure)."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    from oracle.block import block_step, fp_target
    from oracle.let import let_init
    from paper_2308_13137_amd import inputs
    import torch

    ws = w.with_tokens(tokens)

    def bf(a):
        return torch.from_numpy(a).to(torch.bfloat16).float().numpy() if ws.bf16 else a
    X = [bf(inputs.activations(inputs.rng_for(77, k), tokens, s.width)) for k, s in enumerate(ws.sites)]
    W = [bf(inputs.weights(inputs.rng_for(78, i), l.c_out, ws.c_in(i), ws.w_sigma, ws.w_outlier))
         for i, l in enumerate(ws.linears)]
    Y = [fp_target(X[l.site], W[i], None, bf16=ws.bf16) for i, l in enumerate(ws.linears)]
    gl = [np.full((l.c_out, ws.c_in(i) // l.group), 4.0, np.float32) for i, l in enumerate(ws.linears)]
    s = [let_init(X[k], [W[i] for i, l in enumerate(ws.linears) if l.site == k])[0] if st.let else None
         for k, st in enumerate(ws.sites)]
    d = [let_init(X[k], [W[i] for i, l in enumerate(ws.linears) if l.site == k])[1] if st.let else None
         for k, st in enumerate(ws.sites)]
    params = dict(W=W, B=[None] * len(W), gamma_logit=gl, beta_logit=[g.copy() for g in gl], s=s, delta=d)
    t0 = time.perf_counter()
    block_step(ws.oracle_desc(), X, Y, params)
    dt = time.perf_counter() - t0
    out = dict(cpu_facts(), value=round(tokens / dt, 3), unit="calibration tokens/s", kind="oracle",
               sample=f"one full {w.name} block step (all {len(w.linears)} linears, LWC fwd/bwd on "
                      f"every weight, fp64 products) at {tokens} tokens, {dt:.1f} s")
    t1 = max(tokens // 8, 64)
    ws1 = w.with_tokens(t1)
    X1 = [x[:t1] for x in X]
    Y1 = [y[:t1] for y in Y]
    with threadpool_limits(1):
        t0 = time.perf_counter()
        block_step(ws1.oracle_desc(), X1, Y1, params)
        dt1 = time.perf_counter() - t0
    out["one_core"] = {"value": round(t1 / dt1, 3), "unit": "calibration tokens/s",
                       "sample": f"the same step at its first {t1} tokens, one thread, {dt1:.1f} s"}
    return out


# The deployment workload (Sec. 4.5, Table "tab:speed"): one decoded token
# through the linears of all blocks of a LLaMA model (32 for 7B, 80 for
# 65B), weights stored as packed
# low-bit codes.  Linears that read the same input are stacked (q,k,v and
# gate,up), as a deployment would: 4 launches per block.
DECODE_MODELS = {
    # name: (blocks, hidden, ffn); LLaMA-1 shapes of the paper's speed table
    "llama7b": (32, 4096, 11008),
    "llama65b": (80, 8192, 22016),
}


def decode_linears(model):
    _, hid, ffn = DECODE_MODELS[model]
    return (("qkv", 3 * hid, hid), ("o", hid, hid), ("gate_up", 2 * ffn, hid), ("down", hid, ffn))


def decode_inputs(bits, group, model, n_tok, device="cuda"):
    """Seeded random packed codes (every code value equally likely), step
    sizes, zero points and activations, distinct for every block so that no
    block's weights are cached when the next one is read."""
    import torch

    from paper_2308_13137_amd import inputs
    gen = torch.Generator(device=device)
    gen.manual_seed(inputs.SEED + 5)
    lins = []
    for _ in range(DECODE_MODELS[model][0]):
        for name, c_out, c_in in decode_linears(model):
            P = torch.randint(0, 256, (c_out, c_in * bits // 8), generator=gen, device=device,
                              dtype=torch.uint8)
            h = torch.rand((c_out, c_in // group), generator=gen, device=device) * 0.02 + 1e-3
            z = torch.randint(0, 2 ** bits, (c_out, c_in // group), generator=gen,
                              device=device).float()
            lins.append((name, c_in, P, h, z))
    X = {c_in: inputs.torch_activations(gen, n_tok, c_in, dtype=torch.bfloat16, device=device)
         .contiguous() for c_in in {c for _, _, c in decode_linears(model)}}
    return lins, X


def decode_cpu_baseline(bits, group, model, min_seconds=10.0):
    """The oracle's packed linear on the first eighth of the rows of one
    block's four stacked linears, one token, repeated on fresh inputs until
    ``min_seconds`` have passed; rows are independent, so the time per pass
    scales by 8 to the block and by the block count to the model."""
    import numpy as np

    from oracle.packed import packed_linear
    rng = np.random.default_rng(5)
    dt, passes = 0.0, 0
    while dt < min_seconds:
        for name, c_out, c_in in decode_linears(model):
            rows = c_out // 8
            P = rng.integers(0, 256, size=(rows, c_in * bits // 8), dtype=np.uint8)
            h = rng.uniform(1e-3, 2.1e-2, size=(rows, c_in // group)).astype(np.float32)
            z = rng.integers(0, 2 ** bits, size=(rows, c_in // group)).astype(np.float32)
            x = rng.standard_normal((1, c_in))
            t0 = time.perf_counter()
            packed_linear(x, P, bits, group, h, z)
            dt += time.perf_counter() - t0
        passes += 1
    blocks = DECODE_MODELS[model][0]
    return dict(cpu_facts(), value=float(f"{passes / (8 * dt * blocks):.4g}"),
                unit="decoded tokens/s", kind="oracle",
                sample=f"{passes} pass(es) over one eighth of the rows of one block's four stacked "
                       f"linears, one token ({dt:.1f} s), scaled by 8 x {blocks} blocks")


def decode_name(args):
    name = f"{args.decode_model}_w{args.decode_bits}a16_g{args.decode_group}_decode"
    return name if args.decode_tokens == 1 else f"{name}_t{args.decode_tokens}"


def bench_decode(args):
    import torch

    from paper_2308_13137_amd import oq
    bits, group, n_tok = args.decode_bits, args.decode_group, args.decode_tokens
    torch.cuda.set_device(0)
    oq.lib()
    name = decode_name(args)
    n_blocks = DECODE_MODELS[args.decode_model][0]
    shapes = decode_linears(args.decode_model)
    log(f"[bench] {name}: {n_blocks} blocks x {len(shapes)} stacked linears, "
        f"{n_tok} token(s) per step")
    lins, X = decode_inputs(bits, group, args.decode_model, n_tok)
    outs = [torch.empty((n_tok, P.shape[0]), dtype=torch.float32, device="cuda")
            for _, _, P, _, _ in lins]

    def step():
        for (nm, c_in, P, h, z), y in zip(lins, outs):
            oq.packed_linear_into(X[c_in], P, bits, group, h, z, y)
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # kernel durations: eager steps, each launch bracketed by HIP events on its stream
    oq.profile_reset()
    oq.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    oq.profile_enable(False)
    n, kms, work = oq.profile_read()["packed_linear"]
    eager_ms = (t1 - t0) * 1e3 / args.steps
    # step time: a decode loop launches the same kernels for every token, so
    # the step is captured once in a HIP graph and replayed
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for _ in range(args.warmup):
        graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / args.steps
    # every launch of the replayed step is the packed linear, back to back on
    # the replay stream: the events around the replays over the launch count
    # give its average duration (events around each eager launch add their
    # own overhead to these few-microsecond kernels)
    launches = n / args.steps
    launch_ms = e0.elapsed_time(e1) / (args.steps * launches)
    achieved = work / n / (launch_ms / 1e3) / 1e9
    weight_bytes = sum(P.numel() + 8 * h.numel() for _, _, P, h, _ in lins)
    line = {
        "metric": "decoded tokens/s through the block linears (packed weights)",
        "value": round(n_tok / (ms / 1e3), 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "eager_ms_per_step": round(eager_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": name, "blocks": n_blocks, "tokens_per_step": n_tok,
                   "w_bits": bits, "group": group, "weight_bytes": weight_bytes,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "kernel": "packed_linear", "achieved": round(achieved, 1),
                     "peak": PEAK["hbm_gbs"], "unit": "GB/s",
                     "frac": round(achieved / PEAK["hbm_gbs"], 4),
                     "avg_launch_ms": round(launch_ms, 5),
                     "traffic": read_traffic(name, "packed_linear")},
        "kernels": {"packed_linear": {"launches_per_step": launches,
                                      "bytes_per_launch": round(work / n),
                                      "eager_event_bracketed_launch_ms": round(kms / n, 5)}},
    }
    # per shape: its 32 launches replayed from a graph, against a torch copy
    # of the same packed bytes (read + write): the practical streaming rate at
    # these launch sizes
    per_shape = {}
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for si, (nm, c_out, c_in) in enumerate(shapes):
        idx = [b * len(shapes) + si for b in range(n_blocks)]
        g_lin, g_cp = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_lin):
            for i in idx:
                _, _, P, h, z = lins[i]
                oq.packed_linear_into(X[c_in], P, bits, group, h, z, outs[i])
        dsts = [torch.empty_like(lins[i][2]) for i in idx]
        with torch.cuda.graph(g_cp):
            for i, d in zip(idx, dsts):
                d.copy_(lins[i][2])
        g_lin.replay()
        g_cp.replay()
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(5):
            g_lin.replay()
        ev[1].record()
        for _ in range(5):
            g_cp.replay()
        ev[2].record()
        torch.cuda.synchronize()
        lin_us = ev[0].elapsed_time(ev[1]) * 1e3 / (5 * len(idx))
        cp_us = ev[1].elapsed_time(ev[2]) * 1e3 / (5 * len(idx))
        _, _, P, h, _ = lins[idx[0]]
        nbytes = P.numel() + 8 * h.numel()
        per_shape[nm] = {"c_out": c_out, "c_in": c_in, "weight_bytes": nbytes,
                         "linear_us": round(lin_us, 2), "linear_gbs": round(nbytes / lin_us / 1e3, 1),
                         "copy_us": round(cp_us, 2),
                         "copy_gbs": round(2 * P.numel() / cp_us / 1e3, 1)}
        del g_lin, g_cp, dsts
    line["per_shape"] = per_shape
    del lins, X, outs
    torch.cuda.empty_cache()
    if args.copy_calibration:
        src = torch.ones(COPY_BYTES // 4, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        log("[bench] CPU oracle on one block")
        line["cpu_baseline"] = decode_cpu_baseline(bits, group, args.decode_model)
    else:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)


# The whole LLaMA block (Sec. 3.1 and 3.3): RMSNorm, the seven linears with
# LWC (and LET at three sites), RoPE, causal attention with the [Q, K] scale
# s_a and per-token Q/K/V quantisation, SiLU gating, residuals; the loss on the
# block output.  LLaMA-7B shapes, one 2048-token calibration sample per step
# by default (Algorithm 1's batch).
BLOCK_MODELS = {
    # name: (hidden, heads, kv_heads, ffn)
    "llama7b": (4096, 32, 32, 11008),
}


def block_name(args):
    g = "ch" if args.block_group == 0 else str(args.block_group)
    name = (f"{args.block_model}_block_w{args.block_bits}a{args.block_act_bits}_g{g}"
            f"{'_let' if args.block_let else ''}"
            f"{f'_p{args.block_softmax_bits}' if args.block_softmax_bits < 16 else ''}")
    return name if args.block_tokens == args.block_seq else f"{name}_t{args.block_tokens}"


def block_inputs(args, device="cuda"):
    """Seeded synthetic block on the GPU: bf16 weights N(0, 0.02) with 0.1%
    x10 outliers, bf16 inputs with 1% heavy-tailed outlier channels (RMS 1 per
    token), norm gains U(0.8, 1.2), clipping logits 4 (sigmoid 0.982), LET at
    its identity (s = 1, delta = 0, s_a = 1), the target the block's own
    full-precision output."""
    import torch

    from paper_2308_13137_amd import inputs, oq
    D, H, Hkv, F = BLOCK_MODELS[args.block_model]
    d = D // H
    T = args.block_tokens
    gen = torch.Generator(device=device)
    gen.manual_seed(inputs.SEED + 7)
    shapes = [(H * d, D), (Hkv * d, D), (Hkv * d, D), (D, H * d), (F, D), (F, D), (D, F)]
    W = [inputs.torch_weights(gen, a, b, 0.02, 0.001, dtype=torch.bfloat16, device=device).contiguous()
         for a, b in shapes]
    h0 = inputs.torch_activations(gen, T, D, dtype=torch.bfloat16, device=device).contiguous()
    g1 = 0.8 + 0.4 * torch.rand(D, generator=gen, device=device)
    g2 = 0.8 + 0.4 * torch.rand(D, generator=gen, device=device)
    groups = [b if args.block_group == 0 else args.block_group for _, b in shapes]
    gl = [torch.full((a, b // g), 4.0, device=device) for (a, b), g in zip(shapes, groups)]
    bl = [t.clone() for t in gl]
    let = None
    if args.block_let:
        sw = [D, H * d, D]
        let = dict(s=[torch.ones(n, device=device) for n in sw],
                   delta=[torch.zeros(n, device=device) for n in sw],
                   s_a=torch.ones(Hkv * d, device=device))
    blk = oq.LlamaBlock(T, args.block_seq, D, H, Hkv, F, [args.block_bits] * 7, groups,
                        act_bits=args.block_act_bits, let=args.block_let,
                        softmax_bits=args.block_softmax_bits)
    target = blk.forward(h0, W, g1, g2, quantised=False)
    return blk, h0, target, W, g1, g2, gl, bl, let, groups


def block_cpu_baseline(args, groups):
    """The oracle's whole-block step on one calibration sample of the same
    block (all seven linears at full width, attention over the sample)."""
    import numpy as np

    from oracle import llama_block as lb
    from paper_2308_13137_amd import inputs
    D, H, Hkv, F = BLOCK_MODELS[args.block_model]
    d = D // H
    T = args.block_seq
    rng = inputs.rng_for(79, T)
    import torch

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).float().numpy()
    shapes = [(H * d, D), (Hkv * d, D), (Hkv * d, D), (D, H * d), (F, D), (F, D), (D, F)]
    W = [bf(inputs.weights(rng, a, b, 0.02, 0.001)) for a, b in shapes]
    desc = dict(hidden=D, heads=H, kv_heads=Hkv, ffn=F, seq_len=T, norm_eps=1e-6, rope_base=10000.0,
                w_bits=[args.block_bits] * 7, w_group=groups, act_bits=args.block_act_bits,
                let=args.block_let, softmax_bits=args.block_softmax_bits)
    gl = [np.full((a, b // g), 4.0, np.float32) for (a, b), g in zip(shapes, groups)]
    p = dict(W=W, gamma_logit=gl, beta_logit=[g.copy() for g in gl],
             g1=np.ones(D, np.float32), g2=np.ones(D, np.float32),
             s=[np.ones(n, np.float32) for n in (D, H * d, D)],
             delta=[np.zeros(n, np.float32) for n in (D, H * d, D)], s_a=np.ones(Hkv * d, np.float32))
    h0 = bf(inputs.activations(rng, T, D))
    target = bf(lb.fp_block(desc, h0, p))
    t0 = time.perf_counter()
    lb.block_step(desc, h0, target, p)
    dt = time.perf_counter() - t0
    return dict(cpu_facts(), value=round(T / dt, 3), unit="calibration tokens/s", kind="oracle",
                sample=f"one whole-block step of the same block on one {T}-token sample "
                       f"(fp64 products, fp32 quantisers), {dt:.1f} s")


def bench_block(args):
    import torch

    from paper_2308_13137_amd import oq
    torch.cuda.set_device(0)
    oq.lib()
    name = block_name(args)
    log(f"[bench] {name}: T={args.block_tokens} in samples of {args.block_seq}")
    blk, h0, target, W, g1, g2, gl, bl, let, groups = block_inputs(args)
    blk.init_optimizer()
    kw = dict(let) if let else {}

    def step():
        blk.step(h0, target, W, g1, g2, gl, bl, update=True, **kw)
    torch.cuda.synchronize()
    log(f"[bench] inputs resident, workspace {blk.ws_bytes / 2**30:.2f} GiB; warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # the timed steps run without per-launch events: at about 85 launches in
    # 5 ms the two event records around each launch add about 6% to the step
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / args.steps
    # the same number of steps again with the events, for the per-kernel
    # breakdown and the roofline
    oq.profile_reset()
    oq.profile_enable(True)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    oq.profile_enable(False)
    prof = oq.profile_read()
    loss = float(blk.loss.cpu())
    ms_prof = (t3 - t2) * 1e3 / args.steps
    kernels = {}
    for kind, (n, kms, work) in prof.items():
        if n == 0:
            continue
        ent = {"launches_per_step": n / args.steps, "ms_per_step": round(kms / args.steps, 4)}
        if kind in GEMM_KINDS or kind.startswith("attn"):
            ent["tflops"] = round(work / (kms / 1e3) / 1e12, 1)
        elif work > 0:
            ent["gbs"] = round(work / (kms / 1e3) / 1e9, 1)
        kernels[kind] = ent
    dom = max(prof, key=lambda k: prof[k][1])
    n, kms, work = prof[dom]
    if dom in GEMM_KINDS or dom.startswith("attn"):
        achieved = work / n / (kms / n / 1e3) / 1e12
        roof = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 1),
                "peak": PEAK["mfma_bf16_tflops"], "unit": "TFLOP/s"}
    else:
        achieved = work / n / (kms / n / 1e3) / 1e9
        roof = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1),
                "peak": PEAK["hbm_gbs"], "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["avg_launch_ms"] = round(kms / n, 4)
    roof["traffic"] = None
    D, H, Hkv, F = BLOCK_MODELS[args.block_model]
    line = {
        "metric": "calibration tokens/s per whole-block fwd+bwd step",
        "value": round(args.block_tokens / (ms / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": name, "tokens_per_step": args.block_tokens,
                   "seq_len": args.block_seq, "hidden": D, "heads": H, "kv_heads": Hkv, "ffn": F,
                   "w_bits": args.block_bits, "group": args.block_group or "per-channel",
                   "act_bits": args.block_act_bits, "let": args.block_let,
                   "softmax_bits": args.block_softmax_bits,
                   "parallelism": "single GPU"},
        "loss": loss,
        "profiled_ms_per_step": round(ms_prof, 3),
        "block_seconds_at_20_epochs_128_samples": round(20 * 128 * args.block_seq / args.block_tokens
                                                       * ms / 1e3, 2),
        "roofline": roof,
        "kernels": kernels,
    }
    del blk, h0, target, W, gl, bl
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log("[bench] CPU oracle on one sample of the block")
        line["cpu_baseline"] = block_cpu_baseline(args, groups)
    else:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="llama7b_w3a16_g128")
    ap.add_argument("--tokens", type=int, default=None, help="tokens per step (default: the workload's)")
    ap.add_argument("--cpu-tokens", type=int, default=16384)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--step-times", action="store_true",
                    help="also report each timed step's duration (events between steps)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed steps, run a plain copy of known size (counter scale)")
    ap.add_argument("--summarize-traffic", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "CMD_FETCH",
                                                             "CMD_WRITE"),
                    help="write the HBM traffic summary from two rocprofv3 --pmc passes")
    ap.add_argument("--schedule", type=int, default=0, metavar="EPOCHS",
                    help="time Algorithm 1's loop instead: EPOCHS passes over the workload's "
                         "tokens as segments of --segment-tokens, one step per segment, in one "
                         "oq_block_calibrate call")
    ap.add_argument("--segment-tokens", type=int, default=2048)
    ap.add_argument("--decode", action="store_true",
                    help="time the deployment workload instead: packed-weight linears of "
                         "all blocks of --decode-model for one decoded token per step")
    ap.add_argument("--decode-model", default="llama7b", choices=sorted(DECODE_MODELS))
    ap.add_argument("--decode-bits", type=int, default=4)
    ap.add_argument("--decode-group", type=int, default=128)
    ap.add_argument("--decode-tokens", type=int, default=1)
    ap.add_argument("--block", action="store_true",
                    help="time the whole LLaMA block's step instead (attention, norms, RoPE, "
                         "SiLU, residuals and the seven quantised linears)")
    ap.add_argument("--block-model", default="llama7b", choices=sorted(BLOCK_MODELS))
    ap.add_argument("--block-bits", type=int, default=4)
    ap.add_argument("--block-group", type=int, default=0, help="0: per output channel")
    ap.add_argument("--block-act-bits", type=int, default=4)
    ap.add_argument("--block-let", type=int, default=1)
    ap.add_argument("--block-softmax-bits", type=int, default=16,
                    help="2..8: quantise the softmax output too (16: not)")
    ap.add_argument("--block-seq", type=int, default=2048)
    ap.add_argument("--block-tokens", type=int, default=2048)
    ap.add_argument("--summarize-trace", nargs=3, metavar=("DB", "TITLE", "CMD"),
                    help="print the per-kernel summary of a rocprofv3 trace over the last "
                         "--steps steps")
    args = ap.parse_args()
    args.block_let = bool(args.block_let)
    if args.summarize_trace:
        summarize_trace(args.summarize_trace[0], args.steps, *args.summarize_trace[1:])
        return
    if args.summarize_traffic:
        if args.decode:
            summarize_traffic(*args.summarize_traffic[:2], decode_name(args),
                              *args.summarize_traffic[2:], kind="packed_linear")
            return
        w = args.config if not args.tokens else f"{args.config}_t{args.tokens}"
        summarize_traffic(*args.summarize_traffic[:2], w, *args.summarize_traffic[2:])
        return
    if args.decode and args.gpus == 1:
        bench_decode(args)
        return
    if args.block and args.gpus == 1:
        bench_block(args)
        return

    if args.gpus != 1:
        print(f"bench.py measures the calibration step on one GPU; --gpus {args.gpus} is not "
              "supported (the step is single-GPU; sharding is described, not run).", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2308_13137_amd import configs, oq

    w = configs.BY_NAME[args.config]
    if args.tokens:
        w = w.with_tokens(args.tokens)
    torch.cuda.set_device(0)
    oq.lib()
    log(f"[bench] {w.name}: T={w.T}, {len(w.linears)} linears, {w.n_params / 1e6:.1f} M weights")
    X, W, Y, gl, bl, s, d = make_inputs(w)
    dt = torch.bfloat16 if w.bf16 else torch.float32
    T_step, n_seg = w.T, 1
    if args.schedule:
        # Algorithm 1's schedule: the same tokens as segments of T_step, one
        # step per segment, LET initialised over all of them (make_inputs)
        T_step = args.segment_tokens
        n_seg = w.T // T_step
        Xs = [[x[g * T_step:(g + 1) * T_step] for x in X] for g in range(n_seg)]
        del Y
        torch.cuda.empty_cache()
        Ys = [[oq.fp_target(xs[l.site], W[i]) for i, l in enumerate(w.linears)] for xs in Xs]
        X, Y = Xs[0], Ys[0]
    blk = oq.Block(T_step, [(st.width, st.let, st.act_bits) for st in w.sites],
                   [(l.site, l.c_out, l.bits, l.group) for l in w.linears], dtype=dt)
    blk.init_optimizer()
    torch.cuda.synchronize()
    log(f"[bench] inputs resident, workspace {blk.ws_bytes / 2**30:.1f} GiB; warmup {args.warmup}")
    for _ in range(args.warmup):
        blk.step(X, Y, W, gl, bl, s=s, delta=d, update=True)
    torch.cuda.synchronize()
    steps = args.schedule * n_seg if args.schedule else args.steps
    log(f"[bench] timing {steps} steps")

    oq.profile_reset()
    oq.profile_enable(True)
    torch.cuda.synchronize()
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)] \
        if args.step_times else None
    t0 = time.perf_counter()
    if args.schedule:
        losses = blk.calibrate(Xs, Ys, W, gl, bl, epochs=args.schedule, s=s, delta=d)
    else:
        for i in range(args.steps):
            if marks:
                marks[i].record()
            blk.step(X, Y, W, gl, bl, s=s, delta=d, update=True)
        if marks:
            marks[-1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    oq.profile_enable(False)
    prof = oq.profile_read()
    loss = float(losses[-1].cpu()) if args.schedule else float(blk.loss.cpu())

    ms = (t1 - t0) * 1e3 / steps
    value = T_step / (ms / 1e3)

    kernels = {}
    for kind, (n, kms, work) in prof.items():
        if n == 0:
            continue
        ent = {"launches_per_step": n / steps, "ms_per_step": round(kms / steps, 4)}
        if kind in GEMM_KINDS:
            ent["tflops"] = round(work / (kms / 1e3) / 1e12, 1)
        elif work > 0:
            ent["gbs"] = round(work / (kms / 1e3) / 1e9, 1)
        kernels[kind] = ent
    dom = max(prof, key=lambda k: prof[k][1])
    n, kms, work = prof[dom]
    if dom in GEMM_KINDS:
        achieved = work / n / (kms / n / 1e3) / 1e12
        roof = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 1),
                "peak": PEAK["mfma_bf16_tflops"] if w.bf16 else PEAK["fp32_tflops"],
                "unit": "TFLOP/s"}
    else:
        achieved = work / n / (kms / n / 1e3) / 1e9
        roof = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1),
                "peak": PEAK["hbm_gbs"], "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["avg_launch_ms"] = round(kms / n, 4)
    roof["traffic"] = None
    if dom == "gemm_fwd" and not args.schedule:
        tb = read_traffic(args.config if not args.tokens else f"{args.config}_t{args.tokens}")
        if tb is not None:
            roof["traffic"] = tb          # HBM bytes per launch (counter passes, copy-scaled)

    line = {
        "metric": ("calibration tokens/s, one step per calibration segment" if args.schedule
                   else "calibration tokens/s per block fwd+bwd step"),
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.bf16 else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "tokens_per_step": T_step, "linears": len(w.linears),
                   "weights": w.n_params, "w_bits": w.linears[0].bits,
                   "group": w.linears[0].group, "let": any(st.let for st in w.sites),
                   "act_bits": w.sites[0].act_bits, "parallelism": "single GPU"},
        "loss": loss,
        "roofline": roof,
        "kernels": kernels,
    }
    if args.schedule:
        line["config"].update(segments=n_seg, epochs=args.schedule)
        line["block_seconds_at_20_epochs"] = round(20 * n_seg * ms / 1e3, 3)
        line["first_last_loss"] = [float(losses[0].cpu()), loss]
    if marks:
        line["step_ms"] = [round(marks[i].elapsed_time(marks[i + 1]), 3) for i in range(args.steps)]
    if args.copy_calibration:
        src = torch.ones(COPY_BYTES // 4, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        del X, W, Y, blk
        torch.cuda.empty_cache()
        log(f"[bench] CPU oracle on a {args.cpu_tokens}-token sample")
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_tokens)
    else:
        line["cpu_baseline"] = None
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
