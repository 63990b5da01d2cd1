#!/usr/bin/env python3
"""Decode throughput of parallel decoding vs greedy decoding on one MI355X.

Headline workload: the large multilingual-shaped model (12+12 layers,
d = 1024, 16 heads, FFN 4096 GELU, pre-LN, vocabulary 250,027, bf16) with
seeded random weights, batch 1 (the paper's online setting), sources of
n ~ U[20, 120] tokens and m = min(n + 10, 256) target positions (50 sentences
plus one with m = 256).  A step is the decode of one sentence (pd_decode,
batch 1) with its source already encoded and resident in HBM; the timed region
covers the first K sentences (--steps), after W warm-up decodes (--warmup) of
the same first sentences.  Every mode decodes the same K sentences.

One JSON line on stdout: value = target tokens/s of GS-Jacobi b = 16, next to
greedy decoding, Jacobi and hybrid b = 16 with their k/m; the roofline of the
time-dominant kernel family (the decoder's streaming matrix products) and of
the fused vocabulary projection + argmax, from the kernels' own dispatch
timestamps; the block-iteration / greedy-step cost ratio and the break-even
k/m it implies; the CPU oracle baseline on the host cores; and, as side
records, the Transformer-base-shaped model at batch 1 (float32 and bfloat16),
the tiny model's iteration latency, and the batched workloads.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0   # dense bf16 matrix peak of MI355X
HEADLINE = ("gs_jacobi", 16)
# (mode, block[, stopping condition]); "prefix" is PD_STOP_PREFIX, the
# stopping-condition variant (the default is Eq. (3))
LARGE_MODES = [("ar", 1), ("jacobi", 0), ("gs_jacobi", 16), ("hybrid", 16), ("gs_jacobi", 16, "prefix")]
MT_MODES = [("ar", 1), ("jacobi", 0), ("gs_jacobi", 5), ("hybrid", 5), ("gs_jacobi", 5, "prefix"),
            ("hybrid", 5, "prefix"), ("jacobi", 0, "prefix")]


def mode_key(spec):
    mode, b = spec[0], spec[1]
    stop = spec[2] if len(spec) > 2 else "block"
    return f"{mode}_b{b}" + ("" if stop == "block" else f"_{stop}")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


_MODELS = {}


def load_model(cfg):
    """Seed-0 weights of a model shape and their device copy, drawn once per run."""
    from paper_2305_10427_amd import pdec, synth
    if cfg not in _MODELS:
        w = synth.make_weights(cfg, seed=0)
        _MODELS[cfg] = (w, pdec.Model(cfg, w))
    return _MODELS[cfg]


def run_mode(ctxs, sents, outs, mode, block, steps, warmup, timing=False, stop="block"):
    """Decodes sentences 0..steps-1 (each its own context, already encoded)
    after warm-up decodes of sentences 0..warmup-1; returns the timed totals."""
    import torch
    n = len(sents)
    assert steps <= n, f"{steps} steps but only {n} sentences"
    # one-time setup: every context captures and instantiates its iteration
    # graph for this mode on its first decode
    for i in range(steps):
        ctxs[i].decode(mode, [sents[i][1]], block=block, out=outs[i], stop=stop)
    torch.cuda.synchronize()
    for i in range(warmup):
        ctxs[i % steps].decode(mode, [sents[i % steps][1]], block=block, out=outs[i % steps], stop=stop)
    torch.cuda.synchronize()
    if timing:
        for c in ctxs[:steps]:
            c.set_timing(True)
    t0 = time.perf_counter()
    for i in range(steps):
        ctxs[i].decode(mode, [sents[i][1]], block=block, out=outs[i], stop=stop)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    toks = ks = ms = 0
    for i in range(steps):
        toks += int(outs[i][1][0])
        ks += int(outs[i][2][0])
        ms += sents[i][1]
    res = {"tokens": toks, "seconds": dt, "tokens_per_s": toks / dt, "k": ks, "m": ms, "k_over_m": ks / ms,
           "ms_per_step": 1e3 * dt / steps, "us_per_iteration": 1e6 * dt / ks,
           "kernels_per_iteration": ctxs[0].iteration_kernels()}
    if timing:
        v_n = v_ms = p_n = p_ms = p_b = 0
        for c in ctxs[:steps]:
            n_l, t_ms = c.vocab_timing()
            q_n, q_ms, q_b = c.product_timing()
            v_n, v_ms, p_n, p_ms, p_b = v_n + n_l, v_ms + t_ms, p_n + q_n, p_ms + q_ms, p_b + q_b
            c.set_timing(False)
        res.update(vocab_launches=v_n, vocab_ms=v_ms, product_launches=p_n, product_ms=p_ms, product_bytes=p_b)
    return res


def setup_batch1(wl_name, n_sent):
    import torch
    from paper_2305_10427_amd import configs as C, pdec, synth
    wl = C.WORKLOADS[wl_name]
    t0 = time.perf_counter()
    w, model = load_model(wl.model)
    sents = synth.make_sentences(wl, seed=1)[:n_sent]
    max_src = max(len(s) for s, _ in sents)
    ctxs, outs = [], []
    for src, m in sents:
        c = pdec.Context(model, 1, max_src, wl.tgt_cap)
        c.encode(torch.from_numpy(src[None]).cuda(), [len(src)])
        ctxs.append(c)
        outs.append((torch.empty((1, wl.tgt_cap), dtype=torch.int32, device="cuda"),
                     torch.empty(1, dtype=torch.int32, device="cuda"),
                     torch.empty(1, dtype=torch.int32, device="cuda"),
                     torch.empty(1, dtype=torch.int32, device="cuda")))
    torch.cuda.synchronize()
    log(f"[{wl_name}] weights {model.weight_bytes() / 1e6:.1f} MB, {len(sents)} sentences encoded "
        f"in {time.perf_counter() - t0:.1f}s")
    return wl, w, model, sents, ctxs, outs


def encode_rate(ctxs, sents, cfg, steps, warmup):
    """pd_encode of one source per call (batch 1), the step before the
    decoding iterations: wall time per sentence over `steps` calls, against
    the weights it must read (encoder layers and every decoder layer's
    cross-attention K/V projection)."""
    import torch
    n = len(sents)
    srcs = [torch.from_numpy(src[None]).cuda() for src, _ in sents]
    torch.cuda.synchronize()
    for i in range(warmup):
        ctxs[i % n].encode(srcs[i % n], [len(sents[i % n][0])])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        ctxs[i % n].encode(srcs[i % n], [len(sents[i % n][0])])
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    es = 2 if cfg.dtype == "bf16" else 4
    d, f = cfg.d_model, cfg.d_ff
    wbytes = (cfg.n_enc * (4 * d * d + 2 * d * f + 9 * d + f) + cfg.n_dec * (2 * d * d + 2 * d)) * es
    return {"us_per_sentence": round(1e6 * dt, 2), "weight_bytes": wbytes,
            "achieved": round(wbytes / dt / 1e9, 1), "unit": "GB/s", "frac": round(wbytes / dt / 1e9 / HBM_PEAK_GBS, 4)}


def mode_table(res):
    return {k: {"tokens_per_s": round(v["tokens_per_s"], 1), "k_over_m": round(v["k_over_m"], 4),
                "ms_per_sentence": round(v["ms_per_step"], 3), "us_per_iteration": round(v["us_per_iteration"], 2),
                "kernels_per_iteration": v["kernels_per_iteration"]} for k, v in res.items()}


def cost_ratio(res, block_key):
    """Wall time of one iteration of the block mode against one greedy step.
    The block mode decodes m tokens in k iterations, greedy decoding in m
    steps, so it is faster exactly when k/m < greedy step / block iteration."""
    it_b = res[block_key]["us_per_iteration"]
    it_g = res["ar_b1"]["us_per_iteration"]
    return {"mode": block_key, "block_iteration_us": round(it_b, 2), "greedy_step_us": round(it_g, 2),
            "ratio": round(it_b / it_g, 3), "break_even_k_over_m": round(it_g / it_b, 3),
            "measured_k_over_m": round(res[block_key]["k_over_m"], 4)}


def source_sha(files):
    return hashlib.sha256(b"".join(open(os.path.join(ROOT, "paper_2305_10427_amd", "csrc", f), "rb").read()
                                   for f in files)).hexdigest()


def measured_traffic(name):
    """HBM bytes per launch from a committed rocprofv3 counter record
    (profiles/<name>.json), or None once the kernel sources it covers changed."""
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", name + ".json")))
        if source_sha(rec["kernel_sources"]) != rec["kernel_source_sha256"]:
            return None
        return rec["traffic_bytes_per_launch"]
    except (OSError, KeyError, ValueError):
        return None


KERNEL_SOURCES = ["gemm.hip", "vocab.hip", "mma.h", "common.h", "kernels.h"]


def rooflines(cfg, t):
    """The decoder's streaming products (time-dominant at batch 1) and the
    fused vocabulary kernel of the event-timed pass."""
    p_avg = t["product_ms"] / max(t["product_launches"], 1)
    p_bytes = t["product_bytes"] / max(t["product_launches"], 1)
    p_ach = p_bytes / (p_avg * 1e-3) / 1e9 if p_avg > 0 else 0.0
    v_bytes = cfg.vocab * (cfg.d_model + 1) * (2 if cfg.dtype == "bf16" else 4)
    v_avg = t["vocab_ms"] / max(t["vocab_launches"], 1)
    v_ach = v_bytes / (v_avg * 1e-3) / 1e9 if v_avg > 0 else 0.0
    tag = cfg.name.split("@")[0]
    products = {"kernel": "k_gemm (the decoder's streaming matrix products: QKV, attention output, cross-attention "
                          "query and output, FFN; every launch of the timed iterations)",
                "bound": "hbm", "achieved": round(p_ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(p_ach / HBM_PEAK_GBS, 4), "traffic": measured_traffic(f"gemm_products_{tag}"),
                "avg_launch_us": round(p_avg * 1e3, 2), "launches": t["product_launches"],
                "bytes_per_launch": round(p_bytes), "ms_per_iteration": round(t["product_ms"] / max(t["k"], 1), 4)}
    vocab = {"kernel": "k_vocab (streaming vocabulary projection + LayerNorm + argmax, <= 16 rows)", "bound": "hbm",
             "achieved": round(v_ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(v_ach / HBM_PEAK_GBS, 4),
             "traffic": measured_traffic(f"vocab_argmax_{tag}"), "avg_launch_us": round(v_avg * 1e3, 2),
             "launches": t["vocab_launches"], "bytes_per_launch": v_bytes}
    return products, vocab


def iteration_roofline(cfg, res):
    d, f, L = cfg.d_model, cfg.d_ff, cfg.n_dec
    es = 2 if cfg.dtype == "bf16" else 4
    it_bytes = (L * (6 * d * d + 2 * d * f + 13 * d + f) + cfg.vocab * (d + 1)) * es
    us = res["us_per_iteration"]
    return {"us": round(us, 2), "bytes": it_bytes, "achieved": round(it_bytes / us / 1e3, 1), "unit": "GB/s",
            "frac": round(it_bytes / us / 1e3 / HBM_PEAK_GBS, 4),
            "note": "one decoding iteration (every kernel of the decoder pass, vocabulary and control step) at "
                    "batch 1, against the weight bytes it must read"}


def host_threads():
    info = {"os_cpu_count": os.cpu_count(), "affinity": len(os.sched_getaffinity(0))}
    try:
        from threadpoolctl import threadpool_info
        info["blas_threads"] = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:                       # noqa: BLE001
        info["blas_threads"] = None
    return info


def cpu_baseline(wl, w, sents, ctxs, mode, block, m_cap, n_sent):
    """The oracle as it stands (float64) and the same code in float32, on all
    host threads and on one, over a bounded sample: the first n_sent sentences
    with their targets cut to m_cap positions.  The GPU decodes the same cut
    sentences; their ids and k are compared with the float64 oracle's
    (exact / near tie)."""
    import numpy as np
    import torch
    import oracle
    from threadpoolctl import threadpool_limits
    cfg = wl.model
    sample = [(src, min(m, m_cap)) for src, m in sents[:n_sent]]
    host = host_threads()
    out = {"sample": f"the first {n_sent} sentence(s) of the same workload with m cut to {m_cap}, {mode} b={block}, "
                     "decode only (encoder excluded)", "host": host, "variants": {}}
    results = None
    for dt_name, dtype in (("f64", np.float64), ("f32", np.float32)):
        M = oracle.Model(cfg, w.values, dtype=dtype)
        encs = [M.encode(src) for src, _ in sample]
        for threads in ("all", 1):
            lim = host["blas_threads"] if threads == "all" else 1
            with threadpool_limits(limits=lim):
                toks, t0 = 0, time.perf_counter()
                res = []
                for enc, (_, m) in zip(encs, sample):
                    r = oracle.decode(M, enc, m, mode, block)
                    toks += len(r.out)
                    res.append(r)
                dt = time.perf_counter() - t0
            out["variants"][f"{dt_name}_{threads}_threads" if threads == "all" else f"{dt_name}_1_thread"] = {
                "tokens_per_s": round(toks / dt, 2), "threads": lim, "seconds": round(dt, 2)}
            log(f"[cpu] oracle {dt_name} on {lim} thread(s): {toks / dt:.2f} tok/s ({dt:.1f}s)")
            if dt_name == "f64" and threads == "all":
                results = res
        del M
    v = out["variants"]["f64_all_threads"]
    out.update(value=v["tokens_per_s"], unit="tokens/s", cores=v["threads"], kind="oracle")
    # the GPU's decodes of the same cut sentences against the float64 oracle
    exact = near = 0
    for i, ((src, m), r) in enumerate(zip(sample, results)):
        ids, ln, k, fl = ctxs[i].decode(mode, [m], block=block)
        torch.cuda.synchronize()
        g = ids[0, : int(ln[0])].cpu().numpy()
        if np.array_equal(g, r.out) and int(k[0]) == r.k:
            exact += 1
        else:
            near += 1
    # argmaxes of the float64 oracle on the sample whose top-2 margin lies
    # within the logit tolerance (5e-2 of max|logit| in bf16, 1e-3 in fp32):
    # the decisions a correct GPU path may take either way
    tol = 5e-2 if cfg.dtype == "bf16" else 1e-3
    n_arg = sum(len(r.records) for r in results)
    n_tie = sum(1 for r in results for rec in r.records if rec.top1 - rec.top2 < tol * max(rec.linf, 1e-30))
    out["parity_sample"] = {"sentences": len(sample), "exact": exact, "not_exact": near,
                            "argmaxes": n_arg, "near_ties": n_tie, "near_tie_margin": tol,
                            "note": "ids and k of the GPU against the float64 oracle on the baseline sample; "
                                    "near_ties: oracle argmaxes whose top-2 margin is below near_tie_margin x "
                                    "max|logit|; the GPU tests judge every difference"}
    return out


def tiny_latency(steps):
    """The tiny 2+2 model (d = 64, V = 1000, fp32, n = m = 16): every mode over
    its first `steps` sentences; the iteration is launch-bound, so the figures
    are microseconds per iteration and kernels per iteration."""
    wl, _, _, sents, ctxs, outs = setup_batch1("tiny", min(steps, 100))
    res = {}
    for mode, b in wl.modes:
        r = run_mode(ctxs, sents, outs, mode, b, len(sents), 5)
        res[f"{mode}_b{b}"] = r
        log(f"[tiny] {mode:9s} b={b:2d}: {r['us_per_iteration']:7.2f} us/iteration, "
            f"{r['kernels_per_iteration']} kernels/iteration, k/m={r['k_over_m']:.3f}")
    return {"workload": f"tiny 2+2 layers, d=64, V=1000, fp32, batch 1, first {len(sents)} sources, n=m=16",
            **mode_table(res)}


def batch1_workload(wl_name, steps, warmup, modes, headline, trace=False, encode=False):
    wl, w, model, sents, ctxs, outs = setup_batch1(wl_name, max(steps, warmup))
    cfg = wl.model
    res = {}
    for spec in modes:
        mode, b = spec[0], spec[1]
        r = run_mode(ctxs, sents, outs, mode, b, steps, warmup, stop=spec[2] if len(spec) > 2 else "block")
        res[mode_key(spec)] = r
        log(f"[{wl_name}] {mode_key(spec):18s}: {r['tokens_per_s']:9.1f} tok/s  {r['ms_per_step']:8.3f} ms/sentence  "
            f"k/m={r['k_over_m']:.3f}  {r['us_per_iteration']:7.1f} us/iteration")
    # the event-timed pass of the headline mode: dispatch timestamps of every
    # decoder product and vocabulary launch (iterations launched kernel by
    # kernel); the throughput above comes from the graph-replayed pass
    timed = run_mode(ctxs, sents, outs, headline[0], headline[1], steps, warmup, timing=True)
    extra = {}
    if encode:
        extra["encode"] = encode_rate(ctxs, sents[:steps], cfg, steps, warmup)
        log(f"[{wl_name}] encode: {extra['encode']['us_per_sentence']:.1f} us/sentence")
    if trace:
        for c in ctxs:
            c.set_trace(4 * wl.tgt_cap, max(headline[1], 1))
        t = run_mode(ctxs, sents, outs, headline[0], headline[1], steps, warmup)
        for c in ctxs:
            c.set_trace(0, 0)
        h = res[f"{headline[0]}_b{headline[1]}"]
        extra["trace"] = {"mode": f"{headline[0]}_b{headline[1]}", "tokens_per_s": round(t["tokens_per_s"], 1),
                          "slowdown": round(h["tokens_per_s"] / t["tokens_per_s"], 3)}
    return wl, w, sents, ctxs, res, timed, extra


def batched_workload(wl_name, n_batches, modes, repeats):
    """Batched decoding (sentences padded to the batch maximum and decoded
    together, each with its own iteration state): target tokens/s and k/m per
    mode over the first n_batches batches of the workload."""
    import torch
    from paper_2305_10427_amd import configs as C, pdec, synth
    wl = C.WORKLOADS[wl_name]
    cfg = wl.model
    _, model = load_model(cfg)
    batches = synth.make_batches(synth.make_sentences(wl, seed=1)[: n_batches * wl.batch], wl.batch)
    ctxs, outs = [], []
    for bt in batches:
        c = pdec.Context(model, wl.batch, bt.src.shape[1], wl.tgt_cap)
        c.encode(torch.from_numpy(bt.src).cuda(), bt.src_len.tolist())
        ctxs.append(c)
        B = len(bt.src_len)
        outs.append((torch.empty((B, wl.tgt_cap), dtype=torch.int32, device="cuda"),
                     torch.empty(B, dtype=torch.int32, device="cuda"),
                     torch.empty(B, dtype=torch.int32, device="cuda"),
                     torch.empty(B, dtype=torch.int32, device="cuda")))
    torch.cuda.synchronize()
    res = {}
    for mode, b in modes:
        for c, bt, o in zip(ctxs, batches, outs):       # graph capture + warm-up
            c.decode(mode, bt.tgt_m.tolist(), block=b, out=o)
        torch.cuda.synchronize()
        toks = ks = ms = 0
        t0 = time.perf_counter()
        for _ in range(repeats):
            for c, bt, o in zip(ctxs, batches, outs):
                c.decode(mode, bt.tgt_m.tolist(), block=b, out=o)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        for bt, o in zip(batches, outs):
            toks += int(o[1].sum()) * repeats
            ks += int(o[2].sum()) * repeats
            ms += int(bt.tgt_m.sum()) * repeats
        # a separate pass with HIP events around the vocabulary launch and the
        # device count of rows evaluated: its MFMA rate
        for c in ctxs:
            c.set_timing(True)
        for c, bt, o in zip(ctxs, batches, outs):
            c.decode(mode, bt.tgt_m.tolist(), block=b, out=o)
        torch.cuda.synchronize()
        launches = rows = 0
        vms = 0.0
        for c in ctxs:
            n_l, t_ms = c.vocab_timing()
            launches += n_l
            vms += t_ms
            rows += c.rows_processed()
            c.set_timing(False)
        flops = 2.0 * rows * cfg.vocab * cfg.d_model
        vocab_tf = flops / (vms * 1e-3) / 1e12 if vms > 0 else 0.0
        res[f"{mode}_b{b}"] = {"tokens_per_s": round(toks / dt, 1), "k_over_m": round(ks / ms, 4),
                               "ms_per_batch": round(1e3 * dt / (repeats * len(batches)), 3),
                               "rows_per_iteration": round(rows / max(launches, 1), 1),
                               "vocab_mfma": {"achieved": round(vocab_tf, 1), "peak": MFMA_BF16_PEAK_TFLOPS,
                                              "unit": "TFLOP/s", "frac": round(vocab_tf / MFMA_BF16_PEAK_TFLOPS, 4),
                                              "avg_launch_us": round(1e3 * vms / max(launches, 1), 2)}}
        log(f"[{wl_name}] {mode:9s} b={b:2d}: {toks / dt:10.1f} tok/s  k/m={ks / ms:.3f}  "
            f"{1e3 * dt / (repeats * len(batches)):8.2f} ms/batch  vocab {vocab_tf:6.1f} TFLOP/s "
            f"({rows / max(launches, 1):.0f} rows/iteration)")
    return res


def copy_calibration():
    """Three plain device copies of 256 MiB (read 256 MiB + write 256 MiB each):
    the reference kernel for scaling the HBM byte counters of a profile."""
    import torch
    src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log("[calibration] 3 x copy of 256 MiB done")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20, help="sentences timed per mode (the first STEPS)")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-sentences", type=int, default=2)
    ap.add_argument("--cpu-m", type=int, default=24, help="target positions of each CPU-baseline sentence")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-mt-base", action="store_true")
    ap.add_argument("--no-tiny", action="store_true")
    ap.add_argument("--no-batched", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--encode-only", default="",
                    help="WORKLOAD — encode its sources one by one (batch 1) and exit (profiling driver)")
    ap.add_argument("--decode-only", default="",
                    help="WORKLOAD:MODE:B:N — decode the first N sentences at batch 1 in one mode (graph replay, "
                         "then an event-timed pass) and exit (profiling driver; prints no JSON line)")
    ap.add_argument("--batched-only", default="",
                    help="WORKLOAD:MODE:B — decode one batch of a batched workload in one mode and exit "
                         "(profiling driver; prints no JSON line)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); sentence-level data "
              "parallelism across GPUs is not built.", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)

    if args.copy_calibration:
        copy_calibration()
    if args.encode_only:
        wl, _, _, sents, ctxs, _ = setup_batch1(args.encode_only, args.steps)
        e = encode_rate(ctxs, sents, wl.model, args.steps, args.warmup)
        log(f"[{args.encode_only}] encode: {e['us_per_sentence']:.1f} us/sentence, {e['achieved']:.0f} GB/s")
        return
    if args.decode_only:
        name, mode, b, n = args.decode_only.split(":")
        wl, _, _, sents, ctxs, outs = setup_batch1(name, int(n))
        r = run_mode(ctxs, sents, outs, mode, int(b), int(n), min(args.warmup, int(n)))
        t = run_mode(ctxs, sents, outs, mode, int(b), int(n), 0, timing=True)
        prod, voc = rooflines(wl.model, t)
        log(f"[{name}] {mode} b={b}: {r['tokens_per_s']:.1f} tok/s, {r['us_per_iteration']:.1f} us/iteration; "
            f"products {prod['achieved']:.0f} GB/s ({prod['avg_launch_us']} us/launch), vocabulary "
            f"{voc['achieved']:.0f} GB/s ({voc['avg_launch_us']} us/launch)")
        return
    if args.batched_only:
        wl_name, mode, b = args.batched_only.split(":")
        batched_workload(wl_name, 1, [(mode, int(b))], 1)
        return

    wl, w, sents, ctxs, res, timed, extra = batch1_workload("large", args.steps, args.warmup, LARGE_MODES,
                                                            HEADLINE, encode=True)
    cfg = wl.model
    key = f"{HEADLINE[0]}_b{HEADLINE[1]}"
    h = res[key]
    products, vocab = rooflines(cfg, timed)
    log(f"[large] products {products['achieved']:.0f} GB/s ({products['frac']:.3f}), vocabulary "
        f"{vocab['achieved']:.0f} GB/s ({vocab['frac']:.3f})")
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, w, sents, ctxs, HEADLINE[0], HEADLINE[1], args.cpu_m, args.cpu_sentences)

    mt = {}
    if not args.no_mt_base:
        for name in ("mt_base_bf16", "mt_base_f32"):
            wl2, _, _, _, r2, t2, x2 = batch1_workload(name, min(args.steps, 200), args.warmup, MT_MODES,
                                                       ("hybrid", 5), trace=name == "mt_base_bf16",
                                                       encode=name == "mt_base_bf16")
            p2, v2 = rooflines(wl2.model, t2)
            mt[name] = {"workload": f"{name}: 6+6 layers, d=512, 8 heads, FFN 2048, V=58101, batch 1, the first "
                                    f"{min(args.steps, 200)} of 200 sources n~U[10,60], m=min(n+10,128)",
                        **mode_table(r2), "cost_ratio": cost_ratio(r2, "hybrid_b5"),
                        "products_roofline": p2, "vocab_roofline": v2,
                        "iteration_roofline": iteration_roofline(wl2.model, r2["hybrid_b5"]), **x2}
    tiny = None if args.no_tiny else tiny_latency(100)
    batched = None
    if not args.no_batched:
        batched = {
            "mt_base_b64": {"workload": "mt_base bf16, batch 64, first 4 batches of 64 sources, n ~ clipped "
                                        "log-normal (median 25, max 128), m = n + 10",
                            **batched_workload("mt_base_b64", 4, [("ar", 1), ("hybrid", 2), ("hybrid", 3),
                                                                  ("hybrid", 5), ("hybrid", 8), ("gs_jacobi", 5),
                                                                  ("jacobi", 0)], 2)},
            "large_b32": {"workload": "large bf16, batch 32, first 2 batches of 32 sources, n ~ U[20,120], "
                                      "m = min(n + 10, 256)",
                          **batched_workload("large_b32", 2, [("ar", 1)] + [(m, b) for m in ("gs_jacobi", "hybrid")
                                                                          for b in (1, 2, 4, 8, 16, 32)]
                                             + [("jacobi", 0)], 1)},
        }

    line = {
        "metric": "target tokens/s (parallel vs greedy AR decode) + iterations/sentence k/m",
        "value": round(h["tokens_per_s"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(h["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random weights and sources)",
        "config": {"workload": "large bf16: 12+12 layers, d=1024, 16 heads, FFN 4096 GELU, pre-LN, V=250027, batch 1, "
                               "51 sources n~U[20,120] (the last with m=256), m=min(n+10,256); "
                               f"timed: sentences 0..{args.steps - 1}",
                   "mode": HEADLINE[0], "block": HEADLINE[1], "global_batch": 1, "parallelism": "none"},
        "modes": mode_table(res),
        "speedup_vs_ar": round(h["tokens_per_s"] / res["ar_b1"]["tokens_per_s"], 3),
        "cost_ratio": cost_ratio(res, key),
        "roofline": products,
        "vocab_roofline": vocab,
        "iteration_roofline": iteration_roofline(cfg, h),
        "cpu_baseline": cpu,
        "encode": {**extra["encode"], "note": "pd_encode at batch 1 over the timed sources (not in the decode timing)"},
    }
    line.update(mt)
    if tiny is not None:
        line["tiny"] = tiny
    if batched is not None:
        line["batched"] = batched
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
