#!/usr/bin/env python3
"""Decode throughput of parallel decoding vs greedy decoding on one MI355X.

Workload (default): the Transformer-base-shaped model (6+6 layers, d=512, 8
heads, FFN 2048, vocabulary 58,101, shared embeddings) with seeded random
weights, 200 synthetic sources with lengths uniform in [10, 60] and
m = min(n + 10, 128) target positions, batch 1 (the paper's online setting).
A step is the decode of one sentence (pd_decode, batch 1) with its source
already encoded and resident in HBM; the timed region covers K steps.

One JSON line on stdout: value = target tokens/s of the headline mode
(hybrid GS-Jacobi, b = 5) in bf16, plus greedy and GS-Jacobi numbers, k/m,
the float32 model, the roofline of the fused vocabulary kernel and the CPU
oracle baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0   # dense bf16 matrix peak of MI355X


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


def run_mode(ctxs, sents, outs, mode, block, steps, warmup, timing=False):
    import torch
    n = len(sents)
    order = [i % n for i in range(warmup + steps)]
    # one-time setup: every context captures and instantiates its iteration
    # graph for this mode (and timing setting) on its first decode
    for i in range(n):
        ctxs[i].set_timing(timing)
        ctxs[i].decode(mode, [sents[i][1]], block=block, out=outs[i])
        ctxs[i].set_timing(False)
    torch.cuda.synchronize()
    for i in order[:warmup]:
        ctxs[i].decode(mode, [sents[i][1]], block=block, out=outs[i])
    torch.cuda.synchronize()
    if timing:
        for c in ctxs:
            c.set_timing(True)
    t0 = time.perf_counter()
    for i in order[warmup:]:
        ctxs[i].decode(mode, [sents[i][1]], block=block, out=outs[i])
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    toks = ks = ms = 0
    for i in order[warmup:]:
        toks += int(outs[i][1][0])
        ks += int(outs[i][2][0])
        ms += sents[i][1]
    res = {"tokens": toks, "seconds": dt, "tokens_per_s": toks / dt, "k": ks, "m": ms, "k_over_m": ks / ms,
           "ms_per_step": 1e3 * dt / steps}
    if timing:
        launches = total_ms = 0
        for c in ctxs:
            n_l, t_ms = c.vocab_timing()
            launches += n_l
            total_ms += t_ms
            c.set_timing(False)
        res["vocab_launches"] = launches
        res["vocab_ms"] = total_ms
    return res


def encode_rate(ctxs, sents, cfg, steps, warmup):
    """pd_encode of one source per call (batch 1), the step before the
    decoding iterations: wall time per sentence over `steps` calls, against
    the weights it must read (encoder layers and every decoder layer's
    cross-attention K/V projection, bf16/f32 storage)."""
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
    return {"us_per_sentence": 1e6 * dt, "weight_bytes": wbytes, "achieved_GBs": wbytes / dt / 1e9,
            "frac": wbytes / dt / 1e9 / HBM_PEAK_GBS}


def encode_only(steps, warmup):
    import torch
    from paper_2305_10427_amd import configs as C, pdec, synth
    wl = C.WORKLOADS["mt_base_bf16"]
    w, model = load_model(wl.model)
    sents = synth.make_sentences(wl, seed=1)
    ctx = pdec.Context(model, 1, max(len(s) for s, _ in sents), wl.tgt_cap)
    e = encode_rate([ctx] * len(sents), sents, wl.model, steps, warmup)
    log(f"[mt_base_bf16] encode: {e['us_per_sentence']:.1f} us/sentence, {e['achieved_GBs']:.0f} GB/s of weights")


def gpu_workload(wl_name, steps, warmup, modes, headline, n_sent=0, trace=False, encode=False):
    import torch
    from paper_2305_10427_amd import configs as C, pdec, synth
    wl = C.WORKLOADS[wl_name]
    cfg = wl.model
    t0 = time.perf_counter()
    w, model = load_model(cfg)
    sents = synth.make_sentences(wl, seed=1)
    if n_sent:
        sents = sents[:n_sent]
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
    res = {}
    for mode, b in modes:
        r = run_mode(ctxs, sents, outs, mode, b, steps, warmup)
        res[f"{mode}_b{b}"] = r
        log(f"[{wl_name}] {mode:9s} b={b}: {r['tokens_per_s']:9.1f} tok/s  {r['ms_per_step']:7.3f} ms/sentence  "
            f"k/m={r['k_over_m']:.3f}")
    # the vocabulary kernel's launch time: a second pass of the headline mode
    # with HIP events around that kernel (the events cost time of their own, so
    # the throughput above comes from the pass without them)
    t = run_mode(ctxs, sents, outs, headline[0], headline[1], steps, warmup, timing=True)
    res[f"{headline[0]}_b{headline[1]}"].update(vocab_launches=t["vocab_launches"], vocab_ms=t["vocab_ms"])
    if encode:
        res["encode"] = encode_rate(ctxs, sents, cfg, steps, warmup)
        e = res["encode"]
        log(f"[{wl_name}] encode: {e['us_per_sentence']:.1f} us/sentence, {e['achieved_GBs']:.0f} GB/s of weights")
    if trace:
        # the same decodes with the DDGviz trace on (records and log-sum-exp
        # partials)
        for c in ctxs:
            c.set_trace(4 * wl.tgt_cap, max(headline[1], 1))
        t = run_mode(ctxs, sents, outs, headline[0], headline[1], steps, warmup)
        for c in ctxs:
            c.set_trace(0, 0)
        res["trace"] = {"mode": f"{headline[0]}_b{headline[1]}", "tokens_per_s": t["tokens_per_s"],
                        "ms_per_step": t["ms_per_step"]}
        log(f"[{wl_name}] traced {headline[0]} b={headline[1]}: {t['tokens_per_s']:9.1f} tok/s")
    return cfg, w, sents, model, res


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
        # a separate pass with HIP events around the fused vocabulary launch and
        # the device count of rows evaluated: its MFMA rate
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


def cpu_baseline(cfg, weights, sents, mode, block, budget_s):
    """The oracle as it stands, on the host cores, on a bounded sample."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:                       # noqa: BLE001
        threads = len(os.sched_getaffinity(0))
    M = oracle.Model(cfg, weights.values)
    toks = n = 0
    t0 = time.perf_counter()
    dec_s = 0.0
    for src, m in sents:
        enc = M.encode(src)
        t1 = time.perf_counter()
        r = oracle.decode(M, enc, m, mode, block)
        dec_s += time.perf_counter() - t1
        toks += len(r.out)
        n += 1
        if time.perf_counter() - t0 > budget_s:
            break
    return {"value": toks / dec_s, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"first {n} sentences of the same workload, {mode} b={block}, decode only "
                      f"(numpy float64 oracle, {dec_s:.1f}s)"}


def measured_traffic():
    """HBM bytes per launch of the fused vocabulary kernel from the committed
    rocprofv3 counter summary, or None once the kernel source has changed."""
    import hashlib
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "vocab_argmax_mt_base_bf16.json")))
        src = b"".join(open(os.path.join(ROOT, "paper_2305_10427_amd", "csrc", f), "rb").read()
                       for f in rec["kernel_sources"])
        if hashlib.sha256(src).hexdigest() != rec["kernel_source_sha256"]:
            return None
        return int(rec["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


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
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--sentences", type=int, default=0, help="use the first N sentences (0: all)")
    ap.add_argument("--modes", default="ar:1,gs_jacobi:5,hybrid:5")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-f32", action="store_true")
    ap.add_argument("--no-large", action="store_true")
    ap.add_argument("--no-batched", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--encode-only", action="store_true",
                    help="encode the MT-base bf16 sources one by one (batch 1) and exit (profiling driver; "
                         "prints no JSON line)")
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
        encode_only(args.steps, args.warmup)
        return
    if args.batched_only:
        wl_name, mode, b = args.batched_only.split(":")
        batched_workload(wl_name, 1, [(mode, int(b))], 1)
        return
    headline = ("hybrid", 5)
    modes = [(m.split(":")[0], int(m.split(":")[1])) for m in args.modes.split(",")]
    if headline not in modes:
        modes.append(headline)
    cfg, w, sents, model, res = gpu_workload("mt_base_bf16", args.steps, args.warmup, modes, headline,
                                             args.sentences, trace=True, encode=True)
    traced = res.pop("trace")
    enc = res.pop("encode")
    f32 = None
    if not args.no_f32:
        _, _, _, _, f32 = gpu_workload("mt_base_f32", args.steps, args.warmup, modes, headline, args.sentences)
    large = None
    if not args.no_large:
        _, _, _, _, large = gpu_workload("large", min(args.steps, 20), min(args.warmup, 2),
                                         [("ar", 1), ("jacobi", 0), ("gs_jacobi", 16)], ("gs_jacobi", 16), 20)

    batched = None
    if not args.no_batched:
        batched = {
            "mt_base_b64": {"workload": "mt_base bf16, batch 64, first 4 batches of 64 sources, n ~ clipped "
                                        "log-normal (median 25, max 128), m = n + 10",
                            **batched_workload("mt_base_b64", 4, [("ar", 1), ("hybrid", 2), ("hybrid", 3),
                                                                  ("hybrid", 5), ("hybrid", 8)], 2)},
            "large_b32": {"workload": "large bf16, batch 32, first 2 batches of 32 sources, n ~ U[20,120], "
                                      "m = min(n + 10, 256)",
                          **batched_workload("large_b32", 2, [("ar", 1)] + [(m, b) for m in ("gs_jacobi", "hybrid")
                                                                          for b in (1, 2, 4, 8, 16, 32)], 1)},
        }

    h = res[f"{headline[0]}_b{headline[1]}"]
    # roofline of the fused vocabulary projection + argmax (bytes: E [V][d] and the output bias, bf16)
    bytes_per_launch = cfg.vocab * (cfg.d_model + 1) * 2
    avg_ms = h["vocab_ms"] / max(h["vocab_launches"], 1)
    achieved = bytes_per_launch / (avg_ms * 1e-3) / 1e9
    roof = {"kernel": "k_vocab<bf16> (streaming vocab projection + LayerNorm + argmax, <= 16 rows)", "bound": "hbm",
            "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(),
            "avg_launch_us": round(avg_ms * 1e3, 2), "launches": h["vocab_launches"],
            "bytes_per_launch": bytes_per_launch}
    # the whole batch-1 iteration against the bytes it must move: decoder
    # weights + vocabulary (the K/V cache reads are a few hundred KB)
    d, f, L = cfg.d_model, cfg.d_ff, cfg.n_dec
    iter_bytes = (L * (6 * d * d + 2 * d * f + 13 * d + f) + cfg.vocab * (d + 1)) * 2
    iter_us = 1e6 * h["seconds"] / h["k"]
    iteration = {"us": round(iter_us, 2), "bytes": iter_bytes, "achieved": round(iter_bytes / iter_us / 1e3, 1),
                 "unit": "GB/s", "frac": round(iter_bytes / iter_us / 1e3 / HBM_PEAK_GBS, 4),
                 "note": "one decoding iteration (every kernel of the decoder pass, vocabulary and control step) "
                         "at batch 1: latency-bound"}
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, w, sents, headline[0], headline[1], args.cpu_seconds)
        log(f"[cpu] oracle {cpu['value']:.1f} tok/s on {cpu['cores']} threads ({cpu['sample']})")

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
        "config": {"workload": "mt_base_bf16: 6+6 layers, d=512, 8 heads, FFN 2048, V=58101, batch 1, "
                               "200 sources n~U[10,60], m=min(n+10,128)",
                   "mode": headline[0], "block": headline[1], "global_batch": 1, "parallelism": "none"},
        "modes": {k: {"tokens_per_s": round(v["tokens_per_s"], 1), "k_over_m": round(v["k_over_m"], 4),
                      "ms_per_sentence": round(v["ms_per_step"], 4)} for k, v in res.items()},
        "speedup_vs_ar": (round(h["tokens_per_s"] / res["ar_b1"]["tokens_per_s"], 3) if "ar_b1" in res else None),
        "roofline": roof,
        "iteration_roofline": iteration,
        "cpu_baseline": cpu,
        "encode": {"us_per_sentence": round(enc["us_per_sentence"], 2), "weight_bytes": enc["weight_bytes"],
                   "achieved": round(enc["achieved_GBs"], 1), "unit": "GB/s", "frac": round(enc["frac"], 4),
                   "note": "pd_encode at batch 1 over the workload's sources (not in the decode timing)"},
        "trace": {"mode": traced["mode"], "tokens_per_s": round(traced["tokens_per_s"], 1),
                  "slowdown": round(h["tokens_per_s"] / traced["tokens_per_s"], 3)},
    }
    if f32 is not None:
        line["f32"] = {k: {"tokens_per_s": round(v["tokens_per_s"], 1), "k_over_m": round(v["k_over_m"], 4)}
                       for k, v in f32.items()}
    if large is not None:
        line["large_bf16"] = {
            "workload": "12+12 layers, d=1024, 16 heads, FFN 4096 GELU, pre-LN, V=250027, batch 1, first 20 "
                        "sources n~U[20,120], m=min(n+10,256)",
            **{k: {"tokens_per_s": round(v["tokens_per_s"], 1), "k_over_m": round(v["k_over_m"], 4),
                   "ms_per_sentence": round(v["ms_per_step"], 3)} for k, v in large.items()}}
        lv = large["gs_jacobi_b16"]
        lb = 250027 * 1025 * 2
        lavg = lv["vocab_ms"] / max(lv["vocab_launches"], 1)
        line["large_bf16"]["vocab_roofline"] = {"achieved": round(lb / (lavg * 1e-3) / 1e9, 1), "peak": HBM_PEAK_GBS,
                                                "unit": "GB/s", "avg_launch_us": round(lavg * 1e3, 2)}
    if batched is not None:
        line["batched"] = batched
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
