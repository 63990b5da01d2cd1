"""Parity at the full sizes of the benchmark workloads, in the launch
configurations bench.py times.

* tiny 2+2 model: all 100 sources, every mode, batch 1, against the oracle;
* MT-base bf16, batch 64 (log-normal source lengths, sources padded to the
  batch maximum): batched greedy, Jacobi, GS-Jacobi b = 5 and hybrid b in
  {2, 3, 5, 8}; every sentence of the batch equals its own batch-1 decode
  bitwise (sentences iterate independently) and sampled sentences equal the
  oracle (ids and k);
* large 12+12 pre-LN bf16 model, batch 32: greedy, Jacobi, and GS-Jacobi and
  hybrid for b in {1, 2, 4, 8, 16, 32}; every mode returns the batched greedy
  ids, sampled sentences equal their batch-1 decodes, the shortest sentence
  equals the oracle, and the oracle's control flow replayed on the GPU's
  recorded evaluations reproduces ids and k of Jacobi and GS-Jacobi b = 32;
* large model, batch 1: the m = 256 sentence in all four modes, and the
  sentences bench.py times (its first --steps sentences), whose greedy ids
  equal the oracle's and whose parallel-mode ids and k the replay reproduces.

Every expected value comes from the oracle or from a property of the method
(Proposition 1: each mode returns the greedy solution; k <= m)."""
import numpy as np
import pytest

import oracle
from paper_2305_10427_amd import configs as C, pdec, synth
from tests.parity import (classify, gpu_decode_batch, gpu_decode_traced, judge_batch, replay_check, spot_check,
                          summarize, workload_model)

pytestmark = pytest.mark.gpu

# bench.py's default number of timed sentences of the large batch-1 workload
# (the driver's --steps 20 times the same first 20)
BENCH_LARGE_SENTENCES = 20


def say(*a):
    print(*a, flush=True)


def no_fail(labels):
    bad = [x for x in labels if x.startswith("FAIL")]
    assert not bad, bad


def test_tiny_workload_every_mode():
    wl = C.WORKLOADS["tiny"]
    _, gm, M = workload_model(wl.model)
    ctx = pdec.Context(gm, 1, 16, wl.tgt_cap)
    labels = []
    for idx, (src, m) in enumerate(synth.make_sentences(wl, seed=1)):
        for mode, b in wl.modes:
            got, labs = judge_batch(ctx, M, [src], [m], mode, b, wl.model.dtype)
            assert not labs[0].startswith("FAIL"), f"sentence {idx} {mode} b={b}: {labs[0]}"
            assert got[0].k <= m
            labels += labs
    s = summarize(labels)
    say("tiny workload", s)
    assert s["exact"] >= 0.98 * len(labels)


def _batch(wl_name, size):
    wl = C.WORKLOADS[wl_name]
    sents = synth.make_sentences(wl, seed=1)[:size]
    return wl, [s for s, _ in sents], [m for _, m in sents]


def test_mt_base_batch64():
    wl, srcs, ms = _batch("mt_base_b64", 64)
    cfg = wl.model
    _, gm, M = workload_model(cfg)
    ctx = pdec.Context(gm, 64, 128, wl.tgt_cap)
    one = pdec.Context(gm, 1, 128, wl.tgt_cap)
    labels = []
    for mode, b in list(wl.modes) + [("jacobi", 0), ("gs_jacobi", 5)]:
        say(f"case mt_base_b64 mode={mode} b={b} B=64 n_max={max(len(s) for s in srcs)} m_max={max(ms)}")
        batch = gpu_decode_batch(ctx, srcs, ms, mode, b)
        for r in range(64):
            assert batch[r].k <= ms[r]
            single = gpu_decode_batch(one, [srcs[r]], [ms[r]], mode, b)[0]
            np.testing.assert_array_equal(batch[r].ids, single.ids)
            assert batch[r].k == single.k, (r, batch[r].k, single.k)
        sample = range(0, 64, 21) if mode == "jacobi" else range(0, 64, 9)
        _, labs = judge_batch(ctx, M, srcs, ms, mode, b, cfg.dtype, idx=sample, got=batch)
        say(f"  sampled sentences {list(sample)}: {labs}")
        no_fail(labs)
        labels += labs
    s = summarize(labels)
    say("mt_base_b64", s)
    assert s["exact"] >= 0.75 * len(labels)


def test_large_batch32_block_sweep():
    wl, srcs, ms = _batch("large_b32", 32)
    cfg = wl.model
    _, gm, M = workload_model(cfg)
    ctx = pdec.Context(gm, 32, 120, wl.tgt_cap)
    one = pdec.Context(gm, 1, 120, wl.tgt_cap)
    say(f"case large_b32 mode=ar B=32 n_max={max(len(s) for s in srcs)} m_max={max(ms)}")
    ar = gpu_decode_batch(ctx, srcs, ms, "ar")
    results = {("ar", 1): ar}
    for mode, b in [("jacobi", 0)] + [x for x in wl.modes if x[0] != "ar"]:
        say(f"case large_b32 mode={mode} b={b}")
        res = gpu_decode_batch(ctx, srcs, ms, mode, b)
        results[(mode, b)] = res
        for r in range(32):
            np.testing.assert_array_equal(res[r].ids, ar[r].ids)      # Proposition 1, same map
            assert res[r].k <= ms[r]
            if b == 1:   # blocks of one position: greedy steps (hybrid stops at EOS, GS-Jacobi solves all m)
                assert res[r].k == (ar[r].k if mode == "hybrid" else ms[r])
    for r in (0, 31):
        for (mode, b), res in results.items():
            say(f"case large_b32 single sentence {r} mode={mode} b={b}")
            single = gpu_decode_batch(one, [srcs[r]], [ms[r]], mode, b)[0]
            np.testing.assert_array_equal(res[r].ids, single.ids)
            assert res[r].k == single.k
    r = int(np.argmin(ms))
    labels = []
    for mode, b in [("ar", 1), ("gs_jacobi", 16), ("hybrid", 8)]:
        _, labs = judge_batch(ctx, M, srcs, ms, mode, b, cfg.dtype, idx=[r], got=results[(mode, b)])
        say(f"  oracle sentence {r} n={len(srcs[r])} m={ms[r]} {mode} b={b}: {labs}")
        labels += labs
    no_fail(labels)
    # Jacobi and GS-Jacobi b = 32 of the whole batch: control replayed per sentence
    spots = []
    for mode, b in [("jacobi", 0), ("gs_jacobi", 32)]:
        res, rows = gpu_decode_traced(ctx, srcs, ms, mode, b)
        for s in range(32):
            assert (res[s].k, res[s].ids.tolist()) == (results[(mode, b)][s].k, results[(mode, b)][s].ids.tolist())
            rep = replay_check(res[s], rows[s], mode, b, ms[s])
            if s == r:
                spots += spot_check(rep, M, M.encode(srcs[s]), cfg.dtype, [0, len(rep.iterations) - 1])
        say(f"  replayed {mode} b={b} on all 32 sentences")
    say("large_b32 spot checks", summarize(spots))
    no_fail(spots)


def _replay_sentence(ctx, M, cfg, src, m, modes, n_spots):
    """ids of every mode against the oracle's greedy output; ids and k of the
    parallel modes through the replay; n_spots whole iterations recomputed."""
    enc = M.encode(src)
    greedy = oracle.greedy(M, enc, m)
    labels = []
    for mode, b in modes:
        say(f"case large m={m} n={len(src)} mode={mode} b={b}")
        if mode == "ar":
            g = gpu_decode_batch(ctx, [src], [m], "ar")[0]
            lab = classify(g, greedy, greedy, cfg.dtype, M, enc)
            say(f"  -> {lab} k={g.k}")
            labels.append(lab)
            continue
        res, rows = gpu_decode_traced(ctx, [src], [m], mode, b)
        g = res[0]
        if not np.array_equal(g.ids, greedy.out):
            labels.append(classify(g, greedy, greedy, cfg.dtype, M, enc))
        rep = replay_check(g, rows[0], mode, b, m)
        n_it = len(rep.iterations)
        picks = [n_it // 2, n_it - 1, 0][:n_spots]
        labels += spot_check(rep, M, enc, cfg.dtype, sorted(set(picks)))
        say(f"  k={g.k} of m={m}, {n_it} iterations replayed")
    return labels


def test_large_full_length_sentence():
    wl = C.WORKLOADS["large"]
    cfg = wl.model
    _, gm, M = workload_model(cfg)
    src, m = synth.make_sentences(wl, seed=1)[-1]
    assert m == wl.tgt_cap == 256
    ctx = pdec.Context(gm, 1, 128, wl.tgt_cap)
    labels = _replay_sentence(ctx, M, cfg, src, m, [("ar", 1), ("jacobi", 0), ("gs_jacobi", 16), ("hybrid", 16)], 2)
    say("large m=256", summarize(labels))
    no_fail(labels)


def test_large_bench_sentences():
    """The sentences bench.py times on the large batch-1 workload (the first
    BENCH_LARGE_SENTENCES, in all four modes): greedy ids equal the oracle's;
    Jacobi, GS-Jacobi b = 16 and hybrid b = 16 return those ids with the k that
    the oracle's control flow gives on their recorded evaluations; one
    iteration of each mode is recomputed by the oracle on every fifth sentence."""
    wl = C.WORKLOADS["large"]
    cfg = wl.model
    _, gm, M = workload_model(cfg)
    sents = synth.make_sentences(wl, seed=1)[:BENCH_LARGE_SENTENCES]
    ctx = pdec.Context(gm, 1, max(len(s) for s, _ in sents), wl.tgt_cap)
    labels = []
    for idx, (src, m) in enumerate(sents):
        labels += _replay_sentence(ctx, M, cfg, src, m, [("ar", 1), ("jacobi", 0), ("gs_jacobi", 16), ("hybrid", 16)],
                                   1 if idx % 5 == 0 else 0)
    s = summarize(labels)
    say("large bench sentences", s)
    no_fail(labels)
