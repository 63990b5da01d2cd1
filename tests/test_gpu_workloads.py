"""Parity at the full sizes of the benchmark workloads, in the launch
configurations bench.py times.

* tiny 2+2 model: all 100 sources, every mode, batch 1, against the oracle;
* MT-base bf16, batch 64 (log-normal source lengths, sources padded to the
  batch maximum): hybrid b in {2, 3, 5, 8} and batched greedy; every sentence of
  the batch equals its own batch-1 decode bitwise (sentences iterate
  independently), eight sampled sentences equal the oracle (ids and k);
* large 12+12 pre-LN bf16 model, batch 32: GS-Jacobi and hybrid for
  b in {1, 2, 4, 8, 16, 32}; every mode returns the batched greedy ids, two
  sampled sentences equal their batch-1 decodes, the shortest sentence of the
  batch equals the oracle (ids and k) in three modes;
* large model, batch 1, the m = 256 sentence: greedy, Jacobi over all 256
  positions and GS-Jacobi b = 16 return the oracle's greedy ids; greedy and
  GS-Jacobi also match the oracle's iteration count.

Every expected value comes from the oracle or from a property of the method
(Proposition 1: each mode returns the greedy solution; k <= m)."""
import numpy as np
import pytest

import oracle
from paper_2305_10427_amd import configs as C, pdec, synth
from tests.parity import TOL, classify, classify_ids, gpu_decode_batch, summarize, workload_model

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)


def test_tiny_workload_every_mode():
    wl = C.WORKLOADS["tiny"]
    _, gm, M = workload_model(wl.model)
    ctx = pdec.Context(gm, 1, 16, wl.tgt_cap)
    labels = []
    for idx, (src, m) in enumerate(synth.make_sentences(wl, seed=1)):
        enc = M.encode(src)
        greedy = oracle.greedy(M, enc, m)
        for mode, b in wl.modes:
            want = oracle.decode(M, enc, m, mode, b)
            g = gpu_decode_batch(ctx, [src], [m], mode, b)[0]
            lab = classify(g, want, greedy, TOL[wl.model.dtype])
            assert not lab.startswith("FAIL"), f"sentence {idx} {mode} b={b}: {lab}"
            assert g.k <= m
            labels.append(lab)
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
    sample = list(range(0, 64, 9))
    enc = {r: M.encode(srcs[r]) for r in sample}
    greedy = {r: oracle.greedy(M, enc[r], ms[r]) for r in sample}
    labels = []
    for mode, b in wl.modes:
        say(f"case mt_base_b64 mode={mode} b={b} B=64 n_max={max(len(s) for s in srcs)} m_max={max(ms)}")
        batch = gpu_decode_batch(ctx, srcs, ms, mode, b)
        for r in range(64):
            assert batch[r].k <= ms[r]
            single = gpu_decode_batch(one, [srcs[r]], [ms[r]], mode, b)[0]
            np.testing.assert_array_equal(batch[r].ids, single.ids)
            assert batch[r].k == single.k, (r, batch[r].k, single.k)
        for r in sample:
            want = oracle.decode(M, enc[r], ms[r], mode, b)
            lab = classify(batch[r], want, greedy[r], TOL[cfg.dtype])
            say(f"  sentence {r} n={len(srcs[r])} m={ms[r]}: {lab} k={batch[r].k}")
            assert not lab.startswith("FAIL"), f"sentence {r}: {lab}"
            labels.append(lab)
    say("mt_base_b64", summarize(labels))


def test_large_batch32_block_sweep():
    wl, srcs, ms = _batch("large_b32", 32)
    cfg = wl.model
    _, gm, M = workload_model(cfg)
    ctx = pdec.Context(gm, 32, 120, wl.tgt_cap)
    one = pdec.Context(gm, 1, 120, wl.tgt_cap)
    say(f"case large_b32 mode=ar B=32 n_max={max(len(s) for s in srcs)} m_max={max(ms)}")
    ar = gpu_decode_batch(ctx, srcs, ms, "ar")
    results = {("ar", 1): ar}
    for mode, b in wl.modes:
        if mode == "ar":
            continue
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
    enc = M.encode(srcs[r])
    greedy = oracle.greedy(M, enc, ms[r])
    for mode, b in [("ar", 1), ("gs_jacobi", 16), ("hybrid", 8)]:
        want = oracle.decode(M, enc, ms[r], mode, b)
        lab = classify(results[(mode, b)][r], want, greedy, TOL[cfg.dtype])
        say(f"  oracle sentence {r} n={len(srcs[r])} m={ms[r]} {mode} b={b}: {lab}")
        assert not lab.startswith("FAIL"), lab


def test_large_full_length_sentence():
    wl = C.WORKLOADS["large"]
    cfg = wl.model
    _, gm, M = workload_model(cfg)
    src, m = synth.make_sentences(wl, seed=1)[-1]
    assert m == wl.tgt_cap == 256
    ctx = pdec.Context(gm, 1, 128, wl.tgt_cap)
    enc = M.encode(src)
    greedy = oracle.greedy(M, enc, m)
    for mode, b in [("ar", 1), ("jacobi", 0), ("gs_jacobi", 16)]:
        say(f"case large m=256 n={len(src)} mode={mode} b={b}")
        g = gpu_decode_batch(ctx, [src], [m], mode, b)[0]
        lab = classify_ids(g.ids, greedy, TOL[cfg.dtype])
        say(f"  -> {lab} k={g.k} len={len(g.ids)}")
        assert not lab.startswith("FAIL"), lab
        assert g.k <= m
        if mode == "ar" and lab == "exact":
            assert g.k == greedy.k
        if mode == "gs_jacobi" and lab == "exact":
            want = oracle.gs_jacobi(M, enc, m, 16)
            assert classify(g, want, greedy, TOL[cfg.dtype]) == "exact"
