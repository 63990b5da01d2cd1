"""Helpers for comparing the HIP decoding path with the CPU oracle.

Token comparison rule: GPU and oracle must return identical ids and identical
iteration counts.  A difference is tolerated only as a *near tie*: at the first
differing position t, the oracle's greedy top-1/top-2 logit margin is below
2 * tol * max|logit| of that row (tol = 1e-3 for float32 models, 5e-2 for
bfloat16 models); a differing k is a near tie only if some argmax on the
oracle's trajectory had such a margin.  Near ties are reported, never silently
accepted as exact.
"""
from __future__ import annotations

import dataclasses
import functools
from typing import List, Optional

import numpy as np

import oracle
from paper_2305_10427_amd import configs as C

TOL = {C.F32: 1e-3, C.BF16: 5e-2}


@dataclasses.dataclass
class GpuResult:
    ids: np.ndarray      # cut to out_len
    k: int
    flags: int


def gpu_decode_batch(ctx, srcs, ms, mode, block=1, max_iters=0, horizon=0, init=None) -> List[GpuResult]:
    """init: optional list of initial drafts (one int array of length >= m per sentence)."""
    import torch
    B = len(srcs)
    n_max = max(len(s) for s in srcs)
    src = np.zeros((B, n_max), np.int32)
    for r, s in enumerate(srcs):
        src[r, :len(s)] = s
    ctx.encode(torch.from_numpy(src).cuda(), [len(s) for s in srcs])
    init_t = None
    if init is not None:
        w = max(len(d) for d in init)
        arr = np.zeros((B, w), np.int32)
        for r, d in enumerate(init):
            arr[r, :len(d)] = d
        init_t = torch.from_numpy(arr).cuda()
    ids, ln, k, fl = ctx.decode(mode, ms, block=block, max_iters=max_iters, horizon=horizon, init=init_t)
    torch.cuda.synchronize()
    ids, ln, k, fl = (t.cpu().numpy() for t in (ids, ln, k, fl))
    out = []
    for r in range(B):
        assert np.all(ids[r, ln[r]:] == C.PAD_ID), "positions after the output must be PAD"
        out.append(GpuResult(ids[r, :ln[r]].copy(), int(k[r]), int(fl[r])))
    return out


def classify(g: GpuResult, want: oracle.Result, greedy: oracle.Result, tol: float) -> str:
    """'exact', 'near_tie:<why>' or 'FAIL:<why>'."""
    if np.array_equal(g.ids, want.out) and g.k == want.k:
        return "exact"
    if not np.array_equal(g.ids, want.out):
        n = min(len(g.ids), len(want.out))
        diff = np.nonzero(g.ids[:n] != want.out[:n])[0]
        t = int(diff[0]) if len(diff) else n
        recs = [r for r in greedy.records if r.position == t]
        if recs:
            r = recs[-1]
            if r.top1 - r.top2 < 2 * tol * r.linf:
                return f"near_tie:token@{t} margin={r.top1 - r.top2:.3g}"
        return f"FAIL:tokens differ at {t}: gpu={g.ids[:t + 3].tolist()} oracle={want.out[:t + 3].tolist()}"
    if want.min_rel_margin() < 2 * tol:
        return f"near_tie:k gpu={g.k} oracle={want.k}"
    return f"FAIL:k gpu={g.k} oracle={want.k}"


def summarize(labels: List[str]) -> dict:
    out = {"exact": 0, "near_tie": 0, "fail": 0}
    for lab in labels:
        out["exact" if lab == "exact" else ("near_tie" if lab.startswith("near_tie") else "fail")] += 1
    return out


@functools.lru_cache(maxsize=None)
def workload_model(cfg: C.ModelConfig):
    """(weights, GPU model, oracle model) of a workload's model with seed-0
    weights, built once per test session (drawing the large model's weights
    takes tens of seconds)."""
    from paper_2305_10427_amd import pdec, synth
    w = synth.make_weights(cfg, seed=0)
    return w, pdec.Model(cfg, w), oracle.Model(cfg, w.values)


def classify_ids(ids: np.ndarray, greedy: oracle.Result, tol: float) -> str:
    """Token ids only (for modes whose iteration count the oracle does not
    replay at this size): 'exact', 'near_tie:...' or 'FAIL:...' as in classify."""
    if np.array_equal(ids, greedy.out):
        return "exact"
    n = min(len(ids), len(greedy.out))
    diff = np.nonzero(ids[:n] != greedy.out[:n])[0]
    t = int(diff[0]) if len(diff) else n
    recs = [r for r in greedy.records if r.position == t]
    if recs and recs[-1].top1 - recs[-1].top2 < 2 * tol * recs[-1].linf:
        return f"near_tie:token@{t}"
    return f"FAIL:tokens differ at {t}: gpu={ids[:t + 3].tolist()} oracle={greedy.out[:t + 3].tolist()}"
