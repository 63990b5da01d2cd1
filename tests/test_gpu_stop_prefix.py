"""The prefix stopping condition (PD_STOP_PREFIX) on the HIP path, against the
oracle's stop="prefix" procedure (oracle/decode.py).

Every expected value comes from the oracle: ids and iteration counts k of the
same decode, greedy decoding's output (Proposition 1 holds for the variant),
and, at full size, the oracle's prefix control flow replayed on the GPU's own
recorded evaluations.  The control kernels that carry the variant are all
exercised: the single-workgroup step of iterations of at most 64 rows, the
row-parallel one (more rows or sentences), and their separate-argmax forms."""
import numpy as np
import pytest

import oracle
from paper_2305_10427_amd import configs as C, pdec, synth
from tests.parity import gpu_decode_batch, gpu_decode_traced, judge_batch, replay_check, spot_check, summarize, \
    workload_model
from tests.test_gpu_parity import CHAIN, SMALL_PRE_BF16, TINY, build, say, sources

pytestmark = pytest.mark.gpu

PREFIX_MODES = [("jacobi", 0), ("gs_jacobi", 4), ("gs_jacobi", 3), ("hybrid", 4), ("hybrid", 1)]


@pytest.mark.parametrize("cfg,wkw", [(TINY, {}), (TINY, dict(bias_std=0.5, ln_std=0.3)),
                                     (CHAIN, dict(bias_std=0.5, ln_std=0.3)),
                                     (SMALL_PRE_BF16, dict(bias_std=0.3, ln_std=0.2))],
                         ids=["tiny", "tiny_bias", "chain", "small_pre_bf16"])
def test_prefix_stop_matches_oracle_small(cfg, wkw):
    """Ids and k equal the oracle's prefix decode; the ids equal the GPU's own
    greedy decode bitwise (the same map), and k never exceeds the Eq. (3)
    decode's by more than the oracle says it should (the oracle's k is the
    reference for both)."""
    _, _, ctx, M = build(cfg, seed=3, **wkw)
    labels = []
    for src in sources(cfg.vocab, 4, seed=11):
        for m in (1, 5, 16):
            ar = gpu_decode_batch(ctx, [src], [m], "ar")[0]
            for mode, b in PREFIX_MODES:
                say(f"case prefix cfg={cfg.name} mode={mode} b={b} m={m}")
                got, labs = judge_batch(ctx, M, [src], [m], mode, b, cfg.dtype, stop="prefix")
                assert not labs[0].startswith("FAIL"), f"{mode} b={b} m={m}: {labs[0]}"
                assert 1 <= got[0].k <= m
                if mode != "hybrid":
                    np.testing.assert_array_equal(got[0].ids, ar.ids)
                labels += labs
    s = summarize(labels)
    say("summary", cfg.name, s)
    assert s["exact"] >= 0.9 * len(labels)


@pytest.mark.parametrize("cfg,seed,wkw", [(TINY, 8, dict(bias_std=0.5, ln_std=0.3)),
                                          (CHAIN, 9, dict(bias_std=0.5, ln_std=0.3)),
                                          (SMALL_PRE_BF16, 13, dict(bias_std=0.3, ln_std=0.2))],
                         ids=["tiny", "chain", "small_pre_bf16"])
def test_prefix_stop_hybrid_eos_fixtures_and_horizons(cfg, seed, wkw):
    """[EOS] at a block start, inside a block, at a block's end or absent,
    crossed with horizons h in {1, b, m/2, m - 1, m}: decoding stops where the
    oracle's prefix decode stops (an [EOS] counts once it is committed)."""
    from tests.test_oracle_decode import eos_cases
    m = 16
    for b in (3, 4):
        found = eos_cases(cfg, seed, wkw, b, m)
        assert {"absent", "start", "mid", "last"} <= set(found), sorted(found)
        for kind, (B, src, q) in found.items():
            _, _, ctx, M = build(cfg, seed=seed, eos_bias=B, **wkw)
            for h in (1, b, m // 2, m - 1, 0):
                say(f"case prefix eos cfg={cfg.name} b={b} kind={kind} q={q} h={h}")
                got, labs = judge_batch(ctx, M, [src], [m], "hybrid", b, cfg.dtype, horizon=h, stop="prefix")
                assert not labs[0].startswith("FAIL"), f"{kind} q={q} h={h}: {labs[0]}"
                if labs[0] == "exact":
                    ends = len(got[0].ids) and got[0].ids[-1] == C.EOS_ID
                    assert bool(got[0].flags & pdec.FLAG_EOS) == bool(ends)


def test_prefix_stop_with_initial_drafts_and_batches():
    """Random initial drafts (pd_decode_init) under the prefix condition give
    the oracle's ids and k; a perfect draft is committed block by block at once
    (k = number of blocks); batched decodes equal single decodes bitwise, on
    the single-workgroup control step (4 sentences) and the row-parallel one
    (8 sentences x blocks of 16 = 128 rows, then 80 sentences)."""
    for cfg, wkw in [(TINY, {}), (CHAIN, dict(bias_std=0.5, ln_std=0.3))]:
        _, _, ctx, M = build(cfg, seed=5, max_batch=8, **wkw)
        srcs = sources(cfg.vocab, 8, seed=14)
        for si, src in enumerate(srcs[:3]):
            enc = M.encode(src)
            for m in (7, 16):
                draft = synth.random_draft(m, cfg.vocab, 200 + si)
                for mode, b in [("jacobi", 0), ("gs_jacobi", 3), ("hybrid", 4)]:
                    say(f"case prefix init cfg={cfg.name} mode={mode} b={b} m={m}")
                    _, labs = judge_batch(ctx, M, [src], [m], mode, b, cfg.dtype, init=[draft], stop="prefix")
                    assert not labs[0].startswith("FAIL"), f"{mode} b={b} m={m}: {labs[0]}"
            y_star = oracle.greedy(M, enc, 16, stop_at_eos=False).y
            for b in (3, 4, 16):
                g = gpu_decode_batch(ctx, [src], [16], "gs_jacobi", b, init=[y_star], stop="prefix")[0]
                assert g.k == -(-16 // b)
        for B, b in [(4, 4), (8, 16)]:
            ms = [16, 11, 16, 3, 9, 16, 14, 5][:B]
            say(f"case prefix batch cfg={cfg.name} B={B} b={b}")
            batch = gpu_decode_batch(ctx, srcs[:B], ms, "gs_jacobi", b, stop="prefix")
            for r in range(B):
                one = gpu_decode_batch(ctx, [srcs[r]], [ms[r]], "gs_jacobi", b, stop="prefix")[0]
                np.testing.assert_array_equal(batch[r].ids, one.ids)
                assert batch[r].k == one.k
            _, labs = judge_batch(ctx, M, srcs[:B], ms, "gs_jacobi", b, cfg.dtype, got=batch, stop="prefix")
            assert not any(lab.startswith("FAIL") for lab in labs), labs
    _, _, ctx, M = build(TINY, seed=3, max_batch=80, max_src=16, max_tgt=24)
    g = np.random.default_rng(31)
    srcs = [g.integers(4, TINY.vocab, int(n)).astype(np.int32) for n in g.integers(4, 17, 80)]
    ms = [int(m) for m in g.integers(1, 25, 80)]
    for mode, b in [("hybrid", 2), ("gs_jacobi", 3)]:
        say(f"case prefix 80 sentences mode={mode} b={b}")
        batch = gpu_decode_batch(ctx, srcs, ms, mode, b, stop="prefix")
        for r in range(80):
            one = gpu_decode_batch(ctx, [srcs[r]], [ms[r]], mode, b, stop="prefix")[0]
            np.testing.assert_array_equal(batch[r].ids, one.ids)
            assert batch[r].k == one.k
        _, labs = judge_batch(ctx, M, srcs, ms, mode, b, C.F32, idx=(0, 41, 79), got=batch, stop="prefix")
        assert not any(lab.startswith("FAIL") for lab in labs), labs


@pytest.mark.parametrize("wl", ["mt_base_f32", "mt_base_bf16"])
def test_prefix_stop_mt_base_sampled_sentences(wl):
    """Sampled MT-base sentences at their full m: GS-Jacobi and hybrid b = 5
    and Jacobi under the prefix condition, against the oracle; the prefix
    decodes never take more iterations than the Eq. (3) ones on these."""
    cfg = C.WORKLOADS[wl].model
    _, gm, M = workload_model(cfg)
    ctx = pdec.Context(gm, 1, 128, C.WORKLOADS[wl].tgt_cap)
    labels = []
    for src, m in synth.make_sentences(C.WORKLOADS[wl], seed=1, count=3):
        for mode, b in [("gs_jacobi", 5), ("hybrid", 5), ("jacobi", 0)]:
            say(f"case prefix {wl} mode={mode} b={b} n={len(src)} m={m}")
            got, labs = judge_batch(ctx, M, [src], [m], mode, b, cfg.dtype, stop="prefix")
            blk = gpu_decode_batch(ctx, [src], [m], mode, b)[0]
            say("  ->", labs[0], "k", got[0].k, "Eq. (3) k", blk.k)
            assert not labs[0].startswith("FAIL"), labs[0]
            assert got[0].k <= blk.k
            labels += labs
    s = summarize(labels)
    say(wl, s)
    assert s["exact"] >= (1.0 if cfg.dtype == C.F32 else 0.5) * len(labels)


def test_prefix_stop_large_replayed():
    """Large model, batch 1: two sentences at their full m in GS-Jacobi and
    hybrid b = 16 under the prefix condition; the ids equal the oracle's greedy
    output, the oracle's prefix control flow run on the GPU's recorded
    evaluations reproduces ids and k, and whole iterations are recomputed by
    the oracle."""
    wl = C.WORKLOADS["large"]
    cfg = wl.model
    _, gm, M = workload_model(cfg)
    ctx = pdec.Context(gm, 1, 128, wl.tgt_cap)
    spots = []
    for src, m in synth.make_sentences(wl, seed=1, count=2):
        enc = M.encode(src)
        greedy = oracle.greedy(M, enc, m)
        for mode, b in [("gs_jacobi", 16), ("hybrid", 16)]:
            say(f"case prefix large replay mode={mode} b={b} n={len(src)} m={m}")
            res, rows = gpu_decode_traced(ctx, [src], [m], mode, b, stop="prefix")
            g = res[0]
            np.testing.assert_array_equal(g.ids, greedy.out)
            rep = replay_check(g, rows[0], mode, b, m, stop="prefix")
            n_it = len(rep.iterations)
            spots += spot_check(rep, M, enc, cfg.dtype, sorted({0, n_it // 2, n_it - 1}))
            say(f"  k={g.k} iterations={n_it}")
    s = summarize(spots)
    say("large prefix spot checks", s)
    assert s["fail"] == 0, [x for x in spots if x.startswith("FAIL")]
