"""Parity of the HIP decoding path (through the C ABI) with the CPU oracle.

Every test is marked gpu: it needs an MI355X and the built libpdec.so.  The
oracle (oracle/) provides every expected value; nothing expected comes from
the GPU path itself."""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2305_10427_amd import configs as C, pdec, synth
from tests.parity import (EPS, TOL, gpu_decode_batch, gpu_decode_traced, judge_batch, replay_check, spot_check,
                          summarize, workload_model)

pytestmark = pytest.mark.gpu

TINY = C.TINY
CHAIN = dataclasses.replace(C.TINY, name="chain", logit_scale=-3.0)
SMALL_PRE_BF16 = dataclasses.replace(C.TINY, name="small_pre", pre_ln=True, act_gelu=True, dtype=C.BF16)
# head widths 64 and 32, and a bf16 width above 512 (LayerNorm rows of more
# than 512 elements per 16-lane group)
MID_F32 = dataclasses.replace(C.TINY, name="mid_f32", d_model=128, n_heads=2, d_ff=256, vocab=700)
MID_BF16 = dataclasses.replace(C.TINY, name="mid_bf16", d_model=256, n_heads=8, d_ff=512, vocab=700, dtype=C.BF16)
WIDE_PRE_BF16 = dataclasses.replace(C.TINY, name="wide_pre", n_dec=1, n_enc=1, d_model=640, n_heads=10, d_ff=640,
                                    vocab=500, pre_ln=True, act_gelu=True, dtype=C.BF16)
# an FFN down-projection with K = 2048: eight K ranges (split over workgroups
# in the tiled products of many rows)
FFN2K_BF16 = dataclasses.replace(C.TINY, name="ffn2k", d_model=256, n_heads=4, d_ff=2048, vocab=700, dtype=C.BF16)


def say(*a):
    print(*a, flush=True)


def build(cfg, seed=0, max_batch=4, max_src=32, max_tgt=32, **wkw):
    w = synth.make_weights(cfg, seed=seed, **wkw)
    gm = pdec.Model(cfg, w)
    ctx = pdec.Context(gm, max_batch, max_src, max_tgt)
    return w, gm, ctx, oracle.Model(cfg, w.values)


def sources(vocab, count, n=16, seed=1):
    g = np.random.default_rng(seed)
    return [g.integers(4, vocab, n).astype(np.int32) for _ in range(count)]


def run_modes(cfg, ctx, M, srcs, m, modes):
    labels = []
    for src in srcs:
        for mode, b in modes:
            say(f"case cfg={cfg.name} mode={mode} b={b} m={m} n={len(src)}")
            got, labs = judge_batch(ctx, M, [src], [m], mode, b, cfg.dtype)
            assert not labs[0].startswith("FAIL"), f"{mode} b={b}: {labs[0]}"
            assert got[0].k <= m
            labels += labs
    return labels


@pytest.mark.parametrize("cfg,wkw", [(TINY, {}), (TINY, dict(bias_std=0.5, ln_std=0.3)),
                                     (CHAIN, dict(bias_std=0.5, ln_std=0.3)),
                                     (SMALL_PRE_BF16, dict(bias_std=0.3, ln_std=0.2))],
                         ids=["tiny", "tiny_bias", "chain", "small_pre_bf16"])
def test_all_modes_match_oracle_small(cfg, wkw):
    _, _, ctx, M = build(cfg, seed=3, **wkw)
    modes = [("ar", 1), ("jacobi", 0), ("gs_jacobi", 4), ("hybrid", 4), ("gs_jacobi", 3), ("hybrid", 1)]
    labels = []
    for m in (1, 5, 16):
        labels += run_modes(cfg, ctx, M, sources(cfg.vocab, 4, seed=11), m, modes)
    s = summarize(labels)
    say("summary", cfg.name, s)
    assert s["exact"] >= 0.9 * len(labels)


def test_parallel_modes_equal_gpu_greedy_bitwise():
    """All modes evaluate the same map on the GPU, so they agree with GPU greedy exactly."""
    _, _, ctx, _ = build(CHAIN, seed=1, bias_std=0.5, ln_std=0.3)
    for src in sources(CHAIN.vocab, 6, seed=5):
        ar = gpu_decode_batch(ctx, [src], [16], "ar")[0]
        for mode, b in [("jacobi", 0), ("gs_jacobi", 2), ("gs_jacobi", 5), ("hybrid", 3)]:
            say(f"case chain mode={mode} b={b}")
            g = gpu_decode_batch(ctx, [src], [16], mode, b)[0]
            np.testing.assert_array_equal(g.ids, ar.ids)


def test_graph_and_direct_launches_agree(monkeypatch):
    """Iterations replayed from a captured HIP graph give the same ids and k as
    directly launched iterations, on the fused (few rows) and separate (many
    rows) control paths."""
    results = {}
    for graphs in ("1", "0"):
        monkeypatch.setenv("PDEC_GRAPHS", graphs)
        _, _, ctx, _ = build(CHAIN, seed=1, max_batch=4, max_tgt=40, bias_std=0.5, ln_std=0.3)
        srcs = sources(CHAIN.vocab, 4, seed=8)
        out = []
        for mode, b, ms in [("ar", 1, [16] * 4), ("gs_jacobi", 5, [16] * 4), ("jacobi", 0, [40, 33, 20, 5])]:
            say(f"case graphs={graphs} mode={mode}")
            out.append([(g.ids.tolist(), g.k) for g in gpu_decode_batch(ctx, srcs, ms, mode, b)])
        results[graphs] = out
    assert results["1"] == results["0"]


def test_context_free_decoder_closed_form_k():
    cfg = dataclasses.replace(TINY, dec_emb_scale=0.0)
    _, _, ctx, M = build(cfg, seed=4, bias_std=0.3)
    for src in sources(cfg.vocab, 3, seed=5):
        for m in (2, 5, 16):
            ref = oracle.greedy(M, M.encode(src), m, stop_at_eos=False).y
            if np.any(ref == C.PAD_ID) or np.any(ref == C.EOS_ID):
                continue
            say(f"case context-free m={m}")
            assert gpu_decode_batch(ctx, [src], [m], "jacobi")[0].k == min(2, m)
            for b in (1, 2, 3, 4):
                want = sum(min(2, min(b, m - i)) for i in range(0, m, b))
                assert gpu_decode_batch(ctx, [src], [m], "gs_jacobi", b)[0].k == want


@pytest.mark.parametrize("cfg,seed,wkw", [(TINY, 8, dict(bias_std=0.5, ln_std=0.3)),
                                          (CHAIN, 9, dict(bias_std=0.5, ln_std=0.3)),
                                          (SMALL_PRE_BF16, 13, dict(bias_std=0.3, ln_std=0.2))],
                         ids=["tiny", "chain", "small_pre_bf16"])
def test_hybrid_eos_fixtures_and_horizons(cfg, seed, wkw):
    """[EOS] at a block start, inside a block, at a block's last position or
    absent (placed past the first block where possible), crossed with the
    hybrid horizon h in {1, b, m/2, m - 1, m}: an [EOS] in a converged block
    before h (CheckEOS) and an [EOS] in the greedy tail after h (IsEOS) both
    stop decoding exactly where the oracle stops."""
    from tests.test_oracle_decode import eos_cases
    m = 16
    for b in (3, 4):
        found = eos_cases(cfg, seed, wkw, b, m)
        assert {"absent", "start", "mid", "last"} <= set(found), sorted(found)
        for kind, (B, src, q) in found.items():
            _, _, ctx, M = build(cfg, seed=seed, eos_bias=B, **wkw)
            runs = [("ar", 1, 0), ("gs_jacobi", b, 0)] + [("hybrid", b, h) for h in (1, b, m // 2, m - 1, 0)]
            for mode, bb, h in runs:
                say(f"case eos cfg={cfg.name} b={b} kind={kind} q={q} mode={mode} h={h}")
                got, labs = judge_batch(ctx, M, [src], [m], mode, bb, cfg.dtype, horizon=h)
                lab = labs[0]
                assert not lab.startswith("FAIL"), f"{kind} q={q} {mode} h={h}: {lab}"
                if mode != "gs_jacobi" and lab == "exact":
                    ends = len(got[0].ids) and got[0].ids[-1] == C.EOS_ID
                    assert bool(got[0].flags & pdec.FLAG_EOS) == bool(ends)
                    if ends and mode == "hybrid":
                        where = "before" if len(got[0].ids) - 1 < (h or m) else "after"
                        say(f"  [EOS] at {len(got[0].ids) - 1}, {where} the horizon")


@pytest.mark.parametrize("cfg", [TINY, SMALL_PRE_BF16, MID_F32, MID_BF16, WIDE_PRE_BF16],
                         ids=["tiny_f32", "small_pre_bf16", "mid_f32", "mid_bf16", "wide_pre_bf16"])
def test_teacher_forced_logits_within_tolerance(cfg):
    import torch
    _, _, ctx, M = build(cfg, seed=6, max_tgt=96, bias_std=0.3, ln_std=0.2)
    srcs = sources(cfg.vocab, 2, n=13, seed=2)
    tgt = np.concatenate([np.ones((2, 1), np.int32),
                          np.random.default_rng(3).integers(0, cfg.vocab, (2, 11)).astype(np.int32)], 1)
    src = np.stack(srcs)
    ctx.encode(torch.from_numpy(src).cuda(), [13, 13])
    got = ctx.debug_logits(torch.from_numpy(tgt)).cpu().numpy()
    for r in range(2):
        ref = M.teacher_forced_logits(M.encode(srcs[r]), tgt[r])
        rel = np.abs(got[r] - ref).max(-1) / np.abs(ref).max(-1)
        say(f"case logits cfg={cfg.name} max rel err {rel.max():.3g}")
        assert rel.max() < EPS[cfg.dtype] <= TOL[cfg.dtype]


@pytest.mark.parametrize("cfg", [TINY, SMALL_PRE_BF16, MID_F32, MID_BF16, WIDE_PRE_BF16, FFN2K_BF16],
                         ids=["tiny_f32", "small_pre_bf16", "mid_f32", "mid_bf16", "wide_pre_bf16", "ffn2k_bf16"])
def test_rows_are_invariant_to_block_and_batch(cfg):
    """A row's logits are bitwise the same whatever else is in the call: fewer
    or more positions (row tiles, fused or separate LayerNorm) and batch mates."""
    import torch
    _, _, ctx, _ = build(cfg, seed=7, max_batch=3, max_tgt=96, bias_std=0.3, ln_std=0.2)
    srcs = sources(cfg.vocab, 3, n=10, seed=4)
    g = np.random.default_rng(9)
    tgt = np.concatenate([np.ones((3, 1), np.int32), g.integers(0, cfg.vocab, (3, 89)).astype(np.int32)], 1)
    ctx.encode(torch.from_numpy(np.stack(srcs)).cuda(), [10, 10, 10])
    full = ctx.debug_logits(torch.from_numpy(tgt)).cpu().numpy()           # 270 rows: separate LN, tiled products
    # 3, 9 and 24 rows: streaming products with the LayerNorm prologue; 90 rows:
    # the same for d <= 512, separate LN and tiled products for wider models
    for T in (1, 3, 8, 30):
        say(f"case row-invariance T={T}")
        part = ctx.debug_logits(torch.from_numpy(np.ascontiguousarray(tgt[:, :T]))).cpu().numpy()
        np.testing.assert_array_equal(part, full[:, :T])
    ctx.encode(torch.from_numpy(np.stack(srcs[1:2])).cuda(), [10])
    alone = ctx.debug_logits(torch.from_numpy(np.ascontiguousarray(tgt[1:2, :8]))).cpu().numpy()
    np.testing.assert_array_equal(alone[0], full[1, :8])


def test_batched_sentences_equal_single_decodes():
    _, _, ctx, M = build(TINY, seed=2, max_batch=4, bias_std=0.5, ln_std=0.3)
    g = np.random.default_rng(21)
    srcs = [g.integers(4, TINY.vocab, n).astype(np.int32) for n in (5, 16, 9, 12)]
    ms = [3, 16, 7, 11]
    for mode, b in [("ar", 1), ("jacobi", 0), ("gs_jacobi", 3), ("hybrid", 4)]:
        say(f"case batch mode={mode} b={b}")
        batch = gpu_decode_batch(ctx, srcs, ms, mode, b)
        for r in range(4):
            one = gpu_decode_batch(ctx, [srcs[r]], [ms[r]], mode, b)[0]
            np.testing.assert_array_equal(batch[r].ids, one.ids)
            assert batch[r].k == one.k
        _, labs = judge_batch(ctx, M, srcs, ms, mode, b, C.F32, got=batch)
        assert not any(lab.startswith("FAIL") for lab in labs), labs


def test_batch_above_the_inline_length_limit():
    """More than 64 sentences: the source and target lengths reach the device
    through the pinned staging copy instead of the first kernel's arguments;
    every sentence still equals its single decode (lengths passed inline)
    and the oracle."""
    _, _, ctx, M = build(TINY, seed=12, max_batch=70, bias_std=0.5, ln_std=0.3)
    g = np.random.default_rng(41)
    srcs = [g.integers(4, TINY.vocab, int(n)).astype(np.int32) for n in g.integers(1, 17, 70)]
    ms = [int(m) for m in g.integers(1, 17, 70)]
    for mode, b in [("gs_jacobi", 4), ("hybrid", 3)]:
        say(f"case batch of 70 mode={mode} b={b}")
        batch = gpu_decode_batch(ctx, srcs, ms, mode, b)
        for r in range(0, 70, 7):
            one = gpu_decode_batch(ctx, [srcs[r]], [ms[r]], mode, b)[0]
            np.testing.assert_array_equal(batch[r].ids, one.ids)
            assert batch[r].k == one.k
        _, labs = judge_batch(ctx, M, srcs, ms, mode, b, C.F32, idx=list(range(0, 70, 7)), got=batch)
        assert not any(lab.startswith("FAIL") for lab in labs), labs


@pytest.mark.parametrize("cfg,wkw", [(TINY, {}), (SMALL_PRE_BF16, dict(bias_std=0.5, ln_std=0.3))],
                         ids=["tiny_f32", "small_pre_bf16"])
def test_launch_bound_shrinks_with_the_rows(cfg, wkw):
    """A batch whose rows fall, as sentences finish, from above 128 through 128
    and 64: its iterations are launched with shrinking bounds (separate
    LayerNorm and tiled products, then LayerNorm prologues, then the control
    step that also embeds the next rows), and every sentence still equals its
    single decode bitwise and the oracle."""
    _, _, ctx, M = build(cfg, seed=5, max_batch=4, max_src=16, max_tgt=48, **wkw)
    srcs = sources(cfg.vocab, 4, n=12, seed=11)
    ms = [44, 6, 14, 33]   # Jacobi: 97 rows, then 91, 77 and 44 as sentences finish (k = 6, 14, 33, 37-44)
    for mode, b in [("jacobi", 0), ("gs_jacobi", 40), ("hybrid", 24)]:
        say(f"case launch-bound cfg={cfg.name} mode={mode} b={b} ms={ms}")
        batch = gpu_decode_batch(ctx, srcs, ms, mode, b)
        for r in range(4):
            one = gpu_decode_batch(ctx, [srcs[r]], [ms[r]], mode, b)[0]
            np.testing.assert_array_equal(batch[r].ids, one.ids)
            assert batch[r].k == one.k
        _, labs = judge_batch(ctx, M, srcs, ms, mode, b, cfg.dtype, got=batch)
        say(f"  {labs}")
        assert not any(lab.startswith("FAIL") for lab in labs), labs


def test_more_than_64_sentences_under_a_fused_control_step():
    """80 sentences of different lengths: once fewer than 65 rows are left,
    the bound selects the control step that also reduces the argmax partials
    and embeds the next rows, here the row-parallel one (more than 64
    sentences).  Every sentence equals its single decode bitwise."""
    _, _, ctx, M = build(TINY, seed=3, max_batch=80, max_src=16, max_tgt=24)
    g = np.random.default_rng(31)
    srcs = [g.integers(4, TINY.vocab, int(n)).astype(np.int32) for n in g.integers(4, 17, 80)]
    ms = [int(m) for m in g.integers(1, 25, 80)]
    for mode, b in [("ar", 1), ("hybrid", 2), ("gs_jacobi", 3)]:
        say(f"case 80 sentences mode={mode} b={b}")
        batch = gpu_decode_batch(ctx, srcs, ms, mode, b)
        for r in range(80):
            one = gpu_decode_batch(ctx, [srcs[r]], [ms[r]], mode, b)[0]
            np.testing.assert_array_equal(batch[r].ids, one.ids)
            assert batch[r].k == one.k
        _, labs = judge_batch(ctx, M, srcs, ms, mode, b, C.F32, idx=(0, 41, 79), got=batch)
        assert not any(lab.startswith("FAIL") for lab in labs), labs


def test_max_iters_and_horizon():
    _, _, ctx, M = build(CHAIN, seed=1, bias_std=0.5, ln_std=0.3)
    src = sources(CHAIN.vocab, 1, seed=3)[0]
    enc = M.encode(src)
    greedy = oracle.greedy(M, enc, 12)
    for mode, b in [("ar", 1), ("jacobi", 0), ("gs_jacobi", 4), ("hybrid", 4)]:
        say(f"case max_iters mode={mode}")
        want = oracle.decode(M, enc, 12, mode, b, max_iters=3)
        g = gpu_decode_batch(ctx, [src], [12], mode, b, max_iters=3)[0]
        assert g.k == 3 and (g.flags & pdec.FLAG_MAX_ITERS)
        n = len(want.out)
        if mode == "ar":      # greedy stops early: compare the produced prefix
            np.testing.assert_array_equal(g.ids[:n], want.out)
        else:
            np.testing.assert_array_equal(g.ids, want.out)
    for h in (1, 4, 7, 12):
        say(f"case horizon h={h}")
        _, labs = judge_batch(ctx, M, [src], [12], "hybrid", 3, C.F32, horizon=h)
        assert labs == ["exact"], labs


@pytest.mark.parametrize("cfg", [CHAIN, SMALL_PRE_BF16], ids=["chain_f32", "small_pre_bf16"])
def test_degenerate_and_extreme_shapes_match_oracle(cfg):
    """One-token targets and sources, blocks longer than the target, ragged
    batches mixing them with full-length sentences, and the context's maximum
    batch, source and target sizes: every mode against the oracle, and each
    batched sentence against its own single decode (bf16: the batched
    iterations of up to 128 rows run on the tiled products and the
    row-parallel control step)."""
    _, _, ctx, M = build(cfg, seed=9, max_batch=4, max_src=32, max_tgt=32, bias_std=0.5, ln_std=0.3)
    g = np.random.default_rng(16)
    modes = [("ar", 1), ("jacobi", 0), ("gs_jacobi", 4), ("gs_jacobi", 40), ("hybrid", 3), ("hybrid", 40)]
    cases = [([1], [1]), ([1], [2]), ([2], [1]), ([32], [32]), ([1, 16, 5, 32], [1, 16, 3, 32]),
             ([32, 32, 32, 32], [32, 1, 32, 2])]
    for lens, ms in cases:
        srcs = [g.integers(4, cfg.vocab, n).astype(np.int32) for n in lens]
        for mode, b in modes:
            say(f"case shapes lens={lens} m={ms} mode={mode} b={b}")
            got, labs = judge_batch(ctx, M, srcs, ms, mode, b, cfg.dtype)
            for r, (src, m) in enumerate(zip(srcs, ms)):
                assert not labs[r].startswith("FAIL"), f"{lens} {ms} {mode} b={b} sentence {r}: {labs[r]}"
                assert got[r].k <= m
                if len(srcs) > 1:
                    one = gpu_decode_batch(ctx, [src], [m], mode, b)[0]
                    np.testing.assert_array_equal(got[r].ids, one.ids)
                    assert got[r].k == one.k


def test_error_paths_on_device():
    import torch
    w = synth.make_weights(TINY, 0)
    gm = pdec.Model(TINY, w)
    ctx = pdec.Context(gm, 2, 16, 16)
    with pytest.raises(pdec.PdError) as e:
        ctx.B = 1
        ctx.decode("ar", [4])
    assert e.value.status == 6                          # decode before encode
    ctx.encode(torch.ones((1, 8), dtype=torch.int32).cuda() * 7, [8])
    for kw, status in [(dict(mode=9, tgt_m=[4]), 1), (dict(mode="ar", tgt_m=[17]), 2),
                       (dict(mode="ar", tgt_m=[0]), 2),
                       (dict(mode="gs_jacobi", tgt_m=[4], block=0), 1)]:
        with pytest.raises(pdec.PdError) as e:
            ctx.decode(**kw)
        assert e.value.status == status
    with pytest.raises(pdec.PdError) as e:
        ctx.encode(torch.ones((3, 8), dtype=torch.int32).cuda(), [8, 8, 8])   # batch > max_batch
    assert e.value.status == 2
    with pytest.raises(pdec.PdError) as e:
        ctx.encode(torch.ones((1, 8), dtype=torch.int32).cuda(), [9])         # length > n_max
    assert e.value.status == 1
    with pytest.raises(pdec.PdError) as e:
        ctx.encode(torch.ones((1, 8), dtype=torch.int32).cuda(), [0])         # empty source
    assert e.value.status == 1
    with pytest.raises(pdec.PdError) as e:
        ctx.encode(torch.ones((0, 8), dtype=torch.int32).cuda(), [])          # empty batch
    assert e.value.status == 1
    # the context still decodes after the refused calls
    ctx.encode(torch.ones((1, 8), dtype=torch.int32).cuda() * 7, [8])
    ids, ln, k, fl = ctx.decode("gs_jacobi", [6], block=3)
    torch.cuda.synchronize()
    assert 1 <= int(ln[0]) <= 6 and 1 <= int(k[0]) <= 6


def _full_size(wl_name, n_sent, m_cap, modes):
    wl = C.WORKLOADS[wl_name]
    cfg = wl.model
    _, gm, M = workload_model(cfg)
    ctx = pdec.Context(gm, 1, 128, wl.tgt_cap)
    labels = []
    for src, m in synth.make_sentences(wl, seed=1, count=n_sent):
        m = min(m, m_cap)
        for mode, b in modes:
            say(f"case {wl_name} mode={mode} b={b} n={len(src)} m={m}")
            got, labs = judge_batch(ctx, M, [src], [m], mode, b, cfg.dtype)
            say("  ->", labs[0], "k", got[0].k)
            assert not labs[0].startswith("FAIL"), labs[0]
            labels += labs
    return labels


@pytest.mark.parametrize("wl", ["mt_base_f32", "mt_base_bf16"])
def test_mt_base_sampled_sentences(wl):
    """Sampled MT-base sentences at their full m in all four modes (Jacobi over
    the whole target included)."""
    labels = _full_size(wl, 3, 128, [("ar", 1), ("jacobi", 0), ("gs_jacobi", 5), ("hybrid", 5)])
    s = summarize(labels)
    say(wl, s)
    # a near tie is a property of a sentence and shows in all four of its
    # decodes (each returns greedy decoding's ids)
    assert s["exact"] >= (1.0 if C.WORKLOADS[wl].model.dtype == C.F32 else 0.5) * len(labels)


def test_large_sampled_sentence_all_modes():
    """The large model at batch 1, one sentence cut to m = 20 so that the
    oracle replays every mode (Jacobi: 20 iterations of 20 rows)."""
    labels = _full_size("large", 1, 20, [("ar", 1), ("jacobi", 0), ("gs_jacobi", 16), ("hybrid", 16)])
    say("large", summarize(labels))


def test_large_sentences_full_length_replayed():
    """Large model, batch 1, two sentences at their full m in Jacobi,
    GS-Jacobi b = 16 and hybrid b = 16: the ids equal the oracle's greedy
    output; the oracle's block procedure run on the GPU's own evaluations of F
    (its decoding trace) reproduces the GPU's ids and k, which checks the
    on-device control at full size; and the GPU's tokens of a few whole
    iterations are recomputed by the oracle."""
    wl = C.WORKLOADS["large"]
    cfg = wl.model
    _, gm, M = workload_model(cfg)
    ctx = pdec.Context(gm, 1, 128, wl.tgt_cap)
    spots = []
    for src, m in synth.make_sentences(wl, seed=1, count=2):
        enc = M.encode(src)
        greedy = oracle.greedy(M, enc, m)
        for mode, b in [("jacobi", 0), ("gs_jacobi", 16), ("hybrid", 16)]:
            say(f"case large replay mode={mode} b={b} n={len(src)} m={m}")
            res, rows = gpu_decode_traced(ctx, [src], [m], mode, b)
            g = res[0]
            np.testing.assert_array_equal(g.ids, greedy.out)
            rep = replay_check(g, rows[0], mode, b, m)
            n_it = len(rep.iterations)
            spots += spot_check(rep, M, enc, cfg.dtype, sorted({0, n_it // 2, n_it - 1}))
            say(f"  k={g.k} iterations={n_it}")
    s = summarize(spots)
    say("large spot checks", s)
    assert s["fail"] == 0, [x for x in spots if x.startswith("FAIL")]
    assert s["exact"] >= 0.9 * len(spots)


def test_more_decoder_layers_than_one_cross_kv_launch_holds():
    """17 decoder layers: the cross-attention K/V products of pd_encode run as
    a 16-layer launch and a 1-layer launch; decodes still match the oracle."""
    cfg = dataclasses.replace(C.TINY, name="deep17", n_enc=1, n_dec=17)
    _, _, ctx, M = build(cfg, seed=8, bias_std=0.3, ln_std=0.2)
    labels = run_modes(cfg, ctx, M, sources(cfg.vocab, 2, seed=15), 12,
                       [("ar", 1), ("jacobi", 0), ("gs_jacobi", 4), ("hybrid", 3)])
    say(f"deep17: {summarize(labels)}")


def test_rows_processed_counts_block_positions():
    """The device row counter equals the positions the oracle's iterations
    evaluated: k for greedy, the sum of the block lengths of every iteration for
    the Jacobi modes."""
    _, _, ctx, M = build(CHAIN, seed=1, bias_std=0.5, ln_std=0.3)
    for src in sources(CHAIN.vocab, 2, seed=12):
        enc = M.encode(src)
        for mode, b in [("ar", 1), ("jacobi", 0), ("gs_jacobi", 3), ("hybrid", 4)]:
            say(f"case rows mode={mode} b={b}")
            want = oracle.decode(M, enc, 16, mode, b)
            ctx.set_timing(False)                   # resets the counter
            g = gpu_decode_batch(ctx, [src], [16], mode, b)[0]
            assert g.k == want.k
            expect = want.k if mode == "ar" else sum(len(blk) for _, _, blk in want.iterates)
            assert ctx.rows_processed() == expect


def test_initial_draft_variants_match_oracle():
    """pd_decode_init (InitT of Section 3.3): random drafts give the oracle's ids
    and k; the greedy solution as the draft is a fixed point recognised at once
    (Jacobi k = 1, GS-Jacobi k = number of blocks); batched drafts equal
    single-sentence decodes."""
    for cfg, wkw in [(TINY, {}), (CHAIN, dict(bias_std=0.5, ln_std=0.3))]:
        _, _, ctx, M = build(cfg, seed=5, **wkw)
        srcs = sources(cfg.vocab, 3, seed=14)
        for si, src in enumerate(srcs):
            enc = M.encode(src)
            for m in (7, 16):
                draft = synth.random_draft(m, cfg.vocab, 200 + si)
                for mode, b in [("jacobi", 0), ("gs_jacobi", 3), ("gs_jacobi", 4), ("hybrid", 4)]:
                    say(f"case init cfg={cfg.name} mode={mode} b={b} m={m}")
                    _, labs = judge_batch(ctx, M, [src], [m], mode, b, cfg.dtype, init=[draft])
                    assert not labs[0].startswith("FAIL"), f"{mode} b={b} m={m}: {labs[0]}"
            y_star = oracle.greedy(M, enc, 16, stop_at_eos=False).y
            say(f"case init fixed point cfg={cfg.name}")
            assert gpu_decode_batch(ctx, [src], [16], "jacobi", init=[y_star])[0].k == 1
            for b in (3, 4, 16):
                assert gpu_decode_batch(ctx, [src], [16], "gs_jacobi", b, init=[y_star])[0].k == -(-16 // b)
        drafts = [synth.random_draft(16, cfg.vocab, 300 + r) for r in range(3)]
        batch = gpu_decode_batch(ctx, srcs, [16, 11, 16], "gs_jacobi", 4, init=drafts)
        for r in range(3):
            one = gpu_decode_batch(ctx, [srcs[r]], [[16, 11, 16][r]], "gs_jacobi", 4, init=[drafts[r]])[0]
            np.testing.assert_array_equal(batch[r].ids, one.ids)
            assert batch[r].k == one.k


def _set_row(w, name, dst, src_row=None, value=None):
    """Weights edit on both the float values and the bf16 bit patterns."""
    if src_row is not None:
        w.values[name][dst] = w.values[name][src_row]
        if w.bf16_bits is not None:
            w.bf16_bits[name][dst] = w.bf16_bits[name][src_row]
    else:
        w.values[name][dst] = value
        if w.bf16_bits is not None:
            w.bf16_bits[name][dst] = np.float32(value).view(np.uint32) >> 16 if np.isfinite(value) \
                else (0x7FC0 if np.isnan(value) else (0x7F80 if value > 0 else 0xFF80))


@pytest.mark.parametrize("cfg", [TINY, SMALL_PRE_BF16], ids=["tiny_f32", "small_pre_bf16"])
@pytest.mark.parametrize("where", ["other_workgroup", "same_tile"])
def test_planted_exact_tie_takes_the_lowest_index(cfg, where):
    """Two vocabulary rows made identical (E[a] = E[t], bias[a] = bias[t], t a
    token the model emits, a unused) give bitwise equal logits, so every row
    where t was the argmax is an exact tie that the lower index of the two must
    win (reading R13) -- across workgroup partials (a in another 64-column
    group) and inside one 16-column tile.  a below t must take t's place, a
    above t must never appear.  Checked on the streaming argmax (blocks of <= 16
    rows), the product / tiled argmax (Jacobi over 32 positions, and 4
    sentences x 8) and greedy decoding, against the oracle."""
    w = synth.make_weights(cfg, seed=12, bias_std=0.3, ln_std=0.2)
    M0 = oracle.Model(cfg, w.values)
    srcs = sources(cfg.vocab, 4, seed=31)
    y = oracle.greedy(M0, M0.encode(srcs[0]), 32, stop_at_eos=False).y
    vals, counts = np.unique(y, return_counts=True)
    t = int(vals[np.argmax(counts)])
    used = set(y.tolist()) | set(np.concatenate(srcs).tolist()) | set(range(4))
    if where == "other_workgroup":
        cands = [c for c in range(cfg.vocab) if c // 64 != t // 64]
    else:
        cands = [c for c in (t - 1, t + 1) if c // 16 == t // 16]
    cands = [c for c in cands if c not in used]
    a = min(cands, key=lambda c: (c > t, abs(c - t)))       # below t where possible
    win, lose = min(a, t), max(a, t)
    _set_row(w, "emb", a, src_row=t)
    _set_row(w, "out_bias", a, src_row=t)
    gm = pdec.Model(cfg, w)
    ctx = pdec.Context(gm, 4, 32, 32)
    M = oracle.Model(cfg, w.values)
    for mode, b, ss, ms in [("ar", 1, srcs[:1], [32]), ("gs_jacobi", 4, srcs[:1], [32]),
                            ("jacobi", 0, srcs[:1], [32]), ("hybrid", 8, srcs, [32, 20, 32, 9])]:
        say(f"case tie {where} cfg={cfg.name} a={a} t={t} mode={mode} b={b} B={len(ss)}")
        got, labs = judge_batch(ctx, M, ss, ms, mode, b, cfg.dtype)
        assert not any(lab.startswith("FAIL") for lab in labs), labs
        assert labs[0] == "exact" and win in got[0].ids
        assert all(lose not in g.ids for g in got)     # the higher index never wins the tie


@pytest.mark.parametrize("cfg", [TINY, SMALL_PRE_BF16], ids=["tiny_f32", "small_pre_bf16"])
@pytest.mark.parametrize("plant", ["nan_bias", "inf_bias", "nan_ffn_weight"])
def test_nonfinite_logits_set_the_flag(cfg, plant):
    """A NaN or an infinity planted in the output bias (one vocabulary column)
    or in a decoder weight (every logit) sets PD_FLAG_NONFINITE for every
    sentence, on the streaming and on the many-row argmax; the oracle refuses
    such logits (reading R13)."""
    w = synth.make_weights(cfg, seed=13)
    if plant == "nan_bias":
        _set_row(w, "out_bias", 700, value=np.nan)
    elif plant == "inf_bias":
        _set_row(w, "out_bias", 700, value=np.inf)
    else:
        w.values["dec.0.ff.w1"][3, 5] = np.nan
        if w.bf16_bits is not None:
            w.bf16_bits["dec.0.ff.w1"][3, 5] = 0x7FC0
    gm = pdec.Model(cfg, w)
    ctx = pdec.Context(gm, 4, 32, 32)
    srcs = sources(cfg.vocab, 4, seed=33)
    for mode, b, ss, ms in [("ar", 1, srcs[:1], [8]), ("gs_jacobi", 4, srcs[:2], [12, 8]),
                            ("jacobi", 0, srcs, [32, 32, 17, 5])]:
        say(f"case nonfinite {plant} cfg={cfg.name} mode={mode} B={len(ss)}")
        got = gpu_decode_batch(ctx, ss, ms, mode, b)
        for g, m in zip(got, ms):
            assert g.flags & pdec.FLAG_NONFINITE, (plant, mode, g.flags)
            assert 1 <= g.k <= m
    M = oracle.Model(cfg, w.values)
    with pytest.raises(FloatingPointError):
        oracle.greedy(M, M.encode(srcs[0]), 4)
