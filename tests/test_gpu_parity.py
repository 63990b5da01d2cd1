"""Parity of the HIP decoding path (through the C ABI) with the CPU oracle.

Every test is marked gpu: it needs an MI355X and the built libpdec.so.  The
oracle (oracle/) provides every expected value; nothing expected comes from
the GPU path itself."""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2305_10427_amd import configs as C, pdec, synth
from tests.parity import TOL, classify, gpu_decode_batch, summarize, workload_model

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


def run_modes(cfg, ctx, M, srcs, m, modes, tol):
    labels = []
    for src in srcs:
        enc = M.encode(src)
        greedy = oracle.greedy(M, enc, m)
        for mode, b in modes:
            say(f"case cfg={cfg.name} mode={mode} b={b} m={m} n={len(src)}")
            want = oracle.decode(M, enc, m, mode, b)
            g = gpu_decode_batch(ctx, [src], [m], mode, b)[0]
            lab = classify(g, want, greedy, tol)
            assert not lab.startswith("FAIL"), f"{mode} b={b}: {lab}"
            assert g.k <= m
            labels.append(lab)
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
        labels += run_modes(cfg, ctx, M, sources(cfg.vocab, 4, seed=11), m, modes, TOL[cfg.dtype])
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


def test_hybrid_eos_fixtures():
    from tests.test_oracle_decode import eos_cases
    for cfg, seed in [(TINY, 8), (CHAIN, 9)]:
        wkw = dict(bias_std=0.5, ln_std=0.3)
        for b in (3, 4):
            found = eos_cases(cfg, seed, wkw, b)
            for kind, (B, src, q) in found.items():
                say(f"case eos cfg={cfg.name} b={b} kind={kind} q={q}")
                _, _, ctx, M = build(cfg, seed=seed, eos_bias=B, **wkw)
                enc = M.encode(src)
                greedy = oracle.greedy(M, enc, 16)
                for mode, bb in [("ar", 1), ("hybrid", b), ("gs_jacobi", b)]:
                    want = oracle.decode(M, enc, 16, mode, bb)
                    g = gpu_decode_batch(ctx, [src], [16], mode, bb)[0]
                    lab = classify(g, want, greedy, TOL[cfg.dtype])
                    assert not lab.startswith("FAIL"), f"{kind} {mode}: {lab}"
                    if mode != "gs_jacobi" and kind != "absent" and lab == "exact":
                        assert g.flags & pdec.FLAG_EOS


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
        assert rel.max() < TOL[cfg.dtype]


@pytest.mark.parametrize("cfg", [TINY, SMALL_PRE_BF16, MID_F32, MID_BF16, WIDE_PRE_BF16],
                         ids=["tiny_f32", "small_pre_bf16", "mid_f32", "mid_bf16", "wide_pre_bf16"])
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
            want = oracle.decode(M, M.encode(srcs[r]), ms[r], mode, b)
            lab = classify(batch[r], want, oracle.greedy(M, M.encode(srcs[r]), ms[r]), TOL[C.F32])
            assert not lab.startswith("FAIL"), lab


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
            enc = M.encode(srcs[r])
            want = oracle.decode(M, enc, ms[r], mode, b)
            lab = classify(batch[r], want, oracle.greedy(M, enc, ms[r]), TOL[cfg.dtype])
            say(f"  sentence {r} m={ms[r]}: {lab} k={batch[r].k}")
            assert not lab.startswith("FAIL"), lab


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
        for r in (0, 41, 79):
            enc = M.encode(srcs[r])
            want = oracle.decode(M, enc, ms[r], mode, b)
            lab = classify(batch[r], want, oracle.greedy(M, enc, ms[r]), TOL[C.F32])
            assert not lab.startswith("FAIL"), lab


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
        want = oracle.hybrid(M, enc, 12, 3, h=h)
        g = gpu_decode_batch(ctx, [src], [12], "hybrid", 3, horizon=h)[0]
        assert classify(g, want, greedy, TOL[C.F32]) == "exact"


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
            got = gpu_decode_batch(ctx, srcs, ms, mode, b)
            for r, (src, m) in enumerate(zip(srcs, ms)):
                enc = M.encode(src)
                want = oracle.decode(M, enc, m, mode, b)
                lab = classify(got[r], want, oracle.greedy(M, enc, m), TOL[cfg.dtype])
                assert not lab.startswith("FAIL"), f"{lens} {ms} {mode} b={b} sentence {r}: {lab}"
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
        enc = M.encode(src)
        greedy = oracle.greedy(M, enc, m)
        for mode, b in modes:
            say(f"case {wl_name} mode={mode} b={b} n={len(src)} m={m}")
            want = oracle.decode(M, enc, m, mode, b)
            g = gpu_decode_batch(ctx, [src], [m], mode, b)[0]
            lab = classify(g, want, greedy, TOL[cfg.dtype])
            say("  ->", lab, "k", g.k, "oracle k", want.k)
            assert not lab.startswith("FAIL"), lab
            labels.append(lab)
    return labels


@pytest.mark.parametrize("wl", ["mt_base_f32", "mt_base_bf16"])
def test_mt_base_sampled_sentences(wl):
    labels = _full_size(wl, 2, 128, [("ar", 1), ("gs_jacobi", 5), ("hybrid", 5)])
    say(wl, summarize(labels))


def test_large_sampled_sentence():
    labels = _full_size("large", 1, 24, [("ar", 1), ("jacobi", 0), ("gs_jacobi", 16)])
    say("large", summarize(labels))


def test_more_decoder_layers_than_one_cross_kv_launch_holds():
    """17 decoder layers: the cross-attention K/V products of pd_encode run as
    a 16-layer launch and a 1-layer launch; decodes still match the oracle."""
    cfg = dataclasses.replace(C.TINY, name="deep17", n_enc=1, n_dec=17)
    _, _, ctx, M = build(cfg, seed=8, bias_std=0.3, ln_std=0.2)
    labels = run_modes(cfg, ctx, M, sources(cfg.vocab, 2, seed=15), 12,
                       [("ar", 1), ("jacobi", 0), ("gs_jacobi", 4), ("hybrid", 3)], TOL[cfg.dtype])
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
            greedy = oracle.greedy(M, enc, 16)
            for m in (7, 16):
                draft = synth.random_draft(m, cfg.vocab, 200 + si)
                for mode, b in [("jacobi", 0), ("gs_jacobi", 3), ("gs_jacobi", 4), ("hybrid", 4)]:
                    say(f"case init cfg={cfg.name} mode={mode} b={b} m={m}")
                    want = oracle.decode(M, enc, m, mode, b, init=draft)
                    g = gpu_decode_batch(ctx, [src], [m], mode, b, init=[draft])[0]
                    lab = classify(g, want, oracle.greedy(M, enc, m), TOL[cfg.dtype])
                    assert not lab.startswith("FAIL"), f"{mode} b={b} m={m}: {lab}"
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
