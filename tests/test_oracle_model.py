"""Pins of the oracle's Transformer (oracle/model.py) against library routines,
invariants and brute force.  CPU only."""
import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import model as om
from paper_2305_10427_amd import configs as C, synth
from tests.torch_ref import TorchSeq2Seq

SMALL_POST = dataclasses.replace(C.TINY, name="small_post", vocab=97)
SMALL_PRE = dataclasses.replace(C.TINY, name="small_pre", vocab=97, pre_ln=True, act_gelu=True)


# --- elementary pieces --------------------------------------------------------

def test_round_bf16_matches_torch_on_float32_inputs():
    g = np.random.default_rng(0)
    x = np.concatenate([
        g.standard_normal(20000).astype(np.float32) * np.float32(10.0) ** g.integers(-20, 20, 20000).astype(np.float32),
        # exact ties: low 16 bits == 0x8000, both even and odd upper halves
        (((g.integers(0, 2 ** 15, 4000).astype(np.uint32) << 16) | 0x8000).view(np.float32)),
        # subnormals and near the bfloat16 overflow threshold
        np.array([1e-40, -3e-39, 1.2e-38, 3.3e38, -3.39e38, 0.0, -0.0], np.float32),
    ])
    x = x[np.isfinite(x)]
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = om.round_bf16(x.astype(np.float64))
    np.testing.assert_array_equal(got, want)


def test_round_bf16_is_idempotent_and_monotone():
    g = np.random.default_rng(1)
    x = np.sort(g.standard_normal(5000) * 100)
    r = om.round_bf16(x)
    np.testing.assert_array_equal(om.round_bf16(r), r)
    assert np.all(np.diff(r) >= 0)
    assert np.all(np.abs(r - x) <= np.abs(x) * 2.0 ** -8)


def test_sinusoid_invariants():
    d = 64
    P = om.sinusoid(np.arange(300), d)
    # position 0: all sines 0, all cosines 1
    np.testing.assert_allclose(P[0, 0::2], 0.0, atol=0)
    np.testing.assert_allclose(P[0, 1::2], 1.0, atol=0)
    # each (sin, cos) pair lies on the unit circle
    np.testing.assert_allclose(P[:, 0::2] ** 2 + P[:, 1::2] ** 2, 1.0, atol=1e-12)
    # relative-position property: pair at p+q is the pair at p rotated by the pair at q
    for p, q in [(3, 5), (17, 200), (250, 49)]:
        s_p, c_p, s_q, c_q = P[p, 0::2], P[p, 1::2], P[q, 0::2], P[q, 1::2]
        np.testing.assert_allclose(P[p + q, 0::2], s_p * c_q + c_p * s_q, atol=1e-10)
        np.testing.assert_allclose(P[p + q, 1::2], c_p * c_q - s_p * s_q, atol=1e-10)
    # frequencies: the first pair turns 1 radian per position, consecutive pairs
    # slow down by the constant factor 10000**(-2/d)
    ang = np.arctan2(P[1, 0::2], P[1, 1::2])
    assert ang[0] == pytest.approx(1.0, abs=1e-12)
    np.testing.assert_allclose(ang[1:] / ang[:-1], 10000.0 ** (-2.0 / d), rtol=1e-10)


def test_layer_norm_gelu_softmax_match_torch():
    g = np.random.default_rng(2)
    x = g.standard_normal((7, 48)) * 3 + 1
    gam, bet = g.standard_normal(48), g.standard_normal(48)
    want = torch.nn.functional.layer_norm(torch.tensor(x), (48,), torch.tensor(gam), torch.tensor(bet), 1e-5)
    np.testing.assert_allclose(om.layer_norm(x, gam, bet, 1e-5), want.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(om.gelu(x), torch.nn.functional.gelu(torch.tensor(x)).numpy(), rtol=1e-12, atol=1e-14)
    s = om.softmax_rows(x)
    np.testing.assert_allclose(s.sum(-1), 1.0, atol=1e-14)
    np.testing.assert_allclose(s, torch.softmax(torch.tensor(x), -1).numpy(), rtol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_attention_matches_torch_sdpa(causal):
    g = np.random.default_rng(3)
    Lq = Lk = 9
    d, H = 32, 4
    q, k, v = (g.standard_normal((Lq, d)) for _ in range(3))
    lim = np.arange(1, Lq + 1) if causal else None
    got = om.attention(q, k, v, H, key_limit=lim)
    tq, tk, tv = (torch.tensor(a).view(-1, H, d // H).transpose(0, 1) for a in (q, k, v))
    want = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=causal)
    np.testing.assert_allclose(got, want.transpose(0, 1).reshape(Lq, d).numpy(), rtol=1e-11, atol=1e-12)


def test_argmax_rows_ties_take_lowest_index_and_top2():
    lg = np.array([[1.0, 5.0, 5.0, 2.0], [0.0, -1.0, 3.0, 2.5], [7.0, 7.0, 7.0, 7.0]])
    recs = om.argmax_rows(lg, 4)
    assert [r.token for r in recs] == [1, 2, 0]
    assert [r.position for r in recs] == [4, 5, 6]
    assert [r.top1 - r.top2 for r in recs] == [0.0, 0.5, 0.0]
    assert recs[1].linf == 3.0
    with pytest.raises(FloatingPointError):
        om.argmax_rows(np.array([[0.0, np.nan]]), 0)


# --- whole model against torch.nn layers ---------------------------------------

@pytest.mark.parametrize("cfg", [SMALL_POST, SMALL_PRE], ids=["post_ln_relu", "pre_ln_gelu"])
def test_model_matches_torch_transformer_layers(cfg):
    w = synth.make_weights(cfg, seed=5, bias_std=0.3, ln_std=0.2, eos_bias=0.7)
    ref = TorchSeq2Seq(cfg, w.values)
    M = oracle.Model(cfg, w.values)
    g = np.random.default_rng(7)
    lens = [11, 6]                       # a padded batch of two sources
    src = np.zeros((2, 11), np.int64)
    srcs = [g.integers(4, cfg.vocab, n) for n in lens]
    for r, s in enumerate(srcs):
        src[r, :len(s)] = s
    tgt = np.concatenate([np.ones((2, 1), np.int64), g.integers(0, cfg.vocab, (2, 8))], 1)
    want = ref.logits(src, lens, tgt)
    for r in range(2):
        enc = M.encode(srcs[r])
        got = M.teacher_forced_logits(enc, tgt[r])
        np.testing.assert_allclose(got, want[r], rtol=1e-9, atol=1e-9)


def test_dec_emb_scale_knob_matches_torch():
    cfg = dataclasses.replace(SMALL_POST, dec_emb_scale=0.0)
    w = synth.make_weights(cfg, seed=9, bias_std=0.3, ln_std=0.2)
    ref = TorchSeq2Seq(cfg, w.values)
    M = oracle.Model(cfg, w.values)
    src = np.arange(4, 14)[None]
    tgt = np.array([[1, 5, 9, 33, 2]])
    np.testing.assert_allclose(M.teacher_forced_logits(M.encode(src[0]), tgt[0]),
                               ref.logits(src, [10], tgt)[0], rtol=1e-9, atol=1e-9)


# --- KV cache, causality ----------------------------------------------------------

@pytest.mark.parametrize("cfg", [SMALL_POST, SMALL_PRE.with_dtype(C.BF16)], ids=["f32", "bf16_pre"])
def test_cached_blocks_equal_full_recompute(cfg):
    w = synth.make_weights(cfg, seed=11, bias_std=0.2, ln_std=0.1)
    M = oracle.Model(cfg, w.values)
    g = np.random.default_rng(0)
    enc = M.encode(g.integers(4, cfg.vocab, 13))
    toks = np.concatenate([[1], g.integers(0, cfg.vocab, 15)])
    full = M.decode_rows(enc, M.new_cache(16), toks, 0)
    cache = M.new_cache(16)
    parts, p0 = [], 0
    for L in [1, 4, 3, 5, 2, 1]:
        parts.append(M.decode_rows(enc, cache, toks[p0:p0 + L], p0))
        p0 += L
    np.testing.assert_allclose(np.concatenate(parts), full, rtol=1e-11, atol=1e-11)


def test_causality_later_inputs_do_not_change_earlier_rows():
    cfg = SMALL_POST
    w = synth.make_weights(cfg, seed=12, bias_std=0.2, ln_std=0.1)
    M = oracle.Model(cfg, w.values)
    enc = M.encode(np.arange(4, 20))
    toks = np.array([1, 7, 8, 9, 10, 11, 12, 13])
    base = M.decode_rows(enc, M.new_cache(8), toks, 0)
    for q in range(1, 8):
        t2 = toks.copy()
        t2[q] = (t2[q] + 31) % cfg.vocab
        h = M.decode_rows(enc, M.new_cache(8), t2, 0)
        np.testing.assert_array_equal(h[:q], base[:q])
        assert not np.allclose(h[q], base[q])


def test_bf16_model_stays_close_to_unrounded_model():
    cfg = SMALL_PRE.with_dtype(C.BF16)
    w = synth.make_weights(cfg, seed=13, bias_std=0.2, ln_std=0.1)
    Mb = oracle.Model(cfg, w.values)
    Mf = oracle.Model(dataclasses.replace(cfg, dtype=C.F32), w.values)   # same bf16-valued weights
    src = np.arange(4, 30)
    tgt = np.array([1, 5, 9, 33, 2, 40, 41])
    lb = Mb.teacher_forced_logits(Mb.encode(src), tgt)
    lf = Mf.teacher_forced_logits(Mf.encode(src), tgt)
    rel = np.abs(lb - lf).max(-1) / np.abs(lf).max(-1)
    assert rel.max() < 5e-2
    assert rel.max() > 0           # rounding really happened


def test_encoded_memory_bf16_values_are_bf16():
    cfg = SMALL_POST.with_dtype(C.BF16)
    w = synth.make_weights(cfg, seed=14)
    M = oracle.Model(cfg, w.values)
    enc = M.encode(np.arange(4, 20))
    for a in [enc.memory] + enc.cross_k + enc.cross_v:
        np.testing.assert_array_equal(om.round_bf16(a), a)


def test_logit_scale_gives_std_near_three():
    """The tied output projection with s = 3 gives logits of standard deviation about 3."""
    cfg = C.TINY
    w = synth.make_weights(cfg, seed=0)
    M = oracle.Model(cfg, w.values)
    lg = M.teacher_forced_logits(M.encode(np.arange(4, 20)), np.array([1] + list(range(30, 45))))
    assert 2.5 < lg.std() < 3.5


def test_argmax_records_log_sum_exp():
    """The records' log-sum-exp is scipy's, and exp(top1 - lse) is the softmax
    probability of the argmax token (the quantity a decoding trace reports)."""
    from scipy.special import logsumexp, softmax
    from oracle.model import argmax_rows
    g = np.random.default_rng(7)
    logits = g.normal(0, 3, size=(5, 257))
    logits[2, 17] = logits[2].max() + 0.5
    recs = argmax_rows(logits, 3)
    for r, rec in enumerate(recs):
        assert rec.position == 3 + r
        assert rec.lse == pytest.approx(float(logsumexp(logits[r])), rel=1e-12, abs=1e-12)
        assert np.exp(rec.top1 - rec.lse) == pytest.approx(float(softmax(logits[r]).max()), rel=1e-12)


# --- the bf16 storage contract, against an independent functional model ----------

def test_reference_bf16_rounding_matches_torch_and_breaks_ties_to_even():
    """tests/bf16_ref.bf16 (integer rounding of the float64 pattern) agrees with
    torch's float32 -> bfloat16 conversion on float32 values, and on float64
    values next to a tie it rounds by the exact value, not by a float32 copy."""
    from tests.bf16_ref import bf16
    g = np.random.default_rng(4)
    x32 = (g.standard_normal(50000) * 10.0 ** g.integers(-30, 30, 50000)).astype(np.float32)
    x32 = np.concatenate([x32, ((g.integers(1, 2 ** 15, 4000).astype(np.uint32) << 16) | 0x8000).view(np.float32)])
    x32 = x32[np.isfinite(x32) & (np.abs(x32) >= 2.0 ** -126) & (np.abs(x32) < 3.3e38)]
    want = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64)
    np.testing.assert_array_equal(bf16(torch.from_numpy(x32.astype(np.float64))).numpy(), want.numpy())
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: a hair larger in magnitude rounds away from zero, a hair smaller towards it
    for tie in (1.0 + 2.0 ** -8, -(1.0 + 2.0 ** -8), 1.5 + 2.0 ** -8, 3.0 + 2.0 ** -7):
        r = bf16(torch.tensor([tie * (1 + 2.0 ** -40), tie * (1 - 2.0 ** -40), tie], dtype=torch.float64)).numpy()
        assert abs(r[0]) > abs(tie) > abs(r[1])
        assert r[2] in (r[0], r[1])
        assert (torch.tensor([r[2]], dtype=torch.float64).view(torch.int64).item() >> 45) & 1 == 0   # the even one
    np.testing.assert_array_equal(bf16(torch.tensor([0.0, -0.0], dtype=torch.float64)).numpy(), [0.0, -0.0])


@pytest.mark.parametrize("cfg", [SMALL_POST.with_dtype(C.BF16), SMALL_PRE.with_dtype(C.BF16)],
                         ids=["post_ln_relu_bf16", "pre_ln_gelu_bf16"])
def test_bf16_storage_contract_matches_functional_reference(cfg):
    """The oracle's bf16 model rounds at exactly the points of the storage
    contract: its teacher-forced logits equal those of tests/bf16_ref (torch
    functional layers, its own rounding) to 1e-12 relative, so one rounding
    more or less anywhere (each moves logits by about 1e-3) fails."""
    from tests.bf16_ref import Bf16Seq2Seq
    w = synth.make_weights(cfg, seed=15, bias_std=0.3, ln_std=0.2)
    M = oracle.Model(cfg, w.values)
    ref = Bf16Seq2Seq(cfg, w.values)
    g = np.random.default_rng(8)
    for n, T in [(11, 9), (5, 14)]:
        src = g.integers(4, cfg.vocab, n)
        tgt = np.concatenate([[1], g.integers(0, cfg.vocab, T - 1)])
        got = M.teacher_forced_logits(M.encode(src), tgt)
        want = ref.logits(src, tgt)
        rel = np.abs(got - want).max(-1) / np.abs(want).max(-1)
        assert rel.max() < 1e-12, rel.max()
    # the same model with no rounding at all differs at the 1e-3 level (the pin has power)
    Mf = oracle.Model(dataclasses.replace(cfg, dtype=C.F32), w.values)
    lf = Mf.teacher_forced_logits(Mf.encode(src), tgt)
    assert (np.abs(lf - want).max(-1) / np.abs(want).max(-1)).max() > 1e-4
