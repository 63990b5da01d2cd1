"""Pins of the oracle's decoding algorithms (oracle/decode.py): Proposition 1,
the triangular structure, brute-force fixed points on a tiny vocabulary,
closed-form iteration counts and special cases.  CPU only."""
import dataclasses
import itertools

import numpy as np
import pytest

import oracle
from oracle.decode import EOS, PAD
from paper_2305_10427_amd import configs as C, synth

TINY = C.TINY
# A fixture whose greedy output alternates between tokens, so each token
# depends on the one before it (a "hard" case for parallel decoding).
CHAIN = dataclasses.replace(C.TINY, name="chain", logit_scale=-3.0)
BRUTE = dataclasses.replace(C.TINY, name="brute", n_enc=1, n_dec=1, d_model=8, n_heads=2,
                            d_ff=16, vocab=8)


def _model(cfg, seed=0, **kw):
    w = synth.make_weights(cfg, seed=seed, **kw)
    return oracle.Model(cfg, w.values)


def _sources(cfg, count, n=16, seed=1):
    g = np.random.default_rng(seed)
    return [g.integers(4, cfg.vocab, n) for _ in range(count)]


CASES = [(TINY, 0, {}), (TINY, 3, dict(bias_std=0.5, ln_std=0.3)), (CHAIN, 1, dict(bias_std=0.5, ln_std=0.3))]


@pytest.mark.parametrize("cfg,seed,kw", CASES, ids=["tiny", "tiny_bias", "chain"])
def test_proposition1_all_modes_equal_greedy(cfg, seed, kw):
    M = _model(cfg, seed, **kw)
    for si, src in enumerate(_sources(cfg, 6, seed=seed + 10)):
        enc = M.encode(src)
        for m in (1, 2, 7, 16):
            ar_full = oracle.greedy(M, enc, m, stop_at_eos=False)
            ar = oracle.greedy(M, enc, m)
            assert ar_full.k == m
            np.testing.assert_array_equal(ar.out, oracle.cut_at_eos(ar_full.y))
            inits = [None, synth.random_draft(m, cfg.vocab, 100 + si)]
            for init in inits:
                for mode, b in [("jacobi", 0), ("gs_jacobi", 1), ("gs_jacobi", 3), ("gs_jacobi", 5),
                                ("hybrid", 2), ("hybrid", 4)]:
                    r = oracle.decode(M, enc, m, mode, b, init=init)
                    np.testing.assert_array_equal(r.out, ar.out, err_msg=f"{mode} b={b} m={m}")
                    assert 1 <= r.k <= m
                    assert not r.hit_max_iters
                    if mode != "hybrid":
                        np.testing.assert_array_equal(r.y, ar_full.y)


@pytest.mark.parametrize("cfg,seed,kw", CASES, ids=["tiny", "tiny_bias", "chain"])
def test_triangle_progress_per_iteration(cfg, seed, kw):
    """After j iterations of a block, its first j tokens are the greedy ones (Eq. (2) is triangular)."""
    M = _model(cfg, seed, **kw)
    for src in _sources(cfg, 4, seed=seed + 20):
        enc = M.encode(src)
        m = 16
        ref = oracle.greedy(M, enc, m, stop_at_eos=False).y
        r = oracle.jacobi(M, enc, m)
        for j, i, blk in r.iterates:
            np.testing.assert_array_equal(blk[:j], ref[:j])
        for b in (3, 4, 6):
            r = oracle.gs_jacobi(M, enc, m, b)
            j_in_block, last_i = 0, -1
            for _, i, blk in r.iterates:
                j_in_block = j_in_block + 1 if i == last_i else 1
                last_i = i
                np.testing.assert_array_equal(blk[:j_in_block], ref[i:i + j_in_block])


def test_chain_fixture_needs_every_iteration():
    """On the alternating fixture most blocks need all L iterations (k/m close to 1)."""
    M = _model(CHAIN, 1, bias_std=0.5, ln_std=0.3)
    ks = [oracle.gs_jacobi(M, M.encode(s), 16, 4).k for s in _sources(CHAIN, 6, seed=11)]
    assert np.mean(ks) / 16 > 0.9


def _brute_table(M, enc, V, m):
    """F(y) for every draft y in [0, V)^m, each recomputed from scratch (no cache)."""
    table = {}
    for y in itertools.product(range(V), repeat=m):
        toks = np.array((1,) + y[:-1])
        h = M.decode_rows(enc, M.new_cache(m), toks, 0)
        table[y] = tuple(int(t) for t in np.argmax(M.logits(h), axis=1))
    return table


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_brute_force_unique_fixed_point_and_trajectories(seed):
    V, m = BRUTE.vocab, 4
    M = _model(BRUTE, seed, bias_std=0.5, ln_std=0.3)
    enc = M.encode(np.array([4, 5, 6, 7, 5]))
    F = _brute_table(M, enc, V, m)
    fixed = [y for y, fy in F.items() if fy == y]
    ar = oracle.greedy(M, enc, m, stop_at_eos=False)
    assert fixed == [tuple(int(t) for t in ar.y)]          # the system has exactly one solution
    # Algorithm 1 step by step from the table, from PAD and from random drafts
    for init in [(PAD,) * m] + [tuple(synth.random_draft(m, V, s)) for s in range(5)]:
        y, traj = init, []
        for j in range(1, m + 1):
            ny = F[y]
            traj.append(ny)
            if ny == y:
                break
            y = ny
        r = oracle.jacobi(M, enc, m, init=np.array(init))
        assert r.k == len(traj)
        assert [tuple(int(t) for t in it) for _, _, it in r.iterates] == traj
    # Algorithm 2 (b = 2 and 3) step by step from the table
    for b in (2, 3):
        y, i, k = [PAD] * m, 0, 0
        while i < m:
            L = min(b, m - i)
            for j in range(1, L + 1):
                new = F[tuple(y)][i:i + L]
                k += 1
                unchanged = list(new) == y[i:i + L]
                y[i:i + L] = new
                if unchanged:
                    break
            i += L
        r = oracle.gs_jacobi(M, enc, m, b)
        assert r.k == k
        assert tuple(int(t) for t in r.y) == tuple(y)


def test_context_free_decoder_closed_form_iterations():
    """With the decoder's token embedding scaled to 0, F no longer depends on the draft:
    PJ needs min(2, m) iterations and PGJ(b) needs sum over blocks of min(2, L)."""
    cfg = dataclasses.replace(TINY, dec_emb_scale=0.0)
    M = _model(cfg, 4, bias_std=0.3)
    for src in _sources(cfg, 4, seed=5):
        enc = M.encode(src)
        for m in (1, 2, 5, 16):
            ref = oracle.greedy(M, enc, m, stop_at_eos=False).y
            assume_no_pad = not np.any(ref == PAD)
            if not assume_no_pad:
                continue
            assert oracle.jacobi(M, enc, m).k == min(2, m)
            for b in (1, 2, 3, 4, 16):
                want = sum(min(2, min(b, m - i)) for i in range(0, m, b))
                assert oracle.gs_jacobi(M, enc, m, b).k == want
            assert oracle.greedy(M, enc, m, stop_at_eos=False).k == m


def test_special_cases_between_modes():
    M = _model(CHAIN, 2, bias_std=0.5, ln_std=0.3)
    for src in _sources(CHAIN, 5, seed=6):
        enc = M.encode(src)
        m = 13
        ar_full = oracle.greedy(M, enc, m, stop_at_eos=False)
        # PGJ with b = 1 is greedy decoding: k = m
        r = oracle.gs_jacobi(M, enc, m, 1)
        assert r.k == m
        np.testing.assert_array_equal(r.y, ar_full.y)
        # PGJ with b >= m is PJ: same iterates, same k
        pj = oracle.jacobi(M, enc, m)
        for b in (m, m + 5):
            g = oracle.gs_jacobi(M, enc, m, b)
            assert g.k == pj.k
            assert [(k, i, list(t)) for k, i, t in g.iterates] == [(k, i, list(t)) for k, i, t in pj.iterates]
        # greedy with EOS stop is HGJ with b = 1
        ar = oracle.greedy(M, enc, m)
        h1 = oracle.hybrid(M, enc, m, 1)
        assert h1.k == ar.k
        np.testing.assert_array_equal(h1.out, ar.out)
        # HGJ without EOS in y_1..y_m is PGJ
        if not np.any(ar_full.y == EOS):
            for b in (2, 4):
                hb, gb = oracle.hybrid(M, enc, m, b), oracle.gs_jacobi(M, enc, m, b)
                assert hb.k == gb.k
                np.testing.assert_array_equal(hb.y, gb.y)


def test_recompute_path_gives_identical_results():
    M = _model(TINY, 3, bias_std=0.5, ln_std=0.3)
    enc = M.encode(_sources(TINY, 1, seed=7)[0])
    for mode, b in [("ar", 1), ("jacobi", 0), ("gs_jacobi", 3), ("hybrid", 4)]:
        a = oracle.decode(M, enc, 11, mode, b)
        r = oracle.decode(M, enc, 11, mode, b, recompute=True)
        assert a.k == r.k
        np.testing.assert_array_equal(a.out, r.out)


def eos_bias_for(cfg, seed, wkw, src, m, q):
    """An output bias on EOS that makes greedy decoding emit its first EOS at
    position q (None: impossible for this source).  Adding a bias B to EOS leaves
    the greedy prefix unchanged until the first position p whose gap
    top1_p - logit_EOS_p falls below B, so q is reachable iff its gap is below
    every earlier gap; B is put halfway between.  q = -1 asks for no EOS at all."""
    M = _model(cfg, seed, **wkw)
    enc = M.encode(src)
    y = oracle.greedy(M, enc, m, stop_at_eos=False).y
    if np.any(y == EOS):
        return None
    lg = M.teacher_forced_logits(enc, np.concatenate([[1], y[:-1]]))
    gap = lg.max(1) - lg[:, EOS]
    if q < 0:
        return 0.0
    lo, hi = gap[q], (gap[:q].min() if q else np.inf)
    if not lo < hi:
        return None
    return float(lo + min(hi - lo, 2.0) / 2)


def eos_cases(cfg, seed, wkw, b, m=16, tries=40):
    """One (bias, source, q) per kind: first EOS at a block start, inside a block,
    at a block's last position, or absent.  Positions past the first block are
    tried first, so that the EOS's block index and its absolute position differ."""
    found = {}
    for t in range(tries):
        src = np.random.default_rng(1000 + t).integers(4, cfg.vocab, 16)
        for q in [-1] + list(range(b, m)) + list(range(min(b, m))):
            if q < 0:
                kind = "absent"
            else:
                off, L = q % b, min(b, m - (q // b) * b)
                kind = "start" if off == 0 else ("last" if off == L - 1 else "mid")
            if kind in found:
                continue
            B = eos_bias_for(cfg, seed, wkw, src, m, q)
            if B is not None:
                found[kind] = (B, src, q)
        if len(found) == 4:
            break
    return found


@pytest.mark.parametrize("cfg,seed", [(TINY, 8), (CHAIN, 9)], ids=["tiny", "chain"])
@pytest.mark.parametrize("b", [3, 4])
def test_hybrid_eos_truncation_matches_greedy(cfg, seed, b):
    wkw = dict(bias_std=0.5, ln_std=0.3)
    found = eos_cases(cfg, seed, wkw, b)
    assert set(found) == {"start", "mid", "last", "absent"}, sorted(found)
    for kind, (B, src, q) in found.items():
        M = _model(cfg, seed, eos_bias=B, **wkw)
        enc = M.encode(src)
        ar = oracle.greedy(M, enc, 16)
        assert (len(ar.out) - 1 if ar.out[-1] == EOS else -1) == q, kind
        h = oracle.hybrid(M, enc, 16, b)
        np.testing.assert_array_equal(h.out, ar.out, err_msg=kind)
        assert h.k <= 16
        g = oracle.gs_jacobi(M, enc, 16, b)
        assert h.k <= g.k
        np.testing.assert_array_equal(g.out, ar.out)


def test_hybrid_finite_horizon_runs_autoregressive_tail():
    M = _model(CHAIN, 1, bias_std=0.5, ln_std=0.3)
    enc = M.encode(_sources(CHAIN, 1, seed=3)[0])
    m = 14
    ar = oracle.greedy(M, enc, m)
    for h in (0, 4, 7, 14):
        r = oracle.hybrid(M, enc, m, 3, h=h)
        np.testing.assert_array_equal(r.out, ar.out)
        assert r.k <= m


def test_max_iters_cap():
    M = _model(CHAIN, 1, bias_std=0.5, ln_std=0.3)
    enc = M.encode(_sources(CHAIN, 1, seed=3)[0])
    m = 12
    full = oracle.gs_jacobi(M, enc, m, 4)
    assert full.k > 3
    for mode, b in [("ar", 1), ("jacobi", 0), ("gs_jacobi", 4), ("hybrid", 4)]:
        r = oracle.decode(M, enc, m, mode, b, max_iters=3)
        assert r.k == 3 and r.hit_max_iters, mode
        r = oracle.decode(M, enc, m, mode, b, max_iters=m)
        assert not r.hit_max_iters


@pytest.mark.parametrize("cfg,seed,kw", CASES, ids=["tiny", "tiny_bias", "chain"])
def test_greedy_solution_as_draft_is_a_fixed_point(cfg, seed, kw):
    """Initialised with the greedy solution y* (the unique solution of the
    triangular system, Eq. (2)), every iteration reproduces its block: Jacobi
    stops after one iteration and GS-Jacobi after one iteration per block."""
    M = _model(cfg, seed, **kw)
    for src in _sources(cfg, 3, seed=seed + 20):
        enc = M.encode(src)
        for m in (1, 7, 16):
            y_star = oracle.greedy(M, enc, m, stop_at_eos=False).y
            r = oracle.jacobi(M, enc, m, init=y_star)
            assert r.k == 1
            np.testing.assert_array_equal(r.y, y_star)
            for b in (1, 3, 4, m):
                r = oracle.gs_jacobi(M, enc, m, b, init=y_star)
                assert r.k == -(-m // b)
                np.testing.assert_array_equal(r.y, y_star)


# ---------------------------------------------------------------------------
# The prefix stopping condition (a variant of Eq. (3); see oracle/decode.py)


@pytest.mark.parametrize("cfg,seed,kw", CASES, ids=["tiny", "tiny_bias", "chain"])
def test_prefix_stop_equals_greedy_and_commits_every_iteration(cfg, seed, kw):
    """Proposition 1 carries over: every mode under stop="prefix" returns the
    greedy output, from [PAD] drafts and from random ones; every iteration
    moves the block start forward (at least one position is committed), so
    k <= m without a cap; and the block start never moves back."""
    M = _model(cfg, seed, **kw)
    for si, src in enumerate(_sources(cfg, 5, seed=seed + 30)):
        enc = M.encode(src)
        for m in (1, 2, 7, 16):
            ar_full = oracle.greedy(M, enc, m, stop_at_eos=False)
            ar = oracle.greedy(M, enc, m)
            for init in (None, synth.random_draft(m, cfg.vocab, 200 + si)):
                for mode, b in [("jacobi", 0), ("gs_jacobi", 1), ("gs_jacobi", 3), ("gs_jacobi", 5),
                                ("hybrid", 2), ("hybrid", 4)]:
                    r = oracle.decode(M, enc, m, mode, b, init=init, stop="prefix")
                    np.testing.assert_array_equal(r.out, ar.out, err_msg=f"prefix {mode} b={b} m={m}")
                    assert 1 <= r.k <= m and not r.hit_max_iters
                    starts = [i for _, i, _ in r.iterates]
                    assert all(b2 > a2 for a2, b2 in zip(starts, starts[1:])), starts
                    if mode != "hybrid":
                        np.testing.assert_array_equal(r.y, ar_full.y)


class _Scripted:
    """A stand-in for the decoder: F(y)[p] = T[p] when p = 0 or y[p-1] = T[p-1],
    else the wrong token 3 (a chain whose links are right only after a right
    predecessor)."""

    def __init__(self, T):
        self.T, self.records, self.calls = list(T), [], []

    def block(self, y, i, L):
        self.calls.append((i, L))
        return np.array([self.T[p] if p == 0 or y[p - 1] == self.T[p - 1] else 3 for p in range(i, i + L)],
                        np.int32)


def test_prefix_stop_worked_example():
    """A hand-worked case, m = 6, b = 3, T = (5 6 7 8 9 10), draft
    (5 6 PAD PAD 9 10):
      prefix: [0,3) -> 5 6 7 (5 6 came out as they went in: commit 3);
              [3,6) -> 8 3 10 (first position changed: commit 1);
              [4,6) -> 9 3 (commit 1); [5,6) -> 10 (commit 1): k = 4.
      Eq. (3): [0,3) 5 6 7, then unchanged (2 iterations); [3,6) 8 3 10,
              8 9 3, 8 9 10 (cap of 3 iterations): k = 5."""
    T = [5, 6, 7, 8, 9, 10]
    draft = np.array([5, 6, PAD, PAD, 9, 10], np.int32)
    ev = _Scripted(T)
    r = oracle.gs_jacobi(None, None, 6, 3, init=draft, evaluator=ev, stop="prefix")
    assert r.k == 4 and ev.calls == [(0, 3), (3, 3), (4, 2), (5, 1)]
    np.testing.assert_array_equal(r.y, T)
    ev = _Scripted(T)
    r = oracle.gs_jacobi(None, None, 6, 3, init=draft, evaluator=ev)
    assert r.k == 5 and ev.calls == [(0, 3), (0, 3), (3, 3), (3, 3), (3, 3)]
    np.testing.assert_array_equal(r.y, T)
    # a perfect draft: every iteration finds its block unchanged and commits it whole
    ev = _Scripted(T)
    r = oracle.gs_jacobi(None, None, 6, 4, init=np.array(T, np.int32), evaluator=ev, stop="prefix")
    assert r.k == 2 and ev.calls == [(0, 4), (4, 2)]
    # [PAD] drafts: only the block start is ever proven, one position per iteration
    ev = _Scripted(T)
    r = oracle.jacobi(None, None, 6, evaluator=ev, stop="prefix")
    assert r.k == 6 and ev.calls == [(i, 6 - i) for i in range(6)]


@pytest.mark.parametrize("cfg,seed", [(TINY, 8), (CHAIN, 9)], ids=["tiny", "chain"])
@pytest.mark.parametrize("b", [3, 4])
def test_prefix_stop_hybrid_eos(cfg, seed, b):
    """[EOS] at a block start, inside a block, at a block's end or absent, crossed
    with horizons: the prefix variant of HGJ stops exactly where greedy
    decoding does (an [EOS] is acted on only once it is committed)."""
    m = 16
    wkw = dict(bias_std=0.5, ln_std=0.3)
    found = eos_cases(cfg, seed, wkw, b, m)
    assert set(found) == {"start", "mid", "last", "absent"}, sorted(found)
    for kind, (B, src, q) in found.items():
        M = _model(cfg, seed, eos_bias=B, **wkw)
        enc = M.encode(src)
        ar = oracle.greedy(M, enc, m)
        for h in (1, b, m // 2, m - 1, m):
            r = oracle.hybrid(M, enc, m, b, h=h, stop="prefix")
            np.testing.assert_array_equal(r.out, ar.out, err_msg=f"{kind} h={h}")
            assert r.k <= len(ar.out)
