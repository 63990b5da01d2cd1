"""CPU oracle, part 2: greedy autoregressive decoding and the paper's three
parallel decoding algorithms.

TEST INFRASTRUCTURE ONLY (see oracle/model.py): never called by the HIP path.

Notation follows Section 3: the target y = (y_1 .. y_m) solves the triangular
system of Eq. (2), f(y_i, y_{1:i-1}, x) = y_i - argmax p_theta(y_i | y_{1:i-1}, x) = 0.
Here y is a 0-based numpy array, so y[t] is y_{t+1}.  The decoder input at
position p is [BOS] for p = 0 and y[p-1] otherwise, and its prediction is the
new value of y[p]; this is the "shift left" of predictions that Appendix A
mentions.  F(y)[p] denotes that prediction.  One iteration is one decoder
forward over the active block.

Greedy decoding (Eq. (1)) is written out on its own, as the plain definition
of the result every parallel mode must reproduce (Proposition 1).

The three parallel algorithms of Section 3.2 (Algorithms 1-3 of Appendix A)
are one procedure with different block schedules.  The m positions are cut
into consecutive blocks, solved one after another (Gauss-Seidel from block
to block); inside the current block [i, i + L) every iteration recomputes
all L positions at once from the committed prefix y[0..i-1] and the block's
previous values (Jacobi), and the block is committed as soon as an iteration
leaves it unchanged (the stopping condition of Eq. (3)):

    mode       block lengths                            stop at [EOS]
    jacobi     one block of all m positions (PJ)        no
    gs_jacobi  b, b, ..., the rest (PGJ)                no
    hybrid     b, b, ... up to the horizon h, then      yes, after a committed
               blocks of one position (HGJ)             block that holds [EOS]

Readings where the paper leaves a detail open (each is listed in the design
notes of the repository as well):

* Algorithms 2 and 3 leave the block loop with a ``break`` when a block stops;
  the text of Section 3.2 says decoding then continues with the next block, so
  ``break`` ends only the current block's Jacobi loop.
* Blocks are half-open, [i, i+L) with L = min(b, m - i); the last one is cut at m.
* Each block runs at most L iterations: after L Jacobi iterations the block is
  exact by the triangular structure (its j-th token is exact after j
  iterations), so it counts as converged.  PJ's cap is the m of its for-loop.
  This keeps Proposition 1's bound of at most m iterations.
* StopC (Eq. (3)) compares the whole block with its previous value.
* CheckEOS returns the absolute index of the first [EOS] of a converged block;
  the output keeps that [EOS].  HGJ's horizon h defaults to m (Section 4.1);
  its autoregressive tail tests the token it just produced and never runs past m.
* PJ and PGJ solve all m equations; their output is cut after the first [EOS].
* Greedy AR stops after producing [EOS] (Eq. (1) with the usual end-of-sentence rule).
* The argmax takes the lowest index on exact ties; non-finite logits raise.

A stopping-condition variant (the paper leaves other stopping conditions to
future work, Section 3.3 and the conclusion): stop="prefix" commits, after
every iteration, the longest prefix of the block that the iteration has
proven exact, instead of waiting for the whole block to repeat (Eq. (3)).
Position i (the block start) is exact after any iteration, since its input is
the committed prefix; if the first t positions of the block came out as they
went in, those inputs were exact, so positions i .. i+t are exact.  With t the
number of leading unchanged positions, the iteration commits all L positions
when t = L (Eq. (3) holds) and t + 1 otherwise; the next block starts right
after the committed positions and keeps the newer values as its draft.  Every
iteration commits at least one position, so k <= m without a per-block cap,
and the output is greedy decoding's (the argument of Proposition 1).  HGJ
stops at an [EOS] among the committed positions only.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

from .model import ArgmaxRecord, Encoded, Model, argmax_rows

PAD, BOS, EOS = 0, 1, 2


@dataclasses.dataclass
class Result:
    y: np.ndarray                 # final iterate: length m, or cut after the [EOS] decoding stopped at
    out: np.ndarray               # output ids, cut after the first EOS (inclusive)
    k: int                        # decoder forwards (iterations) used
    hit_max_iters: bool = False
    records: List[ArgmaxRecord] = dataclasses.field(default_factory=list)
    iterates: List[tuple] = dataclasses.field(default_factory=list)   # (k, i, block tokens)

    def min_rel_margin(self) -> float:
        """Smallest (top1 - top2) / max|logit| over every argmax evaluated."""
        if not self.records:
            return float("inf")
        return min((r.top1 - r.top2) / max(r.linf, 1e-30) for r in self.records)


def cut_at_eos(y: np.ndarray) -> np.ndarray:
    hit = np.nonzero(y == EOS)[0]
    return y[: hit[0] + 1].copy() if len(hit) else y.copy()


class Solver:
    """Evaluates the map F over a block of the draft, with a KV cache.

    F(y)[p] = argmax p_theta(. | BOS, y[0..p-1], x).  ``block(y, i, L)``
    returns the new y[i..i+L-1] given the committed prefix y[0..i-1], whose
    K/V are in the cache, and writes the K/V of positions i..i+L-1.
    With recompute=True it ignores the cache and recomputes positions
    0..i+L-1 from scratch (brute force).
    """

    def __init__(self, model: Model, enc: Encoded, m: int, recompute: bool = False):
        self.model, self.enc, self.m, self.recompute = model, enc, m, recompute
        self.cache = model.new_cache(m)
        self.records: List[ArgmaxRecord] = []

    def inputs(self, y: np.ndarray, i: int, L: int) -> np.ndarray:
        return np.array([BOS if p == 0 else int(y[p - 1]) for p in range(i, i + L)], np.int64)

    def block(self, y: np.ndarray, i: int, L: int) -> np.ndarray:
        if self.recompute:
            cache = self.model.new_cache(self.m)
            h = self.model.decode_rows(self.enc, cache, self.inputs(y, 0, i + L), 0)[i:]
        else:
            h = self.model.decode_rows(self.enc, self.cache, self.inputs(y, i, L), i)
        recs = argmax_rows(self.model.logits(h), i)
        self.records.extend(recs)
        return np.array([r.token for r in recs], np.int32)


def _init(m: int, init: Optional[np.ndarray]) -> np.ndarray:
    """InitT (Section 3.3): all [PAD] unless an explicit draft is given."""
    return np.full(m, PAD, np.int32) if init is None else np.array(init, np.int32).copy()


def _cap(m: int, max_iters: Optional[int]) -> int:
    return m if max_iters is None or max_iters <= 0 else max_iters


def greedy(model: Model, enc: Encoded, m: int, stop_at_eos: bool = True,
           max_iters: Optional[int] = None, recompute: bool = False, evaluator=None) -> Result:
    """Greedy autoregressive decoding, Eq. (1): y[t] = argmax p(. | y[0..t-1], x), t = 0..m-1.

    evaluator: optional stand-in for the model's Solver (see solve_by_blocks)."""
    s = Solver(model, enc, m, recompute) if evaluator is None else evaluator
    cap = _cap(m, max_iters)
    y = np.full(m, PAD, np.int32)
    k, t = 0, 0
    while t < m:
        if k >= cap:
            return Result(y[:t], cut_at_eos(y[:t]), k, True, s.records)
        y[t] = s.block(y, t, 1)[0]
        k += 1
        t += 1
        if stop_at_eos and y[t - 1] == EOS:
            break
    return Result(y[:t].copy(), cut_at_eos(y[:t]), k, False, s.records)


def block_length(mode: str, i: int, m: int, b: int, h: int) -> int:
    """Length of the block that starts at position i (see the table above)."""
    if mode == "jacobi":
        return m - i
    if mode == "gs_jacobi":
        return min(b, m - i)
    if mode == "hybrid":
        return min(b, h - i) if i < h else 1
    raise ValueError(mode)


def solve_by_blocks(model: Model, enc: Encoded, m: int, mode: str, b: int = 1, h: Optional[int] = None,
                    init=None, max_iters: Optional[int] = None, recompute: bool = False,
                    evaluator=None, stop: str = "block") -> Result:
    """The block fixed-point procedure shared by PJ, PGJ and HGJ (Section 3.2).

    evaluator: optional stand-in for the model's Solver (an object with the
    same ``block(y, i, L)`` and ``records``), so that a recorded sequence of
    evaluations of F can be replayed through exactly this control flow.
    stop: "block" (Eq. (3)) or "prefix" (the variant described above).
    """
    if stop == "prefix":
        return _solve_prefix(model, enc, m, mode, b, h, init, max_iters, recompute, evaluator)
    if stop != "block":
        raise ValueError(stop)
    F = Solver(model, enc, m, recompute) if evaluator is None else evaluator
    cap = _cap(m, max_iters)
    h = m if h is None else min(h, m)
    y = _init(m, init)
    res = Result(y, y, 0)
    i = 0
    while i < m:
        L = block_length(mode, i, m, b, h)
        committed = False
        for j in range(1, L + 1):                 # at most L iterations per block
            if res.k >= cap:
                res.hit_max_iters = True
                break
            before = y[i:i + L].copy()
            y[i:i + L] = F.block(y, i, L)
            res.k += 1
            res.iterates.append((res.k, i, y[i:i + L].copy()))
            if np.array_equal(y[i:i + L], before) or j == L:   # Eq. (3), or exact after L iterations
                committed = True
                break
        if not committed:                         # the iteration budget ran out inside the block
            break
        if mode == "hybrid":
            hit = np.nonzero(y[i:i + L] == EOS)[0]
            if len(hit):                          # CheckEOS: stop at the block's first [EOS]
                y = y[: i + int(hit[0]) + 1].copy()
                break
        i += L
    res.y, res.out, res.records = y, cut_at_eos(y), F.records
    return res


def _solve_prefix(model: Model, enc: Encoded, m: int, mode: str, b: int, h: Optional[int], init,
                  max_iters: Optional[int], recompute: bool, evaluator) -> Result:
    """The blocks of solve_by_blocks under stop="prefix": every iteration
    commits the block's proven prefix and the block moves on by that much."""
    F = Solver(model, enc, m, recompute) if evaluator is None else evaluator
    cap = _cap(m, max_iters)
    h = m if h is None else min(h, m)
    y = _init(m, init)
    res = Result(y, y, 0)
    i = 0
    while i < m:
        if res.k >= cap:
            res.hit_max_iters = True
            break
        L = block_length(mode, i, m, b, h)
        before = y[i:i + L].copy()
        y[i:i + L] = F.block(y, i, L)
        res.k += 1
        res.iterates.append((res.k, i, y[i:i + L].copy()))
        t = 0                                     # leading positions that came out as they went in
        while t < L and y[i + t] == before[t]:
            t += 1
        c = L if t == L else t + 1                # positions proven exact
        if mode == "hybrid":
            hit = np.nonzero(y[i:i + c] == EOS)[0]
            if len(hit):                          # an [EOS] among the committed positions
                y = y[: i + int(hit[0]) + 1].copy()
                break
        i += c
    res.y, res.out, res.records = y, cut_at_eos(y), F.records
    return res


def jacobi(model: Model, enc: Encoded, m: int, init=None, max_iters: Optional[int] = None,
           recompute: bool = False, evaluator=None, stop: str = "block") -> Result:
    """Parallel Jacobi decoding (Algorithm 1): one block of all m positions."""
    return solve_by_blocks(model, enc, m, "jacobi", init=init, max_iters=max_iters, recompute=recompute,
                           evaluator=evaluator, stop=stop)


def gs_jacobi(model: Model, enc: Encoded, m: int, b: int, init=None,
              max_iters: Optional[int] = None, recompute: bool = False, evaluator=None,
              stop: str = "block") -> Result:
    """Parallel GS-Jacobi decoding (Algorithm 2): Jacobi inside b-blocks, Gauss-Seidel across them."""
    return solve_by_blocks(model, enc, m, "gs_jacobi", b, init=init, max_iters=max_iters, recompute=recompute,
                           evaluator=evaluator, stop=stop)


def hybrid(model: Model, enc: Encoded, m: int, b: int, h: Optional[int] = None, init=None,
           max_iters: Optional[int] = None, recompute: bool = False, evaluator=None,
           stop: str = "block") -> Result:
    """Hybrid GS-Jacobi decoding (Algorithm 3).

    GS-Jacobi blocks up to the horizon h; a converged block that holds [EOS]
    ends decoding at its first [EOS].  Without [EOS] before h, decoding goes on
    autoregressively from position h until [EOS] or m.
    """
    return solve_by_blocks(model, enc, m, "hybrid", b, h, init=init, max_iters=max_iters, recompute=recompute,
                           evaluator=evaluator, stop=stop)


def decode(model: Model, enc: Encoded, m: int, mode: str, block: int = 1, **kw) -> Result:
    """Dispatch by mode name: ar, jacobi, gs_jacobi, hybrid."""
    if mode == "ar":
        return greedy(model, enc, m, **kw)
    if mode == "jacobi":
        return jacobi(model, enc, m, **kw)
    if mode == "gs_jacobi":
        return gs_jacobi(model, enc, m, block, **kw)
    if mode == "hybrid":
        return hybrid(model, enc, m, block, **kw)
    raise ValueError(mode)
