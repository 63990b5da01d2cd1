"""Mutation check of the oracle's pins (CPU only).

Each case plants one plausible mistake in the oracle (a dropped term, a wrong
index or sign, a rounding point more or less, a missing cap) for the duration
of the case only, and asserts that at least one of the pins in
tests/test_oracle_model.py / tests/test_oracle_decode.py then fails.  A pin
set that let such a mistake through would not pin the oracle."""
import inspect
import sys
import textwrap

import numpy as np
import pytest

import oracle
from oracle import model as om
from tests import test_oracle_decode as TD
from tests import test_oracle_model as TM

OD = sys.modules["oracle.decode"]


def mutate(monkeypatch, owner, name, old, new):
    """Replace `owner.name` by a copy of its source with `old` replaced by `new`."""
    fn = getattr(owner, name)
    src = textwrap.dedent(inspect.getsource(fn))
    assert src.count(old) == 1, f"mutation site not unique in {name}: {old!r}"
    ns = {}
    exec(compile(src.replace(old, new), f"<mutant of {name}>", "exec"), sys.modules[fn.__module__].__dict__, ns)
    monkeypatch.setattr(owner, name, ns[name])
    if getattr(oracle, name, None) is fn:          # the package re-exports it under the same name
        monkeypatch.setattr(oracle, name, ns[name])


def model_pins():
    TM.test_model_matches_torch_transformer_layers(TM.SMALL_POST)
    TM.test_model_matches_torch_transformer_layers(TM.SMALL_PRE)
    TM.test_causality_later_inputs_do_not_change_earlier_rows()


def bf16_pins():
    for cfg in (TM.SMALL_POST.with_dtype("bf16"), TM.SMALL_PRE.with_dtype("bf16")):
        TM.test_bf16_storage_contract_matches_functional_reference(cfg)


def decode_pins():
    for case in TD.CASES:
        TD.test_proposition1_all_modes_equal_greedy(*case)
    TD.test_brute_force_unique_fixed_point_and_trajectories(0)
    TD.test_special_cases_between_modes()


def prefix_pins():
    for case in TD.CASES:
        TD.test_prefix_stop_equals_greedy_and_commits_every_iteration(*case)
    TD.test_prefix_stop_worked_example()
    for cfg, seed in [(TD.TINY, 8), (TD.CHAIN, 9)]:
        TD.test_prefix_stop_hybrid_eos(cfg, seed, 4)


MODEL_MUTANTS = {
    "dropped linear bias": (om.Model, "_lin", "x @ self.w[name_w].T + self.w[name_b]", "x @ self.w[name_w].T"),
    "dropped LayerNorm offset": (om, "layer_norm", "np.sqrt(var + eps) * g + b", "np.sqrt(var + eps) * g"),
    "biased variance replaced by the unbiased one": (om, "layer_norm", ").mean(axis=-1, keepdims=True)\n    return",
                                                     ").sum(axis=-1, keepdims=True) / (x.shape[-1] - 1)\n    return"),
    "causal mask off by one": (om.Model, "decode_rows", "key_limit=pos + 1", "key_limit=pos + 2"),
    "K and V swapped in the self-attention cache": (om.Model, "decode_rows",
                                                    "cache.k[l][p0:p0 + L] = self._r(qkv[:, d:2 * d])",
                                                    "cache.k[l][p0:p0 + L] = self._r(qkv[:, 2 * d:])"),
    "cross-attention reads the self-attention query": (om.Model, "decode_rows",
                                                       "a = self._r(attention(q, enc.cross_k[l]",
                                                       "a = self._r(attention(qkv[:, :d], enc.cross_k[l]"),
    "attention scale 1/d instead of 1/sqrt(d_h)": (om, "attention", "/ math.sqrt(dh)", "/ d"),
    "sin and cos swapped": (om, "sinusoid", "pe[:, 0::2] = np.sin(angle)\n    pe[:, 1::2] = np.cos(angle)",
                            "pe[:, 0::2] = np.cos(angle)\n    pe[:, 1::2] = np.sin(angle)"),
    "tied output projection without its bias": (om.Model, "logits", ' + self.w["out_bias"]', ""),
}

BF16_MUTANTS = {
    "attention output not rounded": (om.Model, "decode_rows", "a = self._r(attention(qkv[:, :d]",
                                     "a = (attention(qkv[:, :d]"),
    "query rounded": (om.Model, "decode_rows", "attention(qkv[:, :d], cache", "attention(self._r(qkv[:, :d]), cache"),
    "FFN hidden not rounded": (om.Model, "decode_rows", "hdn = self._r(self._act(", "hdn = (self._act("),
    "encoder memory not rounded (pre-LN)": (om.Model, "encode", 'mem = self._r(self._ln(x, "enc.ln"))',
                                            'mem = (self._ln(x, "enc.ln"))'),
    "cross-attention V not rounded": (om.Model, "encode", "cv.append(self._r(kv[:, d:]))", "cv.append((kv[:, d:]))"),
}

DECODE_MUTANTS = {
    "inputs not shifted left": (OD.Solver, "inputs", "int(y[p - 1])", "int(y[p])"),
    "no per-block cap of L iterations": (OD, "solve_by_blocks", "or j == L:", ":"),
    "stopping test on the block's first token only": (OD, "solve_by_blocks", "np.array_equal(y[i:i + L], before)",
                                                      "y[i] == before[0]"),
    "next block starts one position late": (OD, "solve_by_blocks", "        i += L\n", "        i += L + 1\n"),
    "greedy predicts position t from the window of t - 1": (OD, "greedy", "y[t] = s.block(y, t, 1)[0]",
                                                            "y[t] = s.block(y, max(t - 1, 0), 1)[0]"),
}


PREFIX_MUTANTS = {
    "one position committed past the proven prefix": (OD, "_solve_prefix", "c = L if t == L else t + 1",
                                                      "c = L if t == L else t + 2"),
    "only the proven positions, never the whole unchanged block": (OD, "_solve_prefix",
                                                                   "c = L if t == L else t + 1", "c = min(t + 1, L - 1) if L > 1 else 1"),
    "[EOS] looked for in the whole block": (OD, "_solve_prefix", "hit = np.nonzero(y[i:i + c] == EOS)[0]",
                                            "hit = np.nonzero(y[i:i + L] == EOS)[0]"),
    "unchanged positions counted from the block's end": (OD, "_solve_prefix", "y[i + t] == before[t]",
                                                         "y[i + L - 1 - t] == before[L - 1 - t]"),
}


@pytest.mark.parametrize("name", list(MODEL_MUTANTS))
def test_model_pins_catch(monkeypatch, name):
    mutate(monkeypatch, *MODEL_MUTANTS[name])
    with pytest.raises(AssertionError):
        model_pins()


@pytest.mark.parametrize("name", list(BF16_MUTANTS))
def test_bf16_contract_pin_catches(monkeypatch, name):
    mutate(monkeypatch, *BF16_MUTANTS[name])
    with pytest.raises(AssertionError):
        bf16_pins()


@pytest.mark.parametrize("name", list(DECODE_MUTANTS))
def test_decode_pins_catch(monkeypatch, name):
    mutate(monkeypatch, *DECODE_MUTANTS[name])
    with pytest.raises((AssertionError, IndexError, ValueError)):
        decode_pins()


@pytest.mark.parametrize("name", list(PREFIX_MUTANTS))
def test_prefix_pins_catch(monkeypatch, name):
    mutate(monkeypatch, *PREFIX_MUTANTS[name])
    with pytest.raises((AssertionError, IndexError, ValueError)):
        prefix_pins()


def test_eos_stop_at_block_index_instead_of_position_is_caught(monkeypatch):
    """CheckEOS read as an index inside the block instead of an absolute position."""
    mutate(monkeypatch, OD, "solve_by_blocks", "y = y[: i + int(hit[0]) + 1].copy()", "y = y[: int(hit[0]) + 1].copy()")
    with pytest.raises(AssertionError):
        for cfg, seed in [(TD.TINY, 8), (TD.CHAIN, 9)]:
            TD.test_hybrid_eos_truncation_matches_greedy(cfg, seed, 4)


def test_argmax_tie_to_the_highest_index_is_caught(monkeypatch):
    mutate(monkeypatch, om, "argmax_rows", "t = int(np.argmax(row))", "t = int(len(row) - 1 - np.argmax(row[::-1]))")
    with pytest.raises(AssertionError):
        TM.test_argmax_rows_ties_take_lowest_index_and_top2()


def test_unmutated_pins_pass():
    """The same pin runs pass on the oracle as it is (the cases above fail
    because of their mutation, not because of the harness)."""
    model_pins()
    bf16_pins()
    decode_pins()
    prefix_pins()
    np.testing.assert_equal(oracle.cut_at_eos(np.array([5, 2, 7, 2])), [5, 2])
