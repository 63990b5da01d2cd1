"""Seeded synthetic weights and source sets.

Both the HIP path and the CPU oracle consume what this module draws; it holds
no arithmetic of the decoding method or of the Transformer itself, only random
draws and their storage type.

Weights (a reading of the initialisation stated for the workloads): every
linear weight W[out, in] is drawn from N(0, 1/in) (standard deviation
1/sqrt(fan_in)); the shared embedding E[V, d] from N(0, 1/d); biases are 0 and
LayerNorm gains/offsets are 1/0, unless a test asks for non-zero values so that
a dropped bias or LayerNorm-affine term is visible.  Each tensor is drawn from
its own PCG64 stream keyed by (seed, tensor index), so a tensor's values do not
depend on which options the others were drawn with.

bf16 models store weights rounded to bfloat16 (round-to-nearest-even); they
are returned as float32 arrays that hold exactly the bf16 values, plus the raw
16-bit patterns for upload.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

from . import configs as C


def _stream(seed: int, index: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, index])))


def _to_bf16_bits(a32: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns of float32 values (round-to-nearest-even), via torch."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a32, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class Weights:
    cfg: C.ModelConfig
    values: Dict[str, np.ndarray]          # float32 arrays (bf16-exact for bf16 models)
    bf16_bits: Optional[Dict[str, np.ndarray]] = None

    def names(self) -> List[str]:
        return [n for n, _ in C.param_shapes(self.cfg)]


def make_weights(cfg: C.ModelConfig, seed: int = 0, bias_std: float = 0.0,
                 ln_std: float = 0.0, eos_bias: float = 0.0) -> Weights:
    """Draw all parameters of `cfg` in canonical order.

    bias_std / ln_std > 0 draw non-zero biases and LayerNorm affines (tests);
    eos_bias adds a constant to the output bias of the EOS token (fixtures
    that make EOS appear at chosen places).
    """
    values: Dict[str, np.ndarray] = {}
    for idx, (name, shape) in enumerate(C.param_shapes(cfg)):
        g = _stream(seed, idx)
        leaf = name.rsplit(".", 1)[-1]
        if name == "emb":
            a = g.standard_normal(shape, dtype=np.float32) * np.float32(1.0 / np.sqrt(shape[1]))
        elif len(shape) == 2:
            a = g.standard_normal(shape, dtype=np.float32) * np.float32(1.0 / np.sqrt(shape[1]))
        elif name.endswith(".g"):
            a = np.ones(shape, np.float32)
            if ln_std > 0:
                a += g.standard_normal(shape, dtype=np.float32) * np.float32(ln_std)
        elif name.endswith(".b") and leaf == "b":
            a = np.zeros(shape, np.float32)
            if ln_std > 0:
                a += g.standard_normal(shape, dtype=np.float32) * np.float32(ln_std)
        else:  # linear biases and the output bias
            a = np.zeros(shape, np.float32)
            if bias_std > 0:
                a += g.standard_normal(shape, dtype=np.float32) * np.float32(bias_std)
            if name == "out_bias" and eos_bias != 0.0:
                a[C.EOS_ID] += np.float32(eos_bias)
        values[name] = np.ascontiguousarray(a, dtype=np.float32)
    bits = None
    if cfg.dtype == C.BF16:
        bits = {}
        for name, a in values.items():
            b = _to_bf16_bits(a)
            bits[name] = b
            values[name] = _bf16_bits_to_f32(b)
    return Weights(cfg, values, bits)


@dataclasses.dataclass
class Batch:
    src: np.ndarray        # int32 [B, n_max], PAD after each sentence's length
    src_len: np.ndarray    # int32 [B]
    tgt_m: np.ndarray      # int32 [B]  number of target positions to solve


def _draw_len(g: np.random.Generator, spec) -> int:
    kind = spec[0]
    if kind == "fixed":
        return int(spec[1])
    if kind == "uniform":
        return int(g.integers(spec[1], spec[2] + 1))
    if kind == "lognormal":
        _, median, sigma, lo, hi = spec
        return int(np.clip(np.round(np.exp(g.normal(np.log(median), sigma))), lo, hi))
    raise ValueError(kind)


def make_sentences(wl: C.Workload, seed: int = 1, count: Optional[int] = None):
    """List of (src_ids int32[n], m) drawn for workload `wl`."""
    g = np.random.Generator(np.random.PCG64(seed))
    count = wl.n_sentences if count is None else count
    out = []
    for _ in range(count):
        n = _draw_len(g, wl.src_len)
        ids = g.integers(C.FIRST_WORD_ID, wl.model.vocab, size=n).astype(np.int32)
        out.append((ids, min(n + wl.tgt_extra, wl.tgt_cap)))
    if wl.extra_full_len and (count is None or count == wl.n_sentences):
        n = wl.src_len[2] if wl.src_len[0] == "uniform" else _draw_len(g, wl.src_len)
        ids = g.integers(C.FIRST_WORD_ID, wl.model.vocab, size=n).astype(np.int32)
        out.append((ids, wl.tgt_cap))
    return out


def make_batches(sentences, batch: int) -> List[Batch]:
    """Group sentences into batches, padding sources to the batch maximum."""
    out = []
    for s0 in range(0, len(sentences), batch):
        chunk = sentences[s0:s0 + batch]
        n_max = max(len(ids) for ids, _ in chunk)
        src = np.full((len(chunk), n_max), C.PAD_ID, np.int32)
        for r, (ids, _) in enumerate(chunk):
            src[r, :len(ids)] = ids
        out.append(Batch(src, np.array([len(i) for i, _ in chunk], np.int32),
                         np.array([m for _, m in chunk], np.int32)))
    return out


def random_draft(m: int, vocab: int, seed: int) -> np.ndarray:
    """A random initial draft (Proposition 1 holds for any initialisation)."""
    g = np.random.Generator(np.random.PCG64(seed))
    return g.integers(0, vocab, size=m).astype(np.int32)
