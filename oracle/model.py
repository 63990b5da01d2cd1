"""CPU oracle, part 1: the encoder-decoder Transformer p_theta(y | x).

TEST INFRASTRUCTURE ONLY.  Only tests, the smoke entry point and the CPU
baseline leg of the benchmark may import this module; the HIP decoding library
never calls it.  It shares no code with the HIP path.

Plain numpy, float64 arithmetic, one sentence at a time, no padding, no fusion
and no reordering beyond what a matrix product in numpy does.

What it computes (the model is the paper's black box p_theta, Section 3.1,
Eq. (1)-(2); its shape follows Section 4.1 "Model Configuration"):

* token embedding E[y] * scale + sinusoidal position encoding (interleaved
  sin/cos, position 0 = the first input position);
* encoder: bidirectional multi-head self-attention + ReLU/GELU FFN;
* decoder: causal self-attention over a KV cache, cross-attention to the
  encoder output, FFN;
* post-LN  (x <- LN(x + Sub(x)))      for the Transformer-base shape,
  pre-LN   (x <- x + Sub(LN(x)), final LN) for the MBart-like shape;
* tied output projection: logits = s * h . E^T + out_bias.

bf16 models follow a storage contract: values are rounded to bfloat16
(round-to-nearest-even) at the embedding output, every K/V entry, every
attention output, the FFN hidden after the activation, the residual stream
after each sublayer and every LayerNorm output that feeds a matrix product;
all other arithmetic is float64 here.  float32 models round nowhere.

Model(..., dtype=np.float32) runs the same code in float32 arithmetic; it is
used only to time the CPU baseline, never for parity.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (ties to even), returned as float64.

    bfloat16 keeps 8 significant bits and float32's exponent range; below
    2**-126 it keeps a fixed quantum of 2**-133 (subnormals).
    """
    x = np.asarray(x, dtype=np.float64)
    mant, expo = np.frexp(x)                       # x = mant * 2**expo, 0.5 <= |mant| < 1
    normal = np.ldexp(np.round(mant * 256.0), expo - 8)   # np.round: half to even
    sub = np.round(np.ldexp(x, 133)) * 2.0 ** -133
    out = np.where(np.abs(x) < 2.0 ** -126, sub, normal)
    big = np.abs(out) > 3.3895313892515355e38      # largest finite bfloat16
    return np.where(big, np.copysign(np.inf, x), out)


def sinusoid(positions: np.ndarray, d: int) -> np.ndarray:
    """Sinusoidal position encoding: columns 2i, 2i+1 = sin, cos of pos / 10000**(2i/d)."""
    pos = np.asarray(positions, dtype=np.float64)[:, None]
    i = np.arange(d // 2, dtype=np.float64)[None, :]
    angle = pos / np.power(10000.0, 2.0 * i / d)
    pe = np.zeros((pos.shape[0], d), np.float64)
    pe[:, 0::2] = np.sin(angle)
    pe[:, 1::2] = np.cos(angle)
    return pe


def layer_norm(x, g, b, eps):
    """(x - mean) / sqrt(biased variance + eps) * g + b, per row."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def gelu(x):
    """Exact GELU: x * Phi(x) with the Gaussian CDF written through erf."""
    from scipy.special import erf
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def softmax_rows(s):
    s = s - s.max(axis=-1, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=-1, keepdims=True)


def attention(q, k, v, n_heads, key_limit=None):
    """Multi-head scaled dot-product attention.

    q [Lq, d], k/v [Lk, d].  key_limit[r] (optional) = number of keys row r may
    see (keys 0 .. key_limit[r]-1); None lets every row see every key.
    """
    Lq, d = q.shape
    dh = d // n_heads
    out = np.zeros((Lq, d), q.dtype)
    for h in range(n_heads):
        sl = slice(h * dh, (h + 1) * dh)
        scores = (q[:, sl] @ k[:, sl].T) / math.sqrt(dh)          # [Lq, Lk]
        if key_limit is not None:
            cols = np.arange(k.shape[0])[None, :]
            scores = np.where(cols < np.asarray(key_limit)[:, None], scores, -np.inf)
        out[:, sl] = softmax_rows(scores) @ v[:, sl]
    return out


@dataclasses.dataclass
class Encoded:
    memory: np.ndarray              # [n, d]
    cross_k: List[np.ndarray]       # per decoder layer [n, d]
    cross_v: List[np.ndarray]


@dataclasses.dataclass
class Cache:
    """Decoder self-attention K/V per layer for input positions 0..T-1."""
    k: List[np.ndarray]
    v: List[np.ndarray]


@dataclasses.dataclass
class ArgmaxRecord:
    """One row's argmax over the vocabulary."""
    position: int          # input position (predicts y at the same 0-based index)
    token: int             # argmax, lowest index on exact ties
    top1: float
    top2: float            # largest logit among the other indices
    linf: float            # max |logit|
    lse: float = 0.0       # log sum_v exp(logit_v): p(token) = exp(top1 - lse)


class Model:
    """p_theta with weights given as a {name: array} dict (canonical names)."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray], dtype=np.float64):
        self.cfg = cfg
        self.d = cfg.d_model
        self.H = cfg.n_heads
        self.bf16 = cfg.dtype == "bf16"
        self.dt = np.dtype(dtype)
        self.w = {k: np.asarray(v, dtype=self.dt) for k, v in weights.items()}
        self.enc_scale = math.sqrt(self.d)
        des = getattr(cfg, "dec_emb_scale", None)
        self.dec_scale = math.sqrt(self.d) if des is None else float(des)

    # -- helpers -------------------------------------------------------------
    def _r(self, x):
        return round_bf16(x).astype(self.dt, copy=False) if self.bf16 else x

    def _lin(self, x, name_w, name_b):
        return x @ self.w[name_w].T + self.w[name_b]

    def _ln(self, x, prefix):
        return layer_norm(x, self.w[prefix + ".g"], self.w[prefix + ".b"], self.cfg.ln_eps)

    def _act(self, x):
        return gelu(x) if self.cfg.act_gelu else np.maximum(x, 0.0)

    def embed(self, tokens, positions, scale):
        pe = sinusoid(positions, self.d).astype(self.dt, copy=False)
        return self._r(self.w["emb"][np.asarray(tokens)] * self.dt.type(scale) + pe)

    # -- encoder ---------------------------------------------------------------
    def encode(self, src) -> Encoded:
        cfg, d = self.cfg, self.d
        src = np.asarray(src)
        x = self.embed(src, np.arange(len(src)), self.enc_scale)
        for l in range(cfg.n_enc):
            p = f"enc.{l}."
            u = self._r(self._ln(x, p + "ln1")) if cfg.pre_ln else x
            qkv = self._lin(u, p + "sa.w_qkv", p + "sa.b_qkv")
            q, k, v = qkv[:, :d], self._r(qkv[:, d:2 * d]), self._r(qkv[:, 2 * d:])
            a = self._r(attention(q, k, v, self.H))
            y = self._lin(a, p + "sa.w_o", p + "sa.b_o")
            x = self._r(x + y) if cfg.pre_ln else self._r(self._ln(x + y, p + "ln1"))
            u = self._r(self._ln(x, p + "ln2")) if cfg.pre_ln else x
            hdn = self._r(self._act(self._lin(u, p + "ff.w1", p + "ff.b1")))
            y = self._lin(hdn, p + "ff.w2", p + "ff.b2")
            x = self._r(x + y) if cfg.pre_ln else self._r(self._ln(x + y, p + "ln2"))
        mem = self._r(self._ln(x, "enc.ln")) if cfg.pre_ln else x
        ck, cv = [], []
        for l in range(cfg.n_dec):
            kv = self._lin(mem, f"dec.{l}.ca.w_kv", f"dec.{l}.ca.b_kv")
            ck.append(self._r(kv[:, :d]))
            cv.append(self._r(kv[:, d:]))
        return Encoded(mem, ck, cv)

    # -- decoder ---------------------------------------------------------------
    def new_cache(self, T: int) -> Cache:
        return Cache([np.zeros((T, self.d), self.dt) for _ in range(self.cfg.n_dec)],
                     [np.zeros((T, self.d), self.dt) for _ in range(self.cfg.n_dec)])

    def decode_rows(self, enc: Encoded, cache: Cache, tokens, p0: int) -> np.ndarray:
        """Final hidden states of input positions p0 .. p0+L-1.

        tokens[r] is the decoder input at position p0 + r.  The cache must hold
        K/V of positions < p0; this call writes K/V of positions p0 .. p0+L-1
        and row r attends to positions 0 .. p0 + r (causal).
        """
        cfg, d = self.cfg, self.d
        L = len(tokens)
        pos = np.arange(p0, p0 + L)
        x = self.embed(tokens, pos, self.dec_scale)
        for l in range(cfg.n_dec):
            p = f"dec.{l}."
            u = self._r(self._ln(x, p + "ln1")) if cfg.pre_ln else x
            qkv = self._lin(u, p + "sa.w_qkv", p + "sa.b_qkv")
            cache.k[l][p0:p0 + L] = self._r(qkv[:, d:2 * d])
            cache.v[l][p0:p0 + L] = self._r(qkv[:, 2 * d:])
            a = self._r(attention(qkv[:, :d], cache.k[l][:p0 + L], cache.v[l][:p0 + L], self.H,
                                  key_limit=pos + 1))
            y = self._lin(a, p + "sa.w_o", p + "sa.b_o")
            x = self._r(x + y) if cfg.pre_ln else self._r(self._ln(x + y, p + "ln1"))
            u = self._r(self._ln(x, p + "ln2")) if cfg.pre_ln else x
            q = self._lin(u, p + "ca.w_q", p + "ca.b_q")
            a = self._r(attention(q, enc.cross_k[l], enc.cross_v[l], self.H))
            y = self._lin(a, p + "ca.w_o", p + "ca.b_o")
            x = self._r(x + y) if cfg.pre_ln else self._r(self._ln(x + y, p + "ln2"))
            u = self._r(self._ln(x, p + "ln3")) if cfg.pre_ln else x
            hdn = self._r(self._act(self._lin(u, p + "ff.w1", p + "ff.b1")))
            y = self._lin(hdn, p + "ff.w2", p + "ff.b2")
            x = self._r(x + y) if cfg.pre_ln else self._r(self._ln(x + y, p + "ln3"))
        return self._r(self._ln(x, "dec.ln")) if cfg.pre_ln else x

    def logits(self, h: np.ndarray) -> np.ndarray:
        """Tied output projection s * h . E^T + out_bias, one row per hidden state."""
        return self.dt.type(self.cfg.logit_scale) * (h @ self.w["emb"].T) + self.w["out_bias"]

    def teacher_forced_logits(self, enc: Encoded, tgt_in) -> np.ndarray:
        """Logits of every position for decoder inputs tgt_in (BOS first), recomputed from scratch."""
        cache = self.new_cache(len(tgt_in))
        return self.logits(self.decode_rows(enc, cache, tgt_in, 0))


def argmax_rows(logits: np.ndarray, p0: int) -> List[ArgmaxRecord]:
    """Per-row argmax with the lowest index winning exact ties, plus the top-2 margin."""
    if not np.all(np.isfinite(logits)):
        raise FloatingPointError("non-finite logits")
    out = []
    for r in range(logits.shape[0]):
        row = logits[r]
        t = int(np.argmax(row))              # first maximal index
        top1 = float(row[t])
        rest = np.delete(row, t)
        lse = top1 + float(np.log(np.sum(np.exp(row - top1))))    # log-sum-exp, shifted by the maximum
        out.append(ArgmaxRecord(p0 + r, t, top1, float(rest.max()), float(np.abs(row).max()), lse))
    return out
