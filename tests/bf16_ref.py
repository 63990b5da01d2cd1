"""A bfloat16-storage encoder-decoder written with torch.nn.functional (CPU, float64).

Used only to pin where the oracle rounds to bfloat16 (its storage contract):
values are stored as bfloat16 (round to nearest, ties to even) at

  * the token + position embedding,
  * every K and V entry of self- and cross-attention,
  * every attention output (before its output projection),
  * the FFN hidden values after the activation,
  * the residual stream after every sublayer,
  * every LayerNorm output that feeds a matrix product (post-LN: the
    normalised residual itself; pre-LN: the sublayer input, the encoder
    memory and the final decoder state),

and everything else (queries, scores, softmax, products, logits) stays float64.
The rounding is done here on the float64 bit pattern with integer arithmetic
(drop 45 of the 52 mantissa bits, round half to even), not with the oracle's
frexp/ldexp routine, and the layers are torch's own functional ops: linear,
layer_norm, scaled_dot_product_attention (causal for the decoder's
self-attention over the whole target at once, no KV cache), relu / erf GELU.
"""
import math

import numpy as np
import torch
import torch.nn.functional as F

_DROP = 45                       # float64 mantissa bits that bfloat16 does not keep (52 - 7)
_HALF = 1 << (_DROP - 1)
_MASK = ~((1 << _DROP) - 1)


def bf16(x: torch.Tensor) -> torch.Tensor:
    """Round float64 values to the nearest bfloat16 (ties to even), kept in float64."""
    assert x.dtype == torch.float64
    a = x.abs()
    # only normal bfloat16 magnitudes (and zero) occur in these models
    assert bool(torch.all((a == 0) | ((a >= 2.0 ** -126) & (a < 3.3e38)))), "value outside the normal bf16 range"
    bits = x.contiguous().view(torch.int64)
    lsb = (bits >> _DROP) & 1
    rounded = (bits + (_HALF - 1) + lsb) & _MASK
    return rounded.view(torch.float64)


def _pe(T, d):
    pos = torch.arange(T, dtype=torch.float64)[:, None]
    inv = torch.pow(torch.tensor(10000.0, dtype=torch.float64),
                    -torch.arange(0, d, 2, dtype=torch.float64) / d)[None, :]
    pe = torch.zeros(T, d, dtype=torch.float64)
    pe[:, 0::2] = torch.sin(pos * inv)
    pe[:, 1::2] = torch.cos(pos * inv)
    return pe


class Bf16Seq2Seq:
    def __init__(self, cfg, weights):
        self.cfg = cfg
        self.W = {k: torch.tensor(np.asarray(v, np.float64)) for k, v in weights.items()}

    def _ln(self, x, p):
        return F.layer_norm(x, (self.cfg.d_model,), self.W[p + ".g"], self.W[p + ".b"], self.cfg.ln_eps)

    def _heads(self, t):
        L = t.shape[0]
        H = self.cfg.n_heads
        return t.reshape(L, H, -1).transpose(0, 1)

    def _attend(self, q, k, v, causal):
        o = F.scaled_dot_product_attention(self._heads(q), self._heads(k), self._heads(v), is_causal=causal)
        return o.transpose(0, 1).reshape(q.shape[0], -1)

    def _act(self, x):
        return F.gelu(x) if self.cfg.act_gelu else F.relu(x)

    def _block(self, x, p, ln_name, sub):
        """One sublayer with its residual: pre-LN x + sub(LN(x)), post-LN LN(x + sub(x))."""
        if self.cfg.pre_ln:
            return bf16(x + sub(bf16(self._ln(x, p + ln_name))))
        return bf16(self._ln(x + sub(x), p + ln_name))

    def _self_attn(self, p, causal):
        d = self.cfg.d_model

        def sub(u):
            qkv = F.linear(u, self.W[p + "sa.w_qkv"], self.W[p + "sa.b_qkv"])
            q, k, v = qkv[:, :d], bf16(qkv[:, d:2 * d]), bf16(qkv[:, 2 * d:])
            a = bf16(self._attend(q, k, v, causal))
            return F.linear(a, self.W[p + "sa.w_o"], self.W[p + "sa.b_o"])
        return sub

    def _ffn(self, p):
        def sub(u):
            h = bf16(self._act(F.linear(u, self.W[p + "ff.w1"], self.W[p + "ff.b1"])))
            return F.linear(h, self.W[p + "ff.w2"], self.W[p + "ff.b2"])
        return sub

    def logits(self, src, tgt_in):
        """src [n] token ids, tgt_in [T] decoder inputs (BOS first) -> logits [T, V]."""
        cfg, W = self.cfg, self.W
        d = cfg.d_model
        src = torch.as_tensor(np.asarray(src, np.int64))
        tgt = torch.as_tensor(np.asarray(tgt_in, np.int64))
        x = bf16(W["emb"][src] * math.sqrt(d) + _pe(len(src), d))
        for l in range(cfg.n_enc):
            p = f"enc.{l}."
            x = self._block(x, p, "ln1", self._self_attn(p, causal=False))
            x = self._block(x, p, "ln2", self._ffn(p))
        mem = bf16(self._ln(x, "enc.ln")) if cfg.pre_ln else x
        dec_scale = math.sqrt(d) if cfg.dec_emb_scale is None else cfg.dec_emb_scale
        y = bf16(W["emb"][tgt] * dec_scale + _pe(len(tgt), d))
        for l in range(cfg.n_dec):
            p = f"dec.{l}."
            y = self._block(y, p, "ln1", self._self_attn(p, causal=True))

            def cross(u, p=p):
                q = F.linear(u, W[p + "ca.w_q"], W[p + "ca.b_q"])
                kv = F.linear(mem, W[p + "ca.w_kv"], W[p + "ca.b_kv"])
                a = bf16(self._attend(q, bf16(kv[:, :d]), bf16(kv[:, d:]), causal=False))
                return F.linear(a, W[p + "ca.w_o"], W[p + "ca.b_o"])
            y = self._block(y, p, "ln2", cross)
            y = self._block(y, p, "ln3", self._ffn(p))
        if cfg.pre_ln:
            y = bf16(self._ln(y, "dec.ln"))
        return (cfg.logit_scale * (y @ W["emb"].T) + W["out_bias"]).numpy()
