"""An encoder-decoder built from torch.nn Transformer layers (CPU, float64).

Used only to pin the numpy oracle: torch's TransformerEncoderLayer /
TransformerDecoderLayer implement post-LN (norm_first=False) and pre-LN
(norm_first=True) blocks, multi-head attention with packed in-projections,
key-padding and causal masks, ReLU / erf-GELU FFNs and LayerNorm, independently
of the oracle's code.  Weights are copied in from the canonical dict.
"""
import math

import numpy as np
import torch
import torch.nn as nn


def _t(a):
    return torch.tensor(np.asarray(a, np.float64))


def _pe(T, d):
    pos = torch.arange(T, dtype=torch.float64)[:, None]
    inv = torch.pow(torch.tensor(10000.0, dtype=torch.float64),
                    -torch.arange(0, d, 2, dtype=torch.float64) / d)[None, :]
    pe = torch.zeros(T, d, dtype=torch.float64)
    pe[:, 0::2] = torch.sin(pos * inv)
    pe[:, 1::2] = torch.cos(pos * inv)
    return pe


class TorchSeq2Seq:
    def __init__(self, cfg, weights):
        self.cfg = cfg
        d, H = cfg.d_model, cfg.n_heads
        act = "gelu" if cfg.act_gelu else "relu"
        kw = dict(dim_feedforward=cfg.d_ff, dropout=0.0, activation=act, layer_norm_eps=cfg.ln_eps,
                  batch_first=True, norm_first=cfg.pre_ln, dtype=torch.float64)
        W = {k: _t(v) for k, v in weights.items()}
        self.W = W
        self.enc = []
        with torch.no_grad():
            for l in range(cfg.n_enc):
                p = f"enc.{l}."
                m = nn.TransformerEncoderLayer(d, H, **kw)
                m.self_attn.in_proj_weight.copy_(W[p + "sa.w_qkv"])
                m.self_attn.in_proj_bias.copy_(W[p + "sa.b_qkv"])
                m.self_attn.out_proj.weight.copy_(W[p + "sa.w_o"])
                m.self_attn.out_proj.bias.copy_(W[p + "sa.b_o"])
                m.linear1.weight.copy_(W[p + "ff.w1"]); m.linear1.bias.copy_(W[p + "ff.b1"])
                m.linear2.weight.copy_(W[p + "ff.w2"]); m.linear2.bias.copy_(W[p + "ff.b2"])
                m.norm1.weight.copy_(W[p + "ln1.g"]); m.norm1.bias.copy_(W[p + "ln1.b"])
                m.norm2.weight.copy_(W[p + "ln2.g"]); m.norm2.bias.copy_(W[p + "ln2.b"])
                self.enc.append(m)
            self.dec = []
            for l in range(cfg.n_dec):
                p = f"dec.{l}."
                m = nn.TransformerDecoderLayer(d, H, **kw)
                m.self_attn.in_proj_weight.copy_(W[p + "sa.w_qkv"])
                m.self_attn.in_proj_bias.copy_(W[p + "sa.b_qkv"])
                m.self_attn.out_proj.weight.copy_(W[p + "sa.w_o"])
                m.self_attn.out_proj.bias.copy_(W[p + "sa.b_o"])
                m.multihead_attn.in_proj_weight.copy_(torch.cat([W[p + "ca.w_q"], W[p + "ca.w_kv"]]))
                m.multihead_attn.in_proj_bias.copy_(torch.cat([W[p + "ca.b_q"], W[p + "ca.b_kv"]]))
                m.multihead_attn.out_proj.weight.copy_(W[p + "ca.w_o"])
                m.multihead_attn.out_proj.bias.copy_(W[p + "ca.b_o"])
                m.linear1.weight.copy_(W[p + "ff.w1"]); m.linear1.bias.copy_(W[p + "ff.b1"])
                m.linear2.weight.copy_(W[p + "ff.w2"]); m.linear2.bias.copy_(W[p + "ff.b2"])
                m.norm1.weight.copy_(W[p + "ln1.g"]); m.norm1.bias.copy_(W[p + "ln1.b"])
                m.norm2.weight.copy_(W[p + "ln2.g"]); m.norm2.bias.copy_(W[p + "ln2.b"])
                m.norm3.weight.copy_(W[p + "ln3.g"]); m.norm3.bias.copy_(W[p + "ln3.b"])
                self.dec.append(m)
        for m in self.enc + self.dec:
            m.eval()

    def _final_ln(self, x, name):
        return nn.functional.layer_norm(x, (self.cfg.d_model,), self.W[name + ".g"],
                                        self.W[name + ".b"], self.cfg.ln_eps)

    def logits(self, src_batch, src_len, tgt_in):
        """src_batch [B, n] padded, src_len [B], tgt_in [B, T] -> logits [B, T, V]."""
        cfg = self.cfg
        d = cfg.d_model
        src = torch.tensor(np.asarray(src_batch, np.int64))
        tgt = torch.tensor(np.asarray(tgt_in, np.int64))
        B, n = src.shape
        T = tgt.shape[1]
        pad = torch.arange(n)[None, :] >= torch.tensor(np.asarray(src_len))[:, None]
        E = self.W["emb"]
        dec_scale = math.sqrt(d) if cfg.dec_emb_scale is None else cfg.dec_emb_scale
        x = E[src] * math.sqrt(d) + _pe(n, d)[None]
        for m in self.enc:
            x = m(x, src_key_padding_mask=pad)
        if cfg.pre_ln:
            x = self._final_ln(x, "enc.ln")
        mem = x
        causal = torch.triu(torch.full((T, T), float("-inf"), dtype=torch.float64), diagonal=1)
        y = E[tgt] * dec_scale + _pe(T, d)[None]
        for m in self.dec:
            y = m(y, mem, tgt_mask=causal, memory_key_padding_mask=pad)
        if cfg.pre_ln:
            y = self._final_ln(y, "dec.ln")
        return (cfg.logit_scale * (y @ E.T) + self.W["out_bias"]).detach().numpy()
