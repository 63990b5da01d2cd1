"""Model shapes and workload recipes for the synthetic decoding benchmarks.

The paper evaluates a Transformer-base model (d=512, 6+6 layers, Opus-MT, 58K
vocabulary) and a Transformer-big model (d=1024, 12+12 layers, MBart50, 250K
vocabulary) at batch size 1 with a KV cache (Section 4.1, "Model
Configuration" and "Evaluation"; vocabulary sizes in Section 4.3 "Speedup
Analysis").  Trained weights and the WMT/IWSLT/IITB/FLORES test sets are not
available, so every workload here is a seeded random-weight model of the same
shape and a seeded synthetic source set with a stated length distribution.

This module holds only shapes and recipes: no arithmetic of the method.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

# Special token ids.  The paper initialises drafts with [PAD] (Section 3.3,
# "Initialization") and uses [BOS]/[EOS] (Section 3.2); their numeric values
# are not given, so the first four ids are reserved: PAD 0, BOS 1, EOS 2, UNK 3.
PAD_ID = 0
BOS_ID = 1
EOS_ID = 2
UNK_ID = 3
FIRST_WORD_ID = 4

F32 = "f32"
BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    """Shape of an encoder-decoder Transformer p_theta(y | x)."""

    name: str
    n_enc: int
    n_dec: int
    d_model: int
    n_heads: int
    d_ff: int
    vocab: int
    pre_ln: bool          # False: post-LN (Transformer-base); True: pre-LN + final LN (MBart-like)
    act_gelu: bool        # False: ReLU FFN; True: exact (erf) GELU FFN
    dtype: str            # storage type of weights/activations: "f32" or "bf16"
    ln_eps: float = 1e-5
    logit_scale: float = 3.0   # tied output projection: logits = s * h . E^T + b
    # Scale of the decoder's token embedding (None: sqrt(d_model), the usual
    # choice).  0 gives a decoder whose prediction at a position ignores the
    # draft tokens (a fixture with closed-form iteration counts).
    dec_emb_scale: Optional[float] = None

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    def with_dtype(self, dtype: str) -> "ModelConfig":
        return dataclasses.replace(self, dtype=dtype, name=f"{self.name.split('@')[0]}@{dtype}")

    def param_count(self) -> int:
        return sum(int(_numel(s)) for _, s in param_shapes(self))


@dataclasses.dataclass(frozen=True)
class Workload:
    """A synthetic source set plus the decode modes run on it."""

    name: str
    model: ModelConfig
    batch: int
    n_sentences: int
    src_len: Tuple            # ("uniform", lo, hi) | ("fixed", n) | ("lognormal", median, sigma, lo, hi)
    tgt_extra: int            # m = min(n + tgt_extra, tgt_cap)
    tgt_cap: int
    modes: Tuple              # ((mode, block), ...)
    extra_full_len: bool = False   # add one sentence with m == tgt_cap


def _numel(shape):
    n = 1
    for s in shape:
        n *= s
    return n


def param_shapes(cfg: ModelConfig):
    """Canonical (name, shape) list of all parameters, in generation order.

    Linear weights are stored [out, in] (row-major), the layout in which one
    output feature's weights are contiguous.  The token embedding E [V, d] is
    shared by the encoder input, the decoder input and the output projection.
    """
    d, f, V = cfg.d_model, cfg.d_ff, cfg.vocab
    out = [("emb", (V, d)), ("out_bias", (V,))]
    for l in range(cfg.n_enc):
        p = f"enc.{l}."
        out += [(p + "sa.w_qkv", (3 * d, d)), (p + "sa.b_qkv", (3 * d,)),
                (p + "sa.w_o", (d, d)), (p + "sa.b_o", (d,)),
                (p + "ln1.g", (d,)), (p + "ln1.b", (d,)),
                (p + "ff.w1", (f, d)), (p + "ff.b1", (f,)),
                (p + "ff.w2", (d, f)), (p + "ff.b2", (d,)),
                (p + "ln2.g", (d,)), (p + "ln2.b", (d,))]
    if cfg.pre_ln:
        out += [("enc.ln.g", (d,)), ("enc.ln.b", (d,))]
    for l in range(cfg.n_dec):
        p = f"dec.{l}."
        out += [(p + "sa.w_qkv", (3 * d, d)), (p + "sa.b_qkv", (3 * d,)),
                (p + "sa.w_o", (d, d)), (p + "sa.b_o", (d,)),
                (p + "ln1.g", (d,)), (p + "ln1.b", (d,)),
                (p + "ca.w_q", (d, d)), (p + "ca.b_q", (d,)),
                (p + "ca.w_kv", (2 * d, d)), (p + "ca.b_kv", (2 * d,)),
                (p + "ca.w_o", (d, d)), (p + "ca.b_o", (d,)),
                (p + "ln2.g", (d,)), (p + "ln2.b", (d,)),
                (p + "ff.w1", (f, d)), (p + "ff.b1", (f,)),
                (p + "ff.w2", (d, f)), (p + "ff.b2", (d,)),
                (p + "ln3.g", (d,)), (p + "ln3.b", (d,))]
    if cfg.pre_ln:
        out += [("dec.ln.g", (d,)), ("dec.ln.b", (d,))]
    return out


# --- model shapes ---------------------------------------------------------

TINY = ModelConfig("tiny", n_enc=2, n_dec=2, d_model=64, n_heads=4, d_ff=256, vocab=1000,
                   pre_ln=False, act_gelu=False, dtype=F32)
MT_BASE = ModelConfig("mt_base", n_enc=6, n_dec=6, d_model=512, n_heads=8, d_ff=2048,
                      vocab=58101, pre_ln=False, act_gelu=False, dtype=F32)
LARGE = ModelConfig("large", n_enc=12, n_dec=12, d_model=1024, n_heads=16, d_ff=4096,
                    vocab=250027, pre_ln=True, act_gelu=True, dtype=BF16)

# --- workloads ------------------------------------------------------------

WORKLOADS = {
    # Tiny 2+2 model, batch 1, n = 16, m = 16: every mode at once.
    "tiny": Workload("tiny", TINY, batch=1, n_sentences=100, src_len=("fixed", 16),
                     tgt_extra=0, tgt_cap=16,
                     modes=(("ar", 1), ("jacobi", 16), ("gs_jacobi", 4), ("hybrid", 4))),
    # Transformer-base shape, batch 1, n ~ U[10, 60], m = min(n + 10, 128).
    "mt_base_f32": Workload("mt_base_f32", MT_BASE, batch=1, n_sentences=200,
                            src_len=("uniform", 10, 60), tgt_extra=10, tgt_cap=128,
                            modes=(("ar", 1), ("gs_jacobi", 5), ("hybrid", 5))),
    "mt_base_bf16": Workload("mt_base_bf16", MT_BASE.with_dtype(BF16), batch=1, n_sentences=200,
                             src_len=("uniform", 10, 60), tgt_extra=10, tgt_cap=128,
                             modes=(("ar", 1), ("gs_jacobi", 5), ("hybrid", 5))),
    # Transformer-base shape, batch 64, log-normal lengths (median 25), m = n + 10.
    "mt_base_b64": Workload("mt_base_b64", MT_BASE.with_dtype(BF16), batch=64, n_sentences=256,
                            src_len=("lognormal", 25.0, 0.6, 1, 128), tgt_extra=10, tgt_cap=138,
                            modes=(("ar", 1), ("hybrid", 2), ("hybrid", 3), ("hybrid", 5),
                                   ("hybrid", 8))),
    # Transformer-big / multilingual shape, batch 1, n ~ U[20, 120], m = min(n + 10, 256).
    "large": Workload("large", LARGE, batch=1, n_sentences=50, src_len=("uniform", 20, 120),
                      tgt_extra=10, tgt_cap=256,
                      modes=(("ar", 1), ("jacobi", 16), ("gs_jacobi", 16)), extra_full_len=True),
    # Same big model, batch 32, block-size sweep.
    "large_b32": Workload("large_b32", LARGE, batch=32, n_sentences=64, src_len=("uniform", 20, 120),
                          tgt_extra=10, tgt_cap=256,
                          modes=(("ar", 1),) + tuple((m, b) for m in ("gs_jacobi", "hybrid")
                                                     for b in (1, 2, 4, 8, 16, 32))),
}

MODES = {"ar": 0, "jacobi": 1, "gs_jacobi": 2, "hybrid": 3}
