"""Python binding of libpdec.so (include/pdec.h): argument marshalling only.

Device memory and streams come from PyTorch (ROCm); every step of encoding
and decoding runs in the library's HIP kernels.  There is no fallback: if the
library is missing or fails, calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

from . import configs as C

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpdec.so")

PD_AR, PD_JACOBI, PD_GS_JACOBI, PD_HYBRID = 0, 1, 2, 3
MODE_IDS = {"ar": PD_AR, "jacobi": PD_JACOBI, "gs_jacobi": PD_GS_JACOBI, "hybrid": PD_HYBRID}
PD_STOP_PREFIX = 0x100                  # or-ed into the mode: the prefix stopping condition
STOP_FLAGS = {"block": 0, "prefix": PD_STOP_PREFIX}


def mode_word(mode, stop="block") -> int:
    """The mode argument of pd_decode: the mode id, or-ed with the stopping-condition flag."""
    return (MODE_IDS[mode] if isinstance(mode, str) else int(mode)) | STOP_FLAGS[stop]
FLAG_CONVERGED, FLAG_EOS, FLAG_MAX_ITERS, FLAG_NONFINITE = 1, 2, 4, 8
STATUS = {0: "PD_OK", 1: "PD_E_ARG", 2: "PD_E_SHAPE", 3: "PD_E_WORKSPACE", 4: "PD_E_DEVICE",
          5: "PD_E_UNSUPPORTED", 6: "PD_E_STATE"}


class PdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class pd_config(ctypes.Structure):
    _fields_ = [("n_enc", ctypes.c_int32), ("n_dec", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("d_ff", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("pre_ln", ctypes.c_int32), ("act_gelu", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("pad_id", ctypes.c_int32), ("bos_id", ctypes.c_int32), ("eos_id", ctypes.c_int32),
                ("ln_eps", ctypes.c_float), ("logit_scale", ctypes.c_float),
                ("enc_emb_scale", ctypes.c_float), ("dec_emb_scale", ctypes.c_float)]


EXPORTS = ("pd_weight_count", "pd_weight_shape", "pd_model_create", "pd_model_destroy",
           "pd_ctx_workspace_bytes", "pd_ctx_create", "pd_ctx_destroy", "pd_encode", "pd_decode", "pd_decode_init",
           "pd_debug_logits", "pd_ctx_set_timing", "pd_ctx_vocab_timing", "pd_ctx_rows_processed",
           "pd_trace_scratch_bytes", "pd_ctx_set_trace", "pd_ctx_trace_count", "pd_ctx_product_timing",
           "pd_ctx_iteration_kernels", "pd_decode_traced_static", "pd_last_error")
TRACE_STATIC_BYTES = 8 << 20      # PD_TRACE_STATIC_BYTES

_lib = None


def load_library(path: str = LIB_PATH):
    """Load libpdec.so and declare its signatures (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise OSError(f"{path} is not built: run `python -m paper_2305_10427_amd.build`")
    L = ctypes.CDLL(path)
    P, I32, I64, SZ, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p
    L.pd_weight_count.argtypes = [P(pd_config)]
    L.pd_weight_count.restype = I32
    L.pd_weight_shape.argtypes = [P(pd_config), I32, P(I64), P(I64)]
    L.pd_weight_shape.restype = I32
    L.pd_model_create.argtypes = [P(pd_config), P(VP), I32, P(VP)]
    L.pd_model_create.restype = I32
    L.pd_model_destroy.argtypes = [VP]
    L.pd_model_destroy.restype = None
    L.pd_ctx_workspace_bytes.argtypes = [VP, I32, I32, I32, P(SZ)]
    L.pd_ctx_workspace_bytes.restype = I32
    L.pd_ctx_create.argtypes = [VP, I32, I32, I32, VP, SZ, P(VP)]
    L.pd_ctx_create.restype = I32
    L.pd_ctx_destroy.argtypes = [VP]
    L.pd_ctx_destroy.restype = None
    L.pd_encode.argtypes = [VP, VP, P(I32), I32, I32, VP]
    L.pd_encode.restype = I32
    L.pd_decode.argtypes = [VP, I32, I32, I32, I32, P(I32), VP, I32, VP, VP, VP, VP]
    L.pd_decode.restype = I32
    L.pd_decode_init.argtypes = [VP, I32, I32, I32, I32, P(I32), VP, I32, VP, I32, VP, VP, VP, VP]
    L.pd_decode_init.restype = I32
    L.pd_debug_logits.argtypes = [VP, VP, I32, VP, VP]
    L.pd_debug_logits.restype = I32
    L.pd_ctx_set_timing.argtypes = [VP, I32]
    L.pd_ctx_set_timing.restype = I32
    L.pd_ctx_vocab_timing.argtypes = [VP, P(I64), P(ctypes.c_double)]
    L.pd_ctx_vocab_timing.restype = I32
    L.pd_ctx_rows_processed.argtypes = [VP, P(I64)]
    L.pd_ctx_rows_processed.restype = I32
    L.pd_trace_scratch_bytes.argtypes = [VP, I32, P(SZ)]
    L.pd_trace_scratch_bytes.restype = I32
    L.pd_ctx_set_trace.argtypes = [VP, VP, I64, VP, SZ]
    L.pd_ctx_set_trace.restype = I32
    L.pd_ctx_trace_count.argtypes = [VP, P(I64)]
    L.pd_ctx_trace_count.restype = I32
    L.pd_ctx_product_timing.argtypes = [VP, P(I64), P(ctypes.c_double), P(ctypes.c_double)]
    L.pd_ctx_product_timing.restype = I32
    L.pd_ctx_iteration_kernels.argtypes = [VP, P(I64)]
    L.pd_ctx_iteration_kernels.restype = I32
    L.pd_decode_traced_static.argtypes = [VP, I32, I32, I32, I32, P(I32), VP, I32, VP, VP, VP, VP, I64, VP]
    L.pd_decode_traced_static.restype = I32
    L.pd_last_error.argtypes = []
    L.pd_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise PdError(status, load_library().pd_last_error().decode())


def make_config(cfg: C.ModelConfig) -> pd_config:
    return pd_config(cfg.n_enc, cfg.n_dec, cfg.d_model, cfg.n_heads, cfg.d_ff, cfg.vocab,
                     int(cfg.pre_ln), int(cfg.act_gelu), 1 if cfg.dtype == C.BF16 else 0,
                     C.PAD_ID, C.BOS_ID, C.EOS_ID, cfg.ln_eps, cfg.logit_scale, -1.0,
                     -1.0 if cfg.dec_emb_scale is None else float(cfg.dec_emb_scale))


def _stream_handle(stream) -> int:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream)


def _host_i32(a) -> ctypes.Array:
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return (ctypes.c_int32 * len(a))(*a.tolist())


class Model:
    """Weights uploaded to the GPU plus the library's pd_model handle."""

    def __init__(self, cfg: C.ModelConfig, weights, device: str = "cuda"):
        import torch
        L = load_library()
        self.cfg = cfg
        self.c_cfg = make_config(cfg)
        n = L.pd_weight_count(ctypes.byref(self.c_cfg))
        names = [nm for nm, _ in C.param_shapes(cfg)]
        if n != len(names):
            raise PdError(1, f"library expects {n} weights, configuration has {len(names)}")
        self.tensors = []
        for i, nm in enumerate(names):
            rows, cols = ctypes.c_int64(), ctypes.c_int64()
            _check(L.pd_weight_shape(ctypes.byref(self.c_cfg), i, ctypes.byref(rows), ctypes.byref(cols)))
            want = (rows.value, cols.value) if cols.value > 1 else (rows.value,)
            if tuple(weights.values[nm].shape) != want:
                raise PdError(2, f"weight {nm}: shape {weights.values[nm].shape} != {want}")
            if cfg.dtype == C.BF16:
                host = torch.from_numpy(weights.bf16_bits[nm].view(np.int16).copy()).view(torch.bfloat16)
            else:
                host = torch.from_numpy(np.ascontiguousarray(weights.values[nm], np.float32))
            self.tensors.append(host.to(device).contiguous())
        ptrs = (ctypes.c_void_p * n)(*[t.data_ptr() for t in self.tensors])
        h = ctypes.c_void_p()
        _check(L.pd_model_create(ctypes.byref(self.c_cfg), ptrs, n, ctypes.byref(h)))
        self.handle = h

    def weight_bytes(self) -> int:
        return sum(t.numel() * t.element_size() for t in self.tensors)

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.pd_model_destroy(self.handle)
            self.handle = None


class Context:
    """A decoding context: caller-owned workspace + the library's pd_ctx."""

    def __init__(self, model: Model, max_batch: int, max_src: int, max_tgt: int, device: str = "cuda"):
        import torch
        L = load_library()
        self.model = model
        self.max_batch, self.max_src, self.max_tgt = max_batch, max_src, max_tgt
        nbytes = ctypes.c_size_t()
        _check(L.pd_ctx_workspace_bytes(model.handle, max_batch, max_src, max_tgt, ctypes.byref(nbytes)))
        self.workspace = torch.empty(nbytes.value + 256, dtype=torch.uint8, device=device)
        base = self.workspace.data_ptr()
        self.ws_ptr = (base + 255) // 256 * 256
        h = ctypes.c_void_p()
        _check(L.pd_ctx_create(model.handle, max_batch, max_src, max_tgt, ctypes.c_void_p(self.ws_ptr),
                               nbytes.value, ctypes.byref(h)))
        self.handle = h
        self.B = 0
        self.device = device

    def encode(self, src, src_len: Sequence[int], stream=None):
        """src: int32 device tensor [B, n_max]; src_len: host ints."""
        import torch
        src = src.to(device=self.device, dtype=torch.int32).contiguous()
        B, n_max = src.shape
        self._src = src                      # keep alive until the kernels have read it
        _check(load_library().pd_encode(self.handle, ctypes.c_void_p(src.data_ptr()), _host_i32(src_len),
                                        B, n_max, ctypes.c_void_p(_stream_handle(stream))))
        self.B = B

    def decode(self, mode, tgt_m: Sequence[int], block: int = 1, max_iters: int = 0, horizon: int = 0,
               stream=None, out=None, init=None, stop: str = "block"):
        """Returns (ids [B, m_max], lengths [B], k [B], flags [B]) as device int32 tensors.
        init: optional int32 tensor [B, >= max(tgt_m)], the initial draft (default all [PAD]).
        stop: "block" (Eq. (3)) or "prefix" (PD_STOP_PREFIX)."""
        import torch
        mode_id = mode_word(mode, stop)
        tgt_m = [int(x) for x in tgt_m]
        if len(tgt_m) != self.B:
            raise PdError(1, f"tgt_m has {len(tgt_m)} entries, the encoded batch has {self.B}")
        m_max = max(tgt_m)
        B = len(tgt_m)
        if out is None:   # at least one column, so that the library itself reports a bad tgt_m
            out = (torch.empty((B, max(m_max, 1)), dtype=torch.int32, device=self.device),
                   torch.empty(B, dtype=torch.int32, device=self.device),
                   torch.empty(B, dtype=torch.int32, device=self.device),
                   torch.empty(B, dtype=torch.int32, device=self.device))
        ids, ln, k, fl = out
        if init is None:
            _check(load_library().pd_decode(self.handle, mode_id, int(block), int(horizon), int(max_iters),
                                            _host_i32(tgt_m), ctypes.c_void_p(ids.data_ptr()), ids.shape[1],
                                            ctypes.c_void_p(ln.data_ptr()), ctypes.c_void_p(k.data_ptr()),
                                            ctypes.c_void_p(fl.data_ptr()), ctypes.c_void_p(_stream_handle(stream))))
        else:
            init = init.to(device=self.device, dtype=torch.int32).contiguous()
            if init.dim() != 2 or init.shape[0] != B:
                raise PdError(1, f"init must be [B, >= m_max], got {tuple(init.shape)}")
            self._init = init                # keep alive until the kernels have read it
            _check(load_library().pd_decode_init(self.handle, mode_id, int(block), int(horizon), int(max_iters),
                                                 _host_i32(tgt_m), ctypes.c_void_p(init.data_ptr()), init.shape[1],
                                                 ctypes.c_void_p(ids.data_ptr()), ids.shape[1],
                                                 ctypes.c_void_p(ln.data_ptr()), ctypes.c_void_p(k.data_ptr()),
                                                 ctypes.c_void_p(fl.data_ptr()),
                                                 ctypes.c_void_p(_stream_handle(stream))))
        return ids, ln, k, fl

    def decode_traced_static(self, mode, tgt_m: Sequence[int], capacity: int, block: int = 1, max_iters: int = 0,
                             horizon: int = 0, stream=None, stop: str = "block"):
        """pd_decode_traced_static: decode with the trace on, the trace scratch
        in the library's static array.  Returns (ids, lengths, k, flags,
        records, count); records is a numpy structured array (TRACE_DTYPE) of
        the first min(count, capacity) records."""
        import torch
        mode_id = mode_word(mode, stop)
        tgt_m = [int(x) for x in tgt_m]
        if len(tgt_m) != self.B:
            raise PdError(1, f"tgt_m has {len(tgt_m)} entries, the encoded batch has {self.B}")
        B = len(tgt_m)
        ids = torch.empty((B, max(max(tgt_m), 1)), dtype=torch.int32, device=self.device)
        ln, k, fl = (torch.empty(B, dtype=torch.int32, device=self.device) for _ in range(3))
        rec = torch.empty(max(int(capacity), 1) * 6, dtype=torch.int32, device=self.device)
        _check(load_library().pd_decode_traced_static(
            self.handle, mode_id, int(block), int(horizon), int(max_iters), _host_i32(tgt_m),
            ctypes.c_void_p(ids.data_ptr()), ids.shape[1], ctypes.c_void_p(ln.data_ptr()),
            ctypes.c_void_p(k.data_ptr()), ctypes.c_void_p(fl.data_ptr()), ctypes.c_void_p(rec.data_ptr()),
            int(capacity), ctypes.c_void_p(_stream_handle(stream))))
        torch.cuda.current_stream().synchronize() if stream is None else stream.synchronize()
        n = ctypes.c_int64()
        _check(load_library().pd_ctx_trace_count(self.handle, ctypes.byref(n)))
        kept = min(n.value, int(capacity))
        raw = rec[: kept * 6].cpu().numpy()
        return ids, ln, k, fl, raw.view(np.dtype(self.TRACE_DTYPE)), n.value

    def debug_logits(self, tgt_in, stream=None):
        """Teacher-forced logits [B, T, V] for decoder inputs tgt_in [B, T] (BOS first)."""
        import torch
        tgt_in = tgt_in.to(device=self.device, dtype=torch.int32).contiguous()
        B, T = tgt_in.shape
        logits = torch.empty((B, T, self.model.cfg.vocab), dtype=torch.float32, device=self.device)
        _check(load_library().pd_debug_logits(self.handle, ctypes.c_void_p(tgt_in.data_ptr()), T,
                                              ctypes.c_void_p(logits.data_ptr()),
                                              ctypes.c_void_p(_stream_handle(stream))))
        return logits

    def set_timing(self, enable: bool):
        _check(load_library().pd_ctx_set_timing(self.handle, int(enable)))

    def vocab_timing(self):
        """(launches, total_ms) of the fused vocabulary kernel since set_timing(True)."""
        n, ms = ctypes.c_int64(), ctypes.c_double()
        _check(load_library().pd_ctx_vocab_timing(self.handle, ctypes.byref(n), ctypes.byref(ms)))
        return n.value, ms.value

    def product_timing(self):
        """(launches, total_ms, bytes) of the decoder's timed product launches since set_timing(True)."""
        n, ms, b = ctypes.c_int64(), ctypes.c_double(), ctypes.c_double()
        _check(load_library().pd_ctx_product_timing(self.handle, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(b)))
        return n.value, ms.value, b.value

    def iteration_kernels(self) -> int:
        """Kernels in the iteration graph replayed last."""
        n = ctypes.c_int64()
        _check(load_library().pd_ctx_iteration_kernels(self.handle, ctypes.byref(n)))
        return n.value

    def rows_processed(self) -> int:
        """Rows evaluated by all iterations since set_timing (synchronous)."""
        n = ctypes.c_int64()
        _check(load_library().pd_ctx_rows_processed(self.handle, ctypes.byref(n)))
        return n.value

    TRACE_DTYPE = [("iteration", "<i4"), ("sentence", "<i4"), ("position", "<i4"), ("token", "<i4"),
                   ("top1", "<f4"), ("lse", "<f4")]

    def set_trace(self, capacity: int, max_rows: int):
        """Turn the decoding trace on (capacity records, iterations of up to
        max_rows rows; both buffers allocated here) or off (capacity 0)."""
        import torch
        L = load_library()
        if capacity <= 0:
            _check(L.pd_ctx_set_trace(self.handle, None, 0, None, 0))
            self._trace = None
            return
        nbytes = ctypes.c_size_t()
        _check(L.pd_trace_scratch_bytes(self.model.handle, int(max_rows), ctypes.byref(nbytes)))
        rec = torch.empty(capacity * 6, dtype=torch.int32, device=self.device)
        scratch = torch.empty(nbytes.value // 8, dtype=torch.float64, device=self.device)
        _check(L.pd_ctx_set_trace(self.handle, ctypes.c_void_p(rec.data_ptr()), int(capacity),
                                  ctypes.c_void_p(scratch.data_ptr()), nbytes.value))
        self._trace = (rec, scratch)

    def trace(self):
        """Records appended since set_trace, as a numpy structured array
        (fields of TRACE_DTYPE), and the full count (may exceed capacity)."""
        if getattr(self, "_trace", None) is None:
            raise PdError(6, "tracing is off: call set_trace first")
        n = ctypes.c_int64()
        _check(load_library().pd_ctx_trace_count(self.handle, ctypes.byref(n)))
        rec = self._trace[0]
        kept = min(n.value, rec.numel() // 6)
        raw = rec[: kept * 6].cpu().numpy()
        return raw.view(np.dtype(self.TRACE_DTYPE)), n.value

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.pd_ctx_destroy(self.handle)
            self.handle = None
