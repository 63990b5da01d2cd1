"""pd_decode_traced_static (the traced decode for callers that cannot
allocate: the log-sum-exp scratch in the library's static device array)
against the existing pd_ctx_set_trace + pd_decode with a caller scratch,
through the C ABI: ids, lengths, k, flags and every trace record equal
(records bitwise), on two calls in a row, the second with a smaller input,
and a decode too large for the static array is refused before anything runs."""
import dataclasses

import numpy as np
import pytest

from paper_2305_10427_amd import configs as C, pdec, synth
from tests.parity import gpu_decode_batch, max_rows

pytestmark = pytest.mark.gpu

SMALL_PRE_BF16 = dataclasses.replace(C.TINY, name="small_pre", pre_ln=True, act_gelu=True, dtype=C.BF16)


def say(*a):
    print(*a, flush=True)


def sources(vocab, lens, seed):
    g = np.random.default_rng(seed)
    return [g.integers(4, vocab, n).astype(np.int32) for n in lens]


def reference(ctx, srcs, ms, mode, b, cap):
    ctx.set_trace(cap, max_rows(mode, b, ms))
    try:
        got = gpu_decode_batch(ctx, srcs, ms, mode, b)
        rec, n = ctx.trace()
    finally:
        ctx.set_trace(0, 0)
    return got, rec, n


def static_call(ctx, srcs, ms, mode, b, cap):
    import torch
    n_max = max(len(s) for s in srcs)
    src = np.zeros((len(srcs), n_max), np.int32)
    for r, s in enumerate(srcs):
        src[r, :len(s)] = s
    ctx.encode(torch.from_numpy(src).cuda(), [len(s) for s in srcs])
    ids, ln, k, fl, rec, n = ctx.decode_traced_static(mode, ms, cap, block=b)
    ids, ln, k, fl = (t.cpu().numpy() for t in (ids, ln, k, fl))
    return [(ids[r, :ln[r]], int(k[r]), int(fl[r])) for r in range(len(srcs))], rec, n


@pytest.mark.parametrize("cfg", [C.TINY, SMALL_PRE_BF16], ids=["tiny_f32", "small_pre_bf16"])
def test_static_trace_scratch_matches_caller_scratch(cfg):
    w = synth.make_weights(cfg, seed=21, bias_std=0.3, ln_std=0.2)
    ctx = pdec.Context(pdec.Model(cfg, w), 4, 24, 32)
    calls = [(sources(cfg.vocab, [20, 16, 24, 9], 40), [30, 16, 24, 9], "jacobi", 0),   # 120 rows
             (sources(cfg.vocab, [11], 41), [7], "gs_jacobi", 3)]                        # then 3 rows
    for srcs, ms, mode, b in calls:
        cap = len(ms) * max(ms) * max_rows(mode, b, ms)
        say(f"case static-scratch cfg={cfg.name} mode={mode} b={b} B={len(ms)} m={ms}")
        got, rec, n = static_call(ctx, srcs, ms, mode, b, cap)
        ref, rec_ref, n_ref = reference(ctx, srcs, ms, mode, b, cap)
        for (ids, k, fl), r in zip(got, ref):
            np.testing.assert_array_equal(ids, r.ids)
            assert (k, fl) == (r.k, r.flags)
        assert n == n_ref == len(rec) == len(rec_ref) > 0
        for f in ("iteration", "sentence", "position", "token"):
            np.testing.assert_array_equal(rec[f], rec_ref[f])
        np.testing.assert_array_equal(rec["top1"].view(np.uint32), rec_ref["top1"].view(np.uint32))
        np.testing.assert_array_equal(rec["lse"].view(np.uint32), rec_ref["lse"].view(np.uint32))


def test_static_trace_scratch_refuses_decodes_beyond_its_size():
    """A 200,000-word vocabulary needs 3,125 partials (25 KB) per row, so the
    8 MiB array holds 335 rows: Jacobi over 4 x 100 positions is refused, the
    context then decodes a smaller batch through the same entry point."""
    cfg = dataclasses.replace(C.TINY, name="wide_vocab", vocab=200_000)
    w = synth.make_weights(cfg, seed=22)
    ctx = pdec.Context(pdec.Model(cfg, w), 4, 16, 100)
    per_row = -(-cfg.vocab // 64) * 8
    assert 4 * 100 * per_row > pdec.TRACE_STATIC_BYTES >= 2 * 100 * per_row
    srcs = sources(cfg.vocab, [16, 16, 16, 16], 42)
    with pytest.raises(pdec.PdError) as ei:
        static_call(ctx, srcs, [100] * 4, "jacobi", 0, 4 * 100 * 100)
    assert ei.value.status == 3 and "static" in str(ei.value)
    got, rec, n = static_call(ctx, srcs[:2], [100, 60], "jacobi", 0, 2 * 100 * 100)
    ref, rec_ref, n_ref = reference(ctx, srcs[:2], [100, 60], "jacobi", 0, 2 * 100 * 100)
    for (ids, k, fl), r in zip(got, ref):
        np.testing.assert_array_equal(ids, r.ids)
        assert (k, fl) == (r.k, r.flags)
    assert n == n_ref
    np.testing.assert_array_equal(rec["top1"].view(np.uint32), rec_ref["top1"].view(np.uint32))
