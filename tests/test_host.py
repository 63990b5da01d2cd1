"""Host-side logic (no GPU): the seeded workload generators, batching, the
bench script's one-GPU guard and its check that the committed traffic figure
belongs to the current kernel sources."""
import hashlib
import json
import os
import shutil
import subprocess
import sys

import numpy as np
import pytest

from paper_2305_10427_amd import configs as C, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("name", sorted(C.WORKLOADS))
def test_workload_sentences_follow_their_recipe(name):
    wl = C.WORKLOADS[name]
    sents = synth.make_sentences(wl, seed=1)
    expect = wl.n_sentences + (1 if wl.extra_full_len else 0)
    assert len(sents) == expect
    kind = wl.src_len[0]
    for ids, m in sents:
        n = len(ids)
        assert ids.dtype == np.int32
        assert np.all(ids >= C.FIRST_WORD_ID) and np.all(ids < wl.model.vocab)   # no special ids in sources
        if kind == "fixed":
            assert n == wl.src_len[1]
        elif kind == "uniform":
            assert wl.src_len[1] <= n <= wl.src_len[2]
        else:
            assert wl.src_len[3] <= n <= wl.src_len[4]
        assert m == min(n + wl.tgt_extra, wl.tgt_cap) or (wl.extra_full_len and m == wl.tgt_cap)
    # seeded: the same draw twice, a different one for another seed
    again = synth.make_sentences(wl, seed=1)
    assert all(np.array_equal(a[0], b[0]) and a[1] == b[1] for a, b in zip(sents, again))
    other = synth.make_sentences(wl, seed=2)
    assert any(not np.array_equal(a[0], b[0]) for a, b in zip(sents, other))


def test_lognormal_lengths_have_the_stated_median():
    wl = C.WORKLOADS["mt_base_b64"]
    n = np.array([len(i) for i, _ in synth.make_sentences(wl, seed=1)])
    assert 20 <= np.median(n) <= 30            # median 25, 256 draws


def test_batches_pad_sources_and_keep_lengths():
    wl = C.WORKLOADS["mt_base_b64"]
    sents = synth.make_sentences(wl, seed=1)
    batches = synth.make_batches(sents, 64)
    assert [b.src.shape[0] for b in batches] == [64] * 4
    k = 0
    for b in batches:
        assert b.src.shape[1] == b.src_len.max()
        for r in range(b.src.shape[0]):
            ids, m = sents[k]
            k += 1
            assert b.src_len[r] == len(ids) and b.tgt_m[r] == m
            np.testing.assert_array_equal(b.src[r, :len(ids)], ids)
            assert np.all(b.src[r, len(ids):] == C.PAD_ID)


def test_weights_are_seeded_and_bf16_values_are_representable():
    cfg = C.TINY.with_dtype(C.BF16)
    a = synth.make_weights(cfg, seed=0)
    b = synth.make_weights(cfg, seed=0)
    for name in a.values:
        np.testing.assert_array_equal(a.values[name], b.values[name])
        bits = a.values[name].view(np.uint32)
        assert np.all((bits & 0xFFFF) == 0), name        # float32 values that are exact bfloat16
        np.testing.assert_array_equal(a.bf16_bits[name], (bits >> 16).astype(np.uint16))


def test_bench_refuses_more_than_one_gpu():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout.strip() == ""


@pytest.mark.parametrize("name", ["vocab_argmax_large", "gemm_products_large", "vocab_argmax_mt_base",
                                  "gemm_products_mt_base"])
def test_bench_traffic_figure_is_tied_to_the_kernel_sources(tmp_path, monkeypatch, name):
    import bench
    rec = json.load(open(os.path.join(ROOT, "profiles", name + ".json")))
    assert abs(rec["traffic_bytes_per_launch"] - rec["fetch_bytes_per_launch"] - rec["write_bytes_per_launch"]) <= 1
    csrc = tmp_path / "paper_2305_10427_amd" / "csrc"
    csrc.mkdir(parents=True)
    (tmp_path / "profiles").mkdir()
    for f in rec["kernel_sources"]:
        shutil.copy(os.path.join(ROOT, "paper_2305_10427_amd", "csrc", f), csrc / f)
    src = b"".join((csrc / f).read_bytes() for f in rec["kernel_sources"])
    good = dict(rec, kernel_source_sha256=hashlib.sha256(src).hexdigest())
    (tmp_path / "profiles" / (name + ".json")).write_text(json.dumps(good))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic(name) == int(rec["traffic_bytes_per_launch"])
    # any change to a kernel source voids the figure
    with open(csrc / rec["kernel_sources"][0], "ab") as f:
        f.write(b"\n")
    assert bench.measured_traffic(name) is None
