"""bench.py's host-side accounting, checked without a GPU: the algorithmic bytes each bench
line divides by, against the oracle's own record sizes and cache layout (an independent
implementation of the record format), the per-token bytes of the attention step, and the two
CPU baselines on tiny samples."""
import importlib.util
import os

import numpy as np
import pytest

import oracle
import workloads

ROOT = os.path.join(os.path.dirname(__file__), "..")


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test",
                                                  os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _oracle_codec(w):
    kinds = []
    for t in w.table:
        kinds += [oracle.Kind(t.n_k, t.norm_mode_k, t.norm_bits_k),
                  oracle.Kind(t.n_v, t.norm_mode_v, t.norm_bits_v)]
    return oracle.Codec(w.L, w.H, w.d, kinds, workloads.sign_table(w.sign_seed, w.L, w.d))


@pytest.mark.parametrize("key", ["C2", "C3", "C4", "C5"])
def test_algorithmic_bytes_match_the_oracle_records(key):
    b, w = _bench(), workloads.get(key)
    c = _oracle_codec(w)
    rec = sum(sum(c.record_bytes(l, k)) for l in range(w.L) for k in range(2))
    total, _ = c.layout(w.B, w.T)
    ab = b.algorithmic_bytes(w)
    elem = 2 if w.dtype == "bf16" else 4
    assert ab["kv"] == 2 * w.L * w.B * w.H * w.T * w.d * elem
    assert ab["compressed"] == rec * w.B * w.H * w.T == total
    assert ab["per_launch"] == ab["kv"] + ab["compressed"]
    assert ab["vectors"] == 2 * w.L * w.B * w.H * w.T
    if key == "C2":
        # Mistral-7B shape, n = 64, K 8-bit linear, V 4-bit log: 256 B in, 120 + 88 B out
        assert ab["per_launch"] == 754_974_720


@pytest.mark.parametrize("key", ["C4", "C5"])
def test_attention_step_bytes(key):
    b, w = _bench(), workloads.get(key)
    c = _oracle_codec(w)
    rec_tok, kv_tok, qo = b.longctx_bytes(w)
    assert rec_tok == sum(sum(c.record_bytes(l, k)) for l in range(w.L)
                          for k in range(2)) * w.B * w.H
    assert kv_tok == 2 * w.L * w.B * w.H * w.d * 2
    assert qo == 2 * w.L * w.B * w.H * b.ATTN_GROUP * w.d * 2
    if key == "C5":
        assert rec_tok == 868_352


def test_cpu_baselines_run_on_small_samples():
    b = _bench()
    w = workloads.get("C4")
    att = b.cpu_baseline_attention(w, budget_s=0.2, tokens=64)
    assert att["value"] > 0 and att["value_1core"] > 0 and att["kind"] == "oracle"
    assert att["cores"] == (os.cpu_count() or 1)
    tiny = workloads.get("C1")
    codec = b.cpu_baseline(tiny, budget_s=0.2)
    assert codec["value"] > 0 and codec["value_1core"] > 0 and codec["kind"] == "oracle"


def test_gpu_count_above_one_is_refused():
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


@pytest.mark.parametrize("extra", [["--workload", "C5"], ["--attention"], ["--encode-mfma"]])
def test_pool_takes_the_codec_step_only(extra):
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--pool", *extra],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "--pool" in r.stderr


def test_codec_counter_summaries_exist_for_their_workloads():
    """Each workload with a codec counter summary has it committed and taken on that workload
    (its bench line quotes it while the summary's kernel-source hash matches the tree)."""
    import json
    b = _bench()
    for key in b.CODEC_COUNTER_FILES:
        path = b.codec_counters(key)
        d = json.load(open(path))
        assert d["workload"] == workloads.get(key).name
        assert len(d["kernel_source_hash"]) == 16, key
        assert set(d["kernels"]) == {"tvq_encode", "tvq_decode"}
    assert b.codec_counters("C5") is None
    d = json.load(open(b.LONGCTX_DECODE_COUNTERS))
    assert d["workload"] == workloads.get("C5").name
    assert 1.0 <= d["hbm_bytes_per_step"] / d["algorithmic_bytes_per_step"] < 1.1
