"""The benchmark's algorithmic accounting, on the CPU: attention flops per
layer (4 D H_q per visible (query, key) pair) and fetch payload bytes, at
the benchmark shapes, against values computed by hand from the shapes."""

import importlib.util
import os

import pytest

from paper_2606_16135_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_module", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_attention_flops_at_benchmark_shapes(bench):
    # 8B shape: pairs = N P + N (N + 1) / 2 = 512 * 8192 + 512 * 513 / 2
    assert bench.attention_flops(W.config(2)) == 4 * 128 * 32 * (512 * 8192 + 512 * 513 // 2) == 70871154688
    # 14B shape: 40 query heads, P = 32768, N = 1024
    assert bench.attention_flops(W.config(4)) == 4 * 128 * 40 * (1024 * 32768 + 1024 * 1025 // 2)
    # tiny shape: 8 heads of 64 dims, P = 256, N = 64
    assert bench.attention_flops(W.config(1)) == 4 * 64 * 8 * (64 * 256 + 64 * 65 // 2) == 37814272


def test_fetch_payload(bench):
    # K and V of every prefix token: 2 * H_kv * D * 2 bytes per token
    assert bench.fetch_payload_bytes(W.config(2)) == 8192 * 2 * 8 * 128 * 2 == 32 << 20
    # with half of the full prefix blocks in the regular cache only the rest moves
    assert bench.fetch_payload_bytes(W.config(2, rc_fraction=0.5)) == 16 << 20
    wl = W.config(3)
    assert bench.fetch_payload_bytes(wl) == int(wl.prefix_len.sum()) * 4096


def test_traffic_counters_match_the_attention_code(bench):
    """Every benchmark workload has HBM byte counters, taken on the attention
    code as it stands (the hash ignores comments): the bench line's
    roofline.traffic is never stale or missing for them."""
    code = bench._src_sha16("attn_fwd.hip")
    for name in ("llama3-8b-P8192-N512", "llama3-8b-batch16-varlen", "qwen-14b-P32768-N1024",
                 "llama3-8b-P131072-N2048-hosttier"):
        nbytes, key = bench.PMC_TRAFFIC[name]
        assert key == code, f"{name}: counters taken on code {key}, the source is now {code}"
        assert nbytes > 0
