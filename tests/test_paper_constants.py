"""Eq. 1 against the per-token KV sizes printed in Table 2."""

import json
import os

import pytest

from oracle import kvcache as ok

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table2_per_token_kv.json")


def _models():
    with open(GOLDEN) as f:
        return json.load(f)["models"]


@pytest.mark.parametrize("m", _models(), ids=lambda m: m["name"])
def test_eq1_times_layers_matches_table2(m):
    per_token = ok.per_token_bytes(m["layers"], m["kv_heads"], m["head_dim"], 2)
    assert per_token / 2 ** 20 == pytest.approx(m["mib_per_token"], abs=5e-4)


def test_eq1_block_bytes_of_the_benchmark_shapes():
    # B = 16, 8 KV heads, D = 128, bf16: one block of one layer is 64 KiB
    assert ok.m_block_bytes(16, 8, 128, 2) == 65536
    assert ok.m_block_bytes(16, 8, 64, 2) == 32768
