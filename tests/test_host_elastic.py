"""Host entry points for the capacity planner (Eq. 1-5), the elastic unit
(Eq. 6-9), Algorithm 1 and the O(1) pool resize, on the CPU, against the
oracle."""

import json
import os

import numpy as np
import pytest

from oracle import capacity as oc
from oracle import elastic as oe

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table2_per_token_kv.json")
FAKE_BASE = 0x10000   # never dereferenced: no call below touches the device


@pytest.fixture(scope="module")
def sc():
    from paper_2606_16135_amd import swiftcache
    swiftcache.load()
    return swiftcache


def test_capacity_worked_example(sc):
    L, mb_shape = 10, (10, 16, 8, 128, 2)
    mb = oc.m_block_bytes(16, 8, 128, 2)
    out, k = sc.sc_plan_capacity(sc.model_shape(*mb_shape), 100 * mb + mb - 1,
                                 [9 * mb * L + 5, 8 * mb * L])
    assert k == [9, 8]
    assert (out.k_master, out.sum_k_workers, out.n_lsc, out.n_rc) == (100, 17, 17, 8)
    assert out.max_context_tokens == 25 * 16 and out.conventional_blocks == 10
    assert out.m_block_bytes == mb


def test_capacity_matches_oracle_on_random_cases(sc):
    rng = np.random.default_rng(11)
    for _ in range(500):
        L, B, H, D, dt = (int(rng.integers(1, 80)), int(rng.choice([1, 8, 16, 32])), int(rng.integers(1, 33)),
                          int(rng.choice([64, 128])), int(rng.choice([1, 2, 4])))
        cm = int(rng.integers(0, 1 << 40))
        cw = [int(x) for x in rng.integers(0, 1 << 40, size=int(rng.integers(0, 5)))]
        out, k = sc.sc_plan_capacity(sc.model_shape(L, B, H, D, dt), cm, cw)
        ref = oc.plan(cm, cw, L, B, H, D, dt)
        assert k == ref["k_workers"]
        assert (out.m_block_bytes, out.k_master, out.n_lsc, out.n_rc, out.max_context_tokens,
                out.conventional_blocks) == (ref["m_block"], ref["k_master"], ref["n_lsc"], ref["n_rc"],
                                             ref["max_context_tokens"], ref["conventional_blocks"])


def test_elastic_unit_table2_and_random(sc):
    ms = {m["name"]: m for m in json.load(open(GOLDEN))["models"]}
    shape = lambda m: sc.model_shape(m["layers"], 16, m["kv_heads"], m["head_dim"], 2)
    assert sc.sc_elastic_unit(shape(ms["Qwen3-32B"]), shape(ms["Qwen3-8B"])) == (9, 16)
    assert sc.sc_elastic_unit(shape(ms["LWM"]), shape(ms["Qwen3-14B"])) == (5, 16)
    rng = np.random.default_rng(12)
    for _ in range(500):
        a = [int(rng.integers(1, 100)), int(rng.choice([8, 16, 32])), int(rng.integers(1, 40)),
             int(rng.choice([64, 80, 96, 128]))]
        b = [int(rng.integers(1, 100)), int(rng.choice([8, 16, 32])), int(rng.integers(1, 40)),
             int(rng.choice([64, 80, 96, 128]))]
        got = sc.sc_elastic_unit(sc.model_shape(*a, 2), sc.model_shape(*b, 2))
        assert got == oe.meu(oe.block_elems(*a), oe.block_elems(*b))


def test_algorithm1_matches_oracle(sc):
    rng = np.random.default_rng(13)
    for _ in range(2000):
        n, bs = int(rng.integers(0, 10000)), int(rng.choice([1, 8, 16, 32]))
        mi, mm = int(rng.integers(1, 64)), int(rng.integers(1, 64))
        length = int(rng.integers(0, 200000))
        assert sc.sc_scale_up(n, bs, mi, mm, length) == oe.scale_up(n, bs, mi, mm, length)
        window = [int(x) for x in rng.integers(0, 200000, size=int(rng.integers(0, 6)))]
        assert sc.sc_scale_down(n, bs, mi, mm, window) == oe.scale_down(n, bs, mi, mm, window)


@pytest.mark.parametrize("call", [
    lambda sc: sc.sc_scale_up(-1, 16, 1, 1, 5),
    lambda sc: sc.sc_scale_up(1, 0, 1, 1, 5),
    lambda sc: sc.sc_scale_up(1, 16, 0, 1, 5),
    lambda sc: sc.sc_scale_up(1, 16, 1, 1, -5),
    lambda sc: sc.sc_scale_down(1, 16, 1, 1, [-1]),
    lambda sc: sc.sc_elastic_unit(sc.model_shape(0, 16, 8, 128), sc.model_shape(1, 16, 8, 128)),
    lambda sc: sc.sc_plan_capacity(sc.model_shape(4, 16, 8, 128), -1, []),
])
def test_invalid_arguments(sc, call):
    with pytest.raises(sc.SwiftCacheError) as e:
        call(sc)
    assert e.value.status == sc.SC_ERR_INVALID


def test_overflow_is_reported(sc):
    big = sc.model_shape(1 << 30, 1 << 30, 1 << 30, 1 << 30, 2)
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_elastic_unit(big, sc.model_shape(3, 16, 8, 128))
    assert e.value.status == sc.SC_ERR_RANGE


def test_pool_resize_bounds_and_table_check(sc):
    p = sc.sc_pool_create(4, 2, 64, 16, 10, 0, 0, FAKE_BASE, 0)
    try:
        lay = sc.sc_pool_layout_get(p)
        assert (lay.n_device_blocks, lay.device_blocks_lent) == (10, 10)
        sc.sc_pool_resize(p, 3)
        lay = sc.sc_pool_layout_get(p)
        assert (lay.n_device_blocks, lay.device_blocks_lent, lay.device_base) == (10, 3, FAKE_BASE)
        # a table may only use lent blocks (validated before any device work)
        with pytest.raises(sc.SwiftCacheError) as e:
            sc.sc_table_create(p, [0, 5], [0, 2], [20], [0])
        assert e.value.status == sc.SC_ERR_RANGE and "lends" in str(e.value)
        sc.sc_pool_resize(p, 10)
        sc.sc_pool_resize(p, 0)
        for bad in (-1, 11):
            with pytest.raises(sc.SwiftCacheError) as e:
                sc.sc_pool_resize(p, bad)
            assert e.value.status == sc.SC_ERR_RANGE
    finally:
        sc.sc_pool_destroy(p)
