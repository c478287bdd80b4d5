"""Pins of oracle/capacity.py (Eq. 1-5, §3.2): the paper's worked example,
both regimes of Eq. 5, brute-force block counting, and planted mistakes."""

import itertools

from oracle import capacity as oc

MB = oc.m_block_bytes(16, 8, 128, 2)   # 64 KiB


def _bytes_for(blocks, unit, slack):
    return blocks * unit + slack


def test_worked_example_17_plus_8_is_25_against_10():
    # §3.2: L = 10, K_master = 100, K_1 = 9, K_2 = 8.  Byte budgets are chosen
    # with slack just below the next whole block so that the floors matter.
    L = 10
    c_master = _bytes_for(100, MB, MB - 1)
    c_workers = [_bytes_for(9, MB * L, MB * L - 1), _bytes_for(8, MB * L, 0)]
    p = oc.plan(c_master, c_workers, L, 16, 8, 128, 2)
    assert p["k_workers"] == [9, 8]
    assert p["k_master"] == 100
    assert p["n_lsc"] == 17
    assert p["n_rc"] == 8                      # floor(83 / 10)
    assert p["max_context_blocks"] == 25
    assert p["max_context_tokens"] == 25 * 16
    assert p["conventional_blocks"] == 10


def test_workers_fill_the_master_leave_no_regular_cache():
    L = 4
    p = oc.plan(_bytes_for(20, MB, 0), [_bytes_for(30, MB * L, 0)], L, 16, 8, 128, 2)
    assert p["n_lsc"] == 20 and p["n_rc"] == 0
    p = oc.plan(_bytes_for(20, MB, 0), [_bytes_for(20, MB * L, 0)], L, 16, 8, 128, 2)
    assert p["n_lsc"] == 20 and p["n_rc"] == 0


def test_regular_cache_boundary():
    L = 4
    for sum_k, expect_rc in [(19, 0), (16, 1), (15, 1), (12, 2), (0, 5)]:
        p = oc.plan(_bytes_for(20, MB, 0), [_bytes_for(sum_k, MB * L, 0)], L, 16, 8, 128, 2)
        assert p["n_lsc"] == sum_k and p["n_rc"] == expect_rc, (sum_k, p)


def _count_whole(budget, unit):
    n = 0
    while budget >= unit:
        budget -= unit
        n += 1
    return n


def test_block_counts_match_repeated_subtraction():
    for budget, unit, L in itertools.product([0, 1, 99, 100, 101, 1000, 4097], [1, 7, 100], [1, 3]):
        assert oc.master_single_layer_blocks(budget, unit) == _count_whole(budget, unit)
        assert oc.worker_full_layer_blocks(budget, unit, L) == _count_whole(budget, unit * L)


def test_eq1_matches_table2_sizes():
    # Eq. 1 per token (B = 1) times the layer count is Table 2's per-token KV
    # size; Qwen3-8B: 36 layers, 8 KV heads, head_dim 128, fp16 -> 0.141 MiB.
    assert 36 * oc.m_block_bytes(1, 8, 128, 2) == 147456


def test_more_memory_never_shortens_the_context():
    L = 5
    prev = -1
    for extra in range(0, 60):
        p = oc.plan(_bytes_for(40 + extra, MB, 0), [_bytes_for(7, MB * L, 0), _bytes_for(3, MB * L, 0)],
                    L, 16, 8, 128, 2)
        assert p["max_context_blocks"] >= prev
        prev = p["max_context_blocks"]


def test_planted_mistakes_fail_the_worked_example():
    def rc_without_floor_of_layers(kw, km, L):
        return km - sum(kw)                       # forgets the division by L

    def lsc_as_max(kw, km):
        return max(sum(kw), km)                   # min/max swapped

    kw, km, L = [9, 8], 100, 10
    assert oc.lsc_blocks(kw, km) + oc.rc_blocks(kw, km, L) == 25
    assert oc.lsc_blocks(kw, km) + rc_without_floor_of_layers(kw, km, L) != 25
    assert lsc_as_max(kw, km) + oc.rc_blocks(kw, km, L) != 25
