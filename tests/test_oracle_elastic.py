"""Pins of oracle/elastic.py (§3.4, Eq. 6-9, Algorithm 1): MEU values from
Table 2's model shapes by prime factorisation, equal traded bytes and
minimality by brute force, Algorithm 1 against exhaustive search, and resize
move counts against an element-by-element rebuild of both layouts."""

import itertools
import json
import os

import numpy as np

from oracle import elastic as oe

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table2_per_token_kv.json")


def _models():
    return {m["name"]: m for m in json.load(open(GOLDEN))["models"]}


def _factor(n):
    f, p = {}, 2
    while p * p <= n:
        while n % p == 0:
            f[p] = f.get(p, 0) + 1
            n //= p
        p += 1
    if n > 1:
        f[n] = f.get(n, 0) + 1
    return f


def _lcm_by_factors(a, b):
    fa, fb = _factor(a), _factor(b)
    out = 1
    for p in set(fa) | set(fb):
        out *= p ** max(fa.get(p, 0), fb.get(p, 0))
    return out


def _be(m, block_size=16):
    return oe.block_elems(m["layers"], block_size, m["kv_heads"], m["head_dim"])


def test_meu_for_table2_pairs():
    ms = _models()
    # Qwen3-32B master, Qwen3-8B worker: BE 64*16*8*128 = 2^20, 36*16*8*128 = 2^16 * 9.
    be_m, be_i = _be(ms["Qwen3-32B"]), _be(ms["Qwen3-8B"])
    assert (be_m, be_i) == (1048576, 589824)
    assert oe.lcm_elems(be_m, be_i) == _lcm_by_factors(be_m, be_i) == 9437184
    assert oe.meu(be_m, be_i) == (9, 16)
    # LWM master (32 layers, 32 KV heads), Qwen3-14B worker.
    be_m, be_i = _be(ms["LWM"]), _be(ms["Qwen3-14B"])
    assert oe.meu(be_m, be_i) == (5, 16)


def test_meu_trades_equal_bytes_and_is_minimal():
    for a, b in itertools.product([6, 8, 12, 36, 40, 64, 96], [5, 8, 10, 36, 48]):
        be_m, be_i = a * 16 * 8, b * 16 * 8
        mm, mi = oe.meu(be_m, be_i)
        assert mm * be_m == mi * be_i
        # brute force: the first multiple of be_m that is also a multiple of be_i
        k = 1
        while (k * be_m) % be_i:
            k += 1
        assert (k, k * be_m // be_i) == (mm, mi)


def _scale_up_search(n, bs, mi, mm, length):
    need = -(-length // bs)
    if need <= n:
        return 0, 0
    for k in range(1, 10 ** 6):
        if n + k * mi >= need:
            return k * mi, k * mm


def _scale_down_search(n, bs, mi, mm, window):
    max_need = -(-max(window, default=0) // bs)
    best = 0
    for k in range(0, n + 2):
        if n - k * mi >= max_need:
            best = k
    if max_need >= n:
        return 0, 0
    return best * mi, best * mm


def test_algorithm1_against_exhaustive_search():
    rng = np.random.default_rng(5)
    for _ in range(3000):
        n = int(rng.integers(0, 200))
        bs = int(rng.choice([1, 8, 16, 32]))
        mi, mm = int(rng.integers(1, 20)), int(rng.integers(1, 20))
        length = int(rng.integers(0, 5000))
        assert oe.scale_up(n, bs, mi, mm, length) == _scale_up_search(n, bs, mi, mm, length)
        window = [int(x) for x in rng.integers(0, 5000, size=int(rng.integers(0, 5)))]
        assert oe.scale_down(n, bs, mi, mm, window) == _scale_down_search(n, bs, mi, mm, window)


def test_algorithm1_hand_cases():
    # Qwen3-8B worker (B = 16) beside a Qwen3-32B master: MEU_i = 16, MEU_m = 9.
    assert oe.scale_up(100, 16, 16, 9, 1600) == (0, 0)        # exactly 100 blocks
    assert oe.scale_up(100, 16, 16, 9, 1601) == (16, 9)       # one block short -> one unit
    assert oe.scale_up(100, 16, 16, 9, 16 * 133) == (48, 27)  # 33 short -> 3 units
    assert oe.scale_down(100, 16, 16, 9, [16 * 60]) == (32, 18)   # 40 spare -> 2 whole units
    assert oe.scale_down(100, 16, 16, 9, [1600, 3]) == (0, 0)
    assert oe.scale_down(100, 16, 16, 9, []) == (96, 54)      # empty window: keep none


def _rebuild_moves(layout, n_layers, n_old, n_new):
    """Lay out labelled blocks for n_old, then for n_new, and count labels of
    kept blocks whose position changed."""
    def arrange(n):
        pos = {}
        if layout == "layer":
            order = [(l, b) for l in range(n_layers) for b in range(n)]
        else:
            order = [(l, b) for b in range(n) for l in range(n_layers)]
        for i, lb in enumerate(order):
            pos[lb] = i
        return pos
    a, b = arrange(n_old), arrange(n_new)
    return sum(1 for lb in a if lb in b and a[lb] != b[lb])


def test_resize_moves_layer_major_vs_block_major():
    for L, n0, n1 in itertools.product([1, 2, 3, 7], [1, 4, 9], [0, 1, 3, 4, 5, 12]):
        lm = oe.moved_blocks(oe.layer_major_offset, L, n0, n1)
        bm = oe.moved_blocks(oe.block_major_offset, L, n0, n1)
        assert lm == _rebuild_moves("layer", L, n0, n1)
        assert bm == _rebuild_moves("block", L, n0, n1) == 0
        assert lm == ((L - 1) * min(n0, n1) if n0 != n1 else 0)
    # The paper's figure: 3 layers of 4 blocks, one block added or removed.
    assert oe.moved_blocks(oe.layer_major_offset, 3, 4, 5) == 8
    assert oe.moved_blocks(oe.layer_major_offset, 3, 4, 3) == 6
