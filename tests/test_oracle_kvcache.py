"""Pins of the KV-movement oracle (gather / append / store).

The pool is built here by scattering a known dense KV with explicit
per-token loops (an independent construction), so the gather is checked
against data it did not produce.  Planted mistakes at the end must fail.
"""

import numpy as np
import pytest

from oracle import kvcache as ok


def _table(rng, prefix, new, bs, n_blocks):
    per = [(p + n + bs - 1) // bs for p, n in zip(prefix, new)]
    ids = rng.permutation(n_blocks)[:sum(per)].astype(np.int32)
    cu = np.concatenate([[0], np.cumsum(per)]).astype(np.int32)
    return ids, cu


def _dense_and_pool(seed, prefix, new, n_layers=3, bs=4, hkv=2, d=8, n_blocks=40):
    """Dense per-sequence KV [L][2][P+N][H][D] and a pool holding exactly that
    KV at the positions the table names; all other pool bytes are 0xFFFF."""
    rng = np.random.default_rng(seed)
    ids, cu = _table(rng, prefix, new, bs, n_blocks)
    pool = np.full(ok.pool_shape(n_blocks, n_layers, bs, hkv, d), 0xFFFF, dtype=np.uint16)
    dense = []
    for b, (p, n) in enumerate(zip(prefix, new)):
        kv = rng.integers(0, 0x7F00, size=(n_layers, 2, p + n, hkv, d), dtype=np.uint16)
        dense.append(kv)
        for layer in range(n_layers):
            for t in range(p):
                blk = ids[cu[b] + t // bs]
                for s in range(2):
                    pool[blk, layer, s, t % bs] = kv[layer, s, t]
    return pool, ids, cu, dense


@pytest.mark.parametrize("prefix,new,bs", [
    ([8], [3], 4),                # whole blocks
    ([10], [5], 4),               # partial last prefix block
    ([0, 7, 13], [2, 4, 1], 4),   # batch, empty prefix, ragged
    ([33], [0], 16),              # no new tokens
])
def test_gather_reconstructs_dense_prefix(prefix, new, bs):
    pool, ids, cu, dense = _dense_and_pool(3 + sum(prefix), prefix, new, bs=bs)
    _, cu_k = ok.seq_offsets(prefix, new)
    for layer in range(pool.shape[1]):
        k, v = ok.gather_layer(pool, ids, cu, prefix, new, layer)
        for b, p in enumerate(prefix):
            assert np.array_equal(k[cu_k[b]:cu_k[b] + p], dense[b][layer, 0, :p])
            assert np.array_equal(v[cu_k[b]:cu_k[b] + p], dense[b][layer, 1, :p])


def test_gather_is_a_permutation_of_pool_rows_and_reads_only():
    prefix, new, bs = [9, 14], [3, 6], 4
    pool, ids, cu, _ = _dense_and_pool(5, prefix, new, bs=bs)
    before = pool.copy()
    k, v = ok.gather_layer(pool, ids, cu, prefix, new, 1)
    assert np.array_equal(pool, before)
    _, cu_k = ok.seq_offsets(prefix, new)
    expect = []
    for b, p in enumerate(prefix):
        for t in range(p):
            expect.append((int(ids[cu[b] + t // bs]), t % bs))
    # every (block, row) slot appears exactly once and rows hold its bytes
    assert len(set(expect)) == len(expect) == sum(prefix)
    got = np.concatenate([k[cu_k[b]:cu_k[b] + p] for b, p in enumerate(prefix)])
    for r, (blk, row) in enumerate(expect):
        assert np.array_equal(got[r], pool[blk, 1, 0, row])


def test_append_places_new_rows_after_prefix():
    prefix, new = [5, 0, 7], [2, 3, 1]
    rng = np.random.default_rng(8)
    tk = sum(prefix) + sum(new)
    k0 = np.zeros((tk, 2, 4), dtype=np.uint16)
    knew = rng.integers(1, 1000, size=(sum(new), 2, 4), dtype=np.uint16)
    vnew = rng.integers(1, 1000, size=(sum(new), 2, 4), dtype=np.uint16)
    k, v = ok.append_new(k0, k0, knew, vnew, prefix, new)
    assert np.array_equal(k[5:7], knew[0:2])
    assert np.array_equal(k[7:10], knew[2:5])
    assert np.array_equal(v[17:18], vnew[5:6])
    assert np.count_nonzero(k[:5]) == 0 and np.count_nonzero(k[10:17]) == 0


def test_store_then_next_turn_fetch_round_trips():
    prefix, new, bs = [10, 3], [5, 9], 4
    pool, ids, cu, dense = _dense_and_pool(21, prefix, new, bs=bs)
    cu_q, _ = ok.seq_offsets(prefix, new)
    layer = 2
    knew = np.concatenate([dense[b][layer, 0, p:] for b, p in enumerate(prefix)])
    vnew = np.concatenate([dense[b][layer, 1, p:] for b, p in enumerate(prefix)])
    pool2 = ok.store_layer(pool, ids, cu, prefix, new, layer, knew, vnew)
    # next turn: the whole history is the prefix, no new tokens
    prefix2 = [p + n for p, n in zip(prefix, new)]
    k, v = ok.gather_layer(pool2, ids, cu, prefix2, [0, 0], layer)
    _, cu_k2 = ok.seq_offsets(prefix2, [0, 0])
    for b, p2 in enumerate(prefix2):
        assert np.array_equal(k[cu_k2[b]:cu_k2[b] + p2], dense[b][layer, 0])
        assert np.array_equal(v[cu_k2[b]:cu_k2[b] + p2], dense[b][layer, 1])


def test_store_changes_only_new_token_rows():
    prefix, new, bs = [6], [7], 4
    pool, ids, cu, _ = _dense_and_pool(4, prefix, new, bs=bs)
    rng = np.random.default_rng(2)
    knew = rng.integers(0, 100, size=(7, 2, 8), dtype=np.uint16)
    out = ok.store_layer(pool, ids, cu, prefix, new, 0, knew, knew)
    changed = np.argwhere(np.any(out != pool, axis=(4, 5)))
    touched = {(int(ids[(6 + i) // bs]), 0, s, (6 + i) % bs) for i in range(7) for s in range(2)}
    assert {tuple(int(x) for x in c) for c in changed} <= touched


def test_layout_helpers():
    assert ok.blocks_needed([0, 1, 16, 17], [0, 0, 0, 15], 16).tolist() == [0, 1, 1, 2]
    cu_q, cu_k = ok.seq_offsets([3, 4], [1, 2])
    assert cu_q.tolist() == [0, 1, 3] and cu_k.tolist() == [0, 4, 10]


# ---- planted mistakes ------------------------------------------------------

def test_planted_block_index_mistake_is_caught(monkeypatch):
    real = ok._token_locations

    def off_by_one(ids, start, count, bs):
        blk, row = real(ids, start, count, bs)
        return np.roll(blk, 1), row
    prefix, new, bs = [12], [2], 4
    pool, ids, cu, dense = _dense_and_pool(6, prefix, new, bs=bs)
    monkeypatch.setattr(ok, "_token_locations", off_by_one)
    k, _ = ok.gather_layer(pool, ids, cu, prefix, new, 0)
    assert not np.array_equal(k[:12], dense[0][0, 0, :12])


def test_planted_kv_swap_is_caught():
    prefix, new, bs = [8], [1], 4
    pool, ids, cu, dense = _dense_and_pool(9, prefix, new, bs=bs)
    swapped = pool[:, :, ::-1].copy()
    k, _ = ok.gather_layer(swapped, ids, cu, prefix, new, 0)
    assert not np.array_equal(k[:8], dense[0][0, 0, :8])


def test_regular_cache_rows_by_counting():
    """Rows of leading regular-cache blocks, counted block by block: B rows
    per leading regular-cache block at the start of each sequence, none
    elsewhere; the fetched rows are the remaining prefix rows."""
    bs, rc0 = 4, 100
    prefix, new = [12, 9, 0, 8], [3, 2, 5, 0]
    ids = np.array([100, 101, 7,  102, 3, 4,  5, 6,  103, 104], dtype=np.int32)
    cu = np.array([0, 3, 6, 8, 10], dtype=np.int32)
    rows = ok.regular_cache_rows(ids, cu, prefix, new, bs, rc0)
    _, cu_k = ok.seq_offsets(prefix, new)
    expect = np.zeros(int(cu_k[-1]), dtype=bool)
    expect[0:8] = True                       # sequence 0: two blocks
    expect[15:19] = True                     # sequence 1: one block
    expect[31:39] = True                     # sequence 3: its whole prefix
    assert np.array_equal(rows, expect)
    assert rows.sum() == bs * 5
    # a regular-cache block after a donor block, or one that new tokens share
    with pytest.raises(AssertionError):
        ok.regular_cache_rows(np.array([7, 100, 1], dtype=np.int32), np.array([0, 3]), [9], [2], bs, rc0)
    with pytest.raises(AssertionError):
        ok.regular_cache_rows(np.array([100, 101, 102], dtype=np.int32), np.array([0, 3]), [9], [2], bs, rc0)
