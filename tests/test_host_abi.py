"""Host logic of the C ABI, on the CPU: the library loads and exports every
declared symbol; argument validation; the attention work decomposition."""

import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "swiftcache.h")


@pytest.fixture(scope="module")
def sc():
    from paper_2606_16135_amd import swiftcache
    swiftcache.load()
    return swiftcache


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sc_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(sc):
    lib = ctypes.CDLL(sc.LIB_PATH)
    names = declared_functions()
    assert len(names) >= 14
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(sc.EXPORTED) == names


def test_version(sc):
    assert "gfx950" in sc.sc_version()


FAKE_BASE = 0x10000   # never dereferenced: every call below fails validation first


def _pool(sc, n_blocks=8, layers=2, bs=4):
    return sc.sc_pool_create(layers, 2, 64, bs, n_blocks, 0, 0, FAKE_BASE, 0)


def test_pool_validation(sc):
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_pool_create(2, 2, 96, 16, 8, 0, 0, FAKE_BASE, 0)
    assert e.value.status == sc.SC_ERR_UNSUPPORTED
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_pool_create(0, 2, 64, 16, 8, 0, 0, FAKE_BASE, 0)
    assert e.value.status == sc.SC_ERR_INVALID
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_pool_create(2, 2, 64, 16, 0, 0, 0, FAKE_BASE, 0)
    assert e.value.status == sc.SC_ERR_INVALID


def test_pool_rejects_blocks_beyond_32_bit_offsets(sc):
    # 256 tokens x 2^16 KV heads x 128 dims x 2 bytes = 4 GiB of K per block and layer
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_pool_create(1, 1 << 16, 128, 256, 8, 0, 0, FAKE_BASE, 0)
    assert e.value.status == sc.SC_ERR_UNSUPPORTED


def test_pool_element_type(sc):
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_pool_create(2, 2, 64, 16, 8, 0, 0, FAKE_BASE, 0, dtype=2)
    assert e.value.status == sc.SC_ERR_INVALID
    for code in (sc.SC_DTYPE_BF16, sc.SC_DTYPE_F16):
        p = sc.sc_pool_create(2, 2, 64, 16, 8, 0, 0, FAKE_BASE, 0, dtype=code)
        try:
            assert sc.sc_pool_layout_get(p).dtype == code
        finally:
            sc.sc_pool_destroy(p)


def test_pool_layout_follows_eq1(sc):
    p = sc.sc_pool_create(3, 8, 128, 16, 5, 0, 0, FAKE_BASE, 0)
    try:
        lay = sc.sc_pool_layout_get(p)
        assert lay.slice_bytes == 2 * 16 * 8 * 128 * 2 == 65536
        assert lay.block_bytes == 3 * 65536
        assert lay.row_bytes == 8 * 128 * 2
        assert lay.device_base == FAKE_BASE
    finally:
        sc.sc_pool_destroy(p)


@pytest.mark.parametrize("ids,cu,P,N,status", [
    ([0, 1, 2], [0, 3], [9], [4], "INVALID"),       # 13 tokens need ceil(13/4) = 4 entries
    ([0, 1], [0, 2], [9], [2], "INVALID"),          # too few entries
    ([0, 1, 1], [0, 3], [9], [0], "INVALID"),       # duplicate id
    ([0, 1, 8], [0, 3], [9], [0], "RANGE"),         # id outside the pool
    ([0, 1, -1], [0, 3], [9], [0], "RANGE"),        # negative id
    ([0, 1, 2], [0, 3], [-1], [10], "INVALID"),     # negative length
    ([0, 1, 2], [1, 3], [9], [0], "INVALID"),       # cu_blocks[0] != 0
])
def test_table_validation(sc, ids, cu, P, N, status):
    p = _pool(sc)
    try:
        with pytest.raises(sc.SwiftCacheError) as e:
            sc.sc_table_create(p, ids, cu, P, N)
        assert e.value.status == getattr(sc, "SC_ERR_" + status)
    finally:
        sc.sc_pool_destroy(p)


def test_regular_cache_pool_validation(sc):
    with pytest.raises(sc.SwiftCacheError) as e:      # paging needs a power-of-two block
        sc.sc_pool_create(2, 2, 64, 24, 8, 0, 0, FAKE_BASE, 0, 4, FAKE_BASE)
    assert e.value.status == sc.SC_ERR_UNSUPPORTED
    with pytest.raises(sc.SwiftCacheError) as e:      # smaller than a paged row group
        sc.sc_pool_create(2, 2, 64, 8, 8, 0, 0, FAKE_BASE, 0, 4, FAKE_BASE)
    assert e.value.status == sc.SC_ERR_UNSUPPORTED
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_pool_create(2, 2, 64, 16, 8, 0, 0, FAKE_BASE, 0, -1, FAKE_BASE)
    assert e.value.status == sc.SC_ERR_INVALID
    # attention addresses a regular-cache block in 32-bit products: blocks
    # (all layers, K and V) must stay under 4 GiB; 512 layers x 2 x 256 rows
    # x 64 heads x 128 x 2 bytes is exactly 4 GiB, 511 layers is under
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_pool_create(512, 64, 128, 256, 0, 0, 0, 0, 0, 1, FAKE_BASE)
    assert e.value.status == sc.SC_ERR_UNSUPPORTED and "4 GiB" in str(e.value)
    sc.sc_pool_destroy(sc.sc_pool_create(511, 64, 128, 256, 0, 0, 0, 0, 0, 1, FAKE_BASE))
    p = sc.sc_pool_create(2, 2, 64, 16, 0, 0, 0, 0, 0, 4, FAKE_BASE)   # a regular cache alone
    try:
        lay = sc.sc_pool_layout_get(p)
        assert (lay.rc_base, lay.n_rc_blocks, lay.n_device_blocks) == (FAKE_BASE, 4, 0)
    finally:
        sc.sc_pool_destroy(p)


# pool of 8 donor blocks (ids 0..7) and 4 regular-cache blocks (ids 8..11), B = 16
@pytest.mark.parametrize("ids,cu,P,N,status", [
    ([0, 8, 1], [0, 3], [33], [2], "INVALID"),       # regular-cache block after a donor block
    ([8, 9, 10], [0, 3], [33], [2], "INVALID"),      # third block holds new-turn rows
    ([8, 9, 10], [0, 3], [40], [0], "INVALID"),      # third block only partly filled
    ([8, 12, 0], [0, 3], [33], [0], "RANGE"),        # id past the regular cache
    ([8, 8, 0], [0, 3], [33], [0], "INVALID"),       # duplicate regular-cache id
])
def test_regular_cache_table_validation(sc, ids, cu, P, N, status):
    p = sc.sc_pool_create(2, 2, 64, 16, 8, 0, 0, FAKE_BASE, 0, 4, FAKE_BASE)
    try:
        with pytest.raises(sc.SwiftCacheError) as e:
            sc.sc_table_create(p, ids, cu, P, N)
        assert e.value.status == getattr(sc, "SC_ERR_" + status)
    finally:
        sc.sc_pool_destroy(p)


def test_chunked_stack_rejects_bad_chunk(sc):
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_stack_chunked(FAKE_BASE, FAKE_BASE, [1], [1], [1], [1],
                                    [sc.active(1, 1, 1), sc.active(1, 1, 1)], 8, 0)
    assert e.value.status == sc.SC_ERR_INVALID
    assert "chunk_tokens" in str(e.value)


def test_stack_status_validation(sc):
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_table_stack_status(None)
    assert e.value.status == sc.SC_ERR_INVALID


def test_misaligned_pointers_are_rejected(sc):
    """The kernels move 16-byte chunks: element pointers must be 16-byte
    aligned, lse 4-byte aligned; checked before any device work."""
    A = FAKE_BASE
    for q, k, v, out in [(A + 2, A, A, A), (A, A + 8, A, A), (A, A, A + 4, A), (A, A, A, A + 2)]:
        with pytest.raises(sc.SwiftCacheError) as e:
            sc.sc_prefill_attn(q, k, v, 4, 4, 8, 8, 128, out)
        assert e.value.status == sc.SC_ERR_INVALID and "16-byte aligned" in str(e.value)
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn(A, A, A, 4, 4, 8, 8, 128, A, lse=A + 2)
    assert e.value.status == sc.SC_ERR_INVALID and "4-byte aligned" in str(e.value)
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_pool_create(2, 2, 64, 16, 8, 0, 0, FAKE_BASE + 8, 0)
    assert e.value.status == sc.SC_ERR_INVALID and "16-byte aligned" in str(e.value)


def test_attention_argument_validation(sc):
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn(1, 1, 1, 4, 4, 12, 8, 128, 1)
    assert e.value.status == sc.SC_ERR_INVALID
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn(1, 1, 1, 4, 4, 8, 8, 80, 1)
    assert e.value.status == sc.SC_ERR_UNSUPPORTED
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn(1, 1, 1, 4, 4, 64, 2, 128, 1)     # group 32
    assert e.value.status == sc.SC_ERR_UNSUPPORTED
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn(1, 1, 1, -1, 4, 8, 8, 128, 1)
    assert e.value.status == sc.SC_ERR_INVALID
    sc.sc_prefill_attn(0, 0, 0, 5, 0, 8, 8, 128, 0)          # new_len == 0 is a no-op


KEY_TILE = 32
ROWS = 256


def _check_plan(sc, P, N, hq, hkv, target, rc=None):
    items, splits = sc.sc_attn_plan_query(P, N, hq, hkv, target, rc_keys=rc)
    rc = [0] * len(P) if rc is None else rc
    group = hq // hkv
    rows_q = ROWS // group
    assert len(items) % 8 == 0
    real = items[items[:, 0] >= 0]
    # padding slots are only idle workgroups
    assert np.all(items[items[:, 0] < 0][:, 1:] == 0)
    # each (seq, kv head) group lives on one XCD
    xcd_of = {}
    for slot, it in enumerate(items):
        if it[0] < 0:
            continue
        key = (int(it[0]), int(it[1]))
        assert xcd_of.setdefault(key, slot % 8) == slot % 8
    # per query tile, the splits partition [0, P + q0 + nq)
    tiles = {}
    for it in real:
        seq, kvh, q0, nq, kb, ke, s, paged = (int(x) for x in it)
        r = rc[seq]
        # regular-cache items cover [0, r), the others [r, ...): tiles start
        # on the key-tile grid of their own range
        if paged:
            assert ke <= r and kb % KEY_TILE == 0
        else:
            assert kb >= r and (kb - r) % KEY_TILE == 0
        assert ke >= kb
        tiles.setdefault((seq, kvh, q0, nq), []).append((s, kb, ke))
    expect = set()
    for b, (p, n) in enumerate(zip(P, N)):
        for g in range(hkv):
            for q0 in range(0, n, rows_q):
                expect.add((b, g, q0, min(rows_q, n - q0)))
    assert set(tiles) == expect
    for (seq, kvh, q0, nq), parts in tiles.items():
        parts.sort()
        assert [s for s, _, _ in parts] == list(range(splits[seq]))
        pos = 0
        for _, kb, ke in parts:
            if ke > kb:
                assert kb == pos
                pos = ke
        assert pos == P[seq] + q0 + nq
    return items, splits


@pytest.mark.parametrize("P,N,hq,hkv,target", [
    ([8192], [512], 32, 8, 768),
    ([32768], [1024], 40, 8, 768),
    ([131072], [2048], 32, 8, 768),
    ([256], [64], 8, 8, 768),
    ([0], [130], 8, 8, 768),
    ([5000], [40], 8, 2, 768),
    ([33, 0, 1000, 17], [5, 64, 1, 200], 16, 4, 768),
    ([7, 9], [0, 3], 8, 8, 4),
])
def test_plan_covers_every_row_and_key_once(sc, P, N, hq, hkv, target):
    _check_plan(sc, P, N, hq, hkv, target)


@pytest.mark.parametrize("P,N,rc,hq,hkv", [
    ([8192], [512], [4096], 32, 8),
    ([8192], [512], [8192], 32, 8),           # the whole prefix in the regular cache
    ([5000], [40], [16], 8, 2),               # one block, off the key-tile grid
    ([33, 0, 1000, 17], [5, 64, 1, 200], [32, 0, 496, 16], 16, 4),
    ([131072], [2048], [65536], 32, 8),
])
def test_plan_with_regular_cache(sc, P, N, rc, hq, hkv):
    items, splits = _check_plan(sc, P, N, hq, hkv, 768, rc)
    for b, r in enumerate(rc):
        mine = items[items[:, 0] == b]
        if len(mine) == 0:
            continue
        assert bool(np.any(mine[:, 7] == 1)) == (r > 0)
        if r > 0:
            assert splits[b] >= 2               # partials over both ranges are merged


def test_plan_rejects_regular_cache_beyond_prefix(sc):
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_attn_plan_query([100], [10], 8, 8, 0, rc_keys=[112])
    assert e.value.status == sc.SC_ERR_INVALID


def test_plan_random_batches(sc):
    rng = np.random.default_rng(0)
    for _ in range(20):
        b = int(rng.integers(1, 9))
        P = rng.integers(0, 3000, size=b).tolist()
        N = rng.integers(0, 300, size=b).tolist()
        if sum(N) == 0:
            N[0] = 1
        hkv = int(rng.choice([1, 2, 8]))
        group = int(rng.choice([1, 4, 5]))
        _check_plan(sc, P, N, hkv * group, hkv, int(rng.integers(16, 2000)))


def test_planner_counts_the_merge_when_splitting(sc):
    """The split count minimises the forward schedule plus the merge kernel
    that follows it: one 8B-shape conversation (64 query tiles) is split 4
    ways to fill 256 workgroup slots, while a 16-conversation batch whose
    ~1100 unsplit items already balance over the slots is not split (its
    merge would cost more than splitting saves); the 14B shape takes 3."""
    from paper_2606_16135_amd import workloads as W
    _, splits = sc.sc_attn_plan_query([8192], [512], 32, 8, 256)
    assert splits == [4]
    _, splits = sc.sc_attn_plan_query([32768], [1024], 40, 8, 256)
    assert splits == [3]
    wl = W.config(3)
    items, splits = sc.sc_attn_plan_query([int(x) for x in wl.prefix_len], [int(x) for x in wl.new_len],
                                          32, 8, 256)
    assert splits == [1] * 16 and len(items) >= 1024
    # the default slot count is one workgroup per CU of an MI355X
    assert sc.sc_attn_plan_query([8192], [512], 32, 8, 0)[1] == [4]


def test_planner_items_cover_every_query_tile_once(sc):
    """Plan invariants at any shape: every (sequence, KV head) has all its
    query tiles (rows of 256 / group heads' worth of queries); the key ranges
    of one tile's items are contiguous, cover [0, P + q0 + nq) exactly once
    and number the sequence's split count; regular-cache keys [0, rc) and
    slot keys never share an item; all items of one (sequence, KV head) run
    on one XCD (slot w on XCD w % 8)."""
    rng = np.random.default_rng(2606_16135_31)
    for _ in range(60):
        b = int(rng.integers(1, 7))
        hkv = int(rng.choice([1, 2, 4, 8]))
        g = int(rng.choice([1, 2, 4, 5, 8]))
        P = [int(rng.integers(0, 20000)) for _ in range(b)]
        N = [int(rng.integers(1, 1500)) for _ in range(b)]
        rc = [16 * int(rng.integers(0, p // 16 + 1)) if rng.random() < 0.4 else 0 for p in P]
        items, splits = sc.sc_attn_plan_query(P, N, hkv * g, hkv, 256, rc_keys=rc)
        rows_q = 256 // g
        groups, xcd = {}, {}
        for w, it in enumerate(items):
            seq, kvh, q0, nq, kb, ke, _, paged = (int(x) for x in it)
            if seq < 0:
                continue
            groups.setdefault((seq, kvh, q0), []).append((kb, ke, nq, paged))
            xcd.setdefault((seq, kvh), set()).add(w % 8)
        for s in range(b):
            for h in range(hkv):
                assert sorted(q0 for (ss, hh, q0) in groups if ss == s and hh == h) == list(range(0, N[s], rows_q))
                assert len(xcd[(s, h)]) == 1
        for (s, h, q0), v in groups.items():
            v.sort()
            assert len(v) == splits[s]
            pos = 0
            for kb, ke, nq, paged in v:
                assert nq == min(rows_q, N[s] - q0)
                assert kb == pos and ke >= kb
                assert (ke <= rc[s]) if paged else (kb >= rc[s])
                pos = ke
            assert pos == P[s] + v[0][2] + q0


def test_planner_splits_short_turns(sc):
    """Short new turns (a few hundred keys per query tile) are split down to
    two-tile ranges so that enough workgroups run: measured on MI355X this
    takes a P=1024, N=64 attention call (8 query tiles) from 24 to 17 us."""
    for P, N in [(512, 32), (1024, 64), (2048, 64), (2048, 128)]:
        items, splits = sc.sc_attn_plan_query([P], [N], 32, 8, 256)
        assert splits[0] >= 4, (P, N, splits)
        assert len(items) >= 32
        assert min(int(it[5]) - int(it[4]) for it in items if it[0] >= 0 and it[5] > it[4]) >= 32


def test_noalloc_split_choice_equals_the_planner(sc):
    """The allocation-free entry point chooses its key splits in fixed-size
    buffers; for one sequence it must choose what the planner chooses, so
    that its output equals sc_prefill_attn's bit for bit."""
    rng = np.random.default_rng(2606_16135_71)
    shapes = [(8192, 512, 32, 8), (32768, 1024, 40, 8), (131072, 2048, 32, 8), (1024, 64, 32, 8),
              (0, 1, 8, 8), (5, 300, 8, 2), (3000, 4096, 32, 8)]
    for _ in range(150):
        hkv = int(rng.choice([1, 2, 4, 8]))
        g = int(rng.choice([1, 2, 4, 5, 8, 16]))
        shapes.append((int(rng.integers(0, 60000)), int(rng.integers(1, 3000)), hkv * g, hkv))
    for P, N, hq, hkv in shapes:
        for slots in (256, 240, 64):
            _, splits = sc.sc_attn_plan_query([P], [N], hq, hkv, slots)
            assert sc.sc_attn_noalloc_splits(P, N, hq, hkv, slots) == splits[0], (P, N, hq, hkv, slots)


def _implicit_items(P, N, hq, hkv, S):
    """The items the attention kernel derives from its workgroup index when
    it is launched without a work list (the allocation-free entry point):
    workgroup w takes entry (w % 8) * per + w // 8 of the list ordered
    (KV head, query tile, split)."""
    rows_q = ROWS // (hq // hkv)
    n_qt = -(-N // rows_q)
    total = hkv * n_qt * S
    per = -(-total // 8)
    out = []
    for w in range(8 * per):
        j, g = w // 8, (w % 8) * per + w // 8
        if j >= per or g >= total:
            continue
        kvh, r = divmod(g, n_qt * S)
        tile, sp = divmod(r, S)
        q0 = tile * rows_q
        nq = min(rows_q, N - q0)
        keys = P + q0 + nq
        t = -(-keys // KEY_TILE)
        b0 = min(keys, (sp * t // S) * KEY_TILE)
        b1 = min(keys, ((sp + 1) * t // S) * KEY_TILE)
        out.append((0, kvh, q0, nq, b0, max(b0, b1), sp, 0))
    return out


def test_noalloc_implicit_items_equal_the_planned_items(sc):
    """Without a work list each workgroup derives its item from its index;
    the set of items must be the planner's for the same sequence (same
    query tiles, key ranges and split indices, every one exactly once), and
    one KV head's items must sit on as few XCDs as the list allows."""
    rng = np.random.default_rng(2606_16135_72)
    shapes = [(8192, 512, 32, 8), (32768, 1024, 40, 8), (3000, 700, 32, 8), (0, 130, 8, 8), (5000, 40, 8, 2)]
    for _ in range(60):
        hkv = int(rng.choice([1, 2, 4, 8]))
        g = int(rng.choice([1, 2, 4, 5, 8]))
        shapes.append((int(rng.integers(0, 20000)), int(rng.integers(1, 1500)), hkv * g, hkv))
    for P, N, hq, hkv in shapes:
        items, splits = sc.sc_attn_plan_query([P], [N], hq, hkv, 256)
        planned = sorted(tuple(int(x) for x in it) for it in items if it[0] >= 0)
        implicit = _implicit_items(P, N, hq, hkv, splits[0])
        assert sorted(implicit) == planned, (P, N, hq, hkv)
        assert len(set(implicit)) == len(implicit)


def test_noalloc_argument_validation(sc):
    """Checked before any device work, as for sc_prefill_attn."""
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn_noalloc(1, 1, 1, 4, 4, 12, 8, 128, 1)
    assert e.value.status == sc.SC_ERR_INVALID
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn_noalloc(1, 1, 1, 4, 4, 8, 8, 80, 1)
    assert e.value.status == sc.SC_ERR_UNSUPPORTED
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn_noalloc(FAKE_BASE + 2, FAKE_BASE, FAKE_BASE, 4, 4, 8, 8, 128, FAKE_BASE)
    assert e.value.status == sc.SC_ERR_INVALID and "16-byte aligned" in str(e.value)
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn_noalloc(1, 1, 1, -1, 4, 8, 8, 128, 1)
    assert e.value.status == sc.SC_ERR_INVALID
    sc.sc_prefill_attn_noalloc(0, 0, 0, 5, 0, 8, 8, 128, 0)          # new_len == 0 is a no-op
    # Key rows are addressed with signed 32-bit byte offsets, loads past the
    # last tile included: 8 KV heads x 128 dims x 2 bytes = 2 KiB per token,
    # so 2^20 tokens are 2 GiB, and the last 256 below that are refused too.
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn_noalloc(FAKE_BASE, FAKE_BASE, FAKE_BASE, (1 << 20) - 256 - 64, 64, 32, 8, 128, FAKE_BASE)
    assert e.value.status == sc.SC_ERR_UNSUPPORTED and "2 GiB" in str(e.value)
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_attn_noalloc_splits(4, 70000, 32, 8)                   # beyond the fixed buffers
    assert e.value.status == sc.SC_ERR_RANGE
