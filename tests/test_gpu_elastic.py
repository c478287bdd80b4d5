"""GPU: the O(1) resize of the block-major HBM tier leaves every kept block
in place (fetch after shrinking and after growing again is byte-exact
against the oracle) and refuses to release blocks a live table uses."""

import numpy as np
import pytest

from oracle import kvcache as ok
from paper_2606_16135_amd import workloads as W

from _gpu_util import DevicePool, new_active, require_gpu, to_u16

pytestmark = pytest.mark.gpu


def _fetch_matches(sc, dp, wl, pool, table, layer):
    import torch
    k, v, act = new_active(sc, wl)
    sc.sc_fetch_layer_kv(dp.handle, table, layer, act, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    k_ref, v_ref = ok.gather_layer(pool, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, layer)
    _, cu_k = ok.seq_offsets(wl.prefix_len, wl.new_len)
    rows = np.zeros(wl.total_kv, dtype=bool)
    for b, p in enumerate(wl.prefix_len):
        rows[cu_k[b]:cu_k[b] + p] = True
    return np.array_equal(to_u16(k)[rows], k_ref[rows]) and np.array_equal(to_u16(v)[rows], v_ref[rows])


def test_resize_keeps_blocks_in_place_and_protects_live_tables():
    sc = require_gpu()
    wl = W.small_workload(201, [300, 77], [20, 9], 2, 8, 2, 128, pool_factor=3.0)
    pool = W.pool_numpy(wl)
    dp = DevicePool(sc, wl, pool)
    try:
        cap = wl.n_device_blocks
        top = int(np.max(wl.block_ids))
        print(f"\n[elastic] capacity {cap}, highest id in the table {top}", flush=True)
        with pytest.raises(sc.SwiftCacheError) as e:
            sc.sc_pool_resize(dp.handle, top)            # would release a block the table uses
        assert e.value.status == sc.SC_ERR_INVALID
        sc.sc_pool_resize(dp.handle, top + 1)
        assert sc.sc_pool_layout_get(dp.handle).device_blocks_lent == top + 1
        assert _fetch_matches(sc, dp, wl, pool, dp.table, 1)
        sc.sc_pool_resize(dp.handle, cap)
        assert _fetch_matches(sc, dp, wl, pool, dp.table, 0)
        # without the table every block may go; a new table sees the same bytes
        sc.sc_table_destroy(dp.table)
        dp.table = None
        sc.sc_pool_resize(dp.handle, 0)
        with pytest.raises(sc.SwiftCacheError) as e:
            sc.sc_table_create(dp.handle, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len)
        assert e.value.status == sc.SC_ERR_RANGE
        sc.sc_pool_resize(dp.handle, cap)
        dp.table = sc.sc_table_create(dp.handle, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len)
        assert _fetch_matches(sc, dp, wl, pool, dp.table, 1)
    finally:
        if dp.table is not None:
            sc.sc_table_destroy(dp.table)
        sc.sc_pool_destroy(dp.handle)
