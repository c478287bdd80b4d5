"""GPU parity of every C-ABI call against the oracle, element by element, on
seeded inputs small enough for the dense oracle: several key tiles and query
tiles with ragged tails, head groups 1/3/4/5/6/7/8/16, head_dim 64/128, bf16 and fp16 values, empty prefix,
a batch with an empty new turn, split-key work, a half host-pinned pool, and
tables whose leading blocks sit in the regular-cache tier (read in place by
attention; their active-buffer rows hold NaN patterns the kernel must not
read).

Fetch, append and store are compared byte for byte; attention to
|gpu - oracle| <= 2e-2 + 1e-2 |oracle| on every element plus a relative-L2
bound (tests/_gpu_util.py)."""

import numpy as np
import pytest

from oracle import attention as oa
from oracle import kvcache as ok
from paper_2606_16135_amd import workloads as W

from _gpu_util import (DevicePool, bits_to_f64, compare_attention, from_u16, new_active,
                       require_gpu, to_u16)

pytestmark = pytest.mark.gpu


def _case(name):
    sw = W.small_workload
    return {
        "cfg1": lambda: W.config(1),
        "g4_d128_ragged": lambda: sw(101, [100], [77], 2, 32, 8, 128),
        "g5_d128": lambda: sw(102, [300], [50], 1, 40, 8, 128),
        "g1_d64_P0": lambda: sw(103, [0], [130], 1, 8, 8, 64),
        "g4_split_long": lambda: sw(104, [5000], [40], 1, 8, 2, 128),
        "varlen_batch": lambda: sw(105, [33, 0, 1000, 17], [5, 64, 1, 200], 2, 16, 4, 64),
        "varlen_empty_turn": lambda: sw(108, [40, 77], [0, 33], 1, 8, 2, 128),
        "host_tier": lambda: sw(106, [200, 77], [20, 31], 2, 8, 2, 128, host_fraction=0.5),
        "g8_d64": lambda: sw(107, [64], [16], 1, 64, 8, 64),
        # regular-cache tier: leading full prefix blocks read in place
        "rc_varlen": lambda: sw(109, [1000, 40, 0, 300, 16], [30, 17, 50, 1, 5], 2, 16, 4, 64,
                                rc_fraction=0.6),
        "rc_split_d128": lambda: sw(110, [5000], [40], 1, 8, 2, 128, rc_fraction=0.5),
        "rc_whole_prefix": lambda: sw(111, [256, 512], [64, 3], 1, 32, 8, 128, rc_fraction=1.0),
        "rc_host": lambda: sw(112, [200, 77], [20, 31], 2, 8, 2, 128, host_fraction=0.5, rc_fraction=0.5),
        # IEEE fp16 values (the paper's serving precision)
        "f16_g4_d128_ragged": lambda: sw(121, [100], [77], 2, 32, 8, 128, dtype="f16"),
        "f16_varlen": lambda: sw(122, [33, 0, 1000, 17], [5, 64, 1, 200], 2, 16, 4, 64, dtype="f16"),
        "f16_g5_split_rc": lambda: sw(123, [5000, 300], [40, 20], 1, 40, 8, 128, rc_fraction=0.5, dtype="f16"),
        "f16_host": lambda: sw(124, [200, 77], [20, 31], 1, 8, 2, 128, host_fraction=0.5, dtype="f16"),
        # size extremes: largest block (with a regular cache), one-token
        # blocks, many short sequences, the largest GQA group
        "bs256_rc": lambda: sw(131, [700, 300], [30, 2], 1, 8, 2, 128, block_size=256, rc_fraction=0.5),
        "bs1": lambda: sw(132, [50, 3], [9, 20], 1, 8, 8, 64, block_size=1),
        "many_seqs": lambda: sw(133, list(range(0, 400, 10)), [1 + (7 * i) % 40 for i in range(40)], 1, 16, 4, 64),
        "g16_d64": lambda: sw(134, [129], [100], 1, 32, 2, 64),
        # groups that do not divide the 256-row workgroup (its last rows
        # idle), as in 28/4 and 12/2 head layouts, and the largest group at
        # head_dim 128
        "g7_d128_split": lambda: sw(135, [3000], [45], 1, 28, 4, 128),
        "g6_d64_varlen": lambda: sw(136, [500, 90], [37, 70], 2, 12, 2, 64),
        "g3_d128_rc": lambda: sw(137, [800, 41], [60, 9], 1, 24, 8, 128, rc_fraction=0.5),
        "g16_d128": lambda: sw(138, [300], [40], 1, 32, 2, 128),
    }[name]()


CASES = ["cfg1", "g4_d128_ragged", "g5_d128", "g1_d64_P0", "g4_split_long", "varlen_batch",
         "varlen_empty_turn", "host_tier", "g8_d64", "rc_varlen", "rc_split_d128", "rc_whole_prefix",
         "rc_host", "f16_g4_d128_ragged", "f16_varlen", "f16_g5_split_rc", "f16_host", "bs256_rc", "bs1",
         "many_seqs", "g16_d64", "g7_d128_split", "g6_d64_varlen", "g3_d128_rc", "g16_d128"]


def _oracle_layer(wl, pool_u16, layer, q, kn, vn):
    k_act, v_act = ok.gather_layer(pool_u16, wl.block_ids, wl.cu_blocks, wl.prefix_len,
                                   wl.new_len, layer)
    k_full, v_full = ok.append_new(k_act, v_act, kn, vn, wl.prefix_len, wl.new_len)
    o, lse = oa.attention(oa.bits_to_f64(q, wl.dtype), oa.bits_to_f64(k_full, wl.dtype),
                          oa.bits_to_f64(v_full, wl.dtype), wl.prefix_len, wl.new_len)
    return k_act, v_act, k_full, v_full, o, lse


def _prefix_rows(wl):
    _, cu_k = ok.seq_offsets(wl.prefix_len, wl.new_len)
    rows = np.zeros(wl.total_kv, dtype=bool)
    for b, p in enumerate(wl.prefix_len):
        rows[cu_k[b]:cu_k[b] + p] = True
    return rows


def _rc_rows(wl):
    return ok.regular_cache_rows(wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, wl.block_size,
                                 wl.rc_first_id)


@pytest.mark.parametrize("name", CASES)
@pytest.mark.parametrize("q_scale", [1.0, 8.0], ids=["flat", "peaky"])
def test_layer_path_matches_oracle(name, q_scale):
    sc = require_gpu()
    import torch
    wl = _case(name)
    pool_u16 = W.pool_numpy(wl)
    dp = DevicePool(sc, wl, pool_u16)
    stream = torch.cuda.current_stream().cuda_stream
    try:
        for layer in range(wl.n_layers):
            q, kn, vn = W.layer_inputs_numpy(wl, layer, q_scale=q_scale)
            qd, knd, vnd = (from_u16(x, "cuda", wl.dtype) for x in (q, kn, vn))
            k, v, act = new_active(sc, wl, fill_bits=0xFFFF)
            sc.sc_fetch_layer_kv(dp.handle, dp.table, layer, act, stream)
            torch.cuda.synchronize()
            k_act, v_act, k_full, v_full, o_ref, lse_ref = _oracle_layer(wl, pool_u16, layer, q, kn, vn)
            rcr = _rc_rows(wl)
            pre = _prefix_rows(wl) & ~rcr
            kg, vg = to_u16(k), to_u16(v)
            # fetch: prefix rows outside the regular cache bit-exact, other
            # rows untouched (regular-cache rows keep the NaN fill, so
            # attention below fails if it reads them from the slot)
            assert np.array_equal(kg[pre], k_act[pre]), f"{name} layer {layer}: K fetch"
            assert np.array_equal(vg[pre], v_act[pre]), f"{name} layer {layer}: V fetch"
            assert np.all(kg[~pre] == 0xFFFF) and np.all(vg[~pre] == 0xFFFF)
            sc.sc_append_new_kv(dp.handle, dp.table, knd.data_ptr(), vnd.data_ptr(), act, stream)
            torch.cuda.synchronize()
            kg, vg = to_u16(k), to_u16(v)
            assert np.array_equal(kg[~rcr], k_full[~rcr]), f"{name} layer {layer}: K append"
            assert np.array_equal(vg[~rcr], v_full[~rcr]), f"{name} layer {layer}: V append"
            assert np.all(kg[rcr] == 0xFFFF) and np.all(vg[rcr] == 0xFFFF)

            out = torch.full((wl.total_q, wl.n_q_heads, wl.head_dim), float("nan"),
                             dtype=W.torch_dtype(wl), device="cuda")
            lse = torch.full((wl.n_q_heads, max(1, wl.total_q)), float("nan"), device="cuda")
            sc.sc_prefill_attn_varlen(dp.handle, dp.table, layer, qd.data_ptr(), act, wl.n_q_heads,
                                      out.data_ptr(), lse.data_ptr(), 0.0, stream)
            torch.cuda.synchronize()
            compare_attention(to_u16(out), o_ref, f"{name} layer {layer} varlen", wl.dtype)
            lse_g = lse.cpu().numpy().astype(np.float64)[:, :wl.total_q]
            # The kernel's denominator sums the probabilities in fp32
            # (head_dim 128) or rounded to the element type (head_dim 64:
            # the weights that multiply V, each within 2^-9 (bf16) or 2^-11
            # (fp16) relative of its exact value), so ln l is off by at most
            # about 2^-9 plus fp32 accumulation: 2^-8 bounds it.
            np.testing.assert_allclose(lse_g, lse_ref, atol=2.0 ** -8, rtol=1e-4)
            if wl.batch == 1 and not wl.n_rc_blocks:
                out1 = torch.empty_like(out)
                lse1 = torch.empty_like(lse)
                single = sc.sc_prefill_attn if wl.dtype == "bf16" else sc.sc_prefill_attn_f16
                single(qd.data_ptr(), k.data_ptr(), v.data_ptr(), int(wl.prefix_len[0]),
                       int(wl.new_len[0]), wl.n_q_heads, wl.n_kv_heads, wl.head_dim,
                       out1.data_ptr(), lse1.data_ptr(), 0.0, stream)
                torch.cuda.synchronize()
                assert torch.equal(out1.view(torch.int16), out.view(torch.int16))
    finally:
        dp.close()


@pytest.mark.parametrize("name", ["cfg1", "host_tier", "varlen_batch", "rc_host", "f16_host"])
def test_store_matches_oracle(name):
    sc = require_gpu()
    import torch
    wl = _case(name)
    pool_u16 = W.pool_numpy(wl)
    dp = DevicePool(sc, wl, pool_u16)
    stream = torch.cuda.current_stream().cuda_stream
    try:
        expect = pool_u16
        for layer in range(wl.n_layers):
            _, kn, vn = W.layer_inputs_numpy(wl, layer)
            knd, vnd = from_u16(kn, "cuda", wl.dtype), from_u16(vn, "cuda", wl.dtype)
            sc.sc_store_layer_kv(dp.handle, dp.table, layer, knd.data_ptr(), vnd.data_ptr(), stream)
            torch.cuda.synchronize()
            expect = ok.store_layer(expect, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len,
                                    layer, kn, vn)
        assert np.array_equal(dp.full_u16(), expect)
        # next turn: the whole history is the prefix; fetch returns prefix + new bit-exactly
        wl2 = W.Workload(**{**wl.__dict__, "prefix_len": wl.prefix_len + wl.new_len,
                            "new_len": np.zeros_like(wl.new_len)})
        t2 = sc.sc_table_create(dp.handle, wl2.block_ids, wl2.cu_blocks, wl2.prefix_len, wl2.new_len,
                                stream)
        try:
            for layer in range(wl.n_layers):
                k, v, act = new_active(sc, wl2)
                sc.sc_fetch_layer_kv(dp.handle, t2, layer, act, stream)
                torch.cuda.synchronize()
                kr, vr = ok.gather_layer(expect, wl2.block_ids, wl2.cu_blocks, wl2.prefix_len,
                                         wl2.new_len, layer)
                f = ~_rc_rows(wl2)
                assert np.array_equal(to_u16(k)[f], kr[f]) and np.array_equal(to_u16(v)[f], vr[f])
        finally:
            sc.sc_table_destroy(t2)
    finally:
        dp.close()


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_single_visible_key_returns_its_value_row_exactly(dtype):
    sc = require_gpu()
    import torch
    rng = np.random.default_rng(5)
    single = sc.sc_prefill_attn if dtype == "bf16" else sc.sc_prefill_attn_f16
    for hq, hkv, d in [(8, 8, 64), (32, 8, 128), (40, 8, 128)]:
        n = 37
        q = W.normal_bits(rng, (n, hq, d), dtype)
        k = W.normal_bits(rng, (n, hkv, d), dtype)
        v = W.normal_bits(rng, (n, hkv, d), dtype)
        qd, kd, vd = (from_u16(x, "cuda", dtype) for x in (q, k, v))
        out = torch.empty((n, hq, d), dtype=qd.dtype, device="cuda")
        single(qd.data_ptr(), kd.data_ptr(), vd.data_ptr(), 0, n, hq, hkv, d, out.data_ptr(),
               0, 0.0, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        o = to_u16(out)
        g = hq // hkv
        for h in range(hq):
            assert np.array_equal(o[0, h], v[0, h // g]), (hq, hkv, d, h)


@pytest.mark.parametrize("mode", ["overlap", "serial", "overlap-poison", "overlap-event", "overlap-event-poison"])
@pytest.mark.parametrize("name", ["stack_g4", "stack_varlen_host", "stack_rc", "stack_f16_rc"])
def test_layer_stack_matches_oracle(name, mode):
    """The whole layer stack against the oracle, layer by layer, and the pool
    after every store.  "overlap-poison" overwrites each slot with NaN
    patterns before it is refilled, so an attention that ran ahead of its
    slot's fetch and append would leave NaN rows.  The "event" modes order
    the two streams with stream events instead of device-side waits (the
    path taken when dispatches are serialised)."""
    sc = require_gpu()
    import torch
    if name == "stack_g4":
        wl = W.small_workload(201, [300], [70], 4, 32, 8, 128)
    elif name == "stack_varlen_host":
        wl = W.small_workload(202, [150, 0, 500], [20, 40, 7], 3, 8, 2, 64, host_fraction=0.5)
    elif name == "stack_rc":
        wl = W.small_workload(203, [300, 700, 40], [70, 9, 33], 3, 32, 8, 128, host_fraction=0.3,
                              rc_fraction=0.5)
    else:
        wl = W.small_workload(204, [400, 64], [50, 100], 3, 32, 8, 128, rc_fraction=0.5, dtype="f16")
    pool_u16 = W.pool_numpy(wl)
    dp = DevicePool(sc, wl, pool_u16)
    try:
        ins = [W.layer_inputs_numpy(wl, l) for l in range(wl.n_layers)]
        dev = [[from_u16(x, "cuda", wl.dtype) for x in t] for t in ins]
        outs = [torch.full((wl.total_q, wl.n_q_heads, wl.head_dim), float("nan"), dtype=W.torch_dtype(wl),
                           device="cuda") for _ in range(wl.n_layers)]
        slots = [new_active(sc, wl) for _ in range(2)]
        copy = torch.cuda.Stream()
        flags = {"overlap": sc.SC_STACK_OVERLAP, "serial": sc.SC_STACK_SERIAL,
                 "overlap-poison": sc.SC_STACK_OVERLAP | sc.SC_STACK_DEBUG_POISON,
                 "overlap-event": sc.SC_STACK_OVERLAP | sc.SC_STACK_EVENT_WAIT,
                 "overlap-event-poison": sc.SC_STACK_OVERLAP | sc.SC_STACK_EVENT_WAIT | sc.SC_STACK_DEBUG_POISON,
                 }[mode]
        sc.sc_prefill_stack(dp.handle, dp.table, [d[0].data_ptr() for d in dev],
                            [d[1].data_ptr() for d in dev], [d[2].data_ptr() for d in dev],
                            [o.data_ptr() for o in outs], [s[2] for s in slots], wl.n_q_heads, flags,
                            0.0, torch.cuda.current_stream().cuda_stream, copy.cuda_stream)
        torch.cuda.synchronize()
        expect = pool_u16
        for l in range(wl.n_layers):
            q, kn, vn = ins[l]
            *_, o_ref, _ = _oracle_layer(wl, pool_u16, l, q, kn, vn)
            compare_attention(to_u16(outs[l]), o_ref, f"{name} {mode} layer {l}", wl.dtype)
            expect = ok.store_layer(expect, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, l, kn, vn)
        assert np.array_equal(dp.full_u16(), expect)
    finally:
        dp.close()


# Stacks whose plans split keys: each layer's split partials are merged by
# the next layer's forward kernel (claimed in chunks by the workgroups that
# finish first), the last layer's by a merge kernel.  (P, N, Hq, Hkv, D,
# layers, which merge path: at most four splits per row -> four rows per
# lane group, more -> one.)
DEFERRED = {
    "nr4_multi_seq": ([2500, 800, 3000], [200, 100, 250], 32, 8, 128, 3, "le4"),
    "nr1_multi_seq": ([3000, 5000, 1200], [40, 25, 60], 32, 8, 128, 2, "gt4"),
    "one_layer": ([1500], [500], 32, 8, 128, 1, "le4"),
    "d64_nr4": ([2000, 1500], [300, 200], 32, 8, 64, 2, "le4"),
    "d64_nr1": ([3000, 1000], [300, 150], 16, 4, 64, 2, "gt4"),
}


@pytest.mark.parametrize("mode", ["overlap", "serial"])
@pytest.mark.parametrize("name", list(DEFERRED))
def test_stack_deferred_merge_matches_oracle(name, mode):
    """Every layer of a stack with key splits against the oracle: the
    deferred merges (one, several and no sequences split per plan, at most
    and more than four splits per row, head_dim 64 and 128, a single
    layer)."""
    sc = require_gpu()
    import torch
    P, N, hq, hkv, D, L, path = DEFERRED[name]
    _, splits = sc.sc_attn_plan_query(P, N, hq, hkv)
    assert (max(splits) <= 4) == (path == "le4") and max(splits) > 1, splits
    wl = W.small_workload(250 + list(DEFERRED).index(name), P, N, L, hq, hkv, D)
    pool_u16 = W.pool_numpy(wl)
    dp = DevicePool(sc, wl, pool_u16)
    try:
        ins = [W.layer_inputs_numpy(wl, l) for l in range(L)]
        dev = [[from_u16(x, "cuda", wl.dtype) for x in t] for t in ins]
        outs = [torch.full((wl.total_q, hq, D), float("nan"), dtype=W.torch_dtype(wl), device="cuda")
                for _ in range(L)]
        slots = [new_active(sc, wl) for _ in range(2)]
        copy = torch.cuda.Stream()
        flags = sc.SC_STACK_OVERLAP if mode == "overlap" else sc.SC_STACK_SERIAL
        sc.sc_prefill_stack(dp.handle, dp.table, [d[0].data_ptr() for d in dev], [d[1].data_ptr() for d in dev],
                            [d[2].data_ptr() for d in dev], [o.data_ptr() for o in outs], [s[2] for s in slots], hq,
                            flags, 0.0, torch.cuda.current_stream().cuda_stream, copy.cuda_stream)
        torch.cuda.synchronize()
        for l in range(L):
            q, kn, vn = ins[l]
            *_, o_ref, _ = _oracle_layer(wl, pool_u16, l, q, kn, vn)
            compare_attention(to_u16(outs[l]), o_ref, f"{name} {mode} layer {l}", wl.dtype)
    finally:
        dp.close()


def test_overlapped_stacks_on_one_table_from_two_streams():
    """Two overlapped stacks on the same table, enqueued back to back on two
    different caller streams with their own slots and outputs: they share
    the table's slot counter, so the library runs them one after the other;
    both must match the oracle."""
    sc = require_gpu()
    import torch
    wl = W.small_workload(206, [700, 45], [90, 30], 4, 32, 8, 128)
    pool_u16 = W.pool_numpy(wl)
    dp = DevicePool(sc, wl, pool_u16)
    try:
        ins = [W.layer_inputs_numpy(wl, l) for l in range(wl.n_layers)]
        dev = [[from_u16(x, "cuda", wl.dtype) for x in t] for t in ins]
        runs = []
        for _ in range(2):
            outs = [torch.full((wl.total_q, wl.n_q_heads, wl.head_dim), float("nan"), dtype=W.torch_dtype(wl),
                               device="cuda") for _ in range(wl.n_layers)]
            runs.append((outs, [new_active(sc, wl) for _ in range(2)], torch.cuda.Stream(), torch.cuda.Stream()))
        torch.cuda.synchronize()
        for outs, slots, cs, xs in runs:
            sc.sc_prefill_stack(dp.handle, dp.table, [d[0].data_ptr() for d in dev],
                                [d[1].data_ptr() for d in dev], [d[2].data_ptr() for d in dev],
                                [o.data_ptr() for o in outs], [s[2] for s in slots], wl.n_q_heads,
                                sc.SC_STACK_OVERLAP | sc.SC_STACK_NO_STORE, 0.0, cs.cuda_stream, xs.cuda_stream)
        torch.cuda.synchronize()
        assert not sc.sc_table_stack_status(dp.table)
        for r, (outs, *_) in enumerate(runs):
            for l in range(wl.n_layers):
                q, kn, vn = ins[l]
                *_, o_ref, _ = _oracle_layer(wl, pool_u16, l, q, kn, vn)
                compare_attention(to_u16(outs[l]), o_ref, f"stack {r} layer {l}", wl.dtype)
    finally:
        dp.close()


@pytest.mark.parametrize("which", ["ready", "free"])
def test_forced_slot_wait_timeout_is_reported_and_recoverable(which):
    """The failure paths of the overlapped stack's device-side slot waits,
    forced from the host.  SC_STACK_TEST_NEVER_READY: every attention kernel
    waits for a slot count the copy stream never reaches, gives up after a
    few hundred polls and writes NaN rows.  SC_STACK_TEST_NEVER_FREE: every
    copy into a slot (layers 2 and 3) waits for attention workgroups that
    never all finish, gives up and fills the slot with NaN, so those layers'
    rows are NaN.  Either way every kernel exits, the table reports the
    time-out, and after clearing the flag a normal stack on the same table
    is correct again."""
    sc = require_gpu()
    import torch
    flag = sc.SC_STACK_TEST_NEVER_READY if which == "ready" else sc.SC_STACK_TEST_NEVER_FREE
    first_nan = 0 if which == "ready" else 2
    wl = W.small_workload(205, [300, 41], [70, 9], 4, 32, 8, 128)
    pool_u16 = W.pool_numpy(wl)
    dp = DevicePool(sc, wl, pool_u16)
    try:
        ins = [W.layer_inputs_numpy(wl, l) for l in range(wl.n_layers)]
        dev = [[from_u16(x, "cuda", wl.dtype) for x in t] for t in ins]
        outs = [torch.zeros((wl.total_q, wl.n_q_heads, wl.head_dim), dtype=W.torch_dtype(wl), device="cuda")
                for _ in range(wl.n_layers)]
        slots = [new_active(sc, wl) for _ in range(2)]
        copy = torch.cuda.Stream()
        cs = torch.cuda.current_stream().cuda_stream

        def run(flags):
            sc.sc_prefill_stack(dp.handle, dp.table, [d[0].data_ptr() for d in dev],
                                [d[1].data_ptr() for d in dev], [d[2].data_ptr() for d in dev],
                                [o.data_ptr() for o in outs], [s[2] for s in slots], wl.n_q_heads,
                                flags, 0.0, cs, copy.cuda_stream)
            torch.cuda.synchronize()

        assert not sc.sc_table_stack_status(dp.table)
        run(sc.SC_STACK_OVERLAP | sc.SC_STACK_NO_STORE | flag)
        for l in range(first_nan, wl.n_layers):
            assert bool(torch.isnan(outs[l].float()).all()), f"layer {l}: rows written despite the time-out"
        assert sc.sc_table_stack_status(dp.table, clear=True)
        assert not sc.sc_table_stack_status(dp.table)
        run(sc.SC_STACK_OVERLAP | sc.SC_STACK_NO_STORE)
        assert not sc.sc_table_stack_status(dp.table)
        for l in range(wl.n_layers):
            q, kn, vn = ins[l]
            *_, o_ref, _ = _oracle_layer(wl, pool_u16, l, q, kn, vn)
            compare_attention(to_u16(outs[l]), o_ref, f"after recovery, layer {l}", wl.dtype)
        with pytest.raises(sc.SwiftCacheError):
            run(sc.SC_STACK_SERIAL | flag)
        with pytest.raises(sc.SwiftCacheError) as e:       # event waits have no device wait to time out
            run(sc.SC_STACK_OVERLAP | sc.SC_STACK_EVENT_WAIT | flag)
        assert e.value.status == sc.SC_ERR_UNSUPPORTED
    finally:
        dp.close()


def test_stack_under_serialised_dispatch_uses_event_waits():
    """With AMD_SERIALIZE_KERNEL set (each kernel waits for the previous
    one, as under counter collection), a device-side slot wait could only
    time out; the library then orders the streams with events.  A child
    process runs an overlapped stack in that environment and compares every
    layer with the oracle; it must report no time-out."""
    require_gpu()
    import json
    import os
    import subprocess
    import sys
    env = dict(os.environ, AMD_SERIALIZE_KERNEL="3")
    child = os.path.join(os.path.dirname(__file__), "_stack_child.py")
    print("[serialised] child stack with AMD_SERIALIZE_KERNEL=3", flush=True)
    r = subprocess.run([sys.executable, "-u", child], env=env, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    res = json.loads(r.stdout.strip().splitlines()[-1])
    assert res["device_wait"] is False, res
    assert res["timed_out"] is False and res["layers_ok"] == res["layers"], res


def test_stack_wait_kind():
    """Without a serialising environment an overlapped stack at head_dim 128
    waits on the device; SC_STACK_EVENT_WAIT and the other modes do not."""
    sc = require_gpu()
    wl = W.small_workload(207, [100], [20], 1, 32, 8, 128)
    dp = DevicePool(sc, wl, W.pool_numpy(wl))
    try:
        assert sc.sc_stack_wait_kind(dp.table, sc.SC_STACK_OVERLAP)
        assert not sc.sc_stack_wait_kind(dp.table, sc.SC_STACK_OVERLAP | sc.SC_STACK_EVENT_WAIT)
        assert not sc.sc_stack_wait_kind(dp.table, sc.SC_STACK_SERIAL)
        assert not sc.sc_stack_wait_kind(dp.table, sc.SC_STACK_ATTN_ONLY)
    finally:
        dp.close()


@pytest.mark.parametrize("name,chunk,mode", [
    ("g4_d128_ragged", 16, "overlap"), ("g4_d128_ragged", 100, "serial"), ("g4_d128_ragged", 1000, "overlap"),
    ("varlen_batch", 48, "overlap"), ("varlen_empty_turn", 7, "overlap"), ("rc_varlen", 64, "overlap"),
    ("f16_g5_split_rc", 9, "overlap"), ("host_tier", 13, "overlap"), ("g1_d64_P0", 33, "serial"),
])
def test_chunked_stack_matches_oracle(name, chunk, mode):
    """The new turn in chunks over one fetched slot per layer: every output
    row against the oracle's (unchunked) attention, and the pool after the
    stores byte for byte."""
    sc = require_gpu()
    import torch
    wl = _case(name)
    pool_u16 = W.pool_numpy(wl)
    dp = DevicePool(sc, wl, pool_u16)
    try:
        ins = [W.layer_inputs_numpy(wl, l, q_scale=8.0) for l in range(wl.n_layers)]
        dev = [[from_u16(x, "cuda", wl.dtype) for x in t] for t in ins]
        outs = [torch.full((wl.total_q, wl.n_q_heads, wl.head_dim), float("nan"), dtype=W.torch_dtype(wl),
                           device="cuda") for _ in range(wl.n_layers)]
        slots = [new_active(sc, wl) for _ in range(2)]
        copy = torch.cuda.Stream()
        flags = {"overlap": sc.SC_STACK_OVERLAP, "serial": sc.SC_STACK_SERIAL,
                 "overlap-poison": sc.SC_STACK_OVERLAP | sc.SC_STACK_DEBUG_POISON}[mode]
        print(f"\n[chunked] {name} chunk {chunk} {mode}", flush=True)
        sc.sc_prefill_stack_chunked(dp.handle, dp.table, [d[0].data_ptr() for d in dev],
                                    [d[1].data_ptr() for d in dev], [d[2].data_ptr() for d in dev],
                                    [o.data_ptr() for o in outs], [s[2] for s in slots], wl.n_q_heads, chunk,
                                    flags, 0.0, torch.cuda.current_stream().cuda_stream, copy.cuda_stream)
        torch.cuda.synchronize()
        expect = pool_u16
        for l in range(wl.n_layers):
            q, kn, vn = ins[l]
            *_, o_ref, _ = _oracle_layer(wl, pool_u16, l, q, kn, vn)
            compare_attention(to_u16(outs[l]), o_ref, f"{name} chunk {chunk} layer {l}", wl.dtype)
            expect = ok.store_layer(expect, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, l, kn, vn)
        assert np.array_equal(dp.full_u16(), expect)
    finally:
        dp.close()


@pytest.mark.parametrize("name", ["host_tier", "rc_host", "f16_host"])
def test_dma_fetch_matches_oracle(name):
    """The KV Load with the host tier moved by the DMA engines (one
    host-to-device copy per block half and layer): the same bytes as the
    fetch kernel, prefix rows outside the regular cache bit-exact and every
    other row untouched; the batched-copy variant either gives the same
    bytes or reports that the runtime lacks it.  The table's totals match
    the workload."""
    sc = require_gpu()
    import torch
    wl = _case(name)
    pool_u16 = W.pool_numpy(wl)
    dp = DevicePool(sc, wl, pool_u16)
    stream = torch.cuda.current_stream().cuda_stream
    try:
        assert sc.sc_table_totals(dp.table) == (wl.total_q, wl.total_kv)
        pre = _prefix_rows(wl) & ~_rc_rows(wl)
        for layer in range(wl.n_layers):
            k_act, v_act = ok.gather_layer(pool_u16, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, layer)
            for per_copy in (True, False):
                k, v, act = new_active(sc, wl, fill_bits=0xFFFF)
                try:
                    sc.sc_fetch_layer_kv_dma(dp.handle, dp.table, layer, act, per_copy_calls=per_copy, stream=stream)
                except sc.SwiftCacheError as e:
                    assert not per_copy and e.status == sc.SC_ERR_UNSUPPORTED, e
                    continue
                torch.cuda.synchronize()
                kg, vg = to_u16(k), to_u16(v)
                what = f"{name} layer {layer} per_copy={per_copy}"
                assert np.array_equal(kg[pre], k_act[pre]), f"{what}: K"
                assert np.array_equal(vg[pre], v_act[pre]), f"{what}: V"
                assert np.all(kg[~pre] == 0xFFFF) and np.all(vg[~pre] == 0xFFFF), what
    finally:
        dp.close()


def test_sequence_beyond_32_bit_key_offsets_is_rejected():
    """2^21 keys x 8 KV heads x 128 dims x 2 bytes = 4 GiB per sequence: the
    kernel's 32-bit offsets cannot address it, so the call fails before
    any launch (the buffers are never touched)."""
    sc = require_gpu()
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn(16, 16, 16, 1 << 21, 1, 32, 8, 128, 16)
    assert e.value.status == sc.SC_ERR_UNSUPPORTED


def test_longest_accepted_sequence_matches_oracle():
    """The longest sequence the kernel's signed 32-bit key offsets admit at
    8 KV heads x 128 dims: 2 GiB of keys less 256 tokens (2^20 - 257
    tokens), whose last tiles and the loads past them sit just below 2^31
    bytes.  With 4096 new tokens the plan does not split keys, so each work
    item addresses the whole key range from one base.  Sampled rows (first,
    middle and last new token of a head in the first and the last KV group)
    against the oracle, lse included; one more token is refused before any
    launch."""
    sc = require_gpu()
    import torch
    hq, hkv, d, n = 32, 8, 128, 4096
    tokens = (1 << 31) // (hkv * d * 2) - 256 - 1
    p = tokens - n
    items, splits = sc.sc_attn_plan_query([p], [n], hq, hkv)
    assert splits[0] == 1 and all(it[4] == 0 for it in items) and any(it[5] == tokens for it in items)
    q, k, v = W.long_sequence_torch(301, p, n, hq, hkv, d, "cuda")
    out = torch.full((n, hq, d), float("nan"), dtype=torch.bfloat16, device="cuda")
    lse = torch.full((hq, n), float("nan"), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    print(f"[longest] P={p} N={n} heads {hq}/{hkv} D={d}", flush=True)
    sc.sc_prefill_attn(q.data_ptr(), k.data_ptr(), v.data_ptr(), p, n, hq, hkv, d, out.data_ptr(),
                       lse=lse.data_ptr(), stream=stream)
    torch.cuda.synchronize()
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn(q.data_ptr(), k.data_ptr(), v.data_ptr(), p + 1, n, hq, hkv, d, out.data_ptr(),
                           stream=stream)
    assert e.value.status == sc.SC_ERR_UNSUPPORTED
    o_bits = to_u16(out)
    lse_h = lse.cpu().numpy()
    group = hq // hkv
    for h in (0, hq - 1):
        g = h // group
        # One KV head's keys and values, as a one-head problem for the oracle.
        kg = bits_to_f64(to_u16(k[:, g:g + 1]))
        vg = bits_to_f64(to_u16(v[:, g:g + 1]))
        qh = bits_to_f64(to_u16(q[:, h:h + 1]))
        rows = [(0, i, 0) for i in (0, n // 2, n - 1)]
        o_ref, l_ref = oa.attention_rows(qh, kg, vg, [p], [n], rows)
        for r, (_, i, _) in enumerate(rows):
            compare_attention(o_bits[i, h][None, :], o_ref[r][None, :], f"longest row {i} head {h}")
            assert abs(lse_h[h, i] - l_ref[r]) <= 2.0 ** -8 + 1e-4 * abs(l_ref[r]), (h, i, lse_h[h, i], l_ref[r])
        del kg, vg


def test_capacity_and_layer_errors():
    sc = require_gpu()
    wl = W.config(1)
    dp = DevicePool(sc, wl, W.pool_numpy(wl))
    try:
        import torch
        k = torch.empty((wl.total_kv - 1, wl.n_kv_heads, wl.head_dim), dtype=torch.bfloat16, device="cuda")
        act = sc.active(k.data_ptr(), k.data_ptr(), wl.total_kv - 1)
        with pytest.raises(sc.SwiftCacheError) as e:
            sc.sc_fetch_layer_kv(dp.handle, dp.table, 0, act)
        assert e.value.status == sc.SC_ERR_RANGE
        act = sc.active(k.data_ptr(), k.data_ptr(), wl.total_kv)
        with pytest.raises(sc.SwiftCacheError) as e:
            sc.sc_fetch_layer_kv(dp.handle, dp.table, 1, act)
        assert e.value.status == sc.SC_ERR_RANGE
        with pytest.raises(sc.SwiftCacheError) as e:
            sc.sc_prefill_attn_varlen(dp.handle, dp.table, 1, k.data_ptr(), act, wl.n_q_heads, k.data_ptr())
        assert e.value.status == sc.SC_ERR_RANGE
    finally:
        dp.close()
