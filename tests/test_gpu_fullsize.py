"""GPU parity at the five benchmark shapes (two of them also with half of each
sequence's full prefix blocks in the regular cache, the 8B shape also with
fp16 values and with peaky queries), in the launch configuration the
benchmark times: the whole layer stack runs once through sc_prefill_stack
(overlapped mode, two active slots, every layer fetched, appended, attended
and stored), on the same seeded device-generated pool and inputs.  Two more
runs (8B and varlen shapes) add SC_STACK_DEBUG_POISON: every slot is
overwritten with NaN patterns before it is refilled, so an attention that
ran ahead of its slot's fetch and append would leave NaN rows.

Checked layers: every layer of the 8B and varlen shapes' plain runs,
layers {0, L/2, L-2, L-1} otherwise, and the fetch alone on every other layer (fetched
again after the stack and compared byte for byte with the oracle's gather
of the pool, whose prefix rows the store never writes).  On each checked
layer, against the oracle (which works from a host snapshot of the layer
taken before the stack ran):

* fetch + append: every byte of the active layer (all tokens, all KV heads)
  outside the regular-cache rows, which are never copied.  The two slots
  that survive the stack (layers L-2 and L-1, filled by the stack's own
  copy kernel) are compared as the stack left them; every other checked
  layer is fetched again into a spare slot after the stack (prefix rows
  are not touched by the store, so the snapshot still defines them);
* attention: every element (all rows, all heads) of the stack's own output,
  computed by the oracle's dense attention, to
  |gpu - oracle| <= 2e-2 + 1e-2 |oracle| plus the relative-L2 bound;
* store: every byte of every block the table references, after the stack,
  against the oracle's store applied to the snapshot.
"""

import time

import numpy as np
import pytest

from oracle import kvcache as ok
from paper_2606_16135_amd import workloads as W

from _gpu_util import compare_attention, oracle_attention_by_head, require_gpu, to_u16

pytestmark = pytest.mark.gpu


def _sub_pool(dp, layer, ids):
    """Layer `layer` of the referenced blocks only, in table order."""
    return dp.ref_layer_u16(layer, ids)


# cfg, regular-cache fraction, element type, debug poison, q scale, layers checked
CASES = {
    "2": (2, 0.0, "bf16", False, 1.0, "all"),
    "3": (3, 0.0, "bf16", False, 1.0, "all"),
    "4": (4, 0.0, "bf16", False, 1.0, "ends"),
    "5": (5, 0.0, "bf16", False, 1.0, "ends"),
    "2-peaky": (2, 0.0, "bf16", False, 8.0, "ends"),
    "2-rc0.5": (2, 0.5, "bf16", False, 1.0, "ends"),
    "3-rc0.5": (3, 0.5, "bf16", False, 1.0, "ends"),
    "2-f16": (2, 0.0, "f16", False, 1.0, "ends"),
    "2-poison": (2, 0.0, "bf16", True, 1.0, "ends"),
    "3-poison": (3, 0.0, "bf16", True, 1.0, "ends"),
}


@pytest.mark.timeout(600)
@pytest.mark.parametrize("case", list(CASES))
def test_benchmark_shape_stack_matches_oracle(case):
    cfg, rc, dtype, poison, q_scale, which = CASES[case]
    sc = require_gpu()
    import torch
    from paper_2606_16135_amd.torch_pool import DevicePool

    wl = W.config(cfg, rc_fraction=rc, dtype=dtype)
    rc_rows = ok.regular_cache_rows(wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, wl.block_size,
                                    wl.rc_first_id)
    L = wl.n_layers
    check_layers = list(range(L)) if which == "all" else sorted({0, L // 2, max(0, L - 2), L - 1})
    print(f"\n[fullsize] {case} {wl.name}: L={L} total_q={wl.total_q} total_kv={wl.total_kv} "
          f"q_scale={q_scale} layers {check_layers if which != 'all' else 'all'}", flush=True)
    dp = DevicePool(sc, wl, fill="torch")
    try:
        ids = np.asarray(wl.block_ids, dtype=np.int64)
        local_ids = np.arange(len(ids), dtype=np.int32)      # table order in the snapshot
        snap = {l: _sub_pool(dp, l, ids) for l in check_layers}

        inputs = [W.layer_inputs_torch(wl, l, "cuda", q_scale=q_scale) for l in range(L)]
        td = W.torch_dtype(wl)
        outs = [torch.empty((wl.total_q, wl.n_q_heads, wl.head_dim), dtype=td, device="cuda")
                for _ in range(L)]
        slot_t = [(torch.empty((wl.total_kv, wl.n_kv_heads, wl.head_dim), dtype=td, device="cuda"),
                   torch.empty((wl.total_kv, wl.n_kv_heads, wl.head_dim), dtype=td, device="cuda"))
                  for _ in range(3)]
        slots = [sc.active(k.data_ptr(), v.data_ptr(), wl.total_kv) for k, v in slot_t]
        compute = torch.cuda.current_stream()
        copy = torch.cuda.Stream()
        sc.sc_prefill_stack(dp.handle, dp.table, [i[0].data_ptr() for i in inputs],
                            [i[1].data_ptr() for i in inputs], [i[2].data_ptr() for i in inputs],
                            [o.data_ptr() for o in outs], slots[:2], wl.n_q_heads,
                            sc.SC_STACK_OVERLAP | (sc.SC_STACK_DEBUG_POISON if poison else 0), 0.0,
                            compute.cuda_stream, copy.cuda_stream)
        torch.cuda.synchronize()
        print(f"[fullsize] {case}: stack done", flush=True)
        # The slots the stack itself filled last: layer L-1 in slot (L-1) & 1,
        # layer L-2 in the other one.
        survivors = {L - 1: (L - 1) & 1, L - 2: (L - 2) & 1} if L >= 2 else {0: 0}

        f = ~rc_rows                       # regular-cache rows are read in place, never copied
        for l in check_layers:
            t0 = time.perf_counter()
            q, kn, vn = (to_u16(t) for t in inputs[l])
            k_act, v_act = ok.gather_layer(snap[l], local_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, 0)
            k_full, v_full = ok.append_new(k_act, v_act, kn, vn, wl.prefix_len, wl.new_len)

            # fetch + append, every byte
            if l in survivors:
                s = survivors[l]
                kg, vg = to_u16(slot_t[s][0]), to_u16(slot_t[s][1])
                src = f"stack slot {s}"
            else:
                sc.sc_fetch_layer_kv(dp.handle, dp.table, l, slots[2], compute.cuda_stream)
                sc.sc_append_new_kv(dp.handle, dp.table, inputs[l][1].data_ptr(), inputs[l][2].data_ptr(),
                                    slots[2], compute.cuda_stream)
                torch.cuda.synchronize()
                kg, vg = to_u16(slot_t[2][0]), to_u16(slot_t[2][1])
                src = "refetch"
            assert np.array_equal(kg[f], k_full[f]), f"{case} layer {l}: K fetch/append ({src})"
            assert np.array_equal(vg[f], v_full[f]), f"{case} layer {l}: V fetch/append ({src})"

            # attention, every element of the stack's own output
            o_ref = oracle_attention_by_head(q, k_full, v_full, wl.prefix_len, wl.new_len, dtype)
            stats = compare_attention(to_u16(outs[l]), o_ref, f"{case} layer {l}", dtype)

            # store: every referenced block of this layer
            expect = ok.store_layer(snap[l], local_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, 0, kn, vn)
            after = _sub_pool(dp, l, ids)
            assert np.array_equal(after, expect), f"{case} layer {l}: store"
            print(f"[fullsize] {case} layer {l}: fetch/append ({src}) and store exact, attention on all "
                  f"{o_ref.shape[0] * o_ref.shape[1]} rows {stats} ({time.perf_counter() - t0:.1f} s)", flush=True)

        # fetch of every other layer, byte for byte: the store never writes
        # prefix rows, so the pool after the stack still defines them
        _, cu_k = ok.seq_offsets(wl.prefix_len, wl.new_len)
        pre = np.zeros(wl.total_kv, dtype=bool)
        for b, p in enumerate(wl.prefix_len):
            pre[cu_k[b]:cu_k[b] + p] = True
        pre &= f
        rest = [l for l in range(L) if l not in check_layers]
        t0 = time.perf_counter()
        for l in rest:
            sub = dp.ref_layer_u16(l, ids)
            k_act, v_act = ok.gather_layer(sub, local_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, 0)
            sc.sc_fetch_layer_kv(dp.handle, dp.table, l, slots[2], compute.cuda_stream)
            torch.cuda.synchronize()
            kg, vg = to_u16(slot_t[2][0]), to_u16(slot_t[2][1])
            assert np.array_equal(kg[pre], k_act[pre]), f"{case} layer {l}: K fetch"
            assert np.array_equal(vg[pre], v_act[pre]), f"{case} layer {l}: V fetch"
        if rest:
            print(f"[fullsize] {case}: fetch exact on the other {len(rest)} layers "
                  f"({time.perf_counter() - t0:.1f} s)", flush=True)
    finally:
        dp.close()
