"""Child process of test_stack_under_serialised_dispatch_uses_event_waits:
runs one overlapped layer stack in the environment it was started with and
prints one JSON line (layers, layers matching the oracle, time-out flag).
Not a test module itself."""

import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

import numpy as np  # noqa: E402
import torch  # noqa: E402

from oracle import attention as oa  # noqa: E402
from oracle import kvcache as ok  # noqa: E402
from paper_2606_16135_amd import swiftcache as sc  # noqa: E402
from paper_2606_16135_amd import workloads as W  # noqa: E402
from _gpu_util import DevicePool, compare_attention, from_u16, new_active, to_u16  # noqa: E402


def main():
    sc.load()
    wl = W.small_workload(206, [300, 41], [70, 9], 4, 32, 8, 128)
    pool_u16 = W.pool_numpy(wl)
    dp = DevicePool(sc, wl, pool_u16)
    try:
        ins = [W.layer_inputs_numpy(wl, l) for l in range(wl.n_layers)]
        dev = [[from_u16(x, "cuda", wl.dtype) for x in t] for t in ins]
        outs = [torch.full((wl.total_q, wl.n_q_heads, wl.head_dim), float("nan"), dtype=W.torch_dtype(wl),
                           device="cuda") for _ in range(wl.n_layers)]
        slots = [new_active(sc, wl) for _ in range(2)]
        copy = torch.cuda.Stream()
        device_wait = sc.sc_stack_wait_kind(dp.table, sc.SC_STACK_OVERLAP)
        sc.sc_prefill_stack(dp.handle, dp.table, [d[0].data_ptr() for d in dev],
                            [d[1].data_ptr() for d in dev], [d[2].data_ptr() for d in dev],
                            [o.data_ptr() for o in outs], [s[2] for s in slots], wl.n_q_heads,
                            sc.SC_STACK_OVERLAP | sc.SC_STACK_DEBUG_POISON, 0.0,
                            torch.cuda.current_stream().cuda_stream, copy.cuda_stream)
        torch.cuda.synchronize()
        timed_out = bool(sc.sc_table_stack_status(dp.table))
        ok_layers = 0
        for l in range(wl.n_layers):
            q, kn, vn = ins[l]
            k_act, v_act = ok.gather_layer(pool_u16, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, l)
            k_full, v_full = ok.append_new(k_act, v_act, kn, vn, wl.prefix_len, wl.new_len)
            o_ref, _ = oa.attention(oa.bits_to_f64(q, wl.dtype), oa.bits_to_f64(k_full, wl.dtype),
                                    oa.bits_to_f64(v_full, wl.dtype), wl.prefix_len, wl.new_len)
            try:
                compare_attention(to_u16(outs[l]), o_ref, f"layer {l}", wl.dtype)
                ok_layers += 1
            except AssertionError as e:
                print(f"layer {l}: {e}", file=sys.stderr, flush=True)
        print(json.dumps({"layers": wl.n_layers, "layers_ok": ok_layers, "timed_out": timed_out,
                          "device_wait": device_wait}), flush=True)
    finally:
        dp.close()


if __name__ == "__main__":
    main()
