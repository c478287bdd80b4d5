"""Attention calls from several host threads on one shared stream.

The split-key workspace is one grow-only buffer per (device, stream).  A
call holds that buffer's lock from the lookup until its forward and merge
kernels are enqueued, so (a) no other thread's kernels can land between
them on the stream and overwrite the partials the merge is about to read,
and (b) a thread that needs a larger buffer (stream sync, free, allocate)
never frees one that another thread has looked up but not yet launched
with.  Varlen calls on distinct tables take no other lock, so four threads
issuing them concurrently on a fresh stream (whose workspace then grows
while they run) exercise both rules; every output must equal, bit for bit,
the same call made alone (the work decomposition and merge order are
fixed), and one of them is checked against the oracle as well.
"""

import threading

import numpy as np
import pytest

from oracle import attention as oa
from oracle import kvcache as ok
from paper_2606_16135_amd import workloads as W

from _gpu_util import DevicePool, compare_attention, from_u16, new_active, require_gpu, to_u16

pytestmark = pytest.mark.gpu

# (seed, prefix lengths, new-turn lengths): different split-key workspace
# sizes, all with key splits (long prefixes, short turns).
SHAPES = [(201, [3000], [64]), (202, [9000], [48]), (203, [1500, 7000], [40, 90]), (204, [12000], [96])]


@pytest.mark.timeout(300)
def test_varlen_calls_from_threads_on_one_stream():
    sc = require_gpu()
    import torch

    wls = [W.small_workload(seed, P, N, 1, 32, 8, 128) for seed, P, N in SHAPES]
    stream0 = torch.cuda.current_stream()
    pools, acts, qs, refs = [], [], [], []
    try:
        for wl in wls:
            pool_u16 = W.pool_numpy(wl)
            dp = DevicePool(sc, wl, pool_u16)
            pools.append(dp)
            q, kn, vn = W.layer_inputs_numpy(wl, 0)
            qd, knd, vnd = (from_u16(x, "cuda") for x in (q, kn, vn))
            k, v, act = new_active(sc, wl)
            sc.sc_fetch_layer_kv(dp.handle, dp.table, 0, act, stream0.cuda_stream)
            sc.sc_append_new_kv(dp.handle, dp.table, knd.data_ptr(), vnd.data_ptr(), act, stream0.cuda_stream)
            acts.append((k, v, act, knd, vnd))
            qs.append((q, qd))
            out = torch.empty((wl.total_q, wl.n_q_heads, wl.head_dim), dtype=torch.bfloat16, device="cuda")
            sc.sc_prefill_attn_varlen(dp.handle, dp.table, 0, qd.data_ptr(), act, wl.n_q_heads, out.data_ptr(),
                                      stream=stream0.cuda_stream)
            refs.append(out)
        torch.cuda.synchronize()
        splits = [sc.sc_attn_plan_query(wl.prefix_len, wl.new_len, wl.n_q_heads, wl.n_kv_heads)[1] for wl in wls]
        assert all(max(s) > 1 for s in splits), f"every shape must split its keys: {splits}"

        # One of the alone-run outputs against the oracle.
        wl = wls[2]
        pool_u16 = W.pool_numpy(wl)
        q, kn, vn = W.layer_inputs_numpy(wl, 0)
        ka, va = ok.gather_layer(pool_u16, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, 0)
        kf, vf = ok.append_new(ka, va, kn, vn, wl.prefix_len, wl.new_len)
        o_ref, _ = oa.attention(oa.bf16_bits_to_f64(q), oa.bf16_bits_to_f64(kf), oa.bf16_bits_to_f64(vf),
                                wl.prefix_len, wl.new_len)
        compare_attention(to_u16(refs[2]), o_ref, "alone-run varlen output")

        shared = torch.cuda.Stream()       # fresh stream: its workspace starts empty and grows
        reps = 25
        outs = [[torch.full_like(refs[i], float("nan")) for _ in range(reps)] for i in range(len(wls))]
        errors = []
        barrier = threading.Barrier(len(wls))

        def worker(i):
            try:
                barrier.wait()
                dp, wl = pools[i], wls[i]
                for r in range(reps):
                    sc.sc_prefill_attn_varlen(dp.handle, dp.table, 0, qs[i][1].data_ptr(), acts[i][2],
                                              wl.n_q_heads, outs[i][r].data_ptr(), stream=shared.cuda_stream)
            except Exception as e:  # reported below
                errors.append(e)

        threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(wls))]
        for t in threads:
            t.start()
        for t in threads:
            t.join()
        torch.cuda.synchronize()
        assert not errors, errors
        for i in range(len(wls)):
            ref = to_u16(refs[i])
            for r in range(reps):
                assert np.array_equal(to_u16(outs[i][r]), ref), f"shape {i} call {r} differs from the alone run"
    finally:
        for dp in pools:
            dp.close()
