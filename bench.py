"""Benchmark of the layer-wise prefix-KV reload + prefill attention path on one GPU.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 2] [--turn P,N]

A step is one pass of the whole path over one batch: for every layer of the
stack, fetch the layer's prefix KV from the donor pool through the block
table, append the new turn, run causal GQA prefill attention over prefix +
new tokens, and store the new turn back to the pool, with the fetch of layer
l+1 overlapped with the attention of layer l on a second stream.  The
default workload is the Llama-3-8B-shaped stack: 32 layers, 32 query / 8 KV
heads, head_dim 128, one conversation with an 8192-token cached prefix and a
512-token new turn, donor pool 4x the blocks needed with seeded random
placement (synthetic N(0,1) bf16 data; inputs are resident in HBM before the
timed region).

Prints one JSON line.  `value` = new-turn tokens per second through the
whole stack.  `roofline` is for the attention kernel (MFMA-bound), timed
with HIP events on its own stream; `details` adds the fetch kernel's HBM
bandwidth, the attention-only and serial stack times, and the overlap
overhead, plus a plain 1 GiB device-to-device copy's bandwidth as context
for the fetch.  `cpu_baseline` times the CPU oracle on a bounded sample of the
same workload (a few layers, extrapolated to the stack).
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "prefill tokens/s incl. layer-wise prefix-KV reload; fetch HBM GB/s; MFMA util"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
# HBM bytes of one attention call (forward + merge) from two rocprofv3 --pmc
# passes (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0: the factors that map the same
# counters to a plain 256 MiB copy), per workload, for the kernels as they
# are now; profiles/attention_<workload>.md holds the commands and readings.
PMC_TRAFFIC = {"llama3-8b-P8192-N512": 80546600}


def attention_flops(wl):
    """Algorithmic flops of one layer's attention: 4 * D * H_q per visible
    (query, key) pair; pairs per sequence = N * P + N (N + 1) / 2."""
    pairs = sum(int(n) * int(p) + int(n) * (int(n) + 1) // 2 for p, n in zip(wl.prefix_len, wl.new_len))
    return 4.0 * wl.head_dim * wl.n_q_heads * pairs


def fetch_payload_bytes(wl):
    """Prefix KV bytes moved by one layer's fetch (K and V): every prefix
    token outside the regular cache, whose blocks attention reads in place."""
    row = 2 * wl.n_kv_heads * wl.head_dim * 2
    rc_keys = int(np.sum(wl.rc_blocks_per_seq())) * wl.block_size
    return row * (int(np.sum(wl.prefix_len)) - rc_keys)


def cpu_baseline(wl, dp, inputs, budget_s=15.0):
    """The oracle (gather + append + attention) timed on the host cores for
    as many layers as fit in the budget (at least one), extrapolated to the
    whole stack."""
    from oracle import attention as oa
    from oracle import kvcache as ok
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    t_layers = []
    for layer in range(wl.n_layers):
        pool_l = dp.layer_slice_u16(layer)
        q, kn, vn = (t.view(__import__("torch").int16).cpu().numpy().view(np.uint16) for t in inputs[layer])
        t0 = time.perf_counter()
        ka, va = ok.gather_layer(pool_l, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, 0)
        kf, vf = ok.append_new(ka, va, kn, vn, wl.prefix_len, wl.new_len)
        oa.attention(oa.bits_to_f64(q, wl.dtype), oa.bits_to_f64(kf, wl.dtype), oa.bits_to_f64(vf, wl.dtype),
                     wl.prefix_len, wl.new_len)
        t_layers.append(time.perf_counter() - t0)
        if sum(t_layers) >= budget_s:
            break
    per_layer = float(np.mean(t_layers))
    return {"value": wl.total_q / (per_layer * wl.n_layers), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"float64 oracle gather+append+attention on {len(t_layers)} of {wl.n_layers} layers "
                      f"({per_layer:.2f} s/layer), extrapolated to the {wl.n_layers}-layer stack"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--rc-fraction", type=float, default=0.0,
                    help="put this fraction of each sequence's full prefix blocks in the regular "
                         "cache (read in place by attention, never fetched)")
    ap.add_argument("--dtype", choices=["bf16", "f16"], default="bf16",
                    help="element type of the pool, q, K, V and outputs")
    ap.add_argument("--chunk-tokens", type=int, default=0,
                    help="process the new turn in chunks of this many tokens over each fetched layer "
                         "(0: the whole turn in one attention launch per layer)")
    ap.add_argument("--turn", type=str, default=None, metavar="P,N",
                    help="config 2 with prefix P and new turn N tokens (e.g. 1024,64: a short turn)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only", choices=["attention", "fetch", "copy"], default=None,
                    help="run only one kernel of the path, --steps times over every layer "
                         "(for profiler runs), and print its per-layer time; 'copy' runs a "
                         "plain 256 MiB device-to-device copy (reference for byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (--gpus {args.gpus} requested); "
              "the path's multi-GPU sharding is described, not run.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_16135_amd import swiftcache as sc
    from paper_2606_16135_amd import workloads as W
    from paper_2606_16135_amd.torch_pool import DevicePool
    sc.load()
    assert torch.cuda.is_available(), "bench.py needs a GPU"

    turn = tuple(int(x) for x in args.turn.split(",")) if args.turn else None
    wl = W.config(args.config, rc_fraction=args.rc_fraction, dtype=args.dtype, turn=turn)
    td = W.torch_dtype(wl)
    dp = DevicePool(sc, wl, fill="torch")
    L = wl.n_layers
    inputs = [W.layer_inputs_torch(wl, l, "cuda") for l in range(L)]
    outs = [torch.empty((wl.total_q, wl.n_q_heads, wl.head_dim), dtype=td, device="cuda")
            for _ in range(L)]
    slot_t = [(torch.empty((wl.total_kv, wl.n_kv_heads, wl.head_dim), dtype=td, device="cuda"),
               torch.empty((wl.total_kv, wl.n_kv_heads, wl.head_dim), dtype=td, device="cuda"))
              for _ in range(2)]
    slots = [sc.active(k.data_ptr(), v.data_ptr(), wl.total_kv) for k, v in slot_t]
    compute = torch.cuda.current_stream()
    copy = torch.cuda.Stream()
    qp = [i[0].data_ptr() for i in inputs]
    kp = [i[1].data_ptr() for i in inputs]
    vp = [i[2].data_ptr() for i in inputs]
    op = [o.data_ptr() for o in outs]

    def stack(flags):
        if args.chunk_tokens > 0:
            sc.sc_prefill_stack_chunked(dp.handle, dp.table, qp, kp, vp, op, slots, wl.n_q_heads, args.chunk_tokens,
                                        flags, 0.0, compute.cuda_stream, copy.cuda_stream)
        else:
            sc.sc_prefill_stack(dp.handle, dp.table, qp, kp, vp, op, slots, wl.n_q_heads, flags, 0.0,
                                compute.cuda_stream, copy.cuda_stream)

    if args.only is not None:
        # Profiling aid: one op over all layers, warmup then timed steps.
        print(f"bench.py: {wl.name} pool and inputs ready", file=sys.stderr, flush=True)
        copy_src = copy_dst = None
        if args.only == "copy":
            copy_src = torch.empty(128 << 20, dtype=torch.int16, device="cuda").fill_(1)
            copy_dst = torch.empty_like(copy_src)

        def run_op():
            if args.only == "attention":
                stack(sc.SC_STACK_ATTN_ONLY)
            elif args.only == "fetch":
                for l in range(L):
                    sc.sc_fetch_layer_kv(dp.handle, dp.table, l, slots[l & 1], compute.cuda_stream)
            else:
                for _ in range(L):
                    copy_dst.copy_(copy_src)
        # Fill both slots in serial mode: a profiler that serialises
        # dispatches would otherwise hold the overlapped stack's attention,
        # which waits on the device for the copy stream, until its wait
        # gives up.
        sc.sc_prefill_stack(dp.handle, dp.table, qp, kp, vp, op, [slots[0], slots[0]], wl.n_q_heads,
                            sc.SC_STACK_SERIAL, 0.0, compute.cuda_stream, 0)
        sc.sc_prefill_stack(dp.handle, dp.table, qp, kp, vp, op, [slots[1], slots[1]], wl.n_q_heads,
                            sc.SC_STACK_SERIAL, 0.0, compute.cuda_stream, 0)
        for _ in range(args.warmup):
            run_op()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(compute)
        for _ in range(args.steps):
            run_op()
        e1.record(compute)
        torch.cuda.synchronize()
        per_layer_us = e0.elapsed_time(e1) * 1e3 / (args.steps * L)
        print(json.dumps({"only": args.only, "workload": wl.name, "us_per_layer": round(per_layer_us, 2)}),
              flush=True)
        dp.close()
        return

    # ---- headline: overlapped stack --------------------------------------
    for _ in range(args.warmup):
        stack(sc.SC_STACK_OVERLAP)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        stack(sc.SC_STACK_OVERLAP)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = 1e3 * elapsed / args.steps
    value = wl.total_q * args.steps / elapsed
    out_ok = all(bool(torch.isfinite(o.float()).all()) for o in outs)

    def timed_stack(flags, reps):
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(compute)
        for _ in range(reps):
            stack(flags)
        ev1.record(compute)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / reps

    reps = max(1, args.steps)
    t_attn_only = timed_stack(sc.SC_STACK_ATTN_ONLY, reps)      # attention kernels of L layers
    t_serial = timed_stack(sc.SC_STACK_SERIAL, reps)
    t_overlap = timed_stack(sc.SC_STACK_OVERLAP, reps)

    # ---- fetch kernel alone, timed on its own stream ---------------------
    with torch.cuda.stream(copy):
        f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        f0.record(copy)
        for r in range(reps):
            for l in range(L):
                sc.sc_fetch_layer_kv(dp.handle, dp.table, l, slots[l & 1], copy.cuda_stream)
        f1.record(copy)
    torch.cuda.synchronize()
    t_fetch = f0.elapsed_time(f1) / (reps * L) * 1e-3          # seconds per layer
    fetch_gbs = 2.0 * fetch_payload_bytes(wl) / t_fetch / 1e9

    # Context for the fetch: a plain contiguous 1 GiB device-to-device copy
    # (torch copy_, the runtime's copy kernel) on the same stream, read +
    # write bytes per second.
    csrc = torch.empty(1 << 29, dtype=torch.int16, device="cuda").fill_(1)
    cdst = torch.empty_like(csrc)
    with torch.cuda.stream(copy):
        cdst.copy_(csrc)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record(copy)
        for _ in range(5):
            cdst.copy_(csrc)
        c1.record(copy)
    torch.cuda.synchronize()
    copy_gbs = 2.0 * csrc.numel() * 2 * 5 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del csrc, cdst

    flops = attention_flops(wl)
    t_attn_layer = t_attn_only / L * 1e-3
    achieved_tflops = flops / t_attn_layer / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved_tflops, 2), "peak": BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved_tflops / BF16_PEAK_TFLOPS, 4),
                "traffic": PMC_TRAFFIC.get(wl.name),
                "kernel": "attn_fwd_kernel<128> + attn_merge_kernel (one attention call)",
                "flops_per_launch": flops, "avg_launch_us": round(t_attn_layer * 1e6, 2)}

    # Elastic donor tier (§3.4): the block-major pool shrinks / grows in
    # place; time the host call, and state what a layer-major cache would
    # move for the same resize ((L - 1) * kept blocks * slice bytes).
    lay = sc.sc_pool_layout_get(dp.handle)
    cap, keep = lay.n_device_blocks, int(np.max(wl.block_ids[wl.block_ids < lay.n_device_blocks]) + 1
                                        if np.any(wl.block_ids < lay.n_device_blocks) else 0)
    t0r = time.perf_counter()
    for _ in range(1000):
        sc.sc_pool_resize(dp.handle, keep)
        sc.sc_pool_resize(dp.handle, cap)
    resize_us = (time.perf_counter() - t0r) / 2000 * 1e6
    elastic = {"resize_host_us": round(resize_us, 3), "blocks_released": int(cap - keep),
               "bytes_moved": 0,
               "layer_major_bytes_moved": int((L - 1) * keep * lay.slice_bytes)}

    details = {
        "stack_ms": {"overlap": round(t_overlap, 3), "attn_only": round(t_attn_only, 3),
                     "serial": round(t_serial, 3)},
        "overlap_overhead": round(t_overlap / t_attn_only - 1.0, 4),
        "fetch": {"us_per_layer": round(t_fetch * 1e6, 2), "hbm_gbs": round(fetch_gbs, 1),
                  "device_copy_1gib_gbs": round(copy_gbs, 1),
                  "frac_of_hbm_peak": round(fetch_gbs / HBM_PEAK_GBS, 4),
                  "payload_bytes_per_layer": fetch_payload_bytes(wl)},
        "elastic": elastic,
        "outputs_finite": out_ok,
        "device": torch.cuda.get_device_name(0),
    }

    result = {"metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
              "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 3),
              "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
              "data": "synthetic",
              "config": {"workload": wl.name, "layers": L, "q_heads": wl.n_q_heads,
                         "kv_heads": wl.n_kv_heads, "head_dim": wl.head_dim,
                         "prefix_len": [int(x) for x in wl.prefix_len][:16],
                         "new_len": [int(x) for x in wl.new_len][:16], "block_size": wl.block_size,
                         "pool_blocks": wl.n_blocks, "host_tier_blocks": wl.n_host_blocks,
                         "regular_cache_blocks": wl.n_rc_blocks, "chunk_tokens": args.chunk_tokens},
              "roofline": roofline, "details": details}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, dp, inputs)
    print(json.dumps(result), flush=True)
    dp.close()


if __name__ == "__main__":
    main()
