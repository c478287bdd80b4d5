"""Benchmark of the layer-wise prefix-KV reload + prefill attention path on one GPU.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config all|1..5]
                    [--turn P,N] [--rc-fraction F] [--dtype bf16|f16] [--chunk-tokens C]
                    [--only attention|fetch|copy|h2d]

A step is one pass of the whole path over one batch: for every layer of the
stack, fetch the layer's prefix KV from the donor pool through the block
table, append the new turn, run causal GQA prefill attention over prefix +
new tokens, and store the new turn back to the pool, with the fetch of layer
l+1 overlapped with the attention of layer l on a second stream (synthetic
N(0,1) inputs, resident on the device -- the host tier of the long-context
shape in pinned host memory -- before the timed region).

The default run measures all five workloads, one after another:
  1 tiny-L1-H8-D64-P256-N64 (correctness shape: latency only),
  2 llama3-8b-P8192-N512, 3 llama3-8b-batch16-varlen,
  4 qwen-14b-P32768-N1024,
  5 llama3-8b-P131072-N2048-hosttier (the largest; the headline line).
It prints ONE JSON line whose top-level numbers are workload 5's and whose
`details.configs` holds every workload's: prefill tokens/s through the
overlapped stack, the attention call's time and fraction of the bf16 MFMA
peak, the fetch's time and fraction of the HBM peak (destinations rotating
over >= 512 MiB of buffers, so the 256 MiB Infinity Cache cannot hold them
between fetches; for workload 5 the fetch is bound by the host link and is
set against a pinned host-to-device copy measured in the same run, with the
DMA-engine alternatives beside it), the overlap overhead, and a CPU
baseline (the oracle timed on this host on a bounded sample).
`--config N` runs one workload (options --turn/--rc-fraction/--dtype/
--chunk-tokens then apply) and puts it in the headline.
"""

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "prefill tokens/s incl. layer-wise prefix-KV reload; fetch HBM GB/s; MFMA util"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = 2500.0        # dense bf16 (and fp16) MFMA, MI355X
MALL_BYTES = 256 << 20
ROTATE_BYTES = 512 << 20         # destination buffers the standalone fetch cycles through

# HBM bytes of one layer's attention (forward kernel, plus the merge kernels
# spread over the layers when a stack defers its merges) from two
# rocprofv3 --pmc passes (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0: the factors
# that map the same counters to a plain 256 MiB device copy), per workload,
# with the hash of the attention source's code (comments left out) they were
# taken on; a stale entry (the code changed since) is reported as null.
PMC_TRAFFIC = {
    "llama3-8b-P8192-N512": (80481765, "4ba710f1265470eb"),
    "llama3-8b-batch16-varlen": (705816836, "4ba710f1265470eb"),
    "qwen-14b-P32768-N1024": (364153977, "4ba710f1265470eb"),
    "llama3-8b-P131072-N2048-hosttier": (1191660843, "4ba710f1265470eb"),
    "llama3-8b-P8192-N512-rc0.5": (79959614, "4ba710f1265470eb"),
}


def _src_sha16(name):
    """Hash of a source file's code: line comments, trailing blanks and empty
    lines left out, so that editing a comment does not orphan the counters
    taken on that code (the file holds no string with two slashes)."""
    path = os.path.join(ROOT, "paper_2606_16135_amd", "csrc", name)
    with open(path, encoding="utf-8") as f:
        lines = [ln.split("//", 1)[0].rstrip() for ln in f]
    code = "\n".join(ln for ln in lines if ln)
    return hashlib.sha256(code.encode()).hexdigest()[:16]


def plain_copy_reference(torch, timed, stream, nbytes):
    """The runtime's own device-to-device copy (torch copy_) of the fetch's
    byte count, sources and destinations rotating over more than the
    Infinity Cache: what a contiguous copy of the same size reaches on this
    GPU, for comparison with the block gather of the fetch."""
    n = max(1, nbytes // 2)
    pairs = max(2, min(16, -(-(2 * MALL_BYTES) // max(nbytes, 1))))
    with torch.cuda.stream(stream):
        src = [torch.ones(n, dtype=torch.int16, device="cuda") for _ in range(pairs)]
        dst = [torch.empty(n, dtype=torch.int16, device="cuda") for _ in range(pairs)]
    st = {"i": 0}

    def one():
        i = st["i"]
        with torch.cuda.stream(stream):
            dst[i % pairs].copy_(src[(i * 7 + 3) % pairs])
        st["i"] = i + 1

    for _ in range(pairs):
        one()
    reps = max(4 * pairs, 32)
    us = timed(one, reps, stream) * 1e3          # timed() returns ms per call
    del src, dst
    gbs = 2.0 * n * 2 / (us * 1e-6) / 1e9
    return {"us": round(us, 2), "hbm_gbs": round(gbs, 1), "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
            "rotation": f"{pairs} source/destination pairs of {n * 2 >> 20} MiB"}


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


def fetch_tier_bytes(wl):
    """(device-tier bytes, host-tier bytes) of one layer's fetch."""
    row = 2 * wl.n_kv_heads * wl.head_dim * 2
    dev = host = 0
    for b in range(wl.batch):
        ids = wl.block_ids[wl.cu_blocks[b]:wl.cu_blocks[b + 1]]
        P = int(wl.prefix_len[b])
        for j in range(-(-P // wl.block_size)):
            rows = min(wl.block_size, P - j * wl.block_size)
            bid = int(ids[j])
            if bid >= wl.rc_first_id:
                continue
            if bid >= wl.n_device_blocks:
                host += rows * row
            else:
                dev += rows * row
    return dev, host


# ---------------------------------------------------------------------------
# CPU baseline: the oracle on this host
# ---------------------------------------------------------------------------

def cpu_info():
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = {"vendor": "unknown", "threads": None}
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                blas = {"vendor": i.get("internal_api"), "threads": int(i.get("num_threads", 1))}
                break
    except Exception:
        pass
    return {"cpu_model": model, "affinity_cores": len(os.sched_getaffinity(0)), "blas": blas}


def cpu_baseline(wl, dp, inputs, n_layers_sampled=3, reps=3):
    """The oracle (gather + append + attention, float64, numpy) timed on the
    host on a bounded sample of the workload: `n_layers_sampled` layers
    spread over the stack; per layer the gather + append is timed `reps`
    times (median), and attention runs on the whole layer when that layer
    is small (< 2e11 flops), else on the query heads of one KV head (the
    same oracle function on a slice of the heads), scaled by the KV-head
    count.  Extrapolated linearly to the L-layer stack."""
    import torch
    from oracle import attention as oa
    from oracle import kvcache as ok
    info = cpu_info()
    L = wl.n_layers
    layers = sorted({0, L // 2, L - 1})[:n_layers_sampled] if L > 1 else [0]
    ids = np.asarray(wl.block_ids, dtype=np.int64)
    local = np.arange(len(ids), dtype=np.int32)
    whole = attention_flops(wl) < 2e11
    group = wl.n_q_heads // wl.n_kv_heads
    t_gather, t_attn = [], []
    for layer in layers:
        sub = dp.layer_slice_u16(layer)[ids]          # referenced blocks, table order (untimed)
        q, kn, vn = (t.view(torch.int16).cpu().numpy().view(np.uint16) for t in inputs[layer])
        tg = []
        for _ in range(reps):
            t0 = time.perf_counter()
            ka, va = ok.gather_layer(sub, local, wl.cu_blocks, wl.prefix_len, wl.new_len, 0)
            kf, vf = ok.append_new(ka, va, kn, vn, wl.prefix_len, wl.new_len)
            tg.append(time.perf_counter() - t0)
        t_gather.append(float(np.median(tg)))
        if whole:
            qs, ks, vs, scale = q, kf, vf, 1.0
        else:
            qs, ks, vs, scale = q[:, :group], kf[:, :1], vf[:, :1], float(wl.n_kv_heads)
        t0 = time.perf_counter()
        oa.attention(oa.bits_to_f64(qs, wl.dtype), oa.bits_to_f64(ks, wl.dtype), oa.bits_to_f64(vs, wl.dtype),
                     wl.prefix_len, wl.new_len)
        t_attn.append((time.perf_counter() - t0) * scale)
    g = float(np.median(t_gather))
    a = float(np.median(t_attn))
    per_layer = g + a
    payload = fetch_payload_bytes(wl)
    cores = info["blas"]["threads"] or info["affinity_cores"]
    return {"value": wl.total_q / (per_layer * L), "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"float64 numpy oracle on layers {layers} of {L}: gather+append median of {reps}, "
                       f"attention on {'the whole layer' if whole else f'the {group} query heads of one KV head, x{wl.n_kv_heads}'}"
                       f"; median over the sampled layers, extrapolated to the {L}-layer stack"),
            "extrapolated": True,
            "gather_append_s_per_layer": round(g, 4), "attention_s_per_layer": round(a, 3),
            "gather_gbs": round(2.0 * payload / g / 1e9, 2) if payload else None,
            **info}


# ---------------------------------------------------------------------------
# One workload
# ---------------------------------------------------------------------------

def run_workload(args, cfg, torch, sc, W, DevicePool, with_cpu, turn=None, rc_fraction=0.0, dtype="bf16",
                 chunk_tokens=0):
    wl = W.config(cfg, rc_fraction=rc_fraction, dtype=dtype, turn=turn)
    print(f"bench.py: {wl.name}: building pool ({wl.n_blocks} blocks)", file=sys.stderr, flush=True)
    td = W.torch_dtype(wl)
    dp = DevicePool(sc, wl, fill="torch")
    L = wl.n_layers
    inputs = [W.layer_inputs_torch(wl, l, "cuda") for l in range(L)]
    outs = [torch.empty((wl.total_q, wl.n_q_heads, wl.head_dim), dtype=td, device="cuda") for _ in range(L)]

    def new_slot():
        k = torch.empty((wl.total_kv, wl.n_kv_heads, wl.head_dim), dtype=td, device="cuda")
        v = torch.empty_like(k)
        return k, v, sc.active(k.data_ptr(), v.data_ptr(), wl.total_kv)

    slot_t = [new_slot() for _ in range(2)]
    slots = [s[2] for s in slot_t]
    compute = torch.cuda.current_stream()
    copy = torch.cuda.Stream()
    qp = [i[0].data_ptr() for i in inputs]
    kp = [i[1].data_ptr() for i in inputs]
    vp = [i[2].data_ptr() for i in inputs]
    op = [o.data_ptr() for o in outs]

    def stack(flags):
        if chunk_tokens > 0:
            sc.sc_prefill_stack_chunked(dp.handle, dp.table, qp, kp, vp, op, slots, wl.n_q_heads, chunk_tokens,
                                        flags, 0.0, compute.cuda_stream, copy.cuda_stream)
        else:
            sc.sc_prefill_stack(dp.handle, dp.table, qp, kp, vp, op, slots, wl.n_q_heads, flags, 0.0,
                                compute.cuda_stream, copy.cuda_stream)

    def timed(fn, reps, stream):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps          # ms

    # Slots for a standalone fetch whose destinations rotate over >= 512 MiB.
    slot_bytes = 2 * wl.total_kv * wl.n_kv_heads * wl.head_dim * 2
    n_rot = max(2, -(-ROTATE_BYTES // slot_bytes))
    rot = [new_slot() for _ in range(n_rot - 2)]
    rot_slots = slots + [s[2] for s in rot]

    if args.only is not None:
        def fill_other_slot():
            l = max(0, L - 2)
            sc.sc_fetch_layer_kv(dp.handle, dp.table, l, slots[1], compute.cuda_stream)
            sc.sc_append_new_kv(dp.handle, dp.table, kp[l], vp[l], slots[1], compute.cuda_stream)
        return profile_only(args, wl, dp, sc, torch, stack, rot_slots, compute, L, fill_other_slot)

    # ---- headline: the overlapped stack, wall clock -------------------------
    print(f"bench.py: {wl.name}: timing", file=sys.stderr, flush=True)
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
    timed_out = sc.sc_table_stack_status(dp.table, clear=True)

    reps = max(1, args.steps)
    t_attn_only = timed(lambda: stack(sc.SC_STACK_ATTN_ONLY), reps, compute)
    t_serial = timed(lambda: stack(sc.SC_STACK_SERIAL), reps, compute)
    t_overlap = timed(lambda: stack(sc.SC_STACK_OVERLAP), reps, compute)

    # ---- attention call: the dominant kernel ------------------------------
    flops = attention_flops(wl)
    t_attn_layer = t_attn_only / L * 1e-3
    tflops = flops / t_attn_layer / 1e12
    traffic = PMC_TRAFFIC.get(wl.name)
    traffic = traffic[0] if traffic and traffic[1] == _src_sha16("attn_fwd.hip") else None
    roofline = {"bound": "mfma", "achieved": round(tflops, 2), "peak": MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tflops / MFMA_PEAK_TFLOPS, 4), "traffic": traffic,
                "kernel": f"attn_fwd_kernel<{wl.head_dim}> (+ attn_merge_kernel when keys are split): "
                          "one layer's attention call",
                "flops_per_launch": flops, "avg_launch_us": round(t_attn_layer * 1e6, 2)}

    # ---- fetch alone, destinations rotating over >= 512 MiB ---------------
    n_f = reps * L
    state = {"i": 0}

    def one_fetch():
        i = state["i"]
        sc.sc_fetch_layer_kv(dp.handle, dp.table, i % L, rot_slots[i % len(rot_slots)], copy.cuda_stream)
        state["i"] = i + 1

    t_fetch = timed(one_fetch, n_f, copy) * 1e-3            # seconds per layer
    payload = fetch_payload_bytes(wl)
    dev_b, host_b = fetch_tier_bytes(wl)
    fetch = {"us_per_layer": round(t_fetch * 1e6, 2), "payload_bytes_per_layer": payload,
             "mall_control": f"destinations rotate over {n_rot} slot pairs = {n_rot * slot_bytes >> 20} MiB "
                             f"(> the {MALL_BYTES >> 20} MiB Infinity Cache); sources are {L} distinct layer "
                             "slices of the pool"}
    if host_b == 0:
        gbs = 2.0 * payload / t_fetch / 1e9
        fetch.update({"hbm_gbs": round(gbs, 1), "payload_gbs": round(gbs / 2.0, 1),
                      "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4), "bound": "hbm"})
        fetch["plain_copy_reference"] = plain_copy_reference(torch, timed, copy, payload)
        fetch["vs_plain_copy"] = round(fetch["plain_copy_reference"]["us"] / (t_fetch * 1e6), 3)
    else:
        fetch.update(host_tier_detail(args, wl, dp, sc, torch, timed, rot_slots, copy, t_fetch, dev_b, host_b))

    entry = {
        "workload": wl.name, "description": wl.description,
        "value": round(value, 1), "unit": "tokens/s", "ms_per_step": round(ms_step, 3),
        # every token the step's attention covers (prefix + new turn), per second
        "context_tokens_per_s": round(float(np.sum(wl.prefix_len) + wl.total_q) * args.steps / elapsed, 1),
        "steps": args.steps, "warmup": args.warmup,
        "shape": {"layers": L, "q_heads": wl.n_q_heads, "kv_heads": wl.n_kv_heads, "head_dim": wl.head_dim,
                  "batch": wl.batch, "prefix_len_total": int(np.sum(wl.prefix_len)),
                  "new_len_total": wl.total_q, "block_size": wl.block_size, "pool_blocks": wl.n_blocks,
                  "host_tier_blocks": wl.n_host_blocks, "regular_cache_blocks": wl.n_rc_blocks,
                  "chunk_tokens": chunk_tokens, "dtype": wl.dtype},
        "attention": {"us_per_layer": round(t_attn_layer * 1e6, 2), "tflops": round(tflops, 1),
                      "frac_of_mfma_peak": round(tflops / MFMA_PEAK_TFLOPS, 4), "flops_per_layer": flops},
        "fetch": fetch,
        "stack_ms": {"overlap": round(t_overlap, 3), "attn_only": round(t_attn_only, 3),
                     "serial": round(t_serial, 3)},
        "overlap_overhead": round(t_overlap / t_attn_only - 1.0, 4),
        "outputs_finite": out_ok, "device_wait_timed_out": bool(timed_out),
        "roofline": roofline,
    }
    if with_cpu:
        print(f"bench.py: {wl.name}: CPU oracle sample", file=sys.stderr, flush=True)
        entry["cpu_baseline"] = cpu_baseline(wl, dp, inputs)
    del rot, slot_t, outs, inputs
    dp.close()
    del dp
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return entry


def elastic_resize(torch, sc, W, reps=5):
    """The elastic donor tier (§3.4): a library-owned HBM tier of workload
    2's pool shape (L = 32, 2 MiB blocks) shrinks by a quarter and grows back;
    both calls are timed on the host and the device's free memory is read
    around them.  A layer-major cache would have to move every kept block of
    every layer but the first for the same resize; that count is the
    formula (L - 1) * kept * slice_bytes."""
    wl = W.config(2)
    cap = wl.n_device_blocks
    keep = cap - cap // 4
    pool = sc.sc_pool_create(wl.n_layers, wl.n_kv_heads, wl.head_dim, wl.block_size, cap)
    try:
        lay = sc.sc_pool_layout_get(pool)
        t_shrink, t_grow, freed, taken = [], [], [], []
        for _ in range(reps):
            torch.cuda.synchronize()
            f0 = torch.cuda.mem_get_info()[0]
            t0 = time.perf_counter()
            sc.sc_pool_resize(pool, keep)
            t1 = time.perf_counter()
            f1 = torch.cuda.mem_get_info()[0]
            sc.sc_pool_resize(pool, cap)
            t2 = time.perf_counter()
            f2 = torch.cuda.mem_get_info()[0]
            t_shrink.append(t1 - t0)
            t_grow.append(t2 - t1)
            freed.append(f1 - f0)
            taken.append(f1 - f2)
        return {"pool_blocks": cap, "released_blocks": cap - keep, "block_bytes": lay.block_bytes,
                "chunk_blocks": lay.device_chunk_blocks,
                "shrink_ms": round(1e3 * float(np.median(t_shrink)), 3),
                "grow_ms": round(1e3 * float(np.median(t_grow)), 3),
                "device_free_bytes_after_shrink": int(np.median(freed)),
                "device_free_bytes_taken_by_grow": int(np.median(taken)),
                "kept_blocks_moved": 0,
                "layer_major_bytes_to_move": int((wl.n_layers - 1) * keep * lay.slice_bytes)}
    finally:
        sc.sc_pool_destroy(pool)


def h2d_peak_gbs(torch, nbytes=1 << 30, reps=5):
    """Pinned host -> device hipMemcpyAsync (DMA) bandwidth of one large
    contiguous copy: the host link's roofline."""
    h = torch.empty(nbytes, dtype=torch.uint8).pin_memory()
    d = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        d.copy_(h, non_blocking=True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        for _ in range(reps):
            d.copy_(h, non_blocking=True)
        e1.record(s)
    torch.cuda.synchronize()
    gbs = nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del h, d
    return gbs


def host_tier_detail(args, wl, dp, sc, torch, timed, rot_slots, copy, t_fetch, dev_b, host_b):
    """The fetch of a pool with a host tier is bound by the host link: set
    it against a pinned H2D copy measured now, and time the DMA-engine
    alternatives for the host-tier blocks (one hipMemcpyBatchAsync per layer,
    or one hipMemcpyAsync per block half)."""
    L = wl.n_layers
    link = h2d_peak_gbs(torch)
    host_gbs = host_b / t_fetch / 1e9
    out = {"bound": "host link", "device_tier_bytes": dev_b, "host_tier_bytes": host_b,
           "host_link_gbs": round(host_gbs, 2), "h2d_peak_gbs": round(link, 2),
           "frac_of_h2d_peak": round(host_gbs / link, 4),
           "hbm_gbs_device_part": None}
    alts = {}
    layers = list(range(min(L, 4)))
    for name, per_copy in (("dma_batch", False), ("dma_per_copy", True)):
        state = {"i": 0}

        def one():
            i = state["i"]
            sc.sc_fetch_layer_kv_dma(dp.handle, dp.table, layers[i % len(layers)], rot_slots[i % len(rot_slots)],
                                     per_copy, copy.cuda_stream)
            state["i"] = i + 1
        try:
            one()
            torch.cuda.synchronize()
            state["i"] = 0
            w0 = time.perf_counter()
            t = timed(one, len(layers), copy) * 1e-3
            wall = (time.perf_counter() - w0) / len(layers)
            alts[name] = {"us_per_layer": round(t * 1e6, 1), "wall_us_per_layer": round(wall * 1e6, 1),
                          "host_link_gbs": round(host_b / t / 1e9, 2)}
        except sc.SwiftCacheError as e:
            alts[name] = {"unsupported": str(e)}
    out["dma_alternatives"] = alts
    out["zero_copy_kernel_us_per_layer"] = round(t_fetch * 1e6, 1)
    return out


def profile_only(args, wl, dp, sc, torch, stack, rot_slots, compute, L, fill_other_slot):
    """Profiling aid: one op of the path over every layer, warmup then timed
    steps; prints its per-layer time."""
    copy_src = copy_dst = None
    if args.only == "copy":
        copy_src = torch.empty(128 << 20, dtype=torch.int16, device="cuda").fill_(1)
        copy_dst = torch.empty_like(copy_src)
    state = {"i": 0}

    def run_op():
        if args.only == "attention":
            stack(sc.SC_STACK_ATTN_ONLY)
        elif args.only == "fetch":
            for l in range(L):
                i = state["i"]
                sc.sc_fetch_layer_kv(dp.handle, dp.table, l, rot_slots[i % len(rot_slots)], compute.cuda_stream)
                state["i"] = i + 1
        else:
            for _ in range(L):
                copy_dst.copy_(copy_src)
    # Fill both slots without the overlapped stack: a profiler that
    # serialises dispatches would otherwise hold the overlapped stack's
    # attention, which waits on the device for the copy stream, until its
    # wait gives up.  The serial stack leaves layer L-1 in slot 0; slot 1 gets
    # layer L-2 (or 0), so every attention-only layer reads a real layer's
    # K/V rather than whatever the slot's memory held.
    stack(sc.SC_STACK_SERIAL)
    fill_other_slot()
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
    return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="all", help="all (default: every workload, headline = 5) or 1..5")
    ap.add_argument("--rc-fraction", type=float, default=0.0,
                    help="put this fraction of each sequence's full prefix blocks in the regular "
                         "cache (read in place by attention, never fetched)")
    ap.add_argument("--dtype", choices=["bf16", "f16"], default="bf16",
                    help="element type of the pool, q, K, V and outputs")
    ap.add_argument("--chunk-tokens", type=int, default=0,
                    help="process the new turn in chunks of this many tokens over each fetched layer")
    ap.add_argument("--turn", type=str, default=None, metavar="P,N",
                    help="workload 2 with prefix P and new turn N tokens")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only", choices=["attention", "fetch", "copy"], default=None,
                    help="run only one kernel of the path over every layer, --steps times (for "
                         "profiler runs; needs --config N); 'copy' runs a plain 256 MiB "
                         "device-to-device copy (reference for byte counters)")
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

    single = args.config != "all"
    if args.only is not None and not single:
        ap.error("--only needs --config N")
    if not single and (args.turn or args.rc_fraction or args.dtype != "bf16" or args.chunk_tokens):
        ap.error("--turn/--rc-fraction/--dtype/--chunk-tokens need --config N")
    with_cpu = not args.no_cpu_baseline
    entries = {}
    if single:
        cfg = int(args.config)
        turn = tuple(int(x) for x in args.turn.split(",")) if args.turn else None
        e = run_workload(args, cfg, torch, sc, W, DevicePool, with_cpu, turn=turn, rc_fraction=args.rc_fraction,
                         dtype=args.dtype, chunk_tokens=args.chunk_tokens)
        if e is None:
            return
        head = e
        entries[e["workload"]] = e
    else:
        for cfg in (1, 2, 3, 4, 5):
            e = run_workload(args, cfg, torch, sc, W, DevicePool, with_cpu)
            entries[e["workload"]] = e
        head = e
    details = {"configs": entries, "device": torch.cuda.get_device_name(0),
               "elastic_resize": elastic_resize(torch, sc, W) if not single else None,
               "headline": f"{head['workload']} (the largest single-GPU workload)" if not single
               else head["workload"]}
    result = {"metric": METRIC, "value": head["value"], "unit": "tokens/s", "n_gpus": 1,
              "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
              "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": head["shape"]["dtype"],
              "data": "synthetic",
              "config": {"workload": head["workload"], **head["shape"]},
              "roofline": head["roofline"], "details": details}
    if with_cpu:
        result["cpu_baseline"] = head["cpu_baseline"]
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
