"""A seeded random sweep of small workloads through the whole layer stack,
against the oracle: batch 1-5, prefixes 0-3000 tokens (empty ones
included, lengths not multiples of the block), new turns 0-300 tokens,
head_dim 64 and 128, GQA groups 1-8 and 16, block sizes 8-128, half
host-pinned pools, regular-cache tables, bf16 and fp16, 1-3 layers;
overlapped stacks with device-side or event waits and serial stacks, whole
or chunked new turns.  Each case checks
every attention output element of every layer, the last layer's active slot
byte for byte, and the pool after every store, so together they cover the
combinations the hand-picked parity cases do not."""

import numpy as np
import pytest

from oracle import attention as oa
from oracle import kvcache as ok
from paper_2606_16135_amd import workloads as W

from _gpu_util import DevicePool, compare_attention, from_u16, new_active, require_gpu, to_u16

N_CASES = 60
N_LARGE = 16


def random_case(i, large=False):
    """Workload parameters of sweep case i (pure function of i).  The large
    draw (2-3 layers, prefixes to 8000 tokens, turns to 600) reaches plans
    with many key splits, merged by the next layer's forward kernel."""
    base = 88_000 if large else 77_000
    rng = np.random.default_rng(base + i)
    batch = int(rng.integers(1, 4 if large else 6))
    head_dim = int(rng.choice([64, 128]))
    group = int(rng.choice([1, 2, 3, 4, 5, 6, 7, 8, 16]))
    if large:
        n_kv = int(rng.choice([1, 2, 4])) if group <= 8 else 1
    else:
        n_kv = int(rng.choice([1, 2, 4, 8])) if group <= 8 else int(rng.choice([1, 2]))
    block = int(rng.choice([8, 16, 32, 64, 128]))
    max_p, max_n = (8000, 600) if large else (3000, 300)
    prefix = [int(rng.integers(0, max_p + 1)) if rng.random() > 0.15 else 0 for _ in range(batch)]
    new = [int(rng.integers(1, max_n + 1)) if rng.random() > 0.1 else 0 for _ in range(batch)]
    if sum(new) == 0:
        new[0] = int(rng.integers(1, max_n + 1))
    host = float(rng.choice([0.0, 0.0, 0.4]))
    rc = float(rng.choice([0.0, 0.0, 0.5])) if block >= 16 else 0.0
    dtype = str(rng.choice(["bf16", "f16"]))
    layers = int(rng.integers(2, 4)) if large else int(rng.integers(1, 4))
    mode = str(rng.choice(["overlap", "overlap", "serial", "event"]))
    chunk = int(rng.choice([0, 0, 0, 32, 100]))
    return dict(seed=base + i, prefix_len=prefix, new_len=new, n_layers=layers,
                n_q_heads=n_kv * group, n_kv_heads=n_kv, head_dim=head_dim, block_size=block,
                host_fraction=host, rc_fraction=rc, dtype=dtype, mode=mode, chunk=chunk)


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(N_CASES))
def test_random_stack_matches_oracle(i):
    _run_case(random_case(i), f"sweep {i}")


@pytest.mark.gpu
@pytest.mark.parametrize("i", range(N_LARGE))
def test_random_large_stack_matches_oracle(i):
    _run_case(random_case(i, large=True), f"large sweep {i}")


def _run_case(p, label):
    sc = require_gpu()
    import torch
    print(f"\n[{label}] {p}", flush=True)
    wl = W.small_workload(p["seed"], p["prefix_len"], p["new_len"], p["n_layers"], p["n_q_heads"],
                          p["n_kv_heads"], p["head_dim"], block_size=p["block_size"],
                          host_fraction=p["host_fraction"], rc_fraction=p["rc_fraction"], dtype=p["dtype"])
    pool_u16 = W.pool_numpy(wl)
    dp = DevicePool(sc, wl, pool_u16)
    try:
        ins = [W.layer_inputs_numpy(wl, l) for l in range(wl.n_layers)]
        dev = [[from_u16(x, "cuda", wl.dtype) for x in t] for t in ins]
        outs = [torch.full((max(1, wl.total_q), wl.n_q_heads, wl.head_dim), float("nan"),
                           dtype=W.torch_dtype(wl), device="cuda") for _ in range(wl.n_layers)]
        slots = [new_active(sc, wl) for _ in range(2)]
        copy = torch.cuda.Stream()
        flags = {"overlap": sc.SC_STACK_OVERLAP, "serial": sc.SC_STACK_SERIAL,
                 "event": sc.SC_STACK_OVERLAP | sc.SC_STACK_EVENT_WAIT}[p["mode"]]
        args = (dp.handle, dp.table, [d[0].data_ptr() for d in dev], [d[1].data_ptr() for d in dev],
                [d[2].data_ptr() for d in dev], [o.data_ptr() for o in outs], [s[2] for s in slots],
                wl.n_q_heads)
        cs = torch.cuda.current_stream().cuda_stream
        if p["chunk"]:
            sc.sc_prefill_stack_chunked(*args, p["chunk"], flags, 0.0, cs, copy.cuda_stream)
        else:
            sc.sc_prefill_stack(*args, flags, 0.0, cs, copy.cuda_stream)
        torch.cuda.synchronize()
        rc_rows = ok.regular_cache_rows(wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len,
                                        wl.block_size, wl.rc_first_id)
        expect = pool_u16
        for l in range(wl.n_layers):
            q, kn, vn = ins[l]
            k_act, v_act = ok.gather_layer(pool_u16, wl.block_ids, wl.cu_blocks, wl.prefix_len,
                                           wl.new_len, l)
            k_full, v_full = ok.append_new(k_act, v_act, kn, vn, wl.prefix_len, wl.new_len)
            if wl.total_q:
                o_ref, _ = oa.attention(oa.bits_to_f64(q, wl.dtype), oa.bits_to_f64(k_full, wl.dtype),
                                        oa.bits_to_f64(v_full, wl.dtype), wl.prefix_len, wl.new_len)
                compare_attention(to_u16(outs[l])[:wl.total_q], o_ref, f"{label} layer {l}", wl.dtype)
            if l == wl.n_layers - 1:
                k_slot, v_slot, _ = slots[0] if p["mode"] == "serial" else slots[l & 1]
                keep = ~rc_rows
                assert np.array_equal(to_u16(k_slot)[keep], k_full[keep]), f"{label}: K slot"
                assert np.array_equal(to_u16(v_slot)[keep], v_full[keep]), f"{label}: V slot"
            expect = ok.store_layer(expect, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, l, kn, vn)
        assert np.array_equal(dp.full_u16(), expect), f"{label}: pool after the stores"
    finally:
        dp.close()


def test_sweep_covers_the_stated_combinations():
    """CPU check (no GPU needed) that the seeded sweep really contains the
    combinations its docstring lists."""
    cases = [random_case(k) for k in range(N_CASES)]
    assert random_case(7) == random_case(7)
    large = [random_case(k, large=True) for k in range(N_LARGE)]
    assert all(c["n_layers"] >= 2 for c in large) and max(max(c["prefix_len"]) for c in large) > 5000
    assert {c["head_dim"] for c in cases} == {64, 128}
    assert {c["dtype"] for c in cases} == {"bf16", "f16"}
    assert {c["n_q_heads"] // c["n_kv_heads"] for c in cases} == {1, 2, 3, 4, 5, 6, 7, 8, 16}
    assert {c["block_size"] for c in cases} == {8, 16, 32, 64, 128}
    assert {c["mode"] for c in cases} == {"overlap", "serial", "event"}
    assert any(c["chunk"] for c in cases) and any(not c["chunk"] for c in cases)
    assert all(any(c["chunk"] and c["mode"] == m for c in cases) for m in ("overlap", "serial", "event"))
    assert any(c["host_fraction"] > 0 for c in cases) and any(c["rc_fraction"] > 0 for c in cases)
    assert any(c["host_fraction"] > 0 and c["rc_fraction"] > 0 for c in cases)
    assert any(0 in c["prefix_len"] for c in cases) and any(0 in c["new_len"] for c in cases)
    assert any(p % c["block_size"] for c in cases for p in c["prefix_len"])
    assert {len(c["prefix_len"]) for c in cases} == {1, 2, 3, 4, 5}
    assert {c["n_layers"] for c in cases} == {1, 2, 3}
