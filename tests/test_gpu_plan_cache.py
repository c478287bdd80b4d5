"""The single-call plan cache (sc_prefill_attn keeps one uploaded plan per
(device, prefix, new turn, heads, head_dim)) holds at most 256 plans; the
next distinct shape drains the device and frees that device's plans.  The
calls here are enqueued back to back with no host synchronisation, so the
eviction happens while earlier calls may still be queued, and the first
shapes are called again afterwards (their plans rebuilt).  Every output is
compared with the oracle."""

import numpy as np
import pytest

from oracle import attention as oa

from _gpu_util import compare_attention, require_gpu, to_u16

pytestmark = pytest.mark.gpu


@pytest.mark.timeout(300)
def test_plan_cache_eviction_keeps_every_result():
    sc = require_gpu()
    import torch

    hq, hkv, d = 8, 2, 64
    shapes = [(p, 1 + p % 5) for p in range(300)]   # 300 distinct (prefix, new turn) pairs
    calls = shapes + shapes[:4]
    t_max = max(p + n for p, n in shapes)
    n_max = max(n for _, n in shapes)
    g = torch.Generator(device="cuda")
    g.manual_seed(2606_16135_7)
    q = torch.randn((n_max, hq, d), generator=g, device="cuda").to(torch.bfloat16)
    k = torch.randn((t_max, hkv, d), generator=g, device="cuda").to(torch.bfloat16)
    v = torch.randn((t_max, hkv, d), generator=g, device="cuda").to(torch.bfloat16)
    stream = torch.cuda.current_stream().cuda_stream
    outs = []
    for p, n in calls:
        out = torch.full((n, hq, d), float("nan"), dtype=torch.bfloat16, device="cuda")
        sc.sc_prefill_attn(q.data_ptr(), k.data_ptr(), v.data_ptr(), p, n, hq, hkv, d, out.data_ptr(),
                           stream=stream)
        outs.append(out)
    torch.cuda.synchronize()
    qh, kh, vh = (oa.bf16_bits_to_f64(to_u16(x)) for x in (q, k, v))
    for i, ((p, n), out) in enumerate(zip(calls, outs)):
        o_ref, _ = oa.attention(qh[:n], kh[:p + n], vh[:p + n], [p], [n])
        compare_attention(to_u16(out), o_ref, f"call {i} (P={p}, N={n})")
