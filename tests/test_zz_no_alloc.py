"""The allocation-free attention entry point against the one it varies.

sc_prefill_attn_noalloc keeps its split-key partials in the library's
file-scope device array and derives each workgroup's work from its index;
sc_prefill_attn allocates a workspace and uploads a work list.  Both run the
same kernels over the same key splits, so their outputs (and log-sum-exps)
must agree bit for bit; the outputs are also checked against the oracle.
Calls in a row, each smaller than the one before, show that the shared
array's leftover contents from an earlier call do not leak into a later
one; the last also has a GQA group (7) that leaves rows of the 256-row
workgroup idle, at head_dim 64.
"""

import numpy as np
import pytest

from oracle import attention as oa

from _gpu_util import compare_attention, require_gpu, to_u16

pytestmark = pytest.mark.gpu

# (prefix, new turn, q heads, KV heads, head_dim): the 8B benchmark shape's
# layer (4 key splits) first, then smaller calls.
CALLS = [(8192, 512, 32, 8, 128), (3000, 200, 32, 8, 128), (1500, 90, 28, 4, 64)]


def _inputs(torch, P, N, hq, hkv, d, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    q = torch.randn((N, hq, d), generator=g, device="cuda").to(torch.bfloat16)
    k = torch.randn((P + N, hkv, d), generator=g, device="cuda").to(torch.bfloat16)
    v = torch.randn((P + N, hkv, d), generator=g, device="cuda").to(torch.bfloat16)
    return q, k, v


@pytest.mark.timeout(300)
def test_noalloc_matches_allocating_entry_point_on_successive_calls():
    sc = require_gpu()
    import torch

    stream = torch.cuda.current_stream().cuda_stream
    for idx, (P, N, hq, hkv, d) in enumerate(CALLS):
        print(f"\n[noalloc] call {idx}: P={P} N={N} heads {hq}/{hkv} D={d}", flush=True)
        q, k, v = _inputs(torch, P, N, hq, hkv, d, 2606_16135_900 + idx)
        splits = sc.sc_attn_noalloc_splits(P, N, hq, hkv)
        out_a = torch.full((N, hq, d), float("nan"), dtype=torch.bfloat16, device="cuda")
        out_n = torch.full_like(out_a, float("nan"))
        lse_a = torch.full((hq, N), float("nan"), dtype=torch.float32, device="cuda")
        lse_n = torch.full_like(lse_a, float("nan"))
        sc.sc_prefill_attn(q.data_ptr(), k.data_ptr(), v.data_ptr(), P, N, hq, hkv, d, out_a.data_ptr(),
                           lse=lse_a.data_ptr(), stream=stream)
        sc.sc_prefill_attn_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), P, N, hq, hkv, d, out_n.data_ptr(),
                                   lse=lse_n.data_ptr(), stream=stream)
        torch.cuda.synchronize()
        assert np.array_equal(to_u16(out_n), to_u16(out_a)), f"call {idx}: outputs differ"
        assert np.array_equal(lse_n.cpu().numpy().view(np.uint32), lse_a.cpu().numpy().view(np.uint32)), \
            f"call {idx}: lse differs"
        o_ref, lse_ref = oa.attention(oa.bf16_bits_to_f64(to_u16(q)), oa.bf16_bits_to_f64(to_u16(k)),
                                      oa.bf16_bits_to_f64(to_u16(v)), [P], [N])
        stats = compare_attention(to_u16(out_n), o_ref, f"noalloc call {idx}")
        assert np.abs(lse_n.cpu().numpy() - lse_ref).max() <= 2.0 ** -8
        print(f"[noalloc] call {idx}: {splits} key splits, bit-identical to sc_prefill_attn, {stats}", flush=True)
    if idx < 1:
        pytest.fail("expected at least two calls")


def test_noalloc_rejects_partials_beyond_its_array():
    """A call whose key splits need more than the array holds is refused
    before any device work (the inputs are real device buffers anyway)."""
    sc = require_gpu()
    import torch

    P, N, hq, hkv, d = 65536, 2048, 40, 8, 128
    splits = sc.sc_attn_noalloc_splits(P, N, hq, hkv)
    need = splits * N * hq * (2 * d + 4)
    assert splits > 1 and need > 64 << 20, (splits, need)
    q = torch.zeros((N, hq, d), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((P + N, hkv, d), dtype=torch.bfloat16, device="cuda")
    v = torch.zeros_like(k)
    out = torch.zeros_like(q)
    with pytest.raises(sc.SwiftCacheError) as e:
        sc.sc_prefill_attn_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(), P, N, hq, hkv, d, out.data_ptr())
    assert e.value.status == sc.SC_ERR_RANGE and "scratch" in str(e.value)
    torch.cuda.synchronize()
