"""The parity check used by the GPU tests must reject wrong answers.

Each wrong answer is produced on the CPU by the oracle with a planted
mistake (or is trivially wrong), rounded to bf16 like a GPU output, and must
fail ``compare_attention``; the correct answer must pass it."""

import numpy as np
import pytest

from oracle import attention as oa
from oracle import kvcache as ok
from paper_2606_16135_amd import workloads as W

from _gpu_util import compare_attention


def _round_bf16(x):
    return W.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def _setup(q_scale, seed=1):
    wl = W.small_workload(seed, [40], [24], 2, 8, 2, 64)
    pool = W.pool_numpy(wl)
    res = []
    for layer in range(2):
        q, kn, vn = W.layer_inputs_numpy(wl, layer, q_scale=q_scale)
        ka, va = ok.gather_layer(pool, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, layer)
        kf, vf = ok.append_new(ka, va, kn, vn, wl.prefix_len, wl.new_len)
        res.append(tuple(oa.bf16_bits_to_f64(x) for x in (q, kf, vf)))
    return wl, res


def test_correct_answer_passes():
    wl, res = _setup(1.0)
    q, k, v = res[0]
    o, _ = oa.attention(q, k, v, wl.prefix_len, wl.new_len)
    compare_attention(_round_bf16(o), o, "correct")


def test_all_zero_output_fails():
    wl, res = _setup(8.0)
    q, k, v = res[0]
    o, _ = oa.attention(q, k, v, wl.prefix_len, wl.new_len)
    with pytest.raises(AssertionError):
        compare_attention(_round_bf16(np.zeros_like(o)), o, "zeros")


def test_output_of_another_layer_fails():
    wl, res = _setup(1.0)
    o0, _ = oa.attention(*res[0], wl.prefix_len, wl.new_len)
    q, k1, v1 = res[1]
    o_wrong, _ = oa.attention(res[0][0], k1, v1, wl.prefix_len, wl.new_len)
    with pytest.raises(AssertionError):
        compare_attention(_round_bf16(o_wrong), o0, "wrong layer")


def test_mask_shifted_by_one_fails_on_peaky_inputs(monkeypatch):
    wl, res = _setup(8.0)
    q, k, v = res[0]
    o, _ = oa.attention(q, k, v, wl.prefix_len, wl.new_len)

    def shifted(prefix_len, q_rows, n_keys):
        q_rows = np.asarray(q_rows)
        return np.arange(n_keys)[None, :] <= (prefix_len + q_rows + 1)[:, None]
    monkeypatch.setattr(oa, "causal_visible", shifted)
    o_wrong, _ = oa.attention(q, k, v, wl.prefix_len, wl.new_len)
    with pytest.raises(AssertionError):
        compare_attention(_round_bf16(o_wrong), o, "shifted mask")


def test_dropped_prefix_block_fails_on_peaky_inputs():
    wl, res = _setup(8.0)
    q, k, v = res[0]
    o, _ = oa.attention(q, k, v, wl.prefix_len, wl.new_len)
    k2, v2 = k.copy(), v.copy()
    k2[16:32] = -30.0          # block 1 of the prefix is never attended
    o_wrong, _ = oa.attention(q, k2, v2, wl.prefix_len, wl.new_len)
    with pytest.raises(AssertionError):
        compare_attention(_round_bf16(o_wrong), o, "dropped block")
