"""Pins of the attention oracle against things other than itself.

Each test targets a plausible mistake: a dropped or extra key (single key,
q = 0 mean, causality), a wrong sign or scale (brute force, SDPA), a wrong
GQA index (brute force with distinct KV heads, GQA = replicated MHA), a
broken merge (split/merge), a transposed operand (brute force with
non-square shapes).  The last tests plant mistakes in the oracle and check
that the pins catch them.
"""

import math

import numpy as np
import pytest

from oracle import attention as oa


def _rand(rng, shape):
    return rng.standard_normal(shape)


def _packed(rng, prefix, new, hq, hkv, d):
    tq = sum(new)
    tk = sum(prefix) + sum(new)
    return _rand(rng, (tq, hq, d)), _rand(rng, (tk, hkv, d)), _rand(rng, (tk, hkv, d))


def brute_force(q, k, v, prefix, new, scale):
    """Pure-Python float64 definition: for each new token i of sequence b and
    query head h, weights exp(scale * q.k_j) over keys j <= P + i of KV head
    h // group, normalised, applied to V."""
    hq, d = q.shape[1], q.shape[2]
    hkv = k.shape[1]
    group = hq // hkv
    out = np.zeros(q.shape)
    lse = np.zeros((hq, q.shape[0]))
    qoff = koff = 0
    for p, n in zip(prefix, new):
        for i in range(n):
            for h in range(hq):
                g = h // group
                scores = []
                for j in range(p + i + 1):
                    dot = 0.0
                    for x in range(d):
                        dot += float(q[qoff + i, h, x]) * float(k[koff + j, g, x])
                    scores.append(scale * dot)
                mx = max(scores)
                w = [math.exp(s - mx) for s in scores]
                tot = sum(w)
                for x in range(d):
                    acc = 0.0
                    for j, wj in enumerate(w):
                        acc += wj * float(v[koff + j, g, x])
                    out[qoff + i, h, x] = acc / tot
                lse[h, qoff + i] = mx + math.log(tot)
        qoff += n
        koff += p + n
    return out, lse


@pytest.mark.parametrize("prefix,new,hq,hkv,d", [
    ([0], [5], 2, 2, 8),
    ([7], [3], 4, 1, 8),
    ([13, 2], [4, 3], 5, 1, 8),
    ([40], [12], 8, 2, 8),
    ([20, 0, 9], [6, 4, 1], 4, 4, 64),
])
def test_matches_brute_force(prefix, new, hq, hkv, d):
    rng = np.random.default_rng(1234 + sum(prefix) + hq)
    q, k, v = _packed(rng, prefix, new, hq, hkv, d)
    scale = 1.0 / math.sqrt(d)
    o, lse = oa.attention(q, k, v, prefix, new)
    ob, lb = brute_force(q, k, v, prefix, new, scale)
    np.testing.assert_allclose(o, ob, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lb, rtol=0, atol=1e-12)


def test_single_visible_key_returns_its_value_row():
    rng = np.random.default_rng(7)
    prefix, new = [0], [6]
    q, k, v = _packed(rng, prefix, new, 8, 2, 16)
    o, lse = oa.attention(q, k, v, prefix, new)
    for h in range(8):
        g = h // 4
        assert np.array_equal(o[0, h], v[0, g])
        assert lse[h, 0] == pytest.approx(q[0, h] @ k[0, g] / 4.0, abs=1e-14)


def test_split_and_merge_equals_unsplit():
    rng = np.random.default_rng(11)
    p, n, d = 37, 9, 16
    qh = _rand(rng, (n, d))
    kh = _rand(rng, (p + n, d))
    vh = _rand(rng, (p + n, d))
    vis = oa.causal_visible(p, np.arange(n), p + n)
    full_o, full_l = oa.softmax_attention(qh, kh, vh, vis, 0.25)
    for cut in (16, 21, p, p + 4):          # block boundary, mid-block, prefix end, inside new turn
        a = vis.copy()
        a[:, cut:] = False
        b = vis.copy()
        b[:, :cut] = False
        oa_, la_ = oa.softmax_attention(qh, kh, vh, a, 0.25)
        ob_, lb_ = oa.softmax_attention(qh, kh, vh, b, 0.25)
        mo, ml = oa.lse_merge([(oa_, la_), (ob_, lb_)])
        np.testing.assert_allclose(mo, full_o, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(ml, full_l, rtol=1e-12, atol=1e-13)


def test_merge_with_empty_part_is_identity():
    rng = np.random.default_rng(3)
    o = _rand(rng, (4, 8))
    lse = _rand(rng, 4)
    mo, ml = oa.lse_merge([(o, lse), (np.zeros((4, 8)), np.full(4, -np.inf))])
    np.testing.assert_allclose(mo, o, rtol=1e-15)
    np.testing.assert_allclose(ml, lse, rtol=1e-15)


def test_uniform_values_return_that_value():
    rng = np.random.default_rng(5)
    prefix, new = [30], [7]
    q, k, _ = _packed(rng, prefix, new, 4, 2, 8)
    c = _rand(rng, (2, 8))
    v = np.broadcast_to(c, (37, 2, 8)).copy()
    o, _ = oa.attention(q, k, v, prefix, new)
    for h in range(4):
        np.testing.assert_allclose(o[:, h], np.broadcast_to(c[h // 2], (7, 8)), rtol=1e-13, atol=1e-14)


def test_zero_query_gives_mean_of_visible_values():
    rng = np.random.default_rng(9)
    prefix, new = [19], [5]
    _, k, v = _packed(rng, prefix, new, 2, 1, 8)
    q = np.zeros((5, 2, 8))
    o, lse = oa.attention(q, k, v, prefix, new)
    for i in range(5):
        expect = v[:19 + i + 1, 0].mean(axis=0)
        np.testing.assert_allclose(o[i, 0], expect, rtol=1e-13, atol=1e-14)
        assert lse[0, i] == pytest.approx(math.log(19 + i + 1), abs=1e-13)


def test_rows_do_not_depend_on_later_tokens():
    rng = np.random.default_rng(13)
    prefix, new = [10], [8]
    q, k, v = _packed(rng, prefix, new, 4, 2, 8)
    o, _ = oa.attention(q, k, v, prefix, new)
    for i in range(8):
        k2, v2 = k.copy(), v.copy()
        k2[10 + i + 1:] = _rand(rng, k2[10 + i + 1:].shape)
        v2[10 + i + 1:] = 100.0
        o2, _ = oa.attention(q, k2, v2, prefix, new)
        assert np.array_equal(o2[i], o[i])
        if i < 7:
            assert not np.allclose(o2[i + 1], o[i + 1])


def test_gqa_equals_mha_with_replicated_kv():
    rng = np.random.default_rng(17)
    prefix, new, hq, hkv = [23], [6], 10, 2
    q, k, v = _packed(rng, prefix, new, hq, hkv, 8)
    o, lse = oa.attention(q, k, v, prefix, new)
    krep = np.repeat(k, hq // hkv, axis=1)
    vrep = np.repeat(v, hq // hkv, axis=1)
    o2, lse2 = oa.attention(q, krep, vrep, prefix, new)
    np.testing.assert_array_equal(o, o2)
    np.testing.assert_array_equal(lse, lse2)


def test_prefix_order_does_not_matter():
    rng = np.random.default_rng(19)
    prefix, new = [48], [5]
    q, k, v = _packed(rng, prefix, new, 4, 1, 8)
    o, _ = oa.attention(q, k, v, prefix, new)
    perm = np.concatenate([rng.permutation(48), np.arange(48, 53)])
    o2, _ = oa.attention(q, k[perm], v[perm], prefix, new)
    np.testing.assert_allclose(o2, o, rtol=1e-12, atol=1e-13)


def test_matches_torch_sdpa_float64():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(23)
    p, n, hq, hkv, d = 29, 11, 8, 2, 16
    q, k, v = _packed(rng, [p], [n], hq, hkv, d)
    o, _ = oa.attention(q, k, v, [p], [n])
    g = hq // hkv
    tq = torch.from_numpy(q).permute(1, 0, 2)                         # [H][N][D]
    tk = torch.from_numpy(np.repeat(k, g, axis=1)).permute(1, 0, 2)   # [H][P+N][D]
    tv = torch.from_numpy(np.repeat(v, g, axis=1)).permute(1, 0, 2)
    mask = torch.from_numpy(oa.causal_visible(p, np.arange(n), p + n))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask)
    np.testing.assert_allclose(o, ref.permute(1, 0, 2).numpy(), rtol=1e-12, atol=1e-12)


def test_row_sampled_variant_matches_dense():
    rng = np.random.default_rng(29)
    prefix, new = [33, 5], [7, 4]
    q, k, v = _packed(rng, prefix, new, 6, 3, 8)
    o, lse = oa.attention(q, k, v, prefix, new)
    rows = [(0, 0, 0), (0, 6, 5), (1, 3, 2), (1, 0, 4)]
    orow, lrow = oa.attention_rows(q, k, v, prefix, new, rows)
    cu_q = [0, 7]
    for r, (b, i, h) in enumerate(rows):
        np.testing.assert_allclose(orow[r], o[cu_q[b] + i, h], rtol=1e-12, atol=1e-13)
        assert lrow[r] == pytest.approx(lse[h, cu_q[b] + i], abs=1e-12)


def test_bf16_upcast_is_exact():
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x0000, 0x8000, 0x7F80, 0x0001], dtype=np.uint16)
    vals = oa.bf16_bits_to_f64(bits)
    assert vals[0] == 1.0 and vals[1] == -1.0
    assert vals[2] == pytest.approx(3.140625, abs=0)
    assert vals[3] == 0.0 and math.copysign(1.0, vals[4]) == -1.0
    assert math.isinf(vals[5])
    assert vals[6] == 2.0 ** -133


def test_f16_upcast_is_exact():
    """Hand-decoded binary16 patterns, and every one of the 65536 patterns
    against numpy's own float16 type (a library routine)."""
    bits = np.array([0x3C00, 0xC000, 0x7BFF, 0x0001, 0x03FF, 0x0400, 0x8000, 0x7C00, 0xFC00, 0x3555],
                    dtype=np.uint16)
    v = oa.f16_bits_to_f64(bits)
    assert v[0] == 1.0 and v[1] == -2.0
    assert v[2] == 65504.0                        # largest finite
    assert v[3] == 2.0 ** -24                     # smallest subnormal
    assert v[4] == 1023 * 2.0 ** -24              # largest subnormal
    assert v[5] == 2.0 ** -14                     # smallest normal
    assert v[6] == 0.0 and math.copysign(1.0, v[6]) == -1.0
    assert v[7] == math.inf and v[8] == -math.inf
    assert v[9] == 1365 / 4096                    # 0x3555 = 1.0101010101b * 2^-2
    allbits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    mine = oa.f16_bits_to_f64(allbits)
    ref = allbits.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(mine), nan)
    assert np.array_equal(mine[~nan], ref[~nan])
    assert np.array_equal(np.signbit(mine[~nan]), np.signbit(ref[~nan]))
    assert np.array_equal(oa.bits_to_f64(allbits[:100], "f16"), mine[:100])
    with pytest.raises(ValueError):
        oa.bits_to_f64(allbits[:4], "f32")


# ---- planted mistakes: the pins above must catch them ---------------------

def test_planted_diagonal_exclusion_is_caught(monkeypatch):
    def strict(prefix_len, q_rows, n_keys):
        q_rows = np.asarray(q_rows)
        return np.arange(n_keys)[None, :] < (prefix_len + q_rows)[:, None]
    monkeypatch.setattr(oa, "causal_visible", strict)
    rng = np.random.default_rng(7)
    q, k, v = _packed(rng, [3], [4], 2, 2, 8)
    o, _ = oa.attention(q, k, v, [3], [4])
    ob, _ = brute_force(q, k, v, [3], [4], 1 / math.sqrt(8))
    assert not np.allclose(o, ob, atol=1e-6)


def test_planted_gqa_index_mistake_is_caught(monkeypatch):
    rng = np.random.default_rng(31)
    prefix, new, hq, hkv = [9], [3], 4, 2
    q, k, v = _packed(rng, prefix, new, hq, hkv, 8)
    ob, _ = brute_force(q, k, v, prefix, new, 1 / math.sqrt(8))
    # a mapping h % H_kv instead of h // group
    swapped = np.stack([q[:, 0], q[:, 2], q[:, 1], q[:, 3]], axis=1)
    o_wrong, _ = oa.attention(swapped, k, v, prefix, new)
    o_wrong = np.stack([o_wrong[:, 0], o_wrong[:, 2], o_wrong[:, 1], o_wrong[:, 3]], axis=1)
    assert not np.allclose(o_wrong, ob, atol=1e-6)


def test_per_head_parallel_helper_equals_the_oracle():
    """The GPU tests run the oracle one query head at a time in threads at
    the benchmark shapes; that must be the same function as one call."""
    from paper_2606_16135_amd import workloads as W
    from _gpu_util import oracle_attention_by_head
    wl = W.small_workload(7, [40, 0, 300], [9, 20, 33], 1, 20, 4, 64)
    pool = W.pool_numpy(wl)
    q, kn, vn = W.layer_inputs_numpy(wl, 0)
    from oracle import kvcache as ok
    ka, va = ok.gather_layer(pool, wl.block_ids, wl.cu_blocks, wl.prefix_len, wl.new_len, 0)
    kf, vf = ok.append_new(ka, va, kn, vn, wl.prefix_len, wl.new_len)
    o_ref, _ = oa.attention(oa.bf16_bits_to_f64(q), oa.bf16_bits_to_f64(kf), oa.bf16_bits_to_f64(vf), wl.prefix_len,
                         wl.new_len)
    o = oracle_attention_by_head(q, kf, vf, wl.prefix_len, wl.new_len, "bf16", workers=4)
    assert np.array_equal(o, o_ref)
