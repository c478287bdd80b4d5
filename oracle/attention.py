"""Oracle for causal GQA prefill attention over prefix + new tokens.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What it follows
---------------
* §2.2 "Transformer architecture": causal attention, i.e. a token's output
  depends on its own key/value and on those of earlier positions only;
  §2.2 "Multi-turn conversations": in a new turn only the new tokens are
  computed, their attention combining the history's cached KV with the new
  tokens' KV.  New token ``i`` of a sequence with
  ``P`` cached prefix tokens therefore sees keys ``0 .. P + i`` (all of the
  prefix, the new tokens before it, and itself).
* §5 "Model": the models use GQA; query head ``h`` reads KV head
  ``h // (H_q / H_kv)`` (consecutive query heads share a KV head).
* Softmax scale ``1/sqrt(D)`` unless given (the paper is silent; this is the
  standard attention scale).

This is exact attention written as its definition: a dense score matrix,
an explicit visibility mask, a max-subtracted exponential, a row sum and a
weighted sum of V, all in float64 after an exact bf16 (or IEEE fp16, the
paper's serving precision, §5) -> float64 upcast.  No
tiling, no online softmax.  The natural-log log-sum-exp of each row's scores
is returned alongside the output.

``lse_merge`` is the identity that attention over the union of two disjoint
key sets equals the log-sum-exp weighted combination of the attentions over
each set; the HIP path uses that identity for split-key work, so the oracle
carries it as a separately pinned function.

Pins (tests/test_oracle_attention.py): pure-Python brute force on tiny
inputs for head groups 1, 4 and 5; a single visible key returns its V row;
split-and-merge equals the unsplit result; uniform V returns that V; q = 0
returns the mean of the visible V rows; rows do not depend on later tokens;
GQA equals MHA with replicated KV heads; permuting the prefix leaves the
output unchanged; the library routine
``torch.nn.functional.scaled_dot_product_attention`` (float64, explicit mask)
agrees; the fp16 upcast matches hand-decoded patterns and numpy's float16
on all 65536 patterns.
"""

import math

import numpy as np


def bf16_bits_to_f64(bits):
    """Exact upcast of bf16 bit patterns (uint16) to float64: a bf16 value is
    the upper half of the float32 with the same bits."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def f16_bits_to_f64(bits):
    """Exact upcast of IEEE 754 binary16 bit patterns (uint16) to float64,
    from the format's definition: sign bit, 5-bit exponent with bias 15,
    10-bit fraction; exponent 0 encodes subnormals 2^-14 * f / 2^10,
    exponent 31 encodes infinities (f = 0) and NaNs."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.int64)
    sign = np.where((u >> 15) & 1, -1.0, 1.0)
    e = (u >> 10) & 0x1F
    f = (u & 0x3FF).astype(np.float64)
    normal = sign * np.ldexp(1.0 + f / 1024.0, (e - 15).astype(np.int64))
    sub = sign * np.ldexp(f / 1024.0, -14)
    special = np.where(f == 0, sign * np.inf, np.nan)
    return np.where(e == 0, sub, np.where(e == 31, special, normal))


def bits_to_f64(bits, dtype="bf16"):
    """Exact upcast of 16-bit patterns of the given element type."""
    if dtype == "bf16":
        return bf16_bits_to_f64(bits)
    if dtype == "f16":
        return f16_bits_to_f64(bits)
    raise ValueError(f"unknown element type {dtype}")


def default_scale(head_dim):
    return 1.0 / math.sqrt(head_dim)


def softmax_attention(qh, kh, vh, visible, scale):
    """Attention of one head: rows ``qh[n][D]`` over keys ``kh[m][D]`` with
    values ``vh[m][D]``; ``visible[n][m]`` says which keys each row sees.

    Returns ``(o[n][D], lse[n])``.  A row that sees no key gets ``o = 0`` and
    ``lse = -inf`` (the neutral element of :func:`lse_merge`)."""
    s = (qh @ kh.T) * scale
    s = np.where(visible, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    empty = ~np.isfinite(m)
    m = np.where(empty, 0.0, m)
    p = np.exp(s - m)
    ell = p.sum(axis=1, keepdims=True)
    safe = np.where(ell > 0, ell, 1.0)
    o = (p @ vh) / safe
    lse = np.where(ell[:, 0] > 0, m[:, 0] + np.log(safe[:, 0]), -np.inf)
    return o, lse


def causal_visible(prefix_len, q_rows, n_keys):
    """Visibility of keys ``0..n_keys-1`` for new-turn query indices
    ``q_rows``: new token ``i`` sees keys ``j <= P + i``."""
    q_rows = np.asarray(q_rows, dtype=np.int64)
    j = np.arange(n_keys, dtype=np.int64)
    return j[None, :] <= (prefix_len + q_rows)[:, None]


def attention(q, k, v, prefix_len, new_len, scale=None, chunk_elems=1 << 24):
    """Causal GQA prefill attention for a packed batch.

    ``q[sum N][H_q][D]``, ``k, v[sum(P + N)][H_kv][D]`` (float arrays, packed
    as in :mod:`oracle.kvcache`).  Returns ``o[sum N][H_q][D]`` and
    ``lse[H_q][sum N]`` in float64."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    total_q, hq, d = q.shape
    hkv = k.shape[1]
    assert hq % hkv == 0
    group = hq // hkv
    if scale is None:
        scale = default_scale(d)
    p_arr = np.asarray(prefix_len, dtype=np.int64)
    n_arr = np.asarray(new_len, dtype=np.int64)
    cu_q = np.concatenate([[0], np.cumsum(n_arr)])
    cu_k = np.concatenate([[0], np.cumsum(p_arr + n_arr)])
    o = np.zeros((total_q, hq, d), dtype=np.float64)
    lse = np.full((hq, total_q), -np.inf, dtype=np.float64)
    for b in range(len(p_arr)):
        p, n = int(p_arr[b]), int(n_arr[b])
        if n == 0:
            continue
        kb = k[cu_k[b]:cu_k[b] + p + n]
        vb = v[cu_k[b]:cu_k[b] + p + n]
        rows_per_chunk = max(1, chunk_elems // (p + n))
        for h in range(hq):
            g = h // group
            for i0 in range(0, n, rows_per_chunk):
                i1 = min(n, i0 + rows_per_chunk)
                vis = causal_visible(p, np.arange(i0, i1), p + n)
                oc, lc = softmax_attention(q[cu_q[b] + i0:cu_q[b] + i1, h],
                                           kb[:, g], vb[:, g], vis, scale)
                o[cu_q[b] + i0:cu_q[b] + i1, h] = oc
                lse[h, cu_q[b] + i0:cu_q[b] + i1] = lc
    return o, lse


def attention_rows(q, k, v, prefix_len, new_len, rows, scale=None):
    """The same attention for selected rows only, for shapes too large to
    compute whole.  ``rows`` is a list of ``(b, i, h)``: sequence, new-token
    index within the sequence, query head.  Returns ``o[len(rows)][D]`` and
    ``lse[len(rows)]``."""
    d = q.shape[2]
    hq = q.shape[1]
    hkv = k.shape[1]
    group = hq // hkv
    if scale is None:
        scale = default_scale(d)
    p_arr = np.asarray(prefix_len, dtype=np.int64)
    n_arr = np.asarray(new_len, dtype=np.int64)
    cu_q = np.concatenate([[0], np.cumsum(n_arr)])
    cu_k = np.concatenate([[0], np.cumsum(p_arr + n_arr)])
    o = np.zeros((len(rows), d), dtype=np.float64)
    lse = np.zeros(len(rows), dtype=np.float64)
    for r, (b, i, h) in enumerate(rows):
        p = int(p_arr[b])
        g = h // group
        n_vis = p + i + 1
        kk = np.asarray(k[cu_k[b]:cu_k[b] + n_vis, g], dtype=np.float64)
        vv = np.asarray(v[cu_k[b]:cu_k[b] + n_vis, g], dtype=np.float64)
        qq = np.asarray(q[cu_q[b] + i, h], dtype=np.float64)[None, :]
        oc, lc = softmax_attention(qq, kk, vv, np.ones((1, n_vis), dtype=bool), scale)
        o[r] = oc[0]
        lse[r] = lc[0]
    return o, lse


def lse_merge(parts):
    """Combine ``[(o_s, lse_s), ...]`` computed over disjoint key sets into
    attention over their union: ``lse = log sum_s exp(lse_s)`` and
    ``o = sum_s exp(lse_s - lse) o_s``.  Rows with every ``lse_s = -inf``
    stay ``o = 0, lse = -inf``."""
    lses = np.stack([np.asarray(l, dtype=np.float64) for _, l in parts])
    m = lses.max(axis=0)
    m_safe = np.where(np.isfinite(m), m, 0.0)
    w = np.exp(lses - m_safe)
    tot = w.sum(axis=0)
    lse = np.where(tot > 0, m_safe + np.log(np.where(tot > 0, tot, 1.0)), -np.inf)
    o = np.zeros_like(np.asarray(parts[0][0], dtype=np.float64))
    for (o_s, _), w_s in zip(parts, w):
        coef = np.where(tot > 0, w_s / np.where(tot > 0, tot, 1.0), 0.0)
        o = o + coef[..., None] * np.asarray(o_s, dtype=np.float64)
    return o, lse
