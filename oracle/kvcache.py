"""Oracle for the KV-cache data movement of the layer stream cache.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What it follows
---------------
* Eq. 1 (§3.2): the bytes of one block of one layer,
  ``M_block = 2 * B * H_kv * D_kv * d_type`` (K and V).
* §3.4 "Block-Major Layout": the donor pool is shaped
  ``(n_blocks, n_layers, block_elems)`` so that all layers of a block are
  contiguous.  Eq. 1's factor of two is made explicit, K half first:
  ``pool[n_blocks][n_layers][2][B][H_kv][D]``.  ``block_elems`` counts KV
  heads (the heads that own KV entries under GQA).
* §3.2 "Layer Stream Cache" and §3.3 "KV Load": before a layer's attention,
  that layer's prefix KV is loaded from the donor into a local buffer that
  holds only the active layer; the new turn's KV is written into the same
  buffer.
* §3.3 "KV Store": the new turn's KV is written back to donor blocks.

Active-buffer layout: sequences are packed one after another, sequence ``b``
occupying rows ``[cu_k[b], cu_k[b] + P_b + N_b)`` of ``K[T][H_kv][D]`` and
``V[T][H_kv][D]``: its ``P_b`` prefix tokens first, then its ``N_b`` new
tokens.  The block table of sequence ``b`` lists ``ceil((P_b + N_b) / B)``
pool block ids in token order; prefix token ``t`` lives in block
``ids_b[t // B]`` at row ``t % B``, and new token ``i`` continues at logical
position ``P_b + i`` (a partially filled last prefix block is filled up
first).

Regular cache (§3.2 "Regular Cache"): when the workers' memory cannot hold
the whole context, the master keeps some blocks with all their layers in its
own memory.  A table may list such blocks (ids at or above ``rc_first_id``)
as the leading entries of a sequence, for blocks the prefix fills
completely; their keys are used where they are and the KV Load skips them
(:func:`regular_cache_rows`).  Attention still runs over every key, so the
gathered K/V of :func:`gather_layer` defines its input either way.

Values are handled as raw 16-bit patterns (numpy ``uint16``) so that every
comparison is on bytes.

Pins (tests/test_oracle_kvcache.py, tests/test_paper_constants.py):
Eq. 1 times the layer count against the per-token sizes printed in Table 2;
gather of a pool that was built by scattering a known dense KV returns that
dense KV exactly; gather output is an exact permutation of pool rows and
leaves the pool untouched; store followed by a gather of the extended prefix
equals the concatenation of the old prefix and the new turn.
"""

import numpy as np


def m_block_bytes(block_size, n_kv_heads, head_dim, dtype_bytes):
    """Eq. 1: bytes of one block of one layer (K and V)."""
    return 2 * block_size * n_kv_heads * head_dim * dtype_bytes


def per_token_bytes(n_layers, n_kv_heads, head_dim, dtype_bytes):
    """KV bytes one token occupies over all layers: Eq. 1 divided by the block
    size and multiplied by the layer count (the "overhead/token" column of
    Table 2)."""
    return n_layers * m_block_bytes(1, n_kv_heads, head_dim, dtype_bytes)


def pool_shape(n_blocks, n_layers, block_size, n_kv_heads, head_dim):
    """Block-major pool shape with the K/V axis made explicit (§3.4)."""
    return (n_blocks, n_layers, 2, block_size, n_kv_heads, head_dim)


def seq_offsets(prefix_len, new_len):
    """Row offsets of each sequence in the packed query array (cu_q) and in
    the packed active-layer buffer (cu_k)."""
    p = np.asarray(prefix_len, dtype=np.int64)
    n = np.asarray(new_len, dtype=np.int64)
    cu_q = np.concatenate([[0], np.cumsum(n)])
    cu_k = np.concatenate([[0], np.cumsum(p + n)])
    return cu_q, cu_k


def blocks_needed(prefix_len, new_len, block_size):
    """Block-table entries per sequence: ceil((P + N) / B)."""
    p = np.asarray(prefix_len, dtype=np.int64)
    n = np.asarray(new_len, dtype=np.int64)
    return (p + n + block_size - 1) // block_size


def _token_locations(ids, start, count, block_size):
    """Pool (block id, row) of logical token positions start..start+count-1
    of one sequence whose block table is ``ids``."""
    t = np.arange(start, start + count, dtype=np.int64)
    return np.asarray(ids, dtype=np.int64)[t // block_size], t % block_size


def gather_layer(pool, block_ids, cu_blocks, prefix_len, new_len, layer):
    """KV Load of one layer (§3.2, §3.3): copy every prefix token of every
    sequence from its pool block into the packed active-layer buffer.

    ``pool`` is the 6-D block-major pool (uint16).  Returns ``(K, V)`` of
    shape ``[sum(P + N)][H_kv][D]``; rows of new tokens are left zero (they
    are filled by :func:`append_new`)."""
    n_blocks, n_layers, two, bs, hkv, d = pool.shape
    assert two == 2 and 0 <= layer < n_layers
    _, cu_k = seq_offsets(prefix_len, new_len)
    total = int(cu_k[-1])
    k_out = np.zeros((total, hkv, d), dtype=pool.dtype)
    v_out = np.zeros((total, hkv, d), dtype=pool.dtype)
    for b, p in enumerate(prefix_len):
        ids = block_ids[cu_blocks[b]:cu_blocks[b + 1]]
        blk, row = _token_locations(ids, 0, int(p), bs)
        k_out[cu_k[b]:cu_k[b] + p] = pool[blk, layer, 0, row]
        v_out[cu_k[b]:cu_k[b] + p] = pool[blk, layer, 1, row]
    return k_out, v_out


def append_new(k_act, v_act, k_new, v_new, prefix_len, new_len):
    """Write the new turn's KV after each sequence's prefix in the active
    buffer (§3.2: newly generated entries are written into the buffer).
    Returns new arrays; the inputs are not modified."""
    k_act = k_act.copy()
    v_act = v_act.copy()
    cu_q, cu_k = seq_offsets(prefix_len, new_len)
    for b, (p, n) in enumerate(zip(prefix_len, new_len)):
        dst = slice(int(cu_k[b] + p), int(cu_k[b] + p + n))
        src = slice(int(cu_q[b]), int(cu_q[b] + n))
        k_act[dst] = k_new[src]
        v_act[dst] = v_new[src]
    return k_act, v_act


def store_layer(pool, block_ids, cu_blocks, prefix_len, new_len, layer, k_new, v_new):
    """KV Store of one layer (§3.3): write each new token ``i`` of sequence
    ``b`` to logical position ``P_b + i`` of its block table.  Returns the
    updated pool; every other byte equals the input pool."""
    out = pool.copy()
    bs = pool.shape[3]
    cu_q, _ = seq_offsets(prefix_len, new_len)
    for b, (p, n) in enumerate(zip(prefix_len, new_len)):
        ids = block_ids[cu_blocks[b]:cu_blocks[b + 1]]
        blk, row = _token_locations(ids, int(p), int(n), bs)
        src = slice(int(cu_q[b]), int(cu_q[b] + n))
        out[blk, layer, 0, row] = k_new[src]
        out[blk, layer, 1, row] = v_new[src]
    return out


def regular_cache_rows(block_ids, cu_blocks, prefix_len, new_len, block_size, rc_first_id):
    """Rows of the packed active buffer whose keys live in the regular cache:
    the tokens of each sequence's leading regular-cache blocks.  The KV Load
    writes exactly the prefix rows outside this set."""
    _, cu_k = seq_offsets(prefix_len, new_len)
    rows = np.zeros(int(cu_k[-1]), dtype=bool)
    for b, p in enumerate(prefix_len):
        ids = np.asarray(block_ids[cu_blocks[b]:cu_blocks[b + 1]])
        lead = 0
        while lead < len(ids) and ids[lead] >= rc_first_id:
            lead += 1
        assert not np.any(ids[lead:] >= rc_first_id), "regular-cache blocks lead the table"
        assert lead * block_size <= p, "regular-cache blocks are full prefix blocks"
        rows[cu_k[b]:cu_k[b] + lead * block_size] = True
    return rows
