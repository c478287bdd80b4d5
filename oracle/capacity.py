"""Oracle for the master's cache capacity: layer stream cache (LSC) and
regular cache (RC) sizing.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What it follows (§3.2 "Layer Stream Cache" and "Regular Cache"):

* Eq. 1: ``M_block = 2 * B * H_kv * D_kv * d_type`` bytes per block per layer.
* Eq. 2: worker i can hold ``K_i = floor(C_worker_i / (M_block * L))`` of the
  master's full-layer blocks (``L`` = the master's layer count).
* Eq. 3: the master's own memory holds ``K_master = floor(C_master / M_block)``
  single-layer blocks.
* Eq. 4: ``N_LSC = min(sum_i K_i, K_master)`` single-layer blocks of LSC.
* Eq. 5: the rest of the master's memory holds
  ``N_RC = floor((K_master - sum_i K_i) / L)`` full-layer blocks when
  ``sum_i K_i < K_master``, else none.
* The longest context the master supports is ``(N_LSC + N_RC) * B`` tokens; a
  master without LSC holds ``floor(K_master / L)`` full-layer blocks.

Everything is integer arithmetic, written out as the equations state it.

Pins (tests/test_oracle_capacity.py): the paper's worked example (L = 10,
K_master = 100, K = (9, 8) gives 17 + 8 = 25 blocks against 10), the two
regimes of Eq. 5 at and around the boundary, monotonicity in every capacity,
and brute-force counting of how many whole blocks fit in a byte budget.
"""


def m_block_bytes(block_size, n_kv_heads, head_dim, dtype_bytes):
    """Eq. 1."""
    return 2 * block_size * n_kv_heads * head_dim * dtype_bytes


def worker_full_layer_blocks(worker_cache_bytes, m_block, n_layers):
    """Eq. 2: master full-layer blocks one worker's KV cache can hold."""
    return worker_cache_bytes // (m_block * n_layers)


def master_single_layer_blocks(master_cache_bytes, m_block):
    """Eq. 3: single-layer blocks the master's own KV cache can hold."""
    return master_cache_bytes // m_block


def lsc_blocks(k_workers, k_master):
    """Eq. 4."""
    return min(sum(k_workers), k_master)


def rc_blocks(k_workers, k_master, n_layers):
    """Eq. 5 (zero when the workers' capacity fills the master)."""
    s = sum(k_workers)
    if s >= k_master:
        return 0
    return (k_master - s) // n_layers


def plan(master_cache_bytes, worker_cache_bytes, n_layers, block_size, n_kv_heads, head_dim,
         dtype_bytes):
    """All of §3.2's capacity quantities for one master and its workers.

    Returns a dict with m_block, k_workers (list), k_master, n_lsc, n_rc,
    max_context_blocks, max_context_tokens and conventional_blocks (a master
    that keeps every layer of every block locally)."""
    mb = m_block_bytes(block_size, n_kv_heads, head_dim, dtype_bytes)
    kw = [worker_full_layer_blocks(c, mb, n_layers) for c in worker_cache_bytes]
    km = master_single_layer_blocks(master_cache_bytes, mb)
    n_lsc = lsc_blocks(kw, km)
    n_rc = rc_blocks(kw, km, n_layers)
    return {
        "m_block": mb,
        "k_workers": kw,
        "k_master": km,
        "n_lsc": n_lsc,
        "n_rc": n_rc,
        "max_context_blocks": n_lsc + n_rc,
        "max_context_tokens": (n_lsc + n_rc) * block_size,
        "conventional_blocks": km // n_layers,
    }
