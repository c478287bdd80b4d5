"""Oracle for the worker's elastic cache: block-major resizing, the shared
scaling unit (MEU) and the scale-up / scale-down decisions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What it follows (§3.4 "Worker Cache Manager Design"):

* Layouts.  Layer-major KV cache ``(n_layers, n_blocks, block_elems)``: block
  b of layer l starts at element ``(l * n_blocks + b) * block_elems``.
  Block-major ``(n_blocks, n_layers, block_elems)``: at
  ``(b * n_layers + l) * block_elems``.  Resizing from n to n' blocks keeps
  blocks 0 .. min(n, n') - 1; a block "moves" when its start changes.
* Eq. 6-7: elements of one block of a model over all its layers,
  ``BE = L * B * H_kv * D_kv``.
* Eq. 8: ``LCM_elem = lcm(BE_m, BE_i)``.
* Eq. 9: ``MEU_m = LCM_elem / BE_m``, ``MEU_i = LCM_elem / BE_i``: the master
  scales by multiples of MEU_m blocks exactly when worker i scales by the
  same multiple of MEU_i blocks, so the bytes traded are equal.
* Algorithm 1.  ScaleUp(N_i, B_i, MEU_i, MEU_m, request_len): the worker
  needs ceil(request_len / B_i) blocks; if it holds at least that many
  nothing changes, otherwise it grows by the smallest multiple k of MEU_i
  that covers the shortfall and the master gives up k * MEU_m blocks.
  ScaleDown(N_i, B_i, MEU_i, MEU_m, lengths in the last t seconds): the
  worker keeps ceil(max length / B_i) blocks; if it holds more, it releases
  the largest multiple k of MEU_i that fits in the surplus and the master
  gains k * MEU_m blocks.  Both return (worker blocks, master blocks).

Reading taken where the paper is silent: ScaleDown over an empty window
uses a maximum length of 0 (no recent request needs any block).

Pins (tests/test_oracle_elastic.py): MEU values derived from Table 2's model
shapes by prime factorisation (Qwen3-32B master with a Qwen3-8B worker:
MEU 9 / 16; LWM with Qwen3-14B: 5 / 16), equal traded bytes and minimality
of the unit checked by brute force, Algorithm 1 against an exhaustive search
over k, and resize move counts against a simulation that rebuilds both
layouts element by element.
"""

import math


def block_elems(n_layers, block_size, n_kv_heads, head_dim):
    """Eq. 6 / Eq. 7."""
    return n_layers * block_size * n_kv_heads * head_dim


def lcm_elems(be_master, be_worker):
    """Eq. 8."""
    return be_master * be_worker // math.gcd(be_master, be_worker)


def meu(be_master, be_worker):
    """Eq. 9: (MEU_m, MEU_i)."""
    lcm = lcm_elems(be_master, be_worker)
    return lcm // be_master, lcm // be_worker


def _ceil_div(a, b):
    return -(-a // b)


def scale_up(n_i, block_size_i, meu_i, meu_m, request_len):
    """Algorithm 1's scale-up decision, from what it guarantees: after it the
    worker holds enough blocks for the request, it changes by whole elastic
    units only (MEU_i of its blocks, traded for MEU_m of the master's), and
    no smaller number of units would do.  Returns (worker blocks to add,
    master blocks to give)."""
    shortfall = max(0, _ceil_div(request_len, block_size_i) - n_i)
    units = _ceil_div(shortfall, meu_i)          # least u with u * MEU_i >= shortfall
    return units * meu_i, units * meu_m


def scale_down(n_i, block_size_i, meu_i, meu_m, window_lengths):
    """Algorithm 1's scale-down decision, from what it guarantees: the worker
    keeps enough blocks for the longest request seen in the last t seconds
    (none if there was none), gives back whole elastic units only, and as
    many of them as fit in its surplus.  Returns (worker blocks to release,
    master blocks to gain)."""
    longest = max(window_lengths) if len(window_lengths) else 0
    surplus = max(0, n_i - _ceil_div(longest, block_size_i))
    units = surplus // meu_i                     # most u with u * MEU_i <= surplus
    return units * meu_i, units * meu_m


def layer_major_offset(layer, block, n_layers, n_blocks, block_elems_):
    """Element offset of (layer, block) in a layer-major cache."""
    del n_layers
    return (layer * n_blocks + block) * block_elems_


def block_major_offset(layer, block, n_layers, n_blocks, block_elems_):
    """Element offset of (layer, block) in a block-major cache."""
    del n_blocks
    return (block * n_layers + layer) * block_elems_


def moved_blocks(offset_fn, n_layers, n_old, n_new, block_elems_=1):
    """Blocks (one layer of one block each) whose start moves when the cache
    is resized from n_old to n_new blocks (the kept blocks are 0 .. min - 1)."""
    moved = 0
    for layer in range(n_layers):
        for block in range(min(n_old, n_new)):
            a = offset_fn(layer, block, n_layers, n_old, block_elems_)
            b = offset_fn(layer, block, n_layers, n_new, block_elems_)
            moved += a != b
    return moved
