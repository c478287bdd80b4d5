"""Seeded synthetic inputs for the layer-wise prefix-KV reload + prefill path.

This module only draws inputs: block placements, sequence lengths, pool
contents and per-layer q / k_new / v_new.  It holds none of the method's
arithmetic (no gather, no attention) and is the one module both the HIP path
and the oracle consume.

The paper evaluates on multi-turn conversation datasets that are not
available here; the workloads below are synthetic stand-ins with the shapes
and length distributions of those conversations: a long cached history
(prefix) plus a short new turn, KV blocks of 16 tokens scattered over a donor
pool in block-major layout.

Values are N(0, 1) draws rounded to bf16 (or to IEEE fp16 for fp16
workloads; round to nearest even) and kept as raw 16-bit patterns.  Pool
blocks that no table references are filled with the element type's
quiet-NaN pattern (bf16 0x7FC0, fp16 0x7E00), so any stray read poisons
attention.
"""

import dataclasses
import math

import numpy as np

BF16_NAN_SENTINEL = 0x7FC0
F16_NAN_SENTINEL = 0x7E00
DTYPES = ("bf16", "f16")


def nan_sentinel(dtype):
    return BF16_NAN_SENTINEL if dtype == "bf16" else F16_NAN_SENTINEL
SEED_BASE = 26061613500


@dataclasses.dataclass
class Workload:
    name: str
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    block_size: int
    prefix_len: np.ndarray          # int32 [batch]
    new_len: np.ndarray             # int32 [batch]
    n_device_blocks: int
    n_host_blocks: int
    block_ids: np.ndarray           # int32 [sum ceil((P+N)/B)]
    cu_blocks: np.ndarray           # int32 [batch + 1]
    seed: int
    description: str = ""
    n_rc_blocks: int = 0            # regular-cache tier (ids after the host tier)
    dtype: str = "bf16"             # element type: "bf16" or "f16"

    @property
    def batch(self):
        return len(self.prefix_len)

    @property
    def n_blocks(self):
        return self.n_device_blocks + self.n_host_blocks + self.n_rc_blocks

    @property
    def rc_first_id(self):
        return self.n_device_blocks + self.n_host_blocks

    def rc_blocks_per_seq(self):
        """Leading regular-cache entries of each sequence's table."""
        out = np.zeros(self.batch, dtype=np.int32)
        for b in range(self.batch):
            ids = self.block_ids[self.cu_blocks[b]:self.cu_blocks[b + 1]]
            r = 0
            while r < len(ids) and ids[r] >= self.rc_first_id:
                r += 1
            out[b] = r
        return out

    @property
    def total_q(self):
        return int(np.sum(self.new_len))

    @property
    def total_kv(self):
        return int(np.sum(self.prefix_len) + np.sum(self.new_len))

    @property
    def row_elems(self):
        """Elements of one token of one layer for K (or V)."""
        return self.n_kv_heads * self.head_dim

    @property
    def block_elems(self):
        """Elements of one pool block (all layers, K and V)."""
        return self.n_layers * 2 * self.block_size * self.row_elems

    def pool_shape(self):
        return (self.n_blocks, self.n_layers, 2, self.block_size,
                self.n_kv_heads, self.head_dim)

    def seed_for(self, tag):
        """Sub-seed for one named stream of random numbers."""
        ss = np.random.SeedSequence([self.seed, _tag_int(tag)])
        return int(ss.generate_state(1, dtype=np.uint64)[0] >> 1)


def _tag_int(tag):
    h = 1469598103934665603
    for ch in str(tag).encode():
        h = ((h ^ ch) * 1099511628211) % (1 << 63)
    return h


def _blocks_for(p, n, bs):
    return (int(p) + int(n) + bs - 1) // bs


def _place(rng, total_blocks, needed):
    """Seeded random placement: ``needed`` distinct pool block ids."""
    return rng.permutation(total_blocks)[:needed].astype(np.int32)


def make_workload(name, n_layers, n_q_heads, n_kv_heads, head_dim, prefix_len,
                  new_len, seed, block_size=16, pool_factor=4, host_fraction=0.0,
                  description="", rc_fraction=0.0, dtype="bf16"):
    """Build a workload with a seeded block placement.

    The donor pool holds ``pool_factor`` times the donor blocks the batch
    needs; a fraction ``host_fraction`` of its slots is the host-pinned tier
    (its ids follow the device tier's).  Table entries are drawn without
    replacement from all donor slots, so about ``host_fraction`` of the
    blocks of each sequence land on the host tier.

    ``rc_fraction`` > 0 moves the first floor(rc_fraction * (P // B)) blocks
    of each sequence -- blocks its prefix fills completely -- to a regular
    cache tier (ids after the host tier, ``pool_factor`` times the blocks
    placed there, seeded placement of their own).  ``dtype`` is the element
    type of every value ("bf16" or "f16")."""
    if dtype not in DTYPES:
        raise ValueError(f"unknown element type {dtype}")
    prefix_len = np.asarray(prefix_len, dtype=np.int32)
    new_len = np.asarray(new_len, dtype=np.int32)
    per_seq = np.array([_blocks_for(p, n, block_size) for p, n in zip(prefix_len, new_len)],
                       dtype=np.int64)
    rc_seq = np.array([int(math.floor(rc_fraction * (int(p) // block_size))) for p in prefix_len],
                      dtype=np.int64)
    needed = int(per_seq.sum() - rc_seq.sum())
    total = max(needed, int(round(pool_factor * needed)))
    n_host = int(round(host_fraction * total))
    n_dev = total - n_host
    rng = np.random.default_rng(np.random.SeedSequence([seed, _tag_int("placement")]))
    donor = _place(rng, total, needed)
    n_rc_needed = int(rc_seq.sum())
    n_rc = max(n_rc_needed, int(round(pool_factor * n_rc_needed))) if n_rc_needed else 0
    rc_ids = np.zeros(0, dtype=np.int32)
    if n_rc_needed:
        rng_rc = np.random.default_rng(np.random.SeedSequence([seed, _tag_int("placement-rc")]))
        rc_ids = (_place(rng_rc, n_rc, n_rc_needed) + total).astype(np.int32)
    parts, di, ri = [], 0, 0
    for b in range(len(prefix_len)):
        r, rest = int(rc_seq[b]), int(per_seq[b] - rc_seq[b])
        parts += [rc_ids[ri:ri + r], donor[di:di + rest]]
        ri, di = ri + r, di + rest
    ids = np.concatenate(parts).astype(np.int32) if parts else donor
    cu = np.concatenate([[0], np.cumsum(per_seq)]).astype(np.int32)
    return Workload(name=name, n_layers=n_layers, n_q_heads=n_q_heads, n_kv_heads=n_kv_heads,
                    head_dim=head_dim, block_size=block_size, prefix_len=prefix_len,
                    new_len=new_len, n_device_blocks=n_dev, n_host_blocks=n_host,
                    block_ids=ids, cu_blocks=cu, seed=seed, description=description,
                    n_rc_blocks=n_rc, dtype=dtype)


def config(index, seed=None, rc_fraction=0.0, dtype="bf16", turn=None):
    """The five benchmark shapes, numbered 1..5.

    1 tiny: 1 layer, 8/8 heads, D=64, prefix 256 (16 blocks) + new 64, pool of
      64 blocks, placement = a seeded permutation of the pool.
    2 Llama-3-8B shape: 32 layers, 32 q / 8 KV heads, D=128, prefix 8192, new
      512, donor pool 4x what is needed.
    3 the 8B shape with 16 conversations: prefix ~ lognormal(ln 4096, 0.8)
      clipped to [512, 32768] and floored; new-turn length uniform integer in
      [64, 1024]; ragged tables.
    4 Qwen-14B shape: 48 layers, 40 q / 8 KV heads, D=128, prefix 32768, new
      1024, pool 4x.
    5 long context, 8B shape: prefix 131072, new 2048; pool 2x what is needed,
      half of it on the host-pinned tier.

    ``turn`` = (P, N) replaces shape 2's prefix and new-turn lengths (one
    conversation of the 8B shape, e.g. a short turn on a short prefix).
    ``rc_fraction`` > 0 gives each sequence a regular-cache tier for that
    fraction of its full prefix blocks (see make_workload); ``dtype="f16"``
    draws fp16 values; the name and description say so.
    """
    if seed is None:
        seed = SEED_BASE + index
    kw = {}
    if index == 1:
        name, shape, p, n = "tiny-L1-H8-D64-P256-N64", (1, 8, 8, 64), [256], [64]
        kw = dict(pool_factor=64 / 20)
        desc = "1 layer, 8/8 heads, D=64, P=256, N=64"
    elif index == 2:
        tp, tn = turn if turn is not None else (8192, 512)
        if tp < 0 or tn < 1:
            raise ValueError(f"turn {turn}: need P >= 0 and N >= 1")
        name, shape, p, n = f"llama3-8b-P{tp}-N{tn}", (32, 32, 8, 128), [tp], [tn]
        desc = f"32 layers, 32q/8kv heads, D=128, P={tp}, N={tn}, batch 1"
    elif index == 3:
        rng = np.random.default_rng(np.random.SeedSequence([seed, _tag_int("lengths")]))
        p = np.floor(np.clip(rng.lognormal(math.log(4096.0), 0.8, size=16), 512, 32768)).astype(np.int32)
        n = rng.integers(64, 1024, size=16, endpoint=True).astype(np.int32)
        name, shape = "llama3-8b-batch16-varlen", (32, 32, 8, 128)
        desc = ("32 layers, 32q/8kv, D=128, 16 conversations, "
                "P~lognormal(ln4096,0.8) in [512,32768], N~U[64,1024]")
    elif index == 4:
        name, shape, p, n = "qwen-14b-P32768-N1024", (48, 40, 8, 128), [32768], [1024]
        desc = "48 layers, 40q/8kv heads, D=128, P=32768, N=1024"
    elif index == 5:
        name, shape, p, n = "llama3-8b-P131072-N2048-hosttier", (32, 32, 8, 128), [131072], [2048]
        kw = dict(pool_factor=2, host_fraction=0.5)
        desc = "32 layers, 32q/8kv, D=128, P=131072, N=2048, pool 2x, half host-pinned"
    else:
        raise ValueError(f"unknown config {index}")
    if turn is not None and index != 2:
        raise ValueError("turn applies to config 2 only")
    if rc_fraction:
        name += f"-rc{rc_fraction:g}"
        desc += f", regular cache for {rc_fraction:g} of the full prefix blocks"
    if dtype != "bf16":
        name += f"-{dtype}"
        desc += f", {dtype} values"
    wl = make_workload(name, *shape, p, n, seed, description=desc, rc_fraction=rc_fraction, dtype=dtype, **kw)
    if index == 1 and not rc_fraction:
        assert wl.n_blocks == 64
    return wl


def small_workload(seed, prefix_len, new_len, n_layers=2, n_q_heads=8, n_kv_heads=2,
                   head_dim=64, block_size=16, pool_factor=2.0, host_fraction=0.0, rc_fraction=0.0,
                   dtype="bf16"):
    """A custom small workload for parity edge cases."""
    return make_workload(f"small-{seed}", n_layers, n_q_heads, n_kv_heads, head_dim,
                         prefix_len, new_len, seed, block_size=block_size,
                         pool_factor=pool_factor, host_fraction=host_fraction,
                         rc_fraction=rc_fraction, dtype=dtype)



# ----------------------------------------------------------------------------
# numpy generation (small shapes; CPU tests and parity cases)
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(x):
    """Round float32 to bf16 (nearest even) and return the 16-bit patterns.
    Inputs here are finite normal draws."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def normal_bf16(rng, shape, scale=1.0):
    return f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32) * np.float32(scale))


def normal_bits(rng, shape, dtype="bf16", scale=1.0):
    """N(0, scale^2) draws rounded to the element type (nearest even), as
    16-bit patterns.  numpy's float16 conversion rounds to nearest even."""
    x = rng.standard_normal(shape, dtype=np.float32) * np.float32(scale)
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    return x.astype(np.float16).view(np.uint16)


def pool_numpy(wl):
    """Pool contents as uint16 of shape ``wl.pool_shape()``: N(0,1) values of
    the workload's element type in every referenced block, the NaN sentinel
    in every other block."""
    rng = np.random.default_rng(wl.seed_for("pool"))
    pool = np.full(wl.pool_shape(), nan_sentinel(wl.dtype), dtype=np.uint16)
    used = np.unique(wl.block_ids)
    pool[used] = normal_bits(rng, (len(used),) + wl.pool_shape()[1:], wl.dtype)
    return pool


def layer_inputs_numpy(wl, layer, q_scale=1.0):
    """q[sum N][H_q][D], k_new and v_new[sum N][H_kv][D] of one layer as
    uint16 patterns of the element type.  ``q_scale`` > 1 makes the softmax
    peaky."""
    rng = np.random.default_rng(wl.seed_for(f"layer{layer}"))
    t = wl.total_q
    q = normal_bits(rng, (t, wl.n_q_heads, wl.head_dim), wl.dtype, q_scale)
    k = normal_bits(rng, (t, wl.n_kv_heads, wl.head_dim), wl.dtype)
    v = normal_bits(rng, (t, wl.n_kv_heads, wl.head_dim), wl.dtype)
    return q, k, v


# ----------------------------------------------------------------------------
# torch generation on the device (large shapes).  torch is imported lazily so
# that CPU-only users of this module do not need it.
# ----------------------------------------------------------------------------

def torch_dtype(wl):
    import torch
    return torch.bfloat16 if wl.dtype == "bf16" else torch.float16


def _torch_gen(wl, tag, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(wl.seed_for(tag))
    return g


def fill_pool_torch(wl, dev_pool, host_pool=None, chunk_blocks=256, rc_pool=None):
    """Fill a device pool tensor (and the host-tier and regular-cache
    tensors, if any) in place.

    ``dev_pool`` is a bf16 tensor of ``n_device_blocks * block_elems``
    elements; ``host_pool`` is a pinned CPU tensor for the host tier;
    ``rc_pool`` a device tensor of ``n_rc_blocks * block_elems`` elements.
    Referenced blocks get N(0,1) bf16 values, all others the NaN sentinel.
    Values are drawn on the device in chunks of blocks."""
    import torch
    device = dev_pool.device
    td = torch_dtype(wl)
    sentinel = nan_sentinel(wl.dtype)
    used = np.zeros(wl.n_blocks, dtype=bool)
    used[wl.block_ids] = True
    be = wl.block_elems
    gen = _torch_gen(wl, "pool-device", device)
    dv = dev_pool.view(torch.int16).view(wl.n_device_blocks, be)
    dv.fill_(sentinel)
    dev_used = np.nonzero(used[:wl.n_device_blocks])[0]
    for i in range(0, len(dev_used), chunk_blocks):
        idx = torch.from_numpy(dev_used[i:i + chunk_blocks]).to(device)
        vals = torch.randn((len(idx), be), generator=gen, device=device, dtype=torch.float32)
        dv.index_copy_(0, idx, vals.to(td).view(torch.int16))
    if wl.n_host_blocks:
        assert host_pool is not None
        hv = host_pool.view(torch.int16).view(wl.n_host_blocks, be)
        hv.fill_(sentinel)
        host_used = np.nonzero(used[wl.n_device_blocks:])[0]
        genh = _torch_gen(wl, "pool-host", device)
        for i in range(0, len(host_used), chunk_blocks):
            sel = host_used[i:i + chunk_blocks]
            vals = torch.randn((len(sel), be), generator=genh, device=device, dtype=torch.float32)
            hv[torch.from_numpy(sel)] = vals.to(td).view(torch.int16).cpu()
    if wl.n_rc_blocks:
        assert rc_pool is not None
        rv = rc_pool.view(torch.int16).view(wl.n_rc_blocks, be)
        rv.fill_(sentinel)
        rc_used = np.nonzero(used[wl.rc_first_id:])[0]
        genr = _torch_gen(wl, "pool-rc", device)
        for i in range(0, len(rc_used), chunk_blocks):
            idx = torch.from_numpy(rc_used[i:i + chunk_blocks]).to(device)
            vals = torch.randn((len(idx), be), generator=genr, device=device, dtype=torch.float32)
            rv.index_copy_(0, idx, vals.to(td).view(torch.int16))


def layer_inputs_torch(wl, layer, device, q_scale=1.0):
    """Device tensors q[sum N][H_q][D], k_new, v_new[sum N][H_kv][D] of the
    workload's element type."""
    import torch
    g = _torch_gen(wl, f"layer{layer}", device)
    t = wl.total_q
    q = (torch.randn((t, wl.n_q_heads, wl.head_dim), generator=g, device=device) * q_scale)
    k = torch.randn((t, wl.n_kv_heads, wl.head_dim), generator=g, device=device)
    v = torch.randn((t, wl.n_kv_heads, wl.head_dim), generator=g, device=device)
    td = torch_dtype(wl)
    return q.to(td), k.to(td), v.to(td)


def long_sequence_torch(seed, prefix_len, new_len, n_q_heads, n_kv_heads, head_dim, device):
    """One sequence's q[new_len][H_q][D] and active K, V[prefix_len +
    new_len][H_kv][D] as bf16 device tensors of N(0,1) draws, for lengths
    too large to draw on the host (the longest sequence the attention
    accepts)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    t = prefix_len + new_len
    q = torch.randn((new_len, n_q_heads, head_dim), generator=g, device=device).to(torch.bfloat16)
    k = torch.empty((t, n_kv_heads, head_dim), dtype=torch.bfloat16, device=device)
    v = torch.empty_like(k)
    step = 1 << 16
    for dst in (k, v):
        for i in range(0, t, step):
            n = min(step, t - i)
            dst[i:i + n] = torch.randn((n, n_kv_heads, head_dim), generator=g, device=device).to(torch.bfloat16)
    return q, k, v

