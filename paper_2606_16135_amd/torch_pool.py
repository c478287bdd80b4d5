"""Device memory for the library from torch: a donor pool over a caller-owned
device tensor (HBM tier) and a pinned host tensor (host tier), its block
table, and active-layer buffers.  torch provides memory and streams only;
every step of the path runs in libswiftcache's kernels."""

import numpy as np
import torch


_TORCH_DTYPES = {"bf16": torch.bfloat16, "f16": torch.float16}


def to_u16(t):
    """16-bit tensor (any device) -> numpy uint16 bit patterns."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def from_u16(a, device, dtype="bf16"):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(_TORCH_DTYPES[dtype])


class DevicePool:
    """A workload's pool in caller-owned memory: a device tensor for the HBM
    tier, a pinned host tensor for the host tier and a device tensor for the
    regular-cache tier."""

    def __init__(self, sc, wl, pool_u16=None, fill="numpy"):
        self.sc, self.wl = sc, wl
        be = wl.block_elems
        self.dev = torch.empty(max(1, wl.n_device_blocks) * be, dtype=_TORCH_DTYPES[wl.dtype], device="cuda")
        self.host = None
        if wl.n_host_blocks:
            self.host = torch.empty(wl.n_host_blocks * be, dtype=_TORCH_DTYPES[wl.dtype]).pin_memory()
        self.rc = None
        if wl.n_rc_blocks:
            self.rc = torch.empty(wl.n_rc_blocks * be, dtype=_TORCH_DTYPES[wl.dtype], device="cuda")
        if pool_u16 is not None:
            flat = pool_u16.reshape(wl.n_blocks, be)
            self.dev.view(torch.int16)[: wl.n_device_blocks * be].copy_(
                torch.from_numpy(flat[: wl.n_device_blocks].reshape(-1).view(np.int16)))
            if self.host is not None:
                self.host.view(torch.int16).copy_(
                    torch.from_numpy(flat[wl.n_device_blocks:wl.rc_first_id].reshape(-1).view(np.int16)))
            if self.rc is not None:
                self.rc.view(torch.int16).copy_(
                    torch.from_numpy(flat[wl.rc_first_id:].reshape(-1).view(np.int16)))
        elif fill == "torch":
            from paper_2606_16135_amd.workloads import fill_pool_torch
            fill_pool_torch(wl, self.dev, self.host, rc_pool=self.rc)
        torch.cuda.synchronize()
        self.handle = sc.sc_pool_create(wl.n_layers, wl.n_kv_heads, wl.head_dim, wl.block_size,
                                        wl.n_device_blocks, wl.n_host_blocks, 0,
                                        self.dev.data_ptr(),
                                        self.host.data_ptr() if self.host is not None else 0,
                                        wl.n_rc_blocks, self.rc.data_ptr() if self.rc is not None else 0,
                                        sc.DTYPE_CODES[wl.dtype])
        self.table = sc.sc_table_create(self.handle, wl.block_ids, wl.cu_blocks, wl.prefix_len,
                                        wl.new_len, torch.cuda.current_stream().cuda_stream)

    def layer_slice_u16(self, layer):
        """Layer `layer` of every pool block, as a 6-D uint16 array with a
        single layer: [n_blocks][1][2][B][H_kv][D] (input for the oracle)."""
        wl = self.wl
        shp = (2, wl.block_size, wl.n_kv_heads, wl.head_dim)
        parts = []
        if wl.n_device_blocks:
            d = self.dev.view(torch.int16)[: wl.n_device_blocks * wl.block_elems]
            d = d.view(wl.n_device_blocks, wl.n_layers, *shp)[:, layer].cpu().numpy()
            parts.append(d)
        if wl.n_host_blocks:
            h = self.host.view(torch.int16).view(wl.n_host_blocks, wl.n_layers, *shp)[:, layer].numpy()
            parts.append(h.copy())
        if wl.n_rc_blocks:
            r = self.rc.view(torch.int16).view(wl.n_rc_blocks, wl.n_layers, *shp)[:, layer].cpu().numpy()
            parts.append(r)
        return np.concatenate(parts).view(np.uint16)[:, None]

    def ref_layer_u16(self, layer, ids):
        """Layer `layer` of the pool blocks `ids` (table order), as a 6-D
        uint16 array [len(ids)][1][2][B][H_kv][D]; only those blocks cross
        to the host."""
        wl = self.wl
        shp = (2, wl.block_size, wl.n_kv_heads, wl.head_dim)
        ids = np.asarray(ids, dtype=np.int64)
        out = np.zeros((len(ids), 1) + shp, dtype=np.int16)
        tiers = [(self.dev, 0, wl.n_device_blocks), (self.host, wl.n_device_blocks, wl.n_host_blocks),
                 (self.rc, wl.rc_first_id, wl.n_rc_blocks)]
        for t, first, n in tiers:
            sel = np.nonzero((ids >= first) & (ids < first + n))[0]
            if t is None or n == 0 or len(sel) == 0:
                continue
            v = t.view(torch.int16)[: n * wl.block_elems].view(n, wl.n_layers, *shp)[:, layer]
            local = torch.from_numpy(ids[sel] - first)
            if t.is_cuda:
                out[sel, 0] = v.index_select(0, local.to(t.device)).cpu().numpy()
            else:
                out[sel, 0] = v[local].numpy()
        return out.view(np.uint16)

    def full_u16(self):
        wl = self.wl
        parts = []
        if wl.n_device_blocks:
            parts.append(self.dev.view(torch.int16)[: wl.n_device_blocks * wl.block_elems].cpu().numpy())
        if wl.n_host_blocks:
            parts.append(self.host.view(torch.int16).numpy().copy())
        if wl.n_rc_blocks:
            parts.append(self.rc.view(torch.int16).cpu().numpy())
        return np.concatenate(parts).view(np.uint16).reshape(wl.pool_shape())

    def close(self):
        self.sc.sc_table_destroy(self.table)
        self.sc.sc_pool_destroy(self.handle)


def new_active(sc, wl, fill_bits=0xFFFF, extra=0):
    """K and V active-layer buffers of sum(P+N) (+ extra) rows of the
    workload's element type, filled with the 16-bit pattern `fill_bits`
    (0xFFFF is a NaN in bf16 and fp16), and their sc_active descriptor."""
    cap = wl.total_kv + extra
    fill = int(np.uint16(fill_bits).view(np.int16))
    k = torch.full((cap, wl.n_kv_heads, wl.head_dim), fill, dtype=torch.int16, device="cuda")
    v = torch.full_like(k, fill)
    k = k.view(_TORCH_DTYPES[wl.dtype])
    v = v.view(_TORCH_DTYPES[wl.dtype])
    return k, v, sc.active(k.data_ptr(), v.data_ptr(), cap)
