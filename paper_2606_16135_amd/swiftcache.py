"""ctypes binding of libswiftcache.so (include/swiftcache.h).

Argument marshalling only: every function forwards to the C entry point of
the same name and raises :class:`SwiftCacheError` on a negative status.
Device buffers are passed as integer device addresses (``tensor.data_ptr()``)
and streams as integer ``hipStream_t`` handles
(``torch.cuda.current_stream().cuda_stream``).

torch is imported before the library is loaded so that both share one HIP
runtime (same SONAME), which makes torch's streams and allocations valid
for the library.
"""

import ctypes
import os

import torch  # noqa: F401  (loads the HIP runtime the library binds to)

_PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG_DIR, "libswiftcache.so")

SC_OK = 0
SC_ERR_INVALID = -1
SC_ERR_OOM = -2
SC_ERR_HIP = -3
SC_ERR_RANGE = -4
SC_ERR_UNSUPPORTED = -5

SC_DTYPE_BF16 = 0
SC_DTYPE_F16 = 1
DTYPE_CODES = {"bf16": SC_DTYPE_BF16, "f16": SC_DTYPE_F16}

SC_STACK_OVERLAP = 0
SC_STACK_SERIAL = 1
SC_STACK_ATTN_ONLY = 2
SC_STACK_NO_STORE = 4
SC_STACK_TEST_NEVER_READY = 8
SC_STACK_DEBUG_POISON = 16
SC_STACK_TEST_NEVER_FREE = 32
SC_STACK_EVENT_WAIT = 64

EXPORTED = [
    "sc_pool_create", "sc_pool_destroy", "sc_pool_layout_get", "sc_table_create",
    "sc_table_destroy", "sc_table_totals", "sc_table_stack_status", "sc_stack_wait_kind", "sc_fetch_layer_kv",
    "sc_fetch_layer_kv_dma", "sc_append_new_kv",
    "sc_prefill_attn", "sc_prefill_attn_f16", "sc_prefill_attn_noalloc", "sc_attn_noalloc_splits",
    "sc_prefill_attn_varlen", "sc_store_layer_kv",
    "sc_prefill_stack", "sc_prefill_stack_chunked", "sc_attn_plan_query", "sc_pool_resize", "sc_plan_capacity", "sc_elastic_unit", "sc_scale_up",
    "sc_scale_down", "sc_last_error", "sc_version",
]


class SwiftCacheError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"status {status}: {message}")
        self.status = status


class sc_pool_desc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("n_device_blocks", ctypes.c_int64), ("n_host_blocks", ctypes.c_int64),
                ("device", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("device_base", ctypes.c_void_p), ("host_base", ctypes.c_void_p),
                ("n_rc_blocks", ctypes.c_int64), ("rc_base", ctypes.c_void_p)]


class sc_pool_layout(ctypes.Structure):
    _fields_ = [("device_base", ctypes.c_void_p), ("host_base", ctypes.c_void_p),
                ("slice_bytes", ctypes.c_size_t), ("block_bytes", ctypes.c_size_t),
                ("row_bytes", ctypes.c_size_t), ("n_device_blocks", ctypes.c_int64),
                ("n_host_blocks", ctypes.c_int64), ("device_blocks_lent", ctypes.c_int64),
                ("rc_base", ctypes.c_void_p), ("n_rc_blocks", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("device_bytes_mapped", ctypes.c_int64),
                ("device_chunk_blocks", ctypes.c_int64)]


class sc_model_shape(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("block_size", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("dtype_bytes", ctypes.c_int32)]


class sc_capacity(ctypes.Structure):
    _fields_ = [("m_block_bytes", ctypes.c_int64), ("k_master", ctypes.c_int64),
                ("sum_k_workers", ctypes.c_int64), ("n_lsc", ctypes.c_int64), ("n_rc", ctypes.c_int64),
                ("max_context_tokens", ctypes.c_int64), ("conventional_blocks", ctypes.c_int64)]


class sc_active(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("capacity_tokens", ctypes.c_int64)]


_lib = None


def load():
    """Load the library; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_16135_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, F32, VP = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                            ctypes.c_void_p)
    i32p = ctypes.POINTER(ctypes.c_int32)
    sig = {
        "sc_pool_create": (I32, [ctypes.POINTER(sc_pool_desc), ctypes.POINTER(P)]),
        "sc_pool_destroy": (None, [P]),
        "sc_pool_layout_get": (I32, [P, ctypes.POINTER(sc_pool_layout)]),
        "sc_table_create": (I32, [P, I32, i32p, i32p, i32p, i32p, VP, ctypes.POINTER(P)]),
        "sc_table_destroy": (None, [P]),
        "sc_table_totals": (I32, [P, ctypes.POINTER(I64), ctypes.POINTER(I64)]),
        "sc_table_stack_status": (I32, [P, ctypes.POINTER(I32), I32]),
        "sc_stack_wait_kind": (I32, [P, ctypes.c_uint32, ctypes.POINTER(I32)]),
        "sc_fetch_layer_kv": (I32, [P, P, I32, ctypes.POINTER(sc_active), VP]),
        "sc_fetch_layer_kv_dma": (I32, [P, P, I32, ctypes.POINTER(sc_active), I32, VP]),
        "sc_append_new_kv": (I32, [P, P, VP, VP, ctypes.POINTER(sc_active), VP]),
        "sc_prefill_attn": (I32, [VP, VP, VP, I32, I32, I32, I32, I32, F32, VP, VP, VP]),
        "sc_prefill_attn_f16": (I32, [VP, VP, VP, I32, I32, I32, I32, I32, F32, VP, VP, VP]),
        "sc_prefill_attn_noalloc": (I32, [VP, VP, VP, I32, I32, I32, I32, I32, F32, VP, VP, VP]),
        "sc_attn_noalloc_splits": (I32, [I32, I32, I32, I32, I32, i32p]),
        "sc_prefill_attn_varlen": (I32, [P, P, I32, VP, ctypes.POINTER(sc_active), I32, F32, VP, VP, VP]),
        "sc_store_layer_kv": (I32, [P, P, I32, VP, VP, VP]),
        "sc_prefill_stack": (I32, [P, P, I32, ctypes.POINTER(VP), ctypes.POINTER(VP),
                                   ctypes.POINTER(VP), ctypes.POINTER(VP),
                                   ctypes.POINTER(sc_active), I32, F32, ctypes.c_uint32, VP, VP]),
        "sc_prefill_stack_chunked": (I32, [P, P, I32, ctypes.POINTER(VP), ctypes.POINTER(VP),
                                           ctypes.POINTER(VP), ctypes.POINTER(VP),
                                           ctypes.POINTER(sc_active), I32, F32, ctypes.c_uint32, I32, VP, VP]),
        "sc_attn_plan_query": (I32, [I32, i32p, i32p, VP, I32, I32, I32, i32p, i32p, I32, i32p]),
        "sc_pool_resize": (I32, [P, I64]),
        "sc_plan_capacity": (I32, [ctypes.POINTER(sc_model_shape), I64, ctypes.POINTER(I64), I32,
                                   ctypes.POINTER(I64), ctypes.POINTER(sc_capacity)]),
        "sc_elastic_unit": (I32, [ctypes.POINTER(sc_model_shape), ctypes.POINTER(sc_model_shape),
                                  ctypes.POINTER(I64), ctypes.POINTER(I64)]),
        "sc_scale_up": (I32, [I64, I32, I64, I64, I64, ctypes.POINTER(I64), ctypes.POINTER(I64)]),
        "sc_scale_down": (I32, [I64, I32, I64, I64, ctypes.POINTER(I64), I32, ctypes.POINTER(I64),
                                ctypes.POINTER(I64)]),
        "sc_last_error": (ctypes.c_char_p, []),
        "sc_version": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status):
    if status != SC_OK:
        raise SwiftCacheError(status, load().sc_last_error().decode())


def _i32_array(values):
    arr = (ctypes.c_int32 * max(1, len(values)))(*[int(x) for x in values])
    return arr


def sc_version():
    return load().sc_version().decode()


def sc_pool_create(n_layers, n_kv_heads, head_dim, block_size, n_device_blocks, n_host_blocks=0,
                   device=0, device_base=0, host_base=0, n_rc_blocks=0, rc_base=0, dtype=SC_DTYPE_BF16):
    d = sc_pool_desc(n_layers, n_kv_heads, head_dim, block_size, n_device_blocks, n_host_blocks,
                     device, dtype, device_base or None, host_base or None, n_rc_blocks, rc_base or None)
    h = ctypes.c_void_p()
    _check(load().sc_pool_create(ctypes.byref(d), ctypes.byref(h)))
    return h.value


def sc_pool_destroy(pool):
    load().sc_pool_destroy(pool)


def sc_pool_layout_get(pool):
    lay = sc_pool_layout()
    _check(load().sc_pool_layout_get(pool, ctypes.byref(lay)))
    return lay


def sc_table_create(pool, block_ids, cu_blocks, prefix_len, new_len, stream=0):
    h = ctypes.c_void_p()
    batch = len(prefix_len)
    _check(load().sc_table_create(pool, batch, _i32_array(block_ids), _i32_array(cu_blocks),
                                  _i32_array(prefix_len), _i32_array(new_len), stream or None,
                                  ctypes.byref(h)))
    return h.value


def sc_table_destroy(table):
    load().sc_table_destroy(table)


def sc_table_totals(table):
    tq, tk = ctypes.c_int64(), ctypes.c_int64()
    _check(load().sc_table_totals(table, ctypes.byref(tq), ctypes.byref(tk)))
    return tq.value, tk.value


def sc_stack_wait_kind(table, flags):
    """True when an sc_prefill_stack call with these flags would use the
    device-side slot waits, False when stream events."""
    t = ctypes.c_int32()
    _check(load().sc_stack_wait_kind(table, flags, ctypes.byref(t)))
    return bool(t.value)


def sc_table_stack_status(table, clear=False):
    """True when an overlapped stack's attention gave up waiting for a slot
    (call after synchronising the stack's streams)."""
    t = ctypes.c_int32()
    _check(load().sc_table_stack_status(table, ctypes.byref(t), 1 if clear else 0))
    return bool(t.value)


def active(k_ptr, v_ptr, capacity_tokens):
    return sc_active(k_ptr, v_ptr, capacity_tokens)


def sc_fetch_layer_kv(pool, table, layer, dst, stream=0):
    _check(load().sc_fetch_layer_kv(pool, table, layer, ctypes.byref(dst), stream or None))


def sc_fetch_layer_kv_dma(pool, table, layer, dst, per_copy_calls=False, stream=0):
    _check(load().sc_fetch_layer_kv_dma(pool, table, layer, ctypes.byref(dst), int(per_copy_calls),
                                        stream or None))


def sc_append_new_kv(pool, table, k_new, v_new, dst, stream=0):
    _check(load().sc_append_new_kv(pool, table, k_new, v_new, ctypes.byref(dst), stream or None))


def sc_store_layer_kv(pool, table, layer, k_new, v_new, stream=0):
    _check(load().sc_store_layer_kv(pool, table, layer, k_new, v_new, stream or None))


def sc_prefill_attn(q, k_active, v_active, prefix_len, new_len, n_q_heads, n_kv_heads, head_dim,
                    out, lse=0, scale=0.0, stream=0):
    _check(load().sc_prefill_attn(q, k_active, v_active, prefix_len, new_len, n_q_heads, n_kv_heads,
                                  head_dim, scale, out, lse or None, stream or None))


def sc_prefill_attn_f16(q, k_active, v_active, prefix_len, new_len, n_q_heads, n_kv_heads, head_dim,
                        out, lse=0, scale=0.0, stream=0):
    _check(load().sc_prefill_attn_f16(q, k_active, v_active, prefix_len, new_len, n_q_heads, n_kv_heads,
                                      head_dim, scale, out, lse or None, stream or None))


def sc_prefill_attn_noalloc(q, k_active, v_active, prefix_len, new_len, n_q_heads, n_kv_heads, head_dim,
                            out, lse=0, scale=0.0, stream=0):
    _check(load().sc_prefill_attn_noalloc(q, k_active, v_active, prefix_len, new_len, n_q_heads, n_kv_heads,
                                          head_dim, scale, out, lse or None, stream or None))


def sc_attn_noalloc_splits(prefix_len, new_len, n_q_heads, n_kv_heads, slots=0):
    s = ctypes.c_int32()
    _check(load().sc_attn_noalloc_splits(prefix_len, new_len, n_q_heads, n_kv_heads, slots, ctypes.byref(s)))
    return s.value


def sc_prefill_attn_varlen(pool, table, layer, q, kv, n_q_heads, out, lse=0, scale=0.0, stream=0):
    _check(load().sc_prefill_attn_varlen(pool, table, layer, q, ctypes.byref(kv), n_q_heads, scale, out,
                                         lse or None, stream or None))


def sc_prefill_stack(pool, table, q_ptrs, knew_ptrs, vnew_ptrs, out_ptrs, slots, n_q_heads,
                     flags=SC_STACK_OVERLAP, scale=0.0, compute_stream=0, copy_stream=0):
    n = len(q_ptrs)
    arr = ctypes.c_void_p * n
    slot_arr = (sc_active * 2)(*slots)
    _check(load().sc_prefill_stack(pool, table, n, arr(*q_ptrs), arr(*knew_ptrs), arr(*vnew_ptrs),
                                   arr(*out_ptrs), slot_arr, n_q_heads, scale, flags,
                                   compute_stream or None, copy_stream or None))


def sc_attn_plan_query(prefix_len, new_len, n_q_heads, n_kv_heads, target_items=0, rc_keys=None):
    """Returns (items [n][8] int32 list, splits per sequence)."""
    import numpy as np
    batch = len(prefix_len)
    n = ctypes.c_int32()
    P, N = _i32_array(prefix_len), _i32_array(new_len)
    rc_arr = _i32_array(rc_keys) if rc_keys is not None else None
    rc = ctypes.cast(rc_arr, ctypes.c_void_p) if rc_arr is not None else None
    _check(load().sc_attn_plan_query(batch, P, N, rc, n_q_heads, n_kv_heads, target_items,
                                     ctypes.byref(n), None, 0, None))
    items = (ctypes.c_int32 * (8 * max(1, n.value)))()
    splits = (ctypes.c_int32 * batch)()
    _check(load().sc_attn_plan_query(batch, P, N, rc, n_q_heads, n_kv_heads, target_items,
                                     ctypes.byref(n), items, n.value, splits))
    arr = np.frombuffer(items, dtype=np.int32)[: 8 * n.value].reshape(n.value, 8).copy()
    return arr, list(splits)


def sc_pool_resize(pool, n_device_blocks):
    _check(load().sc_pool_resize(pool, int(n_device_blocks)))


def model_shape(n_layers, block_size, n_kv_heads, head_dim, dtype_bytes=2):
    return sc_model_shape(n_layers, block_size, n_kv_heads, head_dim, dtype_bytes)


def sc_plan_capacity(master, master_cache_bytes, worker_cache_bytes):
    """Returns (sc_capacity, [K_i per worker])."""
    n = len(worker_cache_bytes)
    w = (ctypes.c_int64 * max(1, n))(*[int(x) for x in worker_cache_bytes])
    k = (ctypes.c_int64 * max(1, n))()
    out = sc_capacity()
    _check(load().sc_plan_capacity(ctypes.byref(master), int(master_cache_bytes), w, n, k, ctypes.byref(out)))
    return out, [int(k[i]) for i in range(n)]


def sc_elastic_unit(master, worker):
    mm, mw = ctypes.c_int64(), ctypes.c_int64()
    _check(load().sc_elastic_unit(ctypes.byref(master), ctypes.byref(worker), ctypes.byref(mm), ctypes.byref(mw)))
    return mm.value, mw.value


def sc_scale_up(worker_blocks, worker_block_size, meu_worker, meu_master, request_len):
    dw, dm = ctypes.c_int64(), ctypes.c_int64()
    _check(load().sc_scale_up(int(worker_blocks), int(worker_block_size), int(meu_worker), int(meu_master),
                              int(request_len), ctypes.byref(dw), ctypes.byref(dm)))
    return dw.value, dm.value


def sc_scale_down(worker_blocks, worker_block_size, meu_worker, meu_master, window_lens):
    n = len(window_lens)
    w = (ctypes.c_int64 * max(1, n))(*[int(x) for x in window_lens])
    dw, dm = ctypes.c_int64(), ctypes.c_int64()
    _check(load().sc_scale_down(int(worker_blocks), int(worker_block_size), int(meu_worker), int(meu_master),
                                w, n, ctypes.byref(dw), ctypes.byref(dm)))
    return dw.value, dm.value


def sc_prefill_stack_chunked(pool, table, q_ptrs, knew_ptrs, vnew_ptrs, out_ptrs, slots, n_q_heads, chunk_tokens,
                             flags=SC_STACK_OVERLAP, scale=0.0, compute_stream=0, copy_stream=0):
    n = len(q_ptrs)
    arr = ctypes.c_void_p * n
    slot_arr = (sc_active * 2)(*slots)
    _check(load().sc_prefill_stack_chunked(pool, table, n, arr(*q_ptrs), arr(*knew_ptrs), arr(*vnew_ptrs),
                                           arr(*out_ptrs), slot_arr, n_q_heads, scale, flags, chunk_tokens,
                                           compute_stream or None, copy_stream or None))
