// Row-copy kernel behind the layer KV load (§3.2 "Layer Stream Cache", §3.3
// "KV Load"), the append of the new turn into the active buffer (§3.2) and
// the layer KV store back to donor blocks (§3.3 "KV Store").
//
// All three move whole token rows (n_kv_heads * head_dim bf16 = row_bytes)
// between a block of the block-major pool (§3.4) and a packed buffer, so one
// body serves them: workgroup 2*i copies item i's K rows, workgroup 2*i+1
// its V rows (a grid capped below 2 * n_items, as the overlapped layer stack
// launches it beside attention, strides over the item halves).  A block slice of one layer is contiguous in the pool (K half
// then V half, Eq. 1), and consecutive rows of a sequence are contiguous in
// the active buffer, so each item is one contiguous range on both sides.
//
// The overlapped layer stack launches all three of a layer in one grid
// (kv_layer_copy_kernel) after a one-wave gate kernel that waits on the
// device for the attention that last read the slot.
//
// HBM-bound: every lane moves 16-byte chunks with kUnroll loads in flight
// before the matching stores, through buffer resources over the item's two
// ranges.  Both sides are streamed once per call: the loads are
// system-coherent and non-temporal (sc0 sc1 nt: no cache keeps the source),
// the stores non-temporal (nt), so neither evicts the attention's K/V
// working set from L2.  Measured on MI355X against non-temporal loads, the
// fetch of the 8B shape runs about 7% faster (11.9 vs 12.8 us per layer);
// against cached stores, non-temporal stores about 6% faster.  The data a
// copy reads was written by earlier kernels, whose completion wrote it back
// beyond the caches.  Host-tier blocks are read or written through their
// device-visible pinned mapping, over the host link.
#include "sc_internal.h"

namespace sc {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 8;
// Buffer instruction cache-policy bits on gfx950: sc0 = 1, nt = 2, sc1 = 16.
constexpr int kLoadPolicy = 1 | 2 | 16;
constexpr int kStorePolicy = 2;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// poison: write nan2 over the destination instead of copying (fetch and
// append into a slot whose gate timed out).
template <int MODE>
__device__ __forceinline__ void copy_rows(const CopyArgs &a, int g, bool poison = false, uint32_t nan2 = 0) {
  const int item_idx = g >> 1;
  const int is_v = g & 1;
  const CopyItem it = a.items[item_idx];
  if (MODE != COPY_APPEND && !((a.tier_mask >> it.tier) & 1)) return;
  const int64_t nchunks = ((int64_t)it.nrows * a.row_bytes) >> 4;
  const int64_t half_off = is_v ? a.v_half_off : 0;
  const char *src;
  char *dst;
  if (MODE == COPY_FETCH) {
    src = a.tier_base[it.tier] + it.pool_off + a.layer_off + half_off;
    dst = (is_v ? a.act_v : a.act_k) + it.act_row * a.row_bytes;
  } else if (MODE == COPY_APPEND) {
    src = (is_v ? a.new_v : a.new_k) + it.src_row * a.row_bytes;
    dst = (is_v ? a.act_v : a.act_k) + it.act_row * a.row_bytes;
  } else {
    src = (is_v ? a.new_v : a.new_k) + it.src_row * a.row_bytes;
    dst = a.tier_base[it.tier] + it.pool_off + a.layer_off + half_off;
  }
  // One item is at most 256 rows of one KV layer (under 4 MiB), so 32-bit
  // byte offsets cover it.
  const int bytes = (int)(nchunks * 16);
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(src), (short)0, bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(dst, (short)0, bytes, 0x00020000);
  for (int64_t base = 0; base < nchunks; base += (int64_t)kThreads * kUnroll) {
    u32x4 r[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t idx = base + u * kThreads + threadIdx.x;
      if (poison)
        r[u] = u32x4{nan2, nan2, nan2, nan2};
      else if (idx < nchunks)
        r[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(idx * 16), 0, kLoadPolicy));
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t idx = base + u * kThreads + threadIdx.x;
      if (idx < nchunks) __builtin_amdgcn_raw_buffer_store_b128(r[u], rd, (int)(idx * 16), 0, kStorePolicy);
    }
  }
}

// One kernel symbol per direction, so that profiles tell them apart.
// Workgroup g copies half g & 1 of item g >> 1; a grid smaller than
// 2 * n_items walks the halves with a stride of the grid size.
template <int MODE>
__device__ __forceinline__ void copy_all(const CopyArgs &a) {
  for (int g = blockIdx.x; g < 2 * a.n_items; g += gridDim.x) copy_rows<MODE>(a, g);
}
__global__ __launch_bounds__(kThreads) void kv_fetch_kernel(CopyArgs a) { copy_all<COPY_FETCH>(a); }
__global__ __launch_bounds__(kThreads) void kv_append_kernel(CopyArgs a) { copy_all<COPY_APPEND>(a); }
__global__ __launch_bounds__(kThreads) void kv_store_kernel(CopyArgs a) { copy_all<COPY_STORE>(a); }

// The overlapped stack's per-layer copy: fetch, append and store item
// halves in that order, strided over a capped grid.
__global__ __launch_bounds__(kThreads) void kv_layer_copy_kernel(LayerCopyArgs a) {
  const bool poison =
      a.fail_word != nullptr && __hip_atomic_load(a.fail_word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == a.fail_tag;
  const int n0 = 2 * a.part[0].n_items;
  const int n1 = n0 + 2 * a.part[1].n_items;
  const int n2 = n1 + 2 * a.part[2].n_items;
  for (int g = blockIdx.x; g < n2; g += gridDim.x) {
    if (g < n0)
      copy_rows<COPY_FETCH>(a.part[0], g, poison, a.nan2);
    else if (g < n1)
      copy_rows<COPY_APPEND>(a.part[1], g - n0, poison, a.nan2);
    else
      copy_rows<COPY_STORE>(a.part[2], g - n1);
  }
}

// Holds its stream until *counter >= value.  The poll is a relaxed
// device-scope load with a sleep between polls; the counter only rises.
__global__ __launch_bounds__(64) void slot_gate_kernel(const uint64_t *counter, uint64_t value, uint32_t *timeout,
                                                       uint64_t *fail_word, uint64_t fail_tag, int spin_limit) {
  if (threadIdx.x != 0) return;
  int spins = 0;
  while (__hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < value) {
    if (++spins > spin_limit) {
      __hip_atomic_store(timeout, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(fail_word, fail_tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    __builtin_amdgcn_s_sleep(8);
  }
}

// Fills n16 16-byte chunks with a repeated 16-bit pattern (the debug
// poisoning of an active slot before it is refilled).
__global__ __launch_bounds__(kThreads) void kv_fill_kernel(u32x4 *p, int64_t n16, uint32_t pattern2) {
  const u32x4 v = {pattern2, pattern2, pattern2, pattern2};
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n16; i += (int64_t)gridDim.x * kThreads)
    p[i] = v;
}

}  // namespace

hipError_t launch_kv_fill(void *p, size_t bytes, uint16_t pattern, hipStream_t stream) {
  const int64_t n16 = (int64_t)(bytes / 16);
  if (n16 <= 0) return hipSuccess;
  const int64_t want = (n16 + kThreads - 1) / kThreads;
  const unsigned blocks = (unsigned)(want < 4096 ? want : 4096);
  hipLaunchKernelGGL(kv_fill_kernel, dim3(blocks), dim3(kThreads), 0, stream, static_cast<u32x4 *>(p), n16,
                     (uint32_t)pattern * 0x10001u);
  return hipGetLastError();
}

int kv_copy_vgprs() {
  int m = 0;
  for (const void *f : {reinterpret_cast<const void *>(&kv_fetch_kernel), reinterpret_cast<const void *>(&kv_append_kernel),
                        reinterpret_cast<const void *>(&kv_store_kernel),
                        reinterpret_cast<const void *>(&kv_layer_copy_kernel)}) {
    hipFuncAttributes at{};
    if (hipFuncGetAttributes(&at, f) != hipSuccess) return -1;
    m = at.numRegs > m ? at.numRegs : m;
  }
  return m;
}

hipError_t launch_kv_copy(const CopyArgs &a, hipStream_t stream, size_t lds_reserve, int max_groups) {
  if (a.n_items <= 0) return hipSuccess;
  const int groups = max_groups > 0 && max_groups < 2 * a.n_items ? max_groups : 2 * a.n_items;
  const dim3 grid(groups), block(kThreads);
  if (a.mode == COPY_FETCH)
    hipLaunchKernelGGL(kv_fetch_kernel, grid, block, lds_reserve, stream, a);
  else if (a.mode == COPY_APPEND)
    hipLaunchKernelGGL(kv_append_kernel, grid, block, lds_reserve, stream, a);
  else
    hipLaunchKernelGGL(kv_store_kernel, grid, block, lds_reserve, stream, a);
  return hipGetLastError();
}

hipError_t launch_kv_layer_copy(const LayerCopyArgs &a, hipStream_t stream, size_t lds_reserve, int max_groups) {
  const int halves = 2 * (a.part[0].n_items + a.part[1].n_items + a.part[2].n_items);
  if (halves <= 0) return hipSuccess;
  const int groups = max_groups > 0 && max_groups < halves ? max_groups : halves;
  hipLaunchKernelGGL(kv_layer_copy_kernel, dim3(groups), dim3(kThreads), lds_reserve, stream, a);
  return hipGetLastError();
}

hipError_t launch_slot_gate(const uint64_t *counter, uint64_t value, uint32_t *timeout, uint64_t *fail_word,
                            uint64_t fail_tag, int spin_limit, hipStream_t stream) {
  hipLaunchKernelGGL(slot_gate_kernel, dim3(1), dim3(64), 0, stream, counter, value, timeout, fail_word, fail_tag,
                     spin_limit);
  return hipGetLastError();
}

}  // namespace sc
