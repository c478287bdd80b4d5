// Row-copy kernel behind the layer KV load (§3.2 "Layer Stream Cache", §3.3
// "KV Load"), the append of the new turn into the active buffer (§3.2) and
// the layer KV store back to donor blocks (§3.3 "KV Store").
//
// All three move whole token rows (n_kv_heads * head_dim bf16 = row_bytes)
// between a block of the block-major pool (§3.4) and a packed buffer, so one
// body serves them: workgroup 2*i copies item i's K rows, workgroup 2*i+1
// its V rows (a grid capped below 2 * n_items, as the overlapped layer
// stack launches it beside attention, strides over the item halves).  A
// block slice of one layer is contiguous in the pool (K half then V half,
// Eq. 1), and consecutive rows of a sequence are contiguous in the active
// buffer, so each item is one contiguous range on both sides.
//
// The overlapped layer stack launches all three of a layer in one grid
// (kv_layer_copy_kernel) after a one-wave gate kernel that waits on the
// device for the attention that last read the slot.
//
// HBM-bound: every lane moves 16-byte chunks with kUnroll loads in flight
// before the matching stores (one store or all of them in flight, see
// launch_kv_copy), through buffer resources over the item's two ranges.
// Both sides are streamed once per call: the loads are
// system-coherent and non-temporal (sc0 sc1 nt: no cache keeps the source),
// the stores non-temporal (nt), so neither evicts the attention's K/V
// working set from L2.  Measured on MI355X, every other combination of
// cached and non-temporal loads and stores is slower (up to a third with
// both cached).  The data a
// copy reads was written by earlier kernels, whose completion wrote it back
// beyond the caches.  Host-tier blocks are read or written through their
// device-visible pinned mapping, over the host link.
#include "sc_internal.h"

#include <map>
#include <mutex>
#include <tuple>

namespace sc {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 8;
// Buffer instruction cache-policy bits on gfx950: sc0 = 1, nt = 2, sc1 = 16.
constexpr int kLoadPolicy = 1 | 2 | 16;
constexpr int kStorePolicy = 2;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// A record of 32-bit fields read through the constant address space: the
// host writes the copy items before the launch and nothing writes them
// during it, so a uniform index gives one scalar load, the item stays in
// scalar registers and the buffer resources built from it need no
// per-lane loop.  (Read as ordinary global memory, the fields came back
// one dependent vector load at a time and every buffer access was wrapped
// in a loop over the distinct resources of the wave.)
typedef int32_t i32x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ CopyItem load_item(const CopyItem *p) {
  static_assert(sizeof(CopyItem) == sizeof(i32x8), "one 32-byte record");
  const i32x8 v = *(const __attribute__((address_space(4))) i32x8 *)p;
  CopyItem r;
  __builtin_memcpy(&r, &v, sizeof(r));
  return r;
}

// poison: write nan2 over the destination instead of copying (fetch and
// append into a slot whose gate timed out).  kSerialStores: one store in
// flight per wave (see launch_kv_copy).
template <int MODE, bool kSerialStores>
__device__ __forceinline__ void copy_rows(const CopyArgs &a, int g, bool poison = false, uint32_t nan2 = 0) {
  const int item_idx = g >> 1;
  const int is_v = g & 1;
  const CopyItem it = load_item(a.items + item_idx);
  if (MODE != COPY_APPEND && !((a.tier_mask >> it.tier) & 1)) return;
  // One item is at most 256 rows of one KV layer (under 4 MiB), so 32-bit
  // chunk indices and byte offsets cover it.
  const int nchunks = (int)(((int64_t)it.nrows * a.row_bytes) >> 4);
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
  const int bytes = nchunks * 16;
  // Lanes past the item's last chunk are not masked off: the buffer
  // resources end at the item's last byte, so their loads return zeros and
  // their stores are dropped by the hardware's range check.
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(src), (short)0, bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(dst, (short)0, bytes, 0x00020000);
  for (int base = 0; base < nchunks; base += kThreads * kUnroll) {
    u32x4 r[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int idx = base + u * kThreads + (int)threadIdx.x;
      if (poison)
        r[u] = u32x4{nan2, nan2, nan2, nan2};
      else
        r[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, idx * 16, 0, kLoadPolicy));
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int idx = base + u * kThreads + (int)threadIdx.x;
      if constexpr (kSerialStores) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __builtin_amdgcn_raw_buffer_store_b128(r[u], rd, idx * 16, 0, kStorePolicy);
    }
  }
}

// One kernel symbol per direction, so that profiles tell them apart.
// Workgroup g copies half g & 1 of item g >> 1; a grid smaller than
// 2 * n_items walks the halves with a stride of the grid size.
template <int MODE>
__device__ __forceinline__ void copy_all(const CopyArgs &a) {
  if (a.serial_stores)
    for (int g = blockIdx.x; g < 2 * a.n_items; g += gridDim.x) copy_rows<MODE, true>(a, g);
  else
    for (int g = blockIdx.x; g < 2 * a.n_items; g += gridDim.x) copy_rows<MODE, false>(a, g);
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
      copy_rows<COPY_FETCH, true>(a.part[0], g, poison, a.nan2);
    else if (g < n1)
      copy_rows<COPY_APPEND, true>(a.part[1], g - n0, poison, a.nan2);
    else
      copy_rows<COPY_STORE, true>(a.part[2], g - n1);
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

// Workgroups of a copy kernel that the device runs at once (all CUs),
// computed once per (device, kernel, LDS reservation).
int copy_resident_groups(const void *kernel, size_t lds_reserve) {
  static std::mutex mu;
  static std::map<std::tuple<int, const void *, size_t>, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  const auto key = std::make_tuple(dev, kernel, lds_reserve);
  std::lock_guard<std::mutex> lk(mu);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, lds_reserve) != hipSuccess)
    return 0;
  return cache[key] = cus * per_cu;
}

hipError_t launch_kv_copy(const CopyArgs &args, hipStream_t stream, size_t lds_reserve, int max_groups) {
  if (args.n_items <= 0) return hipSuccess;
  const int groups = max_groups > 0 && max_groups < 2 * args.n_items ? max_groups : 2 * args.n_items;
  const void *kernel = args.mode == COPY_FETCH    ? reinterpret_cast<const void *>(&kv_fetch_kernel)
                       : args.mode == COPY_APPEND ? reinterpret_cast<const void *>(&kv_append_kernel)
                                                  : reinterpret_cast<const void *>(&kv_store_kernel);
  // Store policy, by measurement: when the whole grid is resident at once
  // (one round of workgroups, e.g. the 8B shape's 32 MiB layer in 1024
  // workgroups) or runs capped beside attention, one store in flight per
  // wave (eight in flight: 11% slower there, and burstier writes slow the
  // attention beside them); with several rounds of workgroups (128-330 MiB
  // layers) eight in flight, 4-6% faster.
  CopyArgs a = args;
  a.serial_stores = (max_groups > 0 || groups <= copy_resident_groups(kernel, lds_reserve)) ? 1 : 0;
  const dim3 grid(groups), block(kThreads);
  if (a.mode == COPY_FETCH)
    hipLaunchKernelGGL(kv_fetch_kernel, grid, block, lds_reserve, stream, a);
  else if (a.mode == COPY_APPEND)
    hipLaunchKernelGGL(kv_append_kernel, grid, block, lds_reserve, stream, a);
  else
    hipLaunchKernelGGL(kv_store_kernel, grid, block, lds_reserve, stream, a);
  return hipGetLastError();
}

hipError_t launch_kv_layer_copy(const LayerCopyArgs &args, hipStream_t stream, size_t lds_reserve, int max_groups) {
  const int halves = 2 * (args.part[0].n_items + args.part[1].n_items + args.part[2].n_items);
  if (halves <= 0) return hipSuccess;
  // Beside attention: one store in flight per wave (see launch_kv_copy;
  // the kernel always stores that way).
  const LayerCopyArgs &a = args;
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
