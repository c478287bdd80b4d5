// Internal declarations shared by the host runtime (sc_api.cpp) and the
// kernel translation units (kv_copy.hip, attn_fwd.hip).  Not installed.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <map>
#include <set>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/swiftcache.h"

namespace sc {

// ---------------------------------------------------------------------------
// Error state
// ---------------------------------------------------------------------------
sc_status fail(sc_status st, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
sc_status fail_hip(hipError_t e, const char *what);
void clear_error();

#define SC_HIP(call)                                   \
  do {                                                 \
    hipError_t e_ = (call);                            \
    if (e_ != hipSuccess) return ::sc::fail_hip(e_, #call); \
  } while (0)

// ---------------------------------------------------------------------------
// Copy work items (fetch / append / store).  One item moves `nrows` token
// rows of K and, in a second workgroup, of V.
//   FETCH : pool tier `tier` at byte offset pool_off (+ layer slice) -> active
//           rows starting at act_row.
//   APPEND: k_new rows starting at src_row -> active rows starting at act_row.
//   STORE : k_new rows starting at src_row -> pool tier at pool_off (+ layer).
// ---------------------------------------------------------------------------
struct CopyItem {
  int64_t pool_off;   // bytes from the tier base to the first row (layer 0, K half)
  int64_t act_row;    // first row in the active buffer (FETCH/APPEND)
  int64_t src_row;    // first row of k_new / v_new (APPEND/STORE)
  int32_t nrows;
  int32_t tier;       // 0 = device tier, 1 = host tier
};
static_assert(sizeof(CopyItem) == 32, "CopyItem layout");

enum CopyMode { COPY_FETCH = 0, COPY_APPEND = 1, COPY_STORE = 2 };

struct CopyArgs {
  const CopyItem *items;
  int32_t n_items;
  int32_t mode;
  int64_t row_bytes;      // bytes of one token row of K (or V) of one layer
  int64_t layer_off;      // layer * slice_bytes
  int64_t v_half_off;     // slice_bytes / 2: V half of a block slice
  char *tier_base[2];     // device-visible bases of the device and host tiers
  int32_t tier_mask;      // FETCH / STORE: bit t set = copy the items of tier t
  char *act_k;
  char *act_v;
  const char *new_k;
  const char *new_v;
  int32_t serial_stores;  // set by the launch: one store in flight per wave
};

// lds_reserve: bytes of LDS each copy workgroup reserves without using them
// (limits how many copy workgroups share a CU with attention; 0 = none).
// max_groups > 0 caps the grid; the workgroups then loop over the items.
hipError_t launch_kv_copy(const CopyArgs &a, hipStream_t stream, size_t lds_reserve = 0, int max_groups = 0);
// bytes (a multiple of 16, 16-byte aligned p) filled with a 16-bit pattern.
hipError_t launch_kv_fill(void *p, size_t bytes, uint16_t pattern, hipStream_t stream);

// One layer's fetch, append and store in one launch (overlapped layer
// stack): workgroups take fetch item halves first, then append, then store.
// If *fail_word == fail_tag when a workgroup starts (the slot gate below
// timed out for this layer), fetch and append write the NaN pattern nan16
// into the slot instead of data.
struct LayerCopyArgs {
  CopyArgs part[3];                // COPY_FETCH, COPY_APPEND, COPY_STORE
  const uint64_t *fail_word;       // nullable
  uint64_t fail_tag;
  uint32_t nan2;                   // nan16 repeated in both halves
};
hipError_t launch_kv_layer_copy(const LayerCopyArgs &a, hipStream_t stream, size_t lds_reserve, int max_groups);
// One-wave kernel that holds the stream until *counter >= value (the
// attention workgroups that read a slot are all done with it), polling at
// most spin_limit times; on time-out it sets *timeout and *fail_word =
// fail_tag and ends.  One wave cannot keep an attention workgroup off a CU.
hipError_t launch_slot_gate(const uint64_t *counter, uint64_t value, uint32_t *timeout, uint64_t *fail_word,
                            uint64_t fail_tag, int spin_limit, hipStream_t stream);

// ---------------------------------------------------------------------------
// Attention work decomposition
// ---------------------------------------------------------------------------
struct SeqDesc {
  int32_t cu_q;       // first query row of the sequence
  int32_t cu_k;       // first active-buffer row of the sequence
  int32_t prefix;     // P
  int32_t n_new;      // N
  int32_t n_splits;   // key splits of every query tile of this sequence
  int32_t rc_keys;    // leading keys read in place from the regular cache
  int32_t rc_off;     // first entry of the sequence in AttnArgs::rc_ids
  int32_t q_off;      // first row of the sequence's queries in q / out (== cu_q unless
                      // the plan covers one chunk of the new turn)
};
static_assert(sizeof(SeqDesc) == 32, "SeqDesc layout");

// One workgroup: rows (query, head) = queries [q0, q0 + nq) of sequence `seq`
// times the `group` query heads of KV head `kvh`; keys [k_begin, k_end).
struct WorkItem {
  int32_t seq;        // -1: padding slot, the workgroup exits
  int32_t kvh;
  int32_t q0;
  int32_t nq;
  int32_t k_begin;
  int32_t k_end;
  int32_t split;
  int32_t paged;      // 1: keys [k_begin, k_end) come from the regular cache in place
};
static_assert(sizeof(WorkItem) == 32, "WorkItem layout");

struct AttnArgs {
  const uint16_t *q;
  const uint16_t *k;
  const uint16_t *v;
  uint16_t *out;
  float *lse;             // nullable, [Hq][total_q]
  const WorkItem *items;
  const SeqDesc *seqs;
  uint16_t *part_o;       // [max_splits][total_q][Hq][D] normalised partial outputs, element type
  float *part_lse;        // [max_splits][total_q][Hq]
  int32_t n_seqs;
  int32_t total_q;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t group;
  int32_t rows_q;         // queries per workgroup tile
  int32_t dtype;          // sc_dtype of q, K, V and out
  float scale_log2;       // softmax scale * log2(e)
  // Optional device-side dependency (overlapped layer stack): before reading
  // K/V, each workgroup waits until *ready_flag >= ready_value, polling at
  // most ready_spin_limit times; on time-out it sets *ready_timeout and
  // writes NaN rows instead of results.  ready_flag == nullptr: no wait.
  const uint64_t *ready_flag;
  uint64_t ready_value;
  uint32_t *ready_timeout;
  int32_t ready_spin_limit;
  // Nonzero: once the flag is seen, an agent-scope acquire (invalidates
  // this XCD's L2) before any K/V read.  For stacks in which another kernel
  // writes the slot after this kernel's dispatch (the debug poisoning):
  // that kernel's lines may stay valid in this XCD's L2 while the copy
  // kernel's newer data was written from another XCD.
  int32_t ready_acquire;
  // Optional: every workgroup adds 1 to *done_counter once it has finished
  // reading K/V (after its last key tile; timed-out and empty workgroups
  // too), so that the next refill of the slot can wait on the device.
  uint64_t *done_counter;
  // Regular cache (paged items): block i of sequence s is local block
  // rc_ids[seqs[s].rc_off + i] of the tier at rc_base, whose layer-l K rows
  // start at rc_base + id * rc_block_elems + rc_layer_elems (V rows
  // rc_half_elems further); block_shift = log2(block_size).
  const uint16_t *rc_base;
  const int32_t *rc_ids;
  int64_t rc_block_elems;
  int64_t rc_layer_elems;
  int64_t rc_half_elems;
  int32_t block_shift;
  // Implicit work list (one sequence, no regular cache; the allocation-free
  // entry point): items == nullptr and seqs == nullptr.  The sequence is
  // seq0; workgroup w takes item g = (w % 8) * imp_per_xcd + w / 8 of the
  // list ordered (KV head, query tile, key split), so consecutive items --
  // one KV head's -- share an XCD.  Split sp of a tile with `keys` keys
  // covers tiles [sp * t / S, (sp + 1) * t / S) of its t = ceil(keys / 32)
  // key tiles, exactly as plan_attention divides them.
  SeqDesc seq0;
  int32_t imp_tiles;      // query tiles per KV head
  int32_t imp_splits;     // key splits per query tile (S)
  int32_t imp_per_xcd;    // items per XCD (grid = 8 * imp_per_xcd)
  // Optional deferred merge (layer stack, same plan for every layer): once
  // its own item is done, a workgroup claims chunks of rows of the previous
  // layer's split partials (dm_part_o, dm_part_lse, laid out like part_o /
  // part_lse; at most dm_max_splits splits per row) from *dm_counter (zero
  // before the launch) and merges them into dm_out exactly as
  // attn_merge_kernel would, until every chunk is claimed; workgroups that
  // finish early take more.  dm_out == nullptr: none.
  const uint16_t *dm_part_o;
  const float *dm_part_lse;
  uint16_t *dm_out;
  uint32_t *dm_counter;
  int32_t dm_max_splits;
};

// Tile geometry the planner and the kernel agree on.
constexpr int kAttnRows = 256;   // (query, head) rows per workgroup
constexpr int kAttnKeyTile = 32; // keys per LDS tile
// The attention kernel addresses one sequence's key rows (all KV heads)
// with signed 32-bit byte offsets, including the loads of up to a few tiles
// past the last one (which the buffer range turns into zeros): a sequence
// must fit in 2 GiB of keys less this many tokens.
constexpr int kKeyOffsetMarginTokens = 8 * kAttnKeyTile;
inline bool keys_fit_offsets(int64_t tokens, int n_kv_heads, int head_dim) {
  const int64_t row_bytes = (int64_t)n_kv_heads * head_dim * 2;   // head_dim is 64 or 128
  return row_bytes > 0 && tokens >= 0 && tokens + kKeyOffsetMarginTokens <= (((int64_t)1 << 31) - 1) / row_bytes;
}
constexpr int kAttnMaxSplits = 16; // key splits per sequence (merge kernel bound)
// Polls of the ready flag before an attention workgroup gives up (about a
// second), and the limit a forced time-out uses.
constexpr int kAttnReadySpinLimit = 1 << 22;
constexpr int kAttnTestSpinLimit = 256;

hipError_t launch_attn_fwd(const AttnArgs &a, int head_dim, int n_items, hipStream_t stream);
// Allocation-free calls: the device address of this device's file-scope
// split-key scratch array (looked up once per device, with that device
// current) and its size in bytes.
hipError_t noalloc_scratch(int device, void **ptr, size_t *bytes);
size_t attn_fwd_lds_bytes(int head_dim);
int attn_fwd_vgprs(int head_dim);   // per work item, -1 if unknown
int kv_copy_vgprs();                // largest of the three copy kernels
hipError_t launch_attn_merge(const AttnArgs &a, int head_dim, hipStream_t stream);

struct AttnPlan {
  bool paged = false;              // some items read the regular cache in place
  int group = 0;
  int rows_q = 0;
  int max_splits = 1;
  int n_items = 0;                 // grid size (includes padding slots)
  int n_real_items = 0;
  std::vector<WorkItem> items;
  std::vector<SeqDesc> seqs;
  WorkItem *d_items = nullptr;
  SeqDesc *d_seqs = nullptr;
  int64_t total_q = 0;
};

// Builds the work list for a batch (host only; no device work).
// `slots` = workgroups the device runs at once (CUs x resident workgroups).
// rc_keys[b] (may be empty = none) leading keys of sequence b are read in
// place from the regular cache: they get items of their own (a split
// boundary at rc_keys[b]).  cu_k / q_off (may be empty = packed from P + N
// and N): the sequence's first active-buffer row and first q / out row,
// for plans over one chunk of a longer new turn.
void plan_attention(const std::vector<int32_t> &P, const std::vector<int32_t> &N, int n_q_heads,
                    int n_kv_heads, int slots, AttnPlan *plan, const std::vector<int32_t> &rc_keys = {},
                    const std::vector<int32_t> &rc_off = {}, const std::vector<int32_t> &cu_k = {},
                    const std::vector<int32_t> &q_off = {});
int attn_slots(int device);


}  // namespace sc

// ---------------------------------------------------------------------------
// Opaque objects
// ---------------------------------------------------------------------------
struct sc_pool {
  sc_pool_desc desc;
  char *rc_base = nullptr;        // regular-cache tier (device)
  bool own_rc = false;
  // Elastic HBM tier (sc_pool_resize): ids [0, dev_lent) are usable; the
  // largest HBM id each live table references (-1: none), for the shrink check.
  int64_t dev_lent = 0;
  std::mutex mu;
  std::multiset<int64_t> live_max_dev;
  char *dev_base = nullptr;
  // Library-owned HBM tier backed chunk by chunk: dev_base starts a reserved
  // virtual range of vmm_reserved bytes; physical chunks of vmm_chunk_bytes
  // (whole blocks, a multiple of the allocation granularity) are mapped at
  // its start, vmm_handles[i] at dev_base + i * vmm_chunk_bytes.
  // sc_pool_resize appends or releases chunks at the tail; the mapped ones
  // never move.
  bool vmm = false;
  size_t vmm_reserved = 0;
  size_t vmm_chunk_bytes = 0;
  int64_t vmm_chunk_blocks = 0;
  std::vector<hipMemGenericAllocationHandle_t> vmm_handles;
  char *host_base = nullptr;      // host address of the host tier
  char *host_dev = nullptr;       // device-visible address of the host tier
  bool own_dev = false;
  bool own_host = false;
  size_t slice_bytes = 0;
  size_t block_bytes = 0;
  size_t row_bytes = 0;
};

struct sc_table {
  sc_pool *pool = nullptr;
  int64_t max_dev_id = -1;           // largest HBM block id in the table
  std::vector<int32_t> rc_keys, rc_off; // per sequence: keys read in place, offset into rc ids
  std::vector<int32_t> h_rc_ids;     // local regular-cache block index per leading block
  int32_t *d_rc_ids = nullptr;
  int32_t batch = 0;
  std::vector<int32_t> P, N;
  std::vector<int64_t> cu_q, cu_k;
  int64_t total_q = 0, total_kv = 0;
  std::vector<sc::CopyItem> h_items; // host copy (source of the upload)
  sc::CopyItem *d_items = nullptr;   // fetch items, then append, then store
  int32_t n_fetch = 0, n_append = 0, n_store = 0;
  int32_t n_fetch_host = 0;          // fetch items that read the host tier
  std::mutex mu;
  // keyed by (n_q_heads, slots, chunk tokens, chunk index); chunk tokens 0:
  // the whole new turn
  std::map<std::tuple<int, int, int, int>, sc::AttnPlan> plans;
  // Overlapped stack: [0] = count of layers whose active slot is filled
  // (written by the copy stream, polled by attention), [1] = time-out flag,
  // [2] = forward workgroups of the running stack done with their slot
  // (reset at its start, polled by the slot gates), [3] = tag of the last
  // layer whose slot gate timed out.
  uint64_t *d_sync = nullptr;
  uint64_t sync_gen = 1;
  // Overlapped stacks on one table share d_sync, so their device work must
  // not interleave: stack_mu is held while one is enqueued, and each starts
  // after the previous one's end event (last_overlap, recorded on its
  // caller's compute stream).
  std::mutex stack_mu;
  hipEvent_t last_overlap = nullptr;
  bool last_overlap_recorded = false;
};
