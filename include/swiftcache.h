/*
 * swiftcache.h — C ABI of the MI355X layer-wise prefix-KV reload and prefill
 * attention library (libswiftcache.so, gfx950).
 *
 * The library implements the per-layer hot path of a layer stream cache
 * (paper §3.2 "Layer Stream Cache"): a conversation's cached prefix KV lives
 * in a donor pool in block-major layout (§3.4); before each layer's attention
 * the layer's prefix blocks are loaded through a block table into a local
 * buffer that holds only the active layer (§3.2, §3.3 "KV Load"); the new
 * turn's K/V are written into that buffer; causal GQA prefill attention runs
 * over prefix + new tokens (§2.2); the new turn's K/V are written back to
 * donor blocks (§3.3 "KV Store").
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Element type of every KV, q and output tensor: the pool's sc_dtype,
 *    bf16 by default or IEEE fp16 (raw 16-bit patterns either way);
 *    sc_prefill_attn is bf16, sc_prefill_attn_f16 its fp16 twin.
 *  - Device pointers are HIP device addresses on the pool's device.  Host
 *    arrays (block tables, lengths) are read synchronously during the call
 *    and may be freed when it returns.
 *  - Alignment: every pointer to K/V, q, k_new, v_new, output or pool-tier
 *    data must be 16-byte aligned (the kernels move 16-byte chunks), lse
 *    4-byte aligned; a misaligned pointer returns SC_ERR_INVALID.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *    device work is enqueued asynchronously on it; no call synchronises the
 *    caller's stream.  Caller-owned buffers must stay alive until that work
 *    has completed.
 *  - Errors: argument, shape and range errors are detected before any work
 *    is enqueued and return a negative sc_status; sc_last_error() then gives
 *    a message (thread-local, valid until the next call on the thread).
 *    A failed kernel launch returns SC_ERR_HIP.  Faults during asynchronous
 *    execution surface at the caller's next synchronisation.
 *  - Packed varlen layout: sequence b of a batch owns query rows
 *    [cu_q[b], cu_q[b] + N_b) of q/out/k_new/v_new and active-buffer rows
 *    [cu_k[b], cu_k[b] + P_b + N_b), prefix first, where
 *    cu_q = exclusive prefix sum of N_b and cu_k = exclusive prefix sum of
 *    P_b + N_b.
 *  - Thread safety: distinct objects may be used from distinct threads.
 *    Calls that enqueue work on the same stream are ordered by the stream.
 */
#ifndef SWIFTCACHE_H
#define SWIFTCACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SC_OK = 0,
  SC_ERR_INVALID = -1,      /* null pointer, bad enum/flag, malformed table  */
  SC_ERR_OOM = -2,          /* device or pinned host allocation failed       */
  SC_ERR_HIP = -3,          /* a HIP runtime call or kernel launch failed    */
  SC_ERR_RANGE = -4,        /* index or size outside the object's bounds     */
  SC_ERR_UNSUPPORTED = -5   /* shape the kernels are not built for           */
} sc_status;

/* Element type of every K/V, q, k_new, v_new and output element of a pool
 * (and of the active buffers used with it): bf16, or IEEE fp16 as the paper
 * serves its models (§5).  Attention accumulates in fp32 for both; the
 * probabilities of the PV product and the output are rounded to the same
 * type (round to nearest even). */
typedef enum {
  SC_DTYPE_BF16 = 0,
  SC_DTYPE_F16 = 1
} sc_dtype;

typedef struct sc_pool sc_pool;     /* opaque, library-owned */
typedef struct sc_table sc_table;   /* opaque, library-owned */

/*
 * Donor pool description.  Eq. 1 (§3.2) gives the bytes of one block of one
 * layer: slice_bytes = 2 * block_size * n_kv_heads * head_dim * 2 (16-bit
 * elements).
 * Block-major layout (§3.4), with Eq. 1's K/V factor made explicit and the
 * K half first:
 *     pool[n_blocks][n_layers][2][block_size][n_kv_heads][head_dim]
 * so one block occupies block_bytes = n_layers * slice_bytes contiguous
 * bytes, and its layer-l slice starts at l * slice_bytes.
 *
 * Block ids [0, n_device_blocks) address the HBM tier (a device allocation
 * standing in for a co-located model's idle KV memory); ids
 * [n_device_blocks, n_device_blocks + n_host_blocks) address the host-pinned
 * tier, whose block k is id n_device_blocks + k; ids
 * [n_device_blocks + n_host_blocks, ... + n_rc_blocks) address the regular
 * cache (§3.2 "Regular Cache"): full-layer blocks in the master's own HBM,
 * which attention reads in place through the block table instead of
 * fetching them (needs a power-of-two block_size of at least 16 and blocks
 * under 4 GiB over all layers; SC_ERR_UNSUPPORTED otherwise).
 *
 * device_base / host_base: when non-NULL the pool indexes caller-owned
 * memory of at least n_device_blocks * block_bytes (device memory on
 * `device`) and n_host_blocks * block_bytes (pinned host memory from
 * hipHostMalloc, mapped for device access) bytes, and never frees it.  When
 * NULL the library allocates the tier and frees it in sc_pool_destroy: the
 * host tier with hipHostMalloc; the HBM tier as one reserved virtual address
 * range of the full capacity whose physical memory is mapped in chunks of
 * whole blocks (hipMemCreate / hipMemMap, plain cached device memory), so
 * that sc_pool_resize really appends and releases memory, or, where the
 * runtime lacks virtual memory management, with one hipMalloc.  rc_base
 * likewise for n_rc_blocks * block_bytes of device memory (hipMalloc).
 */
typedef struct {
  int32_t n_layers;
  int32_t n_kv_heads;
  int32_t head_dim;          /* 64 or 128 */
  int32_t block_size;        /* tokens per block, 1..256 */
  int64_t n_device_blocks;
  int64_t n_host_blocks;
  int32_t device;            /* HIP device ordinal */
  int32_t dtype;             /* sc_dtype (0 = bf16) */
  void *device_base;         /* optional caller-owned HBM tier */
  void *host_base;           /* optional caller-owned pinned host tier */
  int64_t n_rc_blocks;       /* regular-cache blocks (0: none) */
  void *rc_base;             /* optional caller-owned regular-cache tier */
} sc_pool_desc;

typedef struct {
  void *device_base;         /* HBM tier base (device address) */
  void *host_base;           /* pinned host tier base (host address), or NULL */
  size_t slice_bytes;        /* Eq. 1: bytes of one block of one layer */
  size_t block_bytes;        /* n_layers * slice_bytes */
  size_t row_bytes;          /* one token of one layer, K or V: n_kv_heads*head_dim*2 */
  int64_t n_device_blocks;   /* HBM tier capacity (fixes the id split)   */
  int64_t n_host_blocks;
  int64_t device_blocks_lent;/* HBM blocks currently usable (sc_pool_resize), <= n_device_blocks */
  void *rc_base;             /* regular-cache tier base (device address), or NULL */
  int64_t n_rc_blocks;
  int32_t dtype;             /* sc_dtype */
  int64_t device_bytes_mapped;  /* physical bytes behind the HBM tier now (0: caller-owned) */
  int64_t device_chunk_blocks;  /* blocks per physical chunk of an elastic tier (0: one allocation) */
} sc_pool_layout;

/* Active-layer buffer (the layer stream cache slot, §3.2): caller-owned
 * device arrays K and V, each [capacity_tokens][n_kv_heads][head_dim] of the
 * pool's element type. */
typedef struct {
  void *k;
  void *v;
  int64_t capacity_tokens;
} sc_active;

/* Create a pool (see sc_pool_desc).  Errors: SC_ERR_INVALID for a null
 * argument, non-positive sizes or an unknown dtype; SC_ERR_UNSUPPORTED for a
 * head_dim other than 64/128; SC_ERR_OOM when an allocation fails. */
sc_status sc_pool_create(const sc_pool_desc *desc, sc_pool **out);

/* Free a pool and any tiers it allocated.  Call only after every stream that
 * used it has drained.  NULL is ignored. */
void sc_pool_destroy(sc_pool *pool);

/* Bases and strides of the pool (for filling or reading it). */
sc_status sc_pool_layout_get(const sc_pool *pool, sc_pool_layout *out);

/*
 * Block table of a batch of conversations: the master's replica of the donor
 * block table (§3.5).  Host arrays, copied during the call:
 *   prefix_len[batch]  P_b >= 0 cached tokens;   new_len[batch]  N_b >= 0;
 *   cu_blocks[batch+1] offsets into block_ids; sequence b owns exactly
 *                      ceil((P_b + N_b) / block_size) entries, in token
 *                      order: logical token t lives in block
 *                      block_ids[cu_blocks[b] + t / block_size], row
 *                      t % block_size.  The new turn continues the last,
 *                      possibly partial, prefix block.
 *   block_ids[...]     pool block ids, each in range and used at most once
 *                      within the table.  Regular-cache ids may only be the
 *                      leading entries of a sequence and only for blocks the
 *                      prefix fills completely (R_b * block_size <= P_b): those
 *                      R_b blocks are read in place by attention and never
 *                      fetched, stored or appended to.
 * The table copies its index arrays to the device with hipMemcpyAsync on
 * `stream` (work issued on other streams must be ordered after it).
 * Errors: SC_ERR_INVALID (null pointer, batch <= 0, negative length, wrong
 * entry count, duplicate id, a regular-cache id after a non-regular one or
 * in a partially filled block), SC_ERR_RANGE (id outside the pool, or an HBM
 * id beyond the blocks the pool lends, see sc_pool_resize).
 */
sc_status sc_table_create(sc_pool *pool, int32_t batch, const int32_t *block_ids,
                          const int32_t *cu_blocks, const int32_t *prefix_len,
                          const int32_t *new_len, void *stream, sc_table **out);
void sc_table_destroy(sc_table *table);

/* Totals of a table: sum N_b (query rows) and sum (P_b + N_b) (active rows). */
sc_status sc_table_totals(const sc_table *table, int64_t *total_q, int64_t *total_kv);

/*
 * KV Load of one layer (§3.2, §3.3): for every sequence b and prefix token
 * t < P_b, copy K and V of token t of layer `layer` from its pool block to
 * rows cu_k[b] + t of dst->k and dst->v.  Token-exact: a partial last prefix
 * block copies P_b mod block_size rows; rows of new tokens are not written.
 * Host-tier blocks are read by the kernel over the host link (zero-copy).
 * Regular-cache blocks are not copied (attention reads them in place), so
 * their rows of dst keep whatever they held.  The pool is only read.
 * Errors: SC_ERR_INVALID (null), SC_ERR_RANGE (layer outside [0, n_layers)
 * or sum(P+N) > dst->capacity_tokens).
 */
sc_status sc_fetch_layer_kv(sc_pool *pool, const sc_table *table, int32_t layer,
                            const sc_active *dst, void *stream);

/*
 * The same KV Load with the host tier moved by the DMA engines instead of
 * the kernel (the PCIe reload of §1): each host-tier block's K and V halves
 * of the layer are two host-to-device copies (one hipMemcpyBatchAsync call
 * for all of them, or, with per_copy_calls != 0, one hipMemcpyAsync call
 * each); device-tier blocks are copied by the fetch kernel as above.  In
 * the block-major layout one layer's slice of a block is never contiguous
 * with another block's, so copies cannot be merged across blocks.  Same
 * result, arguments and errors as sc_fetch_layer_kv, plus
 * SC_ERR_UNSUPPORTED when per_copy_calls == 0 and the HIP runtime loaded in
 * the process has no hipMemcpyBatchAsync.
 */
sc_status sc_fetch_layer_kv_dma(sc_pool *pool, const sc_table *table, int32_t layer,
                                const sc_active *dst, int32_t per_copy_calls, void *stream);

/*
 * Append the new turn (§3.2: new entries are written into the active
 * buffer): rows cu_q[b] + i of k_new / v_new ([sum N][n_kv_heads][head_dim]
 * the pool's element type, device) go to rows cu_k[b] + P_b + i of dst->k /
 * dst->v.
 * Errors: as sc_fetch_layer_kv.
 */
sc_status sc_append_new_kv(sc_pool *pool, const sc_table *table, const void *k_new,
                           const void *v_new, const sc_active *dst, void *stream);

/*
 * Causal GQA prefill attention of one sequence (§2.2; GQA as in §5):
 *   out[i][h][:] = sum_{j <= P + i} softmax_j(scale * q[i][h] . k[j][g]) v[j][g]
 *   with g = h / (n_q_heads / n_kv_heads), for i < new_len, h < n_q_heads.
 * q, out: [new_len][n_q_heads][head_dim] bf16; k_active, v_active:
 * [prefix_len + new_len][n_kv_heads][head_dim] bf16 (the prefix rows then
 * the new rows).  scale <= 0 selects 1/sqrt(head_dim).  lse (nullable):
 * float [n_q_heads][new_len], the natural-log log-sum-exp of each row's
 * scaled scores.  Arithmetic: bf16 MFMA products, fp32 accumulation and
 * softmax, probabilities rounded to bf16 for the PV product, output rounded
 * to nearest even.  The library may use a device workspace of its own for
 * split-key partials (one per device and stream, grown on demand).
 * Errors: SC_ERR_INVALID (null, negative length, n_q_heads not a multiple
 * of n_kv_heads), SC_ERR_UNSUPPORTED (head_dim not 64/128, group > 16, or
 * (prefix_len + new_len + 256) x n_kv_heads x head_dim x 2 bytes of keys
 * reaching 2 GiB: key rows are addressed with signed 32-bit offsets, the
 * loads of a few tiles past the last one included; the same bound applies
 * to every sequence of the varlen, layer and stack calls).
 * new_len == 0 is a no-op.
 */
sc_status sc_prefill_attn(const void *q, const void *k_active, const void *v_active,
                          int32_t prefix_len, int32_t new_len, int32_t n_q_heads,
                          int32_t n_kv_heads, int32_t head_dim, float scale, void *out,
                          float *lse, void *stream);

/* The same with IEEE fp16 q, K, V and out (the paper's serving precision,
 * §5): fp16 MFMA products, fp32 accumulation and softmax, probabilities
 * rounded to fp16 for the PV product, output rounded to nearest even.
 * Arguments and errors as sc_prefill_attn. */
sc_status sc_prefill_attn_f16(const void *q, const void *k_active, const void *v_active,
                              int32_t prefix_len, int32_t new_len, int32_t n_q_heads,
                              int32_t n_kv_heads, int32_t head_dim, float scale, void *out,
                              float *lse, void *stream);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, arithmetic, work decomposition and result (bit for bit) as
 * sc_prefill_attn, but the call allocates nothing: no hipMalloc, hipFree or
 * other allocating routine, and no device work list (each workgroup derives
 * its (KV head, query tile, key split) from its index).  The split-key
 * partials live in a file-scope device array of 64 MiB that the library's
 * code object holds on every device it runs on until the process ends.
 * That array is shared by every call on the device and keeps the last
 * call's contents; calls that overlap on one device race on it (issue them
 * on one stream, or serialise them).
 * Errors: as sc_prefill_attn, plus SC_ERR_RANGE when the call's key splits
 * need more than the 64 MiB of partials (splits x new_len x n_q_heads x
 * (2 head_dim + 4) bytes) or more than 4096 (query tile, split) pairs.
 */
sc_status sc_prefill_attn_noalloc(const void *q, const void *k_active, const void *v_active,
                                  int32_t prefix_len, int32_t new_len, int32_t n_q_heads,
                                  int32_t n_kv_heads, int32_t head_dim, float scale, void *out,
                                  float *lse, void *stream);

/* Host only: the key-split count sc_prefill_attn_noalloc uses for one
 * sequence on `slots` resident workgroups (<= 0: 256), which equals the
 * split count sc_attn_plan_query reports for the same sequence.
 * Errors: SC_ERR_INVALID (null splits, negative length, heads),
 * SC_ERR_RANGE (shape beyond the allocation-free planner's buffers). */
sc_status sc_attn_noalloc_splits(int32_t prefix_len, int32_t new_len, int32_t n_q_heads,
                                 int32_t n_kv_heads, int32_t slots, int32_t *splits);

/* The same attention for every sequence of a table (packed varlen layout)
 * at layer `layer`: q, out [sum N][n_q_heads][head_dim]; kv = the active
 * buffer filled by sc_fetch_layer_kv + sc_append_new_kv; lse (nullable)
 * [n_q_heads][sum N].  Keys in the table's regular-cache blocks are read in
 * place from layer `layer` of the pool's regular-cache tier (their rows of
 * kv are not read); the partial results over those keys and over the rest
 * are combined exactly by their log-sum-exp.
 * Errors: as sc_prefill_attn, plus SC_ERR_RANGE (layer out of range). */
sc_status sc_prefill_attn_varlen(sc_pool *pool, const sc_table *table, int32_t layer, const void *q,
                                 const sc_active *kv, int32_t n_q_heads, float scale,
                                 void *out, float *lse, void *stream);

/*
 * KV Store of one layer (§3.3): write row cu_q[b] + i of k_new / v_new to
 * logical position P_b + i of sequence b's block table, layer `layer`.
 * Only those rows of the pool change.  Host-tier blocks are written over the
 * host link.
 * Errors: SC_ERR_INVALID (null), SC_ERR_RANGE (layer out of range).
 */
sc_status sc_store_layer_kv(sc_pool *pool, const sc_table *table, int32_t layer,
                            const void *k_new, const void *v_new, void *stream);

/*
 * The whole layer stack with layer-wise pipelining (§3.3).  Per layer l, slot
 * s = l % 2 of `slots`:
 *   copy stream:    wait until attention(l-2) released slot s; fetch(l),
 *                   append(l) into slot s and store(l); mark slot s ready.
 *   compute stream: wait for slot s; attention(l) into out_per_layer[l];
 *                   release slot s.
 * so the fetch of layer l+1 runs while layer l's attention runs.  Two slots
 * are needed because this path has no FFN to hide the load behind (the
 * paper loads layer i while the FFN of layer i-1 runs).  On return all work
 * is enqueued and the compute stream is ordered after every store.
 * "Wait for slot s" is done by the attention kernel itself on a device
 * counter the copy stream advances (no stream-level wait in front of every
 * attention), and "wait until released" by a one-wave kernel on the copy
 * stream polling a count of finished attention workgroups, whenever a copy
 * workgroup can always run beside an attention workgroup (and kernel
 * dispatches are not serialised, see SC_STACK_EVENT_WAIT); otherwise both
 * are stream event waits.  The device waits are bounded (about a second); an
 * attention workgroup that gives up writes NaN rows, and a copy whose wait
 * gave up writes NaN into the slot instead of K/V, so a lost dependency is
 * visible in the output, never silent.  Overlapped
 * stacks on one table share its slot counter, so the library runs them one
 * after another on the device even when they are enqueued from different
 * threads or caller streams (each starts after the previous one ended).
 * When the attention plan splits key ranges, layer l's split partials are
 * merged by the forward kernel of layer l+1 (its workgroups take chunks of
 * rows once their own work items are done) and the last layer's by one
 * merge kernel; out_per_layer[l] is therefore complete only when the whole
 * stack is, which is when the compute stream reaches the end of the stack.
 * The partials use the library's split-key workspace of the attention
 * stream (two layers' worth while the stack is enqueued).
 * Arrays of per-layer device pointers (host arrays of length n_layers):
 *   q_per_layer, knew_per_layer, vnew_per_layer, out_per_layer.
 * flags: SC_STACK_OVERLAP (two streams, two slots), SC_STACK_SERIAL
 * (everything on `compute`, slot 0 only), SC_STACK_ATTN_ONLY (attention
 * only, over whatever the slots hold: the reference point for the overlap
 * overhead), optionally | SC_STACK_NO_STORE.  `copy` may be NULL unless
 * SC_STACK_OVERLAP is set.
 * SC_STACK_DEBUG_POISON (overlapped or serial): before each layer's fetch
 * the slot it fills is overwritten with quiet-NaN patterns (bf16 0x7FC0,
 * fp16 0x7E00), on the stream that then fetches into it, so an attention
 * that read a slot before its fetch and append had landed (a lost ordering)
 * would produce NaN rows instead of another layer's plausible values.
 * Costs one slot-sized fill per layer; for tests.
 * SC_STACK_TEST_NEVER_READY (with SC_STACK_OVERLAP only, for tests of the
 * failure path): every attention kernel waits for a slot count the copy
 * stream never reaches and gives up after a few hundred polls, so its rows
 * come out NaN and sc_table_stack_status reports the time-out; every kernel
 * still exits.  SC_ERR_UNSUPPORTED if this stack would use the stream-level
 * wait (no device-side wait to time out).
 * SC_STACK_TEST_NEVER_FREE (likewise): every wait for a slot's release
 * (layers 2 and up) waits for a count the attention never reaches and gives
 * up after a few hundred polls; those layers' slots are filled with NaN, so
 * their rows come out NaN (layers whose slot was refilled while they read it
 * may too), and sc_table_stack_status reports the time-out.
 * SC_STACK_EVENT_WAIT (with SC_STACK_OVERLAP): both directions wait on
 * stream events instead of on the device.  The library also chooses this
 * by itself when the environment serialises kernel dispatches (the ROCm
 * profiler collecting counters, AMD_SERIALIZE_KERNEL or HIP_LAUNCH_BLOCKING
 * set): a device-side wait needs the copy kernel to run while the attention
 * kernel holds the GPU.
 */
enum {
  SC_STACK_OVERLAP = 0,
  SC_STACK_SERIAL = 1,
  SC_STACK_ATTN_ONLY = 2,
  SC_STACK_MODE_MASK = 3,
  SC_STACK_NO_STORE = 4,
  SC_STACK_TEST_NEVER_READY = 8,
  SC_STACK_DEBUG_POISON = 16,
  SC_STACK_TEST_NEVER_FREE = 32,
  SC_STACK_EVENT_WAIT = 64
};
sc_status sc_prefill_stack(sc_pool *pool, const sc_table *table, int32_t n_layers,
                           const void *const *q_per_layer, const void *const *knew_per_layer,
                           const void *const *vnew_per_layer, void *const *out_per_layer,
                           const sc_active *slots /* [2] */, int32_t n_q_heads, float scale,
                           uint32_t flags, void *compute_stream, void *copy_stream);

/*
 * The same layer stack with the new turn processed in chunks of at most
 * chunk_tokens tokens per sequence, for very long new turns (the paper does
 * not describe chunking): each layer's slot is fetched and appended once,
 * then attention runs one launch per chunk c over that same slot, chunk c's
 * queries (new tokens [c*C, min(N_b, (c+1)*C)) of each sequence) seeing the prefix
 * and the earlier chunks.  The result equals sc_prefill_stack's (same
 * definition; only the rounding order of the split-key merge differs);
 * chunking bounds the split-key workspace and the length of any single
 * launch to those of a C-token turn.  Arguments as sc_prefill_stack.
 * Errors: as sc_prefill_stack, plus SC_ERR_INVALID (chunk_tokens <= 0).
 */
sc_status sc_prefill_stack_chunked(sc_pool *pool, const sc_table *table, int32_t n_layers,
                                   const void *const *q_per_layer, const void *const *knew_per_layer,
                                   const void *const *vnew_per_layer, void *const *out_per_layer,
                                   const sc_active *slots /* [2] */, int32_t n_q_heads, float scale,
                                   uint32_t flags, int32_t chunk_tokens, void *compute_stream,
                                   void *copy_stream);

/*
 * Host-only introspection of the attention work decomposition (no device
 * work, no allocation).  For a batch with the given lengths, returns in
 * *n_items the number of workgroup slots; when `items` is non-NULL it also
 * receives them as int32 octets
 *   {seq, kv_head, q0, n_queries, key_begin, key_end, split, paged}
 * (seq = -1 marks an idle padding slot; slot w runs on XCD w % 8), and when
 * `splits` is non-NULL it receives each sequence's key-split count.  Every
 * workgroup covers rows (queries [q0, q0 + n_queries) x the group of query
 * heads of kv_head) and keys [key_begin, key_end); the splits of one query
 * tile partition [0, P + q0 + n_queries).  rc_keys (nullable) gives each
 * sequence's leading keys held in the regular cache, as a table with that
 * many leading regular-cache blocks would: no workgroup straddles that
 * boundary and paged = 1 marks those that read it.  `slots` is the number
 * of workgroups the device runs at once (<= 0: 256, one per CU of an MI355X,
 * as the library plans its own calls).
 * Errors: SC_ERR_INVALID (null, negative length, rc_keys outside [0, P],
 * heads as in sc_prefill_attn), SC_ERR_RANGE (items non-NULL and capacity
 * too small).
 */
sc_status sc_attn_plan_query(int32_t batch, const int32_t *prefix_len, const int32_t *new_len,
                             const int32_t *rc_keys, int32_t n_q_heads, int32_t n_kv_heads, int32_t slots,
                             int32_t *n_items, int32_t *items, int32_t capacity, int32_t *splits);

/* ------------------------------------------------------------------------
 * Elastic donor tier and capacity planning (host only, no device work).
 * ---------------------------------------------------------------------- */

/*
 * Resize the pool's HBM tier in place (§3.4 "Block-Major Layout": the
 * elastic cache grows by appending blocks at the end and shrinks by
 * releasing the last ones; with all layers of a block contiguous, nothing
 * else moves, so the cost does not depend on the layer count).  Afterwards
 * ids [0, n_device_blocks) are usable; ids of the host tier do not change
 * (they start at the HBM capacity given at creation).  Tables created later
 * may only use ids below the new count.
 * A library-owned HBM tier (device_base NULL at creation) changes its
 * physical memory: shrinking unmaps and frees the chunks wholly past the new
 * count (after waiting for the device to finish the work already queued,
 * which may still read them), growing maps fresh chunks after the last one
 * (their contents are undefined until stored).  Kept blocks keep their
 * addresses and bytes.  Over caller-owned memory the call only moves the
 * bound on usable ids.
 * Errors: SC_ERR_INVALID (null pool); SC_ERR_RANGE (n_device_blocks < 0 or
 * above the capacity the pool was created with); SC_ERR_INVALID when a live
 * table still references an HBM block at or above the new count (the
 * message names it); SC_ERR_OOM when growing cannot map memory (the tier
 * is left as it was); SC_ERR_HIP when unmapping fails.
 */
sc_status sc_pool_resize(sc_pool *pool, int64_t n_device_blocks);

/* Shape of a model's KV cache (one entry per model in the formulas below). */
typedef struct {
  int32_t n_layers;
  int32_t block_size;        /* tokens per block */
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t dtype_bytes;
} sc_model_shape;

/* Capacity of the master's caches, §3.2. */
typedef struct {
  int64_t m_block_bytes;      /* Eq. 1: 2 * B * H_kv * D * dtype           */
  int64_t k_master;           /* Eq. 3: floor(C_master / M_block)          */
  int64_t sum_k_workers;      /* sum over workers of Eq. 2                 */
  int64_t n_lsc;              /* Eq. 4: min(sum K_i, K_master)             */
  int64_t n_rc;               /* Eq. 5: floor((K_master - sum K_i) / L), 0 if negative */
  int64_t max_context_tokens; /* (N_LSC + N_RC) * B                        */
  int64_t conventional_blocks;/* floor(K_master / L): without the LSC      */
} sc_capacity;

/*
 * LSC / RC sizing (§3.2, Eq. 1-5) for a master of shape `master` with
 * master_cache_bytes of its own KV memory and n_workers workers lending
 * worker_cache_bytes[i] bytes.  k_workers (nullable) receives Eq. 2 per
 * worker.  Errors: SC_ERR_INVALID (null, non-positive shape, negative bytes,
 * n_workers < 0); SC_ERR_RANGE (a product overflows 64 bits).
 */
sc_status sc_plan_capacity(const sc_model_shape *master, int64_t master_cache_bytes,
                           const int64_t *worker_cache_bytes, int32_t n_workers,
                           int64_t *k_workers, sc_capacity *out);

/*
 * Minimum elastic unit (§3.4, Eq. 6-9): BE = L * B * H_kv * D elements per
 * block of each model, LCM = lcm(BE_master, BE_worker), MEU = LCM / BE.
 * Scaling the master by k * meu_master blocks and the worker by
 * k * meu_worker blocks trades the same number of elements.
 * Errors: SC_ERR_INVALID (null, non-positive shape); SC_ERR_RANGE (overflow).
 */
sc_status sc_elastic_unit(const sc_model_shape *master, const sc_model_shape *worker,
                          int64_t *meu_master, int64_t *meu_worker);

/*
 * Algorithm 1, ScaleUp: a worker holding worker_blocks blocks of
 * worker_block_size tokens receives a request of request_len tokens.  If it
 * needs more than it holds, it grows by the smallest multiple k of
 * meu_worker covering the shortfall and the master gives up k * meu_master
 * blocks; otherwise both deltas are 0.
 * Errors: SC_ERR_INVALID (null, negative counts, non-positive block size or
 * units); SC_ERR_RANGE (overflow).
 */
sc_status sc_scale_up(int64_t worker_blocks, int32_t worker_block_size, int64_t meu_worker,
                      int64_t meu_master, int64_t request_len, int64_t *worker_delta,
                      int64_t *master_delta);

/*
 * Algorithm 1, ScaleDown: window_lens[n_window] are the lengths of the
 * requests seen in the last t seconds (an empty window keeps no block).  If
 * the worker holds more than the longest of them needs, it releases the
 * largest multiple k of meu_worker that fits in the surplus and the master
 * gains k * meu_master blocks; otherwise both deltas are 0.
 * Errors: as sc_scale_up; window_lens may be NULL when n_window is 0.
 */
sc_status sc_scale_down(int64_t worker_blocks, int32_t worker_block_size, int64_t meu_worker,
                        int64_t meu_master, const int64_t *window_lens, int32_t n_window,
                        int64_t *worker_delta, int64_t *master_delta);

/*
 * Whether a device-side wait of an overlapped stack on this table gave up
 * since the table was created or the flag was last cleared: an attention
 * workgroup waiting for its slot to be filled (it wrote NaN rows), or the
 * copy stream's wait for a slot to be released (that layer's slot was
 * filled with NaN).  Reads device memory synchronously: call it only after
 * the streams passed to the stack have been synchronised.  *timed_out = 0
 * or 1; clear != 0 resets the flag.  A table that never ran an overlapped
 * stack reports 0.
 */
sc_status sc_table_stack_status(const sc_table *table, int32_t *timed_out, int32_t clear);

/*
 * Host-side introspection (no device work): *device_wait = 1 when
 * sc_prefill_stack(table, ..., flags, ...) would order its copy and compute
 * streams with the device-side slot waits, 0 when with stream events (see
 * SC_STACK_EVENT_WAIT; serial and attention-only stacks have no such
 * waits and report 0).  Errors: SC_ERR_INVALID (null).
 */
sc_status sc_stack_wait_kind(const sc_table *table, uint32_t flags, int32_t *device_wait);

/* Message of the last failed call on this thread ("" if none). */
const char *sc_last_error(void);

/* Library version string. */
const char *sc_version(void);

#ifdef __cplusplus
}
#endif
#endif /* SWIFTCACHE_H */
