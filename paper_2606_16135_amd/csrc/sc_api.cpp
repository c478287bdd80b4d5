// Host runtime behind the C ABI in include/swiftcache.h: donor pool tiers,
// block-table validation and device work lists, the attention planner and
// split-key workspace, and the two-stream layer pipeline (§3.3).
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <cstdlib>
#include <dlfcn.h>
#include <memory>
#include <numeric>

#include "sc_internal.h"

namespace sc {

// ---------------------------------------------------------------------------
// Errors
// ---------------------------------------------------------------------------
static thread_local std::string g_last_error;

sc_status fail(sc_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

sc_status fail_hip(hipError_t e, const char *what) {
  g_last_error = std::string(what) + ": " + hipGetErrorString(e);
  return e == hipErrorOutOfMemory ? SC_ERR_OOM : SC_ERR_HIP;
}

void clear_error() { g_last_error.clear(); }

// Makes `dev` current for the duration of a call and restores the caller's.
class DeviceGuard {
 public:
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&old_) != hipSuccess) old_ = -1;
    if (old_ != dev) ok_ = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    if (old_ >= 0) (void)hipSetDevice(old_);
  }
  bool ok() const { return ok_; }

 private:
  int old_ = -1;
  bool ok_ = true;
};

// ---------------------------------------------------------------------------
// Attention planner
// ---------------------------------------------------------------------------
namespace {
constexpr int kXcds = 8;                 // MI355X: workgroup w is dispatched to XCD w % 8
constexpr int kMinSplitKeys = 2 * kAttnKeyTile;   // the schedule model below picks among the rest
constexpr int kMaxSplits = kAttnMaxSplits;
constexpr int kResidentPerCu = 1;        // one 8-wave workgroup per CU (LDS ring, 2 waves per SIMD)
constexpr int kQueryDefaultSlots = 256 * kResidentPerCu;   // MI355X: 256 CUs
constexpr int64_t kItemOverheadKeys = 128;  // prologue + epilogue, in keys
constexpr int64_t kMergeOverheadKeys = 64;  // partial write of a split item, in keys
// The merge kernel runs after the forward kernel, so its time adds to the
// schedule: a launch plus a term proportional to the partial rows it reads
// and the output rows it writes.  Calibrated on MI355X, where a key of one
// workgroup's range costs ~33 ns: the 8B shape's merge (16384 rows, 4
// splits) takes ~5.8 us, the 16-conversation batch's (~520k row-splits)
// ~33 us.
constexpr int64_t kMergeLaunchKeys = 45;
constexpr int64_t kMergeRowSplitsPerKey = 600;  // (rows x (splits + 1)) per key of merge time
// Every item also reads its Q tile and writes its output or partial tile
// (256 rows each way, 128 KiB at head_dim 128), and that traffic shares HBM
// with every other item in flight: about 30 ns, one key, per item.  With
// this term and two-tile splits allowed, the split count chosen for 21
// single-sequence shapes (P 256..32768, N 16..1024, 32 or 40 query heads)
// came within 2% of the fastest of 1..16 splits measured on MI355X for each;
// short turns (P <= 4096, N <= 256) run 10-35% faster than with a 512-key
// floor and no such term.
constexpr int64_t kItemSharedKeys = 1;

struct TileDesc {
  int32_t seq, kvh, q0, nq, keys;
};

// Longest-processing-time schedule of `costs` on `slots` identical slots.
int64_t lpt_makespan(std::vector<int64_t> &costs, int slots) {
  std::sort(costs.begin(), costs.end(), std::greater<int64_t>());
  std::vector<int64_t> heap(std::max(1, slots), 0);   // min-heap of slot loads
  auto cmp = std::greater<int64_t>();
  std::make_heap(heap.begin(), heap.end(), cmp);
  for (int64_t c : costs) {
    std::pop_heap(heap.begin(), heap.end(), cmp);
    heap.back() += c;
    std::push_heap(heap.begin(), heap.end(), cmp);
  }
  return *std::max_element(heap.begin(), heap.end());
}
}  // namespace

// The split count plan_attention chooses for one sequence without a
// regular cache, computed in fixed-size buffers (no heap memory): the same
// candidates, item costs, LPT schedule and merge term.  Each (query tile,
// split) cost stands for n_kv_heads identical items.  Returns false when the
// candidates' item lists exceed the buffers.
constexpr int kNoAllocMaxCosts = 4096;
constexpr int kNoAllocMaxSlots = 2048;

bool single_splits_noalloc(int P, int N, int hq, int hkv, int slots, int *splits_out) {
  const int group = hq / hkv;
  const int rows_q = kAttnRows / group;
  const int n_qt = (N + rows_q - 1) / rows_q;
  const int64_t max_kv = (int64_t)P + N;
  if (slots < 1 || slots > kNoAllocMaxSlots) return false;
  int64_t costs[kNoAllocMaxCosts];
  int64_t heap[kNoAllocMaxSlots];
  auto splits_of = [&](int64_t chunk) {
    return (int)std::min<int64_t>(kMaxSplits, std::max<int64_t>(1, (max_kv + chunk - 1) / chunk));
  };
  int64_t best_chunk = std::max<int64_t>(max_kv, 1), best_span = -1, best_items = 0;
  for (int s = 1; s <= kMaxSplits && n_qt > 0; ++s) {
    int64_t chunk = (max_kv + s - 1) / s;
    chunk = ((chunk + kAttnKeyTile - 1) / kAttnKeyTile) * kAttnKeyTile;
    if (s > 1 && chunk < kMinSplitKeys) break;
    const int S = splits_of(chunk);
    if ((int64_t)n_qt * S > kNoAllocMaxCosts) return false;
    int nc = 0;
    for (int tile = 0; tile < n_qt; ++tile) {
      const int q0 = tile * rows_q;
      const int keys = P + q0 + std::min(rows_q, N - q0);
      const int t = (keys + kAttnKeyTile - 1) / kAttnKeyTile;
      for (int sp = 0; sp < S; ++sp) {
        const int b0 = std::min(keys, (int)((int64_t)sp * t / S) * kAttnKeyTile);
        const int b1 = std::min(keys, (int)((int64_t)(sp + 1) * t / S) * kAttnKeyTile);
        costs[nc++] = (std::max(b0, b1) - b0) + kItemOverheadKeys + (S > 1 ? kMergeOverheadKeys : 0);
      }
    }
    std::sort(costs, costs + nc, std::greater<int64_t>());
    std::fill(heap, heap + slots, (int64_t)0);   // all zero: already a heap
    auto cmp = std::greater<int64_t>();
    for (int i = 0; i < nc; ++i)
      for (int g = 0; g < hkv; ++g) {
        std::pop_heap(heap, heap + slots, cmp);
        heap[slots - 1] += costs[i];
        std::push_heap(heap, heap + slots, cmp);
      }
    const int64_t makespan = *std::max_element(heap, heap + slots);
    const int64_t n = (int64_t)nc * hkv;
    const int64_t row_splits = S > 1 ? (int64_t)N * hq * (S + 1) : 0;
    const int64_t merge = row_splits > 0 ? kMergeLaunchKeys + row_splits / kMergeRowSplitsPerKey : 0;
    const int64_t span = makespan + merge + kItemSharedKeys * n;
    if (best_span < 0 || span < best_span || (span == best_span && n < best_items)) {
      best_span = span;
      best_chunk = chunk;
      best_items = n;
    }
  }
  *splits_out = splits_of(best_chunk);
  return true;
}

int attn_slots(int device) {
  static std::mutex mu;
  static std::map<int, int> cache;
  std::lock_guard<std::mutex> lk(mu);
  auto it = cache.find(device);
  if (it != cache.end()) return it->second;
  int cus = 256;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess || cus <= 0)
    cus = 256;
  const int slots = cus * kResidentPerCu;
  cache[device] = slots;
  return slots;
}

struct GroupItems {
  int64_t cost = 0;
  std::vector<WorkItem> items;
};

// Places the items of each (sequence, KV head) group on one XCD (workgroup
// w runs on XCD w mod 8), groups by decreasing cost onto the least loaded
// XCD, longest items first within an XCD.
void place_items(std::vector<GroupItems> &groups, AttnPlan *plan) {
  std::stable_sort(groups.begin(), groups.end(),
                   [](const GroupItems &x, const GroupItems &y) { return x.cost > y.cost; });
  std::vector<int64_t> load(kXcds, 0);
  std::vector<std::vector<WorkItem>> per_xcd(kXcds);
  for (auto &gi : groups) {
    const int x = (int)(std::min_element(load.begin(), load.end()) - load.begin());
    load[x] += gi.cost;
    per_xcd[x].insert(per_xcd[x].end(), gi.items.begin(), gi.items.end());
  }
  size_t max_len = 0;
  int n_real = 0;
  for (auto &v : per_xcd) {
    // Longest items first; equal costs keep split-major order so that the
    // workgroups resident together read the same key range.
    std::stable_sort(v.begin(), v.end(), [](const WorkItem &x, const WorkItem &y) {
      const int cx = x.k_end - x.k_begin, cy = y.k_end - y.k_begin;
      if (cx != cy) return cx > cy;
      if (x.seq != y.seq) return x.seq < y.seq;
      if (x.split != y.split) return x.split < y.split;
      return x.q0 < y.q0;
    });
    max_len = std::max(max_len, v.size());
    n_real += (int)v.size();
  }
  plan->items.assign(max_len * kXcds, WorkItem{-1, 0, 0, 0, 0, 0, 0, 0});
  for (int x = 0; x < kXcds; ++x)
    for (size_t j = 0; j < per_xcd[x].size(); ++j) plan->items[j * kXcds + x] = per_xcd[x][j];
  plan->n_items = (int)plan->items.size();
  plan->n_real_items = n_real;
}

void plan_attention(const std::vector<int32_t> &P, const std::vector<int32_t> &N, int n_q_heads,
                    int n_kv_heads, int slots, AttnPlan *plan, const std::vector<int32_t> &rc_keys,
                    const std::vector<int32_t> &rc_off, const std::vector<int32_t> &cu_k,
                    const std::vector<int32_t> &q_off) {
  const int group = n_q_heads / n_kv_heads;
  const int rows_q = kAttnRows / group;
  const int batch = (int)P.size();
  plan->group = group;
  plan->rows_q = rows_q;
  plan->seqs.assign(batch, SeqDesc{});
  int64_t cq = 0, ck = 0, max_kv = 0;
  std::vector<TileDesc> tiles;
  for (int b = 0; b < batch; ++b) {
    SeqDesc &s = plan->seqs[b];
    s.cu_q = (int32_t)cq;
    s.cu_k = cu_k.empty() ? (int32_t)ck : cu_k[b];
    s.q_off = q_off.empty() ? (int32_t)cq : q_off[b];
    s.prefix = P[b];
    s.n_new = N[b];
    s.n_splits = 1;
    s.rc_keys = rc_keys.empty() ? 0 : rc_keys[b];
    s.rc_off = rc_off.empty() ? 0 : rc_off[b];
    if (s.rc_keys > 0) plan->paged = true;
    cq += N[b];
    ck += (int64_t)P[b] + N[b];
    max_kv = std::max<int64_t>(max_kv, (int64_t)P[b] + N[b]);
    for (int g = 0; g < n_kv_heads; ++g)
      for (int q0 = 0; q0 < N[b]; q0 += rows_q) {
        const int nq = std::min(rows_q, N[b] - q0);
        tiles.push_back(TileDesc{b, g, q0, nq, P[b] + q0 + nq});
      }
  }
  plan->total_q = cq;

  // Key-split choice: every sequence is split into chunks of at most `chunk`
  // keys; try the chunk sizes that give 1..kMaxSplits splits to the longest
  // sequence and keep the one with the shortest simulated schedule.  The
  // keys read in place from the regular cache [0, rc) and the keys of the
  // active slot [rc, keys) never share an item.
  struct Range {
    int32_t k_begin, k_end, paged;
  };
  auto split_counts = [&](int64_t chunk, int b, int *s_rc, int *s_sl) {
    const int64_t rc = rc_keys.empty() ? 0 : rc_keys[b];
    const int64_t kv = (int64_t)P[b] + N[b];
    *s_rc = rc > 0 ? (int)std::min<int64_t>(kMaxSplits - 1, std::max<int64_t>(1, (rc + chunk - 1) / chunk)) : 0;
    *s_sl = (int)std::min<int64_t>(kMaxSplits - *s_rc, std::max<int64_t>(1, (kv - rc + chunk - 1) / chunk));
  };
  auto ranges_for = [&](int64_t chunk, int b, int keys, std::vector<Range> *out) {
    int s_rc, s_sl;
    split_counts(chunk, b, &s_rc, &s_sl);
    const int rc = rc_keys.empty() ? 0 : rc_keys[b];
    out->clear();
    const int rc_t = (rc + kAttnKeyTile - 1) / kAttnKeyTile;
    for (int sp = 0; sp < s_rc; ++sp) {
      const int b0 = std::min(rc, (int)((int64_t)sp * rc_t / s_rc) * kAttnKeyTile);
      const int b1 = std::min(rc, (int)((int64_t)(sp + 1) * rc_t / s_rc) * kAttnKeyTile);
      out->push_back(Range{b0, std::max(b0, b1), 1});
    }
    const int len = keys - rc;
    const int sl_t = (len + kAttnKeyTile - 1) / kAttnKeyTile;
    for (int sp = 0; sp < s_sl; ++sp) {
      const int b0 = rc + (int)((int64_t)sp * sl_t / s_sl) * kAttnKeyTile;
      const int b1 = std::min(keys, rc + (int)((int64_t)(sp + 1) * sl_t / s_sl) * kAttnKeyTile);
      out->push_back(Range{std::min(b0, keys), std::max(std::min(b0, keys), b1), 0});
    }
  };
  auto splits_for = [&](int64_t chunk, int b) {
    int s_rc, s_sl;
    split_counts(chunk, b, &s_rc, &s_sl);
    return s_rc + s_sl;
  };
  int64_t best_chunk = std::max<int64_t>(max_kv, 1), best_span = -1;
  size_t best_items = 0;
  for (int s = 1; s <= kMaxSplits && !tiles.empty(); ++s) {
    int64_t chunk = (max_kv + s - 1) / s;
    chunk = ((chunk + kAttnKeyTile - 1) / kAttnKeyTile) * kAttnKeyTile;
    if (s > 1 && chunk < kMinSplitKeys) break;
    std::vector<int64_t> costs;
    std::vector<Range> rs;
    for (const TileDesc &t : tiles) {
      ranges_for(chunk, t.seq, t.keys, &rs);
      const int S = (int)rs.size();
      for (const Range &r : rs)
        costs.push_back((r.k_end - r.k_begin) + kItemOverheadKeys + (S > 1 ? kMergeOverheadKeys : 0));
    }
    const size_t n = costs.size();
    int64_t row_splits = 0;
    for (int b = 0; b < batch; ++b) {
      const int S = splits_for(chunk, b);
      if (S > 1) row_splits += (int64_t)N[b] * n_q_heads * (S + 1);
    }
    const int64_t merge = row_splits > 0 ? kMergeLaunchKeys + row_splits / kMergeRowSplitsPerKey : 0;
    const int64_t span = lpt_makespan(costs, slots) + merge + kItemSharedKeys * (int64_t)n;
    if (best_span < 0 || span < best_span || (span == best_span && n < best_items)) {
      best_span = span;
      best_chunk = chunk;
      best_items = n;
    }
  }
  int max_splits = 1;
  for (int b = 0; b < batch; ++b) {
    plan->seqs[b].n_splits = splits_for(best_chunk, b);
    max_splits = std::max(max_splits, plan->seqs[b].n_splits);
  }
  plan->max_splits = max_splits;

  // Items, grouped by (sequence, KV head) so that one group's K/V stays in
  // one XCD's L2.
  std::vector<GroupItems> groups;
  size_t ti = 0;
  for (int b = 0; b < batch; ++b) {
    for (int g = 0; g < n_kv_heads; ++g) {
      GroupItems gi;
      std::vector<Range> rs;
      for (; ti < tiles.size() && tiles[ti].seq == b && tiles[ti].kvh == g; ++ti) {
        const TileDesc &t = tiles[ti];
        ranges_for(best_chunk, b, t.keys, &rs);
        for (int s = 0; s < (int)rs.size(); ++s) {
          WorkItem w{};
          w.seq = b;
          w.kvh = g;
          w.q0 = t.q0;
          w.nq = t.nq;
          w.k_begin = rs[s].k_begin;
          w.k_end = rs[s].k_end;
          w.split = s;
          w.paged = rs[s].paged;
          gi.cost += (w.k_end - w.k_begin) + kItemOverheadKeys;
          gi.items.push_back(w);
        }
      }
      if (!gi.items.empty()) groups.push_back(std::move(gi));
    }
  }
  place_items(groups, plan);
}

namespace {

// ---------------------------------------------------------------------------
// Split-key workspace: one grow-only buffer per (device, stream).  Work on
// one stream is ordered, so reuse across calls on the same stream is safe.
// Each buffer has its own lock, which a caller holds from the lookup until
// the kernels that use the buffer are enqueued: a thread that must grow the
// buffer (stream sync, free, allocate) can then never free it under another
// thread that has looked it up but not yet launched with it.  The map only
// grows, so a Workspace never moves.
// ---------------------------------------------------------------------------
struct Workspace {
  std::mutex mu;
  void *ptr = nullptr;
  size_t bytes = 0;
};
std::mutex g_ws_mu;   // guards g_ws itself
std::map<std::pair<int, hipStream_t>, std::unique_ptr<Workspace>> g_ws;

// Partial log-sum-exps and outputs of split-key attention.  On success
// *hold owns the buffer's lock; release it after the launches.
sc_status get_workspace(int device, hipStream_t stream, size_t bytes, void **out,
                        std::unique_lock<std::mutex> *hold) {
  Workspace *ws = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_ws_mu);
    std::unique_ptr<Workspace> &slot = g_ws[{device, stream}];
    if (!slot) slot.reset(new Workspace());
    ws = slot.get();
  }
  std::unique_lock<std::mutex> lk(ws->mu);
  if (ws->bytes < bytes) {
    if (ws->ptr) {
      // Earlier launches with this buffer were all enqueued on `stream`
      // before their callers released the lock.
      SC_HIP(hipStreamSynchronize(stream));
      SC_HIP(hipFree(ws->ptr));
      ws->ptr = nullptr;
      ws->bytes = 0;
    }
    SC_HIP(hipMalloc(&ws->ptr, bytes));
    ws->bytes = bytes;
  }
  *out = ws->ptr;
  *hold = std::move(lk);
  return SC_OK;
}

sc_status upload_plan(AttnPlan *plan) {
  if (plan->n_items == 0) return SC_OK;
  SC_HIP(hipMalloc(&plan->d_items, plan->items.size() * sizeof(WorkItem)));
  SC_HIP(hipMalloc(&plan->d_seqs, plan->seqs.size() * sizeof(SeqDesc)));
  SC_HIP(hipMemcpy(plan->d_items, plan->items.data(), plan->items.size() * sizeof(WorkItem),
                   hipMemcpyHostToDevice));
  SC_HIP(hipMemcpy(plan->d_seqs, plan->seqs.data(), plan->seqs.size() * sizeof(SeqDesc),
                   hipMemcpyHostToDevice));
  return SC_OK;
}

void free_plan(AttnPlan *plan) {
  if (plan->d_items) (void)hipFree(plan->d_items);
  if (plan->d_seqs) (void)hipFree(plan->d_seqs);
  plan->d_items = nullptr;
  plan->d_seqs = nullptr;
}

// Plans for single-sequence calls, keyed by (device, P, N, Hq, Hkv).  The
// caller holds g_plan_mu from the lookup until its kernels are enqueued, so
// an eviction (which drains the device first) never frees a plan that
// another thread is about to launch with.
std::mutex g_plan_mu;
std::map<std::tuple<int, int, int, int, int, int>, std::unique_ptr<AttnPlan>> g_single_plans;

sc_status single_plan(int device, int P, int N, int hq, int hkv, int head_dim, AttnPlan **out) {
  auto key = std::make_tuple(device, P, N, hq, hkv, head_dim);
  auto it = g_single_plans.find(key);
  if (it != g_single_plans.end()) {
    *out = it->second.get();
    return SC_OK;
  }
  if (g_single_plans.size() >= 256) {
    // Plans may still be referenced by queued kernels: drain this device
    // before freeing its plans (the caller made it current); other
    // devices' plans stay.
    SC_HIP(hipDeviceSynchronize());
    for (auto i = g_single_plans.begin(); i != g_single_plans.end();) {
      if (std::get<0>(i->first) == device) {
        free_plan(i->second.get());
        i = g_single_plans.erase(i);
      } else {
        ++i;
      }
    }
  }
  auto plan = std::make_unique<AttnPlan>();
  plan_attention({P}, {N}, hq, hkv, attn_slots(device), plan.get());
  sc_status st = upload_plan(plan.get());
  if (st != SC_OK) {
    free_plan(plan.get());
    return st;
  }
  *out = plan.get();
  g_single_plans[key] = std::move(plan);
  return SC_OK;
}

// ready_flag / ready_value: optional device-side wait (overlapped stack);
// after_fwd: optional event recorded once the forward kernel (the only one
// that reads K/V) is enqueued.
// rc: the table's regular cache (pool, layer, device block indices) for
// plans with paged items; required exactly when plan.paged.
struct RcView {
  const sc_pool *pool = nullptr;
  int layer = 0;
  const int32_t *ids = nullptr;
};

// Split-key partials of a layer stack whose merges are deferred: the
// layer's own partial buffer (ws) and the previous layer's (prev_ws, merged
// into prev_out by the forward kernel's workgroups before their own items),
// both laid out as a plan-sized workspace (partials, then lse).
struct StackMerge {
  void *ws = nullptr;
  const void *prev_ws = nullptr;
  void *prev_out = nullptr;
  uint32_t *prev_counter = nullptr;   // zero before the launch
};


// Bytes of a plan's split-key workspace and the lse array's offset in it.
size_t plan_ws_bytes(const AttnPlan &plan, int hq, int head_dim, size_t *lse_off = nullptr) {
  const size_t rows = (size_t)plan.max_splits * plan.total_q * hq;
  if (lse_off) *lse_off = rows * (size_t)head_dim * sizeof(uint16_t);
  return rows * ((size_t)head_dim * sizeof(uint16_t) + sizeof(float));
}

sc_status run_attention(int device, const AttnPlan &plan, const void *q, const void *k, const void *v,
                        void *out, float *lse, int hq, int hkv, int head_dim, int dtype, float scale,
                        hipStream_t stream, const uint64_t *ready_flag = nullptr, uint64_t ready_value = 0,
                        hipEvent_t after_fwd = nullptr, const RcView &rc = RcView(),
                        int spin_limit = kAttnReadySpinLimit, uint64_t *done_counter = nullptr,
                        const StackMerge *sm = nullptr, bool ready_acquire = false) {
  if (plan.n_items == 0) return SC_OK;
  // The kernel addresses one sequence's rows of one KV head with 32-bit
  // byte offsets.
  for (const SeqDesc &s : plan.seqs)
    if (!keys_fit_offsets((int64_t)s.prefix + s.n_new, hkv, head_dim))
      return fail(SC_ERR_UNSUPPORTED,
                  "sequence of %lld tokens x %d KV heads x head_dim %d exceeds 2 GiB of keys less %d tokens",
                  (long long)s.prefix + s.n_new, hkv, head_dim, kKeyOffsetMarginTokens);
  AttnArgs a{};
  a.q = static_cast<const uint16_t *>(q);
  a.k = static_cast<const uint16_t *>(k);
  a.v = static_cast<const uint16_t *>(v);
  a.out = static_cast<uint16_t *>(out);
  a.lse = lse;
  a.items = plan.d_items;
  a.seqs = plan.d_seqs;
  a.n_seqs = (int32_t)plan.seqs.size();
  a.total_q = (int32_t)plan.total_q;
  a.n_q_heads = hq;
  a.n_kv_heads = hkv;
  a.group = plan.group;
  a.rows_q = plan.rows_q;
  a.dtype = dtype;
  if (!(scale > 0.f)) scale = 1.f / std::sqrt((float)head_dim);
  a.scale_log2 = scale * 1.4426950408889634f;
  // Held until the forward and merge kernels are enqueued (see get_workspace).
  std::unique_lock<std::mutex> ws_hold;
  if (plan.max_splits > 1) {
    size_t lse_off = 0;
    const size_t bytes = plan_ws_bytes(plan, hq, head_dim, &lse_off);
    void *ws = sm ? sm->ws : nullptr;
    if (!ws) {
      sc_status st = get_workspace(device, stream, bytes, &ws, &ws_hold);
      if (st != SC_OK) return st;
    }
    a.part_o = static_cast<uint16_t *>(ws);
    a.part_lse = reinterpret_cast<float *>(static_cast<char *>(ws) + lse_off);
    if (sm && sm->prev_ws) {
      a.dm_part_o = static_cast<const uint16_t *>(sm->prev_ws);
      a.dm_part_lse = reinterpret_cast<const float *>(static_cast<const char *>(sm->prev_ws) + lse_off);
      a.dm_out = static_cast<uint16_t *>(sm->prev_out);
      a.dm_counter = sm->prev_counter;
      a.dm_max_splits = plan.max_splits;
    }
  }
  if (plan.paged) {
    if (!rc.pool || !rc.ids || !rc.pool->rc_base)
      return fail(SC_ERR_INVALID, "the table reads regular-cache blocks; the call needs the pool and layer");
    const sc_pool_desc &pd = rc.pool->desc;
    a.rc_base = reinterpret_cast<const uint16_t *>(rc.pool->rc_base);
    a.rc_ids = rc.ids;
    a.rc_block_elems = (int64_t)(rc.pool->block_bytes / 2);
    a.rc_layer_elems = (int64_t)rc.layer * (int64_t)(rc.pool->slice_bytes / 2);
    a.rc_half_elems = (int64_t)(rc.pool->slice_bytes / 4);
    int sh = 0;
    while ((1 << sh) < pd.block_size) ++sh;
    a.block_shift = sh;
  }
  if (ready_flag) {
    a.ready_flag = ready_flag;
    a.ready_value = ready_value;
    a.ready_timeout = reinterpret_cast<uint32_t *>(const_cast<uint64_t *>(ready_flag + 1));
    a.ready_spin_limit = spin_limit;
    a.ready_acquire = ready_acquire ? 1 : 0;
  }
  a.done_counter = done_counter;
  hipError_t e = launch_attn_fwd(a, head_dim, plan.n_items, stream);
  if (e != hipSuccess) return fail_hip(e, "attn_fwd launch");
  if (after_fwd) SC_HIP(hipEventRecord(after_fwd, stream));
  if (plan.max_splits > 1 && !sm) {
    e = launch_attn_merge(a, head_dim, stream);
    if (e != hipSuccess) return fail_hip(e, "attn_merge launch");
  }
  return SC_OK;
}

// The merge kernel alone over a plan-sized workspace (the last layer of a
// stack whose merges are deferred).
sc_status run_merge(const AttnPlan &plan, const void *ws, void *out, int hq, int hkv, int head_dim, int dtype,
                    hipStream_t stream) {
  if (plan.n_items == 0 || plan.max_splits <= 1) return SC_OK;
  size_t lse_off = 0;
  plan_ws_bytes(plan, hq, head_dim, &lse_off);
  AttnArgs a{};
  a.out = static_cast<uint16_t *>(out);
  a.seqs = plan.d_seqs;
  a.n_seqs = (int32_t)plan.seqs.size();
  a.total_q = (int32_t)plan.total_q;
  a.n_q_heads = hq;
  a.n_kv_heads = hkv;
  a.group = plan.group;
  a.rows_q = plan.rows_q;
  a.dtype = dtype;
  a.part_o = static_cast<uint16_t *>(const_cast<void *>(ws));
  a.part_lse = reinterpret_cast<float *>(static_cast<char *>(const_cast<void *>(ws)) + lse_off);
  hipError_t e = launch_attn_merge(a, head_dim, stream);
  return e == hipSuccess ? SC_OK : fail_hip(e, "attn_merge launch");
}

sc_status check_heads(int hq, int hkv, int head_dim) {
  if (hq <= 0 || hkv <= 0 || hq % hkv != 0)
    return fail(SC_ERR_INVALID, "n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)", hq, hkv);
  if (head_dim != 64 && head_dim != 128)
    return fail(SC_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", head_dim);
  if (hq / hkv > 16) return fail(SC_ERR_UNSUPPORTED, "GQA group %d > 16 not supported", hq / hkv);
  return SC_OK;
}

// chunk_tokens > 0: the plan of chunk `chunk` of the new turn, i.e. new
// tokens [chunk * C, min(N_b, (chunk + 1) * C)) of every sequence, which see
// the prefix and the earlier chunks as their prefix (same active rows, q /
// out rows offset by chunk * C within the sequence).
sc_status table_plan(sc_table *t, int hq, AttnPlan **out, int slots = 0, int chunk_tokens = 0, int chunk = 0) {
  const sc_pool_desc &d = t->pool->desc;
  sc_status st = check_heads(hq, d.n_kv_heads, d.head_dim);
  if (st != SC_OK) return st;
  if (slots <= 0) slots = attn_slots(d.device);
  std::lock_guard<std::mutex> lk(t->mu);
  auto key = std::make_tuple(hq, slots, chunk_tokens, chunk);
  auto it = t->plans.find(key);
  if (it != t->plans.end()) {
    *out = &it->second;
    return SC_OK;
  }
  AttnPlan &plan = t->plans[key];
  if (chunk_tokens > 0) {
    const size_t batch = t->P.size();
    std::vector<int32_t> P(batch), N(batch), cu_k(batch), q_off(batch);
    for (size_t b = 0; b < batch; ++b) {
      const int64_t done = std::min<int64_t>(t->N[b], (int64_t)chunk * chunk_tokens);
      P[b] = (int32_t)(t->P[b] + done);
      N[b] = (int32_t)std::min<int64_t>(chunk_tokens, t->N[b] - done);
      cu_k[b] = (int32_t)t->cu_k[b];
      q_off[b] = (int32_t)(t->cu_q[b] + done);
    }
    plan_attention(P, N, hq, d.n_kv_heads, slots, &plan, t->rc_keys, t->rc_off, cu_k, q_off);
  } else {
    plan_attention(t->P, t->N, hq, d.n_kv_heads, slots, &plan, t->rc_keys, t->rc_off);
  }
  st = upload_plan(&plan);
  if (st != SC_OK) {
    free_plan(&plan);
    t->plans.erase(key);
    return st;
  }
  *out = &plan;
  return SC_OK;
}

// ---------------------------------------------------------------------------
// CU-partitioned streams for the layer pipeline when the fetch reads the
// host tier.  Such a fetch takes as long as a layer's attention and its
// workgroups wait on the host link for most of that time, so it must not
// compete with attention for CU slots: the library keeps, per device, a copy
// stream restricted to kHostFetchCus CUs and an attention stream restricted
// to the others.  CU mask bit i selects logical CU i; logical CUs are
// interleaved across the XCDs, so the low bits take the same number of CUs
// from every XCD (on MI355X the low 16 bits are two CUs of each of the 8
// XCDs, as the hardware's XCC_ID and HW_ID registers read by workgroups of
// such a stream show).  The streams live as long as the process.
// ---------------------------------------------------------------------------
constexpr int kHostFetchCus = 16;

struct SplitStreams {
  hipStream_t attn = nullptr;
  hipStream_t copy = nullptr;
  int attn_cus = 0;
};
std::mutex g_split_mu;
std::map<int, SplitStreams> g_split;

sc_status split_streams(int device, SplitStreams **out) {
  std::lock_guard<std::mutex> lk(g_split_mu);
  auto it = g_split.find(device);
  if (it != g_split.end()) {
    *out = &it->second;
    return SC_OK;
  }
  int cus = 0;
  SC_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device));
  if (cus <= 2 * kHostFetchCus) return fail(SC_ERR_UNSUPPORTED, "device has only %d CUs", cus);
  const int words = (cus + 31) / 32;
  std::vector<uint32_t> copy_mask(words, 0u), attn_mask(words, 0u);
  for (int c = 0; c < cus; ++c) {
    std::vector<uint32_t> &m = c < kHostFetchCus ? copy_mask : attn_mask;
    m[c / 32] |= 1u << (c % 32);
  }
  SplitStreams ss;
  SC_HIP(hipExtStreamCreateWithCUMask(&ss.attn, (uint32_t)words, attn_mask.data()));
  const hipError_t e = hipExtStreamCreateWithCUMask(&ss.copy, (uint32_t)words, copy_mask.data());
  if (e != hipSuccess) {
    (void)hipStreamDestroy(ss.attn);
    return fail_hip(e, "copy stream with a CU mask");
  }
  ss.attn_cus = cus - kHostFetchCus;
  *out = &(g_split[device] = ss);
  return SC_OK;
}

// ---------------------------------------------------------------------------
// Copy kernels beside attention (device tier).  In the overlapped stack the
// fetch of layer l+1 is released when attention of layer l-1 ends, the same
// moment attention of layer l becomes ready; if copy workgroups take a CU's
// VGPRs or LDS first, the attention workgroup waits for them and the fetch
// lands on the critical path.  Each copy workgroup therefore reserves enough
// (unused) LDS that at most kCopyBesideAttn of them fit on a CU, and that
// many still leave room for one attention workgroup.
// ---------------------------------------------------------------------------
constexpr int kCopyBesideAttn = 2;
std::mutex g_reserve_mu;
std::map<std::pair<int, int>, size_t> g_reserve;

// Settings under which kernels of different streams do not run at the same
// time: counter collection by the ROCm profiler serialises dispatches, and
// the two runtime switches make every launch wait for the previous kernel.
// The device-side slot waits need a copy kernel to run while an attention
// kernel holds the GPU, so under these the stack waits on stream events.
bool dispatch_is_serialised() {
  static const bool serialised = [] {
    auto on = [](const char *name) {
      const char *e = std::getenv(name);
      return e != nullptr && *e != '\0' && std::strcmp(e, "0") != 0 && std::strcmp(e, "false") != 0 &&
             std::strcmp(e, "False") != 0;
    };
    return on("ROCPROF_COUNTER_COLLECTION") || on("AMD_SERIALIZE_KERNEL") || on("HIP_LAUNCH_BLOCKING");
  }();
  return serialised;
}

// Whether a copy workgroup can always start on a CU that holds an attention
// workgroup (one wave per SIMD beside the attention's two; 512 VGPRs per
// SIMD lane, allocated in steps of 8).  Only then may attention wait for the
// copy stream on the device without risking a wait on itself.
bool copy_fits_beside_attention(int head_dim) {
  const int av = attn_fwd_vgprs(head_dim), cv = kv_copy_vgprs();
  if (av <= 0 || cv <= 0) return false;
  auto alloc = [](int v) { return (v + 7) / 8 * 8; };
  return 2 * alloc(av) + alloc(cv) <= 512;
}

// Whether an sc_prefill_stack call with these flags orders its two streams
// with device-side waits (else stream events): overlapped stacks only, not
// when asked for events or when dispatches are serialised, and only when a
// copy workgroup always fits beside attention or the copies run on CUs of
// their own (a fetch that reaches into the host tier).
bool stack_device_wait(const sc_table *t, uint32_t flags) {
  if ((flags & SC_STACK_MODE_MASK) != SC_STACK_OVERLAP) return false;
  if ((flags & SC_STACK_EVENT_WAIT) != 0 || dispatch_is_serialised()) return false;
  return t->n_fetch_host > 0 || copy_fits_beside_attention(t->pool->desc.head_dim);
}

size_t copy_lds_reserve(int device, int head_dim) {
  std::lock_guard<std::mutex> lk(g_reserve_mu);
  auto key = std::make_pair(device, head_dim);
  auto it = g_reserve.find(key);
  if (it != g_reserve.end()) return it->second;
  int lds_cu = 0, lds_block = 0;
  size_t r = 0;
  if (hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, device) == hipSuccess &&
      hipDeviceGetAttribute(&lds_block, hipDeviceAttributeMaxSharedMemoryPerBlock, device) == hipSuccess &&
      lds_cu > 0) {
    // kCopyBesideAttn of these fit in the LDS an attention workgroup leaves
    // free, one more does not.
    const size_t attn = attn_fwd_lds_bytes(head_dim);
    if (attn < (size_t)lds_cu) {
      const size_t cand = (((size_t)lds_cu - attn) / (kCopyBesideAttn + 1) + 1024 + 255) & ~(size_t)255;
      if (cand <= (size_t)lds_block && kCopyBesideAttn * cand + attn <= (size_t)lds_cu) r = cand;
    }
  }
  g_reserve[key] = r;
  return r;
}

// Width of the copy grids beside attention.  Every copy workgroup that
// shares a CU with attention slows that CU's attention waves (issue slots,
// the vector memory path), so the overlapped stack launches the fewest
// copy workgroups that still finish a layer's fetch, append and store in
// about half of the attention they hide behind; they then loop over the
// items.  Measured on the 8B shape (32 MiB fetched per layer beside ~84 us
// of attention): 1024 workgroups (one per item half) cost 10-11% over
// attention alone, 256 cost 8.6%, 128 cost 7.4%, 64 cost 17% (the copies
// no longer finish in time).  A copy workgroup beside attention moves about
// kCopyGroupBps; attention runs at about kAttnFlops.  Never fewer than half
// the CUs, never more than the items need.
constexpr double kCopyGroupBps = 6.5e9;
constexpr double kAttnFlops = 0.9e15;

int copy_groups_beside_attention(int device, const sc_table *t, int n_q_heads, int head_dim) {
  double pairs = 0.0;
  for (int32_t b = 0; b < t->batch; ++b)
    pairs += (double)t->N[b] * t->P[b] + 0.5 * (double)t->N[b] * (t->N[b] + 1);
  const double flops = 4.0 * head_dim * n_q_heads * pairs;
  int64_t rows = 0;
  for (const CopyItem &it : t->h_items) rows += it.nrows;
  const double bytes = 2.0 * (double)rows * (double)t->pool->row_bytes;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess || cus <= 0) return 0;
  if (flops <= 0.0) return 0;
  const double need = 2.0 * bytes * kAttnFlops / (kCopyGroupBps * flops);
  if (need > 1e9) return 0;
  return std::max(cus / 2, (int)std::ceil(need));
}

CopyArgs copy_args(const sc_pool *p, const sc_table *t, int mode) {
  CopyArgs a{};
  a.mode = mode;
  a.row_bytes = (int64_t)p->row_bytes;
  a.v_half_off = (int64_t)(p->slice_bytes / 2);
  a.tier_base[0] = p->dev_base;
  a.tier_base[1] = p->host_dev;
  a.tier_mask = 3;
  if (mode == COPY_FETCH) {
    a.items = t->d_items;
    a.n_items = t->n_fetch;
  } else if (mode == COPY_APPEND) {
    a.items = t->d_items + t->n_fetch;
    a.n_items = t->n_append;
  } else {
    a.items = t->d_items + t->n_fetch + t->n_append;
    a.n_items = t->n_store;
  }
  return a;
}

// Element data is moved in 16-byte chunks; every row of it is a multiple
// of 16 bytes long, so a 16-byte aligned base keeps every row aligned.
bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

sc_status check_active(const sc_table *t, const sc_active *dst) {
  if (dst == nullptr || dst->k == nullptr || dst->v == nullptr)
    return fail(SC_ERR_INVALID, "null active buffer");
  if (!aligned16(dst->k) || !aligned16(dst->v)) return fail(SC_ERR_INVALID, "active buffer not 16-byte aligned");
  if (dst->capacity_tokens < t->total_kv)
    return fail(SC_ERR_RANGE, "active buffer holds %lld tokens, the table needs %lld",
                (long long)dst->capacity_tokens, (long long)t->total_kv);
  return SC_OK;
}

sc_status do_fetch(sc_pool *p, const sc_table *t, int layer, const sc_active *dst, hipStream_t s,
                   size_t lds_reserve = 0, int max_groups = 0) {
  CopyArgs a = copy_args(p, t, COPY_FETCH);
  a.layer_off = (int64_t)layer * (int64_t)p->slice_bytes;
  a.act_k = static_cast<char *>(dst->k);
  a.act_v = static_cast<char *>(dst->v);
  hipError_t e = launch_kv_copy(a, s, lds_reserve, max_groups);
  return e == hipSuccess ? SC_OK : fail_hip(e, "fetch launch");
}

sc_status do_append(sc_pool *p, const sc_table *t, const void *kn, const void *vn, const sc_active *dst,
                    hipStream_t s, size_t lds_reserve = 0, int max_groups = 0) {
  CopyArgs a = copy_args(p, t, COPY_APPEND);
  a.new_k = static_cast<const char *>(kn);
  a.new_v = static_cast<const char *>(vn);
  a.act_k = static_cast<char *>(dst->k);
  a.act_v = static_cast<char *>(dst->v);
  hipError_t e = launch_kv_copy(a, s, lds_reserve, max_groups);
  return e == hipSuccess ? SC_OK : fail_hip(e, "append launch");
}

sc_status do_store(sc_pool *p, const sc_table *t, int layer, const void *kn, const void *vn, hipStream_t s,
                   size_t lds_reserve = 0, int max_groups = 0) {
  CopyArgs a = copy_args(p, t, COPY_STORE);
  a.layer_off = (int64_t)layer * (int64_t)p->slice_bytes;
  a.new_k = static_cast<const char *>(kn);
  a.new_v = static_cast<const char *>(vn);
  hipError_t e = launch_kv_copy(a, s, lds_reserve, max_groups);
  return e == hipSuccess ? SC_OK : fail_hip(e, "store launch");
}

// Fetch, append and store of one layer as one launch (overlapped stack).
LayerCopyArgs layer_copy_args(const sc_pool *p, const sc_table *t, int layer, const void *kn, const void *vn,
                              const sc_active *dst, bool store) {
  LayerCopyArgs la{};
  const int64_t layer_off = (int64_t)layer * (int64_t)p->slice_bytes;
  for (int m : {COPY_FETCH, COPY_APPEND, COPY_STORE}) {
    CopyArgs &a = la.part[m == COPY_FETCH ? 0 : m == COPY_APPEND ? 1 : 2];
    a = copy_args(p, t, m);
    a.layer_off = m == COPY_APPEND ? 0 : layer_off;
    a.new_k = static_cast<const char *>(kn);
    a.new_v = static_cast<const char *>(vn);
    a.act_k = m == COPY_STORE ? nullptr : static_cast<char *>(dst->k);
    a.act_v = m == COPY_STORE ? nullptr : static_cast<char *>(dst->v);
  }
  if (!store) la.part[2].n_items = 0;
  return la;
}

sc_status prefill_attn_single(const void *q, const void *k_active, const void *v_active, int32_t prefix_len,
                              int32_t new_len, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int dtype,
                              float scale, void *out, float *lse, void *stream) {
  if (prefix_len < 0 || new_len < 0) return fail(SC_ERR_INVALID, "negative length");
  sc_status st = check_heads(n_q_heads, n_kv_heads, head_dim);
  if (st != SC_OK) return st;
  if (new_len == 0) return SC_OK;
  if (!q || !k_active || !v_active || !out) return fail(SC_ERR_INVALID, "null argument");
  if (!aligned16(q) || !aligned16(k_active) || !aligned16(v_active) || !aligned16(out))
    return fail(SC_ERR_INVALID, "q, k_active, v_active and out must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(lse) & 3) != 0) return fail(SC_ERR_INVALID, "lse must be 4-byte aligned");
  int device = 0;
  SC_HIP(hipGetDevice(&device));
  AttnPlan *plan = nullptr;
  std::lock_guard<std::mutex> lk(g_plan_mu);
  st = single_plan(device, prefix_len, new_len, n_q_heads, n_kv_heads, head_dim, &plan);
  if (st != SC_OK) return st;
  return run_attention(device, *plan, q, k_active, v_active, out, lse, n_q_heads, n_kv_heads, head_dim, dtype,
                       scale, (hipStream_t)stream);
}

// ---------------------------------------------------------------------------
// Elastic HBM tier (§3.4 "Block-Major Layout"): one reserved virtual range
// for the tier's capacity, physical memory mapped chunk by chunk at its
// start.  Growing maps chunks after the last one, shrinking unmaps the last
// ones; the blocks that stay keep their addresses and contents.
// ---------------------------------------------------------------------------
hipMemAllocationProp vmm_prop(int device) {
  hipMemAllocationProp prop{};
  prop.type = hipMemAllocationTypePinned;   // plain (cached) device memory
  prop.location.type = hipMemLocationTypeDevice;
  prop.location.id = device;
  return prop;
}

// Maps one more chunk after the mapped ones.
hipError_t vmm_append_chunk(sc_pool *p) {
  const hipMemAllocationProp prop = vmm_prop(p->desc.device);
  char *at = p->dev_base + p->vmm_handles.size() * p->vmm_chunk_bytes;
  if (at + p->vmm_chunk_bytes > p->dev_base + p->vmm_reserved) return hipErrorInvalidValue;
  hipMemGenericAllocationHandle_t h{};
  hipError_t e = hipMemCreate(&h, p->vmm_chunk_bytes, &prop, 0);
  if (e != hipSuccess) return e;
  e = hipMemMap(at, p->vmm_chunk_bytes, 0, h, 0);
  if (e != hipSuccess) {
    (void)hipMemRelease(h);
    return e;
  }
  hipMemAccessDesc ad{};
  ad.location = prop.location;
  ad.flags = hipMemAccessFlagsProtReadWrite;
  e = hipMemSetAccess(at, p->vmm_chunk_bytes, &ad, 1);
  if (e != hipSuccess) {
    (void)hipMemUnmap(at, p->vmm_chunk_bytes);
    (void)hipMemRelease(h);
    return e;
  }
  p->vmm_handles.push_back(h);
  return hipSuccess;
}

// Unmaps and frees the last mapped chunk (no device work may still use it).
hipError_t vmm_release_last_chunk(sc_pool *p) {
  char *at = p->dev_base + (p->vmm_handles.size() - 1) * p->vmm_chunk_bytes;
  hipError_t e = hipMemUnmap(at, p->vmm_chunk_bytes);
  hipError_t e2 = hipMemRelease(p->vmm_handles.back());
  p->vmm_handles.pop_back();
  return e != hipSuccess ? e : e2;
}

// Reserves the tier's range and maps chunks for its first n blocks.  Returns
// hipErrorNotSupported (nothing reserved) when the runtime has no virtual
// memory management for the device.
hipError_t vmm_create(sc_pool *p, int64_t n_blocks) {
  const hipMemAllocationProp prop = vmm_prop(p->desc.device);
  size_t gran = 0;
  hipError_t e = hipMemGetAllocationGranularity(&gran, &prop, hipMemAllocationGranularityMinimum);
  if (e != hipSuccess || gran == 0) return hipErrorNotSupported;
  // Chunks hold whole blocks and are a multiple of the granularity: a
  // multiple of lcm(block_bytes, gran), about kVmmChunkTarget bytes.  Each
  // map or unmap call costs tens to hundreds of microseconds whatever its
  // size (measured on MI355X with 2 MiB chunks: ~70 us to map, ~0.4 ms to
  // unmap), so chunks much smaller than the usual resize step only add
  // calls; 32 MiB is 16 blocks of the 8B shape, the paper's minimum elastic
  // unit for a Qwen3-8B worker beside a Qwen3-32B master (Eq. 9).
  constexpr size_t kVmmChunkTarget = (size_t)32 << 20;
  const size_t g = std::gcd(p->block_bytes, gran);
  const size_t unit = p->block_bytes / g * gran;
  const size_t chunk = unit * std::max<size_t>(1, kVmmChunkTarget / unit);
  const int64_t chunk_blocks = (int64_t)(chunk / p->block_bytes);
  const int64_t cap_chunks = (p->desc.n_device_blocks + chunk_blocks - 1) / chunk_blocks;
  void *base = nullptr;
  e = hipMemAddressReserve(&base, (size_t)cap_chunks * chunk, gran, nullptr, 0);
  if (e != hipSuccess) return e == hipErrorOutOfMemory ? e : hipErrorNotSupported;
  p->dev_base = static_cast<char *>(base);
  p->vmm = true;
  p->vmm_reserved = (size_t)cap_chunks * chunk;
  p->vmm_chunk_bytes = chunk;
  p->vmm_chunk_blocks = chunk_blocks;
  const int64_t need = (n_blocks + chunk_blocks - 1) / chunk_blocks;
  while ((int64_t)p->vmm_handles.size() < need) {
    e = vmm_append_chunk(p);
    if (e != hipSuccess) break;
  }
  if (e != hipSuccess) {
    while (!p->vmm_handles.empty()) (void)vmm_release_last_chunk(p);
    (void)hipMemAddressFree(p->dev_base, p->vmm_reserved);
    p->dev_base = nullptr;
    p->vmm = false;
  }
  return e;
}

void vmm_destroy(sc_pool *p) {
  while (!p->vmm_handles.empty()) (void)vmm_release_last_chunk(p);
  if (p->dev_base) (void)hipMemAddressFree(p->dev_base, p->vmm_reserved);
  p->dev_base = nullptr;
  p->vmm = false;
}

}  // namespace
}  // namespace sc

using namespace sc;

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char *sc_last_error(void) { return g_last_error.c_str(); }

const char *sc_version(void) { return "swiftcache-mi355x 0.1 (gfx950)"; }

sc_status sc_pool_create(const sc_pool_desc *desc, sc_pool **out) {
  clear_error();
  if (desc == nullptr || out == nullptr) return fail(SC_ERR_INVALID, "null argument");
  *out = nullptr;
  const sc_pool_desc &d = *desc;
  if (d.n_layers <= 0 || d.n_kv_heads <= 0 || d.block_size <= 0 || d.block_size > 256 ||
      d.n_device_blocks < 0 || d.n_host_blocks < 0 || d.n_rc_blocks < 0 ||
      d.n_device_blocks + d.n_host_blocks + d.n_rc_blocks <= 0 ||
      (d.dtype != SC_DTYPE_BF16 && d.dtype != SC_DTYPE_F16))
    return fail(SC_ERR_INVALID, "invalid pool description");
  if (d.head_dim != 64 && d.head_dim != 128)
    return fail(SC_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", d.head_dim);
  // The copy kernels address one block's K (or V) rows of a layer with
  // 32-bit byte offsets.
  if ((int64_t)d.block_size * d.n_kv_heads * d.head_dim * 2 >= ((int64_t)1 << 31))
    return fail(SC_ERR_UNSUPPORTED, "block_size x n_kv_heads x head_dim too large (%d x %d x %d)", d.block_size,
                d.n_kv_heads, d.head_dim);
  if (d.n_device_blocks + d.n_host_blocks + d.n_rc_blocks > INT32_MAX)
    return fail(SC_ERR_RANGE, "too many blocks for 32-bit block ids");
  // Attention pages regular-cache keys in groups of up to 8 rows that must
  // not straddle a block.
  if (d.n_rc_blocks > 0 && (d.block_size < 16 || (d.block_size & (d.block_size - 1)) != 0))
    return fail(SC_ERR_UNSUPPORTED, "a regular cache needs a power-of-two block size >= 16 (got %d)",
                d.block_size);
  // Attention addresses a regular-cache block as block index x block bytes
  // in 32 x 32-bit arithmetic.
  if (d.n_rc_blocks > 0 &&
      (int64_t)d.n_layers * 2 * d.block_size * d.n_kv_heads * d.head_dim * 2 >= ((int64_t)1 << 32))
    return fail(SC_ERR_UNSUPPORTED, "a regular cache needs blocks under 4 GiB (all layers, K and V)");
  if (!aligned16(d.device_base) || !aligned16(d.host_base) || !aligned16(d.rc_base))
    return fail(SC_ERR_INVALID, "caller-owned pool tiers must be 16-byte aligned");
  // Pools over caller-owned HBM without a host tier make no HIP call here.
  const bool needs_hip = (d.n_device_blocks > 0 && !d.device_base) || d.n_host_blocks > 0 ||
                         (d.n_rc_blocks > 0 && !d.rc_base);
  std::unique_ptr<DeviceGuard> guard;
  if (needs_hip) {
    guard.reset(new DeviceGuard(d.device));
    if (!guard->ok()) return fail(SC_ERR_INVALID, "cannot select device %d", d.device);
  }
  std::unique_ptr<sc_pool> p(new sc_pool());
  p->desc = d;
  p->dev_lent = d.n_device_blocks;
  p->row_bytes = (size_t)d.n_kv_heads * d.head_dim * 2;
  p->slice_bytes = 2 * (size_t)d.block_size * p->row_bytes;   // Eq. 1 with bf16
  p->block_bytes = (size_t)d.n_layers * p->slice_bytes;
  const size_t dev_bytes = (size_t)d.n_device_blocks * p->block_bytes;
  const size_t host_bytes = (size_t)d.n_host_blocks * p->block_bytes;
  if (d.n_device_blocks > 0) {
    if (d.device_base) {
      p->dev_base = static_cast<char *>(d.device_base);
    } else {
      // Elastic (chunk-mapped) when the runtime supports virtual memory
      // management for the device, one allocation otherwise.
      hipError_t e = vmm_create(p.get(), d.n_device_blocks);
      if (e == hipErrorNotSupported) {
        e = hipMalloc(reinterpret_cast<void **>(&p->dev_base), dev_bytes);
        if (e != hipSuccess) return fail(SC_ERR_OOM, "hipMalloc(%zu) for the device tier: %s", dev_bytes,
                                         hipGetErrorString(e));
      } else if (e != hipSuccess) {
        return fail(SC_ERR_OOM, "mapping %zu bytes for the device tier: %s", dev_bytes, hipGetErrorString(e));
      }
      p->own_dev = true;
    }
  }
  if (d.n_host_blocks > 0) {
    if (d.host_base) {
      p->host_base = static_cast<char *>(d.host_base);
    } else {
      hipError_t e = hipHostMalloc(reinterpret_cast<void **>(&p->host_base), host_bytes,
                                   hipHostMallocMapped | hipHostMallocPortable);
      if (e != hipSuccess) {
        if (p->vmm) vmm_destroy(p.get());
        else if (p->own_dev) (void)hipFree(p->dev_base);
        return fail(SC_ERR_OOM, "hipHostMalloc(%zu) for the host tier: %s", host_bytes, hipGetErrorString(e));
      }
      p->own_host = true;
    }
    void *devp = nullptr;
    hipError_t e = hipHostGetDevicePointer(&devp, p->host_base, 0);
    if (e != hipSuccess || devp == nullptr) {
      if (p->vmm) vmm_destroy(p.get());
      else if (p->own_dev) (void)hipFree(p->dev_base);
      if (p->own_host) (void)hipHostFree(p->host_base);
      return fail(SC_ERR_INVALID, "host tier is not pinned, mapped memory: %s", hipGetErrorString(e));
    }
    p->host_dev = static_cast<char *>(devp);
  }
  if (d.n_rc_blocks > 0) {
    if (d.rc_base) {
      p->rc_base = static_cast<char *>(d.rc_base);
    } else {
      const size_t rc_bytes = (size_t)d.n_rc_blocks * p->block_bytes;
      hipError_t e = hipMalloc(reinterpret_cast<void **>(&p->rc_base), rc_bytes);
      if (e != hipSuccess) {
        if (p->vmm) vmm_destroy(p.get());
        else if (p->own_dev) (void)hipFree(p->dev_base);
        if (p->own_host) (void)hipHostFree(p->host_base);
        return fail(SC_ERR_OOM, "hipMalloc(%zu) for the regular cache: %s", rc_bytes, hipGetErrorString(e));
      }
      p->own_rc = true;
    }
  }
  *out = p.release();
  return SC_OK;
}

void sc_pool_destroy(sc_pool *pool) {
  if (!pool) return;
  if (pool->own_dev || pool->own_host || pool->own_rc) {
    DeviceGuard guard(pool->desc.device);
    if (pool->vmm) vmm_destroy(pool);
    else if (pool->own_dev && pool->dev_base) (void)hipFree(pool->dev_base);
    if (pool->own_host && pool->host_base) (void)hipHostFree(pool->host_base);
    if (pool->own_rc && pool->rc_base) (void)hipFree(pool->rc_base);
  }
  delete pool;
}

sc_status sc_pool_resize(sc_pool *pool, int64_t n_device_blocks) {
  clear_error();
  if (!pool) return fail(SC_ERR_INVALID, "null pool");
  if (n_device_blocks < 0 || n_device_blocks > pool->desc.n_device_blocks)
    return fail(SC_ERR_RANGE, "HBM blocks %lld outside [0, %lld] (the capacity given at creation)",
                (long long)n_device_blocks, (long long)pool->desc.n_device_blocks);
  std::lock_guard<std::mutex> lk(pool->mu);
  if (!pool->live_max_dev.empty() && *pool->live_max_dev.rbegin() >= n_device_blocks)
    return fail(SC_ERR_INVALID, "a live table still references HBM block %lld", (long long)*pool->live_max_dev.rbegin());
  // Block-major layout: the blocks that stay keep their addresses; the ones
  // released (or appended) are the last ones.  No data moves.  A
  // chunk-mapped tier also frees (or maps) the physical memory of the
  // chunks past (up to) the new count.
  if (pool->vmm) {
    DeviceGuard guard(pool->desc.device);
    const int64_t need = (n_device_blocks + pool->vmm_chunk_blocks - 1) / pool->vmm_chunk_blocks;
    const int64_t had = (int64_t)pool->vmm_handles.size();
    if (need < had) {
      // Work already queued (e.g. by tables since destroyed) may still read
      // the chunks about to go.
      SC_HIP(hipDeviceSynchronize());
      while ((int64_t)pool->vmm_handles.size() > need) {
        const hipError_t e = vmm_release_last_chunk(pool);
        if (e != hipSuccess) {
          // The chunk's handle is gone either way: keep every usable id
          // mapped, so no later table can name a block of a lost chunk.
          pool->dev_lent = std::min<int64_t>(pool->dev_lent,
                                             (int64_t)pool->vmm_handles.size() * pool->vmm_chunk_blocks);
          return fail_hip(e, "releasing HBM blocks");
        }
      }
    }
    while ((int64_t)pool->vmm_handles.size() < need) {
      hipError_t e = vmm_append_chunk(pool);
      if (e != hipSuccess) {
        while ((int64_t)pool->vmm_handles.size() > had) (void)vmm_release_last_chunk(pool);
        return fail(SC_ERR_OOM, "mapping HBM blocks [%lld, %lld): %s",
                    (long long)(had * pool->vmm_chunk_blocks), (long long)n_device_blocks, hipGetErrorString(e));
      }
    }
  }
  pool->dev_lent = n_device_blocks;
  return SC_OK;
}

sc_status sc_pool_layout_get(const sc_pool *pool, sc_pool_layout *out) {
  clear_error();
  if (!pool || !out) return fail(SC_ERR_INVALID, "null argument");
  out->device_base = pool->dev_base;
  out->host_base = pool->host_base;
  out->slice_bytes = pool->slice_bytes;
  out->block_bytes = pool->block_bytes;
  out->row_bytes = pool->row_bytes;
  out->n_device_blocks = pool->desc.n_device_blocks;
  out->n_host_blocks = pool->desc.n_host_blocks;
  out->rc_base = pool->rc_base;
  out->n_rc_blocks = pool->desc.n_rc_blocks;
  out->dtype = pool->desc.dtype;
  std::lock_guard<std::mutex> lk(const_cast<sc_pool *>(pool)->mu);
  out->device_blocks_lent = pool->dev_lent;
  out->device_bytes_mapped = pool->vmm ? (int64_t)(pool->vmm_handles.size() * pool->vmm_chunk_bytes)
                                       : (pool->own_dev ? (int64_t)(pool->desc.n_device_blocks * pool->block_bytes) : 0);
  out->device_chunk_blocks = pool->vmm ? pool->vmm_chunk_blocks : 0;
  return SC_OK;
}

sc_status sc_table_create(sc_pool *pool, int32_t batch, const int32_t *block_ids, const int32_t *cu_blocks,
                          const int32_t *prefix_len, const int32_t *new_len, void *stream, sc_table **out) {
  clear_error();
  if (!pool || !cu_blocks || !prefix_len || !new_len || !out) return fail(SC_ERR_INVALID, "null argument");
  *out = nullptr;
  if (batch <= 0) return fail(SC_ERR_INVALID, "batch must be positive (got %d)", batch);
  const int bs = pool->desc.block_size;
  const int64_t n_dev = pool->desc.n_device_blocks;
  const int64_t n_rc0 = n_dev + pool->desc.n_host_blocks;   // first regular-cache id
  const int64_t n_all = n_rc0 + pool->desc.n_rc_blocks;
  if (cu_blocks[0] != 0) return fail(SC_ERR_INVALID, "cu_blocks[0] must be 0");
  int64_t total_kv = 0;
  for (int b = 0; b < batch; ++b) {
    if (prefix_len[b] < 0 || new_len[b] < 0)
      return fail(SC_ERR_INVALID, "negative length in sequence %d", b);
    const int64_t need = ((int64_t)prefix_len[b] + new_len[b] + bs - 1) / bs;
    if ((int64_t)cu_blocks[b + 1] - cu_blocks[b] != need)
      return fail(SC_ERR_INVALID, "sequence %d lists %d blocks, needs ceil((%d+%d)/%d) = %lld", b,
                  cu_blocks[b + 1] - cu_blocks[b], prefix_len[b], new_len[b], bs, (long long)need);
    total_kv += (int64_t)prefix_len[b] + new_len[b];
  }
  if (total_kv >= INT32_MAX) return fail(SC_ERR_RANGE, "batch too long for 32-bit row indices");
  const int64_t n_ids = cu_blocks[batch];
  if (n_ids > 0 && !block_ids) return fail(SC_ERR_INVALID, "null block_ids");
  std::vector<uint8_t> seen((size_t)n_all, 0);
  int64_t lent;
  {
    std::lock_guard<std::mutex> lk(pool->mu);
    lent = pool->dev_lent;
  }
  int64_t max_dev_id = -1;
  for (int64_t i = 0; i < n_ids; ++i) {
    const int32_t id = block_ids[i];
    if (id < 0 || id >= n_all)
      return fail(SC_ERR_RANGE, "block id %d at entry %lld outside the pool [0, %lld)", id, (long long)i,
                  (long long)n_all);
    if (id < n_dev && id >= lent)
      return fail(SC_ERR_RANGE, "block id %d at entry %lld is beyond the %lld HBM blocks the pool lends now", id,
                  (long long)i, (long long)lent);
    if (seen[id]) return fail(SC_ERR_INVALID, "block id %d used twice in one table", id);
    seen[id] = 1;
    if (id < n_dev) max_dev_id = std::max<int64_t>(max_dev_id, id);
  }
  // Regular-cache blocks: the leading, completely filled prefix blocks only.
  std::vector<int32_t> rc_keys(batch, 0), rc_off(batch, 0), rc_ids;
  for (int b = 0; b < batch; ++b) {
    const int32_t *ids = block_ids + cu_blocks[b];
    const int n_b = cu_blocks[b + 1] - cu_blocks[b];
    int r = 0;
    while (r < n_b && ids[r] >= n_rc0) ++r;
    for (int j = r; j < n_b; ++j)
      if (ids[j] >= n_rc0)
        return fail(SC_ERR_INVALID, "sequence %d: regular-cache block %d follows a non-regular block", b, ids[j]);
    if ((int64_t)r * bs > prefix_len[b])
      return fail(SC_ERR_INVALID, "sequence %d: regular-cache block %d is not filled by the prefix", b,
                  ids[r - 1]);
    rc_keys[b] = r * bs;
    rc_off[b] = (int32_t)rc_ids.size();
    for (int j = 0; j < r; ++j) rc_ids.push_back((int32_t)(ids[j] - n_rc0));
  }

  std::unique_ptr<sc_table> t(new sc_table());
  t->pool = pool;
  t->batch = batch;
  t->P.assign(prefix_len, prefix_len + batch);
  t->N.assign(new_len, new_len + batch);
  t->cu_q.assign(batch + 1, 0);
  t->cu_k.assign(batch + 1, 0);
  for (int b = 0; b < batch; ++b) {
    t->cu_q[b + 1] = t->cu_q[b] + new_len[b];
    t->cu_k[b + 1] = t->cu_k[b] + prefix_len[b] + new_len[b];
  }
  t->total_q = t->cu_q[batch];
  t->total_kv = t->cu_k[batch];
  t->rc_keys = rc_keys;
  t->rc_off = rc_off;
  t->h_rc_ids = rc_ids;

  auto locate = [&](int32_t id, CopyItem *it) {
    it->tier = id >= n_dev ? 1 : 0;
    const int64_t local = it->tier ? id - n_dev : id;
    it->pool_off = local * (int64_t)pool->block_bytes;
  };
  std::vector<CopyItem> fetch, append, store;
  for (int b = 0; b < batch; ++b) {
    const int32_t *ids = block_ids + cu_blocks[b];
    const int P = prefix_len[b], N = new_len[b];
    for (int j = rc_keys[b] / bs; j * bs < P; ++j) {   // regular-cache blocks are read in place
      CopyItem it{};
      locate(ids[j], &it);
      it.act_row = t->cu_k[b] + (int64_t)j * bs;
      it.nrows = std::min(bs, P - j * bs);
      fetch.push_back(it);
    }
    for (int i0 = 0; i0 < N; i0 += bs) {
      CopyItem it{};
      it.src_row = t->cu_q[b] + i0;
      it.act_row = t->cu_k[b] + P + i0;
      it.nrows = std::min(bs, N - i0);
      append.push_back(it);
    }
    for (int64_t pos = P; pos < (int64_t)P + N;) {
      const int64_t blk = pos / bs;
      const int64_t end = std::min<int64_t>((blk + 1) * bs, (int64_t)P + N);
      CopyItem it{};
      locate(ids[blk], &it);
      it.pool_off += (pos % bs) * (int64_t)pool->row_bytes;
      it.src_row = t->cu_q[b] + (pos - P);
      it.nrows = (int32_t)(end - pos);
      store.push_back(it);
      pos = end;
    }
  }
  t->n_fetch = (int32_t)fetch.size();
  for (const CopyItem &it : fetch) t->n_fetch_host += it.tier;
  t->n_append = (int32_t)append.size();
  t->n_store = (int32_t)store.size();
  std::vector<CopyItem> &all = t->h_items;
  all.reserve(fetch.size() + append.size() + store.size());
  all.insert(all.end(), fetch.begin(), fetch.end());
  all.insert(all.end(), append.begin(), append.end());
  all.insert(all.end(), store.begin(), store.end());
  DeviceGuard guard(pool->desc.device);
  if (!all.empty()) {
    const size_t bytes = all.size() * sizeof(CopyItem);
    hipError_t e = hipMalloc(reinterpret_cast<void **>(&t->d_items), bytes);
    if (e != hipSuccess) return fail(SC_ERR_OOM, "hipMalloc for table items: %s", hipGetErrorString(e));
    // The source stays alive in the table until it is destroyed.
    e = hipMemcpyAsync(t->d_items, all.data(), bytes, hipMemcpyHostToDevice, (hipStream_t)stream);
    if (e != hipSuccess) {
      (void)hipFree(t->d_items);
      t->d_items = nullptr;
      return fail_hip(e, "table upload");
    }
  }
  if (!t->h_rc_ids.empty()) {
    const size_t bytes = t->h_rc_ids.size() * sizeof(int32_t);
    hipError_t e = hipMalloc(reinterpret_cast<void **>(&t->d_rc_ids), bytes);
    if (e == hipSuccess)
      e = hipMemcpyAsync(t->d_rc_ids, t->h_rc_ids.data(), bytes, hipMemcpyHostToDevice, (hipStream_t)stream);
    if (e != hipSuccess) {
      if (t->d_items) (void)hipFree(t->d_items);
      if (t->d_rc_ids) (void)hipFree(t->d_rc_ids);
      t->d_items = nullptr;
      t->d_rc_ids = nullptr;
      return fail_hip(e, "table upload (regular-cache ids)");
    }
  }
  {
    // Register with the pool; a resize may have shrunk it meanwhile.
    std::lock_guard<std::mutex> lk(pool->mu);
    if (max_dev_id >= pool->dev_lent) {
      if (t->d_items) (void)hipFree(t->d_items);
      if (t->d_rc_ids) (void)hipFree(t->d_rc_ids);
      t->d_items = nullptr;
      t->d_rc_ids = nullptr;
      return fail(SC_ERR_RANGE, "the pool shrank below block %lld while the table was being created",
                  (long long)max_dev_id);
    }
    t->max_dev_id = max_dev_id;
    pool->live_max_dev.insert(max_dev_id);
  }
  *out = t.release();
  return SC_OK;
}

void sc_table_destroy(sc_table *table) {
  if (!table) return;
  {
    std::lock_guard<std::mutex> lk(table->pool->mu);
    auto it = table->pool->live_max_dev.find(table->max_dev_id);
    if (it != table->pool->live_max_dev.end()) table->pool->live_max_dev.erase(it);
  }
  if (table->d_items || table->d_sync || table->d_rc_ids || table->last_overlap || !table->plans.empty()) {
    DeviceGuard guard(table->pool->desc.device);
    if (table->d_items) (void)hipFree(table->d_items);
    if (table->d_sync) (void)hipFree(table->d_sync);
    if (table->last_overlap) (void)hipEventDestroy(table->last_overlap);
    if (table->d_rc_ids) (void)hipFree(table->d_rc_ids);
    for (auto &kv : table->plans) free_plan(&kv.second);
  }
  delete table;
}

sc_status sc_attn_plan_query(int32_t batch, const int32_t *prefix_len, const int32_t *new_len,
                             const int32_t *rc_keys, int32_t n_q_heads, int32_t n_kv_heads, int32_t slots,
                             int32_t *n_items, int32_t *items, int32_t capacity, int32_t *splits) {
  clear_error();
  if (batch <= 0 || !prefix_len || !new_len || !n_items) return fail(SC_ERR_INVALID, "null argument");
  sc_status st = check_heads(n_q_heads, n_kv_heads, 128);
  if (st != SC_OK) return st;
  for (int b = 0; b < batch; ++b) {
    if (prefix_len[b] < 0 || new_len[b] < 0) return fail(SC_ERR_INVALID, "negative length");
    if (rc_keys && (rc_keys[b] < 0 || rc_keys[b] > prefix_len[b]))
      return fail(SC_ERR_INVALID, "sequence %d: regular-cache keys %d outside [0, %d]", b, rc_keys[b],
                  prefix_len[b]);
  }
  std::vector<int32_t> rc;
  if (rc_keys) rc.assign(rc_keys, rc_keys + batch);
  AttnPlan plan;
  plan_attention(std::vector<int32_t>(prefix_len, prefix_len + batch),
                 std::vector<int32_t>(new_len, new_len + batch), n_q_heads, n_kv_heads,
                 slots > 0 ? slots : kQueryDefaultSlots, &plan, rc, std::vector<int32_t>(rc.size(), 0));
  *n_items = plan.n_items;
  if (items) {
    if (capacity < plan.n_items) return fail(SC_ERR_RANGE, "capacity %d < %d items", capacity, plan.n_items);
    std::memcpy(items, plan.items.data(), plan.items.size() * sizeof(WorkItem));
  }
  if (splits)
    for (int b = 0; b < batch; ++b) splits[b] = plan.seqs[b].n_splits;
  return SC_OK;
}

sc_status sc_table_totals(const sc_table *table, int64_t *total_q, int64_t *total_kv) {
  clear_error();
  if (!table) return fail(SC_ERR_INVALID, "null table");
  if (total_q) *total_q = table->total_q;
  if (total_kv) *total_kv = table->total_kv;
  return SC_OK;
}

sc_status sc_stack_wait_kind(const sc_table *table, uint32_t flags, int32_t *device_wait) {
  clear_error();
  if (!table || !device_wait) return fail(SC_ERR_INVALID, "null argument");
  sc::DeviceGuard guard(table->pool->desc.device);
  *device_wait = sc::stack_device_wait(table, flags) ? 1 : 0;
  return SC_OK;
}

sc_status sc_table_stack_status(const sc_table *table, int32_t *timed_out, int32_t clear) {
  clear_error();
  if (!table || !timed_out) return fail(SC_ERR_INVALID, "null argument");
  *timed_out = 0;
  if (!table->d_sync) return SC_OK;
  sc::DeviceGuard guard(table->pool->desc.device);
  uint64_t flag = 0;
  SC_HIP(hipMemcpy(&flag, table->d_sync + 1, sizeof(flag), hipMemcpyDeviceToHost));
  *timed_out = flag != 0 ? 1 : 0;
  if (clear && flag != 0) {
    const uint64_t zero = 0;
    SC_HIP(hipMemcpy(table->d_sync + 1, &zero, sizeof(zero), hipMemcpyHostToDevice));
  }
  return SC_OK;
}

sc_status sc_fetch_layer_kv(sc_pool *pool, const sc_table *table, int32_t layer, const sc_active *dst,
                            void *stream) {
  clear_error();
  if (!pool || !table) return fail(SC_ERR_INVALID, "null argument");
  if (table->pool != pool) return fail(SC_ERR_INVALID, "table belongs to another pool");
  if (layer < 0 || layer >= pool->desc.n_layers)
    return fail(SC_ERR_RANGE, "layer %d outside [0, %d)", layer, pool->desc.n_layers);
  sc_status st = check_active(table, dst);
  if (st != SC_OK) return st;
  DeviceGuard guard(pool->desc.device);
  return do_fetch(pool, table, layer, dst, (hipStream_t)stream);
}

sc_status sc_fetch_layer_kv_dma(sc_pool *pool, const sc_table *table, int32_t layer, const sc_active *dst,
                                int32_t per_copy_calls, void *stream) {
  clear_error();
  if (!pool || !table) return fail(SC_ERR_INVALID, "null argument");
  if (table->pool != pool) return fail(SC_ERR_INVALID, "table belongs to another pool");
  if (layer < 0 || layer >= pool->desc.n_layers)
    return fail(SC_ERR_RANGE, "layer %d outside [0, %d)", layer, pool->desc.n_layers);
  sc_status st = check_active(table, dst);
  if (st != SC_OK) return st;
  DeviceGuard guard(pool->desc.device);
  hipStream_t s = (hipStream_t)stream;
  // Host-tier items: two copies each (the K and V halves of the block's
  // layer slice are contiguous in the pool but go to different buffers).
  std::vector<void *> dsts, srcs;
  std::vector<size_t> sizes;
  const int64_t layer_off = (int64_t)layer * (int64_t)pool->slice_bytes;
  for (int32_t i = 0; i < table->n_fetch; ++i) {
    const CopyItem &it = table->h_items[i];
    if (it.tier != 1) continue;
    char *src = pool->host_base + it.pool_off + layer_off;
    const size_t bytes = (size_t)it.nrows * pool->row_bytes;
    dsts.push_back(static_cast<char *>(dst->k) + it.act_row * (int64_t)pool->row_bytes);
    srcs.push_back(src);
    sizes.push_back(bytes);
    dsts.push_back(static_cast<char *>(dst->v) + it.act_row * (int64_t)pool->row_bytes);
    srcs.push_back(src + pool->slice_bytes / 2);
    sizes.push_back(bytes);
  }
  if (!dsts.empty()) {
    if (per_copy_calls) {
      for (size_t i = 0; i < dsts.size(); ++i)
        SC_HIP(hipMemcpyAsync(dsts[i], srcs[i], sizes[i], hipMemcpyHostToDevice, s));
    } else {
      // Looked up at run time: the HIP runtime a process loads (e.g. the
      // one bundled with its framework) may predate the batch call.
      using BatchFn = hipError_t (*)(void **, void **, size_t *, size_t, hipMemcpyAttributes *, size_t *, size_t,
                                     size_t *, hipStream_t);
      static BatchFn batch = reinterpret_cast<BatchFn>(dlsym(RTLD_DEFAULT, "hipMemcpyBatchAsync"));
      if (batch == nullptr)
        return fail(SC_ERR_UNSUPPORTED, "hipMemcpyBatchAsync is not in the loaded HIP runtime");
      size_t fail_idx = 0;
      SC_HIP(batch(dsts.data(), srcs.data(), sizes.data(), dsts.size(), nullptr, nullptr, 0, &fail_idx, s));
    }
  }
  CopyArgs a = copy_args(pool, table, COPY_FETCH);
  a.tier_mask = 1;   // device-tier items only
  a.layer_off = layer_off;
  a.act_k = static_cast<char *>(dst->k);
  a.act_v = static_cast<char *>(dst->v);
  if (table->n_fetch_host < table->n_fetch) {
    hipError_t e = launch_kv_copy(a, s);
    if (e != hipSuccess) return fail_hip(e, "fetch launch");
  }
  return SC_OK;
}

sc_status sc_append_new_kv(sc_pool *pool, const sc_table *table, const void *k_new, const void *v_new,
                           const sc_active *dst, void *stream) {
  clear_error();
  if (!pool || !table) return fail(SC_ERR_INVALID, "null argument");
  if (table->pool != pool) return fail(SC_ERR_INVALID, "table belongs to another pool");
  if (table->total_q > 0 && (!k_new || !v_new)) return fail(SC_ERR_INVALID, "null k_new/v_new");
  if (!aligned16(k_new) || !aligned16(v_new)) return fail(SC_ERR_INVALID, "k_new/v_new not 16-byte aligned");
  sc_status st = check_active(table, dst);
  if (st != SC_OK) return st;
  DeviceGuard guard(pool->desc.device);
  return do_append(pool, table, k_new, v_new, dst, (hipStream_t)stream);
}

sc_status sc_store_layer_kv(sc_pool *pool, const sc_table *table, int32_t layer, const void *k_new,
                            const void *v_new, void *stream) {
  clear_error();
  if (!pool || !table) return fail(SC_ERR_INVALID, "null argument");
  if (table->pool != pool) return fail(SC_ERR_INVALID, "table belongs to another pool");
  if (layer < 0 || layer >= pool->desc.n_layers)
    return fail(SC_ERR_RANGE, "layer %d outside [0, %d)", layer, pool->desc.n_layers);
  if (table->total_q > 0 && (!k_new || !v_new)) return fail(SC_ERR_INVALID, "null k_new/v_new");
  if (!aligned16(k_new) || !aligned16(v_new)) return fail(SC_ERR_INVALID, "k_new/v_new not 16-byte aligned");
  DeviceGuard guard(pool->desc.device);
  return do_store(pool, table, layer, k_new, v_new, (hipStream_t)stream);
}


sc_status sc_prefill_attn(const void *q, const void *k_active, const void *v_active, int32_t prefix_len,
                          int32_t new_len, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, float scale,
                          void *out, float *lse, void *stream) {
  clear_error();
  return prefill_attn_single(q, k_active, v_active, prefix_len, new_len, n_q_heads, n_kv_heads, head_dim,
                             SC_DTYPE_BF16, scale, out, lse, stream);
}

sc_status sc_prefill_attn_f16(const void *q, const void *k_active, const void *v_active, int32_t prefix_len,
                              int32_t new_len, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, float scale,
                              void *out, float *lse, void *stream) {
  clear_error();
  return prefill_attn_single(q, k_active, v_active, prefix_len, new_len, n_q_heads, n_kv_heads, head_dim,
                             SC_DTYPE_F16, scale, out, lse, stream);
}

sc_status sc_prefill_attn_noalloc(const void *q, const void *k_active, const void *v_active, int32_t prefix_len,
                                  int32_t new_len, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                  float scale, void *out, float *lse, void *stream) {
  clear_error();
  if (prefix_len < 0 || new_len < 0) return fail(SC_ERR_INVALID, "negative length");
  sc_status st = check_heads(n_q_heads, n_kv_heads, head_dim);
  if (st != SC_OK) return st;
  if (new_len == 0) return SC_OK;
  if (!q || !k_active || !v_active || !out) return fail(SC_ERR_INVALID, "null argument");
  if (!aligned16(q) || !aligned16(k_active) || !aligned16(v_active) || !aligned16(out))
    return fail(SC_ERR_INVALID, "q, k_active, v_active and out must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(lse) & 3) != 0) return fail(SC_ERR_INVALID, "lse must be 4-byte aligned");
  if (!keys_fit_offsets((int64_t)prefix_len + new_len, n_kv_heads, head_dim))
    return fail(SC_ERR_UNSUPPORTED,
                "sequence of %lld tokens x %d KV heads x head_dim %d exceeds 2 GiB of keys less %d tokens",
                (long long)prefix_len + new_len, n_kv_heads, head_dim, kKeyOffsetMarginTokens);
  int device = 0;
  SC_HIP(hipGetDevice(&device));
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess || cus <= 0)
    cus = 256;
  int S = 1;
  if (!single_splits_noalloc(prefix_len, new_len, n_q_heads, n_kv_heads, cus * kResidentPerCu, &S))
    return fail(SC_ERR_RANGE, "new turn of %d tokens needs more work items than the allocation-free planner "
                "holds (%d query tiles x splits)", new_len, kNoAllocMaxCosts);
  void *scr = nullptr;
  size_t scr_bytes = 0;
  SC_HIP(noalloc_scratch(device, &scr, &scr_bytes));
  const size_t rows = (size_t)S * new_len * n_q_heads;
  const size_t need = S > 1 ? rows * ((size_t)head_dim * sizeof(uint16_t) + sizeof(float)) : 0;
  if (need > scr_bytes)
    return fail(SC_ERR_RANGE, "%d key splits x %d tokens x %d heads need %zu bytes of split-key scratch; the "
                "allocation-free entry point has %zu", S, new_len, n_q_heads, need, scr_bytes);
  const int group = n_q_heads / n_kv_heads;
  const int rows_q = kAttnRows / group;
  const int n_qt = (new_len + rows_q - 1) / rows_q;
  const int64_t total_items = (int64_t)n_kv_heads * n_qt * S;
  AttnArgs a{};
  a.q = static_cast<const uint16_t *>(q);
  a.k = static_cast<const uint16_t *>(k_active);
  a.v = static_cast<const uint16_t *>(v_active);
  a.out = static_cast<uint16_t *>(out);
  a.lse = lse;
  a.n_seqs = 1;
  a.total_q = new_len;
  a.n_q_heads = n_q_heads;
  a.n_kv_heads = n_kv_heads;
  a.group = group;
  a.rows_q = rows_q;
  a.dtype = SC_DTYPE_BF16;
  if (!(scale > 0.f)) scale = 1.f / std::sqrt((float)head_dim);
  a.scale_log2 = scale * 1.4426950408889634f;
  a.seq0 = SeqDesc{0, 0, prefix_len, new_len, S, 0, 0, 0};
  a.imp_tiles = n_qt;
  a.imp_splits = S;
  a.imp_per_xcd = (int32_t)((total_items + kXcds - 1) / kXcds);
  if (S > 1) {
    a.part_o = static_cast<uint16_t *>(scr);
    a.part_lse = reinterpret_cast<float *>(a.part_o + rows * head_dim);
  }
  hipError_t e = launch_attn_fwd(a, head_dim, kXcds * a.imp_per_xcd, (hipStream_t)stream);
  if (e != hipSuccess) return fail_hip(e, "attn_fwd launch");
  if (S > 1) {
    e = launch_attn_merge(a, head_dim, (hipStream_t)stream);
    if (e != hipSuccess) return fail_hip(e, "attn_merge launch");
  }
  return SC_OK;
}

sc_status sc_attn_noalloc_splits(int32_t prefix_len, int32_t new_len, int32_t n_q_heads, int32_t n_kv_heads,
                                 int32_t slots, int32_t *splits) {
  clear_error();
  if (!splits) return fail(SC_ERR_INVALID, "null argument");
  if (prefix_len < 0 || new_len < 0) return fail(SC_ERR_INVALID, "negative length");
  sc_status st = check_heads(n_q_heads, n_kv_heads, 128);
  if (st != SC_OK) return st;
  int S = 1;
  if (!single_splits_noalloc(prefix_len, new_len, n_q_heads, n_kv_heads, slots > 0 ? slots : kQueryDefaultSlots,
                             &S))
    return fail(SC_ERR_RANGE, "shape exceeds the allocation-free planner's buffers");
  *splits = S;
  return SC_OK;
}

sc_status sc_prefill_attn_varlen(sc_pool *pool, const sc_table *table, int32_t layer, const void *q,
                                 const sc_active *kv, int32_t n_q_heads, float scale, void *out, float *lse,
                                 void *stream) {
  clear_error();
  if (!pool || !table) return fail(SC_ERR_INVALID, "null argument");
  if (table->pool != pool) return fail(SC_ERR_INVALID, "table belongs to another pool");
  if (layer < 0 || layer >= pool->desc.n_layers)
    return fail(SC_ERR_RANGE, "layer %d outside [0, %d)", layer, pool->desc.n_layers);
  sc_status st = check_active(table, kv);
  if (st != SC_OK) return st;
  if (table->total_q == 0) return SC_OK;
  if (!q || !out) return fail(SC_ERR_INVALID, "null argument");
  if (!aligned16(q) || !aligned16(out)) return fail(SC_ERR_INVALID, "q and out must be 16-byte aligned");
  if ((reinterpret_cast<uintptr_t>(lse) & 3) != 0) return fail(SC_ERR_INVALID, "lse must be 4-byte aligned");
  DeviceGuard guard(pool->desc.device);
  AttnPlan *plan = nullptr;
  st = table_plan(const_cast<sc_table *>(table), n_q_heads, &plan);
  if (st != SC_OK) return st;
  const sc_pool_desc &d = pool->desc;
  RcView rc{pool, layer, table->d_rc_ids};
  return run_attention(d.device, *plan, q, kv->k, kv->v, out, lse, n_q_heads, d.n_kv_heads, d.head_dim, d.dtype,
                       scale, (hipStream_t)stream, nullptr, 0, nullptr, rc);
}

}  // extern "C"

namespace sc {
namespace {

// The layer stack (sc_prefill_stack); chunk_tokens > 0 runs each layer's
// attention as one launch per chunk of the new turn over the same fetched
// slot (sc_prefill_stack_chunked).
sc_status prefill_stack(sc_pool *pool, const sc_table *table, int32_t n_layers, const void *const *q_per_layer,
                        const void *const *knew_per_layer, const void *const *vnew_per_layer,
                        void *const *out_per_layer, const sc_active *slots, int32_t n_q_heads, float scale,
                        uint32_t flags, int32_t chunk_tokens, void *compute_stream, void *copy_stream) {
  if (!pool || !table || !q_per_layer || !knew_per_layer || !vnew_per_layer || !out_per_layer || !slots)
    return fail(SC_ERR_INVALID, "null argument");
  if (table->pool != pool) return fail(SC_ERR_INVALID, "table belongs to another pool");
  if (n_layers <= 0 || n_layers > pool->desc.n_layers)
    return fail(SC_ERR_RANGE, "n_layers %d outside [1, %d]", n_layers, pool->desc.n_layers);
  if (flags & ~(uint32_t)(SC_STACK_MODE_MASK | SC_STACK_NO_STORE | SC_STACK_TEST_NEVER_READY |
                          SC_STACK_DEBUG_POISON | SC_STACK_TEST_NEVER_FREE | SC_STACK_EVENT_WAIT))
    return fail(SC_ERR_INVALID, "unknown flags");
  const uint32_t mode = flags & SC_STACK_MODE_MASK;
  if (mode > SC_STACK_ATTN_ONLY) return fail(SC_ERR_INVALID, "unknown stack mode");
  const bool never_ready = (flags & SC_STACK_TEST_NEVER_READY) != 0;
  const bool poison = (flags & SC_STACK_DEBUG_POISON) != 0;
  if (poison && mode == SC_STACK_ATTN_ONLY)
    return fail(SC_ERR_INVALID, "SC_STACK_DEBUG_POISON needs a stack that fetches");
  if (never_ready && mode != SC_STACK_OVERLAP)
    return fail(SC_ERR_INVALID, "SC_STACK_TEST_NEVER_READY needs SC_STACK_OVERLAP");
  const bool never_free = (flags & SC_STACK_TEST_NEVER_FREE) != 0;
  if (never_free && mode != SC_STACK_OVERLAP)
    return fail(SC_ERR_INVALID, "SC_STACK_TEST_NEVER_FREE needs SC_STACK_OVERLAP");
  if ((flags & SC_STACK_EVENT_WAIT) && mode != SC_STACK_OVERLAP)
    return fail(SC_ERR_INVALID, "SC_STACK_EVENT_WAIT needs SC_STACK_OVERLAP");
  const bool do_st = !(flags & SC_STACK_NO_STORE);
  const int n_slots = mode == SC_STACK_SERIAL ? 1 : 2;
  for (int s = 0; s < n_slots; ++s) {
    sc_status st = check_active(table, &slots[s]);
    if (st != SC_OK) return st;
  }
  if (mode == SC_STACK_OVERLAP && copy_stream == nullptr)
    return fail(SC_ERR_INVALID, "overlapped mode needs a copy stream");
  for (int l = 0; l < n_layers; ++l) {
    if (!q_per_layer[l] || !out_per_layer[l] || (table->total_q > 0 && (!knew_per_layer[l] || !vnew_per_layer[l])))
      return fail(SC_ERR_INVALID, "null per-layer pointer at layer %d", l);
    if (!aligned16(q_per_layer[l]) || !aligned16(out_per_layer[l]) || !aligned16(knew_per_layer[l]) ||
        !aligned16(vnew_per_layer[l]))
      return fail(SC_ERR_INVALID, "per-layer pointer at layer %d not 16-byte aligned", l);
  }
  DeviceGuard guard(pool->desc.device);
  const sc_pool_desc &d = pool->desc;
  // A fetch that reaches into the host tier runs on CU-partitioned streams
  // (see split_streams); the caller's streams then only order the work.
  SplitStreams *ss = nullptr;
  if (mode == SC_STACK_OVERLAP && table->n_fetch_host > 0) {
    sc_status st = split_streams(d.device, &ss);
    if (st != SC_OK) return st;
  }
  // One plan, or one per chunk of the new turn.
  int n_chunks = 1;
  if (chunk_tokens > 0) {
    int64_t max_n = 0;
    for (int32_t x : table->N) max_n = std::max<int64_t>(max_n, x);
    n_chunks = (int)std::max<int64_t>(1, (max_n + chunk_tokens - 1) / chunk_tokens);
  }
  std::vector<AttnPlan *> plans(n_chunks, nullptr);
  sc_status st = SC_OK;
  for (int c = 0; c < n_chunks; ++c) {
    st = table_plan(const_cast<sc_table *>(table), n_q_heads, &plans[c], ss ? ss->attn_cus * kResidentPerCu : 0,
                    chunk_tokens > 0 ? chunk_tokens : 0, c);
    if (st != SC_OK) return st;
  }
  hipStream_t caller_cs = (hipStream_t)compute_stream;
  hipStream_t cs = ss ? ss->attn : caller_cs;
  hipStream_t xs = ss ? ss->copy : (hipStream_t)copy_stream;
  // Split-key merges are deferred when every layer runs one plan with key
  // splits: the forward kernel of layer l merges layer l-1's partials
  // (chunks of rows claimed by its workgroups once their own items are
  // done), and one merge kernel follows the last layer.  That saves a merge launch per layer and its ~6 us on the
  // 8B shape.  Partials alternate between two halves of one workspace,
  // held for the whole enqueue.
  const bool defer_merge = n_chunks == 1 && plans[0]->max_splits > 1;
  std::unique_lock<std::mutex> dws_hold;
  char *dws = nullptr;
  size_t dws_half = 0;
  uint32_t *claims = nullptr;             // one claim counter per layer
  if (defer_merge) {
    dws_half = (plan_ws_bytes(*plans[0], n_q_heads, d.head_dim) + 255) & ~(size_t)255;
    const size_t claim_bytes = ((size_t)n_layers * sizeof(uint32_t) + 255) & ~(size_t)255;
    void *w = nullptr;
    st = get_workspace(d.device, cs, 2 * dws_half + claim_bytes, &w, &dws_hold);
    if (st != SC_OK) return st;
    dws = static_cast<char *>(w);
    claims = reinterpret_cast<uint32_t *>(dws + 2 * dws_half);
    // Zeroed by a fill kernel on the attention stream, before any forward
    // kernel of this stack.
    hipError_t e = launch_kv_fill(claims, claim_bytes, 0, cs);
    if (e != hipSuccess) return fail_hip(e, "claim counter reset");
  }
  auto stack_merge = [&](int l) {
    StackMerge m;
    m.ws = dws + (size_t)(l & 1) * dws_half;
    if (l > 0) {
      m.prev_ws = dws + (size_t)((l - 1) & 1) * dws_half;
      m.prev_out = out_per_layer[l - 1];
      m.prev_counter = claims + (l - 1);
    }
    return m;
  };
  auto last_merge = [&]() -> sc_status {
    if (!defer_merge) return SC_OK;
    return run_merge(*plans[0], dws + (size_t)((n_layers - 1) & 1) * dws_half, out_per_layer[n_layers - 1],
                     n_q_heads, d.n_kv_heads, d.head_dim, d.dtype, cs);
  };
  // The first chunk waits for the slot; the slot-free event follows the
  // last chunk's forward kernel.
  // A forced time-out (tests of the failure path) waits for a count the
  // copy stream never reaches, with a spin limit of a few hundred polls.
  const uint64_t never = never_ready ? (uint64_t)1 << 40 : 0;
  const int spin_limit = never_ready ? kAttnTestSpinLimit : kAttnReadySpinLimit;
  auto attn = [&](int l, const sc_active &slot, const uint64_t *ready_flag = nullptr, uint64_t ready_value = 0,
                  hipEvent_t after_fwd = nullptr, uint64_t *done_counter = nullptr) {
    RcView rc{pool, l, table->d_rc_ids};
    const StackMerge sm = defer_merge ? stack_merge(l) : StackMerge();
    for (int c = 0; c < n_chunks; ++c) {
      sc_status r = run_attention(d.device, *plans[c], q_per_layer[l], slot.k, slot.v, out_per_layer[l], nullptr,
                                  n_q_heads, d.n_kv_heads, d.head_dim, d.dtype, scale, cs,
                                  c == 0 ? ready_flag : nullptr, ready_value + (ready_flag ? never : 0),
                                  c == n_chunks - 1 ? after_fwd : nullptr, rc, spin_limit, done_counter,
                                  defer_merge ? &sm : nullptr, poison);
      if (r != SC_OK) return r;
    }
    return SC_OK;
  };

  if (mode == SC_STACK_ATTN_ONLY) {
    for (int l = 0; l < n_layers; ++l) {
      st = attn(l, slots[l & 1]);
      if (st != SC_OK) return st;
    }
    return last_merge();
  }
  // Debug poisoning: NaN patterns over a slot's K and V before it is refilled.
  auto poison_slot = [&](const sc_active &slot, hipStream_t s) -> sc_status {
    const size_t bytes = (size_t)table->total_kv * pool->row_bytes;
    const uint16_t nan16 = d.dtype == SC_DTYPE_F16 ? 0x7E00 : 0x7FC0;
    hipError_t e = launch_kv_fill(slot.k, bytes, nan16, s);
    if (e == hipSuccess) e = launch_kv_fill(slot.v, bytes, nan16, s);
    return e == hipSuccess ? SC_OK : fail_hip(e, "slot poison launch");
  };
  if (mode == SC_STACK_SERIAL) {
    for (int l = 0; l < n_layers; ++l) {
      if (poison && (st = poison_slot(slots[0], cs)) != SC_OK) return st;
      if ((st = do_fetch(pool, table, l, &slots[0], cs)) != SC_OK) return st;
      if ((st = do_append(pool, table, knew_per_layer[l], vnew_per_layer[l], &slots[0], cs)) != SC_OK) return st;
      if ((st = attn(l, slots[0])) != SC_OK) return st;
      if (do_st && (st = do_store(pool, table, l, knew_per_layer[l], vnew_per_layer[l], cs)) != SC_OK) return st;
    }
    return last_merge();
  }

  // Overlapped.  Attention of layer l waits on the device for the copy
  // stream's count of filled slots (table->d_sync[0], written by the copy
  // stream after the layer's copy); a stream-level wait here would put a
  // command-processor round trip (about 12 us measured) in front of every
  // attention.  In the other direction the copy stream runs a one-wave gate
  // kernel that waits until every forward workgroup of the attention that
  // last read slot s has counted itself done (table->d_sync[2]); fetch,
  // append and store of the layer then run as one launch.  Per layer that
  // leaves the host two launches on the copy stream, one counter write and
  // the attention's launches, where separate copy launches and an event
  // record plus a cross-stream wait cost about twice as much host time,
  // which bounded short turns.  Without the device wait (a copy workgroup
  // could be kept off a CU by attention) the streams wait on events.
  // Disjoint CU sets (host tier) never block each other.
  const bool device_wait = stack_device_wait(table, flags);
  if ((never_ready || never_free) && !device_wait)
    return fail(SC_ERR_UNSUPPORTED, "this stack waits on stream events; there is no device wait to time out");
  // One overlapped stack with a device-side wait at a time per table (they
  // share its slot counter, whose values must rise in the order the stacks
  // run on the device): hold the table's stack lock from reserving the
  // counter values until everything is enqueued, and start after the
  // previous such stack ended.
  sc_table *tw = const_cast<sc_table *>(table);
  std::unique_lock<std::mutex> stack_lock(tw->stack_mu, std::defer_lock);
  if (device_wait) {
    stack_lock.lock();
    if (!tw->last_overlap) {
      hipError_t he = hipEventCreateWithFlags(&tw->last_overlap, hipEventDisableTiming);
      if (he != hipSuccess) {
        tw->last_overlap = nullptr;
        return fail_hip(he, "hipEventCreate");
      }
    }
  }
  uint64_t *sync = nullptr, base = 0;
  if (device_wait) {
    std::lock_guard<std::mutex> lk(const_cast<sc_table *>(table)->mu);
    sc_table *t = const_cast<sc_table *>(table);
    if (!t->d_sync) {
      SC_HIP(hipMalloc(reinterpret_cast<void **>(&t->d_sync), 4 * sizeof(uint64_t)));
      const uint64_t zero[4] = {0, 0, 0, 0};
      SC_HIP(hipMemcpy(t->d_sync, zero, sizeof(zero), hipMemcpyHostToDevice));
    }
    sync = t->d_sync;
    base = t->sync_gen;
    t->sync_gen += (uint64_t)n_layers + 1;
  }
  // free_[s] only orders a write after a read of slot s (the next fetch into
  // it after the forward kernel that read it); no data flows through it, so
  // it is recorded without the system-scope release, whose cache write-back
  // (the split-key partials the forward kernel just wrote) measured ~7 us
  // between every forward kernel and its merge.
  hipEvent_t ev[6] = {};
  for (int i = 0; i < 6; ++i) {
    const bool war_only = i == 2 || i == 3;
    hipError_t he = hipEventCreateWithFlags(
        &ev[i], war_only ? (hipEventDisableTiming | hipEventDisableSystemFence) : hipEventDisableTiming);
    if (he != hipSuccess) {
      for (auto &x : ev)
        if (x) (void)hipEventDestroy(x);
      return fail_hip(he, "hipEventCreate");
    }
  }
  hipEvent_t *ready = ev, *free_ = ev + 2, start = ev[4], done = ev[5];
  // Host-tier fetches already run on their own CUs (split streams).
  const size_t reserve = ss ? 0 : copy_lds_reserve(d.device, d.head_dim);
  const int groups = ss ? 0 : copy_groups_beside_attention(d.device, table, n_q_heads, d.head_dim);
  // Forward workgroups per layer (every chunk's launch counts itself).
  uint64_t fwd_groups = 0;
  for (const AttnPlan *pl : plans) fwd_groups += (uint64_t)pl->n_items;
  const uint32_t nan2 = (d.dtype == SC_DTYPE_F16 ? 0x7E00u : 0x7FC0u) * 0x10001u;
  const uint64_t never_f = never_free ? (uint64_t)1 << 40 : 0;
  const int gate_spin = never_free ? kAttnTestSpinLimit : kAttnReadySpinLimit;
  auto body = [&]() -> sc_status {
    sc_status r0;
    if (device_wait && tw->last_overlap_recorded) SC_HIP(hipStreamWaitEvent(caller_cs, tw->last_overlap, 0));
    // The done count starts from zero for this stack; the copy stream
    // starts after this write (event below).
    if (device_wait) SC_HIP(hipStreamWriteValue64(caller_cs, sync + 2, 0, 0));
    // Both streams start after everything already queued on the caller's
    // compute stream.
    SC_HIP(hipEventRecord(start, caller_cs));
    SC_HIP(hipStreamWaitEvent(xs, start, 0));
    if (cs != caller_cs) SC_HIP(hipStreamWaitEvent(cs, start, 0));
    for (int l = 0; l < n_layers; ++l) {
      const int s = l & 1;
      sc_status r;
      if (device_wait) {
        // Slot s was last read by attention(l-2): wait for layers 0..l-2.
        if (l >= 2) {
          hipError_t e = launch_slot_gate(sync + 2, (uint64_t)(l - 1) * fwd_groups + never_f,
                                          reinterpret_cast<uint32_t *>(sync + 1), sync + 3, base + l + 1,
                                          gate_spin, xs);
          if (e != hipSuccess) return fail_hip(e, "slot gate launch");
        }
        if (poison && (r = poison_slot(slots[s], xs)) != SC_OK) return r;
        LayerCopyArgs la = layer_copy_args(pool, table, l, knew_per_layer[l], vnew_per_layer[l], &slots[s], do_st);
        la.fail_word = sync + 3;
        la.fail_tag = base + l + 1;
        la.nan2 = nan2;
        hipError_t e = launch_kv_layer_copy(la, xs, reserve, groups);
        if (e != hipSuccess) return fail_hip(e, "layer copy launch");
        SC_HIP(hipStreamWriteValue64(xs, sync, base + l + 1, 0));
        if ((r = attn(l, slots[s], sync, base + l + 1, nullptr, sync + 2)) != SC_OK) return r;
        continue;
      }
      if (l >= 2) SC_HIP(hipStreamWaitEvent(xs, free_[s], 0));
      if (poison && (r = poison_slot(slots[s], xs)) != SC_OK) return r;
      if ((r = do_fetch(pool, table, l, &slots[s], xs, reserve, groups)) != SC_OK) return r;
      if ((r = do_append(pool, table, knew_per_layer[l], vnew_per_layer[l], &slots[s], xs, reserve, groups)) !=
          SC_OK)
        return r;
      SC_HIP(hipEventRecord(ready[s], xs));
      if (do_st &&
          (r = do_store(pool, table, l, knew_per_layer[l], vnew_per_layer[l], xs, reserve, groups)) != SC_OK)
        return r;
      SC_HIP(hipStreamWaitEvent(cs, ready[s], 0));
      if ((r = attn(l, slots[s], nullptr, 0, free_[s])) != SC_OK) return r;
    }
    if ((r0 = last_merge()) != SC_OK) return r0;
    // The caller's compute stream ends after the last attention and store.
    SC_HIP(hipEventRecord(start, xs));
    SC_HIP(hipStreamWaitEvent(caller_cs, start, 0));
    if (cs != caller_cs) {
      SC_HIP(hipEventRecord(done, cs));
      SC_HIP(hipStreamWaitEvent(caller_cs, done, 0));
    }
    if (device_wait) {
      SC_HIP(hipEventRecord(tw->last_overlap, caller_cs));
      tw->last_overlap_recorded = true;
    }
    return SC_OK;
  };
  st = body();
  for (auto &e : ev) (void)hipEventDestroy(e);
  return st;
}

}  // namespace
}  // namespace sc

extern "C" {

sc_status sc_prefill_stack(sc_pool *pool, const sc_table *table, int32_t n_layers, const void *const *q_per_layer,
                           const void *const *knew_per_layer, const void *const *vnew_per_layer,
                           void *const *out_per_layer, const sc_active *slots, int32_t n_q_heads, float scale,
                           uint32_t flags, void *compute_stream, void *copy_stream) {
  clear_error();
  return prefill_stack(pool, table, n_layers, q_per_layer, knew_per_layer, vnew_per_layer, out_per_layer, slots,
                       n_q_heads, scale, flags, 0, compute_stream, copy_stream);
}

sc_status sc_prefill_stack_chunked(sc_pool *pool, const sc_table *table, int32_t n_layers,
                                   const void *const *q_per_layer, const void *const *knew_per_layer,
                                   const void *const *vnew_per_layer, void *const *out_per_layer,
                                   const sc_active *slots, int32_t n_q_heads, float scale, uint32_t flags,
                                   int32_t chunk_tokens, void *compute_stream, void *copy_stream) {
  clear_error();
  if (chunk_tokens <= 0) return fail(SC_ERR_INVALID, "chunk_tokens must be positive (got %d)", chunk_tokens);
  return prefill_stack(pool, table, n_layers, q_per_layer, knew_per_layer, vnew_per_layer, out_per_layer, slots,
                       n_q_heads, scale, flags, chunk_tokens, compute_stream, copy_stream);
}

}  // extern "C"
