// Capacity planning of the master's caches (§3.2, Eq. 1-5) and the worker's
// elastic-cache decisions (§3.4, Eq. 6-9, Algorithm 1).  Host integer
// arithmetic; every product is checked for 64-bit overflow.  The O(1)
// resize of the block-major donor tier itself is sc_pool_resize (sc_api.cpp),
// since it needs the pool's bookkeeping.
#include <cstdint>
#include <numeric>

#include "sc_internal.h"

namespace sc {
namespace {

bool mul_ok(int64_t a, int64_t b, int64_t *out) { return !__builtin_mul_overflow(a, b, out); }

bool shape_ok(const sc_model_shape *m) {
  return m && m->n_layers > 0 && m->block_size > 0 && m->n_kv_heads > 0 && m->head_dim > 0 && m->dtype_bytes > 0;
}

// Eq. 6 / 7: elements of one block over all layers of a model.
bool block_elems(const sc_model_shape *m, int64_t *out) {
  int64_t v = m->n_layers;
  return mul_ok(v, m->block_size, &v) && mul_ok(v, m->n_kv_heads, &v) && mul_ok(v, m->head_dim, out);
}

int64_t ceil_div(int64_t a, int64_t b) { return a / b + (a % b != 0); }

sc_status check_alg1_args(int64_t worker_blocks, int32_t block_size, int64_t meu_w, int64_t meu_m,
                          const int64_t *dw, const int64_t *dm) {
  if (!dw || !dm) return fail(SC_ERR_INVALID, "null argument");
  if (worker_blocks < 0) return fail(SC_ERR_INVALID, "worker_blocks must be >= 0");
  if (block_size <= 0 || meu_w <= 0 || meu_m <= 0)
    return fail(SC_ERR_INVALID, "block size and elastic units must be positive");
  return SC_OK;
}

}  // namespace
}  // namespace sc

using namespace sc;

extern "C" {

sc_status sc_plan_capacity(const sc_model_shape *master, int64_t master_cache_bytes,
                           const int64_t *worker_cache_bytes, int32_t n_workers, int64_t *k_workers,
                           sc_capacity *out) {
  clear_error();
  if (!out) return fail(SC_ERR_INVALID, "null argument");
  if (!shape_ok(master)) return fail(SC_ERR_INVALID, "master shape must be positive in every field");
  if (n_workers < 0 || (n_workers > 0 && !worker_cache_bytes))
    return fail(SC_ERR_INVALID, "bad worker list");
  if (master_cache_bytes < 0) return fail(SC_ERR_INVALID, "negative master cache size");
  // Eq. 1.
  int64_t mb = 2;
  if (!mul_ok(mb, master->block_size, &mb) || !mul_ok(mb, master->n_kv_heads, &mb) ||
      !mul_ok(mb, master->head_dim, &mb) || !mul_ok(mb, master->dtype_bytes, &mb))
    return fail(SC_ERR_RANGE, "M_block overflows");
  int64_t mb_all_layers;
  if (!mul_ok(mb, master->n_layers, &mb_all_layers)) return fail(SC_ERR_RANGE, "M_block * L overflows");
  // Eq. 2, summed.
  int64_t sum_k = 0;
  for (int32_t i = 0; i < n_workers; ++i) {
    if (worker_cache_bytes[i] < 0) return fail(SC_ERR_INVALID, "negative cache size for worker %d", i);
    const int64_t k = worker_cache_bytes[i] / mb_all_layers;
    if (k_workers) k_workers[i] = k;
    if (__builtin_add_overflow(sum_k, k, &sum_k)) return fail(SC_ERR_RANGE, "sum of K_i overflows");
  }
  // Eq. 3-5.
  const int64_t k_master = master_cache_bytes / mb;
  const int64_t n_lsc = std::min(sum_k, k_master);
  const int64_t n_rc = sum_k < k_master ? (k_master - sum_k) / master->n_layers : 0;
  int64_t tokens;
  if (!mul_ok(n_lsc + n_rc, master->block_size, &tokens)) return fail(SC_ERR_RANGE, "context length overflows");
  out->m_block_bytes = mb;
  out->k_master = k_master;
  out->sum_k_workers = sum_k;
  out->n_lsc = n_lsc;
  out->n_rc = n_rc;
  out->max_context_tokens = tokens;
  out->conventional_blocks = k_master / master->n_layers;
  return SC_OK;
}

sc_status sc_elastic_unit(const sc_model_shape *master, const sc_model_shape *worker, int64_t *meu_master,
                          int64_t *meu_worker) {
  clear_error();
  if (!meu_master || !meu_worker) return fail(SC_ERR_INVALID, "null argument");
  if (!shape_ok(master) || !shape_ok(worker)) return fail(SC_ERR_INVALID, "model shapes must be positive");
  int64_t be_m, be_w;
  if (!block_elems(master, &be_m) || !block_elems(worker, &be_w)) return fail(SC_ERR_RANGE, "BE overflows");
  // Eq. 8-9: lcm = be_m / gcd * be_w, so MEU_m = be_w / gcd and MEU_w = be_m / gcd.
  const int64_t g = std::gcd(be_m, be_w);
  int64_t lcm;
  if (!mul_ok(be_m / g, be_w, &lcm)) return fail(SC_ERR_RANGE, "LCM_elem overflows");
  *meu_master = lcm / be_m;
  *meu_worker = lcm / be_w;
  return SC_OK;
}

sc_status sc_scale_up(int64_t worker_blocks, int32_t worker_block_size, int64_t meu_worker, int64_t meu_master,
                      int64_t request_len, int64_t *worker_delta, int64_t *master_delta) {
  clear_error();
  sc_status st = check_alg1_args(worker_blocks, worker_block_size, meu_worker, meu_master, worker_delta,
                                 master_delta);
  if (st != SC_OK) return st;
  if (request_len < 0) return fail(SC_ERR_INVALID, "negative request length");
  const int64_t need = ceil_div(request_len, worker_block_size);
  int64_t dw = 0, dm = 0;
  if (need > worker_blocks) {
    const int64_t k = ceil_div(need - worker_blocks, meu_worker);
    if (!mul_ok(k, meu_worker, &dw) || !mul_ok(k, meu_master, &dm)) return fail(SC_ERR_RANGE, "delta overflows");
  }
  *worker_delta = dw;
  *master_delta = dm;
  return SC_OK;
}

sc_status sc_scale_down(int64_t worker_blocks, int32_t worker_block_size, int64_t meu_worker, int64_t meu_master,
                        const int64_t *window_lens, int32_t n_window, int64_t *worker_delta,
                        int64_t *master_delta) {
  clear_error();
  sc_status st = check_alg1_args(worker_blocks, worker_block_size, meu_worker, meu_master, worker_delta,
                                 master_delta);
  if (st != SC_OK) return st;
  if (n_window < 0 || (n_window > 0 && !window_lens)) return fail(SC_ERR_INVALID, "bad request window");
  int64_t max_len = 0;
  for (int32_t i = 0; i < n_window; ++i) {
    if (window_lens[i] < 0) return fail(SC_ERR_INVALID, "negative request length at %d", i);
    max_len = std::max(max_len, window_lens[i]);
  }
  const int64_t max_need = ceil_div(max_len, worker_block_size);
  int64_t dw = 0, dm = 0;
  if (max_need < worker_blocks) {
    const int64_t k = (worker_blocks - max_need) / meu_worker;
    if (!mul_ok(k, meu_worker, &dw) || !mul_ok(k, meu_master, &dm)) return fail(SC_ERR_RANGE, "delta overflows");
  }
  *worker_delta = dw;
  *master_delta = dm;
  return SC_OK;
}

}  // extern "C"
