// Causal GQA prefill attention over prefix + new tokens (§2.2: every token
// attends to all tokens before it, and a new turn's tokens attend to the
// cached history plus the new tokens; GQA as used by the models of §5).
//
// Output row (query i of a sequence with P cached tokens, query head h):
//   o = sum_{j <= P + i} softmax_j(scale * q . k_j) v_j,  KV head g = h / group.
//
// Work decomposition (built on the host, see plan_attention): a workgroup
// owns 128 (query, head) rows = rows_q consecutive queries times the `group`
// query heads that share one KV head, and a range of keys.  Packing the
// heads of a group into the rows makes every K/V tile that is staged through
// LDS serve all of them.  Long key ranges are split over several workgroups
// (split-key); each writes a normalised fp32 partial output and its
// log-sum-exp, and attn_merge_kernel combines them exactly
// (o = sum_s exp(lse_s - lse) o_s).
//
// Per workgroup: 4 waves, each owning 32 rows.  Keys are walked in tiles of
// 64 that are double-buffered in LDS: the next tile's global loads are in
// flight while the current tile is consumed.  Per tile and wave:
//   S^T (32 keys x 32 rows) += K_tile . Q^T    MFMA 32x32x16 bf16, K-dim = D
//   online softmax on S^T: every lane holds 16 keys of ONE row per 32-key
//     block, so the row max / sum need only one exchange between the two
//     32-lane halves of the wave; exp2 with scale * log2(e) folded in
//   O^T (D x 32 rows) += V^T . P^T            MFMA 32x32x16 bf16, K-dim = keys
// The probabilities P never leave registers: the S^T accumulator layout is
// already the B-operand layout of the PV product once rounded to bf16, for a
// fixed permutation of the 16 keys of each MFMA step; V^T is read from the
// row-major V tile with that same permutation.
#include "sc_internal.h"

#include <cmath>

namespace sc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int KT = kAttnKeyTile;
static_assert(kAttnRows == 4 * 32, "four waves of 32 rows");
static_assert(KT == 64, "two 32-key MFMA blocks per tile");

// 32x32 MFMA accumulator layout: element r of lane l holds C[m][n] with
// n = l % 32 and m = 8 * (r / 4) + 4 * (l / 32) + r % 4.
__device__ __forceinline__ int acc_m(int r, int half) { return 8 * (r >> 2) + 4 * half + (r & 3); }

template <int D>
struct Geo {
  static constexpr int kChunksPerRow = D / 8;                       // 16-byte chunks
  static constexpr int kChunksPerThread = KT * kChunksPerRow / kThreads;
  static constexpr int kLdsStride = D + 8;                          // bf16 per LDS row (padded)
  static constexpr int kTileElems = KT * kLdsStride;
  static_assert(kChunksPerThread * kThreads == KT * kChunksPerRow, "tile split");
};

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 x) { return __builtin_bit_cast(bf16x8, x); }

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(AttnArgs a) {
  using G_ = Geo<D>;
  constexpr int NCH = G_::kChunksPerThread;
  constexpr int LS = G_::kLdsStride;
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * 2 * G_::kTileElems];

  const WorkItem w = a.items[blockIdx.x];
  if (w.seq < 0) return;
  const SeqDesc sd = a.seqs[w.seq];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int half = lane >> 5;
  const int col = lane & 31;
  const int group = a.group;
  const int row = wave * 32 + col;
  const int qi = row / group;
  const int hg = row - qi * group;
  const bool valid = qi < w.nq;
  const int qpos = w.q0 + (valid ? qi : w.nq - 1);
  const int h = w.kvh * group + hg;
  const int64_t qrow = (int64_t)(sd.cu_q + qpos) * a.n_q_heads + h;

  // Q^T fragments (B operand): lane holds Q[row][16 s + 8 half .. + 7].
  bf16x8 qf[D / 16];
  {
    const u32x4 *qp = reinterpret_cast<const u32x4 *>(a.q + qrow * D);
#pragma unroll
    for (int s = 0; s < D / 16; ++s) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (valid) x = qp[2 * s + half];
      qf[s] = as_bf16x8(x);
    }
  }

  const int64_t kv_stride = (int64_t)a.n_kv_heads * D;
  const uint16_t *kbase = a.k + (int64_t)sd.cu_k * kv_stride + (int64_t)w.kvh * D;
  const uint16_t *vbase = a.v + (int64_t)sd.cu_k * kv_stride + (int64_t)w.kvh * D;
  const int diag_all = sd.prefix + w.q0;   // keys <= diag_all are visible to every row
  const int my_last = sd.prefix + qpos;    // this row sees keys <= my_last
  const int k_end = w.k_end;

  u32x4 kr[NCH], vr[NCH];
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + kThreads * i;
      const int r = c / G_::kChunksPerRow;
      const int cc = c % G_::kChunksPerRow;
      const int key = kt + r;
      u32x4 zk = {0u, 0u, 0u, 0u};
      u32x4 zv = zk;
      if (key < k_end) {
        zk = *reinterpret_cast<const u32x4 *>(kbase + key * kv_stride + cc * 8);
        zv = *reinterpret_cast<const u32x4 *>(vbase + key * kv_stride + cc * 8);
      }
      kr[i] = zk;
      vr[i] = zv;
    }
  };
  auto store_tile = [&](int buf) {
    uint16_t *sk = smem + buf * 2 * G_::kTileElems;
    uint16_t *sv = sk + G_::kTileElems;
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + kThreads * i;
      const int r = c / G_::kChunksPerRow;
      const int cc = c % G_::kChunksPerRow;
      *reinterpret_cast<u32x4 *>(sk + r * LS + cc * 8) = kr[i];
      *reinterpret_cast<u32x4 *>(sv + r * LS + cc * 8) = vr[i];
    }
  };

  float m_run = -INFINITY;  // running max of scaled scores, log2 units
  float l_run = 0.f;        // this lane's share of the running denominator
  f32x16 oacc[D / 32];
#pragma unroll
  for (int c = 0; c < D / 32; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[c][r] = 0.f;

  load_tile(w.k_begin);
  store_tile(0);
  __syncthreads();

  int buf = 0;
  for (int kt = w.k_begin; kt < k_end; kt += KT) {
    const bool has_next = kt + KT < k_end;
    if (has_next) load_tile(kt + KT);

    const uint16_t *sk = smem + buf * 2 * G_::kTileElems;
    const uint16_t *sv = sk + G_::kTileElems;

    // S^T = K . Q^T for two 32-key blocks.
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
      const uint16_t *krow = sk + (32 * kb + col) * LS + 8 * half;
#pragma unroll
      for (int s = 0; s < D / 16; ++s) {
        const bf16x8 kf = as_bf16x8(*reinterpret_cast<const u32x4 *>(krow + 16 * s));
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sacc[kb], 0, 0, 0);
      }
    }

    // Causal mask and the end of the key range; only tiles that reach past
    // the first row's diagonal or past k_end need it.
    if (kt + KT > k_end || kt + KT - 1 > diag_all) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kt + 32 * kb + acc_m(r, half);
          if (key >= k_end || key > my_last) sacc[kb][r] = -INFINITY;
        }
    }

    // Online softmax (log2 domain).
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx * a.scale_log2);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float corr = __builtin_amdgcn_exp2f(m_run - m_use);
    float rs = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(sacc[kb][r] * a.scale_log2 - m_use);
        sacc[kb][r] = p;
        rs += p;
      }
    l_run = l_run * corr + rs;
    m_run = m_new;
#pragma unroll
    for (int c = 0; c < D / 32; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[c][r] *= corr;

    // O^T += V^T . P^T.  MFMA step (kb, t) covers keys 32 kb + 16 t + [0, 16);
    // k-slot e of a lane in half `half` holds key 32 kb + 16 t + 4 half +
    // (e < 4 ? e : e + 4), matching accumulator elements 8 t + e.
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        bf16x8 pf;
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[e] = (__bf16)sacc[kb][8 * t + e];
        const int key0 = 32 * kb + 16 * t + 4 * half;
#pragma unroll
        for (int c = 0; c < D / 32; ++c) {
          const uint16_t *vcol = sv + 32 * c + col;
          bf16x8 vf;
#pragma unroll
          for (int e = 0; e < 8; ++e)
            vf[e] = __builtin_bit_cast(__bf16, vcol[(key0 + (e < 4 ? e : e + 4)) * LS]);
          oacc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, oacc[c], 0, 0, 0);
        }
      }

    if (has_next) store_tile(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  // Epilogue: combine the two halves' denominators, normalise, write.
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_val = l_tot > 0.f ? (m_run + __log2f(l_tot)) * 0.69314718055994530942f : -INFINITY;
  if (!valid) return;
  if (sd.n_splits == 1) {
    uint16_t *orow = a.out + qrow * D;
#pragma unroll
    for (int c = 0; c < D / 32; ++c)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int dim = 32 * c + 8 * g4 + 4 * half;
        u32x2 pk;
        __bf16 b0 = (__bf16)(oacc[c][4 * g4 + 0] * inv), b1 = (__bf16)(oacc[c][4 * g4 + 1] * inv);
        __bf16 b2 = (__bf16)(oacc[c][4 * g4 + 2] * inv), b3 = (__bf16)(oacc[c][4 * g4 + 3] * inv);
        pk[0] = (uint32_t)__builtin_bit_cast(uint16_t, b0) | ((uint32_t)__builtin_bit_cast(uint16_t, b1) << 16);
        pk[1] = (uint32_t)__builtin_bit_cast(uint16_t, b2) | ((uint32_t)__builtin_bit_cast(uint16_t, b3) << 16);
        *reinterpret_cast<u32x2 *>(orow + dim) = pk;
      }
    if (a.lse != nullptr && half == 0) a.lse[(int64_t)h * a.total_q + sd.cu_q + qpos] = lse_val;
  } else {
    const int64_t prow = ((int64_t)w.split * a.total_q + sd.cu_q + qpos) * a.n_q_heads + h;
    float *po = a.part_o + prow * D;
#pragma unroll
    for (int c = 0; c < D / 32; ++c)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int dim = 32 * c + 8 * g4 + 4 * half;
        f32x4 x;
        x[0] = oacc[c][4 * g4 + 0] * inv;
        x[1] = oacc[c][4 * g4 + 1] * inv;
        x[2] = oacc[c][4 * g4 + 2] * inv;
        x[3] = oacc[c][4 * g4 + 3] * inv;
        *reinterpret_cast<f32x4 *>(po + dim) = x;
      }
    if (half == 0) a.part_lse[prow] = lse_val;
  }
}

// One wave per (token, head) row of a split sequence: weights
// exp(lse_s - lse) over the splits, weighted sum of the partial outputs.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  constexpr int PER_LANE = D / 64;
  const int64_t wrow = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t n_rows = (int64_t)a.total_q * a.n_q_heads;
  if (wrow >= n_rows) return;
  const int token = (int)(wrow / a.n_q_heads);
  const int h = (int)(wrow - (int64_t)token * a.n_q_heads);
  int lo = 0, hi = a.n_seqs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.seqs[mid].cu_q <= token) lo = mid; else hi = mid - 1;
  }
  const int S = a.seqs[lo].n_splits;
  if (S <= 1) return;
  const int64_t split_stride = (int64_t)a.total_q * a.n_q_heads;
  float mx = -INFINITY;
  for (int s = 0; s < S; ++s) mx = fmaxf(mx, a.part_lse[s * split_stride + wrow]);
  float acc[PER_LANE];
#pragma unroll
  for (int j = 0; j < PER_LANE; ++j) acc[j] = 0.f;
  float wsum = 0.f;
  for (int s = 0; s < S; ++s) {
    const float ls = a.part_lse[s * split_stride + wrow];
    const float wgt = (ls == -INFINITY) ? 0.f : __expf(ls - mx);
    wsum += wgt;
    const float *po = a.part_o + (s * split_stride + wrow) * D + lane * PER_LANE;
#pragma unroll
    for (int j = 0; j < PER_LANE; ++j) acc[j] += wgt * po[j];
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  uint16_t *orow = a.out + wrow * D + lane * PER_LANE;
#pragma unroll
  for (int j = 0; j < PER_LANE; ++j) orow[j] = __builtin_bit_cast(uint16_t, (__bf16)(acc[j] * inv));
  if (a.lse != nullptr && lane == 0)
    a.lse[(int64_t)h * a.total_q + token] = wsum > 0.f ? mx + __logf(wsum) : -INFINITY;
}

}  // namespace

hipError_t launch_attn_fwd(const AttnArgs &a, int head_dim, int n_items, hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  if (head_dim == 128)
    hipLaunchKernelGGL(attn_fwd_kernel<128>, dim3(n_items), dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<64>, dim3(n_items), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_attn_merge(const AttnArgs &a, int head_dim, hipStream_t stream) {
  const int64_t rows = (int64_t)a.total_q * a.n_q_heads;
  if (rows <= 0) return hipSuccess;
  const int64_t blocks = (rows * 64 + 255) / 256;
  if (head_dim == 128)
    hipLaunchKernelGGL(attn_merge_kernel<128>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(attn_merge_kernel<64>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace sc
