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
// (split-key): each writes a normalised fp32 partial output and its
// log-sum-exp, and attn_merge_kernel combines them exactly
// (o = sum_s exp(lse_s - lse) o_s).  The merge is a separate launch: merging
// in the last-arriving workgroup would need device-scope fences, whose L2
// write-back / invalidate stalls the other workgroups streaming K/V.
//
// Per workgroup: 4 waves, each owning 32 rows.  Keys are walked in tiles of
// 64 that are double-buffered in LDS: the next tile's global loads are in
// flight while the current tile is consumed.  Per tile and wave:
//   S^T (32 keys x 32 rows) += K_tile . Q^T    MFMA 32x32x16 bf16, K-dim = D
//   online softmax on S^T: every lane holds 16 keys of ONE row per 32-key
//     block, so the row max needs one exchange between the two 32-lane
//     halves of the wave; exp2 with scale * log2(e) folded in
//   O^T (D x 32 rows) += V^T . P^T            MFMA 32x32x16 bf16, K-dim = keys
// The probabilities never leave registers: the S^T accumulator layout is the
// B-operand layout of the PV product once rounded to bf16, for a fixed
// permutation of the 16 keys of each MFMA step.  V^T operands come from the
// row-major V tile through LDS transpose reads (ds_read_b64_tr_b16): in each
// 16-lane group, lanes 4r..4r+3 read 4 dims each of key r and lane j gets
// dim j of the 4 keys.
//
// The running max is only moved (and O, l rescaled) when a row's tile max
// exceeds it by more than kRescaleSlack (log2 units); otherwise the
// exponentials stay below 2^kRescaleSlack.  The result is the same softmax,
// with fewer rescale passes over the accumulators.
#include "sc_internal.h"

#include <cmath>
#include <type_traits>

namespace sc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr int kThreads = 256;
constexpr int KT = kAttnKeyTile;
constexpr float kRescaleSlack = 8.0f;
static_assert(kAttnRows == 4 * 32, "four waves of 32 rows");
static_assert(KT == 64, "two 32-key MFMA blocks per tile");

// 32x32 MFMA accumulator layout: element r of lane l holds C[m][n] with
// n = l % 32 and m = 8 * (r / 4) + 4 * (l / 32) + r % 4.
__device__ __forceinline__ int acc_m(int r, int half) { return 8 * (r >> 2) + 4 * half + (r & 3); }

template <int D>
struct Geo {
  static constexpr int kChunksPerRow = D / 8;                        // 16-byte chunks per key row
  static constexpr int kChunksPerThread = KT * kChunksPerRow / kThreads;
  // K rows: 16-byte reads of 16 consecutive keys fall on disjoint banks.
  static constexpr int kLdsK = D + 8;
  // V rows: the 8 rows of one transpose read (64 bytes each) fall on
  // disjoint bank ranges (row stride = 16 dwords mod 64).
  static constexpr int kLdsV = D + 32;
  static constexpr int kTileK = KT * kLdsK;
  static constexpr int kTileV = KT * kLdsV;
  static constexpr int kBuf = kTileK + kTileV;
  static_assert(kChunksPerThread * kThreads == KT * kChunksPerRow, "tile split");
};

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 x) { return __builtin_bit_cast(bf16x8, x); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two floats to packed bf16 (round to nearest even), one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  const bf16x2 p = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, p);
}

// Value of the same lane in the other 32-lane half of the wave.
__device__ __forceinline__ float max_with_other_half(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x),
                                                  __builtin_bit_cast(uint32_t, x), false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}

// One 64-key tile for one wave: S^T, (mask), online softmax, O^T += V^T P^T.
template <int D, bool MASK>
__device__ __forceinline__ void attend_tile(const uint16_t *smem_buf, const bf16x8 (&qf)[D / 16],
                                            f32x16 (&oacc)[D / 32], float &m_run, float &l_run, int lane,
                                            float scale_log2, int kt, int k_end, int my_last) {
  using G_ = Geo<D>;
  const int half = lane >> 5;
  const int col = lane & 31;

  // Two independent accumulation chains (the two 32-key blocks), interleaved.
  f32x16 sacc[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) sacc[kb][r] = 0.f;
  const uint16_t *krow = smem_buf + col * G_::kLdsK + 8 * half;
#pragma unroll
  for (int s = 0; s < D / 16; ++s)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const bf16x8 kf = as_bf16x8(*reinterpret_cast<const u32x4 *>(krow + 32 * kb * G_::kLdsK + 16 * s));
      sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sacc[kb], 0, 0, 0);
    }

  if (MASK) {
    // Element (kb, r) holds key kt + 32 kb + acc_m(r, half); it is visible
    // when that offset is <= lim (the last visible key of this row in the
    // range, relative to kt), i.e. when 32 kb + acc_m(r, 0) <= lim - 4 half.
    const int lim = min(k_end - 1, my_last) - kt - 4 * half;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (32 * kb + acc_m(r, 0) > lim) sacc[kb][r] = -INFINITY;
  }

  // Row max over this lane's 32 scores: four independent chains.
  float m4[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) m4[i] = fmaxf(sacc[i >> 1][8 * (i & 1)], sacc[i >> 1][8 * (i & 1) + 1]);
#pragma unroll
  for (int r = 2; r < 8; ++r)
#pragma unroll
    for (int i = 0; i < 4; ++i) m4[i] = fmaxf(m4[i], sacc[i >> 1][8 * (i & 1) + r]);
  float mx = fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3]));
  mx = max_with_other_half(mx);
  const float tmax = mx * scale_log2;
  const bool need = tmax > m_run + kRescaleSlack;
  if (__ballot(need)) {
    const float m_new = need ? tmax : m_run;
    const float corr = __builtin_amdgcn_exp2f(m_run - m_new);
    l_run *= corr;
#pragma unroll
    for (int c = 0; c < D / 32; ++c)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[c][r] *= corr;
    m_run = m_new;
  }
  const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
  // Exponentials, summed in four independent chains.
  float rs4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float p = __builtin_amdgcn_exp2f(sacc[kb][r] * scale_log2 - m_use);
      sacc[kb][r] = p;
      rs4[(kb << 1) | (r >> 3)] += p;
    }
  l_run += (rs4[0] + rs4[1]) + (rs4[2] + rs4[3]);

  // O^T += V^T . P^T.  MFMA step (kb, t) covers keys 32 kb + 16 t + [0, 16);
  // k-slot e of a lane in half `half` holds key 32 kb + 16 t + 4 half +
  // (e < 4 ? e : e + 4), matching accumulator elements 8 t + e.
  const uint16_t *sv = smem_buf + G_::kTileK;
  const int grp = lane >> 4;                  // 16-lane group: half = grp / 2
  const int tr_row = (lane & 15) >> 2;        // key within the transpose read
  const int tr_dim = 16 * (grp & 1) + 4 * (lane & 3);
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      u32x4 pw;
      pw[0] = pack_bf16(sacc[kb][8 * t + 0], sacc[kb][8 * t + 1]);
      pw[1] = pack_bf16(sacc[kb][8 * t + 2], sacc[kb][8 * t + 3]);
      pw[2] = pack_bf16(sacc[kb][8 * t + 4], sacc[kb][8 * t + 5]);
      pw[3] = pack_bf16(sacc[kb][8 * t + 6], sacc[kb][8 * t + 7]);
      const bf16x8 pf = as_bf16x8(pw);
      const int key_lo = 32 * kb + 16 * t + 4 * half + tr_row;
#pragma unroll
      for (int c = 0; c < D / 32; ++c) {
        const int off = key_lo * G_::kLdsV + 32 * c + tr_dim;
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(sv + off));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(sv + off + 8 * G_::kLdsV));
        u32x4 vw;
        vw[0] = __builtin_bit_cast(u32x2, lo)[0];
        vw[1] = __builtin_bit_cast(u32x2, lo)[1];
        vw[2] = __builtin_bit_cast(u32x2, hi)[0];
        vw[3] = __builtin_bit_cast(u32x2, hi)[1];
        oacc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vw), pf, oacc[c], 0, 0, 0);
      }
    }
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(AttnArgs a) {
  using G_ = Geo<D>;
  constexpr int NCH = G_::kChunksPerThread;
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * G_::kBuf];

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
  // Rows at or past k_end are loaded from row k_end - 1 (valid memory) and
  // masked; only the last tile of the range has such rows.
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + kThreads * i;
      const int key = min(kt + c / G_::kChunksPerRow, k_end - 1);
      const int cc = c % G_::kChunksPerRow;
      kr[i] = *reinterpret_cast<const u32x4 *>(kbase + key * kv_stride + cc * 8);
      vr[i] = *reinterpret_cast<const u32x4 *>(vbase + key * kv_stride + cc * 8);
    }
  };
  auto store_tile = [&](int buf) {
    uint16_t *sk = smem + buf * G_::kBuf;
    uint16_t *sv = sk + G_::kTileK;
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int c = tid + kThreads * i;
      const int r = c / G_::kChunksPerRow;
      const int cc = c % G_::kChunksPerRow;
      *reinterpret_cast<u32x4 *>(sk + r * G_::kLdsK + cc * 8) = kr[i];
      *reinterpret_cast<u32x4 *>(sv + r * G_::kLdsV + cc * 8) = vr[i];
    }
  };

  float m_run = -INFINITY;  // reference max of scaled scores, log2 units
  float l_run = 0.f;        // this lane's share of the denominator
  f32x16 oacc[D / 32];
#pragma unroll
  for (int c = 0; c < D / 32; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[c][r] = 0.f;

  if (w.k_begin < k_end) {
    load_tile(w.k_begin);
    store_tile(0);
    __syncthreads();
    int buf = 0;
    int kt = w.k_begin;
    // Tiles before kt_mask lie wholly inside the range and at or below every
    // row's diagonal; the rest need the mask.  One loop per kind keeps a
    // single tile body live at a time.
    const int kt_full = w.k_begin + ((min(k_end, diag_all + 1) - w.k_begin) / KT) * KT;
    const int kt_mask = max(w.k_begin, kt_full);
    auto run = [&](auto mask_tag, int stop) {
      constexpr bool kMask = decltype(mask_tag)::value;
      for (; kt < stop; kt += KT) {
        const bool has_next = kt + KT < k_end;
        if (has_next) load_tile(kt + KT);
        attend_tile<D, kMask>(smem + buf * G_::kBuf, qf, oacc, m_run, l_run, lane, a.scale_log2, kt, k_end,
                              my_last);
        if (has_next) store_tile(buf ^ 1);
        __syncthreads();
        buf ^= 1;
      }
    };
    run(std::integral_constant<bool, false>(), kt_mask);
    run(std::integral_constant<bool, true>(), k_end);
  }

  // Combine the two halves' denominators and normalise.
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_val = l_tot > 0.f ? (m_run + __log2f(l_tot)) * 0.69314718055994530942f : -INFINITY;
  const int S = sd.n_splits;
  if (S == 1) {
    if (!valid) return;
    uint16_t *orow = a.out + qrow * D;
#pragma unroll
    for (int c = 0; c < D / 32; ++c)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int dim = 32 * c + 8 * g4 + 4 * half;
        u32x2 pk;
        pk[0] = pack_bf16(oacc[c][4 * g4 + 0] * inv, oacc[c][4 * g4 + 1] * inv);
        pk[1] = pack_bf16(oacc[c][4 * g4 + 2] * inv, oacc[c][4 * g4 + 3] * inv);
        *reinterpret_cast<u32x2 *>(orow + dim) = pk;
      }
    if (a.lse != nullptr && half == 0) a.lse[(int64_t)h * a.total_q + sd.cu_q + qpos] = lse_val;
    return;
  }

  // Split-key: write this split's normalised partial and its log-sum-exp.
  if (!valid) return;
  const int64_t prow = (int64_t)w.split * a.total_q * a.n_q_heads + qrow;
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

// 32 lanes per (token, head) row of a split sequence, D / 32 dims per lane:
// weights exp(lse_s - max) over the splits, weighted sum of the partials.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  constexpr int PER_LANE = D / 32;
  const int64_t row = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 5;
  const int sub = threadIdx.x & 31;
  if (row >= (int64_t)a.total_q * a.n_q_heads) return;
  const int token = (int)(row / a.n_q_heads);
  const int h = (int)(row - (int64_t)token * a.n_q_heads);
  int lo = 0, hi = a.n_seqs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.seqs[mid].cu_q <= token) lo = mid; else hi = mid - 1;
  }
  const int S = a.seqs[lo].n_splits;
  if (S <= 1) return;
  const int64_t stride = (int64_t)a.total_q * a.n_q_heads;
  float mx = -INFINITY;
  for (int s = 0; s < S; ++s) mx = fmaxf(mx, a.part_lse[s * stride + row]);
  float acc[PER_LANE];
#pragma unroll
  for (int j = 0; j < PER_LANE; ++j) acc[j] = 0.f;
  float wsum = 0.f;
  for (int s = 0; s < S; ++s) {
    const float ls = a.part_lse[s * stride + row];
    const float wgt = (ls == -INFINITY) ? 0.f : __expf(ls - mx);
    wsum += wgt;
    const float *po = a.part_o + (s * stride + row) * D + sub * PER_LANE;
    if (PER_LANE == 4) {
      const f32x4 x = *reinterpret_cast<const f32x4 *>(po);
#pragma unroll
      for (int j = 0; j < PER_LANE; ++j) acc[j] += wgt * x[j & 3];
    } else {
      const f32x2 x = *reinterpret_cast<const f32x2 *>(po);
#pragma unroll
      for (int j = 0; j < PER_LANE; ++j) acc[j] += wgt * x[j & 1];
    }
  }
  const float winv = wsum > 0.f ? 1.f / wsum : 0.f;
  uint16_t *orow = a.out + row * D + sub * PER_LANE;
  if (PER_LANE == 4) {
    u32x2 pk;
    pk[0] = pack_bf16(acc[0] * winv, acc[1 % PER_LANE] * winv);
    pk[1] = pack_bf16(acc[2 % PER_LANE] * winv, acc[3 % PER_LANE] * winv);
    *reinterpret_cast<u32x2 *>(orow) = pk;
  } else {
    *reinterpret_cast<uint32_t *>(orow) = pack_bf16(acc[0] * winv, acc[1 % PER_LANE] * winv);
  }
  if (a.lse != nullptr && sub == 0)
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
  const unsigned blocks = (unsigned)((rows * 32 + 255) / 256);
  if (head_dim == 128)
    hipLaunchKernelGGL(attn_merge_kernel<128>, dim3(blocks), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(attn_merge_kernel<64>, dim3(blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace sc
