// Causal GQA prefill attention over prefix + new tokens (§2.2: causal
// attention over every earlier position and the token itself; a new turn's tokens attend to the
// cached history plus the new tokens; GQA as used by the models of §5).
//
// Output row (query i of a sequence with P cached tokens, query head h):
//   o = sum_{j <= P + i} softmax_j(scale * q . k_j) v_j,  KV head g = h / group.
//
// Work decomposition (built on the host, see plan_attention): a workgroup
// of 8 waves owns 256 (query, head) rows = rows_q consecutive queries times
// the `group` query heads that share one KV head, and a range of keys.
// Packing the heads of a group into the rows makes every K/V tile staged
// through LDS serve all of them.  Long key ranges are split over several
// workgroups (split-key): each writes a normalised partial output (in the
// element type; it is a convex combination of V rows) and
// its log-sum-exp, and attn_merge_kernel combines them exactly
// (o = sum_s exp(lse_s - lse) o_s).  The merge is not done by the
// last-arriving split's workgroup: that would need device-scope fences,
// whose L2 write-back / invalidate stalls the other workgroups streaming
// K/V.  A single call launches the merge kernel after the forward kernel;
// in a layer stack the forward kernel of the next layer does it, each
// workgroup claiming chunks of rows once its own item is done (the launch
// boundary orders the partials' writes before those reads).
//
// q, K, V and out are bf16 or IEEE fp16 (Elem<DT> below); everything else
// is the same for both types.
//
// Per key tile of 32 and per wave (32 rows):
//   S^T (32 keys x 32 rows) = K_tile . Q^T         MFMA 32x32x16 bf16, fp32 out
//   P = exp2(c S^T - m),  c = scale * log2(e)      online softmax, log2 domain
//   O^T (D x 32 rows) += V^T . P^T                 MFMA 32x32x16 bf16
// The scale stays in fp32: folding it into a bf16 copy of q moves scores by
// about 1% of q's rounding, enough to exceed the tolerance when two keys
// compete for a row.  Every lane holds 16 keys of ONE row (the other 16 are
// in the other half of the wave).  The probabilities never leave registers:
// the S^T accumulator layout is the B-operand layout of the PV product once
// rounded to bf16, for a fixed permutation of the 16 keys of each MFMA step.
// V^T operands come from the row-major V tile through LDS transpose reads
// (ds_read_b64_tr_b16: in each 16-lane group, lanes 4r..4r+3 read 4 dims
// each of key r and lane j gets dim j of the 4 keys).  The row sum adds the
// fp32 probabilities before rounding, in two chains (two v_add_f32 per pair
// measured 1-2% faster at head_dim 128 and 2-4% at 64 than one
// v_dot2c_f32_bf16 on the packed pair); it differs from the sum of the
// rounded weights the PV product uses by the rounding of P, far below the
// tolerance.
//
// Software pipeline.  A single wave issues MFMAs at half the SIMD's matrix
// rate and VALU ops at half its vector rate, so each wave interleaves both:
// iteration j issues QK(j+1) and PV(j-1) (16 MFMAs) in the same basic block
// as the softmax of tile j, and both waves of a SIMD do so.  The MFMAs do
// not hide the vector work completely (measured: each vector instruction
// per score costs 2-3% of the loop), so the softmax is cut to its minimum:
// p = exp2(c s - m), the bf16 packing and the row sum.  The reference max m
// is the exact max of the first tile and moves only when a lane's tile sum
// exceeds kSumLimit: softmax is invariant to the reference, and fp32/bf16
// keep their relative precision at any scale, so a stale reference changes
// nothing but the exponent range, which the limit bounds.  No per-tile row
// max is computed on the common path.
//
// K and V tiles each live in a 4-entry LDS ring (slot = tile mod 4), and
// iteration j reads K(j+1) and V(j-1).  With head_dim 128 the tiles go from
// memory straight into LDS (buffer loads with the LDS flag, swizzled rows
// instead of padded ones, 64 KiB of LDS): the even iteration of each pair
// issues the loads of K(j+3), K(j+4), V(j+1) and V(j+2), and the pair ends
// with one barrier after they have landed.  With head_dim 64 the tiles are
// staged through registers: iteration j writes K(j+3) and V(j+1) loaded in
// iteration j-1 and loads K(j+4) and V(j+2).  Either way a tile is in place
// at least a barrier before it is read and only every second iteration ends
// with a workgroup barrier (one that lets global loads meant for later
// iterations stay in flight), which halves the barrier waits and lets the
// waves drift apart by up to an iteration.  The loop is unrolled so that
// the ring slots, the barrier placement and the score registers are fixed
// at compile time.
#include "sc_internal.h"

#include <cmath>
#include <mutex>
#include <type_traits>

namespace sc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// A record of 32-bit fields read through the constant address space: the
// host writes work items and sequence records before the launch and nothing
// writes them during it, so a uniform index gives scalar loads.
template <class T>
__device__ __forceinline__ T load_const(const T *p) {
  static_assert(sizeof(T) % 4 == 0, "32-bit fields");
  const __attribute__((address_space(4))) int32_t *q = (const __attribute__((address_space(4))) int32_t *)p;
  int32_t v[sizeof(T) / 4];
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) v[i] = q[i];
  T r;
  __builtin_memcpy(&r, v, sizeof(T));
  return r;
}

constexpr int kThreads = 512;            // 8 waves, 2 per SIMD
constexpr int KT = kAttnKeyTile;
static_assert(kAttnRows == 8 * 32, "eight waves of 32 rows");
static_assert(KT == 32, "one 32-key MFMA block per tile");

// 32x32 MFMA accumulator layout: element r of lane l holds C[m][n] with
// n = l % 32 and m = 8 * (r / 4) + 4 * (l / 32) + r % 4.
__device__ __forceinline__ int acc_m(int r, int half) { return 8 * (r >> 2) + 4 * half + (r & 3); }

template <int D>
struct Geo {
  static constexpr int kChunksPerRow = D / 8;                     // 16-byte chunks per key row
  static constexpr int kTileChunks = KT * kChunksPerRow;          // chunks of K (or V) per tile
  static constexpr int kChunksPerThread = 2 * kTileChunks / kThreads;  // K and V of one tile over the workgroup
  // K rows: 16-byte reads of 16 consecutive keys fall on disjoint banks.
  static constexpr int kLdsK = D + 8;
  // V rows: the 8 rows of one transpose read (64 bytes each) fall on
  // disjoint bank ranges (row stride = 16 dwords mod 64).
  static constexpr int kLdsV = D + 32;
  static constexpr int kTileK = KT * kLdsK;
  static constexpr int kTileV = KT * kLdsV;
  static constexpr int kSlots = 4;   // ring entries per operand (K and V)
  static constexpr int kSmem = kSlots * (kTileK + kTileV);
  static_assert(kChunksPerThread * kThreads == 2 * kTileChunks, "tile split");
};

// Element type of q, K, V, the probabilities of the PV product and the
// output: bf16 or IEEE fp16 (the paper's serving precision, §5).  Operands
// travel as raw 16-bit patterns; only the MFMA, the packing of fp32 values
// (round to nearest even) and the unpacking depend on the type.
template <int DT>
struct Elem;

template <>
struct Elem<SC_DTYPE_BF16> {
  // A lane's tile sum above this sends the wave through settle_max.  Every
  // probability is then below 2^20, so O and l stay far from fp32 overflow
  // for any sequence length; rows never pay for a max they do not need.
  static constexpr float kSumLimit = 1048576.0f;
  static __device__ __forceinline__ f32x16 mfma(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  }
  // Two floats to packed bf16, one v_cvt_pk_bf16_f32.
  static __device__ __forceinline__ uint32_t pack(float a, float b) {
    const bf16x2 p = {(__bf16)a, (__bf16)b};
    return __builtin_bit_cast(uint32_t, p);
  }
  // Packed pair back to floats (exact).
  static __device__ __forceinline__ f32x2 unpack(uint32_t p) {
    f32x2 r;
    r[0] = __builtin_bit_cast(float, p << 16);
    r[1] = __builtin_bit_cast(float, p & 0xFFFF0000u);
    return r;
  }
};

template <>
struct Elem<SC_DTYPE_F16> {
  // As for bf16, but fp16 probabilities must also stay below its largest
  // finite value (65504): with a tile sum of at most 2^15 every one does.
  // A probability that overflowed to inf fails the same test.
  static constexpr float kSumLimit = 32768.0f;
  static __device__ __forceinline__ f32x16 mfma(u32x4 a, u32x4 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
  }
  static __device__ __forceinline__ uint32_t pack(float a, float b) {
    const f16x2 p = {(_Float16)a, (_Float16)b};
    return __builtin_bit_cast(uint32_t, p);
  }
  static __device__ __forceinline__ f32x2 unpack(uint32_t p) {
    const f16x2 h = __builtin_bit_cast(f16x2, p);
    f32x2 r;
    r[0] = (float)h[0];
    r[1] = (float)h[1];
    return r;
  }
};

// Max with the same lane of the other 32-lane half of the wave.
__device__ __forceinline__ float max_with_other_half(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x),
                                                  __builtin_bit_cast(uint32_t, x), false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}

// Workgroup barrier that orders LDS only: this wave's LDS accesses complete
// before it, global loads stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// head_dim 128: K/V ring slots loaded straight into LDS (see attn_item).
// One array per slot and operand, so the compiler can tell that a load in
// flight into one slot does not alias reads of another and needs no wait.
struct DmaGeo {
  static constexpr int kRowBytes = 128 * 2;               // one key row of one KV head
  static constexpr int kSlotBytes = KT * kRowBytes;        // one tile, 8 KiB
};
// Pairs of iterations a tile load has to land in, and the ring size that
// allows (tiles read in the A pairs after a load plus the two it loads).
// One pair is enough: with two or three (96 or 128 KiB of LDS) the kernel
// measured 1.5-3% slower on the 8B, 14B and long-prefix shapes.
constexpr int kDmaAhead = 1;
constexpr int kDmaRing = 2 * kDmaAhead + 2;
static_assert(kDmaAhead >= 1 && kDmaRing <= 8, "ring of at most 8 slots");
#define SC_DMA_SLOT(n)                                                          \
  __shared__ __attribute__((aligned(1024))) unsigned char dma_k##n[DmaGeo::kSlotBytes]; \
  __shared__ __attribute__((aligned(1024))) unsigned char dma_v##n[DmaGeo::kSlotBytes];
SC_DMA_SLOT(0)
SC_DMA_SLOT(1)
SC_DMA_SLOT(2)
SC_DMA_SLOT(3)
SC_DMA_SLOT(4)
SC_DMA_SLOT(5)
SC_DMA_SLOT(6)
SC_DMA_SLOT(7)
#undef SC_DMA_SLOT
template <int S>
__device__ __forceinline__ unsigned char *dma_k_slot() {
  static_assert(S >= 0 && S < kDmaRing, "ring slot");
  return S == 0 ? dma_k0 : S == 1 ? dma_k1 : S == 2 ? dma_k2 : S == 3 ? dma_k3
       : S == 4 ? dma_k4 : S == 5 ? dma_k5 : S == 6 ? dma_k6 : dma_k7;
}
template <int S>
__device__ __forceinline__ unsigned char *dma_v_slot() {
  static_assert(S >= 0 && S < kDmaRing, "ring slot");
  return S == 0 ? dma_v0 : S == 1 ? dma_v1 : S == 2 ? dma_v2 : S == 3 ? dma_v3
       : S == 4 ? dma_v4 : S == 5 ? dma_v5 : S == 6 ? dma_v6 : dma_v7;
}

// f(integral_constant<int, i>) for i = B .. E-1, unrolled.
template <int B, int E, class Fn>
__device__ __forceinline__ void static_for(Fn &&f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>());
    static_for<B + 1, E>(f);
  }
}

typedef __attribute__((address_space(3))) void lds_void;

// Wait until at most VM vector-memory operations of this wave (loads into
// LDS included) are in flight and its LDS and scalar loads are done, then a
// workgroup barrier.  No memory-model fence: the fence of __syncthreads
// would wait for every load into LDS, including those meant to stay in
// flight.
template <int VM>
__device__ __forceinline__ void dma_barrier() {
  static_assert(VM >= 0 && VM < 64, "vmcnt field");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4) | (0 << 8));
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Wait for every vector-memory operation of this wave.
__device__ __forceinline__ void dma_wait_all() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0 | (7 << 4) | (15 << 8));
  asm volatile("" ::: "memory");
}

// S^T(tile) = K_tile . Q^T: D / 16 dependent MFMAs.
template <int D, int DT>
__device__ __forceinline__ void qk_tile(const uint16_t *sk, const u32x4 (&qf)[D / 16], f32x16 &s, int lane) {
  using G_ = Geo<D>;
#pragma unroll
  for (int r = 0; r < 16; ++r) s[r] = 0.f;
  const uint16_t *krow = sk + (lane & 31) * G_::kLdsK + 8 * (lane >> 5);
#pragma unroll
  for (int k = 0; k < D / 16; ++k)
    s = Elem<DT>::mfma(*reinterpret_cast<const u32x4 *>(krow + 16 * k), qf[k], s);
}

// O^T += V^T . P^T.  MFMA step t covers keys 16 t + [0, 16); k-slot e of a
// lane in half `half` holds key 16 t + 4 half + (e < 4 ? e : e + 4), which
// is accumulator element 8 t + e of S^T, i.e. pf[t] element e.
template <int D, int DT>
__device__ __forceinline__ void pv_tile(const uint16_t *sv, const u32x4 (&pf)[2], f32x16 (&oacc)[D / 32],
                                        int lane) {
  using G_ = Geo<D>;
  constexpr int NC = D / 32;
  const int tr_row = 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int tr_dim = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const uint16_t *vb = sv + tr_row * G_::kLdsV + tr_dim;
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const uint16_t *p = vb + 16 * t * G_::kLdsV + 32 * c;
      const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)p);
      const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(p + 8 * G_::kLdsV));
      u32x4 vw;
      vw[0] = __builtin_bit_cast(u32x2, lo)[0];
      vw[1] = __builtin_bit_cast(u32x2, lo)[1];
      vw[2] = __builtin_bit_cast(u32x2, hi)[0];
      vw[3] = __builtin_bit_cast(u32x2, hi)[1];
      oacc[c] = Elem<DT>::mfma(vw, pf[t], oacc[c]);
    }
}

// Masks keys past a row's last visible key: element r holds key offset
// acc_m(r, half) within the tile, and lim is the row's last visible offset
// minus 4 half.
__device__ __forceinline__ void apply_mask(f32x16 &s, int lim) {
#pragma unroll
  for (int r = 0; r < 16; ++r)
    if (acc_m(r, 0) > lim) s[r] = -INFINITY;
}

// Row max of sl2 * s over the tile's 32 keys (both wave halves); -inf when
// every key of the row is masked.
__device__ __forceinline__ float tile_max(const f32x16 &s, float sl2) {
  float m4[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) m4[i] = fmaxf(fmaxf(s[4 * i], s[4 * i + 1]), fmaxf(s[4 * i + 2], s[4 * i + 3]));
  return max_with_other_half(fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3]))) * sl2;
}

// p = exp2(sl2 * s - m) for this lane's 16 keys, packed to the element type,
// and their fp32 sum (two chains).
template <int DT>
__device__ __forceinline__ float softmax_tile(const f32x16 &s, u32x4 (&pf)[2], float sl2, float m) {
  float r2[2] = {0.f, 0.f};
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const float x0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[8 * t + e], sl2, -m));
      const float x1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[8 * t + e + 1], sl2, -m));
      pf[t][e >> 1] = Elem<DT>::pack(x0, x1);
      r2[0] += x0;
      r2[1] += x1;
    }
  return r2[0] + r2[1];
}

template <int D>
struct WaveState {
  u32x4 qf[D / 16];   // raw 16-bit patterns
  f32x16 oacc[D / 32];
  f32x16 s[2];        // raw scores of the even / odd tiles
  u32x4 pf_prev[2];   // P(j-1) for the PV product (head_dim 64 loop)
  u32x4 pfb[2][2];    // P of the even / odd tiles (head_dim 128 loop: no copy per tile)
  float m_run;        // reference max of sl2 * s, log2 units (0 until a key is visible)
  float l_run;        // this lane's share of the denominator
};

// Rare path, taken by a whole wave when some lane's tile sum left the safe
// range: move every row's reference max to the true running max, rescale l
// and O (O already holds PV(j-1), computed against the old reference), and
// redo the tile's exponentials.  Returns the new tile sum.
template <int D, int DT>
__device__ __forceinline__ float settle_max(WaveState<D> &w, const f32x16 &s, u32x4 (&pf)[2], float sl2) {
  const float m_new = fmaxf(w.m_run, tile_max(s, sl2));
  const float corr = __builtin_amdgcn_exp2f(w.m_run - m_new);
  w.m_run = m_new;
  w.l_run *= corr;
#pragma unroll
  for (int c = 0; c < D / 32; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) w.oacc[c][r] *= corr;
  return softmax_tile<DT>(s, pf, sl2, m_new);
}

// Writes this lane's row of O (times inv, rounded to the element type) to
// `dst`.  A lane holds 4 consecutive dims of each 8-dim block, the other 4
// are in the same lane of the other half of the wave; one lane swap per
// dword gives half 0 the even and half 1 the odd 8-dim blocks of each 16,
// so every lane writes whole 16-byte chunks (the two halves of a row fill
// 32 contiguous bytes per store).  v_permlane32_swap exchanges lanes 32-63
// of its first operand with lanes 0-31 of its second.
template <int D, int DT>
__device__ __forceinline__ void store_row(const WaveState<D> &w, float inv, int half, uint16_t *dst) {
#pragma unroll
  for (int c = 0; c < D / 32; ++c)
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      // A: dims 32c + 16m + 4 half + [0, 4); B: the same + 8.
      uint32_t A[2], B[2];
      A[0] = Elem<DT>::pack(w.oacc[c][8 * m + 0] * inv, w.oacc[c][8 * m + 1] * inv);
      A[1] = Elem<DT>::pack(w.oacc[c][8 * m + 2] * inv, w.oacc[c][8 * m + 3] * inv);
      B[0] = Elem<DT>::pack(w.oacc[c][8 * m + 4] * inv, w.oacc[c][8 * m + 5] * inv);
      B[1] = Elem<DT>::pack(w.oacc[c][8 * m + 6] * inv, w.oacc[c][8 * m + 7] * inv);
      u32x4 st;
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        // Half 0 receives the other half's A, half 1 the other half's B.
        const auto r = __builtin_amdgcn_permlane32_swap(A[e], B[e], false, false);
        st[e] = (uint32_t)r[0];
        st[2 + e] = (uint32_t)r[1];
      }
      *reinterpret_cast<u32x4 *>(dst + 32 * c + 16 * m + 8 * half) = st;
    }
}

// One work item.  kPaged: its keys are read in place from the regular
// cache; the two kinds of item are separate copies of the whole body so that
// each is register-allocated on its own.
template <int D, int DT, bool kPaged>
__device__ __forceinline__ void attn_item(const AttnArgs &a, const WorkItem &wi, uint16_t *smem) {
  using G_ = Geo<D>;
  constexpr int NCH = G_::kChunksPerThread;
  // Scalar loads (see load_const), so the key-range and address arithmetic
  // built from the record stays in scalar registers.
  const SeqDesc sd = a.seqs != nullptr ? load_const(a.seqs + wi.seq) : a.seq0;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5;
  const int col = lane & 31;
  const int group = a.group;
  const int row = wave * 32 + col;
  const int qi = row / group;
  const int hg = row - qi * group;
  const bool valid = qi < wi.nq;
  const int qpos = wi.q0 + (valid ? qi : wi.nq - 1);
  const int h = wi.kvh * group + hg;
  // qrow: the row in the plan's packed numbering (split partials, lse);
  // io_row: the row of q and out (they differ for a chunk of a new turn).
  const int64_t qrow = (int64_t)(sd.cu_q + qpos) * a.n_q_heads + h;
  const int64_t io_row = (int64_t)(sd.q_off + qpos) * a.n_q_heads + h;

  WaveState<D> w;
  // Q^T fragments (B operand): lane holds Q[row][16 k + 8 half .. + 7].
  {
    const u32x4 *qp = reinterpret_cast<const u32x4 *>(a.q + io_row * D);
#pragma unroll
    for (int k = 0; k < D / 16; ++k) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (valid) x = qp[2 * k + half];
      w.qf[k] = x;
    }
  }
  const float sl2 = a.scale_log2;   // scale * log2(e)
#pragma unroll
  for (int c = 0; c < D / 32; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) w.oacc[c][r] = 0.f;
  w.m_run = 0.f;
  w.l_run = 0.f;

  // This item's keys [k_begin, k_end) of KV head kvh: rows of kv_stride
  // elements, D of them used.  Tile t is read through a buffer resource that
  // starts at its first row and ends after the item's last row, so rows past
  // the range (the ragged last tile, tiles past the end) read as zero
  // without touching memory outside it; those keys are masked.
  const int64_t kv_stride = (int64_t)a.n_kv_heads * D;
  const int k_begin = wi.k_begin;
  const int k_end = wi.k_end;
  const int n = (k_end - k_begin + KT - 1) / KT;
  const int64_t first_row = ((int64_t)sd.cu_k + k_begin) * kv_stride + (int64_t)wi.kvh * D;
  const uint16_t *const kb = a.k + first_row;
  const uint16_t *const vb = a.v + first_row;
  // Byte counts, also of the tiles loaded past the end, fit in 31 bits
  // (checked on the host).
  const uint32_t range_bytes = (uint32_t)((((int64_t)(k_end - k_begin) - 1) * kv_stride + D) * 2);
  const uint32_t tile_bytes = (uint32_t)(KT * kv_stride * 2);
  // Signed 32-bit offset arithmetic stays on the scalar unit (an unsigned
  // saturating subtract would be a vector instruction plus a readfirstlane).
  auto rsrc = [&](const uint16_t *base, int t) {
    const int off = t * (int)tile_bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(reinterpret_cast<const char *>(base) + off),
                                             (short)0, max((int)range_bytes - off, 0), 0x00020000);
  };

  // First tile that needs the mask, the same for the whole workgroup: it
  // reaches past the key range or past the diagonal of the first query.
  const int diag0 = sd.prefix + wi.q0;
  const int j_mask = max(0, min(n, (min(k_end, diag0 + 1) - k_begin) / KT));
  const int my_last = min(k_end - 1, sd.prefix + qpos);
  auto lim_of = [&](int j) { return my_last - (k_begin + j * KT) - 4 * half; };

  // Device-side dependency on the copy stream (see AttnArgs::ready_flag).
  // The poll is a relaxed device-scope load (no cache invalidation per
  // workgroup: an acquire here would invalidate the XCD's L2 under the
  // other workgroups' K/V).  No stale K/V lines can be cached: this kernel's
  // dispatch invalidated the caches after the last reader of the slot (two
  // layers back, same stream) had finished, the only kernel that touches the
  // slot after that is the copy kernel, whose completion wrote its data back
  // before the flag was written, and nothing reads the slot until the flag
  // is set.  A stack that also writes the slot from another kernel after
  // this dispatch (debug poisoning) asks for the acquire (ready_acquire).
  bool timed_out = false;
  if (a.ready_flag != nullptr) {
    __shared__ int s_timeout;
    if (tid == 0) {
      int spins = 0, late = 0;
      while (__hip_atomic_load(a.ready_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < a.ready_value) {
        if (++spins > a.ready_spin_limit) {
          late = 1;
          __hip_atomic_store(a.ready_timeout, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
        __builtin_amdgcn_s_sleep(8);
      }
      if (a.ready_acquire && !late) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
      s_timeout = late;
    }
    __syncthreads();
    timed_out = s_timeout != 0;
  }

  if constexpr (D == 128) {
    // K and V tiles go from memory straight into LDS (buffer loads with the
    // LDS flag; no staging registers).  Wave w loads rows 4 w .. 4 w + 3 of
    // every K and V tile: one 16-byte load per lane and operand, lane i
    // filling bytes 16 i .. 16 i + 15 of the wave's four rows.  Rows are
    // unpadded (256 bytes); chunk c of K row r sits at position c ^ (r mod 16)
    // and of V row r at c ^ 4 (r mod 4), which keeps the K fragment reads and
    // the V transpose reads free of bank conflicts.  Each lane loads the
    // chunk that belongs at its position.
    const int row_bytes = (int)(kv_stride * 2);
    const int l4 = lane >> 4;
    const int p16 = lane & 15;
    const int my_row = 4 * wave;
    const int voff_k = l4 * row_bytes + ((p16 ^ (4 * (wave & 3) + l4)) << 4);
    const int voff_v = l4 * row_bytes + ((p16 ^ (l4 << 2)) << 4);
    // This lane's LDS read offsets within a slot: K fragment k (row col,
    // chunk 2 k + half) and the transpose read of dim block c (key row
    // tr_row; the other key rows of the product are immediates).
    int k_rd[D / 16], v_rd[D / 32];
#pragma unroll
    for (int k = 0; k < D / 16; ++k) k_rd[k] = col * DmaGeo::kRowBytes + (((2 * k + half) ^ (col & 15)) << 4);
    {
      const int tr_row = 4 * half + ((lane & 15) >> 2);
      const int lo = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);
      const int x = (lane >> 2) & 3;
#pragma unroll
      for (int c = 0; c < D / 32; ++c) v_rd[c] = tr_row * DmaGeo::kRowBytes + ((4 * (c ^ x) + lo) << 4) + 8 * (lane & 1);
    }
    // Regular-cache item: key k of the sequence is row k mod B of local
    // block rc_ids[rc_off + k / B], read in place.  A wave's four rows start
    // on a multiple of 4 and B >= 16 is a power of two, so they share one
    // block; its index is a scalar load (the table is read through the
    // constant address space: the host writes it before the launch), made a
    // pair of iterations before the tile's data load.
    const __attribute__((address_space(4))) int32_t *rc_ids_c =
        kPaged ? (const __attribute__((address_space(4))) int32_t *)(a.rc_ids + sd.rc_off) : nullptr;
    // This KV head's K and V rows in block 0 of the layer; block b is
    // b * rc_block_bytes further (under 4 GiB, checked on the host), so the
    // per-tile address is a 32 x 32 -> 64-bit product and two adds.
    const char *rc_kbase =
        kPaged ? reinterpret_cast<const char *>(a.rc_base + a.rc_layer_elems + (int64_t)wi.kvh * D) : nullptr;
    const char *rc_vbase = kPaged ? rc_kbase + a.rc_half_elems * 2 : nullptr;
    const uint32_t rc_block_bytes = kPaged ? (uint32_t)(a.rc_block_elems * 2) : 0u;
    const int rc_mask = (1 << a.block_shift) - 1;
    auto blk_of = [&](int t) -> int {
      if constexpr (!kPaged) {
        return 0;
      } else {
        return rc_ids_c[min(k_begin + t * KT + my_row, k_end - 1) >> a.block_shift];
      }
    };
    // This wave's four rows of tile t, K (kV false) or V, into `slot`.  The
    // buffer resource ends after the last row of the item's range (of the
    // block, for a regular-cache item), so rows past it, and whole tiles
    // past the last one, load zeros without touching memory.
    auto dma = [&](unsigned char *slot, int t, auto v_tag, int blk) {
      constexpr bool kV = decltype(v_tag)::value;
      const int key = k_begin + t * KT + my_row;
      const char *base;
      int range;
      if constexpr (kPaged) {
        const int rib = min(key, k_end - 1) & rc_mask;   // first row within the block
        const int rows = min(rc_mask + 1 - rib, k_end - key);
        base = (kV ? rc_vbase : rc_kbase) + (uint64_t)(uint32_t)blk * rc_block_bytes + (uint32_t)(rib * row_bytes);
        range = rows > 0 ? ((rows - 1) * row_bytes + 2 * D) : 0;
      } else {
        // Signed 32-bit offsets (the host keeps a sequence's keys, plus the
        // tiles loaded past its end, under 2^31 bytes): a subtract and a max
        // on the scalar unit.  A 64-bit compare would be a vector
        // instruction whose result the scalar select then waits for (~2%
        // of the loop), as would a saturating unsigned subtract.
        const int off = t * (int)tile_bytes + my_row * row_bytes;
        base = reinterpret_cast<const char *>(kV ? vb : kb) + off;
        range = max((int)range_bytes - off, 0);
      }
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<char *>(base), (short)0, __builtin_amdgcn_readfirstlane(range), 0x00020000);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)(slot + my_row * DmaGeo::kRowBytes), 16,
                                               kV ? voff_v : voff_k, 0, 0, 0);
    };
    auto qk = [&](const unsigned char *slot, f32x16 &s) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
      for (int k = 0; k < D / 16; ++k)
        s = Elem<DT>::mfma(*reinterpret_cast<const u32x4 *>(slot + k_rd[k]), w.qf[k], s);
    };
    // O^T += V^T . P^T, operands as in pv_tile.
    auto pv = [&](const unsigned char *slot, const u32x4 (&pfp)[2]) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int c = 0; c < D / 32; ++c) {
          const unsigned char *p = slot + v_rd[c] + 16 * t * DmaGeo::kRowBytes;
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)p);
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(p + 8 * DmaGeo::kRowBytes));
          u32x4 vw;
          vw[0] = __builtin_bit_cast(u32x2, lo)[0];
          vw[1] = __builtin_bit_cast(u32x2, lo)[1];
          vw[2] = __builtin_bit_cast(u32x2, hi)[0];
          vw[3] = __builtin_bit_cast(u32x2, hi)[1];
          w.oacc[c] = Elem<DT>::mfma(vw, pfp[t], w.oacc[c]);
        }
    };

    if (n > 0 && !timed_out) {
      using T = std::true_type;
      using F = std::false_type;
      constexpr int A = kDmaAhead;
      constexpr int R = kDmaRing;
      // Regular-cache block indices of the tiles the current pair loads into
      // K (bk0, bk1) and V (bv0, bv1), and of the next pair's K tiles.  The
      // V tiles of a pair are the K tiles of the pair before.
      int bv0 = blk_of(2 * A - 1), bv1 = blk_of(2 * A), bk0 = blk_of(2 * A + 1), bk1 = blk_of(2 * A + 2);
      int bn0 = 0, bn1 = 0;
      // Prologue: K(0 .. 2A) and V(0 .. 2A-2), the operands of the first A
      // pairs; then QK(0).  The first pair loads into the slot QK(0) reads:
      // a second barrier.
      static_for<0, 2 * A + 1>([&](auto t) { dma(dma_k_slot<decltype(t)::value % R>(), t, F(), blk_of(t)); });
      static_for<0, 2 * A - 1>([&](auto t) { dma(dma_v_slot<decltype(t)::value % R>(), t, T(), blk_of(t)); });
      dma_barrier<0>();
      qk(dma_k_slot<0>(), w.s[0]);
      dma_barrier<0>();

      // Iteration j (J = j mod R is the ring slot of tile j; tile j's scores
      // live in s[j mod 2]).  Pair p = iterations 2p, 2p+1 reads K(2p+1),
      // K(2p+2), V(2p-1), V(2p).  Its even iteration loads the operands of
      // pair p+A: K(j+1+2A), K(j+2+2A), V(j-1+2A), V(j+2A), into the slots
      // last read in pair p-1; its odd iteration ends with a barrier once
      // the loads issued A-1 pairs earlier have landed, so a load has A
      // pairs of iterations to land and only every second iteration waits
      // at a barrier.  Loads of tiles past the last one load zeros.  QK(j+1)
      // runs in every iteration, also the last, whose product of a stale
      // slot is never used: one body throughout keeps the MFMA accumulators
      // in place.
      auto iterate = [&](auto j_tag, auto mask_tag, auto first_tag, int j) {
        constexpr int J = decltype(j_tag)::value;
        constexpr bool kMask = decltype(mask_tag)::value;
        constexpr bool kFirst = decltype(first_tag)::value;
        constexpr int PAR = J & 1;
        f32x16 &sc = w.s[PAR];
        f32x16 &sn = w.s[PAR ^ 1];
        if constexpr (kMask) apply_mask(sc, lim_of(j));
        if constexpr (kFirst) {
          const float tm = tile_max(sc, sl2);
          w.m_run = tm > -INFINITY ? tm : 0.f;
        }
        const float mneg = -w.m_run;
        const unsigned char *ks = dma_k_slot<(J + 1) % R>();
        const unsigned char *vs = dma_v_slot<(J + R - 1) % R>();
        // The 16 MFMAs of the iteration alternate between QK(j+1) (even
        // steps, K fragment i / 2) and PV(j-1) (odd steps, V^T block
        // c = (i / 2) mod 4 of key half t = i / 8), and each step also
        // computes one probability of tile j: one MFMA and a sixteenth of
        // the softmax per step, in this order (scheduling barriers keep the
        // compiler from regrouping them).  Operands are read from LDS three
        // steps ahead (two measured ~0.5% slower, four no better).
        auto operand = [&](int i) -> u32x4 {
          if ((i & 1) == 0) return *reinterpret_cast<const u32x4 *>(ks + k_rd[i >> 1]);
          const unsigned char *p = vs + v_rd[(i >> 1) & 3] + 16 * (i >> 3) * DmaGeo::kRowBytes;
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)p);
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(p + 8 * DmaGeo::kRowBytes));
          u32x4 vw;
          vw[0] = __builtin_bit_cast(u32x2, lo)[0];
          vw[1] = __builtin_bit_cast(u32x2, lo)[1];
          vw[2] = __builtin_bit_cast(u32x2, hi)[0];
          vw[3] = __builtin_bit_cast(u32x2, hi)[1];
          return vw;
        };
        u32x4 op[16];
        // Probabilities of tile j go to pfb[j mod 2]; PV(j-1) reads the other.
        u32x4 (&pf)[2] = w.pfb[PAR];
        const u32x4 (&pfp)[2] = w.pfb[PAR ^ 1];
        float rsum0 = 0.f, rsum1 = 0.f;   // row sum: even and odd keys of the tile
        float x_prev = 0.f;
        constexpr int kAhead = 3;         // LDS operand reads, steps ahead of their MFMA
#pragma unroll
        for (int i = 0; i < kAhead; ++i) {
          if (!kFirst || (i & 1) == 0) op[i] = operand(i);
          else op[i] = u32x4{0u, 0u, 0u, 0u};
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          if (i + kAhead < 16) {
            if (!kFirst || ((i + kAhead) & 1) == 0) op[i + kAhead] = operand(i + kAhead);
          }
          if ((i & 1) == 0) {
            sn = Elem<DT>::mfma(op[i], w.qf[i >> 1], i == 0 ? f32x16{} : sn);
          } else if constexpr (!kFirst) {
            w.oacc[(i >> 1) & 3] = Elem<DT>::mfma(op[i], pfp[i >> 3], w.oacc[(i >> 1) & 3]);
          }
          const float x = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[i], sl2, mneg));
          if (i & 1) {
            const uint32_t pk = Elem<DT>::pack(x_prev, x);
            pf[i >> 3][(i & 7) >> 1] = pk;
            rsum0 += x_prev;
            rsum1 += x;
          }
          x_prev = x;
          if constexpr (PAR == 0) {
            if (i == 1) dma(dma_k_slot<(J + 1 + 2 * A) % R>(), j + 1 + 2 * A, F(), bk0);
            if (i == 3) dma(dma_k_slot<(J + 2 + 2 * A) % R>(), j + 2 + 2 * A, F(), bk1);
            if (i == 5) dma(dma_v_slot<(J - 1 + 2 * A) % R>(), j - 1 + 2 * A, T(), bv0);
            if (i == 7) dma(dma_v_slot<(J + 2 * A) % R>(), j + 2 * A, T(), bv1);
            if (i == 9) bn0 = blk_of(j + 3 + 2 * A);
            if (i == 11) bn1 = blk_of(j + 4 + 2 * A);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
        float rs = rsum0 + rsum1;
        if (!kFirst && __builtin_amdgcn_ballot_w64(!(rs <= Elem<DT>::kSumLimit))) rs = settle_max<D, DT>(w, sc, pf, sl2);
        w.l_run += rs;
        if constexpr (PAR == 1) {
          dma_barrier<4 * (A - 1)>();
          bv0 = bk0;
          bv1 = bk1;
          bk0 = bn0;
          bk1 = bn1;
        }
      };
      // j = 0 .. R-1 masked (exact for any tile; j = 0 sets the reference
      // max), then whole rounds of R unmasked tiles, then the rest masked.
      iterate(std::integral_constant<int, 0>(), T(), T(), 0);
      static_for<1, R>([&](auto J) {
        if (decltype(J)::value < n) iterate(J, T(), F(), decltype(J)::value);
      });
      int j = R;
      const int jm = min(j_mask, n);
      for (; j + R - 1 < jm; j += R) static_for<0, R>([&](auto J) { iterate(J, F(), F(), j + decltype(J)::value); });
      for (; j < n; j += R)
        static_for<0, R>([&](auto J) {
          if (j + decltype(J)::value < n) iterate(J, T(), F(), j + decltype(J)::value);
        });
      // PV of the last tile; its V landed before the last pair's barrier.
      const int last = (n - 1) % R;
      static_for<0, R>([&](auto S) {
        constexpr int kS = decltype(S)::value;
        if (last == kS) pv(dma_v_slot<kS>(), w.pfb[kS & 1]);   // R is even: kS has the parity of n-1
      });
      // Loads of tiles past the end may still be in flight.
      dma_wait_all();
    }
  } else {
    // Staging: chunk c = tid + 512 i of a (K tile, V tile) pair; whether it is
    // a K or a V chunk is uniform over a wave.
    int voff[NCH], lds_off[NCH], crow[NCH], ccol[NCH];
    bool is_v[NCH];
  #pragma unroll
    for (int i = 0; i < NCH; ++i) {
      is_v[i] = wave * 64 + kThreads * i >= G_::kTileChunks;
      const int c = tid + kThreads * i - (is_v[i] ? G_::kTileChunks : 0);
      const int r = c / G_::kChunksPerRow, cc = c % G_::kChunksPerRow;
      voff[i] = (int)((r * kv_stride + cc * 8) * 2);
      lds_off[i] = is_v[i] ? G_::kSlots * G_::kTileK + r * G_::kLdsV + cc * 8 : r * G_::kLdsK + cc * 8;
      crow[i] = r;
      ccol[i] = wi.kvh * D + cc * 8;
    }
    // Regular-cache item: key k of the sequence is row k mod B of local block
    // rc_ids[rc_off + k / B], read in place.  A wave's chunk i covers 4 (D=128)
    // or 8 (D=64) consecutive rows of a tile that start on a multiple of that
    // count, and B >= 16 is a power of two, so those rows share one block: its
    // index is wave-uniform and the load goes through a buffer resource over
    // that block's layer slice.  The index of tile t + 1 is read while tile t
    // is loaded (tiles of one chunk are loaded in order, one per call), so the
    // data loads never wait on it.  Rows past the range read the clamped last
    // block; they are masked.
    const int32_t *rc_ids = kPaged ? a.rc_ids + sd.rc_off : nullptr;
    const uint16_t *rc_layer = kPaged ? a.rc_base + a.rc_layer_elems : nullptr;
    const int rc_mask = (1 << a.block_shift) - 1;
    const uint32_t rc_slice_bytes = (uint32_t)(a.rc_half_elems * 4);
    int rc_next[NCH];
  #pragma unroll
    for (int i = 0; i < NCH; ++i) rc_next[i] = 0;
    // The index table is read through the constant address space: the host
    // writes it before the launch and nothing writes it during the kernel, so
    // the uniform index loads are scalar loads.
    const __attribute__((address_space(4))) int32_t *rc_ids_c =
        (const __attribute__((address_space(4))) int32_t *)rc_ids;
    auto rc_block = [&](int t, int i) {
      const int row0 = __builtin_amdgcn_readfirstlane(crow[i]);
      return rc_ids_c[min(k_begin + t * KT + row0, k_end - 1) >> a.block_shift];
    };
    // A negative tile index (prologue only) skips that half of the pair.
    u32x4 lr[NCH];
    auto stage_load = [&](u32x4 (&lr)[NCH], int kj, int vj) {
  #pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int t = is_v[i] ? vj : kj;
        if (t < 0) continue;
        if (kPaged) {
          const int blk = __builtin_amdgcn_readfirstlane(t == 0 ? rc_block(0, i) : rc_next[i]);
          rc_next[i] = rc_block(t + 1, i);
          const uint16_t *base = rc_layer + (int64_t)blk * a.rc_block_elems;
          const int row = (k_begin + t * KT + crow[i]) & rc_mask;
          const int off = (int)((row * kv_stride + ccol[i] + (is_v[i] ? a.rc_half_elems : 0)) * 2);
          lr[i] = __builtin_bit_cast(
              u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                         __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(base), (short)0,
                                                           (int)rc_slice_bytes, 0x00020000),
                         off, 0, 0));
        } else {
          lr[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc(is_v[i] ? vb : kb, t),
                                                                                   voff[i], 0, 0));
        }
      }
    };
    // kt / vt: the tiles the K and V chunks hold (ring slot = tile mod 4); a
    // negative tile skips that half.
    auto stage_store = [&](const u32x4 (&lr)[NCH], int kt, int vt) {
  #pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int t = is_v[i] ? vt : kt;
        if (t >= 0) {
          const int slot_off = is_v[i] ? (t & 3) * G_::kTileV : (t & 3) * G_::kTileK;
          *reinterpret_cast<u32x4 *>(smem + lds_off[i] + slot_off) = lr[i];
        }
      }
    };
    auto slot_k = [&](int t) { return smem + (t & 3) * G_::kTileK; };
    auto slot_v = [&](int t) { return smem + G_::kSlots * G_::kTileK + (t & 3) * G_::kTileV; };

    if (n > 0 && !timed_out) {
      // Prologue: K(0), K(1), K(2) and V(0) into the rings (their loads in
      // flight together), K(3) and V(1) loaded for iteration 0, then QK(0).
      {
        u32x4 lb[NCH], lc[NCH];
        stage_load(lr, 0, 0);
        stage_load(lb, 1, -1);
        stage_load(lc, 2, -1);
        stage_store(lr, 0, 0);
        stage_store(lb, 1, -1);
        stage_store(lc, 2, -1);
        stage_load(lr, 3, 1);
      }
      lds_barrier();
      qk_tile<D, DT>(slot_k(0), w.qf, w.s[0], lane);

      // Iteration j (tile parity PAR): QK(j+1) and PV(j-1) on the MFMA pipe,
      // softmax(j) on the VALU, then K(j+3), V(j+1) into the rings and K(j+4),
      // V(j+2) from memory.  Tile j's scores live in s[PAR].  The rings hold
      // four tiles, so a workgroup barrier is needed only after even
      // iterations: the two iterations between barriers read K(j+1), V(j-1)
      // written at least one barrier earlier and write the two slots read
      // last before that barrier.
      auto iterate = [&](auto par_tag, auto mask_tag, auto qk_tag, auto pv_tag, auto first_tag, int j) {
        constexpr int PAR = decltype(par_tag)::value;
        constexpr bool kMask = decltype(mask_tag)::value;
        constexpr bool kQk = decltype(qk_tag)::value;
        constexpr bool kPv = decltype(pv_tag)::value;
        constexpr bool kFirst = decltype(first_tag)::value;
        __builtin_assume(j >= 0);
        f32x16 &sc = w.s[PAR];
        u32x4 pf[2];
        if (kQk) qk_tile<D, DT>(slot_k(j + 1), w.qf, w.s[PAR ^ 1], lane);
        if (kPv) pv_tile<D, DT>(slot_v(j - 1), w.pf_prev, w.oacc, lane);
        if (kMask) apply_mask(sc, lim_of(j));
        if (kFirst) {
          const float tm = tile_max(sc, sl2);
          w.m_run = tm > -INFINITY ? tm : 0.f;
        }
        float rs = softmax_tile<DT>(sc, pf, sl2, w.m_run);
        if (!kFirst && __builtin_amdgcn_ballot_w64(!(rs <= Elem<DT>::kSumLimit))) rs = settle_max<D, DT>(w, sc, pf, sl2);
        w.l_run += rs;
        stage_store(lr, j + 3, j + 1);
        stage_load(lr, j + 4, j + 2);
        if (PAR == 0) lds_barrier();
        w.pf_prev[0] = pf[0];
        w.pf_prev[1] = pf[1];
      };
      using T = std::true_type;
      using F = std::false_type;
      using P0 = std::integral_constant<int, 0>;
      using P1 = std::integral_constant<int, 1>;
      // j = 0: masked variant (exact for any tile), exact max.
      if (n > 1) iterate(P0(), T(), T(), F(), T(), 0); else iterate(P0(), T(), F(), F(), T(), 0);
      // Steady state j = 1 .. n - 2, unrolled by two so that tile parity is
      // known at compile time: unmasked tiles, then masked ones.
      int j = 1;
      auto steady = [&](auto mask_tag, int j_end) {
        if (j < j_end && (j & 1) == 0) iterate(P0(), mask_tag, T(), T(), F(), j++);
        for (; j + 1 < j_end; j += 2) {
          iterate(P1(), mask_tag, T(), T(), F(), j);
          iterate(P0(), mask_tag, T(), T(), F(), j + 1);
        }
        if (j < j_end) iterate(P1(), mask_tag, T(), T(), F(), j++);
      };
      steady(F(), min(j_mask, n - 1));
      steady(T(), n - 1);
      // j = n - 1: PV(n-2) and softmax(n-1), then drain PV(n-1) (V(n-1) was
      // written in iteration n-2; whichever of n-2, n-1 is even ended with a
      // barrier).
      if (n >= 2) {
        if ((n - 1) & 1) iterate(P1(), T(), F(), T(), F(), n - 1); else iterate(P0(), T(), F(), T(), F(), n - 1);
      }
      pv_tile<D, DT>(slot_v(n - 1), w.pf_prev, w.oacc, lane);
    }

  }

  // Done with K/V: every load of it has been consumed (loads past the range
  // touch no memory), so the slot may be refilled once every workgroup of
  // the launch has counted itself here.  Only the order after these reads
  // matters, no data flows to the refill: a relaxed device-scope add.
  if (a.done_counter != nullptr) {
    __syncthreads();
    if (tid == 0) __hip_atomic_fetch_add(a.done_counter, (uint64_t)1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // Combine the two halves' denominators and normalise.
  const float l_tot = w.l_run + __shfl_xor(w.l_run, 32);
  const float inv = timed_out ? __builtin_nanf("") : l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_val = timed_out ? __builtin_nanf("")
                        : l_tot > 0.f ? (w.m_run + __log2f(l_tot)) * 0.69314718055994530942f : -INFINITY;
  if (!valid) return;
  if (sd.n_splits == 1) {
    store_row<D, DT>(w, inv, half, a.out + io_row * D);
    if (a.lse != nullptr && half == 0) a.lse[(int64_t)h * a.total_q + sd.cu_q + qpos] = lse_val;
    return;
  }

  // Split-key: write this split's normalised partial and its log-sum-exp.
  const int64_t prow = (int64_t)wi.split * a.total_q * a.n_q_heads + qrow;
  // The partial is a convex combination of V rows, so it fits the element
  // type's range; storing it in that type halves the split traffic for one
  // extra rounding (2^-9 relative for bf16, 2^-11 for fp16).
  store_row<D, DT>(w, inv, half, a.part_o + prow * D);
  if (half == 0) a.part_lse[prow] = lse_val;
}

// Split-key merge of NR (token, head) rows per lane group: D / 8 lanes per
// row, 8 dims per lane (`sub`); rows[i] < 0 are skipped; at most SMAX
// splits per row.  Weights
// exp(lse_s - max) over the row's splits, weighted sum of the partials,
// written to `out` (and the row's natural-log lse to lse_out if given).
// Every split's lse and partial chunk of all NR rows are loaded before any
// is used: one memory round trip, whatever the split count (merging a few
// thousand rows is latency-bound, not bandwidth-bound).
template <int D, int DT, int NR, int SMAX = kAttnMaxSplits>
__device__ __forceinline__ void merge_rows(const AttnArgs &a, const int64_t (&rows_i)[NR], int sub,
                                           const uint16_t *part_o, const float *part_lse, uint16_t *out,
                                           float *lse_out) {
  const int64_t rows = (int64_t)a.total_q * a.n_q_heads;
  SeqDesc sd[NR];
  float ls[NR][SMAX];
  u32x4 x[NR][SMAX];
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    const int64_t row = rows_i[i] < 0 ? 0 : rows_i[i];
    const int token = (int)(row / a.n_q_heads);
    int lo = 0;
    if (a.n_seqs > 1) {
      int hi = a.n_seqs - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.seqs[mid].cu_q <= token) lo = mid; else hi = mid - 1;
      }
    }
    sd[i] = a.seqs != nullptr ? a.seqs[lo] : a.seq0;
    const int S = rows_i[i] < 0 ? 0 : sd[i].n_splits;
    const uint16_t *po = part_o + row * D + sub * 8;
#pragma unroll
    for (int s = 0; s < SMAX; ++s) {
      if (s < S && S > 1) {
        ls[i][s] = part_lse[s * rows + row];
        x[i][s] = *reinterpret_cast<const u32x4 *>(po + (int64_t)s * rows * D);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < NR; ++i) {
    const int S = rows_i[i] < 0 ? 0 : sd[i].n_splits;
    if (S <= 1) continue;
    const int64_t row = rows_i[i];
    const int token = (int)(row / a.n_q_heads);
    const int h = (int)(row - (int64_t)token * a.n_q_heads);
    const int64_t io_row = (int64_t)(sd[i].q_off + token - sd[i].cu_q) * a.n_q_heads + h;
    float mx = -INFINITY;
#pragma unroll
    for (int s = 0; s < SMAX; ++s)
      if (s < S) mx = fmaxf(mx, ls[i][s]);
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float wsum = 0.f;
#pragma unroll
    for (int s = 0; s < SMAX; ++s)
      if (s < S) {
        const float wgt = ls[i][s] == -INFINITY ? 0.f : __expf(ls[i][s] - mx);
        wsum += wgt;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const f32x2 v = Elem<DT>::unpack(x[i][s][e]);
          acc[2 * e] += wgt * v[0];
          acc[2 * e + 1] += wgt * v[1];
        }
      }
    const float winv = wsum > 0.f ? 1.f / wsum : 0.f;
    u32x4 pk;
#pragma unroll
    for (int e = 0; e < 4; ++e) pk[e] = Elem<DT>::pack(acc[2 * e] * winv, acc[2 * e + 1] * winv);
    *reinterpret_cast<u32x4 *>(out + io_row * D + sub * 8) = pk;
    if (lse_out != nullptr && sub == 0)
      lse_out[(int64_t)h * a.total_q + token] = wsum > 0.f ? mx + __logf(wsum) : -INFINITY;
  }
}

// The deferred merge of the previous layer (AttnArgs::dm_out), run by a
// workgroup after its own item: it claims chunks of rows (one row per D / 8
// lanes, NR rows per lane group in one memory round trip) until all are
// claimed, so the workgroups that finish their items first do most of it.
// With at most four splits per row (the common plans) a lane group takes
// four rows; with more, one (the registers of the split values).  The
// claims only divide the work; no data flows through the counter (the
// partials were written by the previous launch on the stream).
template <int D, int DT, int NR, int SMAX>
__device__ __forceinline__ void deferred_merge_n(const AttnArgs &a) {
  constexpr int LPR = D / 8;
  constexpr int RPP = kThreads / LPR;   // rows per pass and row slot
  constexpr int64_t kChunk = (int64_t)NR * RPP;
  __shared__ uint32_t s_claim;
  const int64_t rows = (int64_t)a.total_q * a.n_q_heads;
  const int64_t n_chunks = (rows + kChunk - 1) / kChunk;
  const int sub = threadIdx.x % LPR;
  for (;;) {
    __syncthreads();                      // every lane has read the last claim
    if (threadIdx.x == 0)
      s_claim = __hip_atomic_fetch_add(a.dm_counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const int64_t c = (int64_t)s_claim;
    if (c >= n_chunks) break;
    const int64_t base = c * kChunk + threadIdx.x / LPR;
    int64_t rr[NR];
#pragma unroll
    for (int i = 0; i < NR; ++i) rr[i] = base + i * RPP < rows ? base + i * RPP : -1;
    merge_rows<D, DT, NR, SMAX>(a, rr, sub, a.dm_part_o, a.dm_part_lse, a.dm_out, nullptr);
  }
}

template <int D, int DT>
__device__ __forceinline__ void deferred_merge(const AttnArgs &a) {
  if (a.dm_max_splits <= 4)
    deferred_merge_n<D, DT, 4, 4>(a);
  else
    deferred_merge_n<D, DT, 1, kAttnMaxSplits>(a);
}

// Item of workgroup w in an implicit work list (see AttnArgs::seq0).
__device__ __forceinline__ WorkItem implicit_item(const AttnArgs &a, int w) {
  WorkItem wi{-1, 0, 0, 0, 0, 0, 0, 0};
  const int S = a.imp_splits;
  const int per_kvh = a.imp_tiles * S;
  const int j = w >> 3;
  const int g = (w & 7) * a.imp_per_xcd + j;
  if (j >= a.imp_per_xcd || g >= a.n_kv_heads * per_kvh) return wi;
  const int kvh = g / per_kvh;
  const int r = g - kvh * per_kvh;
  const int tile = r / S;
  const int sp = r - tile * S;
  const int q0 = tile * a.rows_q;
  const int nq = min(a.rows_q, a.seq0.n_new - q0);
  const int keys = a.seq0.prefix + q0 + nq;
  const int t = (keys + KT - 1) / KT;
  const int b0 = min(keys, (sp * t / S) * KT);
  const int b1 = min(keys, ((sp + 1) * t / S) * KT);
  wi.seq = 0;
  wi.kvh = kvh;
  wi.q0 = q0;
  wi.nq = nq;
  wi.k_begin = b0;
  wi.k_end = max(b0, b1);
  wi.split = sp;
  return wi;
}

template <int D, int DT>
__device__ __forceinline__ void attn_fwd_body(const AttnArgs &a) {
  const WorkItem wi = a.items != nullptr ? load_const(a.items + blockIdx.x) : implicit_item(a, blockIdx.x);
  if (wi.seq < 0) {
    // Padding slot (XCD placement): no K/V to read, but it counts as done
    // like every other workgroup of the launch.
    if (a.done_counter != nullptr && threadIdx.x == 0)
      __hip_atomic_fetch_add(a.done_counter, (uint64_t)1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  if constexpr (D == 128) {
    // K/V slots are the namespace-scope arrays above.
    if (wi.paged)
      attn_item<D, DT, true>(a, wi, nullptr);
    else
      attn_item<D, DT, false>(a, wi, nullptr);
  } else {
    __shared__ __attribute__((aligned(16))) uint16_t smem[Geo<D>::kSmem];
    if (wi.paged)
      attn_item<D, DT, true>(a, wi, smem);
    else
      attn_item<D, DT, false>(a, wi, smem);
  }
}

// One work item per workgroup, then (in a layer stack with deferred
// merges) its share of the previous layer's merge.
template <int D, int DT>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(AttnArgs a) {
  attn_fwd_body<D, DT>(a);
  if (a.dm_out != nullptr) deferred_merge<D, DT>(a);
}

template <int D, int DT>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  constexpr int LPR = D / 8;
  constexpr int RPB = 256 / LPR;
  const int64_t rows = (int64_t)a.total_q * a.n_q_heads;
  const int64_t row = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;
  if (row >= rows) return;
  const int64_t rr[1] = {row};
  merge_rows<D, DT, 1>(a, rr, threadIdx.x % LPR, a.part_o, a.part_lse, a.out, a.lse);
}

// Split-key partials of the allocation-free entry point: one array per
// device, held by the loaded code object until the process ends.  Host code
// must use the address hipGetSymbolAddress returns, never the symbol.
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

}  // namespace

hipError_t noalloc_scratch(int device, void **ptr, size_t *bytes) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (addr[device] == nullptr) {
    // Each device holds its own copy of the array at its own address, so
    // the lookup runs with that device current.
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device && (e = hipSetDevice(device)) != hipSuccess) return e;
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != device) (void)hipSetDevice(cur);
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[device] = p;
  }
  *ptr = addr[device];
  *bytes = kNoAllocScratchBytes;
  return hipSuccess;
}

hipError_t launch_attn_fwd(const AttnArgs &a, int head_dim, int n_items, hipStream_t stream) {
  if (n_items <= 0) return hipSuccess;
  const dim3 grid(n_items), block(kThreads);
  if (head_dim == 128) {
    if (a.dtype == SC_DTYPE_F16)
      hipLaunchKernelGGL((attn_fwd_kernel<128, SC_DTYPE_F16>), grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL((attn_fwd_kernel<128, SC_DTYPE_BF16>), grid, block, 0, stream, a);
  } else {
    if (a.dtype == SC_DTYPE_F16)
      hipLaunchKernelGGL((attn_fwd_kernel<64, SC_DTYPE_F16>), grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL((attn_fwd_kernel<64, SC_DTYPE_BF16>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

int attn_fwd_vgprs(int head_dim) {
  // The largest of the two element types' kernels for this head_dim.
  int m = -1;
  for (const void *f : {head_dim == 128 ? reinterpret_cast<const void *>(&attn_fwd_kernel<128, SC_DTYPE_BF16>)
                                        : reinterpret_cast<const void *>(&attn_fwd_kernel<64, SC_DTYPE_BF16>),
                        head_dim == 128 ? reinterpret_cast<const void *>(&attn_fwd_kernel<128, SC_DTYPE_F16>)
                                        : reinterpret_cast<const void *>(&attn_fwd_kernel<64, SC_DTYPE_F16>)}) {
    hipFuncAttributes at{};
    if (hipFuncGetAttributes(&at, f) != hipSuccess) return -1;
    m = at.numRegs > m ? at.numRegs : m;
  }
  return m;
}

size_t attn_fwd_lds_bytes(int head_dim) {
  // The largest static LDS of the two element types' kernels; the full LDS
  // of a CU if the runtime cannot tell.
  size_t m = 0;
  for (const void *f : {head_dim == 128 ? reinterpret_cast<const void *>(&attn_fwd_kernel<128, SC_DTYPE_BF16>)
                                        : reinterpret_cast<const void *>(&attn_fwd_kernel<64, SC_DTYPE_BF16>),
                        head_dim == 128 ? reinterpret_cast<const void *>(&attn_fwd_kernel<128, SC_DTYPE_F16>)
                                        : reinterpret_cast<const void *>(&attn_fwd_kernel<64, SC_DTYPE_F16>)}) {
    hipFuncAttributes at{};
    if (hipFuncGetAttributes(&at, f) != hipSuccess) return (size_t)160 << 10;
    m = at.sharedSizeBytes > m ? at.sharedSizeBytes : m;
  }
  return m;
}

hipError_t launch_attn_merge(const AttnArgs &a, int head_dim, hipStream_t stream) {
  const int64_t rows = (int64_t)a.total_q * a.n_q_heads;
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)((rows * (head_dim / 8) + 255) / 256)), block(256);
  if (head_dim == 128) {
    if (a.dtype == SC_DTYPE_F16)
      hipLaunchKernelGGL((attn_merge_kernel<128, SC_DTYPE_F16>), grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL((attn_merge_kernel<128, SC_DTYPE_BF16>), grid, block, 0, stream, a);
  } else {
    if (a.dtype == SC_DTYPE_F16)
      hipLaunchKernelGGL((attn_merge_kernel<64, SC_DTYPE_F16>), grid, block, 0, stream, a);
    else
      hipLaunchKernelGGL((attn_merge_kernel<64, SC_DTYPE_BF16>), grid, block, 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace sc
