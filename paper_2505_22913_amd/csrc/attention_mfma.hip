// Decode attention over compressed K/V for grouped queries (G = 2, 4, 8 query
// heads per kv-head) on gfx950: both contractions of Algorithm 1 on MFMA. The
// default route takes it from 8 query heads per kv-head on (the bit walks are
// faster below that); mustafar_attn_set_route can force it for G = 2 and 4.
//
// Same split-K scheme, staging and bit walks as the G = 1 kernel, but a
// compressed block of NB = 64/T tokens is expanded twice in LDS and contracted
// with v_mfma_f32_16x16x16f16 (fp16 inputs, fp32 accumulation):
//   * the key walk scatters the packed keys into Kd, one row per token; the
//     scores S[token][head] = Kd . Q^T are 16x16x16 MFMAs with Kd as the A
//     operand (16 tokens x 16 channels per lane group of 8-byte LDS reads) and
//     q, held in registers for the whole segment, as the B operand (16 channels
//     x 16 head columns, the G real heads and zeros);
//   * online softmax on the MFMA result layout: lane l holds head l % 16 and
//     tokens 4(l/16) + e, so each head's block maximum and sum are in-lane
//     reductions plus two cross-row shuffles;
//   * that layout is exactly the A operand of the p.V product (row = head,
//     k = token), so the probabilities go from the score registers to the
//     second MFMA without touching LDS; the value walk scatters the packed
//     values into VdT, one row per channel (B operand: 4 consecutive tokens of
//     one channel per 8-byte read), and O[head][channel] accumulates in 16x16
//     MFMA tiles of which the first G rows are real.
// The walks cost the same per key as the value walk of the G = 1 kernel; the G
// multiply-adds per key and channel move to the matrix cores.
#include "attn_common.h"

namespace mf {

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// The probabilities enter the p.V product as fp16, computed against the exact
// running maximum with this exponent bias: the largest is 2^15 (inside fp16),
// and the small ones keep 15 more binades before they flush to zero. The
// partial's maximum is written as m - kMfmaPBias, consistent with l and o.
constexpr float kMfmaPBias = 15.f;

// Slots per tile in Kd and VdT: channel c of half h is slot 4 + 36h + (c % 32);
// slot 3 + 36h is the scratch slot the walks address with channel -1, and the
// 4-channel groups the MFMA operands read stay 8-byte aligned.
constexpr int kMSlots = 72;

struct MfmaLds {
  uint32_t vst, kst, kd, vdt, total;
};

// Lane j T + t of a block walks tile t of token j: NB = 64 / T tokens per block.
// (Half-tile lanes -- 16-token blocks at d = 128, twice the waves per CU by LDS --
// measured 10-15% slower on the grouped-query workloads: their extra walk slots
// and per-block work outweighed the occupancy.)
template <int T>
struct MfmaGeom {
  static constexpr int NB = kWave / T;                     // tokens per block
  static constexpr int NG = NB / 16;                       // 16-token MFMA groups per block
  static constexpr int NC = (kTile * T) / 16;              // 16-channel chunks per token
  static constexpr uint32_t KD_ROW = T * kMSlots * 2 + 8;  // bytes per Kd row (token)
  static constexpr uint32_t VD_ROW = NB * 2 + 8;           // bytes per VdT row (channel slot)
};

// [vst][kst | Kd], with VdT overlaying kst | Kd: the keys are consumed (key walk,
// then the score MFMAs) before VdT is cleared and written.
template <int T>
__host__ __device__ inline MfmaLds mfma_lds_layout(int kmaxK, int kmaxV) {
  using Geo = MfmaGeom<T>;
  MfmaLds L;
  uint32_t o = 0;
  L.vst = o;
  o += (run_region_elems(Geo::NB * kmaxV) * 2 + 15) & ~15u;
  L.kst = o;
  L.vdt = o;
  const uint32_t kst_bytes = (run_region_elems(Geo::NB * kmaxK) * 2 + 15) & ~15u;
  L.kd = o + kst_bytes;
  const uint32_t a = kst_bytes + Geo::NB * Geo::KD_ROW;
  const uint32_t b = T * kMSlots * Geo::VD_ROW;
  L.total = o + (((a > b ? a : b) + 15) & ~15u);
  return L;
}

__device__ __forceinline__ void lds_zero(uint32_t addr, uint32_t bytes, uint32_t lane) {
  const u32x4 z = {0u, 0u, 0u, 0u};
  for (uint32_t i = lane * 16u; i < bytes; i += kWave * 16u) lds_store<u32x4>(addr + i, z);
}

template <int T, int G, int STAGE>
__device__ __forceinline__ void sparse_body_mfma(const AttnArgs& a, int seg, int bh, unsigned char* smem,
                                                 float& m_run, float& l_run,
                                                 f32x4 (&o)[MfmaGeom<T>::NC]) {
  using Geo = MfmaGeom<T>;
  constexpr int d = kTile * T;
  constexpr int NB = Geo::NB, NG = Geo::NG, NC = Geo::NC;
  const MfmaLds L = mfma_lds_layout<T>(a.kmaxK, a.kmaxV);
  const uint32_t base = lds_addr(smem);
  const uint32_t lane = lane_id();
  const uint32_t j = lane / T, t = lane % T;       // walk layout: token j, tile t
  const uint32_t r16 = lane % 16, q4 = lane / 16;  // MFMA layout: column, row quad

  // q as the B operand of the score MFMA: column r16 = head (zero past G),
  // k = 4 q4 + e = channel within the 16-channel chunk.
  half4_t qb[NC];
  {
    const uint16_t* qsrc = a.q + ((int64_t)bh * G + (r16 < (uint32_t)G ? r16 : 0u)) * d;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const u32x2 w = *reinterpret_cast<const u32x2*>(qsrc + 16 * c + 4 * q4);
      const half2_t lo = as_h2(w.x), hi = as_h2(w.y);
      const half4_t v = {lo.x, lo.y, hi.x, hi.y};
      const half4_t z = {(_Float16)0.f, (_Float16)0.f, (_Float16)0.f, (_Float16)0.f};
      qb[c] = r16 < (uint32_t)G ? v : z;
    }
  }

  const int j0 = seg * a.sparse_seg_tokens;
  const int j1 = min(j0 + a.sparse_seg_tokens, stream_tokens(a, bh));
  if (j0 >= j1) return;  // past this stream's tokens: an empty partial
  const int64_t kt0 = (int64_t)bh * a.K.cap_tokens * T;
  const int64_t vt0 = (int64_t)bh * a.V.cap_tokens * T;
  const uint16_t* kv = a.K.values + (int64_t)bh * a.K.val_stride;
  const uint16_t* vv = a.V.values + (int64_t)bh * a.V.val_stride;

  int nb = min(NB, j1 - j0);
  TileMeta cur = load_meta<T>(a, kt0, vt0, j0, nb, lane);
  RunPos pos = segment_start<T>(a, kt0, vt0, j0);
  Runs rcur = runs_of(cur, pos);
  u32x4 stg[STAGE];
  stage_issue<STAGE>(stg, kv, vv, rcur, lane);
  int nb_next = min(NB, j1 - (j0 + NB));
  TileMeta nxt = {0ull, 0ull, 0u, 0u};
  if (nb_next > 0) nxt = load_meta<T>(a, kt0, vt0, j0 + NB, nb_next, lane);
  stage_commit<STAGE>(stg, base + L.kst, base + L.vst, rcur, lane);

  // Walk destinations: channel c of half h of this lane's tile.
  const uint32_t kd_w0 = base + L.kd + j * Geo::KD_ROW + (t * kMSlots + 4u) * 2u;
  const uint32_t kd_w1 = kd_w0 + 36u * 2u;
  const uint32_t vd_w0 = base + L.vdt + (t * kMSlots + 4u) * Geo::VD_ROW + j * 2u;
  const uint32_t vd_w1 = vd_w0 + 36u * Geo::VD_ROW;

  for (int b0 = j0; b0 < j1; b0 += NB) {
    const bool has_next = nb_next > 0;
    Runs rnext = {0u, 0u, 0u, 0u};
    TileMeta nxt2 = {0ull, 0ull, 0u, 0u};
    const int nb_next2 = min(NB, j1 - (b0 + 2 * NB));
    if (has_next) rnext = runs_of(nxt, pos);
    stage_issue<STAGE>(stg, kv, vv, rnext, lane);
    if (nb_next2 > 0) nxt2 = load_meta<T>(a, kt0, vt0, b0 + 2 * NB, nb_next2, lane);

    // Expand the keys (tokens past the block end have empty bitmaps).
    const WalkCounts wc = walk_counts(cur.kb, cur.vb);
    lds_zero(base + L.kd, NB * Geo::KD_ROW, lane);
    {
      const uint32_t va = base + L.kst + ((int)j < nb ? 2u * cur.ko : 0u);
      expand_tile<2u>(wc.klo, wc.khi, cur.kb, va, kd_w0, kd_w1);
    }

    // Scores: S[group g][token 4 q4 + e][head r16].
    f32x4 sc[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      sc[g] = (f32x4){0.f, 0.f, 0.f, 0.f};
      const uint32_t row = base + L.kd + (16u * g + r16) * Geo::KD_ROW;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const uint32_t ch = 16u * (c % 4) + 4u * q4;  // channel within the tile c / 4
        const uint32_t slot = (c / 4) * kMSlots + 4u + (ch >= 32u ? 36u : 0u) + (ch % 32u);
        const half4_t ka = lds_load<half4_t>(row + 2u * slot);
        sc[g] = __builtin_amdgcn_mfma_f32_16x16x16f16(ka, qb[c], sc[g], 0, 0, 0);
        // At most four operand loads ahead of their products (register budget).
        if (c % 4 == 3) __builtin_amdgcn_sched_barrier(0);
      }
    }

    // Online softmax per head (lanes with the same r16 share a head).
    float bmax = -INFINITY;
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int tok = 16 * g + 4 * (int)q4 + e;
        const float v = tok < nb ? sc[g][e] * a.scale_log2 : -INFINITY;
        sc[g][e] = v;
        bmax = fmaxf(bmax, v);
      }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 16, kWave));
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, kWave));
    const float mnew = fmaxf(m_run, bmax);
    const float alpha = __builtin_amdgcn_exp2f(m_run - mnew);
    // p = exp2(score - mnew + kMfmaPBias) in fp16 (at most 2^15); the sum is
    // taken over the same rounded p that the p.V product multiplies.
    float psum = 0.f;
    half4_t pa[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const _Float16 ph =
            r16 < (uint32_t)G ? (_Float16)__builtin_amdgcn_exp2f(sc[g][e] - mnew + kMfmaPBias) : (_Float16)0.f;
        pa[g][e] = ph;
        psum += (float)ph;
      }
    }
    psum += __shfl_xor(psum, 16, kWave);
    psum += __shfl_xor(psum, 32, kWave);
    l_run = l_run * alpha + psum;
    m_run = mnew;

    // Expand the values (VdT overlays the consumed keys).
    lds_zero(base + L.vdt, T * kMSlots * Geo::VD_ROW, lane);
    {
      const uint32_t va = base + L.vst + ((int)j < nb ? 2u * cur.vo : 0u);
      expand_tile<Geo::VD_ROW>(wc.vlo, wc.vhi, cur.vb, va, vd_w0, vd_w1);
    }

    // Rescale the accumulators: row 4 q4 + e of every O tile is head 4 q4 + e.
    if (ballot(alpha != 1.f)) {
      float ar[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float v = 1.f;
#pragma unroll
        for (int h = 0; h < G; ++h)
          v = (4u * q4 + (uint32_t)e == (uint32_t)h) ? readlane_f(alpha, h) : v;
        ar[e] = v;
      }
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int e = 0; e < 4; ++e) o[c][e] *= ar[e];
    }

    // p.V: O[head][channel chunk c] += P[head][16 tokens] . VdT.
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const uint32_t ch = 16u * (c % 4) + r16;  // channel within the tile c / 4
      const uint32_t row = (c / 4) * kMSlots + 4u + (ch >= 32u ? 36u : 0u) + (ch % 32u);
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const half4_t vb = lds_load<half4_t>(base + L.vdt + row * Geo::VD_ROW + (16u * g + 4u * q4) * 2u);
        o[c] = __builtin_amdgcn_mfma_f32_16x16x16f16(pa[g], vb, o[c], 0, 0, 0);
      }
      if (c % 2 == 1) __builtin_amdgcn_sched_barrier(0);
    }

    if (has_next) {
      stage_commit<STAGE>(stg, base + L.kst, base + L.vst, rnext, lane);
      cur = nxt;
      rcur = rnext;
      nxt = nxt2;
    }
    nb = nb_next;
    nb_next = nb_next2;
  }
}

// Waves per SIMD that an instance's register budget is set for: three (168
// VGPRs) where its registers fit without spilling, else two (256), and one for
// the largest staging at d = 256. Unbounded, the compiler took 196-260 VGPRs at
// d = 128 (two waves) and 272-353 at d = 256 (one wave); with the operand loads
// of the two products kept a few MFMAs ahead (the scheduling barriers above)
// these bounds need no spills.
template <int T, int G, int STAGE>
constexpr int mfma_waves() {
  if ((T == 1 && (STAGE <= 6 || (STAGE == 8 && G <= 4))) || (T == 2 && (STAGE == 4 || (STAGE == 6 && G >= 4))))
    return 3;
  return (T == 4 && STAGE == 16) ? 1 : 2;
}

// Sparse call on the matrix cores (G >= 2 query heads per kv-head): grid
// (n_sparse_segs + n_dense_segs, BHkv).
template <int T, int G, int STAGE>
__global__ __launch_bounds__(64, (mfma_waves<T, G, STAGE>())) void k_sparse_attn_mfma(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int seg = blockIdx.x, bh = blockIdx.y;
  if (seg >= a.n_sparse_segs) {
    float m_run[G], l_run[G], od[G][T];
    init_state<T, G>(m_run, l_run, od);
    dense_body<T, G>(a, seg - a.n_sparse_segs, bh, smem, m_run, l_run, od);
    write_partial<T, G>(a, seg, bh, m_run, l_run, od);
    return;
  }
  using Geo = MfmaGeom<T>;
  constexpr int d = kTile * T;
  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[Geo::NC];
#pragma unroll
  for (int c = 0; c < Geo::NC; ++c) o[c] = (f32x4){0.f, 0.f, 0.f, 0.f};
  sparse_body_mfma<T, G, STAGE>(a, seg, bh, smem, m_run, l_run, o);
  m_run -= kMfmaPBias;  // -inf stays -inf for an empty segment

  const uint32_t lane = lane_id();
  const uint32_t r16 = lane % 16, q4 = lane / 16;
  const int64_t row0 = (int64_t)seg * a.BHq + (int64_t)bh * G;
  if (q4 == 0 && r16 < (uint32_t)G) a.ws_ml[row0 + r16] = make_float2(m_run, l_run);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t h = 4u * q4 + (uint32_t)e;
    if (h < (uint32_t)G) {
#pragma unroll
      for (int c = 0; c < Geo::NC; ++c) a.ws_o[(row0 + h) * d + 16 * c + r16] = o[c][e];
    }
  }
}

template <int T, int G, int STAGE>
static hipError_t mfma_launch(const AttnShape& sh, const AttnArgs& a, hipStream_t s) {
  const MfmaLds L = mfma_lds_layout<T>(a.kmaxK, a.kmaxV);
  size_t lds = L.total;
  if (sh.n_dense_segs > 0 && dense_lds_bytes(T, G) > lds) lds = dense_lds_bytes(T, G);
  hipLaunchKernelGGL((k_sparse_attn_mfma<T, G, STAGE>), dim3(sh.n_sparse_segs + sh.n_dense_segs, sh.BHkv),
                     dim3(kWave), lds, s, a);
  return hipGetLastError();
}

template <int T, int G>
static hipError_t mfma_stage(const AttnShape& sh, const AttnArgs& a_in, hipStream_t s) {
  constexpr int NB = MfmaGeom<T>::NB;
  // Staging bounds for this kernel's blocks (a per-channel cache's bound depends
  // on the block length).
  AttnArgs a = a_in;
  a.kmaxK = side_token_bound(kTile * T, a.K, NB);
  a.kmaxV = side_token_bound(kTile * T, a.V, NB);
  const int chunks = (NB * a.kmaxK + 511) / 512 + (NB * a.kmaxV + 511) / 512;
  if (chunks <= 4) return mfma_launch<T, G, 4>(sh, a, s);
  if (chunks <= 6) return mfma_launch<T, G, 6>(sh, a, s);
  if (chunks <= 8) return mfma_launch<T, G, 8>(sh, a, s);
  if (chunks <= 12) return mfma_launch<T, G, 12>(sh, a, s);
  return mfma_launch<T, G, 16>(sh, a, s);
}

template <int T>
static hipError_t mfma_T(const AttnShape& sh, const AttnArgs& a, hipStream_t s) {
  switch (sh.G) {
    case 2: return mfma_stage<T, 2>(sh, a, s);
    case 4: return mfma_stage<T, 4>(sh, a, s);
    case 8: return mfma_stage<T, 8>(sh, a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_sparse_mfma(const AttnShape& sh, const AttnArgs& a, hipStream_t s) {
  switch (sh.T) {
    case 1: return mfma_T<1>(sh, a, s);
    case 2: return mfma_T<2>(sh, a, s);
    case 4: return mfma_T<4>(sh, a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mf
