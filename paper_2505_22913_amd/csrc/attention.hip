// Decode attention over compressed K/V plus a dense window (Algorithm 1) on gfx950.
//
// Split-K: every (batch, kv-head) stream is cut into token segments; a
// one-wave workgroup computes, for the G query heads of its kv-head, the
// running max, running sum and unnormalised output of one segment (online
// softmax), and k_merge combines the segments with their log-sum-exp weights.
// The sparse call launches the compressed segments and the dense-window
// segment in one grid, so the softmax spans concat(S_C, S_L) as Algorithm 1
// states (the merge is order-free). The dense baseline reuses the dense body.
//
// Compressed blocks of NB = 64/T tokens ("load as compressed, expand in LDS"):
//   * the packed values of a block are one contiguous run of the stream; the
//     next block's runs are fetched into registers with 16-byte coalesced
//     loads while the current block is computed, then written to LDS;
//   * lane (j, t) owns tile t of token j and walks the set bits of each
//     32-bit half of its bitmap with v_ffbl, reading its packed values in
//     order, 8 at a time with one 16-byte LDS load. A lane with no bits left
//     gets the index -1, which points at a zero slot of the q table (its
//     product is 0) and at a scratch slot of the expanded value tile, so the
//     walk has no per-element branch; it runs in groups of 8 while any lane
//     has bits left;
//   * p.V runs with one lane per channel over the expanded value tile, two
//     tokens at a time with v_dot2 (fp16 probabilities, fp32 accumulation).
#include "attn_common.h"

namespace mf {

// The walks are software-pipelined: a group is split into an issue step (its
// 16-byte value load, its channels and, for keys, its q loads) and a consume
// step (the products, or the scatter into the expanded tile), and the loop
// issues group g+1 before consuming group g, so each group's LDS round trip
// overlaps the previous group's arithmetic. Two register sets alternate.
template <int G> struct QVal { u32x2 v[G / 4]; };  // q of G heads at one channel (G >= 4)
template <> struct QVal<1> { _Float16 v; };
template <> struct QVal<2> { half2_t v; };

template <int G>
struct KeyGroup {
  u32x4 w;
  QVal<G> q[8];
};

template <int G, bool PEEL>
__device__ __forceinline__ void key_issue(uint32_t& x, uint32_t va, uint32_t qaddr, uint32_t m,
                                          KeyGroup<G>& k) {
  k.w = lds_load<u32x4>(va);
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const uint32_t qa = qaddr + next_channel<PEEL>(x, u, m) * (2u * G);
    if constexpr (G == 1) {
      k.q[u].v = lds_load<_Float16>(qa);
    } else if constexpr (G == 2) {
      k.q[u].v = lds_load<half2_t>(qa);
    } else {
#pragma unroll
      for (int g4 = 0; g4 < G / 4; ++g4) k.q[u].v[g4] = lds_load<u32x2>(qa + 8u * g4);
    }
  }
}

template <int G>
__device__ __forceinline__ void key_consume(const KeyGroup<G>& k, float (&acc)[G]) {
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const float v = (float)group_value(k.w, u);
    if constexpr (G == 1) {
      acc[0] = fmaf((float)k.q[u].v, v, acc[0]);
    } else if constexpr (G == 2) {
      acc[0] = fmaf((float)k.q[u].v.x, v, acc[0]);
      acc[1] = fmaf((float)k.q[u].v.y, v, acc[1]);
    } else {
#pragma unroll
      for (int g4 = 0; g4 < G / 4; ++g4) {
        const half2_t q01 = as_h2(k.q[u].v[g4].x);
        const half2_t q23 = as_h2(k.q[u].v[g4].y);
        acc[4 * g4 + 0] = fmaf((float)q01.x, v, acc[4 * g4 + 0]);
        acc[4 * g4 + 1] = fmaf((float)q01.y, v, acc[4 * g4 + 1]);
        acc[4 * g4 + 2] = fmaf((float)q23.x, v, acc[4 * g4 + 2]);
        acc[4 * g4 + 3] = fmaf((float)q23.y, v, acc[4 * g4 + 3]);
      }
    }
  }
}

// One 32-channel half of a key tile: n groups of 8 from byte address a (n is the
// busiest lane's count, so the loop is uniform and every iteration issues the
// next group before consuming the current one); the first group has m phantom
// slots when PEEL.
template <int G, bool PEEL>
__device__ __forceinline__ void key_half(uint32_t x, uint32_t a, uint32_t qaddr, uint32_t m,
                                         float (&acc)[G]) {
  const int n = wave_max_int((int)(m + (uint32_t)__popc(x) + 7u) >> 3);
  if (n == 0) return;
  KeyGroup<G> k0, k1;
  key_issue<G, PEEL>(x, a, qaddr, m, k0);
  int g = 1;
  for (; g + 1 < n; g += 2) {
    key_issue<G, false>(x, a + 16u * g, qaddr, 0u, k1);
    key_consume<G>(k0, acc);
    key_issue<G, false>(x, a + 16u * (g + 1), qaddr, 0u, k0);
    key_consume<G>(k1, acc);
  }
  if (g < n) {
    key_issue<G, false>(x, a + 16u * g, qaddr, 0u, k1);
    key_consume<G>(k0, acc);
    key_consume<G>(k1, acc);
  } else {
    key_consume<G>(k0, acc);
  }
}

// Scores of one tile: q . k over its 64-bit bitmap `bm`, values at LDS byte address `va`.
template <int G>
__device__ __forceinline__ void key_walk(uint64_t bm, uint32_t va, uint32_t q_w0, uint32_t q_w1,
                                         float (&acc)[G]) {
  const uint32_t lo = (uint32_t)bm, s = (uint32_t)__popc(lo), m = s & 7u;
  key_half<G, false>(lo, va, q_w0, 0u, acc);
  key_half<G, true>((uint32_t)(bm >> 32), va + 2u * (s - m), q_w1, m, acc);
}

// Expansion of one value tile into the dense tile.
__device__ __forceinline__ void value_walk(uint64_t bm, uint32_t va, uint32_t d_w0, uint32_t d_w1) {
  const uint32_t lo = (uint32_t)bm, s = (uint32_t)__popc(lo), m = s & 7u;
  value_half<false, 4u>(lo, va, d_w0, 0u);
  value_half<true, 4u>((uint32_t)(bm >> 32), va + 2u * (s - m), d_w1, m);
}

// LDS layout of the compressed body (byte offsets). The expanded value tile
// shares its bytes with the staged keys: it is cleared after the key walk of a
// block and read by p.V before the next block's keys are committed. A
// workgroup is one wave, whose LDS operations execute in program order, so the
// phases need no barrier.
struct SparseLds {
  uint32_t qtab, ps, dense, kst, vst, total;
};

__host__ __device__ inline SparseLds sparse_lds_layout(int T, int G, int kmaxK, int kmaxV) {
  const int NB = kWave / T;
  SparseLds L;
  uint32_t o = 0;
  L.qtab = o;  o += ((T * kSlots * G * 2) + 15) & ~15;          // [t][slot][g] fp16
  L.ps = o;    o += ((NB / 2) * G * 4 + 15) & ~15;              // [pair][g] half2
  L.vst = o;   o += ((NB * kmaxV + kMargin) * 2 + 15) & ~15;
  const uint32_t kst_bytes = ((NB * kmaxK + kMargin) * 2 + 15) & ~15;
  const uint32_t dense_bytes = (NB / 2) * T * kSlots * 4;      // [pair][t][slot][2] fp16
  L.kst = o;
  L.dense = o;
  o += kst_bytes > dense_bytes ? kst_bytes : dense_bytes;
  L.total = o;
  return L;
}

template <int T, int G, int STAGE>
__device__ __forceinline__ void sparse_body(const AttnArgs& a, int seg, int bh, unsigned char* smem,
                                            float (&m_run)[G], float (&l_run)[G],
                                            float (&o)[G][T]) {
  constexpr int d = kTile * T;
  constexpr int NB = kWave / T;
  const SparseLds L = sparse_lds_layout(T, G, a.kmaxK, a.kmaxV);
  const uint32_t base = lds_addr(smem);
  uint16_t* kst = reinterpret_cast<uint16_t*>(smem + L.kst);
  uint16_t* vst = reinterpret_cast<uint16_t*>(smem + L.vst);
  const uint32_t lane = lane_id();
  const uint32_t j = lane / T, t = lane % T;

  // q table with zero scratch slots: [t][slot][g].
  {
    const uint16_t* qsrc = a.q + (int64_t)bh * G * d;
    uint16_t* qt = reinterpret_cast<uint16_t*>(smem + L.qtab);
    for (int i = lane; i < T * kSlots * G; i += kWave) {
      const int g = i % G, slot = (i / G) % kSlots, tt = i / (G * kSlots);
      const int c = slot < 33 ? slot - 1 : slot - 2;
      qt[i] = (slot == 0 || slot == 33) ? (uint16_t)0 : qsrc[g * d + kTile * tt + c];
    }
  }

  const int j0 = seg * a.sparse_seg_tokens;
  const int j1 = min(j0 + a.sparse_seg_tokens, a.n_s);
  const int64_t kt0 = (int64_t)bh * a.K.cap_tokens * T;
  const int64_t vt0 = (int64_t)bh * a.V.cap_tokens * T;
  const uint16_t* kv = a.K.values + (int64_t)bh * a.K.val_stride;
  const uint16_t* vv = a.V.values + (int64_t)bh * a.V.val_stride;

  // Prologue: block 0 staged in LDS, metadata of block 1 in flight.
  int nb = min(NB, j1 - j0);
  TileMeta cur = load_meta<T>(a, kt0, vt0, j0, nb, lane);
  Runs rcur = runs_of<T>(cur, nb);
  u32x4 stg[STAGE];
  stage_issue<STAGE>(stg, kv, vv, a.K.values, rcur, lane);
  int nb_next = min(NB, j1 - (j0 + NB));
  TileMeta nxt = {0ull, 0ull, 0u, 0u};
  if (nb_next > 0) nxt = load_meta<T>(a, kt0, vt0, j0 + NB, nb_next, lane);
  stage_commit<STAGE>(stg, kst, vst, rcur, lane);

  // Per-lane constant addresses.
  const uint32_t q_w0 = base + L.qtab + (uint32_t)((t * kSlots + 1) * G * 2);
  const uint32_t q_w1 = q_w0 + 33u * G * 2;
  const uint32_t d_w0 = base + L.dense + (uint32_t)((((j >> 1) * T + t) * kSlots + 1) * 4 + (j & 1) * 2);
  const uint32_t d_w1 = d_w0 + 33u * 4;
  const uint32_t pv_slot = lane < 32 ? 1 + lane : 2 + lane;  // PV: lane = channel of each tile

  for (int b0 = j0; b0 < j1; b0 += NB) {
    // Software pipeline: fetch the next block's values and the metadata after it.
    const bool has_next = nb_next > 0;
    Runs rnext = {0u, 0u, 0u, 0u};
    TileMeta nxt2 = {0ull, 0ull, 0u, 0u};
    const int nb_next2 = min(NB, j1 - (b0 + 2 * NB));
    if (has_next) rnext = runs_of<T>(nxt, nb_next);
    stage_issue<STAGE>(stg, kv, vv, a.K.values, rnext, lane);
    if (nb_next2 > 0) nxt2 = load_meta<T>(a, kt0, vt0, b0 + 2 * NB, nb_next2, lane);

    // Scores.
    float acc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g] = 0.f;
    {
      const uint32_t va = base + L.kst + ((int)j < nb ? 2u * (cur.ko - rcur.kstart) : 0u);
      key_walk<G>(cur.kb, va, q_w0, q_w1, acc);
    }
    const bool valid = (int)j < nb;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float sc = valid ? tile_sum<T>(acc[g]) * a.scale_log2 : -INFINITY;
      const float mnew = fmaxf(m_run[g], wave_max_u(sc));
      const float alpha = __builtin_amdgcn_exp2f(m_run[g] - mnew);
      const _Float16 ph = valid ? (_Float16)__builtin_amdgcn_exp2f(sc - mnew) : (_Float16)0.f;
      l_run[g] = l_run[g] * alpha + wave_sum_u(t == 0 ? (float)ph : 0.f);
      m_run[g] = mnew;
#pragma unroll
      for (int tt = 0; tt < T; ++tt) o[g][tt] *= alpha;
      if (t == 0) lds_store<_Float16>(base + L.ps + ((j >> 1) * G + g) * 4 + (j & 1) * 2, ph);
    }

    // Clear the expanded value tile (it overwrites the staged keys, read above).
    {
      constexpr int n16 = (NB / 2) * T * kSlots * 4 / 16;
      const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int i = 0; i < (n16 + kWave - 1) / kWave; ++i)
        if (i * kWave + (int)lane < n16) lds_store<u32x4>(base + L.dense + 16u * (i * kWave + lane), z);
    }

    // Expand the value tiles.
    {
      const uint32_t va = base + L.vst + ((int)j < nb ? 2u * (cur.vo - rcur.vstart) : 0u);
      value_walk(cur.vb, va, d_w0, d_w1);
    }

    // p.V over every token pair of the block (tokens past its end have p = 0
    // and zero values), unrolled so the LDS loads of a batch are in flight
    // together: lane = channel `lane` of every tile.
    constexpr int NP = NB / 2;
    constexpr int PB = G >= 4 ? 4 : 8;
#pragma unroll 1
    for (int pb = 0; pb < NP; pb += PB) {
      half2_t p2[PB][G], v2[PB][T];
#pragma unroll
      for (int i = 0; i < PB; ++i) {
        const int pr = pb + i;
        if constexpr (G == 1) {
          p2[i][0] = lds_load<half2_t>(base + L.ps + pr * 4);
        } else if constexpr (G == 2) {
          const u32x2 w = lds_load<u32x2>(base + L.ps + pr * 8);
          p2[i][0] = as_h2(w.x);
          p2[i][1] = as_h2(w.y);
        } else {
#pragma unroll
          for (int g4 = 0; g4 < G; g4 += 4) {
            const u32x4 w = lds_load<u32x4>(base + L.ps + (pr * G + g4) * 4);
            p2[i][g4 + 0] = as_h2(w.x);
            p2[i][g4 + 1] = as_h2(w.y);
            p2[i][g4 + 2] = as_h2(w.z);
            p2[i][g4 + 3] = as_h2(w.w);
          }
        }
#pragma unroll
        for (int tt = 0; tt < T; ++tt)
          v2[i][tt] = lds_load<half2_t>(base + L.dense + ((pr * T + tt) * kSlots + pv_slot) * 4);
      }
#pragma unroll
      for (int i = 0; i < PB; ++i)
#pragma unroll
        for (int tt = 0; tt < T; ++tt)
#pragma unroll
          for (int g = 0; g < G; ++g) o[g][tt] = __builtin_amdgcn_fdot2(v2[i][tt], p2[i][g], o[g][tt], false);
    }

    if (has_next) {
      stage_commit<STAGE>(stg, kst, vst, rnext, lane);
      cur = nxt;
      rcur = rnext;
      nxt = nxt2;
    }
    nb = nb_next;
    nb_next = nb_next2;
  }
}

// Sparse call: grid (n_sparse_segs + n_dense_segs, BHkv); compressed segments first.
template <int T, int G, int STAGE>
__global__ __launch_bounds__(64) void k_sparse_attn(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int seg = blockIdx.x, bh = blockIdx.y;
  float m_run[G], l_run[G], o[G][T];
  init_state<T, G>(m_run, l_run, o);
  if (seg < a.n_sparse_segs)
    sparse_body<T, G, STAGE>(a, seg, bh, smem, m_run, l_run, o);
  else
    dense_body<T, G>(a, seg - a.n_sparse_segs, bh, smem, m_run, l_run, o);
  write_partial<T, G>(a, seg, bh, m_run, l_run, o);
}

// Dense baseline: grid (n_dense_segs, BHkv).
template <int T, int G>
__global__ __launch_bounds__(64) void k_dense_attn(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int seg = blockIdx.x, bh = blockIdx.y;
  float m_run[G], l_run[G], o[G][T];
  init_state<T, G>(m_run, l_run, o);
  dense_body<T, G>(a, seg, bh, smem, m_run, l_run, o);
  write_partial<T, G>(a, seg, bh, m_run, l_run, o);
}

// grid (BHq, parts), 4 waves: log-sum-exp merge of segments [part * per,
// part * per + per) of one query head. The 256 threads first reduce the
// segments' maxima and weighted sums; then wave w accumulates the weighted
// partial outputs of segments w, w+4, ... (lane = channel, four segments'
// loads in flight) and LDS adds the waves. With FINAL the result is divided
// by the sum and written as fp16 (RNE); otherwise (max, sum, unnormalised
// output) is written as one segment of a second, shorter merge -- used when
// there are many segments and few query heads, so that the merge runs on many
// workgroups instead of one per head.
constexpr int kMergeWaves = 4;
constexpr int kMergeSegsPerPart = 32;

__device__ __forceinline__ float block_reduce(float v, bool is_max, float* red) {
  v = is_max ? wave_max_u(v) : wave_sum_u(v);
  const int wave = threadIdx.x / kWave;
  if (lane_id() == 0) red[wave] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < kMergeWaves; ++w) r = is_max ? fmaxf(r, red[w]) : r + red[w];
  __syncthreads();
  return r;
}

template <int T, bool FINAL>
__global__ __launch_bounds__(kMergeWaves * kWave) void k_merge(const float2* __restrict__ ws_ml,
                                                              const float* __restrict__ ws_o,
                                                              int n_seg, int per, int BHq,
                                                              uint16_t* __restrict__ out,
                                                              float2* __restrict__ part_ml,
                                                              float* __restrict__ part_o) {
  constexpr int d = kTile * T;
  __shared__ float red[kMergeWaves];
  __shared__ float part[kMergeWaves][d];
  const int r = blockIdx.x;
  const int s0 = blockIdx.y * per, s1 = min(n_seg, s0 + per);
  const int tid = threadIdx.x, wave = tid / kWave;
  const uint32_t lane = lane_id();
  float M = -INFINITY;
  for (int s = s0 + tid; s < s1; s += kMergeWaves * kWave) M = fmaxf(M, ws_ml[(int64_t)s * BHq + r].x);
  M = block_reduce(M, true, red);
  float L = 0.f;
  for (int s = s0 + tid; s < s1; s += kMergeWaves * kWave) {
    const float2 ml = ws_ml[(int64_t)s * BHq + r];
    L = fmaf(ml.y, ml.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml.x - M), L);
  }
  L = block_reduce(L, false, red);

  float acc[T];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) acc[tt] = 0.f;
#pragma unroll 4
  for (int s = s0 + wave; s < s1; s += kMergeWaves) {
    const float2 ml = ws_ml[(int64_t)s * BHq + r];
    const float w = ml.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml.x - M);
    const float* o = ws_o + ((int64_t)s * BHq + r) * d + lane;
#pragma unroll
    for (int tt = 0; tt < T; ++tt) acc[tt] = fmaf(o[kTile * tt], w, acc[tt]);
  }
#pragma unroll
  for (int tt = 0; tt < T; ++tt) part[wave][lane + kTile * tt] = acc[tt];
  __syncthreads();
  if (wave == 0) {
    const float inv = 1.f / L;
    const int64_t prow = (int64_t)blockIdx.y * BHq + r;
    if (!FINAL && lane == 0) part_ml[prow] = make_float2(M, L);
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
      float v = part[0][lane + kTile * tt];
#pragma unroll
      for (int w = 1; w < kMergeWaves; ++w) v += part[w][lane + kTile * tt];
      if constexpr (FINAL)
        out[(int64_t)r * d + lane + kTile * tt] = __builtin_bit_cast(uint16_t, (_Float16)(v * inv));
      else
        part_o[prow * d + lane + kTile * tt] = v;
    }
  }
}

// ------------------------------------------------------------------------------------------
// Host-side launch.
// ------------------------------------------------------------------------------------------
template <int T, int G, int STAGE>
static hipError_t sparse_launch(const AttnShape& sh, const AttnArgs& a, hipStream_t s) {
  const SparseLds L = sparse_lds_layout(T, G, a.kmaxK, a.kmaxV);
  size_t lds = L.total;
  if (sh.n_dense_segs > 0 && dense_lds_bytes(T, G) > lds) lds = dense_lds_bytes(T, G);
  hipLaunchKernelGGL((k_sparse_attn<T, G, STAGE>), dim3(sh.n_sparse_segs + sh.n_dense_segs, sh.BHkv),
                     dim3(kWave), lds, s, a);
  return hipGetLastError();
}

template <int T, int G>
static hipError_t sparse_stage(const AttnShape& sh, const AttnArgs& a, hipStream_t s) {
  const int NB = kWave / T;
  const int chunks = (NB * a.kmaxK + 511) / 512 + (NB * a.kmaxV + 511) / 512;
  if (chunks <= 4) return sparse_launch<T, G, 4>(sh, a, s);
  if (chunks <= 6) return sparse_launch<T, G, 6>(sh, a, s);
  if (chunks <= 8) return sparse_launch<T, G, 8>(sh, a, s);
  if (chunks <= 12) return sparse_launch<T, G, 12>(sh, a, s);
  return sparse_launch<T, G, 16>(sh, a, s);
}

template <int T, int G>
static hipError_t attention_TG(const AttnShape& sh, const AttnArgs& a, uint16_t* out, hipStream_t s) {
  const int n_seg = sh.n_sparse_segs + sh.n_dense_segs;
  hipError_t e;
  if (sh.n_sparse_segs > 0) {
    // Grouped queries contract on the matrix cores (attention_mfma.hip).
    e = G >= kMfmaMinGroup ? launch_sparse_mfma(sh, a, s) : sparse_stage<T, G>(sh, a, s);
  } else if (sh.n_s == 0 && sh.n_dense_segs > 0 && a.K.bitmaps != nullptr) {
    // Sparse call with an empty compressed cache: only the window segment.
    e = sparse_launch<T, G, 4>(sh, a, s);
  } else {
    hipLaunchKernelGGL((k_dense_attn<T, G>), dim3(sh.n_dense_segs, sh.BHkv), dim3(kWave),
                       dense_lds_bytes(T, G), s, a);
    e = hipGetLastError();
  }
  if (e != hipSuccess) return e;
  const int parts = merge_parts(n_seg, a.BHq);
  if (parts > 1) {
    // Two levels: parts of kMergeSegsPerPart segments, then the parts.
    float2* part_ml = reinterpret_cast<float2*>(a.ws_o + (int64_t)n_seg * a.BHq * (kTile * T));
    float* part_o = reinterpret_cast<float*>(part_ml + (int64_t)parts * a.BHq);
    hipLaunchKernelGGL((k_merge<T, false>), dim3(a.BHq, parts), dim3(kMergeWaves * kWave), 0, s,
                       a.ws_ml, a.ws_o, n_seg, kMergeSegsPerPart, a.BHq, nullptr, part_ml, part_o);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((k_merge<T, true>), dim3(a.BHq, 1), dim3(kMergeWaves * kWave), 0, s, part_ml,
                       part_o, parts, parts, a.BHq, out, nullptr, nullptr);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((k_merge<T, true>), dim3(a.BHq, 1), dim3(kMergeWaves * kWave), 0, s, a.ws_ml,
                     a.ws_o, n_seg, n_seg, a.BHq, out, nullptr, nullptr);
  return hipGetLastError();
}

template <int T>
static hipError_t attention_T(const AttnShape& sh, const AttnArgs& a, uint16_t* out, hipStream_t s) {
  switch (sh.G) {
    case 1: return attention_TG<T, 1>(sh, a, out, s);
    case 2: return attention_TG<T, 2>(sh, a, out, s);
    case 4: return attention_TG<T, 4>(sh, a, out, s);
    case 8: return attention_TG<T, 8>(sh, a, out, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_attention(const AttnShape& sh, const uint16_t* q, const SparseSide& K,
                            const SparseSide& V, const uint16_t* kd, const uint16_t* vd,
                            float* ws_ml, float* ws_o, uint16_t* out, hipStream_t s) {
  const int d = kTile * sh.T;
  AttnArgs a;
  a.q = q;
  a.K = K;
  a.V = V;
  a.kd = kd;
  a.vd = vd;
  a.n_s = sh.n_s;
  a.n_dense = sh.n_dense;
  a.n_sparse_segs = sh.n_sparse_segs;
  a.sparse_seg_tokens = sh.sparse_seg_tokens;
  a.n_dense_segs = sh.n_dense_segs;
  a.dense_seg_tokens = sh.dense_seg_tokens;
  a.scale_log2 = sh.scale_log2;
  a.ws_ml = reinterpret_cast<float2*>(ws_ml);
  a.ws_o = ws_o;
  a.BHq = sh.BHkv * sh.G;
  a.kmaxK = K.bitmaps != nullptr ? token_max_elems_dev(d, K.n_keep) : 0;
  a.kmaxV = V.bitmaps != nullptr ? token_max_elems_dev(d, V.n_keep) : 0;
  switch (sh.T) {
    case 1: return attention_T<1>(sh, a, out, s);
    case 2: return attention_T<2>(sh, a, out, s);
    case 4: return attention_T<4>(sh, a, out, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mf
