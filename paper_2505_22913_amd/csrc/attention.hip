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
//
// Keys: slots pair up, so one v_dot2 (fp16 pairs, fp32 accumulation) takes two
// products; the two q values of a pair are loaded into the halves of one register.
struct KeyGroup {
  u32x4 w;
  half2_t q[4];
};

template <bool PEEL, bool HI>
__device__ __forceinline__ void key_issue(uint32_t& x, uint32_t va, uint32_t qaddr, uint32_t m,
                                          KeyGroup& k) {
  k.w = group_load<HI>(va);
#pragma unroll
  for (int u = 0; u < 8; u += 2) {
    const uint32_t c0 = next_bit<PEEL>(x, u, m);
    const uint32_t c1 = next_bit<PEEL>(x, u + 1, m);
    half2_t q;
    q.x = lds_load<_Float16>(qaddr + 2u * c0);
    q.y = lds_load<_Float16>(qaddr + 2u * c1);
    k.q[u / 2] = q;
  }
}

__device__ __forceinline__ void key_consume(const KeyGroup& k, float& acc) {
  acc = __builtin_amdgcn_fdot2(as_h2(k.w.x), k.q[0], acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(k.w.y), k.q[1], acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(k.w.z), k.q[2], acc, false);
  acc = __builtin_amdgcn_fdot2(as_h2(k.w.w), k.q[3], acc, false);
}

// One 32-channel half of a key tile (bit 31 left out, see next_bit): n groups of
// 8 from byte address a (n is the busiest lane's count, so the loop is uniform
// and every iteration issues the next group before consuming the current one);
// the upper half (HI) starts with m phantom slots.
template <bool HI>
__device__ __forceinline__ void key_half(int n, uint32_t x, uint32_t a, uint32_t qaddr, uint32_t m,
                                         float& acc) {
  if (n == 0) return;
  KeyGroup k0, k1;
  key_issue<HI, HI>(x, a, qaddr, m, k0);
  int g = 1;
  for (; g + 1 < n; g += 2) {
    key_issue<false, HI>(x, a + 16u * g, qaddr, 0u, k1);
    key_consume(k0, acc);
    key_issue<false, HI>(x, a + 16u * (g + 1), qaddr, 0u, k0);
    key_consume(k1, acc);
  }
  if (g < n) {
    key_issue<false, HI>(x, a + 16u * g, qaddr, 0u, k1);
    key_consume(k0, acc);
    key_consume(k1, acc);
  } else {
    key_consume(k0, acc);
  }
}

// Scores of one tile: q . k over its 64-bit bitmap `bm`, values at LDS byte
// address `va`. Channels 31 and 63 (bit 31 of each half) are added here from
// their ranks s - 1 and c - 1; q31 and q63 are this tile's q at those channels.
__device__ __forceinline__ void key_walk(int nlo, int nhi, uint64_t bm, uint32_t va, uint32_t q_w0,
                                         uint32_t q_w1, _Float16 q31, _Float16 q63, float& acc) {
  const uint32_t lo = (uint32_t)bm, hi = (uint32_t)(bm >> 32);
  const uint32_t s = (uint32_t)__popc(lo), c = s + (uint32_t)__popc(hi), m = s & 3u;
  const _Float16 v31 = lds_load<_Float16>(va + 2u * s - 2u);
  const _Float16 v63 = lds_load<_Float16>(va + 2u * c - 2u);
  key_half<false>(nlo, lo & kLow31, va, q_w0, 0u, acc);
  key_half<true>(nhi, hi & kLow31, va + 2u * (s - m), q_w1, m, acc);
  acc = fmaf((int)lo < 0 ? (float)q31 : 0.f, (float)v31, acc);
  acc = fmaf((int)hi < 0 ? (float)q63 : 0.f, (float)v63, acc);
}

// LDS layout of the compressed body (byte offsets). Values are expanded one
// 32-channel half at a time (both halves of every tile of the block), into a
// channel-major half tile of 32-dword rows: row `slot` (0 = the scratch slot,
// 1 + c = channel c of the half) holds, in dword t * NBH + j % NBH, token j of
// tile t (low half for the block's first NBH = NB / 2 tokens, high half for the
// others). A 32-lane pass of the scatter is then one token half, and its lanes
// write 32 different banks whatever their channels; p.V reads four dwords (eight
// tokens) of one channel per 16-byte load, with the lanes of two tiles
// interleaved and each lane's four chunks rotated by its channel, so eight
// neighbouring lanes read eight different bank groups. The half tile shares its
// bytes with the staged keys: it is cleared after the key walk of a block and
// read by p.V before the next block's keys are committed. A workgroup is one
// wave, whose LDS operations execute in program order, so the phases need no
// barrier.
struct SparseLds {
  uint32_t qtab, ps, dense, kst, vst, total;
};

constexpr int kHalfSlots = 33;
constexpr float kSlack = 8.f;  // log2 headroom of the lazy softmax base
// p is stored as fp16 for p.V; it is computed as exp2(score - base + kPBias),
// base = m_run, so that the largest p (2^(kSlack + kPBias) = 2^15) still fits
// fp16 and the small ones keep 2^kPBias more range before they flush to zero
// (fp16's smallest subnormal is 2^-24). Numerator and denominator sum the same
// rounded p; the partial's maximum is written as m_run - kPBias, so that (m, l)
// stay a consistent pair for the merge.
constexpr float kPBias = 7.f;
constexpr uint32_t kPvRow = 32;  // dwords per half-tile row (T x NBH)

// Bytes per tile of the q table: 49 dwords, so the two tiles of d = 128 sit 17
// banks apart. A half's slots span 17 dwords; the lanes of the two tiles then
// share only two banks in one key-walk load, and never on the slots that the
// walks' surplus slots read (the scratch slot and channel 31 of the half).
__host__ __device__ constexpr uint32_t qtab_stride(int G) {
  return G == 1 ? 196u : ((uint32_t)(kSlots * G * 2) + 15u) & ~15u;
}

__host__ __device__ constexpr uint32_t half_tile_bytes(int) { return kHalfSlots * kPvRow * 4u; }

__host__ __device__ inline SparseLds sparse_lds_layout(int T, int kmaxK, int kmaxV, int G = 1) {
  const int NB = kWave / T;
  SparseLds L;
  uint32_t o = 0;
  L.qtab = o;  o += (T * qtab_stride(G) + 15u) & ~15u;           // [t][slot][g] fp16
  L.ps = o;    o += (G * (NB / 2) * 4 + 15) & ~15;               // [g][j % NBH] half2
  L.vst = o;   o += (run_region_elems(NB * kmaxV) * 2 + 15) & ~15u;
  const uint32_t kst_bytes = (run_region_elems(NB * kmaxK) * 2 + 15) & ~15u;
  L.kst = o;
  L.dense = o;
  o += kst_bytes > half_tile_bytes(T) ? kst_bytes : half_tile_bytes(T);
  L.total = o;
  return L;
}

// p.V work of a lane per half: units (tile u % T, channel u / T of the half).
// With T >= 2 lane L takes units L + 64 k; with T = 1 lanes L and L + 32 share
// unit L % 32 and split its row. NQL 16-byte chunks per unit and lane.
template <int T>
struct PvUnits {
  static constexpr int UPL = T >= 2 ? T / 2 : 1;
  static constexpr int NBH = kWave / T / 2;                // dwords of one tile in a row
  static constexpr int NQL = T == 1 ? NBH / 8 : NBH / 4;
};

// Compressed segment, one head per kv-head.
template <int T, int STAGE>
__device__ __forceinline__ void sparse_body(const AttnArgs& a, int seg, int bh, unsigned char* smem,
                                            float& m_run, float& l_run, float (&o)[T]) {
  constexpr int d = kTile * T;
  constexpr int NB = kWave / T;
  using PU = PvUnits<T>;
  const SparseLds L = sparse_lds_layout(T, a.kmaxK, a.kmaxV);
  const uint32_t base = lds_addr(smem);
  const uint32_t lane = lane_id();
  const uint32_t j = lane / T, t = lane % T;

  const int j0 = seg * a.sparse_seg_tokens;
  const int j1 = min(j0 + a.sparse_seg_tokens, stream_tokens(a, bh));
  if (j0 >= j1) return;  // past this stream's tokens: an empty partial
  const int64_t kt0 = (int64_t)bh * a.K.cap_tokens * T;
  const int64_t vt0 = (int64_t)bh * a.V.cap_tokens * T;
  const uint16_t* kv = a.K.values + (int64_t)bh * a.K.val_stride;
  const uint16_t* vv = a.V.values + (int64_t)bh * a.V.val_stride;

  // q table [t][slot]: slots 0 and 33 are the scratch slots; channels 31 and
  // 63 read zero in the walks (their products are added once per tile). Every
  // load is issued before the first store (a zero slot loads channel 0 and
  // discards it), and the first block's metadata loads go out with them, so
  // that the table, this tile's q at channels 31 and 63 and the metadata cost
  // one memory round trip.
  constexpr int kQn = T * kSlots, kQr = (kQn + kWave - 1) / kWave;
  const uint16_t* qrow = a.q + (int64_t)bh * d + kTile * t;
  const _Float16 q31 = __builtin_bit_cast(_Float16, qrow[31]);
  const _Float16 q63 = __builtin_bit_cast(_Float16, qrow[63]);
  int nb = min(NB, j1 - j0);
  TileMeta cur;
  RunPos pos;
  {
    const uint16_t* qsrc = a.q + (int64_t)bh * d;
    uint16_t qv[kQr];
#pragma unroll
    for (int r = 0; r < kQr; ++r) {
      const int i = (int)lane + r * kWave;
      const int slot = i % kSlots, tt = i / kSlots;
      const int c = slot < 33 ? slot - 1 : slot - 2;
      const bool zero = i >= kQn || slot == 0 || slot == 33 || c == 31 || c == 63;
      qv[r] = qsrc[zero ? 0 : kTile * tt + c];
    }
    cur = load_meta<T>(a, kt0, vt0, j0, nb, lane);
    pos = segment_start<T>(a, kt0, vt0, j0);
#pragma unroll
    for (int r = 0; r < kQr; ++r) {
      const int i = (int)lane + r * kWave;
      const int slot = i % kSlots, tt = i / kSlots;
      const int c = slot < 33 ? slot - 1 : slot - 2;
      const bool zero = slot == 0 || slot == 33 || c == 31 || c == 63;
      uint16_t* qt = reinterpret_cast<uint16_t*>(smem + L.qtab + tt * qtab_stride(1));
      if (i < kQn) qt[slot] = zero ? (uint16_t)0 : qv[r];
    }
    // The key region follows the value region, whose last 16 bytes the commits
    // only ever fill with zeros: zero them once, so that the element before the
    // first key tile (which the channel-31 product of a tile with an empty lower
    // half reads, times 0) is never stale LDS content.
    if (lane == 0) lds_store<u32x4>(lds_addr(smem) + L.kst - 16u, (u32x4){0u, 0u, 0u, 0u});
  }

  // Prologue: block 0 staged in LDS, metadata of block 1 in flight.
  Runs rcur = runs_of(cur, pos);
  u32x4 stg[STAGE];
  stage_issue<STAGE>(stg, kv, vv, rcur, lane);
  int nb_next = min(NB, j1 - (j0 + NB));
  TileMeta nxt = {0ull, 0ull, 0u, 0u};
  if (nb_next > 0) nxt = load_meta<T>(a, kt0, vt0, j0 + NB, nb_next, lane);
  stage_commit<STAGE>(stg, base + L.kst, base + L.vst, rcur, lane);

  // Per-lane constant addresses: walks (token j, tile t) ...
  const uint32_t q_w0 = base + L.qtab + t * qtab_stride(1) + 2u;
  const uint32_t q_w1 = q_w0 + 33u * 2u;
  constexpr uint32_t NBH = PU::NBH;
  constexpr uint32_t kRowB = kPvRow * 4u;  // expanded-tile stride per channel
  const uint32_t d_w = base + L.dense + kRowB + (t * NBH + j % NBH) * 4u + (j / NBH) * 2u;
  // ... and p.V units: row start of each unit, the lane's first dword in it and
  // its chunk rotation.
  const uint32_t pv_dw0 = T == 1 ? (lane / 32u) * (NBH / 2) : 0u;
  uint32_t pv_row[PU::UPL], pv_rot[PU::UPL];
#pragma unroll
  for (int k = 0; k < PU::UPL; ++k) {
    const uint32_t u = T == 1 ? lane % 32u : lane + 64u * k;
    const uint32_t tu = u % T, c = u / T;
    pv_row[k] = base + L.dense + ((1u + c) * kPvRow + tu * NBH + pv_dw0) * 4u;
    pv_rot[k] = c;
  }
  float oh[2][PU::UPL];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int k = 0; k < PU::UPL; ++k) oh[h][k] = 0.f;
  float l_lane = 0.f;

  for (int b0 = j0; b0 < j1; b0 += NB) {
    // Software pipeline: fetch the next block's values and the metadata after it.
    const bool has_next = nb_next > 0;
    Runs rnext = {0u, 0u, 0u, 0u};
    TileMeta nxt2 = {0ull, 0ull, 0u, 0u};
    const int nb_next2 = min(NB, j1 - (b0 + 2 * NB));
    if (has_next) rnext = runs_of(nxt, pos);
    stage_issue<STAGE>(stg, kv, vv, rnext, lane);
    if (nb_next2 > 0) nxt2 = load_meta<T>(a, kt0, vt0, b0 + 2 * NB, nb_next2, lane);

    // Scores.
    const WalkCounts wc = walk_counts(cur.kb, cur.vb);
    float acc = 0.f;
    {
      const uint32_t va = base + L.kst + ((int)j < nb ? 2u * cur.ko : 0u);
      key_walk(wc.klo, wc.khi, cur.kb, va, q_w0, q_w1, q31, q63, acc);
    }
    {
      // Online softmax with a lazy base: m_run moves only when a score passes it
      // by more than kSlack, so p = exp2(score - m_run) stays below 2^kSlack
      // (well inside fp16) and most blocks need neither a wave-wide maximum nor
      // a rescale. The sum of p is kept per lane and reduced once at the end.
      const bool valid = (int)j < nb;
      const float sc = valid ? tile_sum<T>(acc) * a.scale_log2 : -INFINITY;
      if (ballot(sc > m_run + kSlack)) {
        const float mnew = fmaxf(m_run, wave_max_u(sc));
        const float alpha = __builtin_amdgcn_exp2f(m_run - mnew);
        l_lane *= alpha;
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int k = 0; k < PU::UPL; ++k) oh[h][k] *= alpha;
        m_run = mnew;
      }
      const _Float16 ph = valid ? (_Float16)__builtin_amdgcn_exp2f(sc - m_run + kPBias) : (_Float16)0.f;
      l_lane += t == 0 ? (float)ph : 0.f;
      if (t == 0) lds_store<_Float16>(base + L.ps + (j % PU::NBH) * 4 + (j / PU::NBH) * 2, ph);
    }

    // Values, one half of every tile at a time: clear the half tile (it
    // overwrites the staged keys, read above), expand, p.V.
    const uint32_t va = base + L.vst + ((int)j < nb ? 2u * cur.vo : 0u);
    const uint32_t vlo = (uint32_t)cur.vb, vhi = (uint32_t)(cur.vb >> 32);
    const uint32_t vs = (uint32_t)__popc(vlo), vm = vs & 3u;
    const _Float16 v31 = lds_load<_Float16>(va + 2u * vs - 2u);
    const _Float16 v63 = lds_load<_Float16>(va + 2u * (vs + (uint32_t)__popc(vhi)) - 2u);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      {
        // Rows 1..32 (the channels p.V reads; row 0 only takes the walks'
        // surplus writes): 32 rows of 128 bytes, four 16-byte stores per lane.
        constexpr int n16 = (int)((kHalfSlots - 1) * kPvRow * 4u / 16u);
        static_assert(n16 % kWave == 0, "whole stores per lane");
        const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int i = 0; i < n16 / kWave; ++i)
          lds_store<u32x4>(base + L.dense + kRowB + 16u * (i * kWave + lane), z);
      }
      if (h == 0) {
        value_half<false, kRowB>(wc.vlo, vlo & kLow31, va, d_w, 0u);
        lds_store<_Float16>(d_w + kRowB * 31u, (int)vlo < 0 ? v31 : (_Float16)0.f);
      } else {
        value_half<true, kRowB>(wc.vhi, vhi & kLow31, va + 2u * (vs - vm), d_w, vm);
        lds_store<_Float16>(d_w + kRowB * 31u, (int)vhi < 0 ? v63 : (_Float16)0.f);
      }
      // p.V over the lane's tokens (tokens past the block end have p = 0 and
      // zero values): per 16-byte chunk, eight tokens of p and of each unit.
      constexpr int QB = PU::NQL >= 2 ? 2 : 1;  // chunks in flight per unit
#pragma unroll 1
      for (int q0 = 0; q0 < PU::NQL; q0 += QB) {
        u32x4 p4[QB][PU::UPL], v4[QB][PU::UPL];
#pragma unroll
        for (int q = 0; q < QB; ++q)
#pragma unroll
          for (int k = 0; k < PU::UPL; ++k) {
            const uint32_t ch = ((uint32_t)(q0 + q) + pv_rot[k]) % (uint32_t)PU::NQL;
            p4[q][k] = lds_load<u32x4>(base + L.ps + (pv_dw0 + 4u * ch) * 4u);
            v4[q][k] = lds_load<u32x4>(pv_row[k] + 16u * ch);
          }
#pragma unroll
        for (int q = 0; q < QB; ++q)
#pragma unroll
          for (int k = 0; k < PU::UPL; ++k) {
            oh[h][k] = __builtin_amdgcn_fdot2(as_h2(v4[q][k].x), as_h2(p4[q][k].x), oh[h][k], false);
            oh[h][k] = __builtin_amdgcn_fdot2(as_h2(v4[q][k].y), as_h2(p4[q][k].y), oh[h][k], false);
            oh[h][k] = __builtin_amdgcn_fdot2(as_h2(v4[q][k].z), as_h2(p4[q][k].z), oh[h][k], false);
            oh[h][k] = __builtin_amdgcn_fdot2(as_h2(v4[q][k].w), as_h2(p4[q][k].w), oh[h][k], false);
          }
      }
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

  l_run = wave_sum_u(l_lane);
  m_run -= kPBias;  // l and o are sums of exp2(score - (m_run - kPBias))

  // Back to the partial layout (lane = channel of each tile): channel `lane`
  // of tile tt is channel lane % 32 of half lane / 32, unit (lane % 32) T + tt.
  const bool upper = lane >= 32u;
  const int c = (int)(lane % 32u);
#pragma unroll
  for (int tt = 0; tt < T; ++tt) {
    if constexpr (T == 1) {
      const float a0 = __shfl(oh[0][0], c, kWave) + __shfl(oh[0][0], c + 32, kWave);
      const float a1 = __shfl(oh[1][0], c, kWave) + __shfl(oh[1][0], c + 32, kWave);
      o[tt] = upper ? a1 : a0;
    } else if constexpr (T == 2) {
      const int src = c * 2 + tt;
      const float a0 = __shfl(oh[0][0], src, kWave);
      const float a1 = __shfl(oh[1][0], src, kWave);
      o[tt] = upper ? a1 : a0;
    } else {
      const int u = c * T + tt, src = u % 64;
      const bool k1 = u >= 64;
      const float a00 = __shfl(oh[0][0], src, kWave), a01 = __shfl(oh[0][1], src, kWave);
      const float a10 = __shfl(oh[1][0], src, kWave), a11 = __shfl(oh[1][1], src, kWave);
      o[tt] = upper ? (k1 ? a11 : a10) : (k1 ? a01 : a00);
    }
  }
}

// ------------------------------------------------------------------------------------------
// Grouped queries on the walks (G = 2, 4, 8 query heads per kv-head). The q
// table holds the G heads of a channel next to each other (2G bytes per slot),
// so the key walk gathers them with one load per packed key and adds
// v x q_g for every head in fp32 (mixed-precision FMA); the scores, the lazy
// softmax base and the p table are per head. The values are expanded into the
// channel-major half tile exactly as for one head, and p.V takes one v_dot2 per
// head and pair of tokens. Same staging and LDS layout as the one-head body,
// with G-wide q and p tables: no dense key tile, so about half the LDS of the
// matrix-core kernel per wave.
// ------------------------------------------------------------------------------------------
template <int GW>
struct QSlot;  // the q values of GW heads at one channel
template <>
struct QSlot<2> { typedef uint32_t type; };
template <>
struct QSlot<4> { typedef u32x2 type; };

template <int GW>
__device__ __forceinline__ float qslot_head(const typename QSlot<GW>::type& v, int g) {
  uint32_t w;
  if constexpr (GW == 2) w = v;
  else w = v[g >> 1];
  const half2_t h = as_h2(w);
  return (float)((g & 1) ? h.y : h.x);
}

template <int GW>
struct KeyGroupG {
  u32x4 w;
  typename QSlot<GW>::type q[8];
};

template <int GW, bool PEEL, bool HI>
__device__ __forceinline__ void keyg_issue(uint32_t& x, uint32_t va, uint32_t qaddr, uint32_t m,
                                           KeyGroupG<GW>& k) {
  k.w = group_load<HI>(va);
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const uint32_t c = next_bit<PEEL>(x, u, m);
    k.q[u] = lds_load<typename QSlot<GW>::type>(qaddr + (2u * GW) * c);
  }
}

template <int GW>
__device__ __forceinline__ void keyg_consume(const KeyGroupG<GW>& k, float (&acc)[GW]) {
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const float v = (float)group_value(k.w, u);
#pragma unroll
    for (int g = 0; g < GW; ++g) acc[g] = fmaf(v, qslot_head<GW>(k.q[u], g), acc[g]);
  }
}

template <int GW, bool HI>
__device__ __forceinline__ void keyg_half(int n, uint32_t x, uint32_t a, uint32_t qaddr, uint32_t m,
                                          float (&acc)[GW]) {
  if (n == 0) return;
  KeyGroupG<GW> k0, k1;
  keyg_issue<GW, HI, HI>(x, a, qaddr, m, k0);
  int g = 1;
  for (; g + 1 < n; g += 2) {
    keyg_issue<GW, false, HI>(x, a + 16u * g, qaddr, 0u, k1);
    keyg_consume<GW>(k0, acc);
    keyg_issue<GW, false, HI>(x, a + 16u * (g + 1), qaddr, 0u, k0);
    keyg_consume<GW>(k1, acc);
  }
  if (g < n) {
    keyg_issue<GW, false, HI>(x, a + 16u * g, qaddr, 0u, k1);
    keyg_consume<GW>(k0, acc);
    keyg_consume<GW>(k1, acc);
  } else {
    keyg_consume<GW>(k0, acc);
  }
}

// Scores of one tile for GW heads (q table of those heads at q_w0 / q_w1;
// q31 / q63: their q at channels 31 and 63 of the tile, as fp32).
template <int GW>
__device__ __forceinline__ void keyg_walk(int nlo, int nhi, uint64_t bm, uint32_t va, uint32_t q_w0,
                                          uint32_t q_w1, const float (&q31)[GW], const float (&q63)[GW],
                                          float (&acc)[GW]) {
  const uint32_t lo = (uint32_t)bm, hi = (uint32_t)(bm >> 32);
  const uint32_t s = (uint32_t)__popc(lo), c = s + (uint32_t)__popc(hi), m = s & 3u;
  const float v31 = (float)lds_load<_Float16>(va + 2u * s - 2u);
  const float v63 = (float)lds_load<_Float16>(va + 2u * c - 2u);
  keyg_half<GW, false>(nlo, lo & kLow31, va, q_w0, 0u, acc);
  keyg_half<GW, true>(nhi, hi & kLow31, va + 2u * (s - m), q_w1, m, acc);
#pragma unroll
  for (int g = 0; g < GW; ++g) {
    acc[g] = fmaf((int)lo < 0 ? q31[g] : 0.f, v31, acc[g]);
    acc[g] = fmaf((int)hi < 0 ? q63[g] : 0.f, v63, acc[g]);
  }
}

// Compressed segment, G query heads per kv-head (G >= 2).
template <int T, int G, int STAGE>
__device__ __forceinline__ void sparse_body_g(const AttnArgs& a, int seg, int bh, unsigned char* smem,
                                              float (&m_run)[G], float (&l_run)[G], float (&o)[G][T]) {
  constexpr int d = kTile * T;
  constexpr int NB = kWave / T;
  constexpr int GW = G < 4 ? G : 4;       // heads per key walk (G = 8 walks twice)
  constexpr uint32_t QS = 2u * GW;        // bytes per q-table slot
  using PU = PvUnits<T>;
  const SparseLds L = sparse_lds_layout(T, a.kmaxK, a.kmaxV, G);
  const uint32_t base = lds_addr(smem);
  const uint32_t lane = lane_id();
  const uint32_t j = lane / T, t = lane % T;
  constexpr uint32_t QTS = qtab_stride(GW);     // bytes per tile of one head group's table
  constexpr uint32_t QGS = T * QTS;             // bytes per head group

  const int j0 = seg * a.sparse_seg_tokens;
  const int j1 = min(j0 + a.sparse_seg_tokens, stream_tokens(a, bh));
  if (j0 >= j1) return;
  const int64_t kt0 = (int64_t)bh * a.K.cap_tokens * T;
  const int64_t vt0 = (int64_t)bh * a.V.cap_tokens * T;
  const uint16_t* kv = a.K.values + (int64_t)bh * a.K.val_stride;
  const uint16_t* vv = a.V.values + (int64_t)bh * a.V.val_stride;

  // q tables [head group][t][slot][GW heads]: slots 0 and 33 and channels 31
  // and 63 hold zeros (the walks add channels 31 and 63 from their ranks).
  // Every load is issued before the first store (a zero slot loads channel 0
  // and discards it), and the first block's metadata loads go out with them,
  // so that the tables, this tile's q at channels 31 and 63 and the metadata
  // cost one memory round trip.
  constexpr int kQn = G * T * kSlots, kQr = (kQn + kWave - 1) / kWave;
  int nb = min(NB, j1 - j0);
  TileMeta cur;
  RunPos pos;
  float q31[G], q63[G];
  {
    const uint16_t* qrow = a.q + (int64_t)bh * G * d + kTile * t;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      q31[g] = half_bits_to_float(qrow[(int64_t)g * d + 31]);
      q63[g] = half_bits_to_float(qrow[(int64_t)g * d + 63]);
    }
  }
  {
    const uint16_t* qsrc = a.q + (int64_t)bh * G * d;
    uint16_t qv[kQr];
#pragma unroll
    for (int r = 0; r < kQr; ++r) {
      const int i = (int)lane + r * kWave;
      const int gi = i % G, rest = i / G;
      const int slot = rest % kSlots, tt = rest / kSlots;
      const int c = slot < 33 ? slot - 1 : slot - 2;
      const bool zero = i >= kQn || slot == 0 || slot == 33 || c == 31 || c == 63;
      qv[r] = qsrc[zero ? 0 : gi * d + kTile * tt + c];
    }
    cur = load_meta<T>(a, kt0, vt0, j0, nb, lane);
    pos = segment_start<T>(a, kt0, vt0, j0);
#pragma unroll
    for (int r = 0; r < kQr; ++r) {
      const int i = (int)lane + r * kWave;
      const int gi = i % G, rest = i / G;
      const int slot = rest % kSlots, tt = rest / kSlots;
      const int c = slot < 33 ? slot - 1 : slot - 2;
      const bool zero = slot == 0 || slot == 33 || c == 31 || c == 63;
      uint16_t* qt = reinterpret_cast<uint16_t*>(smem + L.qtab + (gi / GW) * QGS + tt * QTS + slot * QS);
      if (i < kQn) qt[gi % GW] = zero ? (uint16_t)0 : qv[r];
    }
    if (lane == 0) lds_store<u32x4>(lds_addr(smem) + L.kst - 16u, (u32x4){0u, 0u, 0u, 0u});
  }

  Runs rcur = runs_of(cur, pos);
  u32x4 stg[STAGE];
  stage_issue<STAGE>(stg, kv, vv, rcur, lane);
  int nb_next = min(NB, j1 - (j0 + NB));
  TileMeta nxt = {0ull, 0ull, 0u, 0u};
  if (nb_next > 0) nxt = load_meta<T>(a, kt0, vt0, j0 + NB, nb_next, lane);
  stage_commit<STAGE>(stg, base + L.kst, base + L.vst, rcur, lane);

  const uint32_t q_w0 = base + L.qtab + t * QTS + QS;   // slot 1: channel 0 of the tile
  const uint32_t q_w1 = q_w0 + 33u * QS;
  constexpr uint32_t NBH = PU::NBH;
  constexpr uint32_t kRowB = kPvRow * 4u;
  const uint32_t d_w = base + L.dense + kRowB + (t * NBH + j % NBH) * 4u + (j / NBH) * 2u;
  const uint32_t pv_dw0 = T == 1 ? (lane / 32u) * (NBH / 2) : 0u;
  uint32_t pv_row[PU::UPL], pv_rot[PU::UPL];
#pragma unroll
  for (int k = 0; k < PU::UPL; ++k) {
    const uint32_t u = T == 1 ? lane % 32u : lane + 64u * k;
    const uint32_t tu = u % T, c = u / T;
    pv_row[k] = base + L.dense + ((1u + c) * kPvRow + tu * NBH + pv_dw0) * 4u;
    pv_rot[k] = c;
  }
  constexpr uint32_t PSG = NBH * 4u;   // bytes of one head's p table
  float oh[G][2][PU::UPL];
  float l_lane[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    l_lane[g] = 0.f;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int k = 0; k < PU::UPL; ++k) oh[g][hh][k] = 0.f;
  }

  for (int b0 = j0; b0 < j1; b0 += NB) {
    const bool has_next = nb_next > 0;
    Runs rnext = {0u, 0u, 0u, 0u};
    TileMeta nxt2 = {0ull, 0ull, 0u, 0u};
    const int nb_next2 = min(NB, j1 - (b0 + 2 * NB));
    if (has_next) rnext = runs_of(nxt, pos);
    stage_issue<STAGE>(stg, kv, vv, rnext, lane);
    if (nb_next2 > 0) nxt2 = load_meta<T>(a, kt0, vt0, b0 + 2 * NB, nb_next2, lane);

    // Scores of every head.
    const WalkCounts wc = walk_counts(cur.kb, cur.vb);
    float acc[G];
    {
      const uint32_t va = base + L.kst + ((int)j < nb ? 2u * cur.ko : 0u);
#pragma unroll
      for (int g0 = 0; g0 < G; g0 += GW) {
        float ag[GW], a31[GW], a63[GW];
#pragma unroll
        for (int g = 0; g < GW; ++g) {
          ag[g] = 0.f;
          a31[g] = q31[g0 + g];
          a63[g] = q63[g0 + g];
        }
        keyg_walk<GW>(wc.klo, wc.khi, cur.kb, va, q_w0 + (uint32_t)(g0 / GW) * QGS,
                      q_w1 + (uint32_t)(g0 / GW) * QGS, a31, a63, ag);
#pragma unroll
        for (int g = 0; g < GW; ++g) acc[g0 + g] = ag[g];
      }
    }
    // Online softmax per head with the lazy base of the one-head body; p as fp16
    // with the exponent bias, the two token halves of the block in one dword.
    {
      const bool valid = (int)j < nb;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float sc = valid ? tile_sum<T>(acc[g]) * a.scale_log2 : -INFINITY;
        if (ballot(sc > m_run[g] + kSlack)) {
          const float mnew = fmaxf(m_run[g], wave_max_u(sc));
          const float alpha = __builtin_amdgcn_exp2f(m_run[g] - mnew);
          l_lane[g] *= alpha;
#pragma unroll
          for (int hh = 0; hh < 2; ++hh)
#pragma unroll
            for (int k = 0; k < PU::UPL; ++k) oh[g][hh][k] *= alpha;
          m_run[g] = mnew;
        }
        const _Float16 ph = valid ? (_Float16)__builtin_amdgcn_exp2f(sc - m_run[g] + kPBias) : (_Float16)0.f;
        l_lane[g] += t == 0 ? (float)ph : 0.f;
        if (t == 0) lds_store<_Float16>(base + L.ps + g * PSG + (j % NBH) * 4 + (j / NBH) * 2, ph);
      }
    }

    // Values, one half of every tile at a time, as in the one-head body.
    const uint32_t va = base + L.vst + ((int)j < nb ? 2u * cur.vo : 0u);
    const uint32_t vlo = (uint32_t)cur.vb, vhi = (uint32_t)(cur.vb >> 32);
    const uint32_t vs = (uint32_t)__popc(vlo), vm = vs & 3u;
    const _Float16 v31 = lds_load<_Float16>(va + 2u * vs - 2u);
    const _Float16 v63 = lds_load<_Float16>(va + 2u * (vs + (uint32_t)__popc(vhi)) - 2u);
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      {
        // Rows 1..32 (the channels p.V reads; row 0 only takes the walks'
        // surplus writes): 32 rows of 128 bytes, four 16-byte stores per lane.
        constexpr int n16 = (int)((kHalfSlots - 1) * kPvRow * 4u / 16u);
        static_assert(n16 % kWave == 0, "whole stores per lane");
        const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int i = 0; i < n16 / kWave; ++i)
          lds_store<u32x4>(base + L.dense + kRowB + 16u * (i * kWave + lane), z);
      }
      if (hh == 0) {
        value_half<false, kRowB>(wc.vlo, vlo & kLow31, va, d_w, 0u);
        lds_store<_Float16>(d_w + kRowB * 31u, (int)vlo < 0 ? v31 : (_Float16)0.f);
      } else {
        value_half<true, kRowB>(wc.vhi, vhi & kLow31, va + 2u * (vs - vm), d_w, vm);
        lds_store<_Float16>(d_w + kRowB * 31u, (int)vhi < 0 ? v63 : (_Float16)0.f);
      }
      // p.V for every head: one chunk (eight tokens) of values per unit, then the
      // same chunk of each head's p.
#pragma unroll 1
      for (int q0 = 0; q0 < PU::NQL; ++q0) {
        u32x4 v4[PU::UPL];
        uint32_t ch[PU::UPL];
#pragma unroll
        for (int k = 0; k < PU::UPL; ++k) {
          ch[k] = ((uint32_t)q0 + pv_rot[k]) % (uint32_t)PU::NQL;
          v4[k] = lds_load<u32x4>(pv_row[k] + 16u * ch[k]);
        }
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
          for (int k = 0; k < PU::UPL; ++k) {
            const u32x4 p4 = lds_load<u32x4>(base + L.ps + g * PSG + (pv_dw0 + 4u * ch[k]) * 4u);
            float r = oh[g][hh][k];
            r = __builtin_amdgcn_fdot2(as_h2(v4[k].x), as_h2(p4.x), r, false);
            r = __builtin_amdgcn_fdot2(as_h2(v4[k].y), as_h2(p4.y), r, false);
            r = __builtin_amdgcn_fdot2(as_h2(v4[k].z), as_h2(p4.z), r, false);
            r = __builtin_amdgcn_fdot2(as_h2(v4[k].w), as_h2(p4.w), r, false);
            oh[g][hh][k] = r;
          }
      }
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

  const bool upper = lane >= 32u;
  const int c = (int)(lane % 32u);
#pragma unroll
  for (int g = 0; g < G; ++g) {
    l_run[g] = wave_sum_u(l_lane[g]);
    m_run[g] -= kPBias;
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
      if constexpr (T == 1) {
        const float a0 = __shfl(oh[g][0][0], c, kWave) + __shfl(oh[g][0][0], c + 32, kWave);
        const float a1 = __shfl(oh[g][1][0], c, kWave) + __shfl(oh[g][1][0], c + 32, kWave);
        o[g][tt] = upper ? a1 : a0;
      } else if constexpr (T == 2) {
        const int src = c * 2 + tt;
        const float a0 = __shfl(oh[g][0][0], src, kWave);
        const float a1 = __shfl(oh[g][1][0], src, kWave);
        o[g][tt] = upper ? a1 : a0;
      } else {
        const int u = c * T + tt, src = u % 64;
        const bool k1 = u >= 64;
        const float a00 = __shfl(oh[g][0][0], src, kWave), a01 = __shfl(oh[g][0][1], src, kWave);
        const float a10 = __shfl(oh[g][1][0], src, kWave), a11 = __shfl(oh[g][1][1], src, kWave);
        o[g][tt] = upper ? (k1 ? a11 : a10) : (k1 ? a01 : a00);
      }
    }
  }
}

// Sparse call: grid (n_sparse_segs + n_dense_segs, BHkv); compressed segments first.
template <int T, int G, int STAGE>
__global__ __launch_bounds__(64) void k_sparse_attn(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int seg = blockIdx.x, bh = blockIdx.y;
  float m_run[G], l_run[G], o[G][T];
  init_state<T, G>(m_run, l_run, o);
  if (seg < a.n_sparse_segs) {
    if constexpr (G == 1) sparse_body<T, STAGE>(a, seg, bh, smem, m_run[0], l_run[0], o[0]);
    else sparse_body_g<T, G, STAGE>(a, seg, bh, smem, m_run, l_run, o);
  } else {
    dense_body<T, G>(a, seg - a.n_sparse_segs, bh, smem, m_run, l_run, o);
  }
  write_partial<T, G>(a, seg, bh, m_run, l_run, o);
}

// Dense baseline: grid (n_dense_segs, BHkv).
template <int T, int G>
__global__ __launch_bounds__(64) void k_dense_attn(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int seg = blockIdx.x, bh = blockIdx.y;
  float m_run[G], l_run[G], o[G][T];
  init_state<T, G>(m_run, l_run, o);
  dense_body<T, G, false>(a, seg, bh, smem, m_run, l_run, o);
  write_partial<T, G>(a, seg, bh, m_run, l_run, o);
}

// grid (BHq, parts), 8 waves: log-sum-exp merge of segments [part * per,
// part * per + per) of one query head. Wave w takes segments w, w + 8, ...,
// kMergeChunk at a time with every load of a chunk issued before the first is
// used (lane = channel), and keeps a running (max, sum, weighted output) over
// them; LDS then combines the eight waves' states. With FINAL the result is
// divided by the sum and written as fp16 (RNE); otherwise (max, sum,
// unnormalised output) is written as one segment of a second, shorter merge --
// used when there are many segments and few query heads, so that the merge runs
// on many workgroups instead of one per head.
constexpr int kMergeWaves = 8;
constexpr int kMergeChunk = 16;
constexpr int kMergeSegsPerPart = 32;

template <int T, bool FINAL>
__global__ __launch_bounds__(kMergeWaves * kWave) void k_merge(const float2* __restrict__ ws_ml,
                                                              const float* __restrict__ ws_o,
                                                              int n_seg, int per, int BHq,
                                                              uint16_t* __restrict__ out,
                                                              float2* __restrict__ part_ml,
                                                              float* __restrict__ part_o,
                                                              float* __restrict__ lse2) {
  constexpr int d = kTile * T;
  __shared__ float wm[kMergeWaves], wl[kMergeWaves];
  __shared__ float part[kMergeWaves][d];
  const int r = blockIdx.x;
  const int s0 = blockIdx.y * per, s1 = min(n_seg, s0 + per);
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const uint32_t lane = lane_id();
  float m = -INFINITY, l = 0.f, acc[T];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) acc[tt] = 0.f;
  for (int c0 = s0 + wave; c0 < s1; c0 += kMergeChunk * kMergeWaves) {
    // Lane k < kMergeChunk loads (max, sum) of the chunk's segment k; every lane
    // loads its channel of each segment's output. Segments past the range load
    // the first one again and weigh 0.
    const int sk = c0 + (int)(lane % kMergeChunk) * kMergeWaves;
    const bool lv = lane < (uint32_t)kMergeChunk && sk < s1;
    const float2 mlv = ws_ml[(int64_t)(lv ? sk : s0) * BHq + r];
    float ov[kMergeChunk][T];
#pragma unroll
    for (int k = 0; k < kMergeChunk; ++k) {
      const int s = c0 + k * kMergeWaves < s1 ? c0 + k * kMergeWaves : s0;
      const float* o = ws_o + ((int64_t)s * BHq + r) * d + lane;
#pragma unroll
      for (int tt = 0; tt < T; ++tt) ov[k][tt] = o[kTile * tt];
    }
    const float xv = lv ? mlv.x : -INFINITY;
    const float cm = fmaxf(m, wave_max_u(xv));
    // Rescale the running state to the new maximum (m = -inf gives 0; with no
    // segment seen yet the state is empty and stays so).
    const float sr = cm == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m - cm);
    const float wv = xv == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(xv - cm);
    l = fmaf(l, sr, wave_sum_u(wv * mlv.y));
#pragma unroll
    for (int tt = 0; tt < T; ++tt) acc[tt] *= sr;
#pragma unroll
    for (int k = 0; k < kMergeChunk; ++k) {
      const float w = readlane_f(wv, k);
#pragma unroll
      for (int tt = 0; tt < T; ++tt) acc[tt] = fmaf(ov[k][tt], w, acc[tt]);
    }
    m = cm;
  }
  if (lane == 0) {
    wm[wave] = m;
    wl[wave] = l;
  }
#pragma unroll
  for (int tt = 0; tt < T; ++tt) part[wave][lane + kTile * tt] = acc[tt];
  __syncthreads();
  if (wave == 0) {
    float M = wm[0];
#pragma unroll
    for (int w = 1; w < kMergeWaves; ++w) M = fmaxf(M, wm[w]);
    float sw[kMergeWaves], L = 0.f;
#pragma unroll
    for (int w = 0; w < kMergeWaves; ++w) {
      sw[w] = wm[w] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(wm[w] - M);
      L = fmaf(wl[w], sw[w], L);
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;  // no token at all (every stream skipped): 0
    const int64_t prow = (int64_t)blockIdx.y * BHq + r;
    if (!FINAL && lane == 0) part_ml[prow] = make_float2(M, L);
    if (FINAL && lse2 != nullptr && lane == 0) lse2[r] = M + __builtin_log2f(L);
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
      float v = 0.f;
#pragma unroll
      for (int w = 0; w < kMergeWaves; ++w) v = fmaf(part[w][lane + kTile * tt], sw[w], v);
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
  size_t lds = sh.n_sparse_segs > 0 ? sparse_lds_layout(T, a.kmaxK, a.kmaxV, G).total : 0;
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
    // Grouped queries contract on the matrix cores (attention_mfma.hip) when
    // the route says so (by default from kMfmaMinGroup heads per kv-head on).
    if constexpr (G >= 2) {
      if (sh.mfma) e = launch_sparse_mfma(sh, a, s);
      else e = sparse_stage<T, G>(sh, a, s);
    } else {
      e = sparse_stage<T, G>(sh, a, s);
    }
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
                       a.ws_ml, a.ws_o, n_seg, kMergeSegsPerPart, a.BHq, nullptr, part_ml, part_o, nullptr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((k_merge<T, true>), dim3(a.BHq, 1), dim3(kMergeWaves * kWave), 0, s, part_ml,
                       part_o, parts, parts, a.BHq, out, nullptr, nullptr, a.lse2);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((k_merge<T, true>), dim3(a.BHq, 1), dim3(kMergeWaves * kWave), 0, s, a.ws_ml,
                     a.ws_o, n_seg, n_seg, a.BHq, out, nullptr, nullptr, a.lse2);
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
  a.kmaxK = side_token_bound(d, K, kWave / sh.T);  // the walk kernel's blocks (the MFMA
  a.kmaxV = side_token_bound(d, V, kWave / sh.T);  // kernel sets its own)
  a.n_comp = sh.n_comp;
  a.win_len = sh.win_len;
  a.win_head = sh.win_head;
  a.Hkv = sh.Hkv;
  a.lse2 = sh.lse2;
  switch (sh.T) {
    case 1: return attention_T<1>(sh, a, out, s);
    case 2: return attention_T<2>(sh, a, out, s);
    case 4: return attention_T<4>(sh, a, out, s);
    default: return hipErrorInvalidValue;
  }
}

// ------------------------------------------------------------------------------------------
// Output-aware scores of per-channel value pruning (Sec. 2): the attention
// probability of every window token younger than 32 steps, summed over the G
// query heads of its kv-head and added to its slot's score. One wave per
// (batch entry, kv-head), lane = window position; q staged in LDS (every lane
// reads the same address, a broadcast). An entry that is not active in this
// step gathers nothing.
// ------------------------------------------------------------------------------------------
constexpr int kScoreSteps = 32;  // steps a token's score accumulates (the current and 31 more)

template <int T, int G>
__global__ __launch_bounds__(kWave) void k_window_scores(WindowView w, const uint16_t* __restrict__ q,
                                                         float scale_log2, const float* __restrict__ lse2,
                                                         const int32_t* __restrict__ active,
                                                         float* __restrict__ acc) {
  constexpr int d = kTile * T;
  __shared__ __attribute__((aligned(16))) uint16_t qs[G * d];
  const int bh = blockIdx.x;
  const int b = bh / w.H;
  if (active != nullptr && active[b] == 0) return;  // uniform over the workgroup
  const uint32_t lane = lane_id();
  for (int i = (int)lane; i < G * d; i += kWave) qs[i] = q[(int64_t)bh * G * d + i];
  __syncthreads();
  const int len = w.len[b], head = w.head[b];
  if (len <= 0 || len > w.W || head < 0 || head >= w.W) return;
  float lse[G];
#pragma unroll
  for (int g = 0; g < G; ++g) lse[g] = lse2[(int64_t)bh * G + g];
  const int p = max(0, len - kScoreSteps) + (int)lane;
  if (p >= len) return;
  const int slot = (head + p) % w.W;
  const uint16_t* kr = w.k + ((int64_t)bh * w.W + slot) * d;
  float s[G];
#pragma unroll
  for (int g = 0; g < G; ++g) s[g] = 0.f;
#pragma unroll 4
  for (int c = 0; c < d; c += 8) {
    const u32x4 kk = *reinterpret_cast<const u32x4*>(kr + c);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const u32x4 qq = *reinterpret_cast<const u32x4*>(qs + g * d + c);
      s[g] = __builtin_amdgcn_fdot2(as_h2(kk.x), as_h2(qq.x), s[g], false);
      s[g] = __builtin_amdgcn_fdot2(as_h2(kk.y), as_h2(qq.y), s[g], false);
      s[g] = __builtin_amdgcn_fdot2(as_h2(kk.z), as_h2(qq.z), s[g], false);
      s[g] = __builtin_amdgcn_fdot2(as_h2(kk.w), as_h2(qq.w), s[g], false);
    }
  }
  float sum = 0.f;
#pragma unroll
  for (int g = 0; g < G; ++g) sum += __builtin_amdgcn_exp2f(fmaf(s[g], scale_log2, -lse[g]));
  acc[(int64_t)bh * w.W + slot] += sum;
}

template <int T>
static hipError_t window_scores_T(const WindowView& w, const uint16_t* q, int G, float scale_log2,
                                  const float* lse2, const int32_t* active, float* acc, hipStream_t s) {
  const dim3 grid((uint32_t)(w.B * w.H));
  switch (G) {
    case 1: hipLaunchKernelGGL((k_window_scores<T, 1>), grid, dim3(kWave), 0, s, w, q, scale_log2, lse2, active, acc); break;
    case 2: hipLaunchKernelGGL((k_window_scores<T, 2>), grid, dim3(kWave), 0, s, w, q, scale_log2, lse2, active, acc); break;
    case 4: hipLaunchKernelGGL((k_window_scores<T, 4>), grid, dim3(kWave), 0, s, w, q, scale_log2, lse2, active, acc); break;
    case 8: hipLaunchKernelGGL((k_window_scores<T, 8>), grid, dim3(kWave), 0, s, w, q, scale_log2, lse2, active, acc); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_window_scores(const WindowView& w, const uint16_t* q, int G, int T, float scale_log2,
                                const float* lse2, const int32_t* active, float* acc, hipStream_t s) {
  switch (T) {
    case 1: return window_scores_T<1>(w, q, G, scale_log2, lse2, active, acc, s);
    case 2: return window_scores_T<2>(w, q, G, scale_log2, lse2, active, acc, s);
    case 4: return window_scores_T<4>(w, q, G, scale_log2, lse2, active, acc, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mf
