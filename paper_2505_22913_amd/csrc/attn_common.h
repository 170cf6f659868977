// Device helpers shared by the decode-attention kernels (attention.hip: the
// bit-walk kernel, one or grouped query heads; attention_mfma.hip: the MFMA
// kernel for grouped queries):
// types, wave reductions, LDS access, the staging of compressed blocks, the
// bit-walk primitives, the dense (window) segment body and the partial-result
// writes of the split-K scheme.
#pragma once

#include "mf_device.h"
#include "mf_launch.h"

namespace mf {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Reinterpret 32 bits as two fp16. Takes the word BY VALUE: __builtin_bit_cast
// applied directly to an ext-vector element (w.y) reinterprets element 0.
__device__ __forceinline__ half2_t as_h2(uint32_t w) { return __builtin_bit_cast(half2_t, w); }

// Per tile and per 32-channel half, one scratch slot precedes the channels:
// [s][ch 0..31][s][ch 32..63] -- slot of channel c is 1 + c + (c >= 32).
constexpr int kSlots = 66;

// Zero fp16 values staged after each packed run (a multiple of 8).
constexpr uint32_t kMargin = 80;

struct AttnArgs {
  const uint16_t* q;
  SparseSide K, V;
  const uint16_t* kd;  // dense keys   [BHkv][n_dense][d]
  const uint16_t* vd;  // dense values [BHkv][n_dense][d]
  int n_s, n_dense;
  int n_sparse_segs, sparse_seg_tokens;
  int n_dense_segs, dense_seg_tokens;
  float scale_log2;
  float2* ws_ml;
  float* ws_o;
  int BHq;
  int kmaxK, kmaxV;  // worst-case fp16 elements per token of each cache
  // Per-batch-entry lengths, null for uniform streams (see AttnShape).
  const int32_t* n_comp;
  const int32_t* win_len;
  const int32_t* win_head;
  int Hkv;
  float* lse2;  // optional: the final merge writes m + log2(l) per query head
};

// Compressed tokens of stream bh (its batch entry's count when ragged); none
// when a bulk compression gave up on the stream (its offsets have holes).
__device__ __forceinline__ int stream_tokens(const AttnArgs& a, int bh) {
  if (a.K.stream_len[bh] == kStreamPoisoned || a.V.stream_len[bh] == kStreamPoisoned) return 0;
  return a.n_comp ? min(a.n_comp[bh / a.Hkv], a.n_s) : a.n_s;
}

__device__ __forceinline__ uint32_t ffbl(uint32_t x) {  // 0xffffffff when x == 0
  uint32_t r;
  asm("v_ffbl_b32 %0, %1" : "=v"(r) : "v"(x));
  return r;
}

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float swz_xor16(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));
}

__device__ __forceinline__ float readlane_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}

// Max / sum over all 64 lanes, returned wave-uniform: DPP within 16-lane rows,
// a swizzle across row pairs, then the two 32-lane halves.
__device__ __forceinline__ float wave_max_u(float v) {
  v = fmaxf(v, dpp<0xB1>(v));   // quad_perm [1,0,3,2]
  v = fmaxf(v, dpp<0x4E>(v));   // quad_perm [2,3,0,1]
  v = fmaxf(v, dpp<0x124>(v));  // row_ror:4
  v = fmaxf(v, dpp<0x128>(v));  // row_ror:8
  v = fmaxf(v, swz_xor16(v));
  return fmaxf(readlane_f(v, 0), readlane_f(v, 32));
}

__device__ __forceinline__ float wave_sum_u(float v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x124>(v);
  v += dpp<0x128>(v);
  v += swz_xor16(v);
  return readlane_f(v, 0) + readlane_f(v, 32);
}

// Sum over the T lanes (adjacent, T in {1,2,4}) that hold the tiles of one token.
template <int T>
__device__ __forceinline__ float tile_sum(float v) {
  if constexpr (T >= 2) v += dpp<0xB1>(v);
  if constexpr (T >= 4) v += dpp<0x4E>(v);
  return v;
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)p;
}

template <typename V>
__device__ __forceinline__ V lds_load(uint32_t byte_addr) {
  return *reinterpret_cast<const __attribute__((address_space(3))) V*>(byte_addr);
}

template <typename V>
__device__ __forceinline__ void lds_store(uint32_t byte_addr, V v) {
  *reinterpret_cast<__attribute__((address_space(3))) V*>(byte_addr) = v;
}

// ------------------------------------------------------------------------------------------
// Dense segment body: the local window of the sparse call, or a range of a dense cache.
// ------------------------------------------------------------------------------------------
// RING: the segment may be a ring window (win_len set) whose unused slots are
// skipped; the dense baseline's segments are plain (RING false).
template <int T, int G, bool RING = true>
__device__ __forceinline__ void dense_body(const AttnArgs& a, int dseg, int bh, unsigned char* smem,
                                           float (&m_run)[G], float (&l_run)[G],
                                           float (&o)[G][T]) {
  constexpr int d = kTile * T;
  constexpr int NB = kWave / T;
  uint16_t* qs = reinterpret_cast<uint16_t*>(smem);           // [G][d]
  float* ps = reinterpret_cast<float*>(smem + G * d * 2);     // [NB][G]
  const uint32_t lane = lane_id();
  const uint32_t j = lane / T, t = lane % T;
  const uint16_t* qsrc = a.q + (int64_t)bh * G * d;
  for (int i = lane; i < G * d; i += kWave) qs[i] = qsrc[i];
  __syncthreads();

  const int j0 = dseg * a.dense_seg_tokens;
  const int j1 = min(j0 + a.dense_seg_tokens, a.n_dense);
  const uint16_t* kd = a.kd + (int64_t)bh * a.n_dense * d;
  const uint16_t* vd = a.vd + (int64_t)bh * a.n_dense * d;
  // A ring window holds win_len tokens from slot win_head on; its other slots
  // are skipped (their contents are arbitrary).
  const bool ring = RING && a.win_len != nullptr;
  const int w_len = ring ? a.win_len[bh / a.Hkv] : a.n_dense;
  const int w_head = ring ? a.win_head[bh / a.Hkv] : 0;
  for (int b0 = j0; b0 < j1; b0 += NB) {
    const int nb = min(NB, j1 - b0);
    const int rel = b0 + (int)j - w_head;  // age rank of the slot's token (ring), or its index
    const bool valid = (int)j < nb && (!RING || (rel < 0 ? rel + a.n_dense : rel) < w_len);
    float acc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g] = 0.f;
    if (valid) {
      const u32x4* kr = reinterpret_cast<const u32x4*>(kd + (int64_t)(b0 + (int)j) * d + kTile * t);
#pragma unroll
      for (int i = 0; i < kTile / 8; ++i) {
        const u32x4 u = kr[i];
        const half2_t k2[4] = {as_h2(u.x), as_h2(u.y),
                               as_h2(u.z), as_h2(u.w)};
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const uint4 qq = *reinterpret_cast<const uint4*>(qs + g * d + kTile * t + 8 * i);
          acc[g] = __builtin_amdgcn_fdot2(k2[0], as_h2(qq.x), acc[g], false);
          acc[g] = __builtin_amdgcn_fdot2(k2[1], as_h2(qq.y), acc[g], false);
          acc[g] = __builtin_amdgcn_fdot2(k2[2], as_h2(qq.z), acc[g], false);
          acc[g] = __builtin_amdgcn_fdot2(k2[3], as_h2(qq.w), acc[g], false);
        }
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float sc = valid ? tile_sum<T>(acc[g]) * a.scale_log2 : -INFINITY;
      const float mnew = fmaxf(m_run[g], wave_max_u(sc));
      const float alpha = __builtin_amdgcn_exp2f(m_run[g] - mnew);
      const float pj = valid ? __builtin_amdgcn_exp2f(sc - mnew) : 0.f;
      l_run[g] = l_run[g] * alpha + wave_sum_u(t == 0 ? pj : 0.f);
      m_run[g] = mnew;
#pragma unroll
      for (int tt = 0; tt < T; ++tt) o[g][tt] *= alpha;
      // Every slot's p is stored (0 for a skipped ring slot): the p.V loop below
      // reads all of the block's slots, and LDS left by an earlier workgroup may
      // hold non-finite bits.
      if (t == 0) ps[j * G + g] = pj;
    }
    __syncthreads();
#pragma unroll 8
    for (int jj = 0; jj < nb; ++jj) {
      float pv[G];
#pragma unroll
      for (int g = 0; g < G; ++g) pv[g] = ps[jj * G + g];
      const uint16_t* vr = vd + (int64_t)(b0 + jj) * d;
      // Skipped ring slots have p = 0 and may hold non-finite bits: read as 0.
      // Every slot is loaded (all lie inside the window buffer) and the skipped
      // ones are dropped after the load, so the loads of successive tokens
      // need not wait for each other.
      const int rj = b0 + jj - w_head;
      const bool live = !RING || (rj < 0 ? rj + a.n_dense : rj) < w_len;
#pragma unroll
      for (int tt = 0; tt < T; ++tt) {
        const float vl = half_bits_to_float(vr[lane + kTile * tt]);
        const float v = live ? vl : 0.f;
#pragma unroll
        for (int g = 0; g < G; ++g) o[g][tt] = fmaf(pv[g], v, o[g][tt]);
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------------------------------
// Compressed segment body.
// ------------------------------------------------------------------------------------------
struct TileMeta {
  uint64_t kb, vb;  // this lane's key / value tile bitmaps (0 past the block end)
  uint32_t ko, vo;  // their offsets from the block's first tile (set by runs_of)
};

// Bitmaps of the block of nb tokens from token b0. The tile offsets are not
// read: a stream's tiles are packed back to back in token order, each taking
// its count padded to 8, so runs_of derives them from the bitmaps.
template <int T>
__device__ __forceinline__ TileMeta load_meta(const AttnArgs& a, int64_t kt0, int64_t vt0, int b0,
                                              int nb, uint32_t lane) {
  TileMeta m = {0ull, 0ull, 0u, 0u};
  if ((int)(lane / T) < nb) {
    const int64_t ti = (int64_t)b0 * T + lane;
    m.kb = __builtin_nontemporal_load(&a.K.bitmaps[kt0 + ti]);
    m.vb = __builtin_nontemporal_load(&a.V.bitmaps[vt0 + ti]);
  }
  return m;
}

// Stream positions (fp16 elements) where the next block's key and value runs
// start: the offsets of the segment's first tiles, then advanced by runs_of.
struct RunPos {
  uint32_t k, v;
};

template <int T>
__device__ __forceinline__ RunPos segment_start(const AttnArgs& a, int64_t kt0, int64_t vt0, int j0) {
  RunPos p;
  p.k = (uint32_t)__builtin_amdgcn_readfirstlane((int)a.K.offsets[kt0 + (int64_t)j0 * T]);
  p.v = (uint32_t)__builtin_amdgcn_readfirstlane((int)a.V.offsets[vt0 + (int64_t)j0 * T]);
  return p;
}

// Packed-value runs of one block: [kstart, kstart + kn) and [vstart, vstart + vn).
struct Runs {
  uint32_t kstart, kn, vstart, vn;
};

// The block's runs and its tiles' offsets: an exclusive wave scan of the
// padded tile counts (tiles past the block end count 0); the run starts at pos,
// which then moves to the next block's run.
__device__ __forceinline__ Runs runs_of(TileMeta& m, RunPos& pos) {
  const uint32_t ck = pad8((uint32_t)__popcll(m.kb)), cv = pad8((uint32_t)__popcll(m.vb));
  const uint32_t ik = wave_incl_scan(ck), iv = wave_incl_scan(cv);
  m.ko = ik - ck;
  m.vo = iv - cv;
  Runs r;
  r.kstart = pos.k;
  r.vstart = pos.v;
  r.kn = (uint32_t)__builtin_amdgcn_readlane((int)ik, kWave - 1);
  r.vn = (uint32_t)__builtin_amdgcn_readlane((int)iv, kWave - 1);
  pos.k += r.kn;
  pos.v += r.vn;
  return r;
}

// Staging chunks: 512 fp16 values, one 16-byte load per lane. A run of n
// values needs ceil(n / 512) chunks; its LDS region holds whole chunks.
constexpr uint32_t kChunk = 512;

__host__ __device__ inline uint32_t run_region_elems(uint32_t max_run) {
  const uint32_t whole = (max_run + kChunk - 1) / kChunk * kChunk;
  const uint32_t need = max_run + kMargin;
  return whole > need ? whole : need;
}

// Raw buffer descriptor (gfx9 word 3) over `elems` fp16 values at p: a load
// past the end returns zeros and reads no memory.
// The arguments are wave-uniform; readfirstlane states it, so the descriptor
// stays in scalar registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t run_rsrc_at(uint64_t a, uint32_t elems) {
  const uint64_t u = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(a >> 32)) << 32) |
                     (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  const int bytes = __builtin_amdgcn_readfirstlane((int)(elems * 2u));
  return __builtin_amdgcn_make_buffer_rsrc(reinterpret_cast<void*>(u), (short)0, bytes, 0x00020000);
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t run_rsrc(const uint16_t* p, uint32_t elems) {
  return run_rsrc_at((uint64_t)(uintptr_t)p, elems);
}

constexpr int kLoadNT = 2;  // non-temporal: the compressed streams are read once per call

// Slot c holds chunk c of the block's key run for c < nck, else chunk c - nck
// of its value run. Every slot is loaded (no divergent register writes), at
// byte offset 16 lane + 1 KiB c of one of two descriptors: the key run's, and
// one that starts nck chunks before the value run and spans those chunks too,
// so that the same slot offsets land on the value chunks. The hardware bounds
// each load by its descriptor's size, immediate and scalar offsets included,
// so the lanes past a run's end get zeros and read no memory.
template <int STAGE>
__device__ __forceinline__ void stage_issue(u32x4 (&r)[STAGE], const uint16_t* kv, const uint16_t* vv,
                                            const Runs& rn, uint32_t lane) {
  const uint32_t nck = (rn.kn + kChunk - 1) / kChunk;
  const __amdgpu_buffer_rsrc_t rk = run_rsrc(kv + rn.kstart, rn.kn);
  const __amdgpu_buffer_rsrc_t rv =
      run_rsrc_at((uint64_t)(uintptr_t)(vv + rn.vstart) - 2ull * kChunk * nck, rn.vn + kChunk * nck);
#pragma unroll
  for (int c = 0; c < STAGE; ++c)
    r[c] = __builtin_amdgcn_raw_buffer_load_b128((uint32_t)c < nck ? rk : rv, 16u * lane,
                                                 2u * kChunk * (uint32_t)c, kLoadNT);
}

// Whole chunks go to LDS (zeros past each run's end), then kMargin zeros after
// each run: the walks read whole groups of 8 up to 72 values past the start of
// a tile (at most 4 groups of the lower half and 5 of the upper half, which
// starts at most 32 values in), and the products of those values with the zero
// q slot must stay 0.
template <int STAGE>
__device__ __forceinline__ void stage_commit(const u32x4 (&r)[STAGE], uint32_t kst, uint32_t vst,
                                             const Runs& rn, uint32_t lane) {
  const uint32_t nck = (rn.kn + kChunk - 1) / kChunk, nvc = (rn.vn + kChunk - 1) / kChunk;
#pragma unroll
  for (int c = 0; c < STAGE; ++c) {
    if ((uint32_t)c < nck + nvc) {
      const uint32_t dst = (uint32_t)c < nck ? kst + 2u * kChunk * c : vst + 2u * kChunk * (c - nck);
      lds_store<u32x4>(dst + 16u * lane, r[c]);
    }
  }
  const u32x4 z = {0u, 0u, 0u, 0u};
  constexpr uint32_t kz = kMargin / 8;
  if (lane < kz) lds_store<u32x4>(kst + 2u * rn.kn + 16u * lane, z);
  else if (lane < 2 * kz) lds_store<u32x4>(vst + 2u * rn.vn + 16u * (lane - kz), z);
}

// Trip counts of the four walks of a block (key and value tiles, lower and
// upper halves; groups of 8 slots, the upper half with its leading phantom
// slots), each the maximum over the wave: one-hot in a byte per walk, one OR
// reduction for all four.
struct WalkCounts {
  int klo, khi, vlo, vhi;
};

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_or(uint32_t v) {
  return v | (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

__device__ __forceinline__ uint32_t half_groups_onehot(uint64_t bm, int shift) {
  const uint32_t s = (uint32_t)__popc((uint32_t)bm);
  const uint32_t lo = (s + 7u) >> 3;
  const uint32_t hi = ((s & 3u) + (uint32_t)__popc((uint32_t)(bm >> 32)) + 7u) >> 3;
  return (1u << (lo + shift)) | (1u << (hi + shift + 8));
}

__device__ __forceinline__ WalkCounts walk_counts(uint64_t kb, uint64_t vb) {
  uint32_t v = half_groups_onehot(kb, 0) | half_groups_onehot(vb, 16);
  v = dpp_or<0xB1>(v);
  v = dpp_or<0x4E>(v);
  v = dpp_or<0x124>(v);
  v = dpp_or<0x128>(v);
  v |= (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x401F);
  v = (uint32_t)__builtin_amdgcn_readlane((int)v, 0) | (uint32_t)__builtin_amdgcn_readlane((int)v, 32);
  WalkCounts w;
  w.klo = 31 - __builtin_clz(v & 0xffu);
  w.khi = 31 - __builtin_clz((v >> 8) & 0xffu);
  w.vlo = 31 - __builtin_clz((v >> 16) & 0xffu);
  w.vhi = 31 - __builtin_clz(v >> 24);
  return w;
}

// The packed values of a tile start 16-byte aligned in LDS (tiles are padded to
// 8 values), so the walks read them 8 at a time with one 16-byte LDS load and
// pair slot u of the group with the next set bit of the 32-bit half word x.
// Channel -1 (all ones: no bit left) addresses the zero slot of the q table
// and the scratch slot of the expanded tile, so the walk has no per-element
// branch.
//
// The values of the upper half start at rank s = popcount(low half). Its groups
// are read from rank s - s % 4 on (8-byte aligned, two 8-byte loads each), and
// the first s % 4 slots (values of the lower half, already consumed) are
// phantom: they take channel -1 and consume no bit.
__device__ __forceinline__ _Float16 group_value(const u32x4& w, int u) {
  const half2_t h = as_h2(w[u >> 1]);
  return (u & 1) ? h.y : h.x;
}

struct ValueGroup {
  u32x4 w;
  uint32_t c[8];
};

// Channel c of the expanded tile is at byte daddr + c * STRIDE.
template <uint32_t STRIDE>
__device__ __forceinline__ void value_consume(const ValueGroup& g, uint32_t daddr) {
#pragma unroll
  for (int u = 0; u < 8; ++u) lds_store<_Float16>(daddr + g.c[u] * STRIDE, group_value(g.w, u));
}

// Walks with a one-instruction bit clear, x += -1 << f (f = the lowest set
// bit). Past the last set bit f alternates between -1 (all ones) and 31, so a
// walk that runs on (the wave's busiest lane sets the trip count) sends its
// surplus slots to the scratch slot and to channel 31 of its half. The walked
// word therefore leaves bit 31 out: channel 31 of each half is handled once per
// tile by the caller (for keys its q slot is zero, for values its expanded slot
// is rewritten after the walk).
constexpr uint32_t kLow31 = 0x7fffffffu;

template <bool PEEL>
__device__ __forceinline__ uint32_t next_bit(uint32_t& x, int u, uint32_t m) {
  const uint32_t f = ffbl(x);
  const uint32_t nx = x + (~0u << (f & 31u));
  if constexpr (PEEL) {
    const bool real = (uint32_t)u >= m;
    x = real ? nx : x;
    return real ? f : 0xffffffffu;
  } else {
    x = nx;
    return f;
  }
}

// 16 bytes of packed values: 16-byte aligned in the lower half (HI false),
// 8-byte aligned in the upper half.
template <bool HI>
__device__ __forceinline__ u32x4 group_load(uint32_t va) {
  if constexpr (HI) {
    const u32x2 a = lds_load<u32x2>(va), b = lds_load<u32x2>(va + 8u);
    return (u32x4){a.x, a.y, b.x, b.y};
  } else {
    return lds_load<u32x4>(va);
  }
}

template <bool PEEL, bool HI>
__device__ __forceinline__ void value_issue(uint32_t& x, uint32_t va, uint32_t m, ValueGroup& g) {
  g.w = group_load<HI>(va);
#pragma unroll
  for (int u = 0; u < 8; ++u) g.c[u] = next_bit<PEEL>(x, u, m);
}

// One 32-channel half of a tile scattered into the expanded tile, pipelined
// like the key walk: n groups (the wave's maximum); the upper half (HI) starts
// with m phantom slots.
template <bool HI, uint32_t STRIDE>
__device__ __forceinline__ void value_half(int n, uint32_t x, uint32_t a, uint32_t daddr, uint32_t m) {
  if (n == 0) return;
  ValueGroup g0, g1;
  value_issue<HI, HI>(x, a, m, g0);
  int g = 1;
  for (; g + 1 < n; g += 2) {
    value_issue<false, HI>(x, a + 16u * g, 0u, g1);
    value_consume<STRIDE>(g0, daddr);
    value_issue<false, HI>(x, a + 16u * (g + 1), 0u, g0);
    value_consume<STRIDE>(g1, daddr);
  }
  if (g < n) {
    value_issue<false, HI>(x, a + 16u * g, 0u, g1);
    value_consume<STRIDE>(g0, daddr);
    value_consume<STRIDE>(g1, daddr);
  } else {
    value_consume<STRIDE>(g0, daddr);
  }
}

// Expansion of one tile (bitmap bm, packed values at LDS byte address va) into
// an expanded tile whose channel c of half h is at byte d_h + c * STRIDE.
// Channels 31 and 63 are written last (value, or zero when dropped), over the
// walks' surplus writes; nlo and nhi are the wave's trip counts.
template <uint32_t STRIDE>
__device__ __forceinline__ void expand_tile(int nlo, int nhi, uint64_t bm, uint32_t va, uint32_t d_w0,
                                            uint32_t d_w1) {
  const uint32_t lo = (uint32_t)bm, hi = (uint32_t)(bm >> 32);
  const uint32_t s = (uint32_t)__popc(lo), c = s + (uint32_t)__popc(hi), m = s & 3u;
  const _Float16 v31 = lds_load<_Float16>(va + 2u * s - 2u);
  const _Float16 v63 = lds_load<_Float16>(va + 2u * c - 2u);
  value_half<false, STRIDE>(nlo, lo & kLow31, va, d_w0, 0u);
  value_half<true, STRIDE>(nhi, hi & kLow31, va + 2u * (s - m), d_w1, m);
  lds_store<_Float16>(d_w0 + STRIDE * 31u, (int)lo < 0 ? v31 : (_Float16)0.f);
  lds_store<_Float16>(d_w1 + STRIDE * 31u, (int)hi < 0 ? v63 : (_Float16)0.f);
}

template <int T, int G>
__device__ __forceinline__ void write_partial(const AttnArgs& a, int seg, int bh, const float (&m_run)[G],
                                              const float (&l_run)[G], const float (&o)[G][T]) {
  constexpr int d = kTile * T;
  const uint32_t lane = lane_id();
  const int64_t row0 = (int64_t)seg * a.BHq + (int64_t)bh * G;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if (lane == 0) a.ws_ml[row0 + g] = make_float2(m_run[g], l_run[g]);
#pragma unroll
    for (int tt = 0; tt < T; ++tt) a.ws_o[(row0 + g) * d + lane + kTile * tt] = o[g][tt];
  }
}

template <int T, int G>
__device__ __forceinline__ void init_state(float (&m_run)[G], float (&l_run)[G], float (&o)[G][T]) {
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m_run[g] = -INFINITY;
    l_run[g] = 0.f;
#pragma unroll
    for (int tt = 0; tt < T; ++tt) o[g][tt] = 0.f;
  }
}

inline size_t dense_lds_bytes(int T, int G) {
  const int d = kTile * T, NB = kWave / T;
  return (size_t)G * d * 2 + (size_t)NB * G * 4;
}

inline int token_max_elems_dev(int d, int k) {
  const int T = d / kTile;
  const int nonempty = k < T ? k : T;
  const int m = (k + (kPad - 1) * nonempty) / kPad * kPad;
  return m < d ? m : d;
}

// Worst-case fp16 elements per token of a per-channel cache (group_keep gk),
// as the bound on the run of any block of NB block-aligned tokens divided by
// NB: a block of 32 or more tokens holds whole groups of 32 (gk * d kept values
// and at most 7 pad slots per tile each); a shorter block (half a group or
// less) holds at most min(NB, gk) values per channel plus its pad slots.
inline int grouped_token_bound(int d, int gk, int NB) {
  const int T = d / kTile;
  const int64_t per_block =
      NB >= kGroup ? (int64_t)(NB / kGroup) * ((int64_t)gk * d + (int64_t)kGroup * T * (kPad - 1))
                   : (int64_t)d * (NB < gk ? NB : gk) + (int64_t)NB * T * (kPad - 1);
  const int m = (int)((per_block + NB - 1) / NB);
  return m < d ? m : d;
}

// Staging bound per token of one cache for blocks of NB tokens.
inline int side_token_bound(int d, const SparseSide& s, int NB) {
  if (s.bitmaps == nullptr) return 0;
  return s.group_keep >= 0 ? grouped_token_bound(d, s.group_keep, NB) : token_max_elems_dev(d, s.n_keep);
}

// The MFMA kernel for grouped queries (attention_mfma.hip; G in {2, 4, 8}); by
// default the sparse call uses it from kMfmaMinGroup query heads per kv-head
// on, the walks below that (mustafar_attn_set_route overrides the choice). Measured on one box (d = 128, 70/70, best split count of each):
// at G = 2 the walks take 47 us against 58 (16K tokens, 32 streams), at G = 4
// 58 against 57 (16K) and 86 against 99 (128K, 8 streams), at G = 8 85 against
// 59: the matrix cores pay from eight query heads per kv-head on, where each
// expanded key and value feeds eight products.
constexpr int kMfmaMinGroup = 8;
hipError_t launch_sparse_mfma(const AttnShape& sh, const AttnArgs& a, hipStream_t s);

}  // namespace mf
