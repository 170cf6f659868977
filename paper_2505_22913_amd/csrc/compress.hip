// Per-token magnitude pruning and bitmap compression on gfx950.
//
// One wavefront handles one token at a time: lane i holds channel 64t+i of
// every tile t, so the keep-mask of a tile is exactly one 64-bit ballot (Sec. 3
// tiles are 1x64 and the wavefront is 64 lanes wide). Selection of the n_keep
// largest magnitudes (Sec. 2, per-token magnitude pruning) is a
// most-significant-bit first radix select on the 15-bit fp16 magnitude with
// ballot+popcount counts, then ties at the threshold go to the lowest channels
// via mbcnt ranks. The packed position of a kept value inside its tile is
// mbcnt(bitmap) -- the number of kept lanes below it -- so a tile is packed by
// one masked 2-byte store.
//
// A stream's per-tile offsets are an exclusive prefix sum of the padded tile
// counts (Sec. 4.3 pads to 8), so bulk compression is a single-pass scan with
// decoupled look-back: each workgroup takes a ticket (tickets order the chunks
// of a stream), stages its chunk of dense tokens in LDS with 16-byte loads,
// selects and packs every token in place, publishes its chunk total, reads the
// totals or prefixes of the chunks before it, and writes its packed run with
// 16-byte stores. k_append handles the one-token-per-stream case of a decode
// step, and k_window_step the dense-window lifecycle around it: the token that
// leaves a full window is the one appended.
#include "mf_device.h"
#include "mf_launch.h"

namespace mf {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

template <typename V>
__device__ __forceinline__ V lds_ld(uint32_t byte_addr) {
  return *reinterpret_cast<const __attribute__((address_space(3))) V*>(byte_addr);
}

template <typename V>
__device__ __forceinline__ void lds_st(uint32_t byte_addr, V v) {
  *reinterpret_cast<__attribute__((address_space(3))) V*>(byte_addr) = v;
}

__device__ __forceinline__ uint32_t ffbl_u32(uint32_t x) {  // 0xffffffff when x == 0
  uint32_t r;
  asm("v_ffbl_b32 %0, %1" : "=v"(r) : "v"(x));
  return r;
}

__device__ __forceinline__ int wave_max_int(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = max(v, __shfl_xor(v, o, kWave));
  return __builtin_amdgcn_readfirstlane(v);
}

// Keep-mask of one token. mag[t] is the key of this lane's channel in tile t:
// the fp16 magnitude (bits & 0x7fff, 15 bits) or a non-negative fp32 score
// (its bits, 31 bits, order like the values). Sets bm[t] (wave-uniform) so that
// exactly k bits are set over the T tiles: the k largest keys, ties to lower
// channels.
template <int T, int NBITS = 15>
__device__ __forceinline__ void select_token(const uint32_t (&mag)[T], int k, uint64_t (&bm)[T]) {
  if (k <= 0) {
#pragma unroll
    for (int t = 0; t < T; ++t) bm[t] = 0;
    return;
  }
  if (k >= kTile * T) {
#pragma unroll
    for (int t = 0; t < T; ++t) bm[t] = ~0ull;
    return;
  }
  // Largest threshold m with #{mag >= m} >= k: that is the k-th largest key.
  uint32_t thr = 0;
#pragma unroll
  for (int b = NBITS - 1; b >= 0; --b) {
    const uint32_t cand = thr | (1u << b);
    int cnt = 0;
#pragma unroll
    for (int t = 0; t < T; ++t) cnt += __popcll(ballot(mag[t] >= cand));
    thr = (cnt >= k) ? cand : thr;
  }
  int n_gt = 0;
  uint64_t eq[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    bm[t] = ballot(mag[t] > thr);
    eq[t] = ballot(mag[t] == thr);
    n_gt += __popcll(bm[t]);
  }
  // The remaining k - n_gt slots go to the lowest-channel elements equal to thr.
  const int need = k - n_gt;
  int before = 0;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int rank = before + (int)mbcnt(eq[t], 0u);
    bm[t] |= ballot(mag[t] == thr && rank < need);
    before += __popcll(eq[t]);
  }
}

// Writes the packed values of one token (tiles start at `start`, relative to
// the stream) and its T offsets. Returns the fp16 elements the token occupies.
template <int T>
__device__ __forceinline__ uint32_t pack_token(const uint16_t (&xv)[T], const uint64_t (&bm)[T],
                                               uint32_t start, uint16_t* __restrict__ vals,
                                               uint32_t* __restrict__ offs, uint32_t lane) {
  uint32_t off = start;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const uint32_t cnt = (uint32_t)__popcll(bm[t]);
    if ((bm[t] >> lane) & 1ull) vals[off + mbcnt(bm[t], 0u)] = xv[t];
    if (lane >= cnt && lane < pad8(cnt)) vals[off + lane] = 0;  // pad slots hold +0.0
    if (lane == (uint32_t)t) offs[t] = off;
    off += pad8(cnt);
  }
  return off - start;
}

template <int T>
__device__ __forceinline__ void load_token(const uint16_t* __restrict__ src, uint32_t lane,
                                           uint16_t (&xv)[T]) {
#pragma unroll
  for (int t = 0; t < T; ++t) xv[t] = src[kTile * t + lane];
}

// Look-back flag of one chunk: status in bits 63:62, a 32-bit count below.
constexpr uint64_t kFlagAgg = 1ull << 62;     // the chunk's own total is known
constexpr uint64_t kFlagPrefix = 2ull << 62;  // the stream offset after the chunk is known
constexpr uint32_t kBadBase = 0xffffffffu;    // look_back gave up

__global__ void k_clear(uint32_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// After a bulk compression (stream-ordered, so every chunk has finished): a
// stream one of whose chunks gave up has holes, so its stream_len becomes
// kStreamPoisoned, which every later call treats as "skip this stream".
__global__ void k_compress_finalize(const uint32_t* __restrict__ gave_up, uint32_t* __restrict__ stream_len,
                                    int BH) {
  const int bh = blockIdx.x * blockDim.x + threadIdx.x;
  if (bh < BH && gave_up[bh] != 0u) stream_len[bh] = kStreamPoisoned;
}

// The flag words are the only data workgroups exchange (the count travels in
// the same 64-bit word as the status, and no workgroup reads what another one
// writes to the cache), so relaxed device-scope atomics suffice: acquire and
// release would write back and invalidate the whole L2 of the XCD on every poll.
//
// Offset in the stream at which chunk `chunk` starts, computed by one whole
// wave after publish_total: the wave reads the flags of the 64 chunks before it
// at once and adds, from the nearest one back, the totals up to and including
// the first known prefix, moving 64 chunks further back while none is found.
// Chunks with lower tickets (of the same stream) are already running and
// publish their totals without waiting, so every poll is eventually answered;
// the number of flag reads is bounded anyway (max_polls; with 0 every chunk
// but a stream's first gives up, which is how the give-up path is tested).
// The chunk's total (chunk 0: its prefix, first_base + total) is published as
// soon as it is known, before the chunk packs, so that the chunks after it
// rarely wait for it.
__device__ void publish_total(uint64_t* __restrict__ fl, int chunk, uint32_t total, uint32_t first_base,
                              uint32_t lane) {
  if (lane != 0) return;
  if (chunk == 0)
    __hip_atomic_store(fl, kFlagPrefix | (uint64_t)(first_base + total), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  else
    __hip_atomic_store(fl + chunk, kFlagAgg | (uint64_t)total, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

// The flags of the 64 chunks before `top` (lane i: chunk top - i); positions
// before chunk 0 read as a known prefix of 0.
__device__ __forceinline__ uint64_t poll_flags(const uint64_t* __restrict__ fl, int top, uint32_t lane) {
  const int p = top - (int)lane;
  return p >= 0 ? __hip_atomic_load(fl + p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : kFlagPrefix;
}

// f0: the first poll, poll_flags(fl, chunk - 1, lane), issued by the caller
// ahead of time so that its latency overlaps other work.
__device__ uint32_t look_back(uint64_t* __restrict__ fl, int chunk, uint32_t total,
                              uint32_t first_base, uint32_t lane, uint32_t max_polls, uint64_t f0) {
  if (chunk == 0) return first_base;
  uint32_t acc = 0, polls = 0;
  for (int top = chunk - 1;;) {
    if (polls++ >= max_polls) return kBadBase;
    const uint64_t f = polls == 1 ? f0 : poll_flags(fl, top, lane);
    const uint32_t st = (uint32_t)(f >> 62);
    const uint64_t pref = ballot(st == 2u);
    const uint64_t none = ballot(st == 0u);
    const uint32_t first = pref ? (uint32_t)__builtin_ctzll(pref) : 64u;  // nearest prefix
    const uint64_t upto = first >= 63u ? ~0ull : ((2ull << first) - 1ull);
    if (none & upto) {  // a chunk between here and that prefix has not published yet
      __builtin_amdgcn_s_sleep(1);
      continue;
    }
    uint32_t v = lane <= first ? (uint32_t)f : 0u;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += (uint32_t)__shfl_xor((int)v, o, kWave);
    acc += v;
    if (first < 64u) break;
    top -= kWave;
  }
  if (lane == 0)
    __hip_atomic_store(fl + chunk, kFlagPrefix | (uint64_t)(acc + total), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  return acc;
}

// Top-k selection with one lane per token, bit-sliced. A lane holds the 15-bit
// magnitudes of its token (of its half of the token when d = 256), two per
// 32-bit register. A 16x16 bit transpose of each group of 16 registers (the low
// and high halves are two independent matrices) turns them into bit planes:
// word b of a group has bit r = bit b of key 2r and bit 16+r = bit b of key
// 2r+1 of the group's 32 keys. The k largest keys are then found most
// significant bit first on whole plane words: `cand` holds the keys that still
// tie with the threshold prefix and `above` those already known to be larger;
// a plane's ones in `cand` either all stay candidates (if, with `above`, they
// reach k) or all move to `above`. At the end the threshold ties (`cand`) are
// taken lowest channel first up to k. This is the same selection as the radix
// search on the magnitude, with a per-plane cost instead of a per-key one.
// (m & a) | (~m & b) in one instruction (the compiler splits the masked
// halves apart when it sees them).
__device__ __forceinline__ uint32_t bit_select(uint32_t m, uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "s"(m), "v"(a), "v"(b));
  return r;
}

// a * b + c on 24-bit signed operands, one instruction (|a|, |b| < 2^23).
__device__ __forceinline__ int mad_i24(int a, int b, int c) {
  int r;
  asm("v_mad_i32_i24 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// (a << s) + b, one instruction (kept as written: a running sum of bits
// would otherwise be rebuilt from a second counter at every step).
__device__ __forceinline__ int lshl_add(int a, int s, int b) {
  int r;
  asm("v_lshl_add_u32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "i"(s), "v"(b));
  return r;
}

// The transpose is four rounds of block swaps (8, 4, 2, 1 bits): in the round
// of s, rows i and i+s (i without bit s) exchange the s-bit blocks that sit
// off the diagonal. The byte round is one byte permute per row; the others
// are a shift and a bit select per row.
__device__ __forceinline__ void transpose16x2(uint32_t* x) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t a = x[i], b = x[i + 8];
    x[i] = __builtin_amdgcn_perm(b, a, 0x06020400u);      // a.byte0, b.byte0, a.byte2, b.byte2
    x[i + 8] = __builtin_amdgcn_perm(b, a, 0x07030501u);  // a.byte1, b.byte1, a.byte3, b.byte3
  }
  constexpr uint32_t kMask[3] = {0x0f0f0f0fu, 0x33333333u, 0x55555555u};
#pragma unroll
  for (int l = 0; l < 3; ++l) {
    const int s = 4 >> l;
    const uint32_t m = kMask[l];  // the low block of each pair; ~m == m << s
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (i & s) continue;
      const uint32_t a = x[i], b = x[i + s];
      x[i] = bit_select(m, a, b << s);
      x[i + s] = bit_select(m, a >> s, b);
    }
  }
}

// Bit r of the low half to bit 2r, bit r of the high half to bit 2r+1.
__device__ __forceinline__ uint32_t interleave_halves(uint32_t x) {
  constexpr uint32_t kMask[4] = {0x0000ff00u, 0x00f000f0u, 0x0c0c0c0cu, 0x22222222u};
#pragma unroll
  for (int l = 0; l < 4; ++l) {
    const int s = 8 >> l;
    const uint32_t t = ((x >> s) ^ x) & kMask[l];
    x ^= t ^ (t << s);
  }
  return x;
}

// The lowest n set bits of w (n >= 0).
__device__ __forceinline__ uint32_t lowest_bits(uint32_t w, int n) {
  if (n >= (int)__popc(w)) return w;
  if (n <= 0) return 0u;
  uint32_t p = 0;  // largest p with popcount(w below bit p) < n
#pragma unroll
  for (int s = 16; s >= 1; s >>= 1)
    if ((int)__popc(w & ((1u << (p + s)) - 1u)) < n) p += s;
  return w & (p >= 31u ? 0xffffffffu : ((2u << p) - 1u));
}

// Workgroup barrier that orders LDS only: the waves of a workgroup exchange
// nothing else, and a full barrier would also wait for loads in flight.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// compress_waves() waves per workgroup; a chunk is that many runs of 64 tokens
// (32 from d = 128 on) of one stream, one run per wave. The waves select and
// pack their runs side by side and share the chunk's ticket, scan total and
// look-back, so those cost once per chunk (two waves: 4% off the bulk
// compression of a 50% cache against one; four measured the same).
// PRESET: the keep-masks are the bitmaps already in the cache for these tokens
// (a pruner variant selected them); only the scan and the packing run.
template <int T>
constexpr int compress_waves() { return 2; }

template <int T, bool PRESET = false>
__global__ __launch_bounds__(compress_waves<T>() * kWave) void k_compress(const uint16_t* __restrict__ x, int n_new, int k_all,
                                                    uint64_t* __restrict__ bitmaps,
                                                    uint32_t* __restrict__ offsets,
                                                    uint16_t* __restrict__ values,
                                                    uint32_t* __restrict__ stream_len,
                                                    int cap_tokens, int tok0, int64_t val_stride,
                                                    uint64_t* __restrict__ flags,
                                                    uint32_t* __restrict__ ticket_ctr, int n_chunks,
                                                    int64_t x_stride, PruneOpts o, uint32_t max_polls,
                                                    uint32_t* __restrict__ gave_up,
                                                    uint32_t* __restrict__ status) {
  constexpr int d = kTile * T;
  constexpr int kCompressWaves = compress_waves<T>();
  constexpr int LPT = T >= 2 ? 2 : 1;      // lanes per token (selection and packing)
  constexpr int TPW = kWave / LPT;          // tokens per wave
  constexpr int CPL = d / LPT;              // channels per lane
  constexpr int NR = CPL / 2;               // packed registers per lane
  constexpr int ROW = d * 2 + 16;           // LDS bytes per token row (pad: conflict-free row reads)
  constexpr int P16 = d / 8;                // 16-byte pieces per row
  __shared__ __align__(16) unsigned char s_rows_all[kCompressWaves][TPW * ROW];  // dense rows
  __shared__ uint32_t s_share[kCompressWaves + 2];  // ticket, the waves' run lengths, the chunk's base

  const uint32_t lane = lane_id();
  const int wave = (int)(threadIdx.x / kWave);
  unsigned char* s_rows = s_rows_all[wave];
  // Workgroups take the streams in turn and, within a stream, ordered tickets
  // from the stream's counter (one counter per stream keeps the atomics spread).
  const int bh = (int)(blockIdx.x % (gridDim.x / (uint32_t)n_chunks));
  // A stream poisoned by an earlier call takes no more tokens: every workgroup
  // of it leaves before drawing a ticket (the last chunk, which rewrites
  // stream_len, draws the last ticket, after every other workgroup's read).
  if (tok0 > 0 && __builtin_amdgcn_readfirstlane((int)stream_len[bh]) == (int)kStreamPoisoned) return;
  constexpr int kChunk = kCompressWaves * TPW;
  constexpr int kIt = TPW * P16 / kWave;  // 16-byte loads per lane for the wave's rows
  // Stage loads of the wave's dense rows of chunk `ch`: 16-byte coalesced
  // non-temporal loads (every load issued; lanes past the rows re-read the
  // chunk's first piece and store nothing).
  auto stage_load = [&](int ch, u32x4_t (&r)[kIt]) {
    const int sj0 = ch * kChunk + wave * TPW;
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(
        x + ((int64_t)bh * x_stride + (sj0 < n_new ? sj0 : ch * kChunk)) * d);
    const int n16 = max(min(TPW, n_new - sj0), 0) * P16;
#pragma unroll
    for (int i = 0; i < kIt; ++i) {
      const int c = i * kWave + (int)lane;
      r[i] = __builtin_nontemporal_load(&src[c < n16 ? c : 0]);
    }
  };
  // The chunk comes with the ticket; the rows of the chunk that workgroups
  // launched in order would draw are loaded meanwhile (and loaded again in
  // the rare case that the ticket differs). The ticket is drawn with an
  // increment: the wave-aggregating rewrite of an add waits for its result
  // at once.
  const int guess = (int)(blockIdx.x / (gridDim.x / (uint32_t)n_chunks));
  uint32_t tk = 0u;
  if (threadIdx.x == 0) tk = atomicInc(ticket_ctr + bh, 0xffffffffu);
  u32x4_t r[kIt];
  stage_load(guess, r);
  if (threadIdx.x == 0) s_share[0] = tk;
  lds_barrier();
  const int chunk = __builtin_amdgcn_readfirstlane((int)s_share[0]);
  if (chunk != guess) stage_load(chunk, r);
  const int k = o.per_head ? o.head_keep[bh % o.H] : k_all;  // kept channels of this stream
  const int jc = chunk * kChunk;                // the chunk's first token
  const int j0 = jc + wave * TPW;               // this wave's first token
  const int nt = min(TPW, n_new - j0);          // <= 0: the chunk ends before this wave's half
  const uint32_t base_lds = (uint32_t)(uintptr_t)s_rows;
  {
    const int n16 = max(nt, 0) * P16;
#pragma unroll
    for (int i = 0; i < kIt; ++i) {
      const int c = i * kWave + (int)lane;
      if (c < n16) *reinterpret_cast<u32x4_t*>(s_rows + (c / P16) * ROW + (c % P16) * 16) = r[i];
    }
  }

  // This lane's half row (lanes past the chunk take a copy of the last row
  // and store nothing), kept in registers for the packing.
  uint32_t raw[NR];
  {
    const unsigned char* row = s_rows + min((int)lane / LPT, max(nt, 1) - 1) * ROW + ((int)lane % LPT) * CPL * 2;
#pragma unroll
    for (int i = 0; i < NR / 4; ++i) {
      const u32x4_t w = *reinterpret_cast<const u32x4_t*>(row + 16 * i);
#pragma unroll
      for (int e = 0; e < 4; ++e) raw[4 * i + e] = w[e];  // channels 8i+2e, 8i+2e+1
    }
  }

  // Keep-mask of this lane's token: NW words of 32 channels, channel order.
  constexpr int NW = NR / 16;
  uint32_t keep[NW];
  if constexpr (PRESET) {
    // (a wave whose run lies past the chunk's end reads nothing: its tokens
    // are past n_new, possibly past the cache's capacity)
    const int jt = min((int)lane / LPT, max(nt, 1) - 1);
    const int64_t tb = ((int64_t)bh * cap_tokens + tok0 + j0 + jt) * T + ((int)lane % LPT) * (T / LPT);
#pragma unroll
    for (int t = 0; t < NW / 2; ++t) {
      const uint64_t bm = nt > 0 ? bitmaps[tb + t] : 0ull;
      keep[2 * t] = (uint32_t)bm;
      keep[2 * t + 1] = (uint32_t)(bm >> 32);
    }
  } else {
    // Register 16 g + i holds the keys of channels 32 g + i (low half) and
    // 32 g + 16 + i (high half), so that bit r of plane word b of group g is
    // bit b of channel 32 g + r: the planes come out in channel order. The
    // sign bits land in plane 15, which the search never reads.
    uint32_t pl[NR];
#pragma unroll
    for (int g = 0; g < NW; ++g) {
      uint32_t r[16];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t a = raw[16 * g + j], b = raw[16 * g + 8 + j];
        r[2 * j] = __builtin_amdgcn_perm(b, a, 0x05040100u);      // low halves of a and b
        r[2 * j + 1] = __builtin_amdgcn_perm(b, a, 0x07060302u);  // high halves
      }
      transpose16x2(r);
#pragma unroll
      for (int i = 0; i < 16; ++i) pl[16 * g + i] = r[i];  // pl[16g + b] = plane b of group g
    }
    uint32_t cand[NW], above[NW];
#pragma unroll
    for (int g = 0; g < NW; ++g) {
      cand[g] = 0xffffffffu;
      above[g] = 0u;
    }
    int need = k;  // keys still to keep beyond `above`
#pragma unroll
    for (int b = 14; b >= 0; --b) {
      uint32_t ones[NW];
      int c1 = 0;
#pragma unroll
      for (int g = 0; g < NW; ++g) {
        ones[g] = cand[g] & pl[16 * g + b];
        c1 += __popc(ones[g]);
      }
      if constexpr (LPT == 2) c1 += __builtin_amdgcn_update_dpp(0, c1, 0xB1, 0xF, 0xF, true);
      // The candidates with a one here reach the rest of k: they stay the
      // candidates. Otherwise (fall = -1) they are all kept and those with a
      // zero stay candidates.
      const int fall = (c1 - need) >> 31;
#pragma unroll
      for (int g = 0; g < NW; ++g) {
        above[g] |= ones[g] & (uint32_t)fall;
        cand[g] = ones[g] ^ (cand[g] & (uint32_t)fall);
      }
      need = mad_i24(c1, fall, need);  // need - c1 when they fell
    }
    // Ties at the threshold: the lowest channels first, up to k (across the two
    // lanes of a token, the lower half of the channels first): `drop` of this
    // lane's candidates, the highest channels, are not kept.
    int n_cand = 0;
#pragma unroll
    for (int g = 0; g < NW; ++g) n_cand += __popc(cand[g]);
    if constexpr (LPT == 2) {
      const int lower = __builtin_amdgcn_mov_dpp(n_cand, 0xB1, 0xF, 0xF, false);
      if (lane & 1u) need -= lower;
    }
    int drop = n_cand - min(max(need, 0), n_cand);
    if (ballot(drop > 2)) {
#pragma unroll
      for (int g = 0; g < NW; ++g) {
        const int c = __popc(cand[g]);
        cand[g] = lowest_bits(cand[g], need);
        need -= c;
      }
    } else {
      // Usually at most one tie: clear the highest candidate drop times.
      while (ballot(drop > 0)) {
        bool done = drop <= 0;
#pragma unroll
        for (int g = NW - 1; g >= 0; --g) {
          const bool here = !done && cand[g] != 0u;
          const uint32_t top = cand[g] != 0u ? 0x80000000u >> __clz(cand[g]) : 0u;
          cand[g] = here ? cand[g] & ~top : cand[g];
          done = done || here;
        }
        --drop;
      }
    }
#pragma unroll
    for (int g = 0; g < NW; ++g) keep[g] = above[g] | cand[g];
  }

  // Tile offsets relative to the chunk's run: the padded tile counts of this
  // lane, scanned over the lanes (token-major, so for d = 256 the lower half
  // of a token comes first).
  constexpr int TPL = T / LPT;               // tiles per lane
  uint32_t tile_pos[TPL];
  uint32_t lane_len = 0;
#pragma unroll
  for (int t = 0; t < TPL; ++t) {
    tile_pos[t] = lane_len;
    lane_len += pad8((uint32_t)(__popc(keep[2 * t]) + __popc(keep[2 * t + 1])));
  }
  if ((int)lane >= nt * LPT) lane_len = 0;   // lanes past the chunk hold no token
  const uint32_t incl = wave_incl_scan(lane_len);
  const uint32_t wave_run = (uint32_t)__builtin_amdgcn_readlane((int)incl, kWave - 1);
  if (lane == 0) s_share[1 + wave] = wave_run;
  lds_barrier();
  uint32_t run = 0, wave_off = 0;           // the chunk's run: the waves' runs in order
#pragma unroll
  for (int w = 0; w < kCompressWaves; ++w) {
    wave_off = w == wave ? run : wave_off;
    run += s_share[1 + w];
  }
  const uint32_t lane_off = incl - lane_len;  // in the wave's run
  const uint32_t first = (chunk == 0 && tok0 > 0) ? stream_len[bh] : 0u;
  if (wave == 0) publish_total(flags + (int64_t)bh * n_chunks, chunk, run, first, lane);
  // The first look-back poll, in flight while the run is packed.
  const uint64_t f0 = (wave == 0 && chunk > 0) ? poll_flags(flags + (int64_t)bh * n_chunks, chunk - 1, lane) : 0ull;

  // Packing, lane = its tiles: from its row held in registers, the lane
  // writes the kept values of each tile in channel order, value r of a tile
  // at r, over the wave's own rows (a wave's LDS operations run in program
  // order, so every row was read before the first write). The run is at most
  // d values per token, so it ends before the last row's pad, the trash slot
  // of the dropped channels. The tile's last group of 8 is zeroed first, so
  // its pad slots hold +0.0.
  {
    const uint32_t trash = base_lds + (uint32_t)(TPW * ROW - 16);
    const bool live = (int)lane < nt * LPT;
#pragma unroll
    for (int t = 0; t < TPL; ++t) {
      const uint32_t lo = live ? keep[2 * t] : 0u, hi = live ? keep[2 * t + 1] : 0u;
      const uint32_t cnt = (uint32_t)(__popc(lo) + __popc(hi));
      const uint32_t pos = base_lds + 2u * (lane_off + tile_pos[t]);
      if (cnt & 7u) lds_st<u32x4_t>(pos + 16u * (cnt / 8u), (u32x4_t){0u, 0u, 0u, 0u});
      // Value c goes to trash + bit * delta: the next packed slot when kept
      // (delta, in bytes from the trash slot, then moves one slot on).
      int delta = (int)pos - (int)trash;  // |delta| < 64 KiB
#pragma unroll
      for (int c = 0; c < kTile; ++c) {
        const int bit = (int)(((c < 32 ? lo : hi) >> (c & 31)) & 1u);
        const uint32_t pair = raw[(kTile / 2) * t + c / 2];
        lds_st<uint16_t>((uint32_t)mad_i24(bit, delta, (int)trash), (uint16_t)(c & 1 ? pair >> 16 : pair));
        delta = lshl_add(bit, 1, delta);
      }
    }
  }

  if (wave == 0) {
    const uint32_t b = look_back(flags + (int64_t)bh * n_chunks, chunk, run, first, lane, max_polls, f0);
    if (lane == 0) s_share[kCompressWaves + 1] = b;
    if (lane == 0 && b == kBadBase) {
      // Mark the stream and the call; k_compress_finalize poisons the stream
      // once every chunk has finished.
      __hip_atomic_store(gave_up + bh, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(status, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (lane == 0 && chunk == n_chunks - 1 && b != kBadBase) stream_len[bh] = b + run;
  }
  lds_barrier();  // the chunk's base
  const uint32_t base = __builtin_amdgcn_readfirstlane((int)s_share[kCompressWaves + 1]);
  if (base == kBadBase) return;  // look-back gave up: nothing is written

  // The wave's packed run (a multiple of 8 values, 16-byte aligned in the
  // stream), after the runs of the waves before it.
  {
    u32x4_t* dst = reinterpret_cast<u32x4_t*>(values + (int64_t)bh * val_stride + base + wave_off);
    const uint32_t n16 = (uint32_t)s_share[1 + wave] / 8u;
    for (uint32_t c = lane; c < n16; c += kWave)
      __builtin_nontemporal_store(lds_ld<u32x4_t>(base_lds + 16u * c), &dst[c]);
  }
  // Bitmaps and offsets of this lane's tiles (tile index = token * T + t).
  if ((int)lane < nt * LPT) {
    const int64_t tile0 = ((int64_t)bh * cap_tokens + tok0 + j0) * T + (int)lane * TPL;
#pragma unroll
    for (int t = 0; t < TPL; ++t) {
      if constexpr (!PRESET) bitmaps[tile0 + t] = (uint64_t)keep[2 * t] | ((uint64_t)keep[2 * t + 1] << 32);
      offsets[tile0 + t] = base + wave_off + lane_off + tile_pos[t];
    }
  }
}

// Output-aware keep-mask of one token, lane = channel: the score |x| * w in
// fp32 (one rounding) of channel 64 t + lane, w the token's fp32 channel
// weights; non-negative, so its bits order like its value (31 significant bits).
template <int T>
__device__ __forceinline__ void select_output_aware(int k, const uint16_t (&xv)[T],
                                                    const float* __restrict__ w, uint32_t lane,
                                                    uint64_t (&bm)[T]) {
  uint32_t key[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const float m = fabsf(half_bits_to_float(xv[t]));
    key[t] = __builtin_bit_cast(uint32_t, m * w[kTile * t + lane]);
  }
  select_token<T, 31>(key, k, bm);
}

// Keep-mask of one token under a pruner variant, lane = channel; xv[t] is the
// lane's fp16 bits in tile t, w the token's fp32 channel weights (output-aware).
template <int T>
__device__ __forceinline__ void select_variant(const PruneOpts& o, int k, const uint16_t (&xv)[T],
                                               const float* __restrict__ w, uint32_t lane,
                                               uint64_t (&bm)[T]) {
  if (o.mode == kPrune24) {
    // 2 of every 4 consecutive channels (the lanes of a quad): a lane is kept if
    // it beats at least two of the other three (larger magnitude, or equal and
    // a lower channel).
    const uint32_t i = lane & 3u;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int key = xv[t] & 0x7fff;
      const int k1 = __builtin_amdgcn_mov_dpp(key, 0xB1, 0xF, 0xF, false);  // lane ^ 1
      const int k2 = __builtin_amdgcn_mov_dpp(key, 0x4E, 0xF, 0xF, false);  // lane ^ 2
      const int k3 = __builtin_amdgcn_mov_dpp(key, 0x1B, 0xF, 0xF, false);  // lane ^ 3
      const int wins = (key > k1 || (key == k1 && i < (i ^ 1u))) + (key > k2 || (key == k2 && i < (i ^ 2u))) +
                       (key > k3 || (key == k3 && i < (i ^ 3u)));
      bm[t] = ballot(wins >= 2);
    }
  } else if (o.mode == kPruneOutputAware) {
    select_output_aware<T>(k, xv, w, lane, bm);
  } else {
    uint32_t mag[T];
#pragma unroll
    for (int t = 0; t < T; ++t) mag[t] = xv[t] & 0x7fffu;
    select_token<T>(mag, k, bm);
  }
}

__device__ __forceinline__ int stream_keep(const PruneOpts& o, int bh, int n_keep) {
  return o.per_head ? o.head_keep[bh % o.H] : n_keep;
}

// Bitmaps of tokens tok0 .. tok0+n_new-1 of every stream under a pruner
// variant: one wave per token, lane = channel, kTokPerWave tokens per wave.
constexpr int kTokPerWave = 8;

template <int T>
__global__ __launch_bounds__(256) void k_select(CacheView c, const uint16_t* __restrict__ x, int n_new,
                                                int64_t x_stride, int tok0, PruneOpts o) {
  constexpr int d = kTile * T;
  const int64_t wave = (int64_t)blockIdx.x * (256 / kWave) + threadIdx.x / kWave;
  const uint32_t lane = lane_id();
  const int64_t total = (int64_t)c.BH * n_new;
  for (int64_t i = wave * kTokPerWave; i < min(total, (wave + 1) * kTokPerWave); ++i) {
    const int bh = (int)(i / n_new), j = (int)(i % n_new);
    const int64_t row = (int64_t)bh * x_stride + j;
    uint16_t xv[T];
#pragma unroll
    for (int t = 0; t < T; ++t) xv[t] = x[row * d + kTile * t + lane];
    uint64_t bm[T];
    select_variant<T>(o, stream_keep(o, bh, c.n_keep), xv, o.weights ? o.weights + row * d : nullptr,
                      lane, bm);
    uint64_t mine = bm[0];
#pragma unroll
    for (int t = 1; t < T; ++t) mine = (lane == (uint32_t)t) ? bm[t] : mine;
    if (lane < (uint32_t)T) c.bitmaps[((int64_t)bh * c.cap_tokens + tok0 + j) * T + lane] = mine;
  }
}

// ---- Per-channel value pruning in groups of 32 tokens (Sec. 2) ---------------------------
// The keep word of one channel over a group (bit j: token j kept): the k
// tokens with the largest keys, equal keys to the lower token. Keys are 15-bit
// fp16 magnitudes (NBITS 15) or the bits of non-negative fp32 scores (NBITS
// 31); both order like the values. Bit-sliced like the token selection of
// k_compress: the 32 keys become bit planes of 32-token words (two 16x16
// transposes of key pairs per 16 bits of key), searched most significant bit
// first; the threshold ties are then taken lowest token first.
template <int NBITS>
__device__ __forceinline__ uint32_t channel_keep_word(const uint32_t (&key)[kGroup], int k) {
  if (k <= 0) return 0u;
  if (k >= kGroup) return 0xffffffffu;
  constexpr int NP = NBITS > 16 ? 2 : 1;  // 16-bit slices of the key
  uint32_t pl[NP][16];
#pragma unroll
  for (int h = 0; h < NP; ++h) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const uint32_t a = (key[2 * r] >> (16 * h)) & 0xffffu, c = (key[2 * r + 1] >> (16 * h)) & 0xffffu;
      pl[h][r] = a | (c << 16);
    }
    transpose16x2(pl[h]);  // pl[h][b]: bit r = bit 16h+b of key 2r, bit 16+r = of key 2r+1
  }
  uint32_t cand = 0xffffffffu, above = 0u;
  int n_above = 0;
#pragma unroll
  for (int b = NBITS - 1; b >= 0; --b) {
    const uint32_t plane = pl[b / 16][b % 16];
    const uint32_t ones = cand & plane;
    const int c1 = (int)__popc(ones);
    const bool take = n_above + c1 >= k;
    above = take ? above : (above | ones);
    cand = take ? ones : (cand & ~plane);
    n_above += take ? 0 : c1;
  }
  return interleave_halves(above) | lowest_bits(interleave_halves(cand), k - n_above);
}

// Key of value x of token j: its fp16 magnitude, or (SCORED) the fp32 product
// |x| * w_j rounded once.
template <bool SCORED>
__device__ __forceinline__ uint32_t channel_key(uint16_t x, float wj) {
  if constexpr (SCORED) return __builtin_bit_cast(uint32_t, fabsf(half_bits_to_float(x)) * wj);
  else return x & 0x7fffu;
}

// Lane (token j, tile t) of the group, j * T + t = r * 64 + lane, takes the
// bitmap of that tile: ballots of bit j of each channel's keep word.
template <int T>
__device__ __forceinline__ void group_bitmaps(const uint32_t (&word)[T], uint32_t lane,
                                              uint64_t (&mine)[(kGroup * T + kWave - 1) / kWave]) {
#pragma unroll
  for (int r = 0; r < (kGroup * T + kWave - 1) / kWave; ++r) mine[r] = 0;
#pragma unroll
  for (int j = 0; j < kGroup; ++j)
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const uint64_t bm = ballot(((word[t] >> j) & 1u) != 0u);
      const int i = j * T + t;
      if (lane == (uint32_t)(i % kWave)) mine[i / kWave] = bm;
    }
}

// Bitmaps of tokens tok0 .. tok0+n_new-1 of every stream under per-channel
// pruning: one wave per (stream, group of 32 tokens), lane = channel of a tile.
template <int T, bool SCORED>
__global__ __launch_bounds__(256) void k_select_channel(CacheView c, const uint16_t* __restrict__ x,
                                                        int n_new, int64_t x_stride, int tok0,
                                                        const float* __restrict__ w) {
  constexpr int d = kTile * T;
  constexpr int R = (kGroup * T + kWave - 1) / kWave;
  const int groups = n_new / kGroup;
  const int64_t wave = (int64_t)blockIdx.x * (256 / kWave) + threadIdx.x / kWave;
  if (wave >= (int64_t)c.BH * groups) return;
  const int bh = (int)(wave / groups), g = (int)(wave % groups);
  const uint32_t lane = lane_id();
  const int64_t row0 = (int64_t)bh * x_stride + (int64_t)g * kGroup;
  uint32_t word[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    uint32_t key[kGroup];
#pragma unroll
    for (int j = 0; j < kGroup; ++j)
      key[j] = channel_key<SCORED>(x[(row0 + j) * d + kTile * t + lane], SCORED ? w[row0 + j] : 0.f);
    word[t] = channel_keep_word<SCORED ? 31 : 15>(key, c.group_keep);
  }
  uint64_t mine[R];
  group_bitmaps<T>(word, lane, mine);
  const int64_t tile0 = ((int64_t)bh * c.cap_tokens + tok0 + (int64_t)g * kGroup) * T;
#pragma unroll
  for (int r = 0; r < R; ++r)
    if (r * kWave + (int)lane < kGroup * T) c.bitmaps[tile0 + r * kWave + lane] = mine[r];
}

// Output-aware weights, one thread per (b, h, T, channel).
__global__ __launch_bounds__(256) void k_query_lookahead(const uint16_t* __restrict__ q, int B, int Hq,
                                                         int Hkv, int n_q, int d, int L,
                                                         float* __restrict__ w) {
  const int G = Hq / Hkv;
  const int64_t n = (int64_t)B * Hkv * n_q * d;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % d);
    const int tq = (int)((i / d) % n_q);
    const int64_t bh = i / ((int64_t)d * n_q);
    const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
    float acc = 0.f;
    const int t1 = min(tq + L, n_q);
    for (int t = tq; t < t1; ++t)
      for (int g = 0; g < G; ++g)
        acc += fabsf(half_bits_to_float(q[(((int64_t)b * Hq + h * G + g) * n_q + t) * d + c]));
    w[i] = acc;
  }
}

// The same weights for L = 32, 32 consecutive positions per thread: the thread
// reads the |q| of the 63 positions its windows cover once (zeros past the
// end, which leave an fp32 sum unchanged) and adds each into the windows that
// contain it, position by position and query head by query head, so every
// output gets exactly the additions, in the order, of the one-thread form.
constexpr int kLookRun = 32;

template <int G>
__global__ __launch_bounds__(256) void k_query_lookahead32(const uint16_t* __restrict__ q, int B, int Hkv,
                                                           int n_q, int d, float* __restrict__ w) {
  constexpr int L = 32;
  const int runs = (n_q + kLookRun - 1) / kLookRun;
  const int64_t n = (int64_t)B * Hkv * runs * d;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int c = (int)(i % d);
  const int run = (int)((i / d) % runs);
  const int64_t bh = i / ((int64_t)d * runs);
  const int b = (int)(bh / Hkv), h = (int)(bh % Hkv);
  const int T0 = run * kLookRun;
  const uint16_t* qb = q + ((int64_t)b * Hkv * G + (int64_t)h * G) * n_q * d + c;
  float acc[kLookRun];
#pragma unroll
  for (int k = 0; k < kLookRun; ++k) acc[k] = 0.f;
#pragma unroll
  for (int s = 0; s < kLookRun + L - 1; ++s) {
    const int t = T0 + s;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float v = t < n_q ? fabsf(half_bits_to_float(qb[((int64_t)g * n_q + t) * d])) : 0.f;
#pragma unroll
      for (int k = 0; k < kLookRun; ++k)
        if (s >= k && s < k + L) acc[k] += v;   // window of output T0 + k: positions k .. k+L-1
    }
  }
  float* wb = w + (bh * n_q + T0) * (int64_t)d + c;
#pragma unroll
  for (int k = 0; k < kLookRun; ++k)
    if (T0 + k < n_q) wb[(int64_t)k * d] = acc[k];
}

// Prune, compress and append one token (d fp16 at src) to stream bh as token
// tok: the token's bitmaps and offsets, its packed values after the stream's
// stream_len values (none when tok == 0), then the new stream_len. One wave.
template <int T>
__device__ __forceinline__ void append_one(const CacheView& c, int bh, int tok,
                                           const uint16_t* __restrict__ src, uint32_t lane) {
  const uint32_t base = tok > 0 ? c.stream_len[bh] : 0u;
  if (base == kStreamPoisoned) return;  // the stream lost tokens: it takes no more
  uint16_t xv[T];
  load_token<T>(src, lane, xv);
  uint32_t mag[T];
#pragma unroll
  for (int t = 0; t < T; ++t) mag[t] = xv[t] & 0x7fffu;
  uint64_t bm[T];
  select_token<T>(mag, c.n_keep, bm);
  const int64_t tile0 = ((int64_t)bh * c.cap_tokens + tok) * T;
  uint64_t mine = bm[0];
#pragma unroll
  for (int t = 1; t < T; ++t) mine = (lane == (uint32_t)t) ? bm[t] : mine;
  if (lane < (uint32_t)T) c.bitmaps[tile0 + lane] = mine;
  const uint32_t used =
      pack_token<T>(xv, bm, base, c.values + (int64_t)bh * c.val_stride, c.offsets + tile0, lane);
  if (lane == 0) c.stream_len[bh] = base + used;
}

// append_one under a pruner variant (w: the token's fp32 weights, output-aware).
template <int T>
__device__ __forceinline__ void append_one_variant(const CacheView& c, const PruneOpts& o, int bh, int tok,
                                                   const uint16_t* __restrict__ src,
                                                   const float* __restrict__ w, uint32_t lane) {
  const uint32_t base = tok > 0 ? c.stream_len[bh] : 0u;
  if (base == kStreamPoisoned) return;
  uint16_t xv[T];
  load_token<T>(src, lane, xv);
  uint64_t bm[T];
  select_variant<T>(o, stream_keep(o, bh, c.n_keep), xv, w, lane, bm);
  const int64_t tile0 = ((int64_t)bh * c.cap_tokens + tok) * T;
  uint64_t mine = bm[0];
#pragma unroll
  for (int t = 1; t < T; ++t) mine = (lane == (uint32_t)t) ? bm[t] : mine;
  if (lane < (uint32_t)T) c.bitmaps[tile0 + lane] = mine;
  const uint32_t used =
      pack_token<T>(xv, bm, base, c.values + (int64_t)bh * c.val_stride, c.offsets + tile0, lane);
  if (lane == 0) c.stream_len[bh] = base + used;
}

template <int T>
__global__ __launch_bounds__(256) void k_append_variant(CacheView c, const uint16_t* __restrict__ x,
                                                        int tok0, PruneOpts o) {
  const int bh = blockIdx.x * (256 / kWave) + threadIdx.x / kWave;
  if (bh >= c.BH) return;
  const int64_t row = (int64_t)bh * kTile * T;
  append_one_variant<T>(c, o, bh, tok0, x + row, o.weights ? o.weights + row : nullptr, lane_id());
}

// One wave per stream, 4 streams per 256-thread block.
template <int T>
__global__ __launch_bounds__(256) void k_append(CacheView c, const uint16_t* __restrict__ x, int tok0) {
  const int bh = blockIdx.x * (256 / kWave) + threadIdx.x / kWave;
  if (bh >= c.BH) return;
  append_one<T>(c, bh, tok0, x + (int64_t)bh * kTile * T, lane_id());
}

// The keys and values of one decode step in one launch: waves 0 .. BH-1 append
// to kc, the next BH to vc (the caches have the same shape and token count).
template <int T>
__global__ __launch_bounds__(256) void k_append_kv(CacheView kc, CacheView vc, const uint16_t* __restrict__ k,
                                                   const uint16_t* __restrict__ v, int tok0) {
  const int i = blockIdx.x * (256 / kWave) + threadIdx.x / kWave;
  if (i >= 2 * kc.BH) return;
  const bool is_v = i >= kc.BH;
  const int bh = is_v ? i - kc.BH : i;
  append_one<T>(is_v ? vc : kc, bh, tok0, (is_v ? v : k) + (int64_t)bh * kTile * T, lane_id());
}

// append_one with output-aware selection: w the token's fp32 channel weights.
template <int T>
__device__ __forceinline__ void append_one_weighted(const CacheView& c, int bh, int tok,
                                                    const uint16_t* __restrict__ src,
                                                    const float* __restrict__ w, uint32_t lane) {
  const uint32_t base = tok > 0 ? c.stream_len[bh] : 0u;
  if (base == kStreamPoisoned) return;
  uint16_t xv[T];
  load_token<T>(src, lane, xv);
  uint64_t bm[T];
  select_output_aware<T>(c.n_keep, xv, w, lane, bm);
  const int64_t tile0 = ((int64_t)bh * c.cap_tokens + tok) * T;
  uint64_t mine = bm[0];
#pragma unroll
  for (int t = 1; t < T; ++t) mine = (lane == (uint32_t)t) ? bm[t] : mine;
  if (lane < (uint32_t)T) c.bitmaps[tile0 + lane] = mine;
  const uint32_t used =
      pack_token<T>(xv, bm, base, c.values + (int64_t)bh * c.val_stride, c.offsets + tile0, lane);
  if (lane == 0) c.stream_len[bh] = base + used;
}

// Window step, one wave per stream: if the batch entry's window is full, its
// oldest token (slot head) goes to both compressed caches as token n_comp and
// the new token takes its slot; otherwise the new token goes to slot
// (head + len) % W. The per-entry counters advance in k_window_commit, after
// every stream of the entry has read them. WEIGHTED: the leaving key is pruned
// output-aware with its slot's accumulated weights kacc [BH][W][d], and the
// new token's weights start at 0.
template <int T, bool WEIGHTED = false>
__global__ __launch_bounds__(256) void k_window_step(CacheView kc, CacheView vc, WindowView w,
                                                     const uint16_t* __restrict__ k_new,
                                                     const uint16_t* __restrict__ v_new,
                                                     const int32_t* __restrict__ active,
                                                     float* __restrict__ kacc = nullptr) {
  constexpr int d = kTile * T;
  const int bh = blockIdx.x * (256 / kWave) + threadIdx.x / kWave;
  if (bh >= kc.BH) return;
  const int b = bh / w.H;
  if (active != nullptr && active[b] == 0) return;
  const uint32_t lane = lane_id();
  const int len = w.len[b], head = w.head[b];
  if (len < 0 || len > w.W || head < 0 || head >= w.W) return;  // not a state these calls produce
  uint16_t* kr = w.k + (int64_t)bh * w.W * d;
  uint16_t* vr = w.v + (int64_t)bh * w.W * d;
  int slot = (head + len) % w.W;
  if (len >= w.W) {
    slot = head;
    const int tok = w.n_comp[b];
    if (tok >= 0 && tok < kc.cap_tokens && tok < vc.cap_tokens) {  // guaranteed by the host's bound
      if constexpr (WEIGHTED)
        append_one_weighted<T>(kc, bh, tok, kr + (int64_t)slot * d, kacc + ((int64_t)bh * w.W + slot) * d,
                               lane);
      else
        append_one<T>(kc, bh, tok, kr + (int64_t)slot * d, lane);
      append_one<T>(vc, bh, tok, vr + (int64_t)slot * d, lane);
    }
  }
  // The old token was consumed above (its loads feed the selection), so the
  // slot can take the new one.
#pragma unroll
  for (int t = 0; t < T; ++t) {
    kr[(int64_t)slot * d + kTile * t + lane] = k_new[(int64_t)bh * d + kTile * t + lane];
    vr[(int64_t)slot * d + kTile * t + lane] = v_new[(int64_t)bh * d + kTile * t + lane];
    if constexpr (WEIGHTED) kacc[((int64_t)bh * w.W + slot) * d + kTile * t + lane] = 0.f;
  }
}

// Output-aware key weights of the window (see mustafar_window_key_weights): a
// 256-thread block per (entry, kv-head); a thread owns four channels of some of
// the newest kKeyWeightSteps slots, loads all of them before it adds and
// stores (no load waits on a store), and adds the |q| of the G query heads one
// by one, head order. An entry that is not active in this step has no query
// of its own here and gathers nothing.
constexpr int kKeyWeightSteps = 32;

template <int T>
__global__ __launch_bounds__(256) void k_window_key_weights(WindowView w, const uint16_t* __restrict__ q,
                                                            int G, const int32_t* __restrict__ active,
                                                            float* __restrict__ kacc) {
  constexpr int d = kTile * T;
  constexpr int C4 = d / 4;                  // four-channel columns per slot
  constexpr int ROWS = 256 / C4;             // slots per pass of the block
  constexpr int PASSES = kKeyWeightSteps / ROWS;
  const int bh = blockIdx.x;
  const int b = bh / w.H;
  if (active != nullptr && active[b] == 0) return;
  const int len = w.len[b], head = w.head[b];
  if (len <= 0 || len > w.W || head < 0 || head >= w.W) return;
  const int c4 = (int)threadIdx.x % C4, r0 = (int)threadIdx.x / C4;
  const int n = min(len, kKeyWeightSteps), p0 = len - n;
  float aq[8][4];
#pragma unroll
  for (int g = 0; g < 8; ++g) {
    uint2 h2 = {0u, 0u};
    if (g < G) h2 = *reinterpret_cast<const uint2*>(q + ((int64_t)bh * G + g) * d + 4 * c4);
    aq[g][0] = fabsf(half_bits_to_float((uint16_t)h2.x));
    aq[g][1] = fabsf(half_bits_to_float((uint16_t)(h2.x >> 16)));
    aq[g][2] = fabsf(half_bits_to_float((uint16_t)h2.y));
    aq[g][3] = fabsf(half_bits_to_float((uint16_t)(h2.y >> 16)));
  }
  float4 v[PASSES];
  float4* a[PASSES];
#pragma unroll
  for (int i = 0; i < PASSES; ++i) {
    const int r = r0 + ROWS * i;
    a[i] = r < n ? reinterpret_cast<float4*>(kacc + ((int64_t)bh * w.W + (head + p0 + r) % w.W) * d) + c4
                 : nullptr;
    if (a[i]) v[i] = *a[i];
  }
#pragma unroll
  for (int i = 0; i < PASSES; ++i) {
    if (!a[i]) continue;
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      if (g < G) {
        v[i].x += aq[g][0];
        v[i].y += aq[g][1];
        v[i].z += aq[g][2];
        v[i].w += aq[g][3];
      }
    }
    *a[i] = v[i];
  }
}

__global__ void k_window_commit(WindowView w, const int32_t* __restrict__ active) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= w.B || (active != nullptr && active[b] == 0)) return;
  if (w.len[b] < 0 || w.len[b] > w.W || w.head[b] < 0 || w.head[b] >= w.W) return;
  if (w.len[b] >= w.W) {
    w.head[b] = (w.head[b] + 1) % w.W;
    w.n_comp[b] += 1;
  } else {
    w.len[b] += 1;
  }
}

// Grouped window step, one wave per stream (see mustafar_window_step_grouped):
// if the entry's window is full, its oldest 32 tokens go to kc pruned per token
// and to vc pruned per channel as one group, as tokens n_comp .. n_comp+31;
// then the new token takes slot (head + len) % W (= head after a graduation)
// and its score starts at 0. k_window_commit_grouped advances the entry.
template <int T, bool SCORED>
__global__ __launch_bounds__(256) void k_window_step_grouped(CacheView kc, CacheView vc, WindowView w,
                                                             const uint16_t* __restrict__ k_new,
                                                             const uint16_t* __restrict__ v_new,
                                                             const int32_t* __restrict__ active,
                                                             float* __restrict__ acc) {
  constexpr int d = kTile * T;
  const int bh = blockIdx.x * (256 / kWave) + threadIdx.x / kWave;
  if (bh >= kc.BH) return;
  const int b = bh / w.H;
  if (active != nullptr && active[b] == 0) return;
  const uint32_t lane = lane_id();
  const int len = w.len[b], head = w.head[b];
  if (len < 0 || len > w.W || head < 0 || head >= w.W) return;  // not a state these calls produce
  uint16_t* kr = w.k + (int64_t)bh * w.W * d;
  uint16_t* vr = w.v + (int64_t)bh * w.W * d;
  float* ac = acc != nullptr ? acc + (int64_t)bh * w.W : nullptr;
  const int slot = (head + len) % w.W;
  const int tok = w.n_comp[b];
  if (len >= w.W && tok >= 0 && tok + kGroup <= kc.cap_tokens && tok + kGroup <= vc.cap_tokens) {
    // Keys, one token at a time (the selection of mustafar_append); a poisoned
    // stream takes no more tokens.
    uint32_t base = tok > 0 ? kc.stream_len[bh] : 0u;
    for (int u = 0; u < kGroup && base != kStreamPoisoned; ++u) {
      uint16_t xv[T];
      load_token<T>(kr + (int64_t)((head + u) % w.W) * d, lane, xv);
      uint32_t mag[T];
#pragma unroll
      for (int t = 0; t < T; ++t) mag[t] = xv[t] & 0x7fffu;
      uint64_t bm[T];
      select_token<T>(mag, kc.n_keep, bm);
      const int64_t tile0 = ((int64_t)bh * kc.cap_tokens + tok + u) * T;
      uint64_t mine = bm[0];
#pragma unroll
      for (int t = 1; t < T; ++t) mine = (lane == (uint32_t)t) ? bm[t] : mine;
      if (lane < (uint32_t)T) kc.bitmaps[tile0 + lane] = mine;
      base += pack_token<T>(xv, bm, base, kc.values + (int64_t)bh * kc.val_stride, kc.offsets + tile0, lane);
    }
    if (lane == 0 && base != kStreamPoisoned) kc.stream_len[bh] = base;
    // Values: per-channel keep words over the group, then each token packed
    // with its tile bitmaps.
    uint32_t word[T];
#pragma unroll
    for (int t = 0; t < T; ++t) {
      uint32_t key[kGroup];
#pragma unroll
      for (int j = 0; j < kGroup; ++j) {
        const int sl = (head + j) % w.W;
        key[j] = channel_key<SCORED>(vr[(int64_t)sl * d + kTile * t + lane], SCORED ? ac[sl] : 0.f);
      }
      word[t] = channel_keep_word<SCORED ? 31 : 15>(key, vc.group_keep);
    }
    base = tok > 0 ? vc.stream_len[bh] : 0u;
    for (int u = 0; u < kGroup && base != kStreamPoisoned; ++u) {
      uint16_t xv[T];
      load_token<T>(vr + (int64_t)((head + u) % w.W) * d, lane, xv);
      uint64_t bm[T];
#pragma unroll
      for (int t = 0; t < T; ++t) bm[t] = ballot(((word[t] >> u) & 1u) != 0u);
      const int64_t tile0 = ((int64_t)bh * vc.cap_tokens + tok + u) * T;
      uint64_t mine = bm[0];
#pragma unroll
      for (int t = 1; t < T; ++t) mine = (lane == (uint32_t)t) ? bm[t] : mine;
      if (lane < (uint32_t)T) vc.bitmaps[tile0 + lane] = mine;
      base += pack_token<T>(xv, bm, base, vc.values + (int64_t)bh * vc.val_stride, vc.offsets + tile0, lane);
    }
    if (lane == 0 && base != kStreamPoisoned) vc.stream_len[bh] = base;
  }
  // The graduated tokens were consumed above, so their slots can be reused.
#pragma unroll
  for (int t = 0; t < T; ++t) {
    kr[(int64_t)slot * d + kTile * t + lane] = k_new[(int64_t)bh * d + kTile * t + lane];
    vr[(int64_t)slot * d + kTile * t + lane] = v_new[(int64_t)bh * d + kTile * t + lane];
  }
  if (ac != nullptr && lane == 0) ac[slot] = 0.f;
}

__global__ void k_window_commit_grouped(WindowView w, const int32_t* __restrict__ active) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= w.B || (active != nullptr && active[b] == 0)) return;
  if (w.len[b] < 0 || w.len[b] > w.W || w.head[b] < 0 || w.head[b] >= w.W) return;
  if (w.len[b] >= w.W) {
    w.head[b] = (w.head[b] + kGroup) % w.W;
    w.n_comp[b] += kGroup;
    w.len[b] -= kGroup - 1;
  } else {
    w.len[b] += 1;
  }
}

// Prefill of one batch entry's window: tokens [first, first + count) of each of
// its H streams (x: [H][x_stride][d]) into ring slots 0.., and its state.
__global__ __launch_bounds__(256) void k_window_fill(WindowView w, int b, int d,
                                                     const uint16_t* __restrict__ xk,
                                                     const uint16_t* __restrict__ xv,
                                                     int64_t x_stride, int first, int count) {
  const int64_t per_stream = (int64_t)count * d;
  const int64_t n = (int64_t)w.H * per_stream;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t h = i / per_stream, r = i % per_stream;
    const int64_t dst = ((int64_t)b * w.H + h) * w.W * d + r;
    const int64_t src = (h * x_stride + first) * d + r;
    w.k[dst] = xk[src];
    w.v[dst] = xv[src];
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    w.len[b] = count;
    w.head[b] = 0;
    w.n_comp[b] = first;
  }
}

// Clears the workspace, runs k_compress (PRESET: with the bitmaps already in the
// cache) and poisons the streams one of whose chunks gave up.
template <int T, bool PRESET>
static hipError_t compress_launch(const CacheView& c, const uint16_t* x, int n_new, int64_t x_stride,
                                  int tok0, uint32_t* ws, hipStream_t s, const PruneOpts& o,
                                  uint32_t max_polls) {
  const int n_chunks = (n_new + compress_chunk_tokens(T) - 1) / compress_chunk_tokens(T);
  const int64_t n_wg = (int64_t)c.BH * n_chunks;
  const CompressWs w = compress_ws(ws, c.BH, n_chunks);
  const int clear_blocks = (int)((w.words + 255) / 256 < 1024 ? (w.words + 255) / 256 : 1024);
  hipLaunchKernelGGL(k_clear, dim3(clear_blocks), dim3(256), 0, s, ws, w.words);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_compress<T, PRESET>), dim3((uint32_t)n_wg), dim3(compress_waves<T>() * kWave),
                     0, s, x, n_new, PRESET ? 0 : c.n_keep,
                     c.bitmaps, c.offsets, c.values, c.stream_len, c.cap_tokens, tok0, c.val_stride,
                     w.flags, w.ticket, n_chunks, x_stride, o, max_polls, w.bad, w.status);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_compress_finalize, dim3((c.BH + 255) / 256), dim3(256), 0, s, w.bad, c.stream_len,
                     c.BH);
  return hipGetLastError();
}

template <int T>
static hipError_t compress_T(const CacheView& c, const uint16_t* x, int n_new, int64_t x_stride,
                             int tok0, uint32_t* ws, hipStream_t s, const PruneOpts& o = PruneOpts{},
                             uint32_t max_polls = kLookbackPolls) {
  return compress_launch<T, false>(c, x, n_new, x_stride, tok0, ws, s, o, max_polls);
}

template <int T>
static hipError_t append_T(const CacheView& c, const uint16_t* x, int tok0, hipStream_t s) {
  dim3 grid((c.BH + 3) / 4);
  hipLaunchKernelGGL(k_append<T>, grid, dim3(256), 0, s, c, x, tok0);
  return hipGetLastError();
}

template <int T>
static hipError_t window_step_T(const CacheView& kc, const CacheView& vc, const WindowView& w,
                                const uint16_t* k_new, const uint16_t* v_new, const int32_t* active,
                                hipStream_t s, float* kacc) {
  if (kacc != nullptr)
    hipLaunchKernelGGL((k_window_step<T, true>), dim3((kc.BH + 3) / 4), dim3(256), 0, s, kc, vc, w, k_new,
                       v_new, active, kacc);
  else
    hipLaunchKernelGGL((k_window_step<T, false>), dim3((kc.BH + 3) / 4), dim3(256), 0, s, kc, vc, w, k_new,
                       v_new, active, nullptr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_window_commit, dim3((w.B + 255) / 256), dim3(256), 0, s, w, active);
  return hipGetLastError();
}

hipError_t launch_compress(const CacheView& c, const uint16_t* x, int n_new, int tok0, uint32_t* ws,
                           hipStream_t s, int64_t x_stride, uint32_t max_polls) {
  if (x_stride <= 0) x_stride = n_new;
  switch (c.T) {
    case 1: return compress_T<1>(c, x, n_new, x_stride, tok0, ws, s, PruneOpts{}, max_polls);
    case 2: return compress_T<2>(c, x, n_new, x_stride, tok0, ws, s, PruneOpts{}, max_polls);
    case 4: return compress_T<4>(c, x, n_new, x_stride, tok0, ws, s, PruneOpts{}, max_polls);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_append(const CacheView& c, const uint16_t* x, int tok0, hipStream_t s) {
  switch (c.T) {
    case 1: return append_T<1>(c, x, tok0, s);
    case 2: return append_T<2>(c, x, tok0, s);
    case 4: return append_T<4>(c, x, tok0, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_append_kv(const CacheView& kc, const CacheView& vc, const uint16_t* k, const uint16_t* v,
                            int tok0, hipStream_t s) {
  const dim3 grid((2 * kc.BH + 3) / 4);
  switch (kc.T) {
    case 1: hipLaunchKernelGGL(k_append_kv<1>, grid, dim3(256), 0, s, kc, vc, k, v, tok0); break;
    case 2: hipLaunchKernelGGL(k_append_kv<2>, grid, dim3(256), 0, s, kc, vc, k, v, tok0); break;
    case 4: hipLaunchKernelGGL(k_append_kv<4>, grid, dim3(256), 0, s, kc, vc, k, v, tok0); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Offsets and packing of tokens whose bitmaps are already in the cache.
template <int T>
static hipError_t pack_preset_T(const CacheView& c, const uint16_t* x, int n_new, int64_t x_stride,
                                int tok0, uint32_t* ws, hipStream_t s, uint32_t max_polls = kLookbackPolls) {
  return compress_launch<T, true>(c, x, n_new, x_stride, tok0, ws, s, PruneOpts{}, max_polls);
}

template <int T>
static hipError_t compress_channel_T(const CacheView& c, const uint16_t* x, int n_new, int tok0,
                                     uint32_t* ws, hipStream_t s, const float* w, int64_t x_stride,
                                     uint32_t max_polls) {
  const int64_t waves = (int64_t)c.BH * (n_new / kGroup);
  const dim3 grid((uint32_t)((waves + 3) / 4));
  if (w != nullptr)
    hipLaunchKernelGGL((k_select_channel<T, true>), grid, dim3(256), 0, s, c, x, n_new, x_stride, tok0, w);
  else
    hipLaunchKernelGGL((k_select_channel<T, false>), grid, dim3(256), 0, s, c, x, n_new, x_stride, tok0, w);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return pack_preset_T<T>(c, x, n_new, x_stride, tok0, ws, s, max_polls);
}

hipError_t launch_compress_channel(const CacheView& c, const uint16_t* x, int n_new, int tok0,
                                   uint32_t* ws, hipStream_t s, const float* w, int64_t x_stride,
                                   uint32_t max_polls) {
  if (x_stride <= 0) x_stride = n_new;
  switch (c.T) {
    case 1: return compress_channel_T<1>(c, x, n_new, tok0, ws, s, w, x_stride, max_polls);
    case 2: return compress_channel_T<2>(c, x, n_new, tok0, ws, s, w, x_stride, max_polls);
    case 4: return compress_channel_T<4>(c, x, n_new, tok0, ws, s, w, x_stride, max_polls);
    default: return hipErrorInvalidValue;
  }
}

template <int T>
static hipError_t compress_variant_T(const CacheView& c, const uint16_t* x, int n_new, int tok0,
                                     uint32_t* ws, hipStream_t s, const PruneOpts& o) {
  // Magnitude pruning with a kept count per head is the bulk compressor with
  // its stream's count.
  if (o.mode == kPruneMagnitude) return compress_T<T>(c, x, n_new, (int64_t)n_new, tok0, ws, s, o);
  const int64_t waves = ((int64_t)c.BH * n_new + kTokPerWave - 1) / kTokPerWave;
  hipLaunchKernelGGL(k_select<T>, dim3((uint32_t)((waves + 3) / 4)), dim3(256), 0, s, c, x, n_new,
                     (int64_t)n_new, tok0, o);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return pack_preset_T<T>(c, x, n_new, (int64_t)n_new, tok0, ws, s);
}

hipError_t launch_compress_variant(const CacheView& c, const uint16_t* x, int n_new, int tok0,
                                   uint32_t* ws, hipStream_t s, const PruneOpts& o) {
  switch (c.T) {
    case 1: return compress_variant_T<1>(c, x, n_new, tok0, ws, s, o);
    case 2: return compress_variant_T<2>(c, x, n_new, tok0, ws, s, o);
    case 4: return compress_variant_T<4>(c, x, n_new, tok0, ws, s, o);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_append_variant(const CacheView& c, const uint16_t* x, int tok0, hipStream_t s,
                                 const PruneOpts& o) {
  dim3 grid((c.BH + 3) / 4);
  switch (c.T) {
    case 1: hipLaunchKernelGGL(k_append_variant<1>, grid, dim3(256), 0, s, c, x, tok0, o); break;
    case 2: hipLaunchKernelGGL(k_append_variant<2>, grid, dim3(256), 0, s, c, x, tok0, o); break;
    case 4: hipLaunchKernelGGL(k_append_variant<4>, grid, dim3(256), 0, s, c, x, tok0, o); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_query_lookahead(const uint16_t* q, int B, int Hq, int Hkv, int n_q, int T, int L,
                                  float* w, hipStream_t s) {
  const int G = Hq / Hkv;
  if (L == 32 && (G == 1 || G == 2 || G == 4 || G == 8)) {
    const int64_t n = (int64_t)B * Hkv * ((n_q + kLookRun - 1) / kLookRun) * kTile * T;
    const dim3 grid((uint32_t)((n + 255) / 256));
    const int d = kTile * T;
    switch (G) {
      case 1: hipLaunchKernelGGL(k_query_lookahead32<1>, grid, dim3(256), 0, s, q, B, Hkv, n_q, d, w); break;
      case 2: hipLaunchKernelGGL(k_query_lookahead32<2>, grid, dim3(256), 0, s, q, B, Hkv, n_q, d, w); break;
      case 4: hipLaunchKernelGGL(k_query_lookahead32<4>, grid, dim3(256), 0, s, q, B, Hkv, n_q, d, w); break;
      default: hipLaunchKernelGGL(k_query_lookahead32<8>, grid, dim3(256), 0, s, q, B, Hkv, n_q, d, w); break;
    }
    return hipGetLastError();
  }
  const int64_t n = (int64_t)B * Hkv * n_q * kTile * T;
  int blocks = (int)((n + 255) / 256);
  blocks = blocks < 1 ? 1 : (blocks > 65536 ? 65536 : blocks);
  hipLaunchKernelGGL(k_query_lookahead, dim3(blocks), dim3(256), 0, s, q, B, Hq, Hkv, n_q, kTile * T, L, w);
  return hipGetLastError();
}

hipError_t launch_window_fill(const WindowView& w, int b, int d, const uint16_t* xk,
                              const uint16_t* xv, int64_t x_stride, int first, int count,
                              hipStream_t s) {
  const int64_t n = (int64_t)w.H * count * d;
  int blocks = (int)((n + 255) / 256);
  blocks = blocks < 1 ? 1 : (blocks > 1024 ? 1024 : blocks);
  hipLaunchKernelGGL(k_window_fill, dim3(blocks), dim3(256), 0, s, w, b, d, xk, xv, x_stride, first,
                     count);
  return hipGetLastError();
}

template <int T>
static hipError_t window_step_grouped_T(const CacheView& kc, const CacheView& vc, const WindowView& w,
                                        const uint16_t* k_new, const uint16_t* v_new,
                                        const int32_t* active, float* acc, hipStream_t s) {
  const dim3 grid((kc.BH + 3) / 4);
  if (acc != nullptr)
    hipLaunchKernelGGL((k_window_step_grouped<T, true>), grid, dim3(256), 0, s, kc, vc, w, k_new, v_new,
                       active, acc);
  else
    hipLaunchKernelGGL((k_window_step_grouped<T, false>), grid, dim3(256), 0, s, kc, vc, w, k_new, v_new,
                       active, acc);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_window_commit_grouped, dim3((w.B + 255) / 256), dim3(256), 0, s, w, active);
  return hipGetLastError();
}

hipError_t launch_window_step_grouped(const CacheView& kc, const CacheView& vc, const WindowView& w,
                                      const uint16_t* k_new, const uint16_t* v_new,
                                      const int32_t* active, float* acc, hipStream_t s) {
  switch (kc.T) {
    case 1: return window_step_grouped_T<1>(kc, vc, w, k_new, v_new, active, acc, s);
    case 2: return window_step_grouped_T<2>(kc, vc, w, k_new, v_new, active, acc, s);
    case 4: return window_step_grouped_T<4>(kc, vc, w, k_new, v_new, active, acc, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_window_step(const CacheView& kc, const CacheView& vc, const WindowView& w,
                              const uint16_t* k_new, const uint16_t* v_new, const int32_t* active,
                              hipStream_t s, float* kacc) {
  switch (kc.T) {
    case 1: return window_step_T<1>(kc, vc, w, k_new, v_new, active, s, kacc);
    case 2: return window_step_T<2>(kc, vc, w, k_new, v_new, active, s, kacc);
    case 4: return window_step_T<4>(kc, vc, w, k_new, v_new, active, s, kacc);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_window_key_weights(const WindowView& w, const uint16_t* q, int G, int T,
                                     const int32_t* active, float* kacc, hipStream_t s) {
  const dim3 grid((uint32_t)(w.B * w.H));
  switch (T) {
    case 1: hipLaunchKernelGGL(k_window_key_weights<1>, grid, dim3(256), 0, s, w, q, G, active, kacc); break;
    case 2: hipLaunchKernelGGL(k_window_key_weights<2>, grid, dim3(256), 0, s, w, q, G, active, kacc); break;
    case 4: hipLaunchKernelGGL(k_window_key_weights<4>, grid, dim3(256), 0, s, w, q, G, active, kacc); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace mf
