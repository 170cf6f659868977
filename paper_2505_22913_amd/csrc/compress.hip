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
// step.
#include "mf_device.h"
#include "mf_launch.h"

namespace mf {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Keep-mask of one token. mag[t] is the fp16 magnitude (bits & 0x7fff) of this
// lane's channel in tile t. Sets bm[t] (wave-uniform) so that exactly k bits
// are set over the T tiles: the k largest magnitudes, ties to lower channels.
template <int T>
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
  // Largest threshold m with #{mag >= m} >= k: that is the k-th largest magnitude.
  uint32_t thr = 0;
#pragma unroll
  for (int b = 14; b >= 0; --b) {
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
constexpr uint32_t kSpinLimit = 1u << 20;     // polls before a chunk gives up (never reached)
constexpr uint32_t kBadBase = 0xffffffffu;

__global__ void k_clear(uint32_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// The flag words are the only data workgroups exchange (the count travels in
// the same 64-bit word as the status, and no workgroup reads what another one
// writes to the cache), so relaxed device-scope atomics suffice: acquire and
// release would write back and invalidate the whole L2 of the XCD on every poll.
//
// Offset in the stream at which chunk `chunk` starts, computed by one whole
// wave. The chunk's total is published first; then the wave reads the flags of
// the 64 chunks before it at once and adds, from the nearest one back, the
// totals up to and including the first known prefix, moving 64 chunks further
// back while none is found. Chunks with lower tickets are already running and
// publish their totals without waiting, so every poll is eventually answered;
// the poll count is bounded anyway.
__device__ uint32_t look_back(uint64_t* __restrict__ fl, int chunk, uint32_t total,
                              uint32_t first_base, uint32_t lane) {
  if (chunk == 0) {
    if (lane == 0)
      __hip_atomic_store(fl, kFlagPrefix | (uint64_t)(first_base + total), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    return first_base;
  }
  if (lane == 0)
    __hip_atomic_store(fl + chunk, kFlagAgg | (uint64_t)total, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  uint32_t acc = 0, polls = 0;
  for (int top = chunk - 1;;) {
    const int p = top - (int)lane;
    // Positions before chunk 0 read as a known prefix of 0.
    const uint64_t f = p >= 0 ? __hip_atomic_load(fl + p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                              : kFlagPrefix;
    const uint32_t st = (uint32_t)(f >> 62);
    const uint64_t pref = ballot(st == 2u);
    const uint64_t none = ballot(st == 0u);
    const uint32_t first = pref ? (uint32_t)__builtin_ctzll(pref) : 64u;  // nearest prefix
    const uint64_t upto = first >= 63u ? ~0ull : ((2ull << first) - 1ull);
    if (none & upto) {  // a chunk between here and that prefix has not published yet
      if (++polls > kSpinLimit) return kBadBase;
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

// 1-D grid of BH * n_chunks workgroups of 4 waves; a chunk is 4 * 64/T tokens of
// one stream, each wave owning 64/T of them (4096 fp16 values, 8 KiB of LDS).
template <int T>
__global__ __launch_bounds__(256) void k_compress(const uint16_t* __restrict__ x, int n_new, int k,
                                                  uint64_t* __restrict__ bitmaps,
                                                  uint32_t* __restrict__ offsets,
                                                  uint16_t* __restrict__ values,
                                                  uint32_t* __restrict__ stream_len, int cap_tokens,
                                                  int tok0, int64_t val_stride,
                                                  uint64_t* __restrict__ flags,
                                                  uint32_t* __restrict__ ticket_ctr, int n_chunks) {
  constexpr int d = kTile * T;
  constexpr int kTPW = kWave / T;            // tokens per wave
  constexpr int kCH = 4 * kTPW;              // tokens per chunk
  constexpr int kRegion = kTPW * d;          // fp16 values per wave region
  __shared__ __align__(16) uint16_t s_x[4][kRegion];  // dense tokens, packed in place
  __shared__ uint64_t s_bm[4][kTPW * T];
  __shared__ uint32_t s_loc[4][kTPW * T];    // tile offsets relative to the wave's run
  __shared__ uint32_t s_wtot[4];
  __shared__ uint32_t s_ticket, s_base;

  const int tid = threadIdx.x;
  const uint32_t lane = lane_id();
  const int wave = tid / kWave;
  if (tid == 0) s_ticket = atomicAdd(ticket_ctr, 1u);
  __syncthreads();
  const int ticket = (int)s_ticket;
  const int bh = ticket / n_chunks, chunk = ticket % n_chunks;
  const int j0 = chunk * kCH + wave * kTPW;
  const int nt = max(0, min(kTPW, n_new - j0));

  // Stage the wave's tokens: 16-byte coalesced loads, 8 per lane. Every load
  // is issued (lanes past the wave's tokens re-read its first 16 bytes) so the
  // staging registers are written unconditionally.
  if (nt > 0) {
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(x + ((int64_t)bh * n_new + j0) * d);
    u32x4_t* dst = reinterpret_cast<u32x4_t*>(s_x[wave]);
    const int n16 = nt * d / 8;
    u32x4_t r[kRegion / 8 / kWave];
#pragma unroll
    for (int i = 0; i < kRegion / 8 / kWave; ++i) {
      const int c = i * kWave + (int)lane;
      r[i] = src[c < n16 ? c : 0];
    }
#pragma unroll
    for (int i = 0; i < kRegion / 8 / kWave; ++i) {
      const int c = i * kWave + (int)lane;
      if (c < n16) dst[c] = r[i];
    }
  }

  // Select and pack token by token (a wave's LDS operations run in order, so a
  // token's packed values may overwrite its own dense values once read; they
  // never reach later tokens because a token packs into at most d values).
  uint16_t* reg = s_x[wave];
  uint32_t run = 0;
  for (int i = 0; i < nt; ++i) {
    uint16_t xv[T];
    uint32_t mag[T];
#pragma unroll
    for (int t = 0; t < T; ++t) {
      xv[t] = reg[i * d + kTile * t + lane];
      mag[t] = xv[t] & 0x7fffu;
    }
    uint64_t bm[T];
    select_token<T>(mag, k, bm);
    uint32_t pos = run;
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const uint32_t cnt = (uint32_t)__popcll(bm[t]);
      const uint32_t below = mbcnt(bm[t], 0u);
      const bool kept = (bm[t] >> lane) & 1ull;
      const uint32_t pad_slot = cnt + (lane - below);  // k-th dropped lane fills pad slot k
      if (kept) reg[pos + below] = xv[t];
      else if (pad_slot < pad8(cnt)) reg[pos + pad_slot] = 0;
      if (lane == (uint32_t)t) {
        s_bm[wave][i * T + t] = bm[t];
        s_loc[wave][i * T + t] = pos;
      }
      pos += pad8(cnt);
    }
    run = pos;
  }
  if (lane == 0) s_wtot[wave] = run;
  __syncthreads();

  if (wave == 0) {
    const uint32_t total = s_wtot[0] + s_wtot[1] + s_wtot[2] + s_wtot[3];
    const uint32_t first = (chunk == 0 && tok0 > 0) ? stream_len[bh] : 0u;
    const uint32_t base = look_back(flags + (int64_t)bh * n_chunks, chunk, total, first, lane);
    if (lane == 0) {
      s_base = base;
      if (chunk == n_chunks - 1) stream_len[bh] = base == kBadBase ? kBadBase : base + total;
    }
  }
  __syncthreads();
  if (s_base == kBadBase) return;  // look-back gave up: nothing is written
  uint32_t wbase = s_base;
  for (int w = 0; w < wave; ++w) wbase += s_wtot[w];

  // Packed run (a multiple of 8 values, 16-byte aligned in the stream).
  {
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(reg);
    u32x4_t* dst = reinterpret_cast<u32x4_t*>(values + (int64_t)bh * val_stride + wbase);
    for (uint32_t c = lane; c < run / 8; c += kWave) dst[c] = src[c];
  }
  // Bitmaps and offsets of the wave's tiles (tile index = token * T + t).
  const int64_t tile0 = ((int64_t)bh * cap_tokens + tok0 + j0) * T;
  if ((int)lane < nt * T) {
    bitmaps[tile0 + lane] = s_bm[wave][lane];
    offsets[tile0 + lane] = wbase + s_loc[wave][lane];
  }
}

// One wave per stream, 4 streams per 256-thread block.
template <int T>
__global__ __launch_bounds__(256) void k_append(const uint16_t* __restrict__ x, int BH, int k,
                                                uint64_t* __restrict__ bitmaps,
                                                uint32_t* __restrict__ offsets,
                                                uint16_t* __restrict__ values,
                                                uint32_t* __restrict__ stream_len, int cap_tokens,
                                                int tok0, int64_t val_stride) {
  constexpr int d = kTile * T;
  const int bh = blockIdx.x * (256 / kWave) + threadIdx.x / kWave;
  if (bh >= BH) return;
  const uint32_t lane = lane_id();
  const uint32_t base = tok0 > 0 ? stream_len[bh] : 0u;
  uint16_t xv[T];
  load_token<T>(x + (int64_t)bh * d, lane, xv);
  uint32_t mag[T];
#pragma unroll
  for (int t = 0; t < T; ++t) mag[t] = xv[t] & 0x7fffu;
  uint64_t bm[T];
  select_token<T>(mag, k, bm);
  const int64_t tile0 = ((int64_t)bh * cap_tokens + tok0) * T;
  uint64_t mine = bm[0];
#pragma unroll
  for (int t = 1; t < T; ++t) mine = (lane == (uint32_t)t) ? bm[t] : mine;
  if (lane < (uint32_t)T) bitmaps[tile0 + lane] = mine;
  const uint32_t used =
      pack_token<T>(xv, bm, base, values + (int64_t)bh * val_stride, offsets + tile0, lane);
  if (lane == 0) stream_len[bh] = base + used;
}

template <int T>
static hipError_t compress_T(const CacheView& c, const uint16_t* x, int n_new, int tok0,
                             uint32_t* ws, hipStream_t s) {
  const int n_chunks = (n_new + compress_chunk_tokens(T) - 1) / compress_chunk_tokens(T);
  const int64_t n_wg = (int64_t)c.BH * n_chunks;
  uint64_t* flags = reinterpret_cast<uint64_t*>(ws);
  uint32_t* ticket = reinterpret_cast<uint32_t*>(flags + n_wg);
  const int64_t words = 2 * n_wg + 1;
  const int clear_blocks = (int)((words + 255) / 256 < 1024 ? (words + 255) / 256 : 1024);
  hipLaunchKernelGGL(k_clear, dim3(clear_blocks), dim3(256), 0, s, ws, words);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_compress<T>, dim3((uint32_t)n_wg), dim3(256), 0, s, x, n_new, c.n_keep,
                     c.bitmaps, c.offsets, c.values, c.stream_len, c.cap_tokens, tok0, c.val_stride,
                     flags, ticket, n_chunks);
  return hipGetLastError();
}

template <int T>
static hipError_t append_T(const CacheView& c, const uint16_t* x, int tok0, hipStream_t s) {
  dim3 grid((c.BH + 3) / 4);
  hipLaunchKernelGGL(k_append<T>, grid, dim3(256), 0, s, x, c.BH, c.n_keep, c.bitmaps, c.offsets,
                     c.values, c.stream_len, c.cap_tokens, tok0, c.val_stride);
  return hipGetLastError();
}

hipError_t launch_compress(const CacheView& c, const uint16_t* x, int n_new, int tok0, uint32_t* ws,
                           hipStream_t s) {
  switch (c.T) {
    case 1: return compress_T<1>(c, x, n_new, tok0, ws, s);
    case 2: return compress_T<2>(c, x, n_new, tok0, ws, s);
    case 4: return compress_T<4>(c, x, n_new, tok0, ws, s);
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

}  // namespace mf
