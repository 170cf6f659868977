// Per-token magnitude pruning and bitmap compression on gfx950.
//
// One wavefront handles one token: lane i holds channel 64t+i of every tile t,
// so the keep-mask of a tile is exactly one 64-bit ballot (Sec. 3 tiles are
// 1x64 and the wavefront is 64 lanes wide). Selection of the n_keep largest
// magnitudes (Sec. 2, per-token magnitude pruning) is a most-significant-bit
// first radix select on the 15-bit fp16 magnitude with ballot+popcount counts,
// then ties at the threshold go to the lowest channels via mbcnt ranks. The
// packed position of a kept value inside its tile is mbcnt(bitmap) -- the
// number of kept lanes below it -- so the scatter is one masked store per tile.
//
// A stream's per-tile offsets are an exclusive prefix sum of the padded tile
// counts (Sec. 4.3 pads to 8). Bulk compression therefore runs in two launches:
// k_select writes the bitmaps and per-chunk padded totals, k_pack scans the
// totals, writes offsets and scatters the values (re-reading the dense tokens).
// k_append handles the one-token-per-stream case of a decode step in one launch.
#include "mf_device.h"
#include "mf_launch.h"

namespace mf {

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

// grid (n_chunks, BH), 256 threads: wave w handles tokens [64w, 64w+64) of the chunk.
template <int T>
__global__ __launch_bounds__(256) void k_select(const uint16_t* __restrict__ x, int n_new, int k,
                                                uint64_t* __restrict__ bitmaps, int cap_tokens,
                                                int tok0, uint32_t* __restrict__ chunk_tot,
                                                uint32_t* __restrict__ base_out,
                                                const uint32_t* __restrict__ stream_len,
                                                int n_chunks) {
  constexpr int d = kTile * T;
  const int chunk = blockIdx.x, bh = blockIdx.y;
  const uint32_t lane = lane_id();
  const int wave = threadIdx.x / kWave;
  const int j_begin = chunk * kCompressChunk + wave * kWave;
  const int j_end = min(j_begin + kWave, n_new);
  const uint16_t* xs = x + (int64_t)bh * n_new * d;
  uint64_t* bms = bitmaps + ((int64_t)bh * cap_tokens + tok0) * T;

  uint32_t total = 0;
  uint16_t cur[T], nxt[T];
  if (j_begin < j_end) load_token<T>(xs + (int64_t)j_begin * d, lane, cur);
  for (int j = j_begin; j < j_end; ++j) {
    if (j + 1 < j_end) load_token<T>(xs + (int64_t)(j + 1) * d, lane, nxt);
    uint32_t mag[T];
#pragma unroll
    for (int t = 0; t < T; ++t) mag[t] = cur[t] & 0x7fffu;
    uint64_t bm[T];
    select_token<T>(mag, k, bm);
    uint64_t mine = bm[0];
#pragma unroll
    for (int t = 1; t < T; ++t) mine = (lane == (uint32_t)t) ? bm[t] : mine;
    if (lane < (uint32_t)T) bms[(int64_t)j * T + lane] = mine;
#pragma unroll
    for (int t = 0; t < T; ++t) total += pad8((uint32_t)__popcll(bm[t]));
#pragma unroll
    for (int t = 0; t < T; ++t) cur[t] = nxt[t];
  }
  __shared__ uint32_t part[kCompressChunk / kWave];
  if (lane == 0) part[wave] = total;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t s = 0;
    for (int w = 0; w < kCompressChunk / kWave; ++w) s += part[w];
    chunk_tot[(int64_t)bh * n_chunks + chunk] = s;
    if (chunk == 0) base_out[bh] = tok0 > 0 ? stream_len[bh] : 0u;
  }
}

// grid (n_chunks, BH), 256 threads. Thread i first owns token i of the chunk
// for the offset scan; then wave w packs tokens [64w, 64w+64).
template <int T>
__global__ __launch_bounds__(256) void k_pack(const uint16_t* __restrict__ x, int n_new,
                                              const uint64_t* __restrict__ bitmaps,
                                              uint32_t* __restrict__ offsets,
                                              uint16_t* __restrict__ values,
                                              uint32_t* __restrict__ stream_len, int cap_tokens,
                                              int tok0, int64_t val_stride,
                                              const uint32_t* __restrict__ chunk_tot,
                                              const uint32_t* __restrict__ base_in, int n_chunks) {
  constexpr int d = kTile * T;
  constexpr int kWaves = kCompressChunk / kWave;
  const int chunk = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x;
  const uint32_t lane = lane_id();
  const int wave = tid / kWave;
  __shared__ uint32_t red[kWaves];
  __shared__ uint32_t start_of[kCompressChunk];
  __shared__ uint64_t bm_of[kCompressChunk][T];

  // Offset of this chunk inside the stream: base + totals of the earlier chunks.
  uint32_t s = 0;
  for (int i = tid; i < chunk; i += kCompressChunk) s += chunk_tot[(int64_t)bh * n_chunks + i];
  s = (uint32_t)wave_sum_i((int)s);
  if (lane == 0) red[wave] = s;
  __syncthreads();
  uint32_t chunk_base = base_in[bh];
  for (int w = 0; w < kWaves; ++w) chunk_base += red[w];
  __syncthreads();

  // Padded length of each token of the chunk and their exclusive scan.
  const int jt = chunk * kCompressChunk + tid;
  const uint64_t* bms = bitmaps + ((int64_t)bh * cap_tokens + tok0) * T;
  uint32_t len = 0;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const uint64_t b = (jt < n_new) ? bms[(int64_t)jt * T + t] : 0ull;
    bm_of[tid][t] = b;
    len += pad8((uint32_t)__popcll(b));
  }
  uint32_t incl = len;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t v = __shfl_up(incl, o, kWave);
    if (lane >= (uint32_t)o) incl += v;
  }
  if (lane == kWave - 1) red[wave] = incl;
  __syncthreads();
  uint32_t before = 0;
  for (int w = 0; w < wave; ++w) before += red[w];
  start_of[tid] = chunk_base + before + incl - len;
  if (tid == kCompressChunk - 1 && chunk == n_chunks - 1) stream_len[bh] = chunk_base + before + incl;
  __syncthreads();

  const uint16_t* xs = x + (int64_t)bh * n_new * d;
  uint16_t* vals = values + (int64_t)bh * val_stride;
  uint32_t* offs = offsets + ((int64_t)bh * cap_tokens + tok0) * T;
  const int j_begin = chunk * kCompressChunk + wave * kWave;
  const int j_end = min(j_begin + kWave, n_new);
  uint16_t cur[T], nxt[T];
  if (j_begin < j_end) load_token<T>(xs + (int64_t)j_begin * d, lane, cur);
  for (int j = j_begin; j < j_end; ++j) {
    if (j + 1 < j_end) load_token<T>(xs + (int64_t)(j + 1) * d, lane, nxt);
    const int jl = j - chunk * kCompressChunk;
    uint64_t bm[T];
#pragma unroll
    for (int t = 0; t < T; ++t) bm[t] = bm_of[jl][t];
    pack_token<T>(cur, bm, start_of[jl], vals, offs + (int64_t)j * T, lane);
#pragma unroll
    for (int t = 0; t < T; ++t) cur[t] = nxt[t];
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
  const int n_chunks = (n_new + kCompressChunk - 1) / kCompressChunk;
  uint32_t* chunk_tot = ws;
  uint32_t* base = ws + (int64_t)c.BH * n_chunks;
  dim3 grid(n_chunks, c.BH);
  hipLaunchKernelGGL(k_select<T>, grid, dim3(256), 0, s, x, n_new, c.n_keep, c.bitmaps,
                     c.cap_tokens, tok0, chunk_tot, base, c.stream_len, n_chunks);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_pack<T>, grid, dim3(256), 0, s, x, n_new, c.bitmaps, c.offsets, c.values,
                     c.stream_len, c.cap_tokens, tok0, c.val_stride, chunk_tot, base, n_chunks);
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
