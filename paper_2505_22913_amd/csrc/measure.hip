// Streaming ceilings the kernels are compared with.
//
// Read: each lane reads one 16-byte word per grid-stride step with a
// non-temporal load and XORs it; one checksum per workgroup keeps the loads
// alive. The rate of this kernel over a buffer much larger than the caches is
// the HBM read rate the decode kernels are compared with. A large grid with one
// word per lane and step, so that the words in flight at any moment form one
// compact front through the buffer, measured fastest on gfx950 (sweeps over
// 4096 to 2097152 workgroups of 256, one to 32 words per lane and step,
// temporal and non-temporal accesses, 8 GiB): reads 6.8-7.25 TB/s against
// 6.6-7.0 with 16384 workgroups and eight words in flight per lane one grid
// apart; a read that also writes 9/16 of its bytes 5.9-6.1 TB/s against
// 5.0-5.2.
#include "mustafar.h"
#include "mf_device.h"

namespace mf {

typedef uint32_t u32x4m __attribute__((ext_vector_type(4)));

constexpr int kReadBlocks = 524288;
constexpr int kReadThreads = 256;

__device__ __forceinline__ void block_checksum(uint32_t acc, uint32_t* __restrict__ sink) {
  __shared__ uint32_t red[kReadThreads / kWave];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o, kWave);
  if (lane_id() == 0) red[threadIdx.x / kWave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

__global__ __launch_bounds__(kReadThreads) void k_stream_read(const u32x4m* __restrict__ src,
                                                              int64_t n16, uint32_t* __restrict__ sink) {
  uint32_t acc = 0;
  const int64_t g = (int64_t)gridDim.x * kReadThreads;
  for (int64_t i = (int64_t)blockIdx.x * kReadThreads + threadIdx.x; i < n16; i += g) {
    const u32x4m a = __builtin_nontemporal_load(&src[i]);
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  block_checksum(acc, sink);
}

// Streaming read + write: every word is read (and XORed into the workgroup's
// checksum, like the read ceiling); of every 16 consecutive 16-byte words the
// first w16 are also written, packed, to dst (word i of group g at
// g * w16 + i), so dst receives w16/16 of the bytes read, interleaved with the
// reads the way a compressing pass writes its output.
__global__ __launch_bounds__(kReadThreads) void k_stream_mix(const u32x4m* __restrict__ src, int64_t n16,
                                                             u32x4m* __restrict__ dst, int w16,
                                                             uint32_t* __restrict__ sink) {
  uint32_t acc = 0;
  const int64_t g = (int64_t)gridDim.x * kReadThreads;
  for (int64_t i = (int64_t)blockIdx.x * kReadThreads + threadIdx.x; i < n16; i += g) {
    const u32x4m a = __builtin_nontemporal_load(&src[i]);
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
    if ((int)(i & 15) < w16) __builtin_nontemporal_store(a, &dst[(i >> 4) * w16 + (i & 15)]);
  }
  block_checksum(acc, sink);
}

// Streaming read + write in the bulk compression's access order: the buffer
// holds n_streams streams of chunks of 16 KiB (stream-major); workgroup g (two
// waves, like a compression chunk at d = 128) takes stream g % n_streams, chunk
// g / n_streams -- the streams take turns chunk by chunk, as the compression's
// workgroups do for its look-back -- reads its chunk with 16-byte non-temporal
// loads (eight per lane), writes the first w16/16 of the chunk's words, packed,
// to the chunk's place in dst, and its checksum to sink[g]. It has the
// compression's bytes and order and none of its arithmetic.
constexpr int kChunkBytes = MUSTAFAR_STREAM_CHUNK_BYTES;
constexpr int kChunkThreads = 128;

__global__ __launch_bounds__(kChunkThreads) void k_stream_chunks(const u32x4m* __restrict__ src,
                                                                 u32x4m* __restrict__ dst, int n_streams,
                                                                 int w16, uint32_t* __restrict__ sink) {
  constexpr int P = kChunkBytes / 16;    // words per chunk
  constexpr int kIt = P / kChunkThreads;  // words per lane
  const int64_t g = blockIdx.x;
  const int64_t n_chunks = gridDim.x / (uint32_t)n_streams;
  const int64_t chunk = (g % n_streams) * n_chunks + g / n_streams;
  const u32x4m* in = src + chunk * P;
  const int out_p = P * w16 / 16;
  u32x4m* out = dst + chunk * out_p;
  u32x4m r[kIt];
#pragma unroll
  for (int i = 0; i < kIt; ++i) r[i] = __builtin_nontemporal_load(&in[i * kChunkThreads + threadIdx.x]);
  uint32_t acc = 0;
#pragma unroll
  for (int i = 0; i < kIt; ++i) {
    const int p = i * kChunkThreads + (int)threadIdx.x;
    if (p < out_p) __builtin_nontemporal_store(r[i], &out[p]);
    acc ^= r[i].x ^ r[i].y ^ r[i].z ^ r[i].w;
  }
  __shared__ uint32_t red[kChunkThreads / kWave];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o, kWave);
  if (lane_id() == 0) red[threadIdx.x / kWave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[g] = red[0] ^ red[1];
}

}  // namespace mf

extern "C" int mustafar_stream_chunks(const void* src, int n_streams, int n_chunks, void* dst,
                                      int write_16ths, void* sink, void* stream) {
  if (!src || !dst || !sink || ((uintptr_t)src % 16) != 0 || ((uintptr_t)dst % 16) != 0 ||
      ((uintptr_t)sink % 4) != 0 || n_streams < 1 || n_chunks < 1 ||
      (int64_t)n_streams * n_chunks > 0x7fffffff || write_16ths < 0 || write_16ths > 16)
    return MUSTAFAR_EINVAL;
  hipLaunchKernelGGL(mf::k_stream_chunks, dim3((uint32_t)((int64_t)n_streams * n_chunks)),
                     dim3(mf::kChunkThreads), 0, (hipStream_t)stream,
                     reinterpret_cast<const mf::u32x4m*>(src), reinterpret_cast<mf::u32x4m*>(dst), n_streams,
                     write_16ths, reinterpret_cast<uint32_t*>(sink));
  return hipGetLastError() == hipSuccess ? MUSTAFAR_OK : MUSTAFAR_ELAUNCH;
}

extern "C" int mustafar_stream_mix(const void* src, size_t bytes, void* dst, int write_16ths, void* sink,
                                   void* stream) {
  if (!src || !dst || !sink || ((uintptr_t)src % 16) != 0 || ((uintptr_t)dst % 16) != 0 ||
      ((uintptr_t)sink % 4) != 0 || bytes % 256 != 0 || write_16ths < 0 || write_16ths > 16)
    return MUSTAFAR_EINVAL;
  hipLaunchKernelGGL(mf::k_stream_mix, dim3(mf::kReadBlocks), dim3(mf::kReadThreads), 0, (hipStream_t)stream,
                     reinterpret_cast<const mf::u32x4m*>(src), (int64_t)(bytes / 16),
                     reinterpret_cast<mf::u32x4m*>(dst), write_16ths, reinterpret_cast<uint32_t*>(sink));
  return hipGetLastError() == hipSuccess ? MUSTAFAR_OK : MUSTAFAR_ELAUNCH;
}

extern "C" size_t mustafar_stream_read_sink_bytes(void) {
  return (size_t)mf::kReadBlocks * sizeof(uint32_t);
}

extern "C" int mustafar_stream_read(const void* src, size_t bytes, void* sink, void* stream) {
  if (!src || !sink || ((uintptr_t)src % 16) != 0 || ((uintptr_t)sink % 4) != 0 || bytes % 16 != 0)
    return MUSTAFAR_EINVAL;
  hipLaunchKernelGGL(mf::k_stream_read, dim3(mf::kReadBlocks), dim3(mf::kReadThreads), 0,
                     (hipStream_t)stream, reinterpret_cast<const mf::u32x4m*>(src),
                     (int64_t)(bytes / 16), reinterpret_cast<uint32_t*>(sink));
  return hipGetLastError() == hipSuccess ? MUSTAFAR_OK : MUSTAFAR_ELAUNCH;
}
