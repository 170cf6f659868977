// Decode attention over compressed K/V plus a dense window (Algorithm 1) on gfx950.
//
// Split-K: every (batch, kv-head) stream is cut into token segments; a
// one-wave workgroup computes, for the G query heads of its kv-head, the
// running max, running sum and unnormalised output of one segment (online
// softmax), and k_merge combines the segments with their log-sum-exp weights.
// Compressed segments come first, then the dense window, so the softmax spans
// concat(S_C, S_L) exactly as Algorithm 1 states; the merge is order-free.
//
// Compressed blocks are handled "load as compressed, expand in LDS":
//   * the packed values of a block of NB = 64/T tokens are one contiguous run
//     of the stream; they are staged into LDS with 16-byte coalesced loads;
//   * lane (j, t) owns tile t of token j and walks the set bits of its bitmap,
//     reading its packed values in order: the q.k partial uses q from LDS, the
//     value tile is expanded into a dense LDS tile (zeros where pruned);
//   * p.V then runs with one lane per channel over the dense value tile.
// All arithmetic on fp16 data accumulates in fp32.
#include "mf_device.h"
#include "mf_launch.h"

namespace mf {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

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
};

__device__ __forceinline__ uint32_t first_set_and_clear(uint32_t& bits) {
  const uint32_t c = (uint32_t)__builtin_ctz(bits);
  bits &= bits - 1u;
  return c;
}

template <int T, int G>
__device__ __forceinline__ void softmax_update(float (&acc)[G], bool valid, uint32_t t, uint32_t j,
                                               float scale_log2, float (&m_run)[G],
                                               float (&l_run)[G], float (&o)[G][T],
                                               float* __restrict__ ps) {
#pragma unroll
  for (int sft = 1; sft < T; sft <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g] += __shfl_xor(acc[g], sft, kWave);
  }
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const float sc = valid ? acc[g] * scale_log2 : -INFINITY;
    const float mnew = fmaxf(m_run[g], wave_max(sc));
    const float alpha = __builtin_amdgcn_exp2f(m_run[g] - mnew);
    const float pj = valid ? __builtin_amdgcn_exp2f(sc - mnew) : 0.f;
    const float bsum = wave_sum(t == 0 ? pj : 0.f);
    l_run[g] = l_run[g] * alpha + bsum;
    m_run[g] = mnew;
#pragma unroll
    for (int tt = 0; tt < T; ++tt) o[g][tt] *= alpha;
    if (t == 0 && valid) ps[j * G + g] = pj;
  }
}

// grid (n_sparse_segs + n_dense_segs, BHkv), one wave per workgroup.
template <int T, int G>
__global__ __launch_bounds__(64) void k_attn_partial(AttnArgs a) {
  constexpr int d = kTile * T;
  constexpr int NB = kWave / T;  // tokens per block: lane = (token j, tile t)
  extern __shared__ __align__(16) unsigned char smem[];
  uint16_t* qs = reinterpret_cast<uint16_t*>(smem);                       // [G][d]
  float* ps = reinterpret_cast<float*>(smem + G * d * 2);                 // [NB][G]
  uint16_t* vdense = reinterpret_cast<uint16_t*>(smem + G * d * 2 + NB * G * 4);  // [NB][d]
  uint16_t* kst = vdense + NB * d;                                        // [NB*kmaxK]
  uint16_t* vst = kst + ((NB * a.kmaxK + 7) & ~7);                        // [NB*kmaxV]

  const int seg = blockIdx.x, bh = blockIdx.y;
  const uint32_t lane = lane_id();
  const uint32_t j = lane / T, t = lane % T;

  const uint16_t* qsrc = a.q + (int64_t)bh * G * d;
  for (int i = lane; i < G * d; i += kWave) qs[i] = qsrc[i];
  __syncthreads();

  float m_run[G], l_run[G], o[G][T];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m_run[g] = -INFINITY;
    l_run[g] = 0.f;
#pragma unroll
    for (int tt = 0; tt < T; ++tt) o[g][tt] = 0.f;
  }

  if (seg < a.n_sparse_segs) {
    const int j0 = seg * a.sparse_seg_tokens;
    const int j1 = min(j0 + a.sparse_seg_tokens, a.n_s);
    const int64_t kt0 = (int64_t)bh * a.K.cap_tokens * T;
    const int64_t vt0 = (int64_t)bh * a.V.cap_tokens * T;
    const uint16_t* kv = a.K.values + (int64_t)bh * a.K.val_stride;
    const uint16_t* vv = a.V.values + (int64_t)bh * a.V.val_stride;
    for (int b0 = j0; b0 < j1; b0 += NB) {
      const int nb = min(NB, j1 - b0);
      const bool valid = (int)j < nb;
      const int64_t ti = (int64_t)(b0 + (int)j) * T + t;
      const uint64_t kb = valid ? a.K.bitmaps[kt0 + ti] : 0ull;
      const uint32_t ko = valid ? a.K.offsets[kt0 + ti] : 0u;
      const uint64_t vb = valid ? a.V.bitmaps[vt0 + ti] : 0ull;
      const uint32_t vo = valid ? a.V.offsets[vt0 + ti] : 0u;
      // The block's packed values are the contiguous runs [kstart, kend), [vstart, vend).
      const uint32_t kstart = __builtin_amdgcn_readfirstlane(ko);
      const uint32_t vstart = __builtin_amdgcn_readfirstlane(vo);
      const uint32_t kend = __builtin_amdgcn_readlane(ko + pad8((uint32_t)__popcll(kb)), nb * T - 1);
      const uint32_t vend = __builtin_amdgcn_readlane(vo + pad8((uint32_t)__popcll(vb)), nb * T - 1);
      {
        const uint4* src = reinterpret_cast<const uint4*>(kv + kstart);
        uint4* dst = reinterpret_cast<uint4*>(kst);
        const int n16 = (int)(kend - kstart) / 8;
        for (int i = lane; i < n16; i += kWave) dst[i] = src[i];
      }
      {
        const uint4* src = reinterpret_cast<const uint4*>(vv + vstart);
        uint4* dst = reinterpret_cast<uint4*>(vst);
        const int n16 = (int)(vend - vstart) / 8;
        for (int i = lane; i < n16; i += kWave) dst[i] = src[i];
      }
      {
        uint4* dz = reinterpret_cast<uint4*>(vdense);
        for (int i = lane; i < NB * d / 8; i += kWave) dz[i] = make_uint4(0, 0, 0, 0);
      }
      __syncthreads();

      // Scores: lane (j, t) dots the kept entries of its key tile with q.
      float acc[G];
#pragma unroll
      for (int g = 0; g < G; ++g) acc[g] = 0.f;
      uint32_t pos = ko - kstart;
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        uint32_t bits = w ? (uint32_t)(kb >> 32) : (uint32_t)kb;
        const uint32_t cb = kTile * t + 32 * w;
        while (bits) {
          const uint32_t c = cb + first_set_and_clear(bits);
          const float kvf = half_bits_to_float(kst[pos++]);
#pragma unroll
          for (int g = 0; g < G; ++g) acc[g] = fmaf(half_bits_to_float(qs[g * d + c]), kvf, acc[g]);
        }
      }
      softmax_update<T, G>(acc, valid, t, j, a.scale_log2, m_run, l_run, o, ps);

      // Expand the value tile into the dense block, channel-interleaved [j][c*T + t].
      pos = vo - vstart;
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        uint32_t bits = w ? (uint32_t)(vb >> 32) : (uint32_t)vb;
        const uint32_t cb = 32 * w;
        while (bits) {
          const uint32_t c = cb + first_set_and_clear(bits);
          vdense[j * d + c * T + t] = vst[pos++];
        }
      }
      __syncthreads();

      // p.V: lane = channel, channels lane + 64*tt.
      for (int jj = 0; jj < nb; ++jj) {
        float pv[G];
#pragma unroll
        for (int g = 0; g < G; ++g) pv[g] = ps[jj * G + g];
#pragma unroll
        for (int tt = 0; tt < T; ++tt) {
          const float v = half_bits_to_float(vdense[jj * d + lane * T + tt]);
#pragma unroll
          for (int g = 0; g < G; ++g) o[g][tt] = fmaf(pv[g], v, o[g][tt]);
        }
      }
      __syncthreads();
    }
  } else {
    // Dense segment: the local window (or a range of a dense cache).
    const int dseg = seg - a.n_sparse_segs;
    const int j0 = dseg * a.dense_seg_tokens;
    const int j1 = min(j0 + a.dense_seg_tokens, a.n_dense);
    const uint16_t* kd = a.kd + (int64_t)bh * a.n_dense * d;
    const uint16_t* vd = a.vd + (int64_t)bh * a.n_dense * d;
    for (int b0 = j0; b0 < j1; b0 += NB) {
      const int nb = min(NB, j1 - b0);
      const bool valid = (int)j < nb;
      float acc[G];
#pragma unroll
      for (int g = 0; g < G; ++g) acc[g] = 0.f;
      if (valid) {
        const uint4* kr = reinterpret_cast<const uint4*>(kd + (int64_t)(b0 + (int)j) * d + kTile * t);
#pragma unroll
        for (int i = 0; i < kTile / 8; ++i) {
          const uint4 u = kr[i];
          const half2_t k2[4] = {__builtin_bit_cast(half2_t, u.x), __builtin_bit_cast(half2_t, u.y),
                                 __builtin_bit_cast(half2_t, u.z), __builtin_bit_cast(half2_t, u.w)};
#pragma unroll
          for (int g = 0; g < G; ++g) {
            const uint4 qq = *reinterpret_cast<const uint4*>(qs + g * d + kTile * t + 8 * i);
            acc[g] = __builtin_amdgcn_fdot2(k2[0], __builtin_bit_cast(half2_t, qq.x), acc[g], false);
            acc[g] = __builtin_amdgcn_fdot2(k2[1], __builtin_bit_cast(half2_t, qq.y), acc[g], false);
            acc[g] = __builtin_amdgcn_fdot2(k2[2], __builtin_bit_cast(half2_t, qq.z), acc[g], false);
            acc[g] = __builtin_amdgcn_fdot2(k2[3], __builtin_bit_cast(half2_t, qq.w), acc[g], false);
          }
        }
      }
      softmax_update<T, G>(acc, valid, t, j, a.scale_log2, m_run, l_run, o, ps);
      __syncthreads();
      for (int jj = 0; jj < nb; ++jj) {
        float pv[G];
#pragma unroll
        for (int g = 0; g < G; ++g) pv[g] = ps[jj * G + g];
        const uint16_t* vr = vd + (int64_t)(b0 + jj) * d;
#pragma unroll
        for (int tt = 0; tt < T; ++tt) {
          const float v = half_bits_to_float(vr[lane + kTile * tt]);
#pragma unroll
          for (int g = 0; g < G; ++g) o[g][tt] = fmaf(pv[g], v, o[g][tt]);
        }
      }
      __syncthreads();
    }
  }

  const int64_t row0 = (int64_t)seg * a.BHq + (int64_t)bh * G;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if (lane == 0) a.ws_ml[row0 + g] = make_float2(m_run[g], l_run[g]);
#pragma unroll
    for (int tt = 0; tt < T; ++tt) a.ws_o[(row0 + g) * d + lane + kTile * tt] = o[g][tt];
  }
}

// grid (BHq), one wave: log-sum-exp merge of the segments, fp16 output (RNE).
template <int T>
__global__ __launch_bounds__(64) void k_merge(const float2* __restrict__ ws_ml,
                                              const float* __restrict__ ws_o, int n_seg, int BHq,
                                              uint16_t* __restrict__ out) {
  constexpr int d = kTile * T;
  const int r = blockIdx.x;
  const uint32_t lane = lane_id();
  float M = -INFINITY;
  for (int s = 0; s < n_seg; ++s) M = fmaxf(M, ws_ml[(int64_t)s * BHq + r].x);
  float L = 0.f, acc[T];
#pragma unroll
  for (int tt = 0; tt < T; ++tt) acc[tt] = 0.f;
  for (int s = 0; s < n_seg; ++s) {
    const float2 ml = ws_ml[(int64_t)s * BHq + r];
    const float w = __builtin_amdgcn_exp2f(ml.x - M);
    L = fmaf(ml.y, w, L);
#pragma unroll
    for (int tt = 0; tt < T; ++tt)
      acc[tt] = fmaf(ws_o[((int64_t)s * BHq + r) * d + lane + kTile * tt], w, acc[tt]);
  }
  const float inv = 1.f / L;
#pragma unroll
  for (int tt = 0; tt < T; ++tt)
    out[(int64_t)r * d + lane + kTile * tt] = __builtin_bit_cast(uint16_t, (_Float16)(acc[tt] * inv));
}

static size_t partial_lds_bytes(int T, int G, int kmaxK, int kmaxV) {
  const int d = kTile * T, NB = kWave / T;
  size_t b = (size_t)G * d * 2 + (size_t)NB * G * 4 + (size_t)NB * d * 2;
  b += (size_t)((NB * kmaxK + 7) & ~7) * 2 + (size_t)NB * kmaxV * 2;
  return (b + 15) & ~size_t(15);
}

template <int T, int G>
static hipError_t attention_TG(const AttnShape& sh, const AttnArgs& a, uint16_t* out, hipStream_t s) {
  const int n_seg = sh.n_sparse_segs + sh.n_dense_segs;
  const size_t lds = partial_lds_bytes(T, G, a.kmaxK, a.kmaxV);
  hipLaunchKernelGGL((k_attn_partial<T, G>), dim3(n_seg, sh.BHkv), dim3(kWave), lds, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_merge<T>, dim3(a.BHq), dim3(kWave), 0, s, a.ws_ml, a.ws_o, n_seg, a.BHq, out);
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

static int token_max_elems_dev(int d, int k) {
  const int T = d / kTile;
  const int nonempty = k < T ? k : T;
  const int m = (k + (kPad - 1) * nonempty) / kPad * kPad;
  return m < d ? m : d;
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
  a.kmaxK = sh.n_sparse_segs > 0 ? token_max_elems_dev(d, K.n_keep) : 0;
  a.kmaxV = sh.n_sparse_segs > 0 ? token_max_elems_dev(d, V.n_keep) : 0;
  switch (sh.T) {
    case 1: return attention_T<1>(sh, a, out, s);
    case 2: return attention_T<2>(sh, a, out, s);
    case 4: return attention_T<4>(sh, a, out, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace mf
