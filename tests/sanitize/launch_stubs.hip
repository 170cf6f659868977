// Stand-ins for the kernel launchers of libmustafar (csrc/mf_launch.h) in the
// host-only sanitizer harness of the C ABI: they launch nothing and count the
// calls, so that every validated entry point can run to its end on a machine
// without a GPU while AddressSanitizer / UndefinedBehaviorSanitizer watch the
// host-side validation, geometry and descriptor bookkeeping of api.hip.
#include "mf_launch.h"

extern "C" long mf_stub_launches = 0;

namespace mf {

static hipError_t ok() { ++mf_stub_launches; return hipSuccess; }

hipError_t launch_compress(const CacheView&, const uint16_t*, int, int, uint32_t*, hipStream_t, int64_t,
                           uint32_t) { return ok(); }
hipError_t launch_append(const CacheView&, const uint16_t*, int, hipStream_t) { return ok(); }
hipError_t launch_append_kv(const CacheView&, const CacheView&, const uint16_t*, const uint16_t*, int,
                            hipStream_t) { return ok(); }
hipError_t launch_compress_variant(const CacheView&, const uint16_t*, int, int, uint32_t*, hipStream_t,
                                   const PruneOpts&) { return ok(); }
hipError_t launch_append_variant(const CacheView&, const uint16_t*, int, hipStream_t, const PruneOpts&) {
  return ok();
}
hipError_t launch_compress_channel(const CacheView&, const uint16_t*, int, int, uint32_t*, hipStream_t,
                                   const float*, int64_t, uint32_t) { return ok(); }
hipError_t launch_query_lookahead(const uint16_t*, int, int, int, int, int, int, float*, hipStream_t) {
  return ok();
}
hipError_t launch_window_fill(const WindowView&, int, int, const uint16_t*, const uint16_t*, int64_t, int,
                              int, hipStream_t) { return ok(); }
hipError_t launch_window_step(const CacheView&, const CacheView&, const WindowView&, const uint16_t*,
                              const uint16_t*, const int32_t*, hipStream_t, float*) { return ok(); }
hipError_t launch_window_key_weights(const WindowView&, const uint16_t*, int, int, const int32_t*, float*,
                                     hipStream_t) { return ok(); }
hipError_t launch_window_step_grouped(const CacheView&, const CacheView&, const WindowView&,
                                      const uint16_t*, const uint16_t*, const int32_t*, float*,
                                      hipStream_t) { return ok(); }
hipError_t launch_window_scores(const WindowView&, const uint16_t*, int, int, float, const float*,
                                const int32_t*, float*, hipStream_t) { return ok(); }
hipError_t launch_attention(const AttnShape& sh, const uint16_t*, const SparseSide&, const SparseSide&,
                            const uint16_t*, const uint16_t*, float* ws_ml, float* ws_o, uint16_t*,
                            hipStream_t) {
  // the partial layout the entry point computed must be ordered and non-empty
  if (sh.n_sparse_segs + sh.n_dense_segs <= 0 || ws_o <= ws_ml) return hipErrorInvalidValue;
  return ok();
}

}  // namespace mf
