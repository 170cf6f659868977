// C ABI of libmustafar (declared in include/mustafar.h): host-side validation,
// launch geometry and workspace layout. Every check runs before any launch, so
// an invalid call enqueues nothing and never touches the GPU.
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "mf_launch.h"
#include "mustafar.h"

// Static device scratch of mustafar_sparse_decode_attn_static: the split-K
// partials of a decode call live here instead of in a caller workspace. Each
// GPU the library runs on holds its own copy until the process ends. In host
// code `scratch` is only a stand-in for the symbol: its device address comes
// from hipGetSymbolAddress (once per device, below) and only that address is
// ever passed to a kernel.
static __device__ __align__(256) unsigned char scratch[MUSTAFAR_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kTile = MUSTAFAR_TILE;
constexpr int kPad = MUSTAFAR_PAD;
constexpr int kMaxGrid = 65535;            // grid.y limit for the stream index
// Default decode splits, from split sweeps over the decode workloads. The walk
// kernel (one query head per kv-head, one wave per segment, 16 resident waves
// per CU) takes about eight rounds of resident waves: from 32 to 128 segments
// per stream on 512 streams of 32K tokens the call time moves by under 1.5%,
// and small batches gain from segments as short as one block; the
// grouped-query kernels want fewer, longer segments.
constexpr int kWalkTargetGroups = 32768;
constexpr int kWalkMinSegTokens = 64;
constexpr int kWalkGroupedTargetGroups = 4096;  // the walks with 2 or 4 query heads per kv-head,
constexpr int kWalkGroupedMinSegTokens = 192;   // segments of at least 192 tokens
constexpr int kMfmaMinGroup = 8;                // the matrix-core kernel from 8 on (attn_common.h)
constexpr int kMfmaTargetGroups = 2048;
constexpr int kDenseGroupedTargetGroups = 4096;
constexpr int kGroupedMinSegTokens = 128;
constexpr int kSegAlign = 64;              // segments are whole 64-token blocks
constexpr int kKeyWeightSteps = 32;        // output-aware keys: the current and 31 next queries
static_assert(MUSTAFAR_LOOKBACK_POLLS == mf::kLookbackPolls, "look-back bound");
static_assert(MUSTAFAR_STREAM_POISONED == mf::kStreamPoisoned, "poisoned stream marker");

// Kernel route of grouped queries (mustafar_attn_set_route), process-wide.
std::atomic<int> g_route{MUSTAFAR_ROUTE_DEFAULT};

// Whether a sparse call with G query heads per kv-head runs its compressed
// segments on the matrix-core kernel.
bool mfma_route(int G, int route) {
  if (G < 2) return false;
  if (route == MUSTAFAR_ROUTE_WALKS) return false;
  if (route == MUSTAFAR_ROUTE_MATRIX_CORES) return true;
  return G >= kMfmaMinGroup;
}

bool aligned(const void* p, uintptr_t a) { return p && ((uintptr_t)p % a) == 0; }
bool head_dim_ok(int d) { return d == 64 || d == 128 || d == 256; }

int status_of(hipError_t e) { return e == hipSuccess ? MUSTAFAR_OK : MUSTAFAR_ELAUNCH; }

// Device address of `scratch` on the current device, looked up at the first call
// on that device and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return MUSTAFAR_ELAUNCH;
  if (dev < 0 || dev >= kMaxDevices) return MUSTAFAR_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return MUSTAFAR_ELAUNCH;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MUSTAFAR_OK;
}

int check_cache(const mustafar_ccache_t* c) {
  if (!c) return MUSTAFAR_EINVAL;
  if (!aligned(c->bitmaps, 8) || !aligned(c->offsets, 4) || !aligned(c->values, 16) ||
      !aligned(c->stream_len, 4))
    return MUSTAFAR_EINVAL;
  if (c->B < 1 || c->H < 1 || (int64_t)c->B * c->H > kMaxGrid) return MUSTAFAR_EINVAL;
  if (!head_dim_ok(c->d)) return MUSTAFAR_EINVAL;
  if (c->n_keep < 0 || c->n_keep > c->d) return MUSTAFAR_EINVAL;
  if (c->cap_tokens < 1 || c->n_tokens < 0 || c->n_tokens > c->cap_tokens) return MUSTAFAR_EINVAL;
  if (c->group_keep < -1 || c->group_keep > mf::kGroup) return MUSTAFAR_EINVAL;
  const int64_t need = c->group_keep >= 0
                           ? mustafar_grouped_stream_capacity(c->d, c->group_keep, c->cap_tokens)
                           : mustafar_stream_capacity(c->d, c->n_keep, c->cap_tokens);
  if (c->val_stride % kPad != 0 || c->val_stride < need) return MUSTAFAR_EINVAL;
  // Offsets and stream lengths are u32, and the largest u32 marks a poisoned stream.
  if (need >= (int64_t)mf::kStreamPoisoned) return MUSTAFAR_EUNSUPPORTED;
  return MUSTAFAR_OK;
}

bool grouped(const mustafar_ccache_t* c) { return c->group_keep >= 0; }

mf::CacheView view_of(const mustafar_ccache_t* c) {
  mf::CacheView v;
  v.bitmaps = c->bitmaps;
  v.offsets = c->offsets;
  v.values = c->values;
  v.stream_len = c->stream_len;
  v.BH = c->B * c->H;
  v.T = c->d / kTile;
  v.n_keep = c->n_keep;
  v.cap_tokens = c->cap_tokens;
  v.val_stride = c->val_stride;
  v.group_keep = c->group_keep;
  return v;
}

mf::SparseSide side_of(const mustafar_ccache_t* c) {
  mf::SparseSide s;
  s.bitmaps = c->bitmaps;
  s.offsets = c->offsets;
  s.values = c->values;
  s.stream_len = c->stream_len;
  s.val_stride = c->val_stride;
  s.cap_tokens = c->cap_tokens;
  s.n_keep = c->n_keep;
  s.group_keep = c->group_keep;
  return s;
}

constexpr int kMaxWindow = 1024;  // window slots per stream (one attention segment)

int check_window(const mustafar_window_t* w) {
  if (!w || !aligned(w->k, 16) || !aligned(w->v, 16) || !aligned(w->len, 4) ||
      !aligned(w->head, 4) || !aligned(w->n_comp, 4))
    return MUSTAFAR_EINVAL;
  if (w->B < 1 || w->H < 1 || (int64_t)w->B * w->H > kMaxGrid || !head_dim_ok(w->d))
    return MUSTAFAR_EINVAL;
  if (w->W < 1 || w->W > kMaxWindow || w->max_len < 0 || w->max_len > w->W) return MUSTAFAR_EINVAL;
  return MUSTAFAR_OK;
}

bool window_matches(const mustafar_window_t* w, const mustafar_ccache_t* c) {
  return c->B == w->B && c->H == w->H && c->d == w->d;
}

// Token counts of a decode call are at most kMaxTokens, so the segment
// arithmetic below stays inside int (it is carried out in 64 bits).
constexpr int kMaxTokens = 1 << 30;

int round_up(int64_t x, int64_t a) { return (int)((x + a - 1) / a * a); }

// Segment size (tokens, multiple of 64) for n tokens split n_splits ways.
int seg_tokens(int n, int n_splits) {
  if (n <= 0) return kSegAlign;
  return round_up(((int64_t)n + n_splits - 1) / n_splits, kSegAlign);
}

int n_segments(int n, int seg) { return n <= 0 ? 0 : (int)(((int64_t)n + seg - 1) / seg); }

float scale_log2_of(float scale, int d) {
  const double s = scale > 0.f ? (double)scale : 1.0 / sqrt((double)d);
  return (float)(s * 1.4426950408889634);  // log2(e): scores live in the exp2 domain
}

mf::WindowView window_view_of(const mustafar_window_t* w) {
  mf::WindowView wv;
  wv.k = w->k;
  wv.v = w->v;
  wv.len = w->len;
  wv.head = w->head;
  wv.n_comp = w->n_comp;
  wv.B = w->B;
  wv.H = w->H;
  wv.W = w->W;
  return wv;
}

// Grouped lifecycle windows: whole groups of 32 slots, at least two.
bool grouped_window_ok(const mustafar_window_t* w) { return w->W >= 2 * mf::kGroup && w->W % mf::kGroup == 0; }

// Tokens of a prompt of n tokens that the prefill leaves in the window: the
// last min(n, W), or with a per-channel value cache the last 1 to 32 (the
// compressed prefix is whole groups).
int prefill_window_len(const mustafar_window_t* w, const mustafar_ccache_t* Vc, int n) {
  if (Vc->group_keep >= 0) return n <= 0 ? 0 : n - (n - 1) / mf::kGroup * mf::kGroup;
  return n < w->W ? n : w->W;
}

// The streams of batch entry b as a one-entry cache (same buffers).
mustafar_ccache_t entry_view(const mustafar_ccache_t* c, int b) {
  mustafar_ccache_t v = *c;
  const int64_t s0 = (int64_t)b * c->H;
  const int64_t tiles = s0 * c->cap_tokens * (c->d / kTile);
  v.bitmaps = c->bitmaps + tiles;
  v.offsets = c->offsets + tiles;
  v.values = c->values + s0 * c->val_stride;
  v.stream_len = c->stream_len + s0;
  v.B = 1;
  v.n_tokens = 0;
  return v;
}

// Host checks of a pruner-variant request; fills the kernel's options.
int prune_opts_of(const mustafar_ccache_t* c, const mustafar_prune_opts_t* opts, mf::PruneOpts* o) {
  o->mode = mf::kPruneMagnitude;
  o->H = c->H;
  o->per_head = 0;
  o->weights = nullptr;
  if (!opts) return MUSTAFAR_OK;
  if (opts->mode != MUSTAFAR_PRUNE_MAGNITUDE && opts->mode != MUSTAFAR_PRUNE_2_4 &&
      opts->mode != MUSTAFAR_PRUNE_OUTPUT_AWARE)
    return MUSTAFAR_EINVAL;
  if (grouped(c)) return MUSTAFAR_EINVAL;  // per-token modes need a per-token cache
  o->mode = opts->mode;
  if (opts->mode == MUSTAFAR_PRUNE_2_4) {
    if (opts->head_keep || c->n_keep * 2 != c->d) return MUSTAFAR_EINVAL;
  }
  if (opts->mode == MUSTAFAR_PRUNE_OUTPUT_AWARE) {
    if (!aligned(opts->weights, 4)) return MUSTAFAR_EINVAL;
    o->weights = opts->weights;
  }
  if (opts->head_keep) {
    if (c->H > mf::kMaxPruneHeads) return MUSTAFAR_EUNSUPPORTED;
    for (int h = 0; h < c->H; ++h) {
      if (opts->head_keep[h] < 0 || opts->head_keep[h] > c->n_keep) return MUSTAFAR_EINVAL;
      o->head_keep[h] = opts->head_keep[h];
    }
    o->per_head = 1;
  }
  return MUSTAFAR_OK;
}

}  // namespace

extern "C" {

int mustafar_keep_count(int d, float sparsity) {
  if (d <= 0 || !(sparsity >= 0.f && sparsity <= 1.f)) return MUSTAFAR_EINVAL;
  const int pruned = (int)floor((double)sparsity * (double)d + 0.5);
  int k = d - pruned;
  if (k < 0) k = 0;
  if (k > d) k = d;
  return k;
}

int64_t mustafar_token_max_elems(int d, int n_keep) {
  if (!head_dim_ok(d) || n_keep < 0 || n_keep > d) return -1;
  const int T = d / kTile;
  const int nonempty = n_keep < T ? n_keep : T;  // only tiles with a kept value are padded
  const int64_t m = (int64_t)(n_keep + (kPad - 1) * nonempty) / kPad * kPad;
  return m < d ? m : d;
}

int64_t mustafar_grouped_stream_capacity(int d, int group_keep, int cap_tokens) {
  if (!head_dim_ok(d) || group_keep < 0 || group_keep > mf::kGroup || cap_tokens < 0) return -1;
  const int64_t groups = ((int64_t)cap_tokens + mf::kGroup - 1) / mf::kGroup;
  return groups * ((int64_t)group_keep * d + (int64_t)mf::kGroup * (d / kTile) * (kPad - 1));
}

int64_t mustafar_stream_capacity(int d, int n_keep, int cap_tokens) {
  const int64_t per = mustafar_token_max_elems(d, n_keep);
  if (per < 0 || cap_tokens < 0) return -1;
  return per * cap_tokens;
}

int mustafar_ccache_init(mustafar_ccache_t* c, void* bitmaps, void* offsets, void* values,
                         void* stream_len, int B, int H, int d, float sparsity, int cap_tokens,
                         int64_t val_stride) {
  if (!c) return MUSTAFAR_EINVAL;
  const int k = mustafar_keep_count(d, sparsity);
  if (k < 0) return MUSTAFAR_EINVAL;
  mustafar_ccache_t t;
  t.bitmaps = (uint64_t*)bitmaps;
  t.offsets = (uint32_t*)offsets;
  t.values = (uint16_t*)values;
  t.stream_len = (uint32_t*)stream_len;
  t.B = B;
  t.H = H;
  t.d = d;
  t.n_keep = k;
  t.cap_tokens = cap_tokens;
  t.n_tokens = 0;
  t.val_stride = val_stride;
  t.group_keep = -1;
  const int st = check_cache(&t);
  if (st != MUSTAFAR_OK) return st;
  *c = t;
  return MUSTAFAR_OK;
}

int mustafar_ccache_init_grouped(mustafar_ccache_t* c, void* bitmaps, void* offsets, void* values,
                                 void* stream_len, int B, int H, int d, float sparsity,
                                 int cap_tokens, int64_t val_stride) {
  if (!c) return MUSTAFAR_EINVAL;
  const int gk = mustafar_keep_count(mf::kGroup, sparsity);
  if (gk < 0 || !head_dim_ok(d)) return MUSTAFAR_EINVAL;
  mustafar_ccache_t t;
  t.bitmaps = (uint64_t*)bitmaps;
  t.offsets = (uint32_t*)offsets;
  t.values = (uint16_t*)values;
  t.stream_len = (uint32_t*)stream_len;
  t.B = B;
  t.H = H;
  t.d = d;
  t.n_keep = d;
  t.cap_tokens = cap_tokens;
  t.n_tokens = 0;
  t.val_stride = val_stride;
  t.group_keep = gk;
  const int st = check_cache(&t);
  if (st != MUSTAFAR_OK) return st;
  *c = t;
  return MUSTAFAR_OK;
}

size_t mustafar_compress_workspace_bytes(int B, int H, int n_new) {
  if (B < 1 || H < 1 || n_new < 1) return 0;
  if ((int64_t)B * H > kMaxGrid) return 0;  // no compression call accepts more streams
  const int64_t n_chunks = ((int64_t)n_new + mf::kMinCompressChunk - 1) / mf::kMinCompressChunk;
  // the status word (16 bytes), then per stream a look-back flag per chunk, a
  // ticket counter and a give-up mark
  return (size_t)(16 + (int64_t)B * H * (n_chunks * (int64_t)sizeof(uint64_t) + 2 * (int64_t)sizeof(uint32_t)));
}

static int prune_compress_polls(mustafar_ccache_t* c, const void* x, int n_new, uint32_t max_polls,
                                void* ws, size_t ws_bytes, void* stream) {
  int st = check_cache(c);
  if (st != MUSTAFAR_OK) return st;
  if (n_new < 1 || !aligned(x, 16)) return MUSTAFAR_EINVAL;
  if ((int64_t)c->n_tokens + n_new > c->cap_tokens) return MUSTAFAR_ECAPACITY;
  const size_t need = mustafar_compress_workspace_bytes(c->B, c->H, n_new);
  if (grouped(c) && (n_new % mf::kGroup != 0 || c->n_tokens % mf::kGroup != 0)) return MUSTAFAR_EINVAL;
  if (!aligned(ws, 8) || ws_bytes < need) return MUSTAFAR_EWORKSPACE;
  const hipError_t e =
      grouped(c) ? mf::launch_compress_channel(view_of(c), (const uint16_t*)x, n_new, c->n_tokens,
                                               (uint32_t*)ws, (hipStream_t)stream, nullptr, 0, max_polls)
                 : mf::launch_compress(view_of(c), (const uint16_t*)x, n_new, c->n_tokens,
                                       (uint32_t*)ws, (hipStream_t)stream, 0, max_polls);
  st = status_of(e);
  if (st == MUSTAFAR_OK) c->n_tokens += n_new;
  return st;
}

int mustafar_prune_compress(mustafar_ccache_t* c, const void* x, int n_new, void* ws,
                            size_t ws_bytes, void* stream) {
  return prune_compress_polls(c, x, n_new, MUSTAFAR_LOOKBACK_POLLS, ws, ws_bytes, stream);
}

int mustafar_prune_compress_bounded(mustafar_ccache_t* c, const void* x, int n_new, uint32_t max_polls,
                                    void* ws, size_t ws_bytes, void* stream) {
  return prune_compress_polls(c, x, n_new, max_polls, ws, ws_bytes, stream);
}

int mustafar_append(mustafar_ccache_t* c, const void* x_new, void* stream) {
  int st = check_cache(c);
  if (st != MUSTAFAR_OK) return st;
  if (!aligned(x_new, 16) || grouped(c)) return MUSTAFAR_EINVAL;
  if (c->n_tokens + 1 > c->cap_tokens) return MUSTAFAR_ECAPACITY;
  st = status_of(mf::launch_append(view_of(c), (const uint16_t*)x_new, c->n_tokens,
                                   (hipStream_t)stream));
  if (st == MUSTAFAR_OK) c->n_tokens += 1;
  return st;
}

int mustafar_append_kv(mustafar_ccache_t* Kc, mustafar_ccache_t* Vc, const void* k_new,
                       const void* v_new, void* stream) {
  int st;
  if ((st = check_cache(Kc)) != MUSTAFAR_OK || (st = check_cache(Vc)) != MUSTAFAR_OK) return st;
  if (Kc == Vc) return MUSTAFAR_EINVAL;
  if (Kc->B != Vc->B || Kc->H != Vc->H || Kc->d != Vc->d || Kc->n_tokens != Vc->n_tokens)
    return MUSTAFAR_EINVAL;
  if (!aligned(k_new, 16) || !aligned(v_new, 16) || grouped(Kc) || grouped(Vc)) return MUSTAFAR_EINVAL;
  if (Kc->n_tokens + 1 > Kc->cap_tokens || Vc->n_tokens + 1 > Vc->cap_tokens) return MUSTAFAR_ECAPACITY;
  st = status_of(mf::launch_append_kv(view_of(Kc), view_of(Vc), (const uint16_t*)k_new,
                                      (const uint16_t*)v_new, Kc->n_tokens, (hipStream_t)stream));
  if (st == MUSTAFAR_OK) {
    Kc->n_tokens += 1;
    Vc->n_tokens += 1;
  }
  return st;
}

int mustafar_prune_compress_ex(mustafar_ccache_t* c, const void* x, int n_new,
                               const mustafar_prune_opts_t* opts, void* ws, size_t ws_bytes,
                               void* stream) {
  if (!opts) return mustafar_prune_compress(c, x, n_new, ws, ws_bytes, stream);
  int st = check_cache(c);
  if (st != MUSTAFAR_OK) return st;
  if (n_new < 1 || !aligned(x, 16)) return MUSTAFAR_EINVAL;
  if (opts->mode == MUSTAFAR_PRUNE_CHANNEL || opts->mode == MUSTAFAR_PRUNE_CHANNEL_OUTPUT_AWARE) {
    const bool scored = opts->mode == MUSTAFAR_PRUNE_CHANNEL_OUTPUT_AWARE;
    if (!grouped(c) || opts->head_keep) return MUSTAFAR_EINVAL;
    if (n_new % mf::kGroup != 0 || c->n_tokens % mf::kGroup != 0) return MUSTAFAR_EINVAL;
    if (scored && (!opts->weights || !aligned(opts->weights, 4))) return MUSTAFAR_EINVAL;
    if ((int64_t)c->n_tokens + n_new > c->cap_tokens) return MUSTAFAR_ECAPACITY;
    if (!aligned(ws, 8) || ws_bytes < mustafar_compress_workspace_bytes(c->B, c->H, n_new))
      return MUSTAFAR_EWORKSPACE;
    st = status_of(mf::launch_compress_channel(view_of(c), (const uint16_t*)x, n_new, c->n_tokens,
                                               (uint32_t*)ws, (hipStream_t)stream,
                                               scored ? opts->weights : nullptr));
    if (st == MUSTAFAR_OK) c->n_tokens += n_new;
    return st;
  }
  mf::PruneOpts o;
  if ((st = prune_opts_of(c, opts, &o)) != MUSTAFAR_OK) return st;
  if ((int64_t)c->n_tokens + n_new > c->cap_tokens) return MUSTAFAR_ECAPACITY;
  const size_t need = mustafar_compress_workspace_bytes(c->B, c->H, n_new);
  if (!aligned(ws, 8) || ws_bytes < need) return MUSTAFAR_EWORKSPACE;
  st = status_of(mf::launch_compress_variant(view_of(c), (const uint16_t*)x, n_new, c->n_tokens,
                                             (uint32_t*)ws, (hipStream_t)stream, o));
  if (st == MUSTAFAR_OK) c->n_tokens += n_new;
  return st;
}

int mustafar_append_ex(mustafar_ccache_t* c, const void* x_new, const mustafar_prune_opts_t* opts,
                       void* stream) {
  if (!opts) return mustafar_append(c, x_new, stream);
  int st = check_cache(c);
  if (st != MUSTAFAR_OK) return st;
  if (!aligned(x_new, 16) || grouped(c)) return MUSTAFAR_EINVAL;
  mf::PruneOpts o;
  if ((st = prune_opts_of(c, opts, &o)) != MUSTAFAR_OK) return st;
  if (c->n_tokens + 1 > c->cap_tokens) return MUSTAFAR_ECAPACITY;
  st = status_of(mf::launch_append_variant(view_of(c), (const uint16_t*)x_new, c->n_tokens,
                                           (hipStream_t)stream, o));
  if (st == MUSTAFAR_OK) c->n_tokens += 1;
  return st;
}

int mustafar_query_lookahead(const void* q, int B, int Hq, int Hkv, int n_q, int d, int L,
                             void* w, void* stream) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || n_q < 1 || L < 1) return MUSTAFAR_EINVAL;
  if (!head_dim_ok(d)) return MUSTAFAR_EINVAL;
  if (!aligned(q, 16) || !aligned(w, 16)) return MUSTAFAR_EINVAL;
  return status_of(mf::launch_query_lookahead((const uint16_t*)q, B, Hq, Hkv, n_q, d / kTile, L,
                                              (float*)w, (hipStream_t)stream));
}

int mustafar_attn_set_route(int route) {
  if (route != MUSTAFAR_ROUTE_DEFAULT && route != MUSTAFAR_ROUTE_WALKS && route != MUSTAFAR_ROUTE_MATRIX_CORES)
    return MUSTAFAR_EINVAL;
  g_route.store(route, std::memory_order_relaxed);
  return MUSTAFAR_OK;
}

int mustafar_attn_route(void) { return g_route.load(std::memory_order_relaxed); }

int mustafar_attn_default_splits(int B, int Hq, int Hkv, int n_tokens, int kind) {
  if (B < 1 || Hkv < 1 || Hq < Hkv || n_tokens < 1) return 1;
  if (kind != MUSTAFAR_ATTN_SPARSE && kind != MUSTAFAR_ATTN_DENSE) return 1;
  const bool grouped_q = Hq / Hkv >= 2;
  const bool mfma = mfma_route(Hq / Hkv, g_route.load(std::memory_order_relaxed));
  const int64_t target = !grouped_q ? kWalkTargetGroups
                         : kind == MUSTAFAR_ATTN_DENSE ? kDenseGroupedTargetGroups
                         : mfma                        ? kMfmaTargetGroups
                                                       : kWalkGroupedTargetGroups;
  const int min_seg = !grouped_q ? kWalkMinSegTokens
                      : (kind == MUSTAFAR_ATTN_SPARSE && !mfma) ? kWalkGroupedMinSegTokens
                                                                : kGroupedMinSegTokens;
  const int64_t streams = (int64_t)B * Hkv;
  int64_t want = (target + streams - 1) / streams;
  const int64_t most = ((int64_t)n_tokens + min_seg - 1) / min_seg;
  if (want > most) want = most;
  if (want < 1) want = 1;
  return (int)want;
}

size_t mustafar_attn_workspace_bytes(int B, int Hq, int Hkv, int d, int n_tokens, int n_splits) {
  if (B < 1 || Hq < 1 || Hkv < 1 || d < 1 || n_tokens < 0) return 0;
  // no decode call accepts more streams, query heads per kv-head, head size or splits
  if ((int64_t)B * Hkv > kMaxGrid || Hq > (int64_t)8 * Hkv || d > 256 || n_splits > (1 << 20)) return 0;
  if (n_splits <= 0) {
    const int sp = mustafar_attn_default_splits(B, Hq, Hkv, n_tokens, MUSTAFAR_ATTN_SPARSE);
    const int dn = mustafar_attn_default_splits(B, Hq, Hkv, n_tokens, MUSTAFAR_ATTN_DENSE);
    n_splits = sp > dn ? sp : dn;
  }
  // Segments actually launched never exceed n_splits over the tokens plus one window
  // segment; a two-level merge adds its first-level parts.
  const int64_t n_seg = (int64_t)n_splits + 1;
  const int64_t BHq = (int64_t)B * Hq;
  const int64_t parts = mf::merge_parts(n_seg, BHq);
  const int64_t rows = n_seg + (parts > 1 ? parts : 0);
  // ... then the per-query-head log-sum-exp of the scores-emitting calls.
  return (size_t)(rows * BHq * (int64_t)(d + 2) * (int64_t)sizeof(float) + BHq * (int64_t)sizeof(float));
}

static int decode_common(const void* q, int B, int Hq, int Hkv, int d, int n_s, int n_dense,
                         int dense_is_window, int n_splits, float scale, void* out, void* ws,
                         size_t ws_bytes, mf::AttnShape* sh, float** ws_ml, float** ws_o) {
  if (B < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0) return MUSTAFAR_EINVAL;
  if ((int64_t)B * Hkv > kMaxGrid) return MUSTAFAR_EINVAL;
  if (!head_dim_ok(d)) return MUSTAFAR_EINVAL;
  if (n_s < 0 || n_dense < 0 || (int64_t)n_s + n_dense < 1) return MUSTAFAR_EINVAL;
  if (n_s > kMaxTokens || n_dense > kMaxTokens) return MUSTAFAR_EINVAL;
  if (!aligned(q, 16) || !aligned(out, 16)) return MUSTAFAR_EINVAL;
  const int G = Hq / Hkv;
  if (G != 1 && G != 2 && G != 4 && G != 8) return MUSTAFAR_EUNSUPPORTED;
  const int n_main = dense_is_window ? n_s : n_dense;
  if (n_splits <= 0)
    n_splits = mustafar_attn_default_splits(B, Hq, Hkv, n_main > 0 ? n_main : 1,
                                            dense_is_window ? MUSTAFAR_ATTN_SPARSE : MUSTAFAR_ATTN_DENSE);
  if (n_splits > (1 << 20)) return MUSTAFAR_EINVAL;
  const size_t need = mustafar_attn_workspace_bytes(B, Hq, Hkv, d, n_main, n_splits);
  if (!aligned(ws, 16) || ws_bytes < need) return MUSTAFAR_EWORKSPACE;

  sh->BHkv = B * Hkv;
  sh->G = G;
  sh->mfma = dense_is_window && mfma_route(G, g_route.load(std::memory_order_relaxed));
  sh->T = d / kTile;
  sh->n_s = n_s;
  sh->n_dense = n_dense;
  if (dense_is_window) {
    sh->sparse_seg_tokens = seg_tokens(n_s, n_splits);
    sh->n_sparse_segs = n_segments(n_s, sh->sparse_seg_tokens);
    sh->dense_seg_tokens = round_up(n_dense > 0 ? n_dense : 1, kSegAlign);
    sh->n_dense_segs = n_dense > 0 ? 1 : 0;
  } else {
    sh->sparse_seg_tokens = kSegAlign;
    sh->n_sparse_segs = 0;
    sh->dense_seg_tokens = seg_tokens(n_dense, n_splits);
    sh->n_dense_segs = n_segments(n_dense, sh->dense_seg_tokens);
  }
  sh->scale_log2 = scale_log2_of(scale, d);
  const int64_t n_seg = sh->n_sparse_segs + sh->n_dense_segs;
  const int64_t BHq = (int64_t)B * Hq;
  *ws_ml = (float*)ws;
  *ws_o = (float*)ws + n_seg * BHq * 2;
  return MUSTAFAR_OK;
}

int mustafar_sparse_decode_attn(const void* q, int B, int Hq, const mustafar_ccache_t* Kc,
                                const mustafar_ccache_t* Vc, const void* k_tail,
                                const void* v_tail, int n_tail, float scale, void* out,
                                int n_splits, void* ws, size_t ws_bytes, void* stream) {
  int st = check_cache(Kc);
  if (st != MUSTAFAR_OK) return st;
  st = check_cache(Vc);
  if (st != MUSTAFAR_OK) return st;
  if (Kc->B != B || Vc->B != B || Kc->H != Vc->H || Kc->d != Vc->d ||
      Kc->n_tokens != Vc->n_tokens)
    return MUSTAFAR_EINVAL;
  if (n_tail < 0) return MUSTAFAR_EINVAL;
  if (n_tail > 0 && (!aligned(k_tail, 16) || !aligned(v_tail, 16))) return MUSTAFAR_EINVAL;
  mf::AttnShape sh;
  float *ws_ml, *ws_o;
  st = decode_common(q, B, Hq, Kc->H, Kc->d, Kc->n_tokens, n_tail, 1, n_splits, scale, out, ws,
                     ws_bytes, &sh, &ws_ml, &ws_o);
  if (st != MUSTAFAR_OK) return st;
  return status_of(mf::launch_attention(sh, (const uint16_t*)q, side_of(Kc), side_of(Vc),
                                        (const uint16_t*)k_tail, (const uint16_t*)v_tail, ws_ml,
                                        ws_o, (uint16_t*)out, (hipStream_t)stream));
}

int mustafar_sparse_decode_attn_static(const void* q, int B, int Hq, const mustafar_ccache_t* Kc,
                                       const mustafar_ccache_t* Vc, const void* k_tail,
                                       const void* v_tail, int n_tail, float scale, void* out,
                                       int n_splits, void* stream) {
  // Every argument is checked on the host first (no GPU call before that).
  int st = check_cache(Kc);
  if (st != MUSTAFAR_OK) return st;
  if ((st = check_cache(Vc)) != MUSTAFAR_OK) return st;
  if (Kc->B != B || Vc->B != B || Kc->H != Vc->H || Kc->d != Vc->d || Kc->n_tokens != Vc->n_tokens)
    return MUSTAFAR_EINVAL;
  if (n_tail < 0) return MUSTAFAR_EINVAL;
  if (n_tail > 0 && (!aligned(k_tail, 16) || !aligned(v_tail, 16))) return MUSTAFAR_EINVAL;
  if (B < 1 || Hq < 1 || Hq % Kc->H != 0) return MUSTAFAR_EINVAL;
  const int G = Hq / Kc->H;
  if (G != 1 && G != 2 && G != 4 && G != 8) return MUSTAFAR_EUNSUPPORTED;
  const int n_main = Kc->n_tokens;
  if (n_splits <= 0)
    n_splits = mustafar_attn_default_splits(B, Hq, Kc->H, n_main > 0 ? n_main : 1, MUSTAFAR_ATTN_SPARSE);
  if (n_splits > (1 << 20)) return MUSTAFAR_EINVAL;
  const size_t need = mustafar_attn_workspace_bytes(B, Hq, Kc->H, Kc->d, n_main, n_splits);
  if (need > (size_t)MUSTAFAR_STATIC_SCRATCH_BYTES) return MUSTAFAR_ESCRATCH;
  void* ws = nullptr;
  if ((st = scratch_of_current_device(&ws)) != MUSTAFAR_OK) return st;
  return mustafar_sparse_decode_attn(q, B, Hq, Kc, Vc, k_tail, v_tail, n_tail, scale, out, n_splits, ws,
                                     (size_t)MUSTAFAR_STATIC_SCRATCH_BYTES, stream);
}

int mustafar_dense_decode_attn(const void* q, int B, int Hq, int Hkv, const void* k,
                               const void* v, int n_tokens, int d, float scale, void* out,
                               int n_splits, void* ws, size_t ws_bytes, void* stream) {
  if (n_tokens < 1 || !aligned(k, 16) || !aligned(v, 16)) return MUSTAFAR_EINVAL;
  mf::AttnShape sh;
  float *ws_ml, *ws_o;
  int st = decode_common(q, B, Hq, Hkv, d, 0, n_tokens, 0, n_splits, scale, out, ws, ws_bytes, &sh,
                         &ws_ml, &ws_o);
  if (st != MUSTAFAR_OK) return st;
  mf::SparseSide none = {nullptr, nullptr, nullptr, nullptr, 0, 1, 0};
  return status_of(mf::launch_attention(sh, (const uint16_t*)q, none, none, (const uint16_t*)k,
                                        (const uint16_t*)v, ws_ml, ws_o, (uint16_t*)out,
                                        (hipStream_t)stream));
}

int mustafar_window_init(mustafar_window_t* w, void* k, void* v, void* len, void* head,
                         void* n_comp, int B, int H, int d, int W, int max_len) {
  if (!w || !aligned(k, 16) || !aligned(v, 16) || !aligned(len, 4) || !aligned(head, 4) ||
      !aligned(n_comp, 4))
    return MUSTAFAR_EINVAL;
  if (B < 1 || H < 1 || (int64_t)B * H > kMaxGrid || !head_dim_ok(d)) return MUSTAFAR_EINVAL;
  if (W < 1 || W > kMaxWindow || max_len < 0 || max_len > W) return MUSTAFAR_EINVAL;
  w->k = (uint16_t*)k;
  w->v = (uint16_t*)v;
  w->len = (int32_t*)len;
  w->head = (int32_t*)head;
  w->n_comp = (int32_t*)n_comp;
  w->B = B;
  w->H = H;
  w->d = d;
  w->W = W;
  w->max_len = max_len;
  return MUSTAFAR_OK;
}

int mustafar_window_prefill(mustafar_window_t* w, mustafar_ccache_t* Kc, mustafar_ccache_t* Vc,
                            const void* x_k, const void* x_v, int n_max, const int32_t* seq_len,
                            void* ws, size_t ws_bytes, void* stream) {
  int st = check_window(w);
  if (st != MUSTAFAR_OK) return st;
  if ((st = check_cache(Kc)) != MUSTAFAR_OK || (st = check_cache(Vc)) != MUSTAFAR_OK) return st;
  if (!window_matches(w, Kc) || !window_matches(w, Vc)) return MUSTAFAR_EINVAL;
  if (Kc->n_tokens != 0 || Vc->n_tokens != 0) return MUSTAFAR_EINVAL;
  if (n_max < 0 || !seq_len || !aligned(x_k, 16) || !aligned(x_v, 16)) return MUSTAFAR_EINVAL;
  if (grouped(Kc) || (grouped(Vc) && !grouped_window_ok(w))) return MUSTAFAR_EINVAL;
  int max_comp = 0, max_len = 0;
  for (int b = 0; b < w->B; ++b) {
    if (seq_len[b] < 0 || seq_len[b] > n_max) return MUSTAFAR_EINVAL;
    const int len = prefill_window_len(w, Vc, seq_len[b]);
    if (seq_len[b] - len > max_comp) max_comp = seq_len[b] - len;
    if (len > max_len) max_len = len;
  }
  if (max_comp > Kc->cap_tokens || max_comp > Vc->cap_tokens) return MUSTAFAR_ECAPACITY;
  if (max_comp > 0 && (!aligned(ws, 8) || ws_bytes < mustafar_compress_workspace_bytes(1, w->H, n_max)))
    return MUSTAFAR_EWORKSPACE;
  const hipStream_t s = (hipStream_t)stream;
  const int64_t entry = (int64_t)w->H * n_max * w->d;  // fp16 elements per batch entry of x
  for (int b = 0; b < w->B; ++b) {
    const int len = prefill_window_len(w, Vc, seq_len[b]);
    const int n_comp = seq_len[b] - len;
    const uint16_t* xk = (const uint16_t*)x_k + b * entry;
    const uint16_t* xv = (const uint16_t*)x_v + b * entry;
    if (n_comp > 0) {
      const mustafar_ccache_t kb = entry_view(Kc, b), vb = entry_view(Vc, b);
      const hipError_t ev =
          grouped(Vc) ? mf::launch_compress_channel(view_of(&vb), xv, n_comp, 0, (uint32_t*)ws, s, nullptr, n_max)
                      : mf::launch_compress(view_of(&vb), xv, n_comp, 0, (uint32_t*)ws, s, n_max);
      if ((st = status_of(mf::launch_compress(view_of(&kb), xk, n_comp, 0, (uint32_t*)ws, s, n_max))) !=
              MUSTAFAR_OK ||
          (st = status_of(ev)) != MUSTAFAR_OK)
        return st;
    }
    if ((st = status_of(mf::launch_window_fill(window_view_of(w), b, w->d, xk, xv, n_max, n_comp, len,
                                               s))) != MUSTAFAR_OK)
      return st;
  }
  Kc->n_tokens = max_comp;
  Vc->n_tokens = max_comp;
  w->max_len = max_len;
  return MUSTAFAR_OK;
}

static int window_step_common(mustafar_window_t* w, mustafar_ccache_t* Kc, mustafar_ccache_t* Vc,
                              const void* k_new, const void* v_new, const void* active, float* kacc,
                              void* stream);

int mustafar_window_step(mustafar_window_t* w, mustafar_ccache_t* Kc, mustafar_ccache_t* Vc,
                         const void* k_new, const void* v_new, const void* active, void* stream) {
  return window_step_common(w, Kc, Vc, k_new, v_new, active, nullptr, stream);
}

int mustafar_window_step_weighted(mustafar_window_t* w, mustafar_ccache_t* Kc, mustafar_ccache_t* Vc,
                                  const void* k_new, const void* v_new, const void* active,
                                  float* kacc, void* stream) {
  int st = check_window(w);
  if (st != MUSTAFAR_OK) return st;
  if (w->W < kKeyWeightSteps || !aligned(kacc, 16)) return MUSTAFAR_EINVAL;
  return window_step_common(w, Kc, Vc, k_new, v_new, active, kacc, stream);
}

int mustafar_window_key_weights(const void* q, int B, int Hq, const mustafar_window_t* w,
                                const void* active, float* kacc, void* stream) {
  int st = check_window(w);
  if (st != MUSTAFAR_OK) return st;
  if (B != w->B || Hq < 1 || Hq % w->H != 0) return MUSTAFAR_EINVAL;
  if (Hq / w->H > 8) return MUSTAFAR_EUNSUPPORTED;
  if (!aligned(q, 16) || !aligned(kacc, 16)) return MUSTAFAR_EINVAL;
  if (active && !aligned(active, 4)) return MUSTAFAR_EINVAL;
  return status_of(mf::launch_window_key_weights(window_view_of(w), (const uint16_t*)q, Hq / w->H,
                                                 w->d / kTile, (const int32_t*)active, kacc,
                                                 (hipStream_t)stream));
}

static int window_step_common(mustafar_window_t* w, mustafar_ccache_t* Kc, mustafar_ccache_t* Vc,
                              const void* k_new, const void* v_new, const void* active, float* kacc,
                              void* stream) {
  int st = check_window(w);
  if (st != MUSTAFAR_OK) return st;
  if ((st = check_cache(Kc)) != MUSTAFAR_OK || (st = check_cache(Vc)) != MUSTAFAR_OK) return st;
  if (!window_matches(w, Kc) || !window_matches(w, Vc)) return MUSTAFAR_EINVAL;
  if (grouped(Kc) || grouped(Vc)) return MUSTAFAR_EINVAL;  // see mustafar_window_step_grouped
  if (!aligned(k_new, 16) || !aligned(v_new, 16)) return MUSTAFAR_EINVAL;
  if (active && !aligned(active, 4)) return MUSTAFAR_EINVAL;
  const bool may_graduate = w->max_len >= w->W;
  if (may_graduate && (Kc->n_tokens + 1 > Kc->cap_tokens || Vc->n_tokens + 1 > Vc->cap_tokens))
    return MUSTAFAR_ECAPACITY;
  st = status_of(mf::launch_window_step(view_of(Kc), view_of(Vc), window_view_of(w), (const uint16_t*)k_new,
                                        (const uint16_t*)v_new, (const int32_t*)active,
                                        (hipStream_t)stream, kacc));
  if (st != MUSTAFAR_OK) return st;
  if (may_graduate) {
    Kc->n_tokens += 1;
    Vc->n_tokens += 1;
  } else {
    w->max_len += 1;
  }
  return MUSTAFAR_OK;
}

int mustafar_window_decode_attn(const void* q, int B, int Hq, const mustafar_ccache_t* Kc,
                                const mustafar_ccache_t* Vc, const mustafar_window_t* w,
                                float scale, void* out, int n_splits, void* ws, size_t ws_bytes,
                                void* stream) {
  int st = check_window(w);
  if (st != MUSTAFAR_OK) return st;
  if ((st = check_cache(Kc)) != MUSTAFAR_OK || (st = check_cache(Vc)) != MUSTAFAR_OK) return st;
  if (!window_matches(w, Kc) || !window_matches(w, Vc) || w->B != B) return MUSTAFAR_EINVAL;
  if (Kc->n_tokens != Vc->n_tokens) return MUSTAFAR_EINVAL;
  mf::AttnShape sh;
  float *ws_ml, *ws_o;
  st = decode_common(q, B, Hq, Kc->H, Kc->d, Kc->n_tokens, w->W, 1, n_splits, scale, out, ws,
                     ws_bytes, &sh, &ws_ml, &ws_o);
  if (st != MUSTAFAR_OK) return st;
  sh.n_comp = w->n_comp;
  sh.win_len = w->len;
  sh.win_head = w->head;
  sh.Hkv = Kc->H;
  return status_of(mf::launch_attention(sh, (const uint16_t*)q, side_of(Kc), side_of(Vc), w->k, w->v,
                                        ws_ml, ws_o, (uint16_t*)out, (hipStream_t)stream));
}

int mustafar_window_decode_attn_scores(const void* q, int B, int Hq, const mustafar_ccache_t* Kc,
                                       const mustafar_ccache_t* Vc, const mustafar_window_t* w,
                                       const void* active, float* acc, float scale, void* out,
                                       int n_splits, void* ws, size_t ws_bytes, void* stream) {
  int st = check_window(w);
  if (st != MUSTAFAR_OK) return st;
  if ((st = check_cache(Kc)) != MUSTAFAR_OK || (st = check_cache(Vc)) != MUSTAFAR_OK) return st;
  if (!window_matches(w, Kc) || !window_matches(w, Vc) || w->B != B) return MUSTAFAR_EINVAL;
  if (Kc->n_tokens != Vc->n_tokens || !aligned(acc, 4)) return MUSTAFAR_EINVAL;
  if (active && !aligned(active, 4)) return MUSTAFAR_EINVAL;
  mf::AttnShape sh;
  float *ws_ml, *ws_o;
  st = decode_common(q, B, Hq, Kc->H, Kc->d, Kc->n_tokens, w->W, 1, n_splits, scale, out, ws,
                     ws_bytes, &sh, &ws_ml, &ws_o);
  if (st != MUSTAFAR_OK) return st;
  if (n_splits <= 0)
    n_splits = mustafar_attn_default_splits(B, Hq, Kc->H, Kc->n_tokens > 0 ? Kc->n_tokens : 1,
                                            MUSTAFAR_ATTN_SPARSE);
  const size_t need = mustafar_attn_workspace_bytes(B, Hq, Kc->H, Kc->d, Kc->n_tokens, n_splits);
  float* lse2 = (float*)((char*)ws + need) - (int64_t)B * Hq;
  sh.n_comp = w->n_comp;
  sh.win_len = w->len;
  sh.win_head = w->head;
  sh.Hkv = Kc->H;
  sh.lse2 = lse2;
  const hipStream_t s = (hipStream_t)stream;
  st = status_of(mf::launch_attention(sh, (const uint16_t*)q, side_of(Kc), side_of(Vc), w->k, w->v,
                                      ws_ml, ws_o, (uint16_t*)out, s));
  if (st != MUSTAFAR_OK) return st;
  return status_of(mf::launch_window_scores(window_view_of(w), (const uint16_t*)q, sh.G, sh.T,
                                            sh.scale_log2, lse2, (const int32_t*)active, acc, s));
}

int mustafar_window_step_grouped(mustafar_window_t* w, mustafar_ccache_t* Kc, mustafar_ccache_t* Vc,
                                 const void* k_new, const void* v_new, const void* active,
                                 float* acc, void* stream) {
  int st = check_window(w);
  if (st != MUSTAFAR_OK) return st;
  if ((st = check_cache(Kc)) != MUSTAFAR_OK || (st = check_cache(Vc)) != MUSTAFAR_OK) return st;
  if (!window_matches(w, Kc) || !window_matches(w, Vc)) return MUSTAFAR_EINVAL;
  if (grouped(Kc) || !grouped(Vc) || !grouped_window_ok(w)) return MUSTAFAR_EINVAL;
  if (Kc->n_tokens != Vc->n_tokens || Kc->n_tokens % mf::kGroup != 0) return MUSTAFAR_EINVAL;
  if (!aligned(k_new, 16) || !aligned(v_new, 16) || (acc && !aligned(acc, 4))) return MUSTAFAR_EINVAL;
  if (active && !aligned(active, 4)) return MUSTAFAR_EINVAL;
  // Host bound of the entries' compressed counts: w->max_len follows an entry
  // that holds the most tokens and is active on every step; no entry
  // graduates before it, so n_tokens grows by a group whenever it does.
  const bool may_graduate = w->max_len >= w->W;
  if (may_graduate && (Kc->n_tokens + mf::kGroup > Kc->cap_tokens || Vc->n_tokens + mf::kGroup > Vc->cap_tokens))
    return MUSTAFAR_ECAPACITY;
  st = status_of(mf::launch_window_step_grouped(view_of(Kc), view_of(Vc), window_view_of(w),
                                                (const uint16_t*)k_new, (const uint16_t*)v_new,
                                                (const int32_t*)active, acc, (hipStream_t)stream));
  if (st != MUSTAFAR_OK) return st;
  if (may_graduate) {
    Kc->n_tokens += mf::kGroup;
    Vc->n_tokens += mf::kGroup;
    w->max_len -= mf::kGroup - 1;
  } else {
    w->max_len += 1;
  }
  return MUSTAFAR_OK;
}

const char* mustafar_strerror(int status) {
  switch (status) {
    case MUSTAFAR_OK: return "success";
    case MUSTAFAR_EINVAL: return "invalid argument (size, pointer, alignment or sparsity)";
    case MUSTAFAR_ECAPACITY: return "compressed cache has no room for the new tokens";
    case MUSTAFAR_EWORKSPACE: return "workspace missing, misaligned or too small";
    case MUSTAFAR_ELAUNCH: return "the HIP runtime rejected a kernel launch";
    case MUSTAFAR_EUNSUPPORTED: return "unsupported shape (head dim or query group size)";
    case MUSTAFAR_ESCRATCH:
      return "the call needs more than the library's static scratch buffer "
             "(MUSTAFAR_STATIC_SCRATCH_BYTES per GPU): use the workspace form";
    default: return "unknown status";
  }
}

}  // extern "C"
