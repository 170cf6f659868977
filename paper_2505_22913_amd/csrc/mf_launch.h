// Internal launch interface between the C-ABI layer (api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mf {

// Tokens per two-wave workgroup of the bulk compression (one lane per token at
// d = 64, two lanes per token from d = 128 on).
constexpr int compress_chunk_tokens(int T) { return T >= 2 ? 64 : 128; }
// Smallest chunk over the supported head sizes, for workspace sizing.
constexpr int kMinCompressChunk = 64;

struct CacheView {
  uint64_t* bitmaps;
  uint32_t* offsets;
  uint16_t* values;
  uint32_t* stream_len;
  int BH;            // streams = batch * kv-heads
  int T;             // tiles per token = d / 64
  int n_keep;        // kept channels per token
  int cap_tokens;    // token capacity per stream
  int64_t val_stride;
  int group_keep;    // per-channel caches: tokens kept per channel and group of 32; else -1
};

// A stream whose bulk compression gave up waiting in the look-back (see
// k_compress) has this stream_len; every later call skips it.
constexpr uint32_t kStreamPoisoned = 0xffffffffu;
// Look-back polls before a chunk gives up (never reached in practice: the
// chunks a chunk waits for are already running).
constexpr uint32_t kLookbackPolls = 1u << 20;

// Workspace of the bulk compression: a u32 status word at byte 0 (nonzero once a
// stream gave up; 16 bytes reserved), then u64 look-back flags [BH][n_chunks],
// u32 ticket counters [BH] and u32 give-up marks [BH]. Cleared by each call.
struct CompressWs {
  uint32_t* status;
  uint64_t* flags;
  uint32_t* ticket;
  uint32_t* bad;
  int64_t words;  // 32-bit words to clear from ws
};
inline CompressWs compress_ws(uint32_t* ws, int64_t BH, int64_t n_chunks) {
  CompressWs w;
  w.status = ws;
  w.flags = reinterpret_cast<uint64_t*>(ws + 4);
  w.ticket = reinterpret_cast<uint32_t*>(w.flags + BH * n_chunks);
  w.bad = w.ticket + BH;
  w.words = 4 + 2 * BH * n_chunks + 2 * BH;
  return w;
}

// Compress n_new tokens per stream (x: [BH][x_stride][64T] fp16, x_stride = n_new
// when 0) after tok0 tokens, with the workspace above; a chunk's look-back gives
// up after max_polls polls.
hipError_t launch_compress(const CacheView& c, const uint16_t* x, int n_new, int tok0, uint32_t* ws,
                           hipStream_t s, int64_t x_stride = 0, uint32_t max_polls = kLookbackPolls);
// Compress one token per stream (x: [BH][64T]) as token tok0.
hipError_t launch_append(const CacheView& c, const uint16_t* x, int tok0, hipStream_t s);
// launch_append of the keys and the values of one step in one launch (same shapes).
hipError_t launch_append_kv(const CacheView& kc, const CacheView& vc, const uint16_t* k, const uint16_t* v,
                            int tok0, hipStream_t s);

// Pruner variants of the same format (the magnitude top-k of k_compress is the
// default): per-head kept counts, 2:4 per token, output-aware key scores.
constexpr int kPruneMagnitude = 0, kPrune24 = 1, kPruneOutputAware = 2, kPruneChannel = 3,
              kPruneChannelOutputAware = 4;
constexpr int kMaxPruneHeads = 256;
struct PruneOpts {
  int mode = 0;
  int H = 1;                  // kv-heads: stream s is head s % H
  int per_head = 0;           // head_keep holds each head's kept count
  const float* weights = nullptr;  // output-aware: fp32 [BH][x_stride][64T] channel weights
  int32_t head_keep[kMaxPruneHeads] = {};
};
// Selection (bitmaps of tokens tok0.., one wave per token) then packing with the
// given bitmaps (k_compress in its preset mode).
hipError_t launch_compress_variant(const CacheView& c, const uint16_t* x, int n_new, int tok0,
                                   uint32_t* ws, hipStream_t s, const PruneOpts& o);
hipError_t launch_append_variant(const CacheView& c, const uint16_t* x, int tok0, hipStream_t s,
                                 const PruneOpts& o);
// Per-channel pruning in groups of 32 tokens (n_new and tok0 multiples of 32):
// selection (bitmaps, one wave per stream and group) then k_compress in its
// preset mode. w: NULL (magnitude) or fp32 token weights [BH][n_new].
constexpr int kGroup = 32;
hipError_t launch_compress_channel(const CacheView& c, const uint16_t* x, int n_new, int tok0,
                                   uint32_t* ws, hipStream_t s, const float* w, int64_t x_stride = 0,
                                   uint32_t max_polls = kLookbackPolls);
// Output-aware weights: w[b][h][T][c] = sum over t = T .. min(T+L, Nq)-1, then over
// the G query heads of h, of |q[b][h*G+g][t][c]| (fp32, in that order).
hipError_t launch_query_lookahead(const uint16_t* q, int B, int Hq, int Hkv, int n_q, int T, int L,
                                  float* w, hipStream_t s);

// One window step per active batch entry (see mustafar_window_step): the ring
// slots k, v [BH][W][64T], device state len/head/n_comp [B], H streams per entry.
struct WindowView {
  uint16_t* k;
  uint16_t* v;
  int32_t* len;
  int32_t* head;
  int32_t* n_comp;
  int B, H, W;
};
hipError_t launch_window_fill(const WindowView& w, int b, int d, const uint16_t* xk,
                              const uint16_t* xv, int64_t x_stride, int first, int count,
                              hipStream_t s);
// kacc: null for magnitude keys, else the window's output-aware key weights
// [BH][W][64T] fp32 (the leaving key is pruned with its slot's weights).
hipError_t launch_window_step(const CacheView& kc, const CacheView& vc, const WindowView& w,
                              const uint16_t* k_new, const uint16_t* v_new, const int32_t* active,
                              hipStream_t s, float* kacc = nullptr);
// kacc[bh][slot] += |q| of the G query heads of bh, for the newest 32 window tokens
// of every active entry (active: int32 [B] or null for all).
hipError_t launch_window_key_weights(const WindowView& w, const uint16_t* q, int G, int T,
                                     const int32_t* active, float* kacc, hipStream_t s);
// Grouped lifecycle step (see mustafar_window_step_grouped): kc per token, vc
// per channel; acc: fp32 [B][H][W] scores or NULL (magnitude).
hipError_t launch_window_step_grouped(const CacheView& kc, const CacheView& vc, const WindowView& w,
                                      const uint16_t* k_new, const uint16_t* v_new,
                                      const int32_t* active, float* acc, hipStream_t s);
// Scores of the window tokens younger than 32 steps: acc[b][h][slot] += sum over
// the G query heads of h of exp2(scale_log2 * q.k - lse2[b][hq]) (lse2: the
// log2-domain log-sum-exp the merge wrote), for the active entries (active:
// int32 [B] or null for all).
hipError_t launch_window_scores(const WindowView& w, const uint16_t* q, int G, int T,
                                float scale_log2, const float* lse2, const int32_t* active, float* acc,
                                hipStream_t s);

struct SparseSide {
  const uint64_t* bitmaps;
  const uint32_t* offsets;
  const uint16_t* values;
  const uint32_t* stream_len;  // a poisoned stream is read as empty
  int64_t val_stride;
  int cap_tokens;
  int n_keep;
  int group_keep = -1;  // per-channel caches (see CacheView)
};

struct AttnShape {
  int BHkv;       // streams
  int G;          // query heads per kv-head
  int T;          // tiles per token
  int n_s;        // compressed tokens per stream (0 for the dense kernel)
  int n_dense;    // dense tokens per stream (window, or the whole dense cache)
  int n_sparse_segs, sparse_seg_tokens;
  int n_dense_segs, dense_seg_tokens;
  float scale_log2;  // score scale times log2(e)
  // Per-batch-entry lengths (all null for uniform streams): compressed tokens
  // n_comp[b] <= n_s, and a ring window of n_dense slots holding len[b] tokens
  // from slot head[b] on. Hkv maps a stream to its batch entry.
  const int32_t* n_comp = nullptr;
  const int32_t* win_len = nullptr;
  const int32_t* win_head = nullptr;
  int Hkv = 1;
  // If set, the final merge also writes each query head's log-sum-exp of the
  // scores in the log2 domain, m + log2(l), to lse2 [BHq].
  float* lse2 = nullptr;
  // Compressed segments on the matrix-core kernel (G >= 2) instead of the walks.
  bool mfma = false;
};

// Split-K merge in two levels when a single level would run on too few
// workgroups (many segments, few query heads): the number of first-level parts
// of 32 segments, or 1 for a single-level merge.
inline int merge_parts(int64_t n_seg, int64_t BHq) {
  return (n_seg > 128 && BHq < 256) ? (int)((n_seg + 31) / 32) : 1;
}

// Partial results of every segment into ws_ml [n_seg][BHq] (max, sum) and
// ws_o [n_seg][BHq][d], then the merge into out [BHq][d] fp16 (a two-level merge
// uses [parts][BHq] (max, sum) and [parts][BHq][d] after ws_o).
hipError_t launch_attention(const AttnShape& sh, const uint16_t* q, const SparseSide& K,
                            const SparseSide& V, const uint16_t* kd, const uint16_t* vd,
                            float* ws_ml, float* ws_o, uint16_t* out, hipStream_t s);

}  // namespace mf
