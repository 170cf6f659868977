/*
 * mustafar.h -- C ABI of the MI355X (gfx950) implementation of MUSTAFAR's
 * decode hot path (arxiv 2505.22913):
 *
 *   1. per-token magnitude pruning of the Key and Value caches to an arbitrary
 *      unstructured sparsity (Sec. 2: the per-token magnitude method is the
 *      one the paper keeps for both caches; Appendix A.4 for 80-90%),
 *   2. compression of the pruned caches into the bitmap-based sparse format
 *      (Sec. 3: 1x64 tiles, a 64-bit bitmap per tile, per-tile offsets,
 *      packed non-zeros; Sec. 4.3: non-zeros padded to a multiple of 8),
 *   3. decode attention computed directly on the compressed caches plus a
 *      dense local window of recent tokens (Algorithm 1, Sec. 3).
 *
 * CONVENTIONS (all entry points)
 *   - fp16 tensors are passed as pointers to IEEE binary16 bit patterns.
 *   - Every tensor pointer is a DEVICE pointer owned by the caller. The library
 *     allocates no device or host memory, keeps no state between calls and
 *     never synchronises: work is enqueued on `stream` (a hipStream_t; NULL is
 *     the default stream) and the call returns at once.
 *   - Arguments are validated on the host before anything is launched; an
 *     invalid call returns a negative status and enqueues nothing.
 *   - Status codes: MUSTAFAR_OK (0) or one of the negative codes below;
 *     mustafar_strerror() gives a message. No exception crosses the ABI.
 *   - Calls that overlap on one stream are ordered by the stream; the caller
 *     must not run two calls that write the same cache on different streams
 *     concurrently.
 *
 * THE COMPRESSED CACHE (one per K or V cache of a layer)
 *   B batch entries x H kv-heads = B*H independent streams. A stream holds the
 *   compressed tokens of one (batch, kv-head) in arrival order. With T = d/64
 *   tiles per token, token j of stream s owns tiles s*cap_tokens*T + j*T + t:
 *     bitmaps[tile]  u64  bit i set  <=> channel 64t+i of the token is kept
 *     offsets[tile]  u32  index (fp16 elements, relative to the stream's first
 *                         value) of the tile's first packed non-zero; always a
 *                         multiple of 8. A stream's tiles are packed back to
 *                         back in token (then tile) order: each offset is the
 *                         previous tile's plus its count padded to 8. The
 *                         decode calls rely on this: they read the offset of
 *                         the first tile of each token range they take and
 *                         derive the others from the bitmaps.
 *     values[s*val_stride + offsets[tile] + r]  r < popcount(bitmap): the
 *                         kept fp16 values of the tile in channel order;
 *                         then zero (+0.0) fill up to the next multiple of 8
 *     stream_len[s]  u32  fp16 elements used by stream s (device-side)
 *   Pruning keeps exactly n_keep = mustafar_keep_count(d, sparsity) channels
 *   per token: the n_keep of largest magnitude, ties broken towards the lower
 *   channel index (magnitudes compare as |x|; +0 and -0 are equal). Inputs
 *   must be finite.
 */
#ifndef MUSTAFAR_H
#define MUSTAFAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MUSTAFAR_TILE 64 /* channels per tile, one bit per wavefront lane */
#define MUSTAFAR_PAD 8   /* packed non-zeros per tile rounded up to this  */
/* stream_len of a stream whose bulk compression gave up (see
 * mustafar_prune_compress); no real stream length reaches it */
#define MUSTAFAR_STREAM_POISONED 0xffffffffu
/* look-back polls before a chunk of mustafar_prune_compress gives up */
#define MUSTAFAR_LOOKBACK_POLLS (1u << 20)

enum mustafar_status {
    MUSTAFAR_OK = 0,
    MUSTAFAR_EINVAL = -1,      /* bad size, pointer, alignment or sparsity      */
    MUSTAFAR_ECAPACITY = -2,   /* cache has no room for the tokens              */
    MUSTAFAR_EWORKSPACE = -3,  /* workspace missing or smaller than required    */
    MUSTAFAR_ELAUNCH = -4,     /* the HIP runtime rejected a launch             */
    MUSTAFAR_EUNSUPPORTED = -5, /* valid but unsupported shape (d, group size)  */
    MUSTAFAR_ESCRATCH = -6      /* needs more than the static scratch buffer    */
};

/* Descriptor of one compressed cache. Pointers are device memory owned by the
 * caller; the integer fields are host-side and are filled by
 * mustafar_ccache_init() and advanced by the compress/append calls. */
typedef struct mustafar_ccache {
    uint64_t* bitmaps;    /* [B*H][cap_tokens][d/64], 8-byte aligned            */
    uint32_t* offsets;    /* [B*H][cap_tokens][d/64], 4-byte aligned            */
    uint16_t* values;     /* [B*H][val_stride] fp16 bits, 16-byte aligned       */
    uint32_t* stream_len; /* [B*H], 4-byte aligned                              */
    int32_t B, H, d;      /* batch, kv-heads, head dimension (64, 128 or 256)   */
    int32_t n_keep;       /* channels kept per token                            */
    int32_t cap_tokens;   /* tokens each stream can hold (a multiple of 64 keeps
                             each stream's bitmaps and offsets line-aligned,
                             which the attention reads block by block)      */
    int32_t n_tokens;     /* tokens compressed so far (same for every stream)   */
    int64_t val_stride;   /* fp16 elements reserved per stream, multiple of 8   */
    int32_t group_keep;   /* -1: per-token cache (n_keep channels per token);   */
                          /* >= 0: per-channel cache, every channel keeps       */
                          /* group_keep tokens of each group of 32 (see         */
                          /* mustafar_ccache_init_grouped); n_keep is then d    */
} mustafar_ccache_t;

/* Channels kept per token for a target sparsity s in [0, 1] (Sec. 2 prunes
 * each token to the target sparsity; the rounding of s*d to a whole number of
 * channels is not given by the paper and is fixed here as
 *   n_keep = d - floor(s*d + 1/2)  (round half up, computed in double).
 * Returns n_keep in [0, d], or MUSTAFAR_EINVAL if d <= 0 or s is outside
 * [0, 1] or NaN. Host only. */
int mustafar_keep_count(int d, float sparsity);

/* Largest number of fp16 elements one token can occupy in a stream:
 * min(d, floor8(n_keep + 7*min(n_keep, d/64))), floor8 rounding down to a
 * multiple of 8 -- each tile holding a kept value adds at most 7 pad slots and
 * the total is a multiple of 8. -1 on invalid arguments. Host only. */
int64_t mustafar_token_max_elems(int d, int n_keep);

/* fp16 elements a stream needs to hold cap_tokens tokens in the worst case
 * (cap_tokens * mustafar_token_max_elems). -1 on invalid arguments. */
int64_t mustafar_stream_capacity(int d, int n_keep, int cap_tokens);

/* Fills *c for caller-allocated buffers and sets n_tokens = 0. Checks shapes,
 * alignment and that val_stride >= mustafar_stream_capacity(d, n_keep,
 * cap_tokens). Host only: touches neither the GPU nor the buffers (the caller
 * need not clear any buffer). */
int mustafar_ccache_init(mustafar_ccache_t* c, void* bitmaps, void* offsets, void* values,
                         void* stream_len, int B, int H, int d, float sparsity,
                         int cap_tokens, int64_t val_stride);

/* PER-CHANNEL CACHES (Sec. 2, value-cache study: each channel is pruned to the
 * target sparsity within groups of 32 consecutive tokens). The format is the
 * same (per-token 1x64 tiles, bitmaps, offsets, padded values), so the decode
 * attention reads these caches like the others; a token keeps a variable number
 * of channels, and every channel keeps group_keep = mustafar_keep_count(32, s)
 * tokens of each group of 32 (tokens 32g .. 32g+31 of the stream).
 * Capacity: per group, group_keep * d kept values plus at most 7 pad slots in
 * each of its 32 * d/64 tiles; mustafar_grouped_stream_capacity returns that
 * bound for ceil(cap_tokens / 32) groups (-1 on invalid arguments). */
int64_t mustafar_grouped_stream_capacity(int d, int group_keep, int cap_tokens);

/* As mustafar_ccache_init for a per-channel cache: sets group_keep =
 * mustafar_keep_count(32, sparsity), n_keep = d, and checks val_stride >=
 * mustafar_grouped_stream_capacity(d, group_keep, cap_tokens). Such a cache is
 * filled by whole groups only: mustafar_prune_compress (per-channel magnitude
 * pruning), mustafar_prune_compress_ex with a CHANNEL mode, or the grouped
 * window lifecycle; the append calls reject it. */
int mustafar_ccache_init_grouped(mustafar_ccache_t* c, void* bitmaps, void* offsets, void* values,
                                 void* stream_len, int B, int H, int d, float sparsity,
                                 int cap_tokens, int64_t val_stride);

/* Device workspace needed by mustafar_prune_compress for n_new tokens. */
size_t mustafar_compress_workspace_bytes(int B, int H, int n_new);

/* Prune and compress n_new tokens per stream and append them after the
 * c->n_tokens tokens already in c (into an empty cache this is the
 * compression of the prefill cache before decoding starts, Sec. 3).
 *   x   [B][H][n_new][d] fp16, 16-byte aligned: the dense new tokens
 *   ws  device workspace of at least mustafar_compress_workspace_bytes(),
 *       8-byte aligned; the call clears and uses it (per-chunk scan flags
 *       and per-stream ticket counters), so calls that share one workspace
 *       must not overlap
 * On success c->n_tokens += n_new. Errors: EINVAL (bad descriptor, n_new < 1,
 * misaligned x), ECAPACITY (n_tokens + n_new > cap_tokens), EWORKSPACE.
 *
 * Completion status. Each chunk of 64 tokens finds its place in the stream by
 * waiting for the running totals of the chunks before it (a single-pass
 * scan). That wait is bounded (MUSTAFAR_LOOKBACK_POLLS reads; the chunks it
 * waits for are always already running, so the bound is a guard, never
 * reached in a healthy run). A chunk that reaches the bound writes nothing;
 * its stream then has a hole and, once the call has finished on the device,
 * its stream_len is MUSTAFAR_STREAM_POISONED. The first 32-bit word of ws is
 * 0 after a call in which every stream was compressed and nonzero if any
 * stream was poisoned; the caller reads it (a device-to-host copy after the
 * stream has synchronised) before it reuses ws. A poisoned stream stays so:
 * every later call skips it (compression and appends write nothing to it, the
 * decode attention treats its compressed part as empty) until the cache is
 * refilled from token 0. */
int mustafar_prune_compress(mustafar_ccache_t* c, const void* x, int n_new, void* ws,
                            size_t ws_bytes, void* stream);

/* mustafar_prune_compress with the caller's bound on the look-back of a chunk,
 * counted in reads of the other chunks' totals (for callers with a latency
 * budget, and to exercise the give-up path: with max_polls = 0 no chunk but the
 * first of a stream may read, so every stream of more than one chunk -- 64
 * tokens, 128 at d = 64 -- is poisoned). Same arguments, status word and
 * errors. */
int mustafar_prune_compress_bounded(mustafar_ccache_t* c, const void* x, int n_new, uint32_t max_polls,
                                    void* ws, size_t ws_bytes, void* stream);

/* Prune, compress and append ONE token per stream (the token that leaves the
 * dense local window at a decode step, Sec. 3 and Appendix C.2). Needs no
 * workspace. x_new [B][H][d] fp16, 16-byte aligned. On success
 * c->n_tokens += 1. The result is bit-identical to compressing all tokens in
 * one mustafar_prune_compress call. */
int mustafar_append(mustafar_ccache_t* c, const void* x_new, void* stream);

/* mustafar_append of a decode step's key (into Kc) and value (into Vc) in one
 * launch. The caches must be two different caches with the same B, H, d and
 * n_tokens (their sparsities may differ). Errors: EINVAL (descriptors, one
 * cache twice, shapes, alignment, per-channel caches), ECAPACITY; on any
 * error neither cache changes. */
int mustafar_append_kv(mustafar_ccache_t* Kc, mustafar_ccache_t* Vc, const void* k_new,
                       const void* v_new, void* stream);

/* PRUNER VARIANTS in the same compressed format (the decode attention reads
 * any bitmaps):
 *   MUSTAFAR_PRUNE_MAGNITUDE     per-token magnitude top-k (the default above),
 *                                optionally with a kept count per head;
 *   MUSTAFAR_PRUNE_2_4           2:4 semi-structured per token (Appendix B): in
 *                                every 4 consecutive channels the 2 of largest
 *                                magnitude, ties to the lower channel; needs a
 *                                cache with n_keep == d/2;
 *   MUSTAFAR_PRUNE_OUTPUT_AWARE  output-aware key pruning (Sec. 2): the n_keep
 *                                channels of largest score |x_c| * w_c, the fp32
 *                                product rounded once, ties to the lower
 *                                channel; w are non-negative fp32 channel
 *                                weights per token (see mustafar_query_lookahead).
 * head_keep (all modes but 2:4): NULL, or a HOST array [H] of kept counts per
 * head, each in [0, c->n_keep] (finer-grained sparsity, named as future work
 * in Conclusion and Limitations; the cache's capacity is the one of n_keep). H <= 256 with head_keep.
 * Per-channel caches only (mustafar_prune_compress_ex; n_new and c->n_tokens
 * multiples of 32; head_keep must be NULL):
 *   MUSTAFAR_PRUNE_CHANNEL       per-channel magnitude pruning in groups of 32
 *                                tokens: every channel keeps the group_keep
 *                                tokens of largest |x|, ties to the lower token
 *                                (the default of mustafar_prune_compress on
 *                                such a cache);
 *   MUSTAFAR_PRUNE_CHANNEL_OUTPUT_AWARE  per-channel output-aware pruning
 *                                (Sec. 2): the key of token j is |x_jc| * w_j,
 *                                the fp32 product rounded once, with w_j >= 0
 *                                the attention probability mass token j
 *                                received (fp32 [B][H][n_new], 4-byte aligned;
 *                                see mustafar_window_decode_attn_scores); ties
 *                                to the lower token. */
enum mustafar_prune_mode {
    MUSTAFAR_PRUNE_MAGNITUDE = 0,
    MUSTAFAR_PRUNE_2_4 = 1,
    MUSTAFAR_PRUNE_OUTPUT_AWARE = 2,
    MUSTAFAR_PRUNE_CHANNEL = 3,
    MUSTAFAR_PRUNE_CHANNEL_OUTPUT_AWARE = 4
};
typedef struct mustafar_prune_opts {
    int32_t mode;
    const int32_t* head_keep; /* host [H] or NULL                                  */
    const float* weights;     /* device fp32, 4-byte aligned: [B][H][n_tokens][d]  */
                              /* (OUTPUT_AWARE) or [B][H][n_tokens] (CHANNEL_      */
                              /* OUTPUT_AWARE); NULL for the other modes           */
} mustafar_prune_opts_t;

/* mustafar_prune_compress / mustafar_append under a pruner variant (opts NULL:
 * the default magnitude pruning). For _ex compress, weights has n_new tokens
 * per stream; for _ex append, one. Same workspace, capacity and errors as the
 * default calls, plus EINVAL for a bad mode, head_keep or weights. */
int mustafar_prune_compress_ex(mustafar_ccache_t* c, const void* x, int n_new,
                               const mustafar_prune_opts_t* opts, void* ws, size_t ws_bytes,
                               void* stream);
int mustafar_append_ex(mustafar_ccache_t* c, const void* x_new, const mustafar_prune_opts_t* opts,
                       void* stream);

/* Channel weights of output-aware key pruning (Sec. 2: the L1 sum of the
 * current and the next L-1 queries, summed over the query heads of a group):
 *   w[b][h][t][c] = sum_{u = t}^{min(t+L, n_q)-1} sum_{g < Hq/Hkv}
 *                   |q[b][h*(Hq/Hkv)+g][u][c]|
 * in fp32, added in that order (u ascending, then g). q [B][Hq][n_q][d] fp16
 * holds the query of every token position; w [B][Hkv][n_q][d] fp32 (both
 * 16-byte aligned). The paper uses L = 32. Errors: EINVAL, EUNSUPPORTED. */
int mustafar_query_lookahead(const void* q, int B, int Hq, int Hkv, int n_q, int d, int L,
                             void* w, void* stream);

/* Kernels behind the decode calls, for mustafar_attn_default_splits:
 * MUSTAFAR_ATTN_SPARSE for the calls over compressed caches, MUSTAFAR_ATTN_DENSE
 * for mustafar_dense_decode_attn. */
enum mustafar_attn_kind {
    MUSTAFAR_ATTN_SPARSE = 0,
    MUSTAFAR_ATTN_DENSE = 1
};

/* Split-K segment count a decode call of the given kind picks when it is
 * passed n_splits <= 0, for B*Hkv streams of n_tokens tokens (the compressed
 * tokens for the sparse calls). It depends on the kernel that runs: with one
 * query head per kv-head, many segments down to one 64-token block; with 2 or
 * 4 query heads per kv-head (the same bit walks), about 4096 workgroups of at
 * least 192 tokens; with 8 (the matrix-core kernel), about 2048 of at least
 * 128; the dense kernel with grouped queries about 4096 of at least 128.
 * With a route other than the default (mustafar_attn_set_route), the split
 * count follows the kernel the route picks. Returns 1 for invalid arguments
 * or kind. */
int mustafar_attn_default_splits(int B, int Hq, int Hkv, int n_tokens, int kind);

/* Kernel route of the sparse calls with grouped queries (2, 4 or 8 query heads
 * per kv-head; one head always takes the bit walks). DEFAULT: the bit walks
 * below 8 query heads per kv-head, the matrix-core kernel (zero-filled tiles
 * contracted with v_mfma) from 8 on, the faster of the two on MI355X at each
 * group size; WALKS and MATRIX_CORES force one kernel for every group size,
 * for comparing them. Both give the same results up to rounding (each within
 * the attention tolerance of the reference). The setting is process-wide and
 * takes effect for calls issued after it; it is not synchronized with calls
 * in flight on other threads. Errors: EINVAL (unknown route). */
enum mustafar_route {
    MUSTAFAR_ROUTE_DEFAULT = 0,
    MUSTAFAR_ROUTE_WALKS = 1,
    MUSTAFAR_ROUTE_MATRIX_CORES = 2
};
int mustafar_attn_set_route(int route);
int mustafar_attn_route(void);

/* Device workspace for the decode-attention calls: fp32 partial results
 * (running max, running sum, d accumulators) for n_splits token ranges plus
 * one dense-window segment, for each of the B*Hq query heads. n_splits <= 0
 * sizes for the larger of the two kinds' default split counts, so the result
 * serves any decode call over n_tokens tokens that also passes n_splits <= 0. */
size_t mustafar_attn_workspace_bytes(int B, int Hq, int Hkv, int d, int n_tokens, int n_splits);

/* Decode attention over compressed caches plus a dense local window
 * (Algorithm 1). For query head h (kv-head h / (Hq/Hkv), grouped-query
 * attention with contiguous groups):
 *   scores = scale * q.k over the Kc->n_tokens compressed tokens (zero-filled
 *            pruned keys), then over the n_tail window tokens;
 *   p      = softmax over all of them;
 *   out    = sum_j p_j v_j (pruned values are zeros).
 *   q       [B][Hq][d] fp16, 16-byte aligned
 *   Kc, Vc  compressed caches with B, H = Hkv, d and n_tokens equal
 *   k_tail, v_tail  [B][Hkv][n_tail][d] fp16, 16-byte aligned; may be NULL
 *           when n_tail == 0
 *   scale   score scale; <= 0 selects 1/sqrt(d)
 *   out     [B][Hq][d] fp16 (round to nearest even), 16-byte aligned
 *   n_splits  token ranges per stream processed in parallel (<= 0: default)
 * Errors: EINVAL (shape mismatch, Hq % Hkv != 0, no tokens at all, bad
 * pointers), EUNSUPPORTED (Hq/Hkv not 1, 2, 4 or 8), EWORKSPACE. */
int mustafar_sparse_decode_attn(const void* q, int B, int Hq, const mustafar_ccache_t* Kc,
                                const mustafar_ccache_t* Vc, const void* k_tail,
                                const void* v_tail, int n_tail, float scale, void* out,
                                int n_splits, void* ws, size_t ws_bytes, void* stream);

/* FOR CALLERS THAT CANNOT ALLOCATE (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): mustafar_sparse_decode_attn without a
 * workspace argument. Its split-K partials go to a static device buffer of
 * MUSTAFAR_STATIC_SCRATCH_BYTES that the library holds on every GPU it runs
 * on until the process ends; the call allocates nothing itself (no hipMalloc,
 * hipFree or allocating library routine). The first call on a device looks up
 * that device's buffer (the current device, which `stream` must belong to).
 * Every call on a GPU shares the one buffer, so calls that overlap on one GPU
 * race: issue them on one stream, or order them. The buffer needs no clearing
 * (every call writes each partial it reads). Same arguments and result as
 * mustafar_sparse_decode_attn (the same kernels), bit for bit for the same
 * n_splits. Errors as mustafar_sparse_decode_attn, plus ESCRATCH when the
 * partials (mustafar_attn_workspace_bytes for the call's sizes and split
 * count) exceed the buffer; an invalid call launches nothing. */
#define MUSTAFAR_STATIC_SCRATCH_BYTES (32u << 20)
int mustafar_sparse_decode_attn_static(const void* q, int B, int Hq, const mustafar_ccache_t* Kc,
                                       const mustafar_ccache_t* Vc, const void* k_tail,
                                       const void* v_tail, int n_tail, float scale, void* out,
                                       int n_splits, void* stream);

/* The same attention over dense fp16 caches k, v [B][Hkv][n_tokens][d]: the
 * in-house dense baseline the sparse path is measured against (the paper
 * compares against a dense batched matrix-vector product, Sec. 4.3). */
int mustafar_dense_decode_attn(const void* q, int B, int Hq, int Hkv, const void* k,
                               const void* v, int n_tokens, int d, float scale, void* out,
                               int n_splits, void* ws, size_t ws_bytes, void* stream);

/* THE DENSE LOCAL WINDOW (Sec. 3: the most recent tokens stay dense and are
 * not pruned; tokens leaving the window are pruned and compressed at decode
 * time). A ring of W token slots per stream, with device-side state per batch
 * entry so that the entries of a batch may hold different numbers of tokens:
 *   k, v     [B][H][W][d] fp16 ring slots, 16-byte aligned
 *   len[b]   tokens in the window of batch entry b (0..W)
 *   head[b]  slot of its oldest token; the i-th oldest is in slot (head+i) % W
 *   n_comp[b] tokens of entry b already in the compressed caches (they are
 *            tokens 0 .. n_comp[b]-1 of every stream of b; the window holds
 *            tokens n_comp[b] .. n_comp[b]+len[b]-1)
 * len, head and n_comp are int32 device arrays owned by the caller, who sets
 * them after filling the caches (a prefill of entry b with P tokens compresses
 * its first P - min(P, W) tokens and copies the rest into slots 0.. with
 * head = 0). The host-side max_len is an upper bound of len[b] over the batch
 * and the caches' n_tokens an upper bound of n_comp[b]; the calls below keep
 * both bounds and use them for capacity checks and launch geometry. */
typedef struct mustafar_window {
    uint16_t* k;      /* [B][H][W][d] fp16                                        */
    uint16_t* v;      /* [B][H][W][d] fp16                                        */
    int32_t* len;     /* [B] device                                               */
    int32_t* head;    /* [B] device                                               */
    int32_t* n_comp;  /* [B] device                                               */
    int32_t B, H, d, W;
    int32_t max_len;  /* host: upper bound of len[b]                              */
} mustafar_window_t;

/* Fills *w for caller-allocated buffers (host only; touches no buffer).
 * 1 <= W <= 1024; 0 <= max_len <= W. Errors: EINVAL. */
int mustafar_window_init(mustafar_window_t* w, void* k, void* v, void* len, void* head,
                         void* n_comp, int B, int H, int d, int W, int max_len);

/* Prefill of the window lifecycle with prompts of different lengths: batch
 * entry b holds the first seq_len[b] tokens of x_k, x_v [B][H][n_max][d] fp16
 * (16-byte aligned; seq_len is a HOST array, 0 <= seq_len[b] <= n_max). Its
 * first seq_len[b] - min(seq_len[b], W) tokens are pruned, compressed and
 * written to the EMPTY caches Kc, Vc (n_tokens == 0); the remaining tokens
 * fill window slots 0.. in order; len[b], head[b] = 0 and n_comp[b] are set.
 * Afterwards Kc/Vc->n_tokens and w->max_len hold the batch maxima. ws: at
 * least mustafar_compress_workspace_bytes(1, H, n_max) bytes, 8-byte aligned
 * (used by one entry after the other). With a per-channel Vc (the grouped
 * lifecycle, see mustafar_window_step_grouped) the compressed prefix is instead
 * the first 32 * floor((seq_len[b] - 1) / 32) tokens, whole groups, values
 * pruned per channel by magnitude. Errors: EINVAL, ECAPACITY, EWORKSPACE. */
int mustafar_window_prefill(mustafar_window_t* w, mustafar_ccache_t* Kc, mustafar_ccache_t* Vc,
                            const void* x_k, const void* x_v, int n_max, const int32_t* seq_len,
                            void* ws, size_t ws_bytes, void* stream);

/* One decode step of the window lifecycle for every batch entry b with
 * active[b] != 0 (active may be NULL: every entry): the new token
 * k_new, v_new [B][H][d] fp16 (16-byte aligned) enters the window; if the
 * window of b was full (len[b] == W), its oldest token first leaves it: it is
 * pruned, compressed and appended to Kc and Vc as token n_comp[b] (the same
 * result as mustafar_append, per batch entry) and n_comp[b] += 1; otherwise
 * len[b] += 1. Kc and Vc must have B, H = w->H and d = w->d. The host bounds
 * advance: if w->max_len == W, Kc->n_tokens and Vc->n_tokens grow by one (the
 * call fails with ECAPACITY, enqueuing nothing, if that would pass
 * cap_tokens), else w->max_len grows by one. */
int mustafar_window_step(mustafar_window_t* w, mustafar_ccache_t* Kc, mustafar_ccache_t* Vc,
                         const void* k_new, const void* v_new, const void* active, void* stream);

/* Output-aware key pruning in the window lifecycle (Sec. 2: a key's channels
 * are scored by |K| times the L1 sum of the query at its position and the 31
 * after it, summed over the query heads of its kv-head). kacc [B][H][W][d] is
 * fp32 device memory, 16-byte aligned, owned by the caller and zeroed by it
 * before the window's prefill; window slot s of (b, h) holds the weights of the
 * token in that slot. Each call adds |q[b][h*G+g][c]| (fp16 q [B][Hq][d],
 * 16-byte aligned; G = Hq/H), for g = 0, 1, ..., G-1 one after the other in
 * fp32, to kacc[b][h][s][c] for every ACTIVE batch entry b (active: int32
 * device [B], 4-byte aligned, nonzero = active; NULL: every entry), kv-head h
 * and slot s holding one of the newest min(len[b], 32) window tokens; an
 * inactive entry's weights do not change. Called once per decode step with
 * that step's queries and the step's active mask, after the step's
 * mustafar_window_step_weighted, it leaves a token that leaves the window with
 * the weights of the queries of its own entry's 32 active steps from its
 * arrival on: those mustafar_query_lookahead (L = 32) computes from that
 * entry's query sequence, bit for bit. Errors: EINVAL, EUNSUPPORTED (G > 8). */
int mustafar_window_key_weights(const void* q, int B, int Hq, const mustafar_window_t* w,
                                const void* active, float* kacc, void* stream);

/* mustafar_window_step whose leaving key (the oldest token of a full window)
 * is pruned output-aware: channel score fl32(|k_c| x kacc[b][h][slot][c]), the
 * larger first, ties to the lower channel (the selection of
 * MUSTAFAR_PRUNE_OUTPUT_AWARE); its value is pruned by magnitude as before. The
 * slot that takes the new token gets weights 0. Needs W >= 32, so that a key
 * leaves with the weights of 32 steps. Errors as mustafar_window_step, and
 * EINVAL for W < 32 or a misaligned kacc. */
int mustafar_window_step_weighted(mustafar_window_t* w, mustafar_ccache_t* Kc, mustafar_ccache_t* Vc,
                                  const void* k_new, const void* v_new, const void* active,
                                  float* kacc, void* stream);

/* Decode attention of Algorithm 1 per batch entry b over its n_comp[b]
 * compressed tokens and the len[b] tokens of its window (the window is
 * Algorithm 1's dense local part). Every batch entry must hold at least one
 * token. Shapes and the other arguments as for mustafar_sparse_decode_attn;
 * the workspace is mustafar_attn_workspace_bytes(B, Hq, H, d, Kc->n_tokens,
 * n_splits). Errors: EINVAL, EUNSUPPORTED, EWORKSPACE. */
int mustafar_window_decode_attn(const void* q, int B, int Hq, const mustafar_ccache_t* Kc,
                                const mustafar_ccache_t* Vc, const mustafar_window_t* w,
                                float scale, void* out, int n_splits, void* ws, size_t ws_bytes,
                                void* stream);

/* Decode attention as mustafar_window_decode_attn, then the output-aware
 * scores of per-channel value pruning (Sec. 2): for every ACTIVE batch entry b
 * (active: int32 device [B], 4-byte aligned, nonzero = active; NULL: every
 * entry), kv-head h and window slot holding one of the entry's tokens that
 * arrived fewer than 32 of its steps ago (the newest 32 of its len[b]),
 *   acc[b][h][slot] += sum over the G query heads of h of the attention
 *                      probability of that token (Algorithm 1's softmax over
 *                      the compressed and window tokens),
 * so that once a token has seen 32 active steps of its entry, its slot holds
 * the sum over the step it arrived in and the 31 following ones; an inactive
 * entry's scores do not change (its output is still computed). acc: device
 * fp32 [B][H][W], 4-byte aligned, zeroed by the caller before the first step
 * (the grouped window step clears the slots it frees). The workspace is the
 * one of mustafar_window_decode_attn. Errors as mustafar_window_decode_attn. */
int mustafar_window_decode_attn_scores(const void* q, int B, int Hq, const mustafar_ccache_t* Kc,
                                       const mustafar_ccache_t* Vc, const mustafar_window_t* w,
                                       const void* active, float* acc, float scale, void* out,
                                       int n_splits, void* ws, size_t ws_bytes, void* stream);

/* One decode step of the GROUPED window lifecycle (per-channel value pruning in
 * groups of 32 tokens, Sec. 2): Kc is a per-token cache, Vc a per-channel
 * cache, the window has W >= 64 slots, W a multiple of 32. For every active
 * batch entry b (active may be NULL): if its window is full (len[b] == W), its
 * oldest 32 tokens leave it together: their keys are pruned per token
 * (magnitude, Kc's n_keep) and their values per channel as one group, with the
 * scores acc[b][h][slot] of their slots (CHANNEL_OUTPUT_AWARE) or by magnitude
 * (acc NULL); both are appended as tokens n_comp[b] .. n_comp[b]+31,
 * n_comp[b] += 32, head[b] advances by 32 and len[b] -= 32. Then the new
 * token enters slot (head + len) % W, whose acc entries are set to 0, and
 * len[b] += 1. A token is thus at least 32 steps old when it leaves,
 * so its score covers exactly its first 32 steps. Host bounds as for
 * mustafar_window_step, by 32 tokens (ECAPACITY if the caches could not take a
 * group). Errors: EINVAL (shapes, W, cache kinds, alignment), ECAPACITY,
 * ELAUNCH. The prefill of such a window (mustafar_window_prefill with a
 * per-channel Vc) compresses the first 32 * floor((n - 1) / 32) tokens of an
 * entry of n tokens, by magnitude, and keeps the rest (1 to 32 tokens) in the
 * window. */
int mustafar_window_step_grouped(mustafar_window_t* w, mustafar_ccache_t* Kc, mustafar_ccache_t* Vc,
                                 const void* k_new, const void* v_new, const void* active,
                                 float* acc, void* stream);

/* Static message for a status code. */
const char* mustafar_strerror(int status);

/* MEASUREMENT HELPER (not a step of the method). Streams `bytes` of device
 * memory at `src` through 16-byte loads and writes one 32-bit checksum per
 * workgroup to `sink` (device, at least mustafar_stream_read_sink_bytes()):
 * the HBM read ceiling the decode kernels are measured against. `src` must be
 * 16-byte aligned and `bytes` a multiple of 16. Errors: EINVAL. */
size_t mustafar_stream_read_sink_bytes(void);
int mustafar_stream_read(const void* src, size_t bytes, void* sink, void* stream);

/* MEASUREMENT HELPER (not a step of the method). Streams `bytes` of device
 * memory at `src` through 16-byte loads, writes one 32-bit checksum per
 * workgroup to `sink` (as mustafar_stream_read does) and writes
 * write_16ths/16 of the words to `dst` (device, at least
 * bytes * write_16ths / 16 bytes): of every 16 consecutive 16-byte words, the
 * first write_16ths are stored, packed. The rate is the HBM ceiling of a pass
 * that reads a dense cache and writes its compressed form in that ratio.
 * `src` and `dst` must be 16-byte aligned, `sink` 4-byte aligned, `bytes` a
 * multiple of 256 and 0 <= write_16ths <= 16. Errors: EINVAL. */
int mustafar_stream_mix(const void* src, size_t bytes, void* dst, int write_16ths, void* sink,
                        void* stream);

/* MEASUREMENT HELPER (not a step of the method). The bytes and access order of
 * the bulk compression (mustafar_prune_compress at d = 128) without its
 * arithmetic: `src` holds n_streams streams of n_chunks chunks of
 * MUSTAFAR_STREAM_CHUNK_BYTES each, stream-major; one two-wave workgroup per
 * chunk, the streams taking turns chunk by chunk (workgroup g: stream
 * g % n_streams, chunk g / n_streams), reads its chunk with 16-byte loads,
 * writes the first write_16ths/16 of the chunk's 16-byte words, packed, to the
 * chunk's place in `dst` (device, at least n_streams * n_chunks *
 * MUSTAFAR_STREAM_CHUNK_BYTES * write_16ths / 16 bytes) and one 32-bit checksum
 * (XOR of the chunk's words) to sink[g] (device, n_streams * n_chunks
 * entries). Its rate is the ceiling of that access order. `src` and `dst` must
 * be 16-byte aligned, `sink` 4-byte aligned, n_streams, n_chunks >= 1 with
 * n_streams * n_chunks < 2^31, 0 <= write_16ths <= 16. Errors: EINVAL. */
#define MUSTAFAR_STREAM_CHUNK_BYTES 16384
int mustafar_stream_chunks(const void* src, int n_streams, int n_chunks, void* dst, int write_16ths,
                           void* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MUSTAFAR_H */
