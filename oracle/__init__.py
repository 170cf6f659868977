"""CPU oracle for MUSTAFAR's decode hot path (arxiv 2505.22913).

TEST INFRASTRUCTURE. Only the test suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package. It shares no code with
the GPU library (``paper_2505_22913_amd``) and never imports it.

The arithmetic lives in ``mustafar_oracle.c`` (plain C, double precision, one
(batch, kv-head) stream per call); this module only marshals numpy arrays and
loops over streams:

* ``keep_count`` -- kept channels per token for a sparsity (Sec. 2).
* ``prune_token`` -- per-token magnitude top-k with the fixed tie rule.
* ``compress`` / ``decompress`` -- the bitmap format (Sec. 3, Sec. 4.3).
* ``decode_attention`` -- Algorithm 1 over zero-filled pruned caches plus a
  dense local window, in float64.
* ``sparse_decode_attention`` -- decompress, then ``decode_attention``.
* ``prune_token_24``, ``prune_token_scored``, ``compress_variant`` -- the
  pruner variants in the same format: 2:4 per token (Appendix B), output-aware
  key pruning (Sec. 2), per-head kept counts (finer-grained sparsity, which
  the Conclusion and Limitations section names as future work);
  ``query_lookahead`` -- the channel weights of output-aware pruning.
* ``prune_channel_group``, ``compress_grouped`` -- per-channel value pruning in
  groups of 32 tokens, by magnitude or output-aware (Sec. 2's value-cache
  study), in the same format; ``attention_probs`` -- the softmax weights of
  Algorithm 1, which the output-aware form accumulates per token.

Streams are independent, so the batched helpers accept ``threads``: ctypes
releases the GIL during each C call and streams are spread over a thread pool.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mustafar_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
TILE = 64
PAD = 8
GROUP = 32  # tokens per per-channel pruning group (Sec. 2, value cache)

_lib = None


def build(force: bool = False) -> str:
    """Compile ``mustafar_oracle.c`` into ``liboracle.so`` with the host C compiler."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build(force=False)
    _lib = _bind(ctypes.CDLL(_LIB_PATH))
    return _lib


@contextlib.contextmanager
def using_library(path: str):
    """Route every oracle call through another build of ``mustafar_oracle.c``
    for the duration of the block (the mutation tests compile deliberately
    broken copies and check that the pins reject them)."""
    global _lib
    saved = _lib
    _lib = _bind(ctypes.CDLL(os.path.abspath(path)))
    try:
        yield
    finally:
        _lib = saved


def _bind(lib):
    P = ctypes.c_void_p
    lib.oracle_half_to_double.argtypes = [ctypes.c_uint16]
    lib.oracle_half_to_double.restype = ctypes.c_double
    lib.oracle_keep_count.argtypes = [ctypes.c_int, ctypes.c_float]
    lib.oracle_keep_count.restype = ctypes.c_int
    lib.oracle_prune_token.argtypes = [P, ctypes.c_int, ctypes.c_int, P]
    lib.oracle_prune_token.restype = None
    lib.oracle_compress_stream.argtypes = [P, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                           P, P, P, ctypes.c_int64, P]
    lib.oracle_compress_stream.restype = ctypes.c_int
    lib.oracle_decompress_stream.argtypes = [P, P, P, ctypes.c_int, ctypes.c_int, P]
    lib.oracle_decompress_stream.restype = ctypes.c_int
    lib.oracle_decode_attention.argtypes = [P, ctypes.c_int, ctypes.c_int, P, P, ctypes.c_int,
                                            P, P, ctypes.c_int, ctypes.c_double, P]
    lib.oracle_decode_attention.restype = ctypes.c_int
    lib.oracle_prune_token_24.argtypes = [P, ctypes.c_int, P]
    lib.oracle_prune_token_24.restype = None
    lib.oracle_prune_token_scored.argtypes = [P, P, ctypes.c_int, ctypes.c_int, P]
    lib.oracle_prune_token_scored.restype = None
    lib.oracle_encode_stream.argtypes = [P, P, ctypes.c_int, ctypes.c_int, P, P, P,
                                         ctypes.c_int64, P]
    lib.oracle_encode_stream.restype = ctypes.c_int
    lib.oracle_prune_channel_group.argtypes = [P, P, ctypes.c_int, ctypes.c_int, ctypes.c_int, P]
    lib.oracle_prune_channel_group.restype = None
    lib.oracle_attention_probs.argtypes = [P, ctypes.c_int, ctypes.c_int, P, ctypes.c_int, P,
                                           ctypes.c_int, ctypes.c_double, P]
    lib.oracle_attention_probs.restype = ctypes.c_int
    return lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data


def _bits(x) -> np.ndarray:
    """fp16 array (or uint16 bit patterns) -> contiguous uint16 bit patterns."""
    x = np.asarray(x)
    if x.dtype == np.float16:
        x = x.view(np.uint16)
    assert x.dtype == np.uint16, f"expected fp16 or uint16, got {x.dtype}"
    return np.ascontiguousarray(x)


def _map(fn, items, threads: int):
    if threads <= 1:
        return [fn(i) for i in items]
    with ThreadPoolExecutor(max_workers=threads) as pool:
        return list(pool.map(fn, items))


def half_to_double(h: int) -> float:
    return _load().oracle_half_to_double(int(h) & 0xFFFF)


def keep_count(d: int, sparsity: float) -> int:
    return _load().oracle_keep_count(int(d), float(sparsity))


def prune_token(x, k: int) -> np.ndarray:
    """Boolean keep-mask of one token (any length d >= 1)."""
    xb = _bits(x).reshape(-1)
    keep = np.zeros(xb.size, dtype=np.uint8)
    _load().oracle_prune_token(_ptr(xb), xb.size, int(k), _ptr(keep))
    return keep.astype(bool)


def token_max_elems(d: int, k: int) -> int:
    """Worst-case fp16 elements of one compressed token (every tile padded)."""
    T = d // TILE
    return min(d, (k + (PAD - 1) * min(k, T)) // PAD * PAD)


def compress(x, sparsity: float | None = None, *, k: int | None = None, threads: int = 1) -> dict:
    """Compress a dense cache x [B][H][N][d] (fp16) stream by stream.

    Returns a dict with ``bitmaps`` u64 [B][H][N][T], ``offsets`` u32 [B][H][N][T],
    ``values`` u16 [B][H][cap] (cap = N * worst case per token; entries past
    ``stream_len`` are zero), ``stream_len`` u32 [B][H], ``n_keep``, ``d``.
    """
    xb = _bits(x)
    B, H, N, d = xb.shape
    if k is None:
        k = keep_count(d, sparsity)
    T = d // TILE
    cap = max(N * token_max_elems(d, k), PAD)
    bitmaps = np.zeros((B, H, N, T), dtype=np.uint64)
    offsets = np.zeros((B, H, N, T), dtype=np.uint32)
    values = np.zeros((B, H, cap), dtype=np.uint16)
    stream_len = np.zeros((B, H), dtype=np.uint32)
    lib = _load()

    def one(bh):
        b, h = bh
        out_len = np.zeros(1, dtype=np.uint32)
        bm = np.zeros((N, T), dtype=np.uint64)
        off = np.zeros((N, T), dtype=np.uint32)
        val = np.zeros(cap, dtype=np.uint16)
        rc = lib.oracle_compress_stream(_ptr(np.ascontiguousarray(xb[b, h])), N, d, int(k),
                                        _ptr(bm), _ptr(off), _ptr(val), cap, _ptr(out_len))
        if rc != 0:
            raise ValueError(f"oracle_compress_stream failed with {rc}")
        bitmaps[b, h], offsets[b, h], values[b, h], stream_len[b, h] = bm, off, val, out_len[0]

    _map(one, [(b, h) for b in range(B) for h in range(H)], threads)
    return {"bitmaps": bitmaps, "offsets": offsets, "values": values,
            "stream_len": stream_len, "n_keep": int(k), "d": d}


def decompress(enc: dict, threads: int = 1) -> np.ndarray:
    """Zero-filled pruned cache [B][H][N][d] as uint16 fp16 bit patterns."""
    bitmaps, offsets, values = enc["bitmaps"], enc["offsets"], enc["values"]
    B, H, N, T = bitmaps.shape
    d = T * TILE
    out = np.zeros((B, H, N, d), dtype=np.uint16)
    lib = _load()

    def one(bh):
        b, h = bh
        dense = np.zeros((N, d), dtype=np.uint16)
        rc = lib.oracle_decompress_stream(_ptr(np.ascontiguousarray(bitmaps[b, h])),
                                          _ptr(np.ascontiguousarray(offsets[b, h])),
                                          _ptr(np.ascontiguousarray(values[b, h])), N, d,
                                          _ptr(dense))
        if rc != 0:
            raise ValueError(f"oracle_decompress_stream failed with {rc}")
        out[b, h] = dense

    _map(one, [(b, h) for b in range(B) for h in range(H)], threads)
    return out


def decode_attention(q, kc, vc, k_tail=None, v_tail=None, scale: float = 0.0,
                     threads: int = 1) -> np.ndarray:
    """Algorithm 1 per (batch, kv-head) in float64.

    q [B][Hq][d]; kc, vc [B][Hkv][Ns][d] zero-filled pruned caches (Ns may be 0);
    k_tail, v_tail [B][Hkv][Nd][d] or None. Query head h uses kv-head h // (Hq//Hkv).
    Returns float64 [B][Hq][d].
    """
    qb, kcb, vcb = _bits(q), _bits(kc), _bits(vc)
    B, Hq, d = qb.shape
    Hkv, Ns = kcb.shape[1], kcb.shape[2]
    if k_tail is None:
        klb = np.zeros((B, Hkv, 0, d), dtype=np.uint16)
        vlb = klb
    else:
        klb, vlb = _bits(k_tail), _bits(v_tail)
    Nd = klb.shape[2]
    G = Hq // Hkv
    out = np.zeros((B, Hq, d), dtype=np.float64)
    lib = _load()

    def one(bh):
        b, h = bh
        o = np.zeros((G, d), dtype=np.float64)
        rc = lib.oracle_decode_attention(
            _ptr(np.ascontiguousarray(qb[b, h * G:(h + 1) * G])), G, d,
            _ptr(np.ascontiguousarray(kcb[b, h])), _ptr(np.ascontiguousarray(vcb[b, h])), Ns,
            _ptr(np.ascontiguousarray(klb[b, h])), _ptr(np.ascontiguousarray(vlb[b, h])), Nd,
            float(scale), _ptr(o))
        if rc != 0:
            raise ValueError(f"oracle_decode_attention failed with {rc}")
        out[b, h * G:(h + 1) * G] = o

    _map(one, [(b, h) for b in range(B) for h in range(Hkv)], threads)
    return out


def sparse_decode_attention(q, enc_k: dict, enc_v: dict, k_tail=None, v_tail=None,
                            scale: float = 0.0, threads: int = 1) -> np.ndarray:
    """Algorithm 1 with the compressed caches given in the oracle's own format."""
    kc = decompress(enc_k, threads=threads)
    vc = decompress(enc_v, threads=threads)
    return decode_attention(q, kc, vc, k_tail, v_tail, scale, threads=threads)


def prune_token_24(x) -> np.ndarray:
    """Keep-mask of one token under 2:4 pruning (2 of every 4 consecutive channels)."""
    xb = _bits(x).reshape(-1)
    keep = np.zeros(xb.size, dtype=np.uint8)
    _load().oracle_prune_token_24(_ptr(xb), xb.size, _ptr(keep))
    return keep.astype(bool)


def prune_token_scored(x, w, k: int) -> np.ndarray:
    """Keep-mask of one key token under output-aware pruning: the k channels of
    largest fp32 score |x_c| * w_c (w: float32 channel weights)."""
    xb = _bits(x).reshape(-1)
    wf = np.ascontiguousarray(np.asarray(w, dtype=np.float32).reshape(-1))
    keep = np.zeros(xb.size, dtype=np.uint8)
    _load().oracle_prune_token_scored(_ptr(xb), _ptr(wf), xb.size, int(k), _ptr(keep))
    return keep.astype(bool)


def compress_variant(x, mode: str = "magnitude", *, k: int | None = None, head_keep=None,
                     weights=None, threads: int = 1) -> dict:
    """The compressed format of x [B][H][N][d] under a pruner variant.

    mode "magnitude": k kept channels per token (head h keeps head_keep[h] if given);
    mode "2:4": 2 of every 4 consecutive channels; mode "output_aware": k (or
    head_keep[h]) channels of largest |x| * weights, weights float32 [B][H][N][d].
    Same dict as ``compress``.
    """
    xb = _bits(x)
    B, H, N, d = xb.shape
    T = d // TILE
    if mode == "2:4":
        ks = [d // 2] * H
    elif head_keep is not None:
        ks = [int(v) for v in head_keep]
    else:
        ks = [int(k)] * H
    cap = max(N * token_max_elems(d, max(ks)), PAD)
    bitmaps = np.zeros((B, H, N, T), dtype=np.uint64)
    offsets = np.zeros((B, H, N, T), dtype=np.uint32)
    values = np.zeros((B, H, cap), dtype=np.uint16)
    stream_len = np.zeros((B, H), dtype=np.uint32)
    if mode == "output_aware":
        wts = np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
    lib = _load()

    def one(bh):
        b, h = bh
        xs = np.ascontiguousarray(xb[b, h])
        keep = np.zeros((N, d), dtype=np.uint8)
        for j in range(N):
            row = np.zeros(d, dtype=np.uint8)
            if mode == "magnitude":
                lib.oracle_prune_token(_ptr(np.ascontiguousarray(xs[j])), d, ks[h], _ptr(row))
            elif mode == "2:4":
                lib.oracle_prune_token_24(_ptr(np.ascontiguousarray(xs[j])), d, _ptr(row))
            elif mode == "output_aware":
                lib.oracle_prune_token_scored(_ptr(np.ascontiguousarray(xs[j])),
                                              _ptr(np.ascontiguousarray(wts[b, h, j])), d, ks[h],
                                              _ptr(row))
            else:
                raise ValueError(mode)
            keep[j] = row
        out_len = np.zeros(1, dtype=np.uint32)
        bm = np.zeros((N, T), dtype=np.uint64)
        off = np.zeros((N, T), dtype=np.uint32)
        val = np.zeros(cap, dtype=np.uint16)
        rc = lib.oracle_encode_stream(_ptr(xs), _ptr(keep), N, d, _ptr(bm), _ptr(off), _ptr(val),
                                      cap, _ptr(out_len))
        if rc != 0:
            raise ValueError(f"oracle_encode_stream failed with {rc}")
        bitmaps[b, h], offsets[b, h], values[b, h], stream_len[b, h] = bm, off, val, out_len[0]

    _map(one, [(b, h) for b in range(B) for h in range(H)], threads)
    return {"bitmaps": bitmaps, "offsets": offsets, "values": values,
            "stream_len": stream_len, "n_keep": max(ks), "d": d}


def query_lookahead(q, Hkv: int, L: int = 32) -> np.ndarray:
    """Channel weights of output-aware key pruning (Sec. 2): for key token T of
    kv-head h, the L1 sum over the queries t = T .. T+L-1 (those that exist) and
    over the query heads of h's group of |q_t|, in float32, added in the order
    t ascending, then query head ascending.

    q [B][Hq][Nq][d] fp16 (one query per token position). Returns float32
    [B][Hkv][Nq][d].
    """
    qb = _bits(q)
    B, Hq, Nq, d = qb.shape
    G = Hq // Hkv
    mag = np.abs(qb.view(np.float16).astype(np.float32))
    out = np.zeros((B, Hkv, Nq, d), dtype=np.float32)
    for b in range(B):
        for h in range(Hkv):
            for T in range(Nq):
                acc = np.zeros(d, dtype=np.float32)
                for t in range(T, min(T + L, Nq)):
                    for g in range(G):
                        acc = acc + mag[b, h * G + g, t]
                out[b, h, T] = acc
    return out


def compressed_bytes(enc: dict) -> int:
    """Bytes of the compressed format: 8-byte bitmap + 4-byte offset per tile plus
    2 bytes per stored fp16 element (padding included)."""
    tiles = enc["bitmaps"].size
    return 12 * tiles + 2 * int(enc["stream_len"].astype(np.int64).sum())


# ---- per-channel value pruning in groups of 32 tokens ------------------------------------
def prune_channel_group(x, k: int, w=None) -> np.ndarray:
    """Keep-mask [n][d] of a group of n tokens x [n][d]: per channel the k tokens
    of largest |x| (or, with token weights w float32 [n], of largest fp32
    |x| * w_j), ties to the lower token."""
    xb = np.ascontiguousarray(_bits(x))
    n, d = xb.shape
    keep = np.zeros((n, d), dtype=np.uint8)
    wf = None if w is None else np.ascontiguousarray(np.asarray(w, dtype=np.float32).reshape(-1))
    _load().oracle_prune_channel_group(_ptr(xb), _ptr(wf), n, d, int(k), _ptr(keep))
    return keep.astype(bool)


def grouped_stream_capacity(d: int, k: int, n_tokens: int) -> int:
    """Worst-case fp16 elements of n_tokens (a multiple of 32) pruned per channel:
    per group k * d kept values plus at most 7 pad slots in each of its 32 * T tiles."""
    T = d // TILE
    return n_tokens // GROUP * (k * d + GROUP * T * (PAD - 1))


def compress_grouped(x, sparsity: float | None = None, *, k: int | None = None, weights=None,
                     threads: int = 1) -> dict:
    """The compressed format of x [B][H][N][d] (N a multiple of 32) pruned per
    channel in groups of 32 consecutive tokens: each channel keeps k =
    keep_count(32, sparsity) of every group (output-aware with token weights
    float32 [B][H][N] if given). Same dict as ``compress``; ``n_keep`` is k."""
    xb = _bits(x)
    B, H, N, d = xb.shape
    if N % GROUP:
        raise ValueError("per-channel pruning takes whole groups of 32 tokens")
    if k is None:
        k = keep_count(GROUP, sparsity)
    T = d // TILE
    cap = max(grouped_stream_capacity(d, k, N), PAD)
    bitmaps = np.zeros((B, H, N, T), dtype=np.uint64)
    offsets = np.zeros((B, H, N, T), dtype=np.uint32)
    values = np.zeros((B, H, cap), dtype=np.uint16)
    stream_len = np.zeros((B, H), dtype=np.uint32)
    wts = None if weights is None else np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
    lib = _load()

    def one(bh):
        b, h = bh
        xs = np.ascontiguousarray(xb[b, h])
        keep = np.zeros((N, d), dtype=np.uint8)
        for g0 in range(0, N, GROUP):
            part = np.zeros((GROUP, d), dtype=np.uint8)
            wg = None if wts is None else np.ascontiguousarray(wts[b, h, g0:g0 + GROUP])
            lib.oracle_prune_channel_group(_ptr(np.ascontiguousarray(xs[g0:g0 + GROUP])), _ptr(wg),
                                           GROUP, d, int(k), _ptr(part))
            keep[g0:g0 + GROUP] = part
        out_len = np.zeros(1, dtype=np.uint32)
        bm = np.zeros((N, T), dtype=np.uint64)
        off = np.zeros((N, T), dtype=np.uint32)
        val = np.zeros(cap, dtype=np.uint16)
        rc = lib.oracle_encode_stream(_ptr(xs), _ptr(keep), N, d, _ptr(bm), _ptr(off), _ptr(val),
                                      cap, _ptr(out_len))
        if rc != 0:
            raise ValueError(f"oracle_encode_stream failed with {rc}")
        bitmaps[b, h], offsets[b, h], values[b, h], stream_len[b, h] = bm, off, val, out_len[0]

    _map(one, [(b, h) for b in range(B) for h in range(H)], threads)
    return {"bitmaps": bitmaps, "offsets": offsets, "values": values,
            "stream_len": stream_len, "n_keep": int(k), "d": d}


def encode(x, keep, threads: int = 1) -> dict:
    """The compressed format of x [B][H][N][d] with the kept channels given by
    keep [B][H][N][d] (bool). Same dict as ``compress`` (``n_keep`` is d)."""
    xb = _bits(x)
    B, H, N, d = xb.shape
    T = d // TILE
    cap = max(N * d, PAD)
    kp = np.ascontiguousarray(np.asarray(keep, dtype=np.uint8))
    bitmaps = np.zeros((B, H, N, T), dtype=np.uint64)
    offsets = np.zeros((B, H, N, T), dtype=np.uint32)
    values = np.zeros((B, H, cap), dtype=np.uint16)
    stream_len = np.zeros((B, H), dtype=np.uint32)
    lib = _load()

    def one(bh):
        b, h = bh
        out_len = np.zeros(1, dtype=np.uint32)
        bm = np.zeros((N, T), dtype=np.uint64)
        off = np.zeros((N, T), dtype=np.uint32)
        val = np.zeros(cap, dtype=np.uint16)
        rc = lib.oracle_encode_stream(_ptr(np.ascontiguousarray(xb[b, h])),
                                      _ptr(np.ascontiguousarray(kp[b, h])), N, d, _ptr(bm),
                                      _ptr(off), _ptr(val), cap, _ptr(out_len))
        if rc != 0:
            raise ValueError(f"oracle_encode_stream failed with {rc}")
        bitmaps[b, h], offsets[b, h], values[b, h], stream_len[b, h] = bm, off, val, out_len[0]

    _map(one, [(b, h) for b in range(B) for h in range(H)], threads)
    return {"bitmaps": bitmaps, "offsets": offsets, "values": values,
            "stream_len": stream_len, "n_keep": d, "d": d}


def attention_probs(q, kc, k_tail=None, scale: float = 0.0) -> np.ndarray:
    """Softmax weights of Algorithm 1 in float64: q [B][Hq][d], kc [B][Hkv][Ns][d]
    zero-filled pruned keys, k_tail [B][Hkv][Nd][d] or None. Returns [B][Hq][Ns+Nd]
    (compressed tokens first, then the dense ones)."""
    qb, kcb = _bits(q), _bits(kc)
    B, Hq, d = qb.shape
    Hkv, Ns = kcb.shape[1], kcb.shape[2]
    klb = np.zeros((B, Hkv, 0, d), dtype=np.uint16) if k_tail is None else _bits(k_tail)
    Nd = klb.shape[2]
    G = Hq // Hkv
    out = np.zeros((B, Hq, Ns + Nd), dtype=np.float64)
    lib = _load()
    for b in range(B):
        for h in range(Hkv):
            p = np.zeros((G, Ns + Nd), dtype=np.float64)
            rc = lib.oracle_attention_probs(
                _ptr(np.ascontiguousarray(qb[b, h * G:(h + 1) * G])), G, d,
                _ptr(np.ascontiguousarray(kcb[b, h])), Ns, _ptr(np.ascontiguousarray(klb[b, h])), Nd,
                float(scale), _ptr(p))
            if rc != 0:
                raise ValueError(f"oracle_attention_probs failed with {rc}")
            out[b, h * G:(h + 1) * G] = p
    return out
