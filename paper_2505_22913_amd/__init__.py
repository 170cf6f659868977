"""MI355X (gfx950) implementation of MUSTAFAR's decode hot path (arxiv 2505.22913).

Thin ctypes binding of ``libmustafar.so``; every step of the path runs in the
library's HIP kernels. Function names mirror the C ABI in ``include/mustafar.h``;
this module only turns torch tensors into device pointers, passes the current
HIP stream and raises ``MustafarError`` on a non-zero status. torch is used for
device memory and streams only.

The library is loaded on first use; if it has not been built the call raises
(there is no CPU fallback). Build it with
``python -m paper_2505_22913_amd.build_lib`` or ``__graft_entry__.build()``.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmustafar.so")
TILE = 64
PAD = 8

OK, EINVAL, ECAPACITY, EWORKSPACE, ELAUNCH, EUNSUPPORTED, ESCRATCH = 0, -1, -2, -3, -4, -5, -6
STATIC_SCRATCH_BYTES = 32 << 20   # the static buffer of mustafar_sparse_decode_attn_static
STREAM_POISONED = 0xFFFFFFFF   # stream_len of a stream whose bulk compression gave up
LOOKBACK_POLLS = 1 << 20

_lib = None


class MustafarError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {status} ({strerror(status)})")
        self.status = status


class ccache_t(ctypes.Structure):
    """Mirror of ``mustafar_ccache_t``."""
    _fields_ = [("bitmaps", ctypes.c_void_p), ("offsets", ctypes.c_void_p),
                ("values", ctypes.c_void_p), ("stream_len", ctypes.c_void_p),
                ("B", ctypes.c_int32), ("H", ctypes.c_int32), ("d", ctypes.c_int32),
                ("n_keep", ctypes.c_int32), ("cap_tokens", ctypes.c_int32),
                ("n_tokens", ctypes.c_int32), ("val_stride", ctypes.c_int64),
                ("group_keep", ctypes.c_int32)]


class window_t(ctypes.Structure):
    """Mirror of ``mustafar_window_t``."""
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("len", ctypes.c_void_p),
                ("head", ctypes.c_void_p), ("n_comp", ctypes.c_void_p),
                ("B", ctypes.c_int32), ("H", ctypes.c_int32), ("d", ctypes.c_int32),
                ("W", ctypes.c_int32), ("max_len", ctypes.c_int32)]


class prune_opts_t(ctypes.Structure):
    """Mirror of ``mustafar_prune_opts_t``."""
    _fields_ = [("mode", ctypes.c_int32), ("head_keep", ctypes.c_void_p),
                ("weights", ctypes.c_void_p)]


PRUNE_MAGNITUDE, PRUNE_2_4, PRUNE_OUTPUT_AWARE = 0, 1, 2
PRUNE_CHANNEL, PRUNE_CHANNEL_OUTPUT_AWARE = 3, 4
ATTN_SPARSE, ATTN_DENSE = 0, 1
GROUP = 32  # tokens per group of per-channel value pruning

_SIGS = {
    "mustafar_keep_count": (ctypes.c_int, [ctypes.c_int, ctypes.c_float]),
    "mustafar_token_max_elems": (ctypes.c_int64, [ctypes.c_int, ctypes.c_int]),
    "mustafar_stream_capacity": (ctypes.c_int64, [ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "mustafar_ccache_init": (ctypes.c_int, [ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                            ctypes.c_float, ctypes.c_int, ctypes.c_int64]),
    "mustafar_grouped_stream_capacity": (ctypes.c_int64, [ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "mustafar_ccache_init_grouped": (ctypes.c_int, [ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                    ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                                    ctypes.c_float, ctypes.c_int, ctypes.c_int64]),
    "mustafar_compress_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int] * 3),
    "mustafar_prune_compress": (ctypes.c_int, [ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                               ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t,
                                               ctypes.c_void_p]),
    "mustafar_prune_compress_bounded": (ctypes.c_int, [ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                                       ctypes.c_int, ctypes.c_uint32, ctypes.c_void_p,
                                                       ctypes.c_size_t, ctypes.c_void_p]),
    "mustafar_append_kv": (ctypes.c_int, [ctypes.POINTER(ccache_t), ctypes.POINTER(ccache_t),
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "mustafar_append": (ctypes.c_int, [ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                       ctypes.c_void_p]),
    "mustafar_attn_default_splits": (ctypes.c_int, [ctypes.c_int] * 5),
    "mustafar_attn_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int] * 6),
    "mustafar_sparse_decode_attn": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                                   ctypes.POINTER(ccache_t),
                                                   ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                                   ctypes.c_void_p, ctypes.c_int, ctypes.c_float,
                                                   ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                                   ctypes.c_size_t, ctypes.c_void_p]),
    "mustafar_sparse_decode_attn_static": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                                          ctypes.POINTER(ccache_t),
                                                          ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                                          ctypes.c_void_p, ctypes.c_int, ctypes.c_float,
                                                          ctypes.c_void_p, ctypes.c_int,
                                                          ctypes.c_void_p]),
    "mustafar_dense_decode_attn": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                                  ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                                  ctypes.c_int, ctypes.c_int, ctypes.c_float,
                                                  ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                                  ctypes.c_size_t, ctypes.c_void_p]),
    "mustafar_window_init": (ctypes.c_int, [ctypes.POINTER(window_t)] + [ctypes.c_void_p] * 5
                             + [ctypes.c_int] * 5),
    "mustafar_window_prefill": (ctypes.c_int, [ctypes.POINTER(window_t), ctypes.POINTER(ccache_t),
                                               ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                               ctypes.c_void_p, ctypes.c_int,
                                               ctypes.POINTER(ctypes.c_int32), ctypes.c_void_p,
                                               ctypes.c_size_t, ctypes.c_void_p]),
    "mustafar_window_step": (ctypes.c_int, [ctypes.POINTER(window_t), ctypes.POINTER(ccache_t),
                                            ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "mustafar_window_step_weighted": (ctypes.c_int, [ctypes.POINTER(window_t), ctypes.POINTER(ccache_t),
                                                     ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                     ctypes.c_void_p]),
    "mustafar_window_key_weights": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                                   ctypes.POINTER(window_t), ctypes.c_void_p,
                                                   ctypes.c_void_p, ctypes.c_void_p]),
    "mustafar_window_decode_attn": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                                   ctypes.POINTER(ccache_t),
                                                   ctypes.POINTER(ccache_t),
                                                   ctypes.POINTER(window_t), ctypes.c_float,
                                                   ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p,
                                                   ctypes.c_size_t, ctypes.c_void_p]),
    "mustafar_window_decode_attn_scores": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                                          ctypes.POINTER(ccache_t),
                                                          ctypes.POINTER(ccache_t),
                                                          ctypes.POINTER(window_t), ctypes.c_void_p,
                                                          ctypes.c_void_p,
                                                          ctypes.c_float, ctypes.c_void_p, ctypes.c_int,
                                                          ctypes.c_void_p, ctypes.c_size_t,
                                                          ctypes.c_void_p]),
    "mustafar_window_step_grouped": (ctypes.c_int, [ctypes.POINTER(window_t), ctypes.POINTER(ccache_t),
                                                    ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                    ctypes.c_void_p]),
    "mustafar_prune_compress_ex": (ctypes.c_int, [ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                                  ctypes.c_int, ctypes.POINTER(prune_opts_t),
                                                  ctypes.c_void_p, ctypes.c_size_t,
                                                  ctypes.c_void_p]),
    "mustafar_append_ex": (ctypes.c_int, [ctypes.POINTER(ccache_t), ctypes.c_void_p,
                                          ctypes.POINTER(prune_opts_t), ctypes.c_void_p]),
    "mustafar_query_lookahead": (ctypes.c_int, [ctypes.c_void_p] + [ctypes.c_int] * 6
                                 + [ctypes.c_void_p, ctypes.c_void_p]),
    "mustafar_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "mustafar_stream_read_sink_bytes": (ctypes.c_size_t, []),
    "mustafar_stream_read": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                            ctypes.c_void_p]),
    "mustafar_attn_set_route": (ctypes.c_int, [ctypes.c_int]),
    "mustafar_attn_route": (ctypes.c_int, []),
    "mustafar_stream_mix": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int,
                                           ctypes.c_void_p, ctypes.c_void_p]),
    "mustafar_stream_chunks": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                              ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]),
}


def lib() -> ctypes.CDLL:
    """The loaded library; raises if libmustafar.so has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2505_22913_amd.build_lib` (no CPU fallback)")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(handle, name)
            fn.restype, fn.argtypes = res, args
        _lib = handle
    return _lib


def strerror(status: int) -> str:
    try:
        return lib().mustafar_strerror(int(status)).decode()
    except Exception:  # noqa: BLE001 - the message is best effort
        return "unknown"


def _check(fn: str, status: int) -> None:
    if status != OK:
        raise MustafarError(fn, status)


def _dptr(t) -> int | None:
    """Device pointer of a CUDA (HIP) tensor; None for None."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("libmustafar takes device tensors only")
    return t.data_ptr()


def _stream(stream) -> int | None:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


# ---- host-only helpers --------------------------------------------------------------------
def mustafar_keep_count(d: int, sparsity: float) -> int:
    k = lib().mustafar_keep_count(int(d), float(sparsity))
    _check("mustafar_keep_count", min(k, 0))
    return k


def mustafar_token_max_elems(d: int, n_keep: int) -> int:
    return lib().mustafar_token_max_elems(int(d), int(n_keep))


def mustafar_stream_capacity(d: int, n_keep: int, cap_tokens: int) -> int:
    return lib().mustafar_stream_capacity(int(d), int(n_keep), int(cap_tokens))


def mustafar_compress_workspace_bytes(B: int, H: int, n_new: int) -> int:
    return lib().mustafar_compress_workspace_bytes(int(B), int(H), int(n_new))


def mustafar_attn_default_splits(B: int, Hq: int, Hkv: int, n_tokens: int,
                                 kind: int = ATTN_SPARSE) -> int:
    return lib().mustafar_attn_default_splits(int(B), int(Hq), int(Hkv), int(n_tokens), int(kind))


def mustafar_attn_workspace_bytes(B: int, Hq: int, Hkv: int, d: int, n_tokens: int,
                                  n_splits: int = 0) -> int:
    return lib().mustafar_attn_workspace_bytes(int(B), int(Hq), int(Hkv), int(d), int(n_tokens),
                                               int(n_splits))


# ---- the compressed cache -----------------------------------------------------------------
class CompressedCache:
    """A compressed K or V cache: device buffers (torch) plus the C descriptor.

    bitmaps u64 [B][H][cap][d/64], offsets u32 [B][H][cap][d/64],
    values fp16 bits [B][H][val_stride], stream_len u32 [B][H].

    The capacity is rounded up to a multiple of ``align`` tokens (64 by default),
    so that every stream's bitmaps and offsets start on a 256-byte boundary: the
    attention kernels read them in 32-token blocks, and a block that straddles
    an extra 128-byte line costs 5% more traffic.
    """

    def __init__(self, B: int, H: int, d: int, sparsity: float, cap_tokens: int, device="cuda",
                 grouped: bool = False, align: int = 64):
        import torch
        T = d // TILE
        cap_tokens = (int(cap_tokens) + align - 1) // align * align
        if grouped:   # per-channel pruning in groups of 32 tokens
            stride = lib().mustafar_grouped_stream_capacity(d, mustafar_keep_count(GROUP, sparsity),
                                                            cap_tokens)
        else:
            stride = mustafar_stream_capacity(d, mustafar_keep_count(d, sparsity), cap_tokens)
        stride = max(PAD, (stride + PAD - 1) // PAD * PAD)
        self.bitmaps = torch.zeros((B, H, cap_tokens, T), dtype=torch.int64, device=device)
        self.offsets = torch.zeros((B, H, cap_tokens, T), dtype=torch.int32, device=device)
        self.values = torch.zeros((B, H, stride), dtype=torch.int16, device=device)
        self.stream_len = torch.zeros((B, H), dtype=torch.int32, device=device)
        self.desc = ccache_t()
        init = "mustafar_ccache_init_grouped" if grouped else "mustafar_ccache_init"
        _check(init, getattr(lib(), init)(
            ctypes.byref(self.desc), self.bitmaps.data_ptr(), self.offsets.data_ptr(),
            self.values.data_ptr(), self.stream_len.data_ptr(), B, H, d, float(sparsity),
            cap_tokens, stride))

    @property
    def n_tokens(self) -> int:
        return self.desc.n_tokens

    @property
    def n_keep(self) -> int:
        return self.desc.n_keep

    @property
    def group_keep(self) -> int:
        return self.desc.group_keep

    @property
    def shape(self):
        return self.desc.B, self.desc.H, self.desc.d


def mustafar_prune_compress(cache: CompressedCache, x, ws=None, stream=None) -> None:
    """Append x [B][H][n_new][d] (fp16, device) to the cache, pruned and compressed."""
    import torch
    n_new = int(x.shape[2])
    need = mustafar_compress_workspace_bytes(cache.desc.B, cache.desc.H, n_new)
    if ws is None:
        ws = torch.empty(max(need, 4), dtype=torch.uint8, device=x.device)
    _check("mustafar_prune_compress", lib().mustafar_prune_compress(
        ctypes.byref(cache.desc), _dptr(x), n_new, _dptr(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def mustafar_prune_compress_bounded(cache: CompressedCache, x, max_polls: int, ws=None,
                                    stream=None) -> None:
    """mustafar_prune_compress with the caller's bound on a chunk's look-back polls."""
    import torch
    n_new = int(x.shape[2])
    need = mustafar_compress_workspace_bytes(cache.desc.B, cache.desc.H, n_new)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=x.device)
    _check("mustafar_prune_compress_bounded", lib().mustafar_prune_compress_bounded(
        ctypes.byref(cache.desc), _dptr(x), n_new, int(max_polls), _dptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def compress_status(ws) -> int:
    """The status word a bulk compression left at the start of its workspace: 0 if
    every stream was compressed, nonzero if a stream was poisoned (synchronises)."""
    return int(ws[:4].view(dtype=__import__("torch").int32).item())


def mustafar_append_kv(Kc: CompressedCache, Vc: CompressedCache, k_new, v_new, stream=None) -> None:
    """Append one decode step's key and value per stream, [B][H][d] fp16 each, in one launch."""
    _check("mustafar_append_kv", lib().mustafar_append_kv(ctypes.byref(Kc.desc), ctypes.byref(Vc.desc),
                                                          _dptr(k_new), _dptr(v_new), _stream(stream)))


def mustafar_append(cache: CompressedCache, x_new, stream=None) -> None:
    """Append one token per stream, x_new [B][H][d] (fp16, device)."""
    _check("mustafar_append", lib().mustafar_append(ctypes.byref(cache.desc), _dptr(x_new),
                                                    _stream(stream)))


def _prune_opts(mode, head_keep, weights):
    """(prune_opts_t, keep-alive objects) for the _ex calls."""
    o = prune_opts_t()
    o.mode = int(mode)
    keep = None
    if head_keep is not None:
        keep = (ctypes.c_int32 * len(head_keep))(*[int(v) for v in head_keep])
        o.head_keep = ctypes.cast(keep, ctypes.c_void_p)
    o.weights = _dptr(weights)
    return o, keep


def mustafar_prune_compress_ex(cache: CompressedCache, x, mode: int = 0, head_keep=None,
                               weights=None, ws=None, stream=None) -> None:
    """mustafar_prune_compress under a pruner variant (PRUNE_MAGNITUDE with optional
    per-head counts, PRUNE_2_4, PRUNE_OUTPUT_AWARE with fp32 weights [B][H][n_new][d];
    on per-channel caches PRUNE_CHANNEL, PRUNE_CHANNEL_OUTPUT_AWARE with fp32 token
    weights [B][H][n_new])."""
    import torch
    n_new = int(x.shape[2])
    need = mustafar_compress_workspace_bytes(cache.desc.B, cache.desc.H, n_new)
    if ws is None:
        ws = torch.empty(max(need, 4), dtype=torch.uint8, device=x.device)
    o, _keep = _prune_opts(mode, head_keep, weights)
    _check("mustafar_prune_compress_ex", lib().mustafar_prune_compress_ex(
        ctypes.byref(cache.desc), _dptr(x), n_new, ctypes.byref(o), _dptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def mustafar_append_ex(cache: CompressedCache, x_new, mode: int = 0, head_keep=None, weights=None,
                       stream=None) -> None:
    """mustafar_append under a pruner variant (weights fp32 [B][H][d] when output-aware)."""
    o, _keep = _prune_opts(mode, head_keep, weights)
    _check("mustafar_append_ex", lib().mustafar_append_ex(
        ctypes.byref(cache.desc), _dptr(x_new), ctypes.byref(o), _stream(stream)))


def mustafar_query_lookahead(q, Hkv: int, L: int = 32, out=None, stream=None):
    """Output-aware channel weights from queries q [B][Hq][n_q][d] fp16: fp32
    [B][Hkv][n_q][d]."""
    import torch
    B, Hq, n_q, d = (int(s) for s in q.shape)
    if out is None:
        out = torch.empty((B, Hkv, n_q, d), dtype=torch.float32, device=q.device)
    _check("mustafar_query_lookahead", lib().mustafar_query_lookahead(
        _dptr(q), B, Hq, int(Hkv), n_q, d, int(L), _dptr(out), _stream(stream)))
    return out


def _attn_ws(B, Hq, Hkv, d, n, n_splits, ws, device):
    import torch
    need = mustafar_attn_workspace_bytes(B, Hq, Hkv, d, n, n_splits)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=device)
    return ws


def mustafar_sparse_decode_attn(q, Kc: CompressedCache, Vc: CompressedCache, k_tail=None,
                                v_tail=None, scale: float = 0.0, out=None, n_splits: int = 0,
                                ws=None, stream=None):
    """Algorithm 1: attention of q [B][Hq][d] over the compressed caches plus the dense
    window [B][Hkv][n_tail][d]. Returns out [B][Hq][d] fp16."""
    import torch
    B, Hq, d = (int(s) for s in q.shape)
    Hkv = Kc.desc.H
    n_tail = 0 if k_tail is None else int(k_tail.shape[2])
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.float16, device=q.device)
    ws = _attn_ws(B, Hq, Hkv, d, Kc.n_tokens, n_splits, ws, q.device)
    _check("mustafar_sparse_decode_attn", lib().mustafar_sparse_decode_attn(
        _dptr(q), B, Hq, ctypes.byref(Kc.desc), ctypes.byref(Vc.desc), _dptr(k_tail),
        _dptr(v_tail), n_tail, float(scale), _dptr(out), int(n_splits), _dptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))
    return out


def mustafar_sparse_decode_attn_static(q, Kc: CompressedCache, Vc: CompressedCache, k_tail=None,
                                       v_tail=None, scale: float = 0.0, out=None, n_splits: int = 0,
                                       stream=None):
    """mustafar_sparse_decode_attn with its partials in the library's static device
    buffer (no workspace; for callers that cannot allocate). out may be preallocated."""
    import torch
    B, Hq, d = (int(s) for s in q.shape)
    n_tail = 0 if k_tail is None else int(k_tail.shape[2])
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.float16, device=q.device)
    _check("mustafar_sparse_decode_attn_static", lib().mustafar_sparse_decode_attn_static(
        _dptr(q), B, Hq, ctypes.byref(Kc.desc), ctypes.byref(Vc.desc), _dptr(k_tail), _dptr(v_tail),
        n_tail, float(scale), _dptr(out), int(n_splits), _stream(stream)))
    return out


def mustafar_dense_decode_attn(q, k, v, scale: float = 0.0, out=None, n_splits: int = 0, ws=None,
                               stream=None):
    """Dense baseline: q [B][Hq][d] over k, v [B][Hkv][N][d] fp16. Returns out fp16."""
    import torch
    B, Hq, d = (int(s) for s in q.shape)
    Hkv, N = int(k.shape[1]), int(k.shape[2])
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.float16, device=q.device)
    ws = _attn_ws(B, Hq, Hkv, d, N, n_splits, ws, q.device)
    _check("mustafar_dense_decode_attn", lib().mustafar_dense_decode_attn(
        _dptr(q), B, Hq, Hkv, _dptr(k), _dptr(v), N, d, float(scale), _dptr(out), int(n_splits),
        _dptr(ws), ws.numel() * ws.element_size(), _stream(stream)))
    return out


# ---- the dense local window (lifecycle) -------------------------------------------------
class DenseWindow:
    """The dense window of the W most recent tokens of every stream: ring slots
    k, v [B][H][W][d] fp16 and int32 device state len, head, n_comp [B]."""

    def __init__(self, B: int, H: int, d: int, W: int, device="cuda"):
        import torch
        self.k = torch.zeros((B, H, W, d), dtype=torch.float16, device=device)
        self.v = torch.zeros((B, H, W, d), dtype=torch.float16, device=device)
        self.len = torch.zeros(B, dtype=torch.int32, device=device)
        self.head = torch.zeros(B, dtype=torch.int32, device=device)
        self.n_comp = torch.zeros(B, dtype=torch.int32, device=device)
        self.desc = window_t()
        _check("mustafar_window_init", lib().mustafar_window_init(
            ctypes.byref(self.desc), self.k.data_ptr(), self.v.data_ptr(), self.len.data_ptr(),
            self.head.data_ptr(), self.n_comp.data_ptr(), B, H, d, W, 0))

    @property
    def W(self) -> int:
        return self.desc.W

    @property
    def max_len(self) -> int:
        return self.desc.max_len


def mustafar_window_prefill(win: DenseWindow, Kc: CompressedCache, Vc: CompressedCache, x_k, x_v,
                            seq_len, ws=None, stream=None) -> None:
    """Prompts of seq_len[b] tokens (host ints) in x_k, x_v [B][H][n_max][d] fp16: the
    tokens before each entry's last min(seq_len[b], W) are compressed, the rest fill
    its window."""
    import torch
    n_max = int(x_k.shape[2])
    lens = (ctypes.c_int32 * len(seq_len))(*[int(n) for n in seq_len])
    need = mustafar_compress_workspace_bytes(1, win.desc.H, max(n_max, 1))
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=x_k.device)
    _check("mustafar_window_prefill", lib().mustafar_window_prefill(
        ctypes.byref(win.desc), ctypes.byref(Kc.desc), ctypes.byref(Vc.desc), _dptr(x_k),
        _dptr(x_v), n_max, lens, _dptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def mustafar_window_step(win: DenseWindow, Kc: CompressedCache, Vc: CompressedCache, k_new, v_new,
                         active=None, stream=None) -> None:
    """One decode step: k_new, v_new [B][H][d] enter the windows of the active entries
    (active: int32 device [B] or None); full windows first hand their oldest token
    to the compressed caches."""
    _check("mustafar_window_step", lib().mustafar_window_step(
        ctypes.byref(win.desc), ctypes.byref(Kc.desc), ctypes.byref(Vc.desc), _dptr(k_new),
        _dptr(v_new), _dptr(active), _stream(stream)))


def mustafar_window_step_weighted(win: DenseWindow, Kc: CompressedCache, Vc: CompressedCache, k_new,
                                  v_new, kacc, active=None, stream=None) -> None:
    """mustafar_window_step whose leaving key is pruned output-aware with its window
    slot's weights in kacc [B][H][W][d] (fp32, device); the new token's weights start
    at 0."""
    _check("mustafar_window_step_weighted", lib().mustafar_window_step_weighted(
        ctypes.byref(win.desc), ctypes.byref(Kc.desc), ctypes.byref(Vc.desc), _dptr(k_new),
        _dptr(v_new), _dptr(active), _dptr(kacc), _stream(stream)))


def mustafar_window_key_weights(q, win: DenseWindow, kacc, active=None, stream=None) -> None:
    """kacc[b][h][slot] += |q| of the query heads of kv-head h (one after the other, in
    fp32) for the newest 32 window tokens of every active entry (active: int32 device
    [B] or None for all); q [B][Hq][d] fp16."""
    B, Hq, _ = (int(s) for s in q.shape)
    _check("mustafar_window_key_weights", lib().mustafar_window_key_weights(
        _dptr(q), B, Hq, ctypes.byref(win.desc), _dptr(active), _dptr(kacc), _stream(stream)))


def mustafar_window_decode_attn(q, Kc: CompressedCache, Vc: CompressedCache, win: DenseWindow,
                                scale: float = 0.0, out=None, n_splits: int = 0, ws=None,
                                stream=None):
    """Algorithm 1 per batch entry over its compressed tokens and its window."""
    import torch
    B, Hq, d = (int(s) for s in q.shape)
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.float16, device=q.device)
    ws = _attn_ws(B, Hq, Kc.desc.H, d, Kc.n_tokens, n_splits, ws, q.device)
    _check("mustafar_window_decode_attn", lib().mustafar_window_decode_attn(
        _dptr(q), B, Hq, ctypes.byref(Kc.desc), ctypes.byref(Vc.desc), ctypes.byref(win.desc),
        float(scale), _dptr(out), int(n_splits), _dptr(ws), ws.numel() * ws.element_size(),
        _stream(stream)))
    return out


def mustafar_window_decode_attn_scores(q, Kc: CompressedCache, Vc: CompressedCache,
                                       win: DenseWindow, acc, scale: float = 0.0, out=None,
                                       n_splits: int = 0, ws=None, active=None, stream=None):
    """mustafar_window_decode_attn, then acc [B][H][W] (fp32, device) += the attention
    probability, summed over each kv-head's query heads, of every window token
    younger than 32 steps, for the active entries (active: int32 device [B] or None)."""
    import torch
    B, Hq, d = (int(s) for s in q.shape)
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.float16, device=q.device)
    ws = _attn_ws(B, Hq, Kc.desc.H, d, Kc.n_tokens, n_splits, ws, q.device)
    _check("mustafar_window_decode_attn_scores", lib().mustafar_window_decode_attn_scores(
        _dptr(q), B, Hq, ctypes.byref(Kc.desc), ctypes.byref(Vc.desc), ctypes.byref(win.desc),
        _dptr(active), _dptr(acc), float(scale), _dptr(out), int(n_splits), _dptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))
    return out


def mustafar_window_step_grouped(win: DenseWindow, Kc: CompressedCache, Vc: CompressedCache,
                                 k_new, v_new, active=None, acc=None, stream=None) -> None:
    """One step of the grouped lifecycle: full windows first hand their oldest 32
    tokens to Kc (per token) and the per-channel cache Vc (one group, scored by acc
    [B][H][W] fp32, or by magnitude when acc is None)."""
    _check("mustafar_window_step_grouped", lib().mustafar_window_step_grouped(
        ctypes.byref(win.desc), ctypes.byref(Kc.desc), ctypes.byref(Vc.desc), _dptr(k_new),
        _dptr(v_new), _dptr(active), _dptr(acc), _stream(stream)))


ROUTE_DEFAULT, ROUTE_WALKS, ROUTE_MATRIX_CORES = 0, 1, 2


def mustafar_attn_set_route(route: int) -> None:
    """Kernel route of grouped-query sparse calls (ROUTE_DEFAULT, ROUTE_WALKS, ROUTE_MATRIX_CORES)."""
    _check("mustafar_attn_set_route", lib().mustafar_attn_set_route(int(route)))


def mustafar_attn_route() -> int:
    return lib().mustafar_attn_route()


def mustafar_stream_mix(src, dst, write_16ths: int, sink=None, stream=None):
    """Measurement helper: stream device tensor `src`, write write_16ths/16 of it to `dst`."""
    import torch
    need = src.numel() * src.element_size() * write_16ths // 16
    if dst.numel() * dst.element_size() < need:
        raise ValueError(f"dst holds {dst.numel() * dst.element_size()} bytes, {need} needed")
    if sink is None:
        sink = torch.empty(lib().mustafar_stream_read_sink_bytes(), dtype=torch.uint8, device=src.device)
    _check("mustafar_stream_mix", lib().mustafar_stream_mix(
        _dptr(src), src.numel() * src.element_size(), _dptr(dst), int(write_16ths), _dptr(sink),
        _stream(stream)))
    return sink


STREAM_CHUNK_BYTES = 16384  # MUSTAFAR_STREAM_CHUNK_BYTES


def mustafar_stream_chunks(src, n_streams: int, dst, write_16ths: int, sink=None, stream=None):
    """Measurement helper: the bulk compression's access order over device tensor
    `src` (n_streams streams of 16 KiB chunks), write_16ths/16 of every chunk to `dst`;
    returns the per-chunk checksums (uint32 as int32, workgroup order)."""
    import torch
    nbytes = src.numel() * src.element_size()
    if n_streams < 1 or nbytes % (n_streams * STREAM_CHUNK_BYTES) != 0:
        raise ValueError(f"{nbytes} bytes are not {n_streams} streams of whole {STREAM_CHUNK_BYTES}-byte chunks")
    n_chunks = nbytes // (n_streams * STREAM_CHUNK_BYTES)
    need = nbytes * write_16ths // 16
    if dst.numel() * dst.element_size() < need:
        raise ValueError(f"dst holds {dst.numel() * dst.element_size()} bytes, {need} needed")
    if sink is None:
        sink = torch.empty(n_streams * n_chunks, dtype=torch.int32, device=src.device)
    _check("mustafar_stream_chunks", lib().mustafar_stream_chunks(
        _dptr(src), int(n_streams), int(n_chunks), _dptr(dst), int(write_16ths), _dptr(sink), _stream(stream)))
    return sink


def mustafar_stream_read(buf, sink=None, stream=None):
    """Measurement helper: stream the bytes of device tensor `buf` through 16-byte loads."""
    import torch
    if sink is None:
        sink = torch.empty(lib().mustafar_stream_read_sink_bytes(), dtype=torch.uint8,
                           device=buf.device)
    _check("mustafar_stream_read", lib().mustafar_stream_read(
        _dptr(buf), buf.numel() * buf.element_size(), _dptr(sink), _stream(stream)))
    return sink
