"""Helpers shared by the GPU parity tests: device upload, read-back of a
compressed cache, the attention error metric, and case announcements that
reach the log even if a GPU failure ends the process."""
from __future__ import annotations

import os
import sys

import numpy as np

# Attention tolerance: per output vector, max_c |o_gpu - o_ref| / max_c |o_ref|.
ATTN_TOL = 2e-3


def announce(msg: str) -> None:
    """Names the case (and, after it, what it measured) on stderr and, when
    MUSTAFAR_CASE_LOG names a file, appended there: pytest's capture holds back
    a passing test's stderr, and a process that a GPU failure ends loses it."""
    line = f"[gpu-case] {msg}\n"
    sys.__stderr__.write(line)
    sys.__stderr__.flush()
    path = os.environ.get("MUSTAFAR_CASE_LOG")
    if path:
        fd = os.open(path, os.O_WRONLY | os.O_APPEND | os.O_CREAT, 0o644)
        try:
            os.write(fd, line.encode())
            os.fsync(fd)
        finally:
            os.close(fd)


def have_lib() -> bool:
    import paper_2505_22913_amd as mf
    return os.path.exists(mf.LIB_PATH)


def to_dev(x: np.ndarray):
    import torch
    if x.dtype == np.float16:
        return torch.from_numpy(np.ascontiguousarray(x)).cuda()
    raise TypeError(x.dtype)


def read_cache(cache) -> dict:
    """Bit patterns of a CompressedCache as numpy arrays (oracle dtypes)."""
    import torch
    torch.cuda.synchronize()
    return {
        "bitmaps": cache.bitmaps.cpu().numpy().view(np.uint64),
        "offsets": cache.offsets.cpu().numpy().view(np.uint32),
        "values": cache.values.cpu().numpy().view(np.uint16),
        "stream_len": cache.stream_len.cpu().numpy().view(np.uint32),
    }


def compare_format(got: dict, want: dict, n_tokens: int, pairs) -> None:
    """pairs: iterable of ((b_gpu, h_gpu), (b_ref, h_ref)) stream index pairs."""
    for (bg, hg), (br, hr) in pairs:
        gb = got["bitmaps"][bg, hg, :n_tokens]
        wb = want["bitmaps"][br, hr, :n_tokens]
        if not np.array_equal(gb, wb):
            bad = np.argwhere(gb != wb)[0]
            raise AssertionError(f"bitmaps differ at stream {(bg, hg)} token/tile {tuple(bad)}: "
                                 f"{int(gb[tuple(bad)]):#x} vs {int(wb[tuple(bad)]):#x}")
        go = got["offsets"][bg, hg, :n_tokens]
        wo = want["offsets"][br, hr, :n_tokens]
        assert np.array_equal(go, wo), f"offsets differ at stream {(bg, hg)}"
        gl, wl = int(got["stream_len"][bg, hg]), int(want["stream_len"][br, hr])
        assert gl == wl, f"stream_len {gl} vs {wl} at stream {(bg, hg)}"
        gv = got["values"][bg, hg, :gl]
        wv = want["values"][br, hr, :wl]
        if not np.array_equal(gv, wv):
            bad = int(np.argwhere(gv != wv)[0][0])
            raise AssertionError(f"values differ at stream {(bg, hg)} element {bad}: "
                                 f"{int(gv[bad]):#06x} vs {int(wv[bad]):#06x}")


def all_pairs(B: int, H: int):
    return [((b, h), (b, h)) for b in range(B) for h in range(H)]


def attn_error(got: np.ndarray, ref: np.ndarray) -> float:
    """max over output vectors of max|got - ref| / max|ref| (last axis = channels)."""
    got = got.astype(np.float64)
    num = np.abs(got - ref).max(axis=-1)
    den = np.maximum(np.abs(ref).max(axis=-1), 1e-6)
    return float((num / den).max())
