"""Host-side checks of the C ABI (no GPU needed).

The library must load on a machine without a GPU, export every function that
include/mustafar.h declares, lay out mustafar_ccache_t as the C compiler does,
and reject every invalid call before anything is launched.
"""
import ctypes
import os
import re
import subprocess

import pytest

import oracle
import paper_2505_22913_amd as mf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mustafar.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(mf.LIB_PATH):
        from paper_2505_22913_amd import build_lib
        build_lib.build()
    return mf.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mustafar_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_expected_entry_points():
    names = declared_functions()
    for n in ("mustafar_prune_compress", "mustafar_append", "mustafar_sparse_decode_attn",
              "mustafar_dense_decode_attn", "mustafar_keep_count", "mustafar_strerror"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", mf.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT\s+(mustafar_\w+)", out))
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing
    for n in declared_functions():
        assert hasattr(lib, n)


def test_struct_layout_matches_the_c_compiler(tmp_path):
    prog = tmp_path / "layout.c"
    prog.write_text(
        '#include <stddef.h>\n#include <stdio.h>\n#include "mustafar.h"\n'
        "int main(void){printf(\"%zu %zu %zu %zu %zu %zu\\n\", sizeof(mustafar_ccache_t),"
        " offsetof(mustafar_ccache_t, B), offsetof(mustafar_ccache_t, n_keep),"
        " offsetof(mustafar_ccache_t, n_tokens), offsetof(mustafar_ccache_t, val_stride),"
        " offsetof(mustafar_ccache_t, group_keep));"
        "return 0;}\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", f"-I{os.path.dirname(HEADER)}", "-o", str(exe), str(prog)],
                   check=True)
    c_vals = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                             check=True).stdout.split()]
    T = mf.ccache_t
    assert c_vals == [ctypes.sizeof(T), T.B.offset, T.n_keep.offset, T.n_tokens.offset,
                      T.val_stride.offset, T.group_keep.offset]


def test_keep_count_agrees_with_the_oracle_reading(lib):
    for d in (64, 128, 256):
        for i in range(0, 1001):
            s = i / 1000.0
            assert mf.mustafar_keep_count(d, s) == oracle.keep_count(d, s), (d, s)
    for bad in (-0.01, 1.01, float("nan")):
        assert lib.mustafar_keep_count(128, bad) == mf.EINVAL
    assert lib.mustafar_keep_count(0, 0.5) == mf.EINVAL


def test_capacity_bounds(lib):
    assert mf.mustafar_token_max_elems(128, 64) == 72    # two tiles, each padded by < 8
    assert mf.mustafar_token_max_elems(128, 128) == 128  # full tiles need no padding
    assert mf.mustafar_token_max_elems(128, 0) == 0
    assert mf.mustafar_token_max_elems(128, 1) == 8
    assert mf.mustafar_token_max_elems(64, 38) == 40
    assert mf.mustafar_token_max_elems(256, 77) == 104
    assert mf.mustafar_token_max_elems(96, 10) == -1      # not a whole number of tiles
    assert mf.mustafar_stream_capacity(128, 38, 1000) == 1000 * 48


def _fake_cache(B=2, H=4, d=128, s=0.5, cap=100, stride=None):
    """Descriptor over fake (never dereferenced) aligned addresses."""
    c = mf.ccache_t()
    k = max(mf.lib().mustafar_keep_count(d, s), 0)
    if stride is None:
        stride = max(mf.mustafar_stream_capacity(d, k, cap), 8)
    st = mf.lib().mustafar_ccache_init(ctypes.byref(c), 0x100000, 0x200000, 0x300000, 0x400000,
                                       B, H, d, s, cap, stride)
    return c, st


def test_ccache_init_validates(lib):
    c, st = _fake_cache()
    assert st == mf.OK and c.n_keep == 64 and c.n_tokens == 0
    assert _fake_cache(d=96)[1] == mf.EINVAL
    assert _fake_cache(s=1.5)[1] == mf.EINVAL
    assert _fake_cache(cap=0)[1] == mf.EINVAL
    assert _fake_cache(stride=8)[1] == mf.EINVAL                    # below worst case
    assert _fake_cache(stride=100 * 72 + 4)[1] == mf.EINVAL         # not a multiple of 8
    c2 = mf.ccache_t()
    assert lib.mustafar_ccache_init(ctypes.byref(c2), 0x100001, 0x200000, 0x300000, 0x400000,
                                    1, 1, 128, 0.5, 10, 720) == mf.EINVAL  # misaligned bitmaps
    assert lib.mustafar_ccache_init(ctypes.byref(c2), 0, 0x200000, 0x300000, 0x400000,
                                    1, 1, 128, 0.5, 10, 720) == mf.EINVAL  # null


def test_compress_and_append_reject_before_launch(lib):
    c, _ = _fake_cache(B=2, H=4, cap=100)
    ws_need = lib.mustafar_compress_workspace_bytes(2, 4, 50)
    # a 16-byte status word, then per stream one 8-byte scan flag per 64-token chunk,
    # a 4-byte ticket counter and a 4-byte give-up mark
    assert ws_need == 16 + 2 * 4 * (1 * 8 + 4 + 4)
    assert lib.mustafar_compress_workspace_bytes(1, 1, 65) == 16 + 2 * 8 + 4 + 4
    # the bounded form checks the same arguments
    assert lib.mustafar_prune_compress_bounded(ctypes.byref(c), x := 0x500000, 50, 0, 0x600000,
                                               ws_need - 1, None) == mf.EWORKSPACE
    assert lib.mustafar_prune_compress_bounded(ctypes.byref(c), x, 0, 0, 0x600000, ws_need,
                                               None) == mf.EINVAL
    x = 0x500000
    assert lib.mustafar_prune_compress(ctypes.byref(c), x, 0, 0x600000, ws_need, None) == mf.EINVAL
    assert lib.mustafar_prune_compress(ctypes.byref(c), x + 2, 50, 0x600000, ws_need,
                                       None) == mf.EINVAL
    assert lib.mustafar_prune_compress(ctypes.byref(c), x, 101, 0x600000, 10 ** 6,
                                       None) == mf.ECAPACITY
    assert lib.mustafar_prune_compress(ctypes.byref(c), x, 50, 0x600000, ws_need - 1,
                                       None) == mf.EWORKSPACE
    assert lib.mustafar_prune_compress(ctypes.byref(c), x, 50, None, ws_need,
                                       None) == mf.EWORKSPACE
    assert lib.mustafar_prune_compress(ctypes.byref(c), x, 50, 0x600004, ws_need,
                                       None) == mf.EWORKSPACE                # not 8-byte aligned
    c.n_tokens = 100
    assert lib.mustafar_append(ctypes.byref(c), x, None) == mf.ECAPACITY
    assert lib.mustafar_prune_compress(ctypes.byref(c), x, 1, 0x600000, 10 ** 6,
                                       None) == mf.ECAPACITY
    c.n_tokens = 101
    assert lib.mustafar_append(ctypes.byref(c), x, None) == mf.EINVAL   # corrupt descriptor
    assert c.n_tokens == 101                                             # nothing changed


def test_append_kv_rejects_before_launch(lib):
    K, _ = _fake_cache(B=2, H=4, cap=10)
    V, _ = _fake_cache(B=2, H=4, s=0.7, cap=10)
    kn, vn = 0xf00000, 0xf10000
    call = lambda **kw: lib.mustafar_append_kv(  # noqa: E731
        ctypes.byref(kw.get("K", K)), ctypes.byref(kw.get("V", V)), kw.get("kn", kn), kw.get("vn", vn), None)
    assert call(kn=kn + 2) == mf.EINVAL
    assert call(vn=None) == mf.EINVAL
    assert call(V=K) == mf.EINVAL                    # the same cache twice
    V3, _ = _fake_cache(B=2, H=3, s=0.7, cap=10)
    assert call(V=V3) == mf.EINVAL                   # shapes differ
    Vg, _ = _fake_grouped(B=2, H=4, cap=64)
    assert call(V=Vg) == mf.EINVAL                   # per-channel groups take no single token
    V.n_tokens = 1
    assert call() == mf.EINVAL                       # token counts differ
    K.n_tokens = V.n_tokens = 10
    assert call() == mf.ECAPACITY
    assert K.n_tokens == 10 and V.n_tokens == 10


def test_decode_attention_rejects_before_launch(lib):
    K, _ = _fake_cache(B=2, H=4)
    V, _ = _fake_cache(B=2, H=4, s=0.7)
    K.n_tokens = V.n_tokens = 50
    q, out, kt, vt = 0x700000, 0x800000, 0x900000, 0xa00000
    need = lib.mustafar_attn_workspace_bytes(2, 16, 4, 128, 50, 0)
    assert need > 0
    call = lambda **kw: lib.mustafar_sparse_decode_attn(  # noqa: E731
        kw.get("q", q), kw.get("B", 2), kw.get("Hq", 16), ctypes.byref(kw.get("K", K)),
        ctypes.byref(kw.get("V", V)), kw.get("kt", kt), kw.get("vt", vt), kw.get("n_tail", 32),
        0.0, kw.get("out", out), kw.get("splits", 0), kw.get("ws", 0xb00000),
        kw.get("ws_bytes", need), None)
    assert call(Hq=12) == mf.EUNSUPPORTED       # group size 3
    assert call(Hq=10) == mf.EINVAL             # not a multiple of Hkv
    assert call(B=3) == mf.EINVAL               # batch mismatch with the caches
    assert call(q=q + 8) == mf.EINVAL           # misaligned q
    assert call(out=None) == mf.EINVAL
    assert call(kt=None) == mf.EINVAL           # window tokens but no window
    assert call(n_tail=-1) == mf.EINVAL
    assert call(ws_bytes=need - 4) == mf.EWORKSPACE
    assert call(ws=None) == mf.EWORKSPACE
    V2, _ = _fake_cache(B=2, H=4, s=0.7)
    V2.n_tokens = 49
    assert call(V=V2) == mf.EINVAL              # K and V token counts differ
    K0, _ = _fake_cache(B=2, H=4)
    V0, _ = _fake_cache(B=2, H=4)
    assert call(K=K0, V=V0, n_tail=0, kt=None, vt=None) == mf.EINVAL   # no tokens at all
    dense = lambda **kw: lib.mustafar_dense_decode_attn(  # noqa: E731
        q, 2, kw.get("Hq", 16), 4, kw.get("k", kt), vt, kw.get("n", 50), kw.get("d", 128), 0.0,
        out, 0, 0xb00000, kw.get("ws_bytes", need), None)
    assert dense(n=0) == mf.EINVAL
    assert dense(d=100) == mf.EINVAL
    assert dense(Hq=24) == mf.EUNSUPPORTED
    assert dense(k=kt + 4) == mf.EINVAL
    assert dense(ws_bytes=16) == mf.EWORKSPACE


def test_default_splits_follow_the_kernel(lib):
    S, D = mf.ATTN_SPARSE, mf.ATTN_DENSE
    ds = lib.mustafar_attn_default_splits
    # one query head per kv-head: ~32768 workgroups, segments down to one 64-token block
    assert ds(16, 32, 32, 32768, S) == 64
    assert ds(1, 32, 32, 4096, S) == 64
    assert ds(1, 8, 8, 1024, S) == 16
    assert ds(1, 8, 8, 1024, D) == 16
    # 2 or 4 query heads per kv-head (the walks): ~4096 workgroups of at least 192 tokens;
    # 8 (the matrix-core kernel): ~2048 of at least 128; dense with grouped queries: ~4096
    assert ds(1, 32, 8, 131072, S) == 512
    assert ds(1, 32, 8, 131072, D) == 512
    assert ds(4, 32, 8, 16384, S) == 86    # 16384 / 192, rounded up
    assert ds(4, 16, 8, 16384, S) == 86
    assert ds(4, 64, 8, 16384, S) == 64
    assert ds(4, 32, 8, 16384, D) == 128
    assert ds(1, 32, 8, 300, S) == 2       # 300 / 192, rounded up
    # invalid arguments
    assert ds(1, 32, 8, 4096, 2) == 1
    assert ds(0, 32, 8, 4096, S) == 1
    assert ds(1, 4, 8, 4096, S) == 1
    assert ds(1, 32, 8, 0, S) == 1
    # the default workspace covers both kinds' default split counts
    for B, Hq, Hkv, n in ((1, 32, 8, 131072), (2, 16, 16, 5000), (3, 8, 2, 700)):
        want = max(lib.mustafar_attn_workspace_bytes(B, Hq, Hkv, 128, n, ds(B, Hq, Hkv, n, k))
                   for k in (S, D))
        assert lib.mustafar_attn_workspace_bytes(B, Hq, Hkv, 128, n, 0) == want


def test_strerror_covers_every_status(lib):
    for code in (mf.OK, mf.EINVAL, mf.ECAPACITY, mf.EWORKSPACE, mf.ELAUNCH, mf.EUNSUPPORTED):
        assert mf.strerror(code) not in ("", "unknown status")
    assert mf.strerror(-99) == "unknown status"


def test_stream_read_helper_rejects_bad_arguments(lib):
    assert lib.mustafar_stream_read_sink_bytes() > 0
    assert lib.mustafar_stream_read(0x100008, 64, 0x200000, None) == mf.EINVAL   # src not 16-aligned
    assert lib.mustafar_stream_read(0x100000, 24, 0x200000, None) == mf.EINVAL   # bytes % 16
    assert lib.mustafar_stream_read(None, 64, 0x200000, None) == mf.EINVAL
    assert lib.mustafar_stream_read(0x100000, 64, None, None) == mf.EINVAL


def _fake_window(B=2, H=4, d=128, W=32, max_len=0):
    w = mf.window_t()
    st = mf.lib().mustafar_window_init(ctypes.byref(w), 0xc00000, 0xd00000, 0xe00000, 0xe10000,
                                       0xe20000, B, H, d, W, max_len)
    return w, st


def test_window_struct_layout_matches_the_c_compiler(tmp_path):
    prog = tmp_path / "wlayout.c"
    prog.write_text(
        '#include <stddef.h>\n#include <stdio.h>\n#include "mustafar.h"\n'
        "int main(void){printf(\"%zu %zu %zu %zu\\n\", sizeof(mustafar_window_t),"
        " offsetof(mustafar_window_t, n_comp), offsetof(mustafar_window_t, B),"
        " offsetof(mustafar_window_t, max_len));return 0;}\n")
    exe = tmp_path / "wlayout"
    subprocess.run(["gcc", "-std=c11", f"-I{os.path.dirname(HEADER)}", "-o", str(exe), str(prog)],
                   check=True)
    c_vals = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                             check=True).stdout.split()]
    T = mf.window_t
    assert c_vals == [ctypes.sizeof(T), T.n_comp.offset, T.B.offset, T.max_len.offset]


def test_window_calls_reject_before_launch(lib):
    w, st = _fake_window()
    assert st == mf.OK and w.W == 32 and w.max_len == 0
    assert _fake_window(W=0)[1] == mf.EINVAL
    assert _fake_window(W=1025)[1] == mf.EINVAL
    assert _fake_window(max_len=33)[1] == mf.EINVAL
    assert _fake_window(d=96)[1] == mf.EINVAL
    w2 = mf.window_t()
    assert lib.mustafar_window_init(ctypes.byref(w2), 0xc00008, 0xd00000, 0xe00000, 0xe10000,
                                    0xe20000, 2, 4, 128, 32, 0) == mf.EINVAL  # ring not 16-aligned
    K, _ = _fake_cache(B=2, H=4, cap=10)
    V, _ = _fake_cache(B=2, H=4, s=0.7, cap=10)
    kn, vn, act = 0xf00000, 0xf10000, 0xf20000
    step = lambda **kw: lib.mustafar_window_step(  # noqa: E731
        ctypes.byref(kw.get("w", w)), ctypes.byref(kw.get("K", K)), ctypes.byref(kw.get("V", V)),
        kw.get("kn", kn), vn, kw.get("act", act), None)
    assert step(kn=kn + 2) == mf.EINVAL
    assert step(act=act + 2) == mf.EINVAL
    K3, _ = _fake_cache(B=3, H=4, cap=10)
    assert step(K=K3) == mf.EINVAL                   # batch differs from the window
    # A full window graduates a token: no room left in the caches.
    wf, _ = _fake_window(max_len=32)
    K.n_tokens = V.n_tokens = 10
    assert step(w=wf) == mf.ECAPACITY
    assert K.n_tokens == 10 and wf.max_len == 32     # nothing changed
    # Prefill: host lengths are validated before anything runs.
    K0, _ = _fake_cache(B=2, H=4, cap=10)
    V0, _ = _fake_cache(B=2, H=4, s=0.7, cap=10)
    lens = (ctypes.c_int32 * 2)(5, 50)
    need = lib.mustafar_compress_workspace_bytes(1, 4, 50)
    pre = lambda **kw: lib.mustafar_window_prefill(  # noqa: E731
        ctypes.byref(w), ctypes.byref(kw.get("K", K0)), ctypes.byref(V0), 0x1000000, 0x2000000,
        kw.get("n_max", 50), kw.get("lens", lens), 0x3000000, kw.get("ws_bytes", need), None)
    assert pre(n_max=49) == mf.EINVAL                # a length beyond n_max
    assert pre() == mf.ECAPACITY                     # 50 - 32 = 18 compressed > cap 10
    lens2 = (ctypes.c_int32 * 2)(5, 40)
    assert pre(lens=lens2, ws_bytes=need - 8) == mf.EWORKSPACE
    K0.n_tokens = 1
    assert pre(lens=lens2) == mf.EINVAL              # caches must start empty
    # Attention over the window: shapes checked against the window.
    K.n_tokens = V.n_tokens = 5
    anb = lib.mustafar_attn_workspace_bytes(2, 8, 4, 128, 5, 0)
    att = lambda **kw: lib.mustafar_window_decode_attn(  # noqa: E731
        0x700000, kw.get("B", 2), kw.get("Hq", 8), ctypes.byref(K), ctypes.byref(V),
        ctypes.byref(w), 0.0, 0x800000, 0, 0xb00000, kw.get("ws_bytes", anb), None)
    assert att(B=3) == mf.EINVAL
    assert att(Hq=12) == mf.EUNSUPPORTED
    assert att(ws_bytes=anb - 4) == mf.EWORKSPACE
    # Output-aware keys in the window.
    kacc = 0x4000000
    wstep = lambda **kw: lib.mustafar_window_step_weighted(  # noqa: E731
        ctypes.byref(kw.get("w", w)), ctypes.byref(K), ctypes.byref(V), kn, vn, act,
        kw.get("kacc", kacc), None)
    assert wstep(kacc=kacc + 8) == mf.EINVAL         # misaligned weights
    assert wstep(kacc=None) == mf.EINVAL
    w16, _ = _fake_window(W=16)
    assert wstep(w=w16) == mf.EINVAL                 # a key must see 32 steps in the window
    kw_ = lambda **kw: lib.mustafar_window_key_weights(  # noqa: E731
        kw.get("q", 0x700000), kw.get("B", 2), kw.get("Hq", 8), ctypes.byref(w), kw.get("act", None),
        kw.get("kacc", kacc), None)
    assert kw_(B=3) == mf.EINVAL
    assert kw_(act=0x900002) == mf.EINVAL            # misaligned activity mask
    assert kw_(Hq=6) == mf.EINVAL                    # not a multiple of H
    assert kw_(Hq=64) == mf.EUNSUPPORTED             # 16 query heads per kv-head
    assert kw_(q=0x700002) == mf.EINVAL
    assert kw_(kacc=kacc + 4) == mf.EINVAL


def test_prune_variants_reject_before_launch(lib):
    c, _ = _fake_cache(B=2, H=4, cap=100, s=0.5)
    x, ws = 0x500000, 0x600000
    need = lib.mustafar_compress_workspace_bytes(2, 4, 50)
    o = mf.prune_opts_t()
    call = lambda opts, **kw: lib.mustafar_prune_compress_ex(  # noqa: E731
        ctypes.byref(kw.get("c", c)), x, kw.get("n", 50), ctypes.byref(opts), ws, need, None)
    o.mode = 7
    assert call(o) == mf.EINVAL                       # unknown mode
    o.mode = mf.PRUNE_OUTPUT_AWARE
    assert call(o) == mf.EINVAL                       # output-aware without weights
    o.mode = mf.PRUNE_2_4
    c7, _ = _fake_cache(B=2, H=4, cap=100, s=0.7)
    assert call(o, c=c7) == mf.EINVAL                 # 2:4 needs n_keep = d/2
    hk = (ctypes.c_int32 * 4)(64, 64, 65, 1)
    o.mode = mf.PRUNE_MAGNITUDE
    o.head_keep = ctypes.cast(hk, ctypes.c_void_p)
    assert call(o) == mf.EINVAL                       # a head above the cache's n_keep
    o2 = mf.prune_opts_t()
    o2.mode = mf.PRUNE_2_4
    o2.head_keep = ctypes.cast(hk, ctypes.c_void_p)
    assert call(o2) == mf.EINVAL                      # 2:4 takes no per-head counts
    assert lib.mustafar_query_lookahead(0x700000, 1, 6, 4, 10, 128, 32, 0x800000, None) == mf.EINVAL
    assert lib.mustafar_query_lookahead(0x700000, 1, 8, 4, 10, 128, 0, 0x800000, None) == mf.EINVAL
    assert lib.mustafar_query_lookahead(0x700008, 1, 8, 4, 10, 128, 32, 0x800000, None) == mf.EINVAL


def _fake_grouped(B=2, H=4, d=128, s=0.7, cap=96, stride=None):
    c = mf.ccache_t()
    gk = mf.lib().mustafar_keep_count(32, s)
    if stride is None:
        stride = max(mf.lib().mustafar_grouped_stream_capacity(d, max(gk, 0), cap), 8)
    st = mf.lib().mustafar_ccache_init_grouped(ctypes.byref(c), 0x100000, 0x200000, 0x300000,
                                               0x400000, B, H, d, s, cap, stride)
    return c, st


def test_grouped_cache_init_and_capacity(lib):
    import oracle
    c, st = _fake_grouped()
    assert st == mf.OK and c.group_keep == 10 and c.n_keep == 128
    per, _ = _fake_cache()
    assert per.group_keep == -1
    # the bound matches the oracle's worst case per group
    for d, gk, cap in ((64, 16, 64), (128, 10, 96), (256, 3, 32), (128, 0, 33)):
        assert lib.mustafar_grouped_stream_capacity(d, gk, cap) == \
            oracle.grouped_stream_capacity(d, gk, (cap + 31) // 32 * 32)
    assert lib.mustafar_grouped_stream_capacity(96, 10, 32) == -1
    assert lib.mustafar_grouped_stream_capacity(128, 33, 32) == -1
    stride = lib.mustafar_grouped_stream_capacity(128, 10, 96)
    assert _fake_grouped(stride=stride - 8)[1] == mf.EINVAL     # too small for the groups
    assert _fake_grouped(s=1.5)[1] == mf.EINVAL


def test_grouped_calls_reject_before_launch(lib):
    c, _ = _fake_grouped(cap=96)
    x, ws = 0x500000, 0x600000
    need = lib.mustafar_compress_workspace_bytes(2, 4, 64)
    comp = lambda n=64, **kw: lib.mustafar_prune_compress(  # noqa: E731
        ctypes.byref(kw.get("c", c)), x, n, ws, need, None)
    assert comp(n=40) == mf.EINVAL                    # not whole groups
    assert comp(n=128) == mf.ECAPACITY
    assert lib.mustafar_append(ctypes.byref(c), x, None) == mf.EINVAL   # groups are whole
    o = mf.prune_opts_t()
    ex = lambda opts, **kw: lib.mustafar_prune_compress_ex(  # noqa: E731
        ctypes.byref(kw.get("c", c)), x, kw.get("n", 64), ctypes.byref(opts), ws, need, None)
    o.mode = mf.PRUNE_MAGNITUDE
    assert ex(o) == mf.EINVAL                         # per-token mode on a per-channel cache
    o.mode = mf.PRUNE_CHANNEL_OUTPUT_AWARE
    assert ex(o) == mf.EINVAL                         # no token weights
    o.weights = 0x700002
    assert ex(o) == mf.EINVAL                         # misaligned weights
    per, _ = _fake_cache(cap=96)
    o.mode = mf.PRUNE_CHANNEL
    o.weights = None
    assert ex(o, c=per) == mf.EINVAL                  # channel mode on a per-token cache
    assert ex(o, n=33) == mf.EINVAL
    assert c.n_tokens == 0
    # Grouped window lifecycle.
    w, _ = _fake_window(W=64)
    K, _ = _fake_cache(B=2, H=4, cap=64)
    V, _ = _fake_grouped(B=2, H=4, cap=64)
    kn, vn, acc = 0xf00000, 0xf10000, 0xf30000
    step = lambda **kw: lib.mustafar_window_step_grouped(  # noqa: E731
        ctypes.byref(kw.get("w", w)), ctypes.byref(kw.get("K", K)), ctypes.byref(kw.get("V", V)),
        kn, vn, None, kw.get("acc", acc), None)
    assert step(V=per) == mf.EINVAL                   # values must be a per-channel cache
    assert step(K=V) == mf.EINVAL                     # keys per token
    w32, _ = _fake_window(W=32)
    assert step(w=w32) == mf.EINVAL                   # at least two groups of slots
    assert step(acc=acc + 2) == mf.EINVAL
    wf, _ = _fake_window(W=64, max_len=64)
    K.n_tokens = V.n_tokens = 64
    assert step(w=wf) == mf.ECAPACITY                 # no room for a group
    assert K.n_tokens == 64 and wf.max_len == 64
    # the per-token step refuses per-channel caches
    assert lib.mustafar_window_step(ctypes.byref(w), ctypes.byref(K), ctypes.byref(V), kn, vn,
                                    None, None) == mf.EINVAL
    # scores: workspace includes the log-sum-exp rows
    K.n_tokens = V.n_tokens = 32
    anb = lib.mustafar_attn_workspace_bytes(2, 8, 4, 128, 32, 0)
    att = lambda **kw: lib.mustafar_window_decode_attn_scores(  # noqa: E731
        0x700000, 2, 8, ctypes.byref(K), ctypes.byref(V), ctypes.byref(w), kw.get("act", None),
        kw.get("acc", acc), 0.0, 0x800000, 0, 0xb00000, kw.get("ws_bytes", anb), None)
    assert att(ws_bytes=anb - 4) == mf.EWORKSPACE
    assert att(act=0x900001) == mf.EINVAL            # misaligned activity mask
    assert att(acc=acc + 1) == mf.EINVAL


def test_static_scratch_decode_rejects_before_touching_the_gpu(lib):
    """mustafar_sparse_decode_attn_static checks every argument, and that the call's
    partials fit the static buffer, before its first HIP call."""
    K, _ = _fake_cache(B=2, H=4, cap=100)
    V, _ = _fake_cache(B=2, H=4, cap=100, s=0.7)
    K.n_tokens = V.n_tokens = 100
    call = lambda **kw: lib.mustafar_sparse_decode_attn_static(  # noqa: E731
        0x700000, kw.get("B", 2), kw.get("Hq", 16), ctypes.byref(K), ctypes.byref(kw.get("V", V)),
        kw.get("kt", 0x900000), 0x980000, kw.get("nt", 32), 0.0, 0x800000, kw.get("splits", 0), None)
    assert call(B=3) == mf.EINVAL
    assert call(Hq=12) == mf.EUNSUPPORTED                    # three query heads per kv-head
    assert call(Hq=6) == mf.EINVAL                           # not a multiple of the kv-heads
    assert call(kt=0x900002) == mf.EINVAL                    # misaligned window
    assert call(nt=-1) == mf.EINVAL
    V.n_tokens = 99
    assert call() == mf.EINVAL                               # K and V differ in length
    V.n_tokens = 100
    need = lib.mustafar_attn_workspace_bytes(2, 16, 4, 128, 100, 1 << 16)
    assert need > mf.STATIC_SCRATCH_BYTES
    assert call(splits=1 << 16) == mf.ESCRATCH
    assert "static scratch" in mf.strerror(mf.ESCRATCH)


def test_stream_chunks_helper_rejects_bad_arguments(lib):
    S = 0x300000
    assert lib.mustafar_stream_chunks(0x100008, 2, 3, 0x200000, 9, S, None) == mf.EINVAL   # src not 16-aligned
    assert lib.mustafar_stream_chunks(0x100000, 2, 3, 0x200008, 9, S, None) == mf.EINVAL   # dst not 16-aligned
    assert lib.mustafar_stream_chunks(0x100000, 2, 3, 0x200000, 9, S + 2, None) == mf.EINVAL
    assert lib.mustafar_stream_chunks(0x100000, 0, 3, 0x200000, 9, S, None) == mf.EINVAL
    assert lib.mustafar_stream_chunks(0x100000, 2, 0, 0x200000, 9, S, None) == mf.EINVAL
    assert lib.mustafar_stream_chunks(0x100000, 1 << 16, 1 << 15, 0x200000, 9, S, None) == mf.EINVAL
    assert lib.mustafar_stream_chunks(0x100000, 2, 3, 0x200000, 17, S, None) == mf.EINVAL
    assert lib.mustafar_stream_chunks(0x100000, 2, 3, 0x200000, -1, S, None) == mf.EINVAL
    assert lib.mustafar_stream_chunks(None, 2, 3, 0x200000, 9, S, None) == mf.EINVAL
    assert lib.mustafar_stream_chunks(0x100000, 2, 3, None, 9, S, None) == mf.EINVAL
    assert lib.mustafar_stream_chunks(0x100000, 2, 3, 0x200000, 9, None, None) == mf.EINVAL


def test_stream_mix_helper_rejects_bad_arguments(lib):
    S = 0x300000
    assert lib.mustafar_stream_mix(0x100008, 256, 0x200000, 9, S, None) == mf.EINVAL   # src not 16-aligned
    assert lib.mustafar_stream_mix(0x100000, 256, 0x200008, 9, S, None) == mf.EINVAL   # dst not 16-aligned
    assert lib.mustafar_stream_mix(0x100000, 240, 0x200000, 9, S, None) == mf.EINVAL   # bytes % 256
    assert lib.mustafar_stream_mix(0x100000, 256, 0x200000, 17, S, None) == mf.EINVAL
    assert lib.mustafar_stream_mix(0x100000, 256, 0x200000, -1, S, None) == mf.EINVAL
    assert lib.mustafar_stream_mix(None, 256, 0x200000, 9, S, None) == mf.EINVAL
    assert lib.mustafar_stream_mix(0x100000, 256, 0x200000, 9, None, None) == mf.EINVAL
    assert lib.mustafar_stream_mix(0x100000, 256, 0x200000, 9, S + 2, None) == mf.EINVAL


def test_attn_route_setting(lib):
    # The route is host state: unknown routes are rejected, the setting sticks
    # and steers the default split count to the chosen kernel's.
    assert lib.mustafar_attn_set_route(3) == mf.EINVAL
    assert lib.mustafar_attn_set_route(-1) == mf.EINVAL
    try:
        assert lib.mustafar_attn_set_route(mf.ROUTE_WALKS) == 0
        assert lib.mustafar_attn_route() == mf.ROUTE_WALKS
        walks = lib.mustafar_attn_default_splits(1, 64, 8, 131072, 0)   # 8 streams, G = 8
        assert lib.mustafar_attn_set_route(mf.ROUTE_MATRIX_CORES) == 0
        cores = lib.mustafar_attn_default_splits(1, 64, 8, 131072, 0)
        cores_g2 = lib.mustafar_attn_default_splits(1, 16, 8, 131072, 0)
    finally:
        assert lib.mustafar_attn_set_route(mf.ROUTE_DEFAULT) == 0
    assert (walks, cores) == (512, 256)   # 4096 and 2048 workgroups over 8 streams
    assert lib.mustafar_attn_default_splits(1, 64, 8, 131072, 0) == cores   # default: cores at G = 8
    assert lib.mustafar_attn_default_splits(1, 16, 8, 131072, 0) == walks   # default: walks at G = 2
    assert cores_g2 == cores
