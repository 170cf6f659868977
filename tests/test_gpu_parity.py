"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Compression: bitmaps, offsets, stream lengths and packed values (padding
included) must equal the oracle bit for bit. Attention: per output vector,
max|o_gpu - o_ref| / max|o_ref| <= 2e-3 (fp16 in/out, fp32 accumulation on
the GPU, float64 in the oracle); the fp16 rounding of the output alone is
below 2.5e-4 of max|o|.
"""
import numpy as np
import pytest

import oracle
import paper_2505_22913_amd as mf
from paper_2505_22913_amd import synth
from tests.gpu_common import (ATTN_TOL, all_pairs, announce, attn_error, compare_format,
                              read_cache, to_dev)

pytestmark = pytest.mark.gpu


def _compress_gpu(x: np.ndarray, s: float, cap=None):
    B, H, N, d = x.shape
    cache = mf.CompressedCache(B, H, d, s, cap or N)
    mf.mustafar_prune_compress(cache, to_dev(x))
    return cache


def _tie_heavy(B, H, N, d, seed):
    rng = np.random.default_rng(seed)
    mags = np.array([0.0, 2.0 ** -24, 2.0 ** -20, 0.5, 1.0, 1.0, 1.0, 2.0], dtype=np.float32)
    x = rng.choice(mags, size=(B, H, N, d)) * rng.choice([-1.0, 1.0], size=(B, H, N, d))
    return x.astype(np.float16)


# ---------------------------------------------------------------------------------------------
# compression
# ---------------------------------------------------------------------------------------------
@pytest.mark.parametrize("s", [0.0, 0.3, 0.5, 0.7, 0.8, 0.9, 1.0])
@pytest.mark.parametrize("N", [1, 63, 64, 65, 257, 1000])
def test_compress_bit_exact_d128(N, s):
    announce(f"compress d=128 N={N} s={s}")
    K, V = synth.make_kv(2, 3, N, 128, seed=100 + N)
    for x in (K, V):
        got = read_cache(_compress_gpu(x, s))
        compare_format(got, oracle.compress(x, s), N, all_pairs(2, 3))


@pytest.mark.parametrize("d", [64, 256])
@pytest.mark.parametrize("s", [0.0, 0.5, 0.7, 0.9, 1.0])
def test_compress_bit_exact_other_head_dims(d, s):
    announce(f"compress d={d} s={s}")
    N = 300
    K, V = synth.make_kv(1, 4, N, d, seed=200 + d)
    for x in (K, V):
        got = read_cache(_compress_gpu(x, s))
        compare_format(got, oracle.compress(x, s), N, all_pairs(1, 4))


@pytest.mark.parametrize("d", [64, 128, 256])
@pytest.mark.parametrize("s", [0.25, 0.5, 0.7, 0.95])
def test_compress_ties_zeros_and_subnormals(d, s):
    announce(f"compress ties d={d} s={s}")
    x = _tie_heavy(2, 2, 130, d, seed=d)
    x[0, 0, 0] = np.float16(1.0)             # a token of all-equal magnitudes
    x[0, 0, 1] = np.float16(-1.0)
    x[0, 0, 2] = np.float16(0.0)             # all zeros: ties everywhere at +0
    x[0, 0, 3, ::2] = np.float16(-0.0)       # -0 and +0 compare equal
    got = read_cache(_compress_gpu(x, s))
    compare_format(got, oracle.compress(x, s), 130, all_pairs(2, 2))


@pytest.mark.parametrize("d", [64, 128, 256])
def test_compress_many_chunks_shared_workspace(d):
    # Tens of chunks per stream (long look-back chains) and one workspace reused
    # by consecutive calls: the call must clear its scan flags itself.
    import torch
    announce(f"compress many chunks d={d}")
    B, H, N = 2, 3, 5000
    K, V = synth.make_kv(B, H, N, d, seed=300 + d)
    ws = torch.empty(mf.mustafar_compress_workspace_bytes(B, H, N), dtype=torch.uint8,
                     device="cuda")
    for x, s in ((K, 0.5), (V, 0.7), (K, 0.0), (V, 1.0)):
        cache = mf.CompressedCache(B, H, d, s, N)
        mf.mustafar_prune_compress(cache, to_dev(x), ws=ws)
        compare_format(read_cache(cache), oracle.compress(x, s), N, all_pairs(B, H))


def test_compress_in_pieces_and_append_equal_compress_all():
    announce("compress pieces + append")
    B, H, d = 2, 4, 128
    n0, n1, n2 = 300, 100, 57
    K, _ = synth.make_kv(B, H, n0 + n1 + n2, d, seed=7)
    for s in (0.5, 0.7):
        cache = mf.CompressedCache(B, H, d, s, n0 + n1 + n2)
        mf.mustafar_prune_compress(cache, to_dev(np.ascontiguousarray(K[:, :, :n0])))
        mf.mustafar_prune_compress(cache, to_dev(np.ascontiguousarray(K[:, :, n0:n0 + n1])))
        for j in range(n0 + n1, n0 + n1 + n2):
            mf.mustafar_append(cache, to_dev(np.ascontiguousarray(K[:, :, j])))
        assert cache.n_tokens == n0 + n1 + n2
        compare_format(read_cache(cache), oracle.compress(K, s), n0 + n1 + n2, all_pairs(B, H))


def test_append_kv_equals_the_oracle():
    announce("append_kv")
    B, H, d, n0, n1 = 2, 3, 128, 70, 9
    K, V = synth.make_kv(B, H, n0 + n1, d, seed=12)
    Kc = mf.CompressedCache(B, H, d, 0.5, n0 + n1)
    Vc = mf.CompressedCache(B, H, d, 0.7, n0 + n1)
    mf.mustafar_prune_compress(Kc, to_dev(np.ascontiguousarray(K[:, :, :n0])))
    mf.mustafar_prune_compress(Vc, to_dev(np.ascontiguousarray(V[:, :, :n0])))
    for j in range(n0, n0 + n1):
        mf.mustafar_append_kv(Kc, Vc, to_dev(np.ascontiguousarray(K[:, :, j])),
                              to_dev(np.ascontiguousarray(V[:, :, j])))
    assert Kc.n_tokens == Vc.n_tokens == n0 + n1
    compare_format(read_cache(Kc), oracle.compress(K, 0.5), n0 + n1, all_pairs(B, H))
    compare_format(read_cache(Vc), oracle.compress(V, 0.7), n0 + n1, all_pairs(B, H))


def test_append_into_empty_cache_and_capacity_error():
    announce("append empty + capacity")
    B, H, d = 1, 2, 64
    K, _ = synth.make_kv(B, H, 3, d, seed=8)
    cache = mf.CompressedCache(B, H, d, 0.5, 3, align=1)
    for j in range(3):
        mf.mustafar_append(cache, to_dev(np.ascontiguousarray(K[:, :, j])))
    compare_format(read_cache(cache), oracle.compress(K, 0.5), 3, all_pairs(B, H))
    with pytest.raises(mf.MustafarError) as e:
        mf.mustafar_append(cache, to_dev(np.ascontiguousarray(K[:, :, 0])))
    assert e.value.status == mf.ECAPACITY


# ---------------------------------------------------------------------------------------------
# decode attention
# ---------------------------------------------------------------------------------------------
def _attn_case(B, Hkv, G, Ns, Nd, d, sK, sV, splits, seed, scale=0.0):
    announce(f"attn B={B} Hkv={Hkv} G={G} Ns={Ns} Nd={Nd} d={d} s=({sK},{sV}) splits={splits}")
    K, V = synth.make_kv(B, Hkv, Ns, d, seed=seed)
    KL, VL = synth.make_tail(B, Hkv, Nd, d, seed=seed)
    q = synth.make_q(B, Hkv * G, d, seed=seed)
    cap = max(Ns, 1)
    Kc = mf.CompressedCache(B, Hkv, d, sK, cap)
    Vc = mf.CompressedCache(B, Hkv, d, sV, cap)
    if Ns > 0:
        mf.mustafar_prune_compress(Kc, to_dev(K))
        mf.mustafar_prune_compress(Vc, to_dev(V))
    kt = to_dev(KL) if Nd > 0 else None
    vt = to_dev(VL) if Nd > 0 else None
    out = mf.mustafar_sparse_decode_attn(to_dev(q), Kc, Vc, kt, vt, scale=scale, n_splits=splits)
    got = out.cpu().numpy()
    ref = oracle.sparse_decode_attention(q, oracle.compress(K, sK), oracle.compress(V, sV),
                                         KL, VL, scale=scale)
    err = attn_error(got, ref)
    assert err <= ATTN_TOL, err
    return err


@pytest.mark.parametrize("G", [1, 2, 4, 8])
@pytest.mark.parametrize("Nd", [0, 1, 31, 32])
def test_attention_group_sizes_and_windows(G, Nd):
    _attn_case(B=2, Hkv=2, G=G, Ns=700, Nd=Nd, d=128, sK=0.5, sV=0.7, splits=0, seed=G * 10 + Nd)


@pytest.mark.parametrize("Ns", [0, 1, 64, 4095])
@pytest.mark.parametrize("splits", [1, 2, 7, 64])
def test_attention_lengths_and_splits(Ns, splits):
    _attn_case(B=1, Hkv=4, G=4, Ns=Ns, Nd=32, d=128, sK=0.7, sV=0.7, splits=splits, seed=Ns + 3)


@pytest.mark.parametrize("d", [64, 256])
@pytest.mark.parametrize("G", [1, 4])
def test_attention_other_head_dims(d, G):
    _attn_case(B=2, Hkv=2, G=G, Ns=333, Nd=32, d=d, sK=0.5, sV=0.5, splits=0, seed=d + G)


# k compressed segments of 64 tokens plus the window segment. The merge runs
# eight waves that take 16 segments at a time: counts around one wave's share
# (8), a full round (128) and several rounds, in one level (256 query heads, or
# at most 128 segments) and in two levels (more segments, fewer heads).
@pytest.mark.parametrize("B,Hkv,G,d,k", [(1, 4, 1, 128, 6), (1, 4, 1, 128, 7), (1, 4, 4, 128, 126),
                                         (1, 4, 1, 128, 127), (1, 2, 2, 128, 128), (1, 2, 1, 128, 300),
                                         (2, 64, 2, 64, 127), (2, 64, 2, 64, 140)])
def test_attention_merge_segment_counts(B, Hkv, G, d, k):
    _attn_case(B=B, Hkv=Hkv, G=G, Ns=64 * k, Nd=32, d=d, sK=0.7, sV=0.7, splits=k, seed=k + G)


# The decode kernels read one tile offset per segment and derive the others from
# the bitmaps (a stream's tiles are packed back to back), so a cache assembled
# from a bulk compression, a second one starting mid-block, single appends and a
# third compression must attend exactly like the oracle's compress-all, with
# segment starts falling in every part (split counts) and on every kernel body
# (one head: walks; four: grouped walks; eight: matrix cores).
@pytest.mark.parametrize("d,G", [(128, 1), (128, 4), (128, 8), (64, 1), (256, 4)])
@pytest.mark.parametrize("splits", [0, 3, 11])
def test_attention_over_caches_built_in_pieces(d, G, splits):
    announce(f"attn pieces d={d} G={G} splits={splits}")
    B, Hkv, Nd = 2, 3, 32
    n0, n1, n2, n3 = 301, 133, 23, 170
    N = n0 + n1 + n2 + n3
    K, V = synth.make_kv(B, Hkv, N, d, seed=d + G)
    KL, VL = synth.make_tail(B, Hkv, Nd, d, seed=d + G)
    q = synth.make_q(B, Hkv * G, d, seed=d + G)
    Kc = mf.CompressedCache(B, Hkv, d, 0.5, N)
    Vc = mf.CompressedCache(B, Hkv, d, 0.7, N)
    for c, x in ((Kc, K), (Vc, V)):
        mf.mustafar_prune_compress(c, to_dev(np.ascontiguousarray(x[:, :, :n0])))
        mf.mustafar_prune_compress(c, to_dev(np.ascontiguousarray(x[:, :, n0:n0 + n1])))
        for j in range(n0 + n1, n0 + n1 + n2):
            mf.mustafar_append(c, to_dev(np.ascontiguousarray(x[:, :, j])))
        mf.mustafar_prune_compress(c, to_dev(np.ascontiguousarray(x[:, :, n0 + n1 + n2:])))
        assert c.n_tokens == N
    out = mf.mustafar_sparse_decode_attn(to_dev(q), Kc, Vc, to_dev(KL), to_dev(VL), n_splits=splits)
    ref = oracle.sparse_decode_attention(q, oracle.compress(K, 0.5), oracle.compress(V, 0.7), KL, VL)
    err = attn_error(out.cpu().numpy(), ref)
    assert err <= ATTN_TOL, err


# The decode kernels read a tile offset only where a segment starts (segments
# are whole 64-token blocks) and rebuild the others from the bitmaps, which the
# bench's needed-bytes figure counts on: with every other offset zeroed (a
# valid position, so a kernel that read them would compute wrong sums rather
# than fault) the attention must not change.
@pytest.mark.parametrize("d,G", [(128, 1), (128, 4), (128, 8), (64, 1), (256, 4)])
def test_attention_reads_offsets_only_at_segment_starts(d, G):
    announce(f"attn segment-start offsets d={d} G={G}")
    B, Hkv, N, Nd = 2, 2, 700, 32
    K, V = synth.make_kv(B, Hkv, N, d, seed=d * 3 + G)
    KL, VL = synth.make_tail(B, Hkv, Nd, d, seed=d * 3 + G)
    q = synth.make_q(B, Hkv * G, d, seed=d * 3 + G)
    Kc = mf.CompressedCache(B, Hkv, d, 0.5, N)
    Vc = mf.CompressedCache(B, Hkv, d, 0.7, N)
    mf.mustafar_prune_compress(Kc, to_dev(K))
    mf.mustafar_prune_compress(Vc, to_dev(V))
    for c in (Kc, Vc):
        starts = c.offsets[:, :, ::64, 0].clone()
        c.offsets.zero_()
        c.offsets[:, :, ::64, 0] = starts
    ref = oracle.sparse_decode_attention(q, oracle.compress(K, 0.5), oracle.compress(V, 0.7), KL, VL)
    for splits in (0, 1, 3, 11):
        out = mf.mustafar_sparse_decode_attn(to_dev(q), Kc, Vc, to_dev(KL), to_dev(VL), n_splits=splits)
        err = attn_error(out.cpu().numpy(), ref)
        assert err <= ATTN_TOL, (splits, err)


@pytest.mark.parametrize("sK,sV", [(0.0, 0.0), (0.9, 0.9), (1.0, 0.5), (0.5, 1.0), (1.0, 1.0)])
def test_attention_extreme_sparsities(sK, sV):
    _attn_case(B=1, Hkv=2, G=2, Ns=200, Nd=5, d=128, sK=sK, sV=sV, splits=3, seed=31)


def test_attention_custom_scale():
    _attn_case(B=1, Hkv=2, G=1, Ns=128, Nd=32, d=128, sK=0.5, sV=0.5, splits=2, seed=5,
               scale=0.02)


def test_attention_only_window():
    _attn_case(B=2, Hkv=2, G=2, Ns=0, Nd=200, d=128, sK=0.5, sV=0.5, splits=0, seed=6)


@pytest.mark.parametrize("G", [1, 4])
@pytest.mark.parametrize("splits", [0, 1, 5])
def test_dense_attention_parity(G, splits):
    announce(f"dense attn G={G} splits={splits}")
    B, Hkv, N, d = 2, 3, 1000, 128
    K, V = synth.make_kv(B, Hkv, N, d, seed=9)
    q = synth.make_q(B, Hkv * G, d, seed=9)
    got = mf.mustafar_dense_decode_attn(to_dev(q), to_dev(K), to_dev(V), n_splits=splits)
    ref = oracle.decode_attention(q, np.zeros((B, Hkv, 0, d), np.float16),
                                  np.zeros((B, Hkv, 0, d), np.float16), K, V)
    assert attn_error(got.cpu().numpy(), ref) <= ATTN_TOL


def test_decode_loop_append_then_attend():
    """Paper's decode step: the token leaving the window is pruned, compressed and
    appended, then attention runs over compressed + window (Sec. 3)."""
    B, Hkv, G, d, n0, steps, W = 1, 4, 4, 128, 500, 12, 32
    announce("decode loop")
    K, V = synth.make_kv(B, Hkv, n0 + steps + W, d, seed=12)
    q = synth.make_q(B, Hkv * G, d, seed=12)
    Kc = mf.CompressedCache(B, Hkv, d, 0.7, n0 + steps)
    Vc = mf.CompressedCache(B, Hkv, d, 0.7, n0 + steps)
    mf.mustafar_prune_compress(Kc, to_dev(np.ascontiguousarray(K[:, :, :n0])))
    mf.mustafar_prune_compress(Vc, to_dev(np.ascontiguousarray(V[:, :, :n0])))
    qd = to_dev(q)
    for step in range(steps + 1):
        ns = n0 + step
        win_k = np.ascontiguousarray(K[:, :, ns:ns + W])
        win_v = np.ascontiguousarray(V[:, :, ns:ns + W])
        got = mf.mustafar_sparse_decode_attn(qd, Kc, Vc, to_dev(win_k), to_dev(win_v))
        if step in (0, 1, steps):
            ref = oracle.sparse_decode_attention(
                q, oracle.compress(np.ascontiguousarray(K[:, :, :ns]), 0.7),
                oracle.compress(np.ascontiguousarray(V[:, :, :ns]), 0.7), win_k, win_v)
            assert attn_error(got.cpu().numpy(), ref) <= ATTN_TOL, step
        if step < steps:
            mf.mustafar_append(Kc, to_dev(np.ascontiguousarray(K[:, :, ns])))
            mf.mustafar_append(Vc, to_dev(np.ascontiguousarray(V[:, :, ns])))


def test_stream_read_checksum():
    # The read-ceiling helper must really read every byte: the XOR of the
    # per-workgroup checksums equals the XOR of all 32-bit words.
    import torch
    announce("stream read checksum")
    rng = np.random.default_rng(3)
    words = rng.integers(0, 2 ** 32, size=(1 << 20) + 12, dtype=np.uint64).astype(np.uint32)
    buf = torch.from_numpy(words.view(np.int32)).cuda()
    sink = mf.mustafar_stream_read(buf).cpu().numpy().view(np.uint32)
    assert int(np.bitwise_xor.reduce(sink)) == int(np.bitwise_xor.reduce(words))


@pytest.mark.parametrize("w16", [0, 9, 16])
def test_stream_mix_writes_the_selected_words(w16):
    # The read+write ceiling helper reads every word (the checksum) and stores
    # words 0..w16-1 of every group of 16 16-byte words, packed; nothing past
    # them.
    import torch
    announce(f"stream mix w16={w16}")
    rng = np.random.default_rng(4)
    n16 = (1 << 16) + 48  # a multiple of 16 words, past one grid-stride pass
    words = rng.integers(0, 2 ** 32, size=(n16, 4), dtype=np.uint64).astype(np.uint32)
    src = torch.from_numpy(words.view(np.int32)).cuda()
    out_words = n16 // 16 * w16
    dst = torch.full((out_words + 16, 4), -1, dtype=torch.int32, device="cuda")
    sink = mf.mustafar_stream_mix(src, dst, w16).cpu().numpy().view(np.uint32)
    assert int(np.bitwise_xor.reduce(sink)) == int(np.bitwise_xor.reduce(words.ravel()))
    got = dst.cpu().numpy().view(np.uint32)
    want = words.reshape(-1, 16, 4)[:, :w16].reshape(-1, 4)
    assert np.array_equal(got[:out_words], want)
    assert (got[out_words:] == 0xffffffff).all()


@pytest.mark.parametrize("n_streams,n_chunks,w16", [(3, 5, 9), (1, 2, 16), (4, 1, 0), (7, 3, 5)])
def test_stream_chunks_writes_each_chunks_share(n_streams, n_chunks, w16):
    # The compression-order helper: workgroup g reads chunk g / n_streams of
    # stream g % n_streams (its checksum goes to sink[g]) and stores the first
    # w16/16 of the chunk's 16-byte words, packed, at the chunk's place.
    import torch
    announce(f"stream chunks {n_streams}x{n_chunks} w16={w16}")
    P = mf.STREAM_CHUNK_BYTES // 16
    rng = np.random.default_rng(n_streams * 31 + w16)
    words = rng.integers(0, 2 ** 32, size=(n_streams, n_chunks, P, 4), dtype=np.uint64).astype(np.uint32)
    src = torch.from_numpy(words.view(np.int32).reshape(-1, 4)).cuda()
    out_p = P * w16 // 16
    dst = torch.full((n_streams * n_chunks * out_p + 16, 4), -1, dtype=torch.int32, device="cuda")
    sink = mf.mustafar_stream_chunks(src, n_streams, dst, w16).cpu().numpy().view(np.uint32)
    g = np.arange(n_streams * n_chunks)
    want_sink = np.bitwise_xor.reduce(words.reshape(n_streams, n_chunks, -1), axis=-1)[g % n_streams,
                                                                                        g // n_streams]
    assert np.array_equal(sink, want_sink)
    got = dst.cpu().numpy().view(np.uint32)
    want = words[:, :, :out_p].reshape(-1, 4)
    assert np.array_equal(got[:n_streams * n_chunks * out_p], want)
    assert (got[n_streams * n_chunks * out_p:] == 0xffffffff).all()


@pytest.fixture
def route():
    """Sets a kernel route for one test and restores the default afterwards."""
    def set_route(r):
        mf.mustafar_attn_set_route(r)
    yield set_route
    mf.mustafar_attn_set_route(mf.ROUTE_DEFAULT)


@pytest.mark.parametrize("kernel", ["walks", "matrix_cores"])
@pytest.mark.parametrize("G", [2, 4, 8])
@pytest.mark.parametrize("d", [64, 128, 256])
def test_attention_both_grouped_kernels(route, kernel, G, d):
    # Either kernel serves every group size (the default picks one per size):
    # both meet the oracle, over several blocks, a ragged tail and a window.
    route(mf.ROUTE_WALKS if kernel == "walks" else mf.ROUTE_MATRIX_CORES)
    announce(f"route {kernel} G={G} d={d}")
    _attn_case(B=2, Hkv=2, G=G, Ns=517, Nd=32, d=d, sK=0.5, sV=0.7, splits=0, seed=40 + G + d)
    _attn_case(B=1, Hkv=2, G=G, Ns=1000, Nd=0, d=d, sK=0.7, sV=0.7, splits=3, seed=41 + G + d)
