"""GPU parity of the pruner variants (mustafar_prune_compress_ex / _append_ex,
mustafar_query_lookahead) against the oracle, bit for bit, and decode attention
over the variant caches within the 2e-3 tolerance.
"""
import numpy as np
import pytest

import oracle
import paper_2505_22913_amd as mf
from tests.gpu_common import ATTN_TOL, all_pairs, announce, attn_error, compare_format, read_cache

pytestmark = pytest.mark.gpu


def _dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _tokens(rng, B, H, N, d, ties=False):
    if ties:
        mags = np.array([0.0, 2.0 ** -24, 0.5, 1.0, 1.0, 2.0], dtype=np.float32)
        return (rng.choice(mags, size=(B, H, N, d)) *
                rng.choice([-1.0, 1.0], size=(B, H, N, d))).astype(np.float16)
    x = rng.standard_normal((B, H, N, d)).astype(np.float16)
    x[..., 3] *= 10
    return x


@pytest.mark.parametrize("d,ties", [(128, False), (128, True), (64, False), (256, True)])
def test_24_compress_and_append(d, ties):
    announce(f"2:4 d={d} ties={ties}")
    rng = np.random.default_rng(d + ties)
    B, H, N = 2, 3, 150
    x = _tokens(rng, B, H, N + 3, d, ties)
    c = mf.CompressedCache(B, H, d, 0.5, N + 3)
    mf.mustafar_prune_compress_ex(c, _dev(x[:, :, :N]), mode=mf.PRUNE_2_4)
    for j in range(N, N + 3):
        mf.mustafar_append_ex(c, _dev(x[:, :, j]), mode=mf.PRUNE_2_4)
    want = oracle.compress_variant(x, "2:4")
    compare_format(read_cache(c), want, N + 3, all_pairs(B, H))


@pytest.mark.parametrize("d", [128, 256])
def test_per_head_counts(d):
    announce(f"per-head counts d={d}")
    rng = np.random.default_rng(11)
    B, H, N = 2, 4, 130
    hk = [d // 2, d // 4, 1, 0] if d == 128 else [128, 77, 3, 100]
    x = _tokens(rng, B, H, N + 2, d)
    c = mf.CompressedCache(B, H, d, 0.5, N + 2)
    mf.mustafar_prune_compress_ex(c, _dev(x[:, :, :N]), head_keep=hk)
    for j in range(N, N + 2):
        mf.mustafar_append_ex(c, _dev(x[:, :, j]), head_keep=hk)
    want = oracle.compress_variant(x, "magnitude", head_keep=hk)
    compare_format(read_cache(c), want, N + 2, all_pairs(B, H))


def test_magnitude_through_the_variant_path_equals_the_default():
    announce("magnitude variant path")
    rng = np.random.default_rng(12)
    B, H, N, d = 2, 3, 200, 128
    x = _tokens(rng, B, H, N, d, ties=True)
    a = mf.CompressedCache(B, H, d, 0.7, N)
    b = mf.CompressedCache(B, H, d, 0.7, N)
    mf.mustafar_prune_compress_ex(a, _dev(x), mode=mf.PRUNE_MAGNITUDE, head_keep=[a.n_keep] * H)
    mf.mustafar_prune_compress(b, _dev(x))
    ga, gb = read_cache(a), read_cache(b)
    compare_format(ga, gb, N, all_pairs(B, H))


@pytest.mark.parametrize("G,L", [(1, 32), (4, 32), (2, 5), (2, 32), (8, 32)])
def test_query_lookahead_bit_exact(G, L):
    announce(f"lookahead G={G} L={L}")
    rng = np.random.default_rng(13 + G)
    B, Hkv, Nq, d = 2, 2, 70, 128
    q = rng.standard_normal((B, Hkv * G, Nq, d)).astype(np.float16)
    got = mf.mustafar_query_lookahead(_dev(q), Hkv, L).cpu().numpy()
    want = oracle.query_lookahead(q, Hkv, L)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("G,s", [(1, 0.5), (4, 0.7)])
def test_output_aware_keys_and_attention(G, s):
    """Keys pruned with the lookahead weights of the queries that follow them
    (the last 32 tokens stay dense, so every compressed key has its 32 queries),
    bit-exact, then Algorithm 1 over them within tolerance."""
    import torch
    announce(f"output-aware G={G} s={s}")
    rng = np.random.default_rng(14 + G)
    B, Hkv, d, N, W = 2, 2, 128, 160, 32
    Hq = Hkv * G
    x = _tokens(rng, B, Hkv, N + W, d)
    v = rng.standard_normal((B, Hkv, N + W, d)).astype(np.float16)
    qs = rng.standard_normal((B, Hq, N + W, d)).astype(np.float16)
    w_dev = mf.mustafar_query_lookahead(_dev(qs), Hkv, 32)
    w_ref = oracle.query_lookahead(qs, Hkv, 32)
    Kc = mf.CompressedCache(B, Hkv, d, s, N)
    Vc = mf.CompressedCache(B, Hkv, d, 0.7, N)
    mf.mustafar_prune_compress_ex(Kc, _dev(x[:, :, :N]), mode=mf.PRUNE_OUTPUT_AWARE,
                                  weights=w_dev[:, :, :N].contiguous())
    mf.mustafar_prune_compress(Vc, _dev(v[:, :, :N]))
    want = oracle.compress_variant(x[:, :, :N], "output_aware", k=Kc.n_keep,
                                   weights=w_ref[:, :, :N])
    compare_format(read_cache(Kc), want, N, all_pairs(B, Hkv))
    q = rng.standard_normal((B, Hq, d)).astype(np.float16)
    out = mf.mustafar_sparse_decode_attn(_dev(q), Kc, Vc, _dev(x[:, :, N:]), _dev(v[:, :, N:]))
    torch.cuda.synchronize()
    ref = oracle.sparse_decode_attention(q, want, oracle.compress(v[:, :, :N], 0.7),
                                         x[:, :, N:], v[:, :, N:])
    err = attn_error(out.cpu().numpy(), ref)
    announce(f"output-aware G={G}: attention error {err:.2e}")
    assert err <= ATTN_TOL


def test_output_aware_append():
    announce("output-aware append")
    rng = np.random.default_rng(15)
    B, H, d, N = 2, 3, 128, 4
    x = _tokens(rng, B, H, N, d)
    w = np.abs(rng.standard_normal((B, H, N, d))).astype(np.float32)
    c = mf.CompressedCache(B, H, d, 0.6, N)
    for j in range(N):
        mf.mustafar_append_ex(c, _dev(x[:, :, j]), mode=mf.PRUNE_OUTPUT_AWARE,
                              weights=_dev(w[:, :, j]))
    want = oracle.compress_variant(x, "output_aware", k=c.n_keep, weights=w)
    compare_format(read_cache(c), want, N, all_pairs(B, H))


def test_attention_over_24_caches():
    import torch
    announce("attention over 2:4 caches")
    rng = np.random.default_rng(16)
    B, Hkv, G, d, N = 2, 2, 2, 128, 300
    k = _tokens(rng, B, Hkv, N + 32, d)
    v = rng.standard_normal((B, Hkv, N + 32, d)).astype(np.float16)
    Kc = mf.CompressedCache(B, Hkv, d, 0.5, N)
    Vc = mf.CompressedCache(B, Hkv, d, 0.5, N)
    mf.mustafar_prune_compress_ex(Kc, _dev(k[:, :, :N]), mode=mf.PRUNE_2_4)
    mf.mustafar_prune_compress_ex(Vc, _dev(v[:, :, :N]), mode=mf.PRUNE_2_4)
    q = rng.standard_normal((B, Hkv * G, d)).astype(np.float16)
    out = mf.mustafar_sparse_decode_attn(_dev(q), Kc, Vc, _dev(k[:, :, N:]), _dev(v[:, :, N:]))
    torch.cuda.synchronize()
    ref = oracle.sparse_decode_attention(q, oracle.compress_variant(k[:, :, :N], "2:4"),
                                         oracle.compress_variant(v[:, :, :N], "2:4"),
                                         k[:, :, N:], v[:, :, N:])
    err = attn_error(out.cpu().numpy(), ref)
    assert err <= ATTN_TOL, err
