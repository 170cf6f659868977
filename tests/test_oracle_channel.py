"""Pins of the oracle's per-channel value pruning and attention probabilities.

Per-channel pruning in groups of 32 tokens (Sec. 2, value-cache study): in each
group every channel keeps the k tokens of largest key, ties to the lower token;
the key is |v| (magnitude) or the fp32 product |v| * A_j (output-aware, A_j the
attention probability mass token j received). Pinned against:

* numpy's stable argsort of each channel's keys (float32 products for the
  output-aware key);
* brute-force enumeration of every k-subset of a channel on tiny groups;
* invariants: exactly k kept per channel and group, unit weights reduce to
  magnitude pruning, power-of-two weight scalings and token permutations act
  as they must, groups are independent;
* the attention probabilities: a numpy float64 softmax of the scores, summing
  to one, and Algorithm 1's output equals probabilities times values.
"""
import itertools

import numpy as np
import pytest

import oracle

GROUP = 32


def _tie_heavy(rng, shape):
    mags = np.array([0.0, 2.0 ** -24, 0.5, 1.0, 1.0, 2.0, 3.0], dtype=np.float32)
    return (rng.choice(mags, size=shape) * rng.choice([-1.0, 1.0], size=shape)).astype(np.float16)


def _numpy_keep(x, k, w=None):
    mag = np.abs(x.astype(np.float32))
    key = mag if w is None else mag * np.asarray(w, dtype=np.float32)[:, None]
    n, d = x.shape
    want = np.zeros((n, d), dtype=bool)
    for c in range(d):
        order = np.argsort(-key[:, c], kind="stable")
        want[order[:k], c] = True
    return want


# ---- magnitude ---------------------------------------------------------------------------
@pytest.mark.parametrize("k", [0, 1, 10, 16, 31, 32])
def test_channel_prune_equals_stable_argsort(k):
    rng = np.random.default_rng(k)
    for ties in (False, True):
        x = _tie_heavy(rng, (GROUP, 128)) if ties else rng.standard_normal((GROUP, 128)).astype(np.float16)
        got = oracle.prune_channel_group(x, k)
        assert np.array_equal(got, _numpy_keep(x, k)), (k, ties)
        assert (got.sum(0) == k).all()


def test_channel_prune_equals_brute_force():
    rng = np.random.default_rng(1)
    n, d = 6, 64
    for _ in range(20):
        x = _tie_heavy(rng, (n, d))
        for k in (1, 2, 4):
            got = oracle.prune_channel_group(x, k)
            mags = np.abs(x.astype(np.float64))
            for c in range(d):
                def key(sub):
                    return sorted(((mags[j, c], -j) for j in sub), reverse=True)
                best = max(itertools.combinations(range(n), k), key=key)
                assert [bool(got[j, c]) for j in range(n)] == [j in best for j in range(n)]


def test_keep_count_of_a_group():
    assert oracle.keep_count(GROUP, 0.7) == 10
    assert oracle.keep_count(GROUP, 0.5) == 16
    assert oracle.keep_count(GROUP, 0.0) == 32
    assert oracle.keep_count(GROUP, 1.0) == 0


# ---- output-aware --------------------------------------------------------------------------
@pytest.mark.parametrize("k", [3, 10, 20])
def test_output_aware_channel_prune_equals_numpy_float32(k):
    rng = np.random.default_rng(2 + k)
    for _ in range(10):
        x = rng.standard_normal((GROUP, 128)).astype(np.float16)
        w = (np.abs(rng.standard_normal(GROUP)) * 0.03).astype(np.float32)
        w[rng.integers(0, GROUP, 3)] = 0.0
        got = oracle.prune_channel_group(x, k, w)
        assert np.array_equal(got, _numpy_keep(x, k, w))


def test_output_aware_invariances():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((GROUP, 64)).astype(np.float16)
    w = np.abs(rng.standard_normal(GROUP)).astype(np.float32)
    base = oracle.prune_channel_group(x, 10, w)
    # unit weights: magnitude pruning
    assert np.array_equal(oracle.prune_channel_group(x, 10, np.ones(GROUP, np.float32)),
                          oracle.prune_channel_group(x, 10))
    # a power-of-two scaling of every weight changes no product's order
    assert np.array_equal(oracle.prune_channel_group(x, 10, w * np.float32(0.25)), base)
    # permuting the tokens (x rows and weights together) permutes the decisions
    perm = rng.permutation(GROUP)
    assert np.array_equal(oracle.prune_channel_group(x[perm], 10, w[perm]), base[perm])
    # a token with an overwhelming weight is kept in every channel where it is non-zero
    w2 = w.copy()
    w2[7] = np.float32(1e30)
    got = oracle.prune_channel_group(x, 1, w2)
    nz = x[7].astype(np.float32) != 0
    assert got[7][nz].all()


# ---- the grouped format ----------------------------------------------------------------------
def test_grouped_compression_round_trip_and_group_independence():
    rng = np.random.default_rng(4)
    B, H, N, d = 1, 2, 96, 128
    x = rng.standard_normal((B, H, N, d)).astype(np.float16)
    w = np.abs(rng.standard_normal((B, H, N))).astype(np.float32)
    for weights in (None, w):
        enc = oracle.compress_grouped(x, 0.7, weights=weights)
        dec = oracle.decompress(enc).view(np.float16)
        for h in range(H):
            for g0 in range(0, N, GROUP):
                grp = x[0, h, g0:g0 + GROUP]
                keep = _numpy_keep(grp, 10, None if weights is None else w[0, h, g0:g0 + GROUP])
                want = np.where(keep, grp, np.float16(0))
                assert np.array_equal(dec[0, h, g0:g0 + GROUP].view(np.uint16),
                                      want.view(np.uint16))
        # each group alone compresses to the same bitmaps
        for g0 in range(0, N, GROUP):
            part = oracle.compress_grouped(x[:, :, g0:g0 + GROUP], 0.7,
                                           weights=None if weights is None else w[:, :, g0:g0 + GROUP])
            assert np.array_equal(part["bitmaps"], enc["bitmaps"][:, :, g0:g0 + GROUP])
        assert (enc["stream_len"] <= oracle.grouped_stream_capacity(d, 10, N)).all()


def test_grouped_compression_rejects_partial_groups():
    with pytest.raises(ValueError):
        oracle.compress_grouped(np.zeros((1, 1, 40, 64), np.float16), 0.5)


# ---- attention probabilities -----------------------------------------------------------------
@pytest.mark.parametrize("G", [1, 4])
def test_attention_probs_equal_numpy_softmax(G):
    rng = np.random.default_rng(5 + G)
    B, Hkv, Ns, Nd, d = 2, 2, 20, 7, 64
    q = rng.standard_normal((B, Hkv * G, d)).astype(np.float16)
    kc = rng.standard_normal((B, Hkv, Ns, d)).astype(np.float16)
    kl = rng.standard_normal((B, Hkv, Nd, d)).astype(np.float16)
    p = oracle.attention_probs(q, kc, kl)
    for b in range(B):
        for hq in range(Hkv * G):
            keys = np.concatenate([kc[b, hq // G], kl[b, hq // G]]).astype(np.float64)
            s = keys @ q[b, hq].astype(np.float64) / np.sqrt(d)
            e = np.exp(s - s.max())
            np.testing.assert_allclose(p[b, hq], e / e.sum(), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=1e-12)


def test_attention_output_equals_probabilities_times_values():
    rng = np.random.default_rng(8)
    B, Hkv, G, Ns, Nd, d = 1, 2, 2, 12, 5, 64
    q = rng.standard_normal((B, Hkv * G, d)).astype(np.float16)
    kc = rng.standard_normal((B, Hkv, Ns, d)).astype(np.float16)
    vc = rng.standard_normal((B, Hkv, Ns, d)).astype(np.float16)
    kl = rng.standard_normal((B, Hkv, Nd, d)).astype(np.float16)
    vl = rng.standard_normal((B, Hkv, Nd, d)).astype(np.float16)
    p = oracle.attention_probs(q, kc, kl, scale=0.3)
    o = oracle.decode_attention(q, kc, vc, kl, vl, scale=0.3)
    for hq in range(Hkv * G):
        vals = np.concatenate([vc[0, hq // G], vl[0, hq // G]]).astype(np.float64)
        np.testing.assert_allclose(o[0, hq], p[0, hq] @ vals, rtol=1e-10, atol=1e-12)


def test_output_aware_key_is_rounded_to_fp32():
    """Two tokens whose exact products differ but round to the same fp32 value tie,
    and the tie goes to the lower token (the key is decided in fp32)."""
    x = np.array([[1.0], [1.0 + 2.0 ** -10]], dtype=np.float16)
    w0 = np.float32(1.0 + 2.0 ** -23)
    target = np.float64(w0)
    w1 = np.float32(target / (1.0 + 2.0 ** -10))
    found = None
    for _ in range(64):
        exact = (1.0 + 2.0 ** -10) * np.float64(w1)
        if np.float32(exact) == w0 and exact > target:
            found = w1
            break
        w1 = np.nextafter(w1, np.float32(2.0))
    assert found is not None
    keep = oracle.prune_channel_group(np.tile(x, (1, 64)), 1, np.array([w0, found], np.float32))
    assert keep[0].all() and not keep[1].any()
