"""Pins of the oracle's pruner variants (same compressed format, other selections).

* 2:4 per token (Appendix B): exhaustive enumeration of each group's pairs, the
  2-of-4 invariant, and a numpy stable sort per group;
* output-aware key pruning (Sec. 2): numpy's float32 products and stable sort,
  unit weights reduce it to magnitude pruning, power-of-two scalings and
  channel permutations act as they must;
* per-head kept counts (finer-grained sparsity, future work in Conclusion and
  Limitations): every head keeps its
  own count, and equals the magnitude compressor run on that head alone;
* the query lookahead weights: closed forms for constant queries.
"""
import itertools

import numpy as np
import pytest

import oracle


def _tie_heavy(rng, shape):
    mags = np.array([0.0, 2.0 ** -24, 0.5, 1.0, 1.0, 2.0, 3.0], dtype=np.float32)
    return (rng.choice(mags, size=shape) * rng.choice([-1.0, 1.0], size=shape)).astype(np.float16)


# ---- 2:4 ---------------------------------------------------------------------------------
def test_24_equals_enumeration_of_each_group():
    rng = np.random.default_rng(0)
    for _ in range(200):
        x = _tie_heavy(rng, 64)
        keep = oracle.prune_token_24(x)
        for g in range(0, 64, 4):
            mags = np.abs(x[g:g + 4].astype(np.float64))
            # the pair whose (magnitude desc, channel asc) key list is largest
            def key(pair):
                return sorted(((mags[i], -i) for i in pair), reverse=True)
            best = max(itertools.combinations(range(4), 2), key=key)
            assert [int(keep[g + i]) for i in range(4)] == [int(i in best) for i in range(4)]


def test_24_numpy_stable_sort_and_invariants():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((2, 3, 40, 128)).astype(np.float16)
    enc = oracle.compress_variant(x, "2:4")
    for b in range(2):
        for h in range(3):
            for j in range(40):
                bm = enc["bitmaps"][b, h, j]
                for t in range(2):
                    w = int(bm[t])
                    for nib in range(16):
                        assert bin((w >> (4 * nib)) & 0xF).count("1") == 2
                tok = np.abs(x[b, h, j].astype(np.float32))
                want = np.zeros(128, dtype=bool)
                for g in range(0, 128, 4):
                    order = np.argsort(-tok[g:g + 4], kind="stable")
                    want[g + order[:2]] = True
                got = np.array([(int(bm[c // 64]) >> (c % 64)) & 1 for c in range(128)], dtype=bool)
                assert np.array_equal(got, want)
    dec = oracle.decompress(enc)
    assert (dec.view(np.float16) != 0).sum() <= x.size // 2   # exactly half kept (zeros aside)


# ---- output-aware ------------------------------------------------------------------------
def test_output_aware_with_unit_weights_is_magnitude_pruning():
    rng = np.random.default_rng(2)
    x = _tie_heavy(rng, (1, 2, 30, 128))
    w = np.ones(x.shape, dtype=np.float32)
    for k in (1, 38, 64, 127):
        a = oracle.compress_variant(x, "output_aware", k=k, weights=w)
        b = oracle.compress(x, k=k)
        for key in ("bitmaps", "offsets", "stream_len"):
            assert np.array_equal(a[key], b[key]), (k, key)


@pytest.mark.parametrize("k", [5, 64, 90])
def test_output_aware_equals_numpy_float32_scores(k):
    rng = np.random.default_rng(3)
    for _ in range(100):
        x = rng.standard_normal(128).astype(np.float16)
        w = np.abs(rng.standard_normal(128)).astype(np.float32) * np.float32(7.0)
        w[rng.integers(0, 128, 5)] = 0.0                      # channels no query reads
        s = np.abs(x.astype(np.float32)) * w                  # IEEE float32 products
        want = np.zeros(128, dtype=bool)
        want[np.argsort(-s, kind="stable")[:k]] = True
        assert np.array_equal(oracle.prune_token_scored(x, w, k), want)


def test_output_aware_invariances():
    rng = np.random.default_rng(4)
    x = rng.standard_normal(128).astype(np.float16)
    w = np.abs(rng.standard_normal(128)).astype(np.float32)
    base = oracle.prune_token_scored(x, w, 40)
    assert np.array_equal(oracle.prune_token_scored(x, w * np.float32(4.0), 40), base)
    # Weights that favour one channel enormously keep it whatever its magnitude.
    w2 = w.copy()
    c = int(np.argmin(np.abs(x.astype(np.float32)) + (x == 0) * 1e9))
    w2[c] = np.float32(1e30)
    assert oracle.prune_token_scored(x, w2, 1)[c]
    # Swapping two channels of x and w swaps their decisions (no other tie).
    perm = np.arange(128)
    perm[[3, 77]] = [77, 3]
    p = oracle.prune_token_scored(x[perm], w[perm], 40)
    assert np.array_equal(p, base[perm])


# ---- per-head kept counts ----------------------------------------------------------------
def test_per_head_counts_and_equivalence_with_one_head_caches():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 4, 25, 128)).astype(np.float16)
    hk = [64, 38, 13, 100]
    enc = oracle.compress_variant(x, "magnitude", head_keep=hk)
    for h in range(4):
        pc = np.zeros(enc["bitmaps"][:, h].shape[:2], dtype=np.int64)
        for t in range(2):
            pc += np.vectorize(lambda v: bin(int(v)).count("1"))(enc["bitmaps"][:, h, :, t])
        assert (pc == hk[h]).all()
        one = oracle.compress(x[:, h:h + 1], k=hk[h])
        for key in ("bitmaps", "offsets", "stream_len"):
            assert np.array_equal(enc[key][:, h:h + 1], one[key]), (h, key)
        n = int(one["stream_len"].max())
        assert np.array_equal(enc["values"][:, h:h + 1, :n], one["values"][:, :, :n])


# ---- query lookahead ---------------------------------------------------------------------
def test_query_lookahead_closed_forms():
    B, Hq, Hkv, Nq, d = 2, 8, 2, 45, 64
    q = np.full((B, Hq, Nq, d), -0.75, dtype=np.float16)     # |q| = 0.75 everywhere
    out = oracle.query_lookahead(q, Hkv, 32)
    G = Hq // Hkv
    for T in range(Nq):
        n = min(32, Nq - T)
        assert np.all(out[:, :, T] == np.float32(0.75 * G * n)), T
    rng = np.random.default_rng(6)
    q2 = rng.standard_normal((1, 2, 10, 64)).astype(np.float16)
    one = oracle.query_lookahead(q2, 2, 1)                    # L = 1, G = 1: |q| itself
    assert np.array_equal(one, np.abs(q2.astype(np.float32)))
