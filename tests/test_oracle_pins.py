"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compare the oracle with itself: each checks it against a library
routine, an exhaustive enumeration, a hand-derived example, a closed form, an
invariant the paper states, or the compression ratios the paper prints
(arxiv 2505.22913). A plausible slip in the oracle -- a reversed tie rule, an
off-by-one in the packed index, a dropped pad, a missing score scale, a swapped
K/V operand -- fails at least one of them.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2505_22913_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _tie_heavy_rows(rng, n, d):
    """fp16 rows drawn from a tiny magnitude set with random signs: many exact
    ties, both zeros, and a subnormal."""
    mags = np.array([0.0, 2.0 ** -24, 0.5, 1.0, 1.0, 2.0, 3.0], dtype=np.float32)
    x = rng.choice(mags, size=(n, d)) * rng.choice([-1.0, 1.0], size=(n, d))
    return x.astype(np.float16)


# ----------------------------------------------------------------------------
# fp16 decoding and the kept count
# ----------------------------------------------------------------------------
def test_half_decoding_matches_numpy_for_every_pattern():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([oracle.half_to_double(int(b)) for b in bits])
    finite = np.isfinite(ref)
    assert np.array_equal(got[finite], ref[finite])
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    assert np.array_equal(got[np.isinf(ref)], ref[np.isinf(ref)])


@pytest.mark.parametrize("d,s,k", [(128, 0.0, 128), (128, 0.5, 64), (128, 0.7, 38),
                                   (128, 1.0, 0), (64, 0.5, 32), (256, 0.7, 77),
                                   (128, 0.50390625, 63)])  # s*d = 64.5: rounds half up
def test_keep_count_values(d, s, k):
    assert oracle.keep_count(d, s) == k


def test_keep_count_is_round_half_up_in_exact_arithmetic():
    rng = np.random.default_rng(0)
    for s in np.concatenate([rng.random(2000, dtype=np.float32), np.arange(257) / 256.0]):
        s = float(np.float32(s))
        for d in (64, 128, 256):
            exact = d - math.floor(Fraction(s) * d + Fraction(1, 2))
            assert oracle.keep_count(d, s) == exact, (s, d)


# ----------------------------------------------------------------------------
# per-token magnitude pruning (Sec. 2)
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("d", [64, 128])
def test_prune_equals_stable_argsort(d):
    """Keeping the k largest |x| with ties to the lower channel is exactly the
    first k entries of a stable ascending argsort of -|x|."""
    rng = np.random.default_rng(1)
    rows = np.concatenate([_tie_heavy_rows(rng, 40, d),
                           rng.standard_normal((40, d)).astype(np.float16)])
    for x in rows:
        order = np.argsort(-np.abs(x.astype(np.float64)), kind="stable")
        for k in range(0, d + 1, 7 if d == 128 else 3):
            want = np.zeros(d, dtype=bool)
            want[order[:k]] = True
            assert np.array_equal(oracle.prune_token(x, k), want), (x, k)


@pytest.mark.parametrize("d", [4, 6, 8])
def test_prune_equals_brute_force_enumeration(d):
    """Over every k-subset: the kept set has the largest total magnitude (only
    top-k sets reach it) and, among those, the lexicographically smallest
    sorted channel list (ties go to lower channels)."""
    rng = np.random.default_rng(2)
    for x in _tie_heavy_rows(rng, 60, d):
        mag = [abs(float(v)) for v in x.astype(np.float64)]
        for k in range(d + 1):
            best = None
            for sub in itertools.combinations(range(d), k):
                key = (-sum(mag[i] for i in sub), sub)
                if best is None or key < best:
                    best = key
            want = np.zeros(d, dtype=bool)
            want[list(best[1])] = True
            assert np.array_equal(oracle.prune_token(x, k), want), (x, k)


def test_every_token_keeps_exactly_k():
    K, V = synth.make_kv(1, 2, 96, 128, seed=3)
    for s in np.round(np.arange(0.0, 1.0001, 0.1), 2):
        for x in (K, V):
            enc = oracle.compress(x, float(s))
            k = oracle.keep_count(128, float(s))
            pop = np.vectorize(lambda b: bin(int(b)).count("1"))(enc["bitmaps"]).sum(axis=-1)
            assert np.all(pop == k), s


def test_zero_and_full_sparsity():
    K, _ = synth.make_kv(1, 2, 33, 128, seed=4)
    enc0 = oracle.compress(K, 0.0)
    assert np.all(enc0["bitmaps"] == np.uint64(0xFFFFFFFFFFFFFFFF))
    assert np.array_equal(oracle.decompress(enc0), K.view(np.uint16))
    enc1 = oracle.compress(K, 1.0)
    assert np.all(enc1["bitmaps"] == 0)
    assert np.all(enc1["offsets"] == 0)
    assert np.all(enc1["stream_len"] == 0)
    assert np.all(oracle.decompress(enc1) == 0)


# ----------------------------------------------------------------------------
# the bitmap format (Sec. 3; padding Sec. 4.3)
# ----------------------------------------------------------------------------
def test_hand_worked_example():
    """d = 128 (two tiles), sparsity 0.5 (k = 64), three tokens, derived by hand:
      token 0: |x| = 2 on channels 0..63, 1 on 64..127 -> tile 0 full, tile 1 empty
      token 1: all |x| = 1 -> ties: the 64 lowest channels, same pattern
      token 2: |x| = 3 on channels 1, 70, 127, 0.5 elsewhere -> the three big
               ones plus the 61 lowest remaining channels {0, 2..61}:
               tile 0 keeps channels 0..61 (62 values, padded to 64),
               tile 1 keeps channels 70 and 127 (bits 6 and 63, padded to 8)
    Offsets run 0, 64 | 64, 128 | 128, 192 and the stream holds 200 elements."""
    d = 128
    sign = np.where(np.arange(d) % 3 == 0, -1.0, 1.0)
    t0 = np.where(np.arange(d) < 64, 2.0, 1.0) * sign
    t1 = np.ones(d) * sign
    t2 = np.full(d, 0.5) * sign
    t2[[1, 70, 127]] = 3.0 * sign[[1, 70, 127]]
    x = np.stack([t0, t1, t2]).astype(np.float16)[None, None]
    enc = oracle.compress(x, 0.5)
    full = np.uint64(0xFFFFFFFFFFFFFFFF)
    assert enc["n_keep"] == 64
    assert enc["bitmaps"][0, 0].tolist() == [[full, 0], [full, 0],
                                             [np.uint64((1 << 62) - 1),
                                              np.uint64((1 << 63) | (1 << 6))]]
    assert enc["offsets"][0, 0].tolist() == [[0, 64], [64, 128], [128, 192]]
    assert int(enc["stream_len"][0, 0]) == 200
    xb = x[0, 0].view(np.uint16)
    vals = enc["values"][0, 0]
    assert np.array_equal(vals[0:64], xb[0, 0:64])
    assert np.array_equal(vals[64:128], xb[1, 0:64])
    assert np.array_equal(vals[128:190], xb[2, 0:62])
    assert np.all(vals[190:192] == 0)
    assert vals[192] == xb[2, 70] and vals[193] == xb[2, 127]
    assert np.all(vals[194:200] == 0)


@pytest.mark.parametrize("s", [0.3, 0.5, 0.7, 0.9])
def test_round_trip_and_layout_invariants(s):
    K, V = synth.make_kv(2, 3, 77, 128, seed=5)
    for x in (K, V):
        enc = oracle.compress(x, s)
        k = enc["n_keep"]
        # decode(encode(x)) is x with everything outside each token's top-k zeroed
        keep = np.stack([oracle.prune_token(t, k) for t in x.reshape(-1, 128)])
        pruned = np.where(keep, x.reshape(-1, 128).view(np.uint16), 0).reshape(x.shape)
        dec = oracle.decompress(enc)
        assert np.array_equal(dec, pruned)
        # encode(decode(enc)) == enc (no kept value is zero in this data)
        enc2 = oracle.compress(dec.view(np.float16), k=k)
        for key in ("bitmaps", "offsets", "values", "stream_len"):
            assert np.array_equal(enc[key], enc2[key]), key
        # offsets: multiples of 8, exclusive prefix sums of the padded counts
        cnt = np.vectorize(lambda b: bin(int(b)).count("1"))(enc["bitmaps"]).astype(np.int64)
        padded = (cnt + 7) // 8 * 8
        flat_pad = padded.reshape(2, 3, -1)
        excl = np.cumsum(flat_pad, axis=-1) - flat_pad
        assert np.array_equal(enc["offsets"].reshape(2, 3, -1), excl)
        assert np.all(enc["offsets"] % 8 == 0)
        assert np.array_equal(enc["stream_len"], flat_pad.sum(axis=-1))
        # pad slots hold +0.0
        for b in range(2):
            for h in range(3):
                off = enc["offsets"][b, h].reshape(-1)
                for o, c, p in zip(off, cnt[b, h].reshape(-1), padded[b, h].reshape(-1)):
                    assert np.all(enc["values"][b, h, o + c:o + p] == 0)


def test_compression_ratio_matches_paper():
    """Per-tile 8-byte bitmap + 4-byte offset + kept values padded to 8 lands on
    the ratios the paper prints for 50% and 70% sparsity."""
    gold = json.load(open(os.path.join(GOLDEN, "paper_compression_ratios.json")))
    tol = gold["tolerance_points"]
    K, V = synth.make_kv(1, 8, 2048, 128, seed=6)
    dense = K.nbytes

    def pct(x, s):
        return 100.0 * oracle.compressed_bytes(oracle.compress(x, s, threads=4)) / dense

    k50, v50, k70, v70 = pct(K, 0.5), pct(V, 0.5), pct(K, 0.7), pct(V, 0.7)
    r = gold["ratios_percent"]
    assert abs((k50 + v50) / 2 - r["k50_v50"]) <= tol
    assert abs((k70 + v70) / 2 - r["k70_v70"]) <= tol
    for single in (k50, v50):
        assert abs((single + 100.0) / 2 - r["one_cache_50_other_dense"]) <= tol
    for single in (k70, v70):
        assert abs((single + 100.0) / 2 - r["one_cache_70_other_dense"]) <= tol


# ----------------------------------------------------------------------------
# Algorithm 1 (decode attention over compressed + dense window)
# ----------------------------------------------------------------------------
def _sdpa64(q, k, v, scale=None):
    """torch's scaled_dot_product_attention in float64 on the CPU."""
    import torch
    qt = torch.from_numpy(q.astype(np.float64))[:, :, None, :]      # [B][Hq][1][d]
    kt = torch.from_numpy(k.astype(np.float64))                     # [B][Hq][N][d]
    vt = torch.from_numpy(v.astype(np.float64))
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)
    return o[:, :, 0, :].numpy()


def _expand_groups(x, G):
    return np.repeat(x, G, axis=1)


@pytest.mark.parametrize("G,n_tail,s", [(1, 0, 0.5), (1, 32, 0.7), (4, 32, 0.7), (2, 5, 0.5),
                                        (8, 1, 0.9)])
def test_attention_equals_torch_sdpa_on_zero_filled_caches(G, n_tail, s):
    B, Hkv, N, d = 2, 2, 150, 128
    K, V = synth.make_kv(B, Hkv, N, d, seed=7)
    KL, VL = synth.make_tail(B, Hkv, n_tail, d, seed=7)
    q = synth.make_q(B, Hkv * G, d, seed=7)
    ek, ev = oracle.compress(K, s), oracle.compress(V, s)
    got = oracle.sparse_decode_attention(q, ek, ev, KL, VL)
    kc = oracle.decompress(ek).view(np.float16)
    vc = oracle.decompress(ev).view(np.float16)
    kall = _expand_groups(np.concatenate([kc, KL], axis=2), G)
    vall = _expand_groups(np.concatenate([vc, VL], axis=2), G)
    ref = _sdpa64(q, kall, vall)
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-13)
    # the scale argument is honoured
    got2 = oracle.sparse_decode_attention(q, ek, ev, KL, VL, scale=0.05)
    assert np.allclose(got2, _sdpa64(q, kall, vall, scale=0.05), rtol=1e-12, atol=1e-13)


def test_zero_sparsity_equals_dense_attention():
    B, Hkv, G, N, d = 1, 4, 2, 200, 128
    K, V = synth.make_kv(B, Hkv, N, d, seed=8)
    q = synth.make_q(B, Hkv * G, d, seed=8)
    got = oracle.sparse_decode_attention(q, oracle.compress(K, 0.0), oracle.compress(V, 0.0))
    ref = _sdpa64(q, _expand_groups(K, G), _expand_groups(V, G))
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-13)


def test_zero_query_gives_the_mean_value_row():
    B, H, N, d = 1, 2, 64, 128
    K, V = synth.make_kv(B, H, N, d, seed=9)
    KL, VL = synth.make_tail(B, H, 7, d, seed=9)
    ek, ev = oracle.compress(K, 0.5), oracle.compress(V, 0.7)
    q = np.zeros((B, H, d), dtype=np.float16)
    got = oracle.sparse_decode_attention(q, ek, ev, KL, VL)
    vc = oracle.decompress(ev).view(np.float16).astype(np.float64)
    want = np.concatenate([vc, VL.astype(np.float64)], axis=2).mean(axis=2)
    assert np.allclose(got, want, rtol=1e-12, atol=1e-14)


def test_dominant_score_selects_one_value_row():
    """If one score beats every other by >= 40, its weight is 1 - O(e^-40)."""
    B, H, N, d = 1, 1, 40, 64
    rng = np.random.default_rng(10)
    K = (rng.standard_normal((B, H, N, d)) * 0.01).astype(np.float16)
    V = rng.standard_normal((B, H, N, d)).astype(np.float16)
    star = 17
    K[0, 0, star, :] = 4.0
    q = np.full((B, H, d), 4.0, dtype=np.float16)   # score(star) = 16*64/8 = 128
    ek, ev = oracle.compress(K, 0.0), oracle.compress(V, 0.0)
    got = oracle.sparse_decode_attention(q, ek, ev)
    assert np.allclose(got[0, 0], V[0, 0, star].astype(np.float64), rtol=0, atol=1e-15)


def test_moving_tokens_between_compressed_and_window_changes_nothing():
    """Algorithm 1 only concatenates the compressed and window scores, so at
    sparsity 0 the split point between the two parts does not matter."""
    B, H, N, d = 1, 2, 96, 128
    K, V = synth.make_kv(B, H, N, d, seed=11)
    q = synth.make_q(B, H, d, seed=11)
    ref = oracle.sparse_decode_attention(q, oracle.compress(K, 0.0), oracle.compress(V, 0.0))
    for split in (0, 1, 31, 64, 95):
        ek = oracle.compress(np.ascontiguousarray(K[:, :, :split]), 0.0)
        ev = oracle.compress(np.ascontiguousarray(V[:, :, :split]), 0.0)
        got = oracle.sparse_decode_attention(q, ek, ev, np.ascontiguousarray(K[:, :, split:]),
                                             np.ascontiguousarray(V[:, :, split:]))
        assert np.allclose(got, ref, rtol=1e-13, atol=1e-15), split
