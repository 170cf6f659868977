"""Pins of the window-lifecycle oracle (oracle/window.py).

The lifecycle is fixed by token positions (Sec. 3): after t arrivals an entry's
window holds its last min(t, W) tokens and every earlier token is compressed.
The pins check the oracle's bookkeeping against that closed form, with tokens
that carry their own arrival index, and its attention against the same
attention computed without the compressed format.
"""
import numpy as np
import pytest

import oracle
from oracle.window import WindowOracle

D = 64


def _indexed_tokens(B, H, n, d, rng, base=0):
    """Random fp16 tokens whose channel 0 holds the arrival index (exact in fp16)."""
    x = rng.standard_normal((B, H, n, d)).astype(np.float16)
    x[..., 0] = (base + np.arange(n, dtype=np.float64)).astype(np.float16)[None, None, :]
    return x


@pytest.mark.parametrize("W", [1, 2, 8, 32])
def test_counts_follow_the_closed_form(W):
    rng = np.random.default_rng(1)
    B, H = 4, 2
    seq = [0, 3, W, W + 5]
    n_max = max(seq) or 1
    xk = _indexed_tokens(B, H, n_max, D, rng)
    xv = _indexed_tokens(B, H, n_max, D, rng)
    o = WindowOracle(B, H, D, W, 0.5, 0.7)
    o.prefill(xk, xv, seq)
    arrived = list(seq)
    masks = [None, [1, 0, 1, 1], [0, 0, 0, 1], None, [1, 1, 0, 0]]
    for s in range(12):
        act = masks[s % len(masks)]
        kn = rng.standard_normal((B, H, D)).astype(np.float16)
        o.step(kn, kn, act)
        for b in range(B):
            if act is None or act[b]:
                arrived[b] += 1
        for b in range(B):
            t = arrived[b]
            assert o.arrived(b) == t
            assert o.window_len(b) == min(t, W)
            assert o.n_comp(b) == max(0, t - W)


def test_window_holds_the_last_tokens_oldest_first():
    rng = np.random.default_rng(2)
    B, H, W = 3, 2, 4
    seq = [2, 4, 9]
    xk = _indexed_tokens(B, H, 9, D, rng)
    o = WindowOracle(B, H, D, W, 0.5, 0.5)
    o.prefill(xk, xk, seq)
    for s in range(6):
        kn = rng.standard_normal((B, H, D)).astype(np.float16)
        kn[..., 0] = np.float16(100 + s)
        o.step(kn, kn, [1, s % 2, 1])
    for b in range(B):
        wk, _ = o.window(b)
        idx = wk[0, :, 0].view(np.float16).astype(np.float64)
        # arrival order of entry b: prefill indices, then the steps it took part in
        order = list(range(seq[b])) + [100 + s for s in range(6) if b != 1 or s % 2]
        assert list(idx) == order[-min(len(order), W):]


def test_hand_example_window_of_two():
    """W = 2, three tokens a, b, c: a is compressed, the window is [b, c]."""
    o = WindowOracle(1, 1, D, 2, 0.5, 0.5)
    toks = [np.full((1, 1, D), v, dtype=np.float16) for v in (1.0, 2.0, 3.0)]
    for t in toks:
        o.step(t, t)
    assert o.n_comp(0) == 1 and o.window_len(0) == 2
    wk, _ = o.window(0)
    assert wk[0, :, 0].view(np.float16).tolist() == [2.0, 3.0]
    enc_k, _ = o.compressed(0)
    # All channels of token a tie at 1.0: the lower half of the channels is kept.
    assert int(enc_k["bitmaps"][0, 0, 0, 0]) == (1 << 32) - 1


@pytest.mark.parametrize("G", [1, 4])
def test_attention_equals_the_direct_computation(G):
    rng = np.random.default_rng(3)
    B, H, W = 3, 2, 5
    seq = [1, 5, 11]
    xk = _indexed_tokens(B, H, 11, D, rng)
    xv = rng.standard_normal((B, H, 11, D)).astype(np.float16)
    o = WindowOracle(B, H, D, W, 0.5, 0.7)
    o.prefill(xk, xv, seq)
    for s in range(4):
        o.step(rng.standard_normal((B, H, D)).astype(np.float16),
               rng.standard_normal((B, H, D)).astype(np.float16), [1, 1, s % 2])
    q = rng.standard_normal((B, H * G, D)).astype(np.float16)
    for b in range(B):
        a = o.attention(q[b], b)
        r = o.attention_direct(q[b], b)
        np.testing.assert_allclose(a, r, rtol=0, atol=1e-12)


# ---- output-aware keys in the lifecycle (Sec. 2) -------------------------------------------
def _output_aware_run(W, S, G, inactive=()):
    rng = np.random.default_rng(40 + W + G)
    B, H, d = 1, 2, 64
    o = WindowOracle(B, H, d, W, 0.5, 0.5, output_aware_keys=True)
    x0 = rng.standard_normal((B, H, 1, d)).astype(np.float16)
    o.prefill(x0, x0, [1])
    keys, qs = [x0[0, :, 0]], []
    for s in range(S):
        k = rng.standard_normal((B, H, d)).astype(np.float16)
        act = [0 if s in inactive else 1]
        o.step(k, rng.standard_normal((B, H, d)).astype(np.float16), act)
        if act[0]:
            keys.append(k[0])
        q = rng.standard_normal((B, H * G, d)).astype(np.float16)
        before = {j: o.key_weights(0, j).copy() for j in range(o.arrived(0))}
        o.accumulate_key_weights(q, act)
        if act[0]:
            qs.append(q[0])
        else:   # a step the entry sits out leaves every weight as it was
            assert all(np.array_equal(o.key_weights(0, j), w) for j, w in before.items())
    return o, np.stack(keys, axis=1)[None], np.stack(qs, axis=1)[None]


@pytest.mark.parametrize("W,G", [(32, 1), (48, 2)])
def test_output_aware_key_weights_equal_the_bulk_lookahead(W, G):
    """A continuously active entry whose prompt is one token: key j >= 1 arrives in
    step j - 1 and leaves with the lookahead weights of the queries of steps
    j - 1 .. j + 30 (query_lookahead with L = 32, bit for bit); the prompt token
    missed its own (prefill) query and carries those of steps 0 .. 30. The
    compressed keys equal compress_variant's output-aware compression with those
    weights, bit for bit."""
    S = 90
    o, K, Q = _output_aware_run(W, S, G)
    H, d = 2, 64
    look = oracle.query_lookahead(Q, H, 32)
    n = o.n_comp(0)
    assert n == S + 1 - W
    want_w = np.stack([oracle.query_lookahead(Q, H, 31)[0, :, 0]] +
                      [look[0, :, j - 1] for j in range(1, n)], axis=1)       # [H][n][d]
    for j in range(n):
        assert np.array_equal(o.key_weights(0, j), want_w[:, j]), j
    want = oracle.compress_variant(K[:, :, :n], "output_aware", k=oracle.keep_count(d, 0.5),
                                   weights=want_w[None])
    got, _ = o.compressed(0)
    for key in ("bitmaps", "offsets", "stream_len"):
        assert np.array_equal(got[key], want[key]), key
    L = int(want["stream_len"][0, 0])
    assert np.array_equal(got["values"][:, :, :L], want["values"][:, :, :L])
    # and the weights matter: some key differs from its magnitude pruning
    mag = oracle.compress(K[:, :, :n], 0.5)
    assert not np.array_equal(got["bitmaps"], mag["bitmaps"])


def test_output_aware_key_pins_reject_planted_mistakes(monkeypatch):
    """The lookahead pin fails when the window oracle gathers one step too few or
    adds the query heads of a step in the other order."""
    import oracle.window as ow

    def weights_match(W=32, G=2):
        o, K, Q = _output_aware_run(W, 90, G)
        look = oracle.query_lookahead(Q, 2, 32)
        return all(np.array_equal(o.key_weights(0, j), look[0, :, j - 1]) for j in range(1, o.n_comp(0)))

    assert weights_match()
    monkeypatch.setattr(ow, "KEY_WEIGHT_STEPS", 31)
    assert not weights_match()
    monkeypatch.undo()

    def reversed_heads(self, q, active=None):
        qa = np.abs(np.asarray(q).view(np.float16).astype(np.float32))
        G = qa.shape[1] // self.H
        for b in range(self.B):
            n, L = self.n_comp(b), self.window_len(b)
            for p in range(max(0, L - ow.KEY_WEIGHT_STEPS), L):
                w = self.key_w[b].setdefault(n + p, np.zeros((self.H, self.d), dtype=np.float32))
                for h in range(self.H):
                    for g in reversed(range(G)):
                        w[h] = w[h] + qa[b, h * G + g]

    monkeypatch.setattr(ow.WindowOracle, "accumulate_key_weights", reversed_heads)
    assert not weights_match()


@pytest.mark.parametrize("G", [1, 2])
def test_output_aware_keys_of_a_paused_entry_gather_only_its_own_queries(G):
    """An entry that sits steps out gathers no query in them: a key that leaves
    carries exactly the lookahead weights (L = 32, bit for bit) of the entry's own
    query sequence -- the queries of the steps it was active in -- from the step
    the key arrived in; the prompt token the 31 first ones. Its caches equal the
    output-aware compression with those weights."""
    W, S, H, d = 32, 90, 2, 64
    pause = set(range(10, 15)) | {40, 41, 60}
    o, K, Q = _output_aware_run(W, S, G, inactive=pause)
    n = o.n_comp(0)
    assert n == S - len(pause) + 1 - W
    look = oracle.query_lookahead(Q, H, 32)           # over the entry's own queries
    want_w = np.stack([oracle.query_lookahead(Q, H, 31)[0, :, 0]] +
                      [look[0, :, j - 1] for j in range(1, n)], axis=1)
    for j in range(n):
        assert np.array_equal(o.key_weights(0, j), want_w[:, j]), j
    want = oracle.compress_variant(K[:, :, :n], "output_aware", k=oracle.keep_count(d, 0.5),
                                   weights=want_w[None])
    got, _ = o.compressed(0)
    for key in ("bitmaps", "offsets", "stream_len"):
        assert np.array_equal(got[key], want[key]), key


# ---- the grouped lifecycle (per-channel value pruning in groups of 32) -------------------
from oracle.window import GroupedWindowOracle  # noqa: E402


@pytest.mark.parametrize("W", [64, 96])
def test_grouped_counts_follow_the_closed_form(W):
    """n_comp stays whole groups; a prefill of n leaves 1..32 tokens dense; a
    window graduates 32 tokens exactly when it holds W before a push."""
    rng = np.random.default_rng(11)
    B, H = 4, 1
    seq = [1, 32, 33, 100]
    xk = _indexed_tokens(B, H, 100, D, rng)
    o = GroupedWindowOracle(B, H, D, W, 0.5, 0.7)
    o.prefill(xk, xk, seq)
    comp = [(n - 1) // 32 * 32 for n in seq]
    lens = [n - c for n, c in zip(seq, comp)]
    assert [o.n_comp(b) for b in range(B)] == comp
    assert all(1 <= L <= 32 for L in lens)
    for s in range(3 * W):
        act = [1, s % 2, 1, s % 3 != 0]
        t = rng.standard_normal((B, H, D)).astype(np.float16)
        o.step(t, t, act)
        for b in range(B):
            if act[b]:
                if lens[b] == W:
                    comp[b] += 32
                    lens[b] -= 32
                lens[b] += 1
            assert o.n_comp(b) == comp[b] and o.window_len(b) == lens[b]
            assert comp[b] % 32 == 0 and 1 <= lens[b] <= W


def test_grouped_window_tokens_and_groups():
    rng = np.random.default_rng(12)
    B, H, W = 1, 2, 64
    xk = _indexed_tokens(B, H, 40, D, rng)
    o = GroupedWindowOracle(B, H, D, W, 0.5, 0.7)
    o.prefill(xk, xk, [40])
    for s in range(60):
        t = rng.standard_normal((B, H, D)).astype(np.float16)
        t[..., 0] = np.float16(40 + s)
        o.step(t, t)
    wk, _ = o.window(0)
    idx = wk[0, :, 0].view(np.float16).astype(np.float64)
    assert list(idx) == list(range(64, 100))      # 100 arrivals, 64 compressed
    # Every compressed group keeps exactly keep_count(32, 0.7) = 10 tokens per channel.
    _, ev = o.compressed(0)
    bm = ev["bitmaps"][0, 0]
    for g in range(2):
        for c in range(D):
            kept = sum((int(bm[g * 32 + j, 0]) >> c) & 1 for j in range(32))
            assert kept == 10


@pytest.mark.parametrize("G", [1, 4])
def test_grouped_attention_and_scores_against_direct_computation(G):
    rng = np.random.default_rng(13 + G)
    B, H, W = 2, 2, 64
    xk = rng.standard_normal((B, H, 70, D)).astype(np.float16)
    xv = rng.standard_normal((B, H, 70, D)).astype(np.float16)
    o = GroupedWindowOracle(B, H, D, W, 0.5, 0.7)
    o.prefill(xk, xv, [70, 9])
    for s in range(40):
        w = {b: np.abs(rng.standard_normal((H, 32))).astype(np.float32) for b in range(B)}
        o.step(rng.standard_normal((B, H, D)).astype(np.float16),
               rng.standard_normal((B, H, D)).astype(np.float16), None, w)
    q = rng.standard_normal((B, H * G, D)).astype(np.float16)
    for b in range(B):
        # attention over the compressed format = dense attention over the decoded tokens
        ek, ev = o.compressed(b)
        wk, wv = o.window(b)
        kk = np.concatenate([oracle.decompress(ek)[0], wk], axis=1)
        vv = np.concatenate([oracle.decompress(ev)[0], wv], axis=1)
        direct = oracle.decode_attention(q[b][None], kk[None], vv[None])[0]
        np.testing.assert_allclose(o.attention(q[b], b), direct, rtol=0, atol=1e-12)
        # score increments: numpy softmax of the scores over all tokens, young window tokens
        inc = o.score_increments(q[b], b)
        L, n = o.window_len(b), o.n_comp(b)
        for h in range(H):
            keys = kk[h].view(np.float16).astype(np.float64)
            tot = np.zeros(n + L)
            for g in range(G):
                s = keys @ q[b, h * G + g].astype(np.float64) / np.sqrt(D)
                e = np.exp(s - s.max())
                tot += e / e.sum()
            want = np.where(np.arange(L) >= L - 32, tot[n:], 0.0)
            np.testing.assert_allclose(inc[h], want, rtol=1e-12, atol=1e-15)
