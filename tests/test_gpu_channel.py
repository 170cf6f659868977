"""GPU parity of per-channel value pruning in groups of 32 tokens (Sec. 2,
value-cache study) against the oracle:

* bulk compression of per-channel caches, magnitude and output-aware (given
  token weights), bit for bit, over several calls;
* decode attention over per-channel value caches (walk and matrix-core
  kernels, every head size) within the 2e-3 tolerance;
* the grouped window lifecycle on ragged batches: the attention scores
  accumulated per window slot against the oracle's probabilities (within
  2e-3 relative), and the caches after every graduation against the oracle
  run with its OWN accumulated scores (float64 sums of its probabilities,
  rounded to fp32 when a group leaves). Keys, offsets and packing are bit for
  bit; a value channel's selection may differ from the oracle's only by a
  boundary pair, two tokens whose oracle keys |v| x A both lie within the score
  tolerance of the channel's threshold (either choice is correct at that
  precision). Such pairs are counted and reported; the GPU's packing of its
  selection is compared bit for bit with the oracle's encoder applied to it,
  and the attention with the oracle's attention over that selection.
"""
import numpy as np
import pytest

import oracle
import paper_2505_22913_amd as mf
from oracle.window import GroupedWindowOracle
from tests.gpu_common import ATTN_TOL, all_pairs, announce, attn_error, compare_format, read_cache

pytestmark = pytest.mark.gpu

SCORE_RTOL = 2e-3
SCORE_ATOL = 1e-7


def _dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _tokens(rng, shape, ties=False):
    if ties:
        mags = np.array([0.0, 2.0 ** -24, 0.5, 1.0, 1.0, 2.0], dtype=np.float32)
        return (rng.choice(mags, size=shape) * rng.choice([-1.0, 1.0], size=shape)).astype(np.float16)
    return rng.standard_normal(shape).astype(np.float16)


@pytest.mark.parametrize("d,ties", [(64, False), (128, False), (128, True), (256, True)])
def test_channel_magnitude_bit_exact(d, ties):
    announce(f"per-channel magnitude d={d} ties={ties}")
    rng = np.random.default_rng(d + 7 * ties)
    B, H, N = 2, 3, 96
    x = _tokens(rng, (B, H, N + 32, d), ties)
    c = mf.CompressedCache(B, H, d, 0.7, N + 32, grouped=True)
    assert c.group_keep == 10
    mf.mustafar_prune_compress(c, _dev(x[:, :, :N]))
    mf.mustafar_prune_compress_ex(c, _dev(x[:, :, N:]), mode=mf.PRUNE_CHANNEL)
    want = oracle.compress_grouped(x, 0.7)
    compare_format(read_cache(c), want, N + 32, all_pairs(B, H))


@pytest.mark.parametrize("d,s", [(128, 0.7), (256, 0.5), (64, 0.3)])
def test_channel_output_aware_bit_exact(d, s):
    announce(f"per-channel output-aware d={d} s={s}")
    rng = np.random.default_rng(31 + d)
    B, H, N = 2, 2, 64
    x = _tokens(rng, (B, H, N, d))
    w = (np.abs(rng.standard_normal((B, H, N))) * 0.05).astype(np.float32)
    w[:, :, 5] = 0.0                       # a token no query attended
    w[:, :, 9] = w[:, :, 10]               # equal weights
    c = mf.CompressedCache(B, H, d, s, N, grouped=True)
    mf.mustafar_prune_compress_ex(c, _dev(x), mode=mf.PRUNE_CHANNEL_OUTPUT_AWARE, weights=_dev(w))
    want = oracle.compress_grouped(x, s, weights=w)
    compare_format(read_cache(c), want, N, all_pairs(B, H))


@pytest.mark.parametrize("G,d", [(1, 128), (4, 128), (1, 256), (2, 64)])
def test_attention_over_grouped_values(G, d):
    import torch
    announce(f"attention over per-channel values G={G} d={d}")
    rng = np.random.default_rng(40 + G + d)
    B, Hkv, N, Nd = 2, 2, 320, 32
    k = _tokens(rng, (B, Hkv, N + Nd, d))
    v = _tokens(rng, (B, Hkv, N + Nd, d))
    Kc = mf.CompressedCache(B, Hkv, d, 0.5, N)
    Vc = mf.CompressedCache(B, Hkv, d, 0.7, N, grouped=True)
    mf.mustafar_prune_compress(Kc, _dev(k[:, :, :N]))
    mf.mustafar_prune_compress(Vc, _dev(v[:, :, :N]))
    q = _tokens(rng, (B, Hkv * G, d))
    for splits in (0, 3):
        out = mf.mustafar_sparse_decode_attn(_dev(q), Kc, Vc, _dev(k[:, :, N:]), _dev(v[:, :, N:]),
                                             n_splits=splits)
        torch.cuda.synchronize()
        ref = oracle.sparse_decode_attention(q, oracle.compress(k[:, :, :N], 0.5),
                                             oracle.compress_grouped(v[:, :, :N], 0.7),
                                             k[:, :, N:], v[:, :, N:])
        err = attn_error(out.cpu().numpy(), ref)
        announce(f"per-channel values G={G} d={d} splits={splits}: error {err:.2e}")
        assert err <= ATTN_TOL


@pytest.mark.parametrize("G,d", [(1, 128), (4, 128), (4, 64), (2, 256), (1, 64)])
def test_attention_over_grouped_values_clustered(G, d):
    """Every channel keeps the same 10 tokens of each group of 32, its first ten
    (their values dominate), so those tokens are dense and the other 22 empty: the
    most values any block of a kernel can meet (a 16-token block holds all of a
    group's kept values). The attention kernels stage such blocks whole."""
    import torch
    announce(f"attention over clustered per-channel values G={G} d={d}")
    rng = np.random.default_rng(60 + G + d)
    B, Hkv, N, Nd = 1, 2, 256, 32
    k = _tokens(rng, (B, Hkv, N + Nd, d))
    v = (rng.standard_normal((B, Hkv, N + Nd, d)) * 0.01).astype(np.float16)
    for g0 in range(0, N, 32):
        v[:, :, g0:g0 + 10] = (8.0 + 2.0 * np.abs(rng.standard_normal((B, Hkv, 10, d)))).astype(np.float16)
    Kc = mf.CompressedCache(B, Hkv, d, 0.5, N)
    Vc = mf.CompressedCache(B, Hkv, d, 0.7, N, grouped=True)
    mf.mustafar_prune_compress(Kc, _dev(k[:, :, :N]))
    mf.mustafar_prune_compress(Vc, _dev(v[:, :, :N]))
    want_v = oracle.compress_grouped(v[:, :, :N], 0.7)
    bm = want_v["bitmaps"][0, 0, :32]
    assert all(int(x) == (1 << 64) - 1 for x in bm[:10].reshape(-1))   # the first ten are dense
    assert not bm[10:].any()
    compare_format(read_cache(Vc), want_v, N, all_pairs(B, Hkv))
    q = _tokens(rng, (B, Hkv * G, d))
    for splits in (0, 1):
        out = mf.mustafar_sparse_decode_attn(_dev(q), Kc, Vc, _dev(k[:, :, N:]), _dev(v[:, :, N:]),
                                             n_splits=splits)
        torch.cuda.synchronize()
        ref = oracle.sparse_decode_attention(q, oracle.compress(k[:, :, :N], 0.5), want_v,
                                             k[:, :, N:], v[:, :, N:])
        err = attn_error(out.cpu().numpy(), ref)
        announce(f"clustered per-channel values G={G} d={d} splits={splits}: error {err:.2e}")
        assert err <= ATTN_TOL


def _state(win, acc):
    import torch
    torch.cuda.synchronize()
    return (win.len.cpu().numpy(), win.head.cpu().numpy(), win.n_comp.cpu().numpy(),
            None if acc is None else acc.cpu().numpy())


def _value_selection(got_bm, want_bm, v, w, gk, n, H):
    """Checks the GPU's per-channel value selection of tokens [0, n) of one entry
    against the oracle's. got_bm, want_bm: u64 [H][n][T]; v: fp16 bits [H][n][d];
    w: per group float32 [H][32] weights of the oracle, or None (magnitude). Returns
    (the GPU's keep mask [H][n][d], the number of boundary pairs)."""
    T = got_bm.shape[-1]
    d = 64 * T
    bits = lambda bm: ((bm[..., None] >> np.arange(64, dtype=np.uint64)) & 1).astype(bool).reshape(  # noqa: E731
        bm.shape[0], bm.shape[1], d)
    keep_g, keep_w = bits(got_bm), bits(want_bm)
    flips = 0
    for g in range(n // 32):
        sl = slice(32 * g, 32 * g + 32)
        if np.array_equal(keep_g[:, sl], keep_w[:, sl]):
            continue
        mag = np.abs(v[:, sl].view(np.float16).astype(np.float32))          # [H][32][d]
        assert w[g] is not None, f"magnitude group {g} differs"
        key = (mag * np.asarray(w[g], dtype=np.float32)[:, :, None]).astype(np.float32)
        for h in range(H):
            for c in np.nonzero((keep_g[h, sl] != keep_w[h, sl]).any(axis=0))[0]:
                kg, kw = keep_g[h, sl, c], keep_w[h, sl, c]
                assert kg.sum() == kw.sum() == gk, (g, h, c)
                theta = np.sort(key[h, :, c])[::-1][gk - 1]           # the oracle's threshold
                tol = 2 * (SCORE_RTOL * theta + SCORE_ATOL * mag[h, :, c].max())
                moved = np.nonzero(kg != kw)[0]
                bad = [int(t) for t in moved if abs(float(key[h, t, c]) - float(theta)) > tol]
                assert not bad, f"group {g} head {h} channel {c}: tokens {bad} are not at the threshold"
                flips += int((kg & ~kw).sum())
    return keep_g, flips


@pytest.mark.parametrize("G,scored", [(1, True), (4, True), (1, False)])
def test_grouped_window_lifecycle(G, scored):
    import torch
    announce(f"grouped lifecycle G={G} scored={scored}")
    rng = np.random.default_rng(50 + G + 2 * scored)
    B, H, d, W = 3, 2, 128, 64
    seq = [1, 40, 100]
    steps = 100
    xk = _tokens(rng, (B, H, 100, d))
    xv = _tokens(rng, (B, H, 100, d))
    cap = 100 + steps
    Kc = mf.CompressedCache(B, H, d, 0.5, cap)
    Vc = mf.CompressedCache(B, H, d, 0.7, cap, grouped=True)
    win = mf.DenseWindow(B, H, d, W)
    acc = torch.zeros((B, H, W), dtype=torch.float32, device="cuda")
    mf.mustafar_window_prefill(win, Kc, Vc, _dev(xk), _dev(xv), seq)
    o = GroupedWindowOracle(B, H, d, W, 0.5, 0.7)
    o.prefill(xk, xv, seq)
    A = [dict() for _ in range(B)]          # oracle scores per token index, float64 [H]
    gw = [[None] * (o.n_comp(b) // 32) for b in range(B)]   # the oracle's weights per group
    graduations = flips = 0
    for s in range(steps):
        act = np.array([1, (s % 3) != 1, 1], dtype=np.int32)
        lens, heads, ncomp, a_now = _state(win, acc if scored else None)
        weights = {}
        for b in range(B):
            assert lens[b] == o.window_len(b) and ncomp[b] == o.n_comp(b), (s, b)
            if act[b] and lens[b] == W:
                graduations += 1
                n = o.n_comp(b)
                weights[b] = (np.stack([A[b].get(n + u, np.zeros(H)) for u in range(32)], axis=1)
                              .astype(np.float32) if scored else None)
                gw[b].append(weights[b])
        kn = _tokens(rng, (B, H, d))
        vn = _tokens(rng, (B, H, d))
        mf.mustafar_window_step_grouped(win, Kc, Vc, _dev(kn), _dev(vn), _dev(act),
                                        acc if scored else None)
        o.step(kn, vn, act, weights if scored else None)
        q = _tokens(rng, (B, H * G, d))
        if scored:
            out = mf.mustafar_window_decode_attn_scores(_dev(q), Kc, Vc, win, acc, active=_dev(act))
            for b in range(B):
                if not act[b]:
                    continue    # an entry that sits the step out gathers no score
                inc = o.score_increments(q[b], b)
                n = o.n_comp(b)
                for p in range(o.window_len(b)):
                    A[b][n + p] = A[b].get(n + p, 0.0) + inc[:, p]
        else:
            out = mf.mustafar_window_decode_attn(_dev(q), Kc, Vc, win)
        if s % 10 == 9 or s == steps - 1:
            lens, heads, ncomp, a_now = _state(win, acc if scored else None)
            got_k, got_v = read_cache(Kc), read_cache(Vc)
            outn = out.cpu().numpy()
            for b in range(B):
                n = int(ncomp[b])
                ek, ev = o.compressed(b)
                if n > 0:
                    pairs = [((b, h), (0, h)) for h in range(H)]
                    compare_format(got_k, ek, n, pairs)
                    vtok = np.stack(o.hist_v[b][:n], axis=1)                  # [H][n][d] bits
                    keep, nf = _value_selection(got_v["bitmaps"][b, :, :n], ev["bitmaps"][0, :, :n],
                                                vtok, gw[b], Vc.group_keep, n, H)
                    flips += nf
                    if nf:
                        ev = oracle.encode(vtok[None], keep[None])
                    compare_format(got_v, ev, n, pairs)
                wk, wv = o.window(b)
                ref = oracle.sparse_decode_attention(q[b][None].view(np.uint16), ek, ev, wk[None],
                                                     wv[None])[0]
                err = attn_error(outn[b], ref)
                assert err <= ATTN_TOL, (s, b, err)
                if scored:
                    for p in range(int(lens[b])):
                        slot = (heads[b] + p) % W
                        want = A[b].get(n + p, np.zeros(H))
                        np.testing.assert_allclose(a_now[b][:, slot], want, rtol=SCORE_RTOL,
                                                   atol=SCORE_ATOL, err_msg=f"step {s} entry {b} pos {p}")
            announce(f"grouped lifecycle G={G} step {s + 1}: n_comp {list(ncomp)}, "
                     f"boundary pairs so far {flips}")
    assert graduations >= 3
    announce(f"grouped lifecycle G={G} scored={scored}: {graduations} graduations, "
             f"{flips} value channels chose the other token of a boundary pair")
