"""GPU parity of the dense-window lifecycle (mustafar_window_prefill / _step /
_decode_attn) against oracle/window.py, on ragged batches.

Entries start from prompts of different lengths (empty, shorter than the window,
exactly one window, longer) and some skip decode steps (the active mask), so the
entries' compressed and window lengths differ throughout. At checkpoints:

* len, n_comp equal the oracle's counts, and the ring read from head in order
  equals the oracle's window, bit for bit;
* every stream's compressed format equals the oracle's one-shot compression of
  the entry's tokens before its window, bit for bit (Sec. 3; the incremental
  graduation must reproduce it exactly);
* the attention output of every entry is within 2e-3 of the oracle's Algorithm 1;
* with output-aware keys, the window's key weights equal the oracle's bit for bit.
"""
import numpy as np
import pytest

import paper_2505_22913_amd as mf
from oracle.window import WindowOracle
from tests.gpu_common import ATTN_TOL, announce, attn_error, compare_format

pytestmark = pytest.mark.gpu


def _check_state(o, win, Kc, Vc, B, H, W):
    import torch
    torch.cuda.synchronize()
    lens = win.len.cpu().numpy()
    heads = win.head.cpu().numpy()
    ncomp = win.n_comp.cpu().numpy()
    rk = win.k.cpu().numpy().view(np.uint16)
    rv = win.v.cpu().numpy().view(np.uint16)
    got_k = {"bitmaps": Kc.bitmaps.cpu().numpy().view(np.uint64),
             "offsets": Kc.offsets.cpu().numpy().view(np.uint32),
             "values": Kc.values.cpu().numpy().view(np.uint16),
             "stream_len": Kc.stream_len.cpu().numpy().view(np.uint32)}
    got_v = {"bitmaps": Vc.bitmaps.cpu().numpy().view(np.uint64),
             "offsets": Vc.offsets.cpu().numpy().view(np.uint32),
             "values": Vc.values.cpu().numpy().view(np.uint16),
             "stream_len": Vc.stream_len.cpu().numpy().view(np.uint32)}
    assert Kc.n_tokens >= int(ncomp.max()) and win.max_len >= int(lens.max())
    for b in range(B):
        assert lens[b] == o.window_len(b), (b, lens[b], o.window_len(b))
        assert ncomp[b] == o.n_comp(b), (b, ncomp[b], o.n_comp(b))
        assert 0 <= heads[b] < W
        wk, wv = o.window(b)
        slots = [(heads[b] + i) % W for i in range(lens[b])]
        assert np.array_equal(rk[b][:, slots], wk), f"window K of entry {b}"
        assert np.array_equal(rv[b][:, slots], wv), f"window V of entry {b}"
        n = int(ncomp[b])
        if n > 0:
            ek, ev = o.compressed(b)
            pairs = [((b, h), (0, h)) for h in range(H)]
            compare_format(got_k, ek, n, pairs)
            compare_format(got_v, ev, n, pairs)


def _check_attention(o, win, Kc, Vc, q, B, G, label):
    out = mf.mustafar_window_decode_attn(q, Kc, Vc, win).cpu().numpy()
    qn = q.cpu().numpy()
    err = max(attn_error(out[b], o.attention(qn[b], b)) for b in range(B))
    announce(f"window {label}: attention error {err:.2e}")
    assert err <= ATTN_TOL, (label, err)


@pytest.mark.parametrize("W,G,sk,sv", [(32, 1, 0.5, 0.7), (8, 2, 0.7, 0.7), (5, 4, 0.5, 0.5)])
def test_window_lifecycle_ragged(W, G, sk, sv):
    import torch
    announce(f"window lifecycle W={W} G={G}")
    rng = np.random.default_rng(100 + W)
    B, H, d = 5, 2, 128
    seq = [0, 3, W, W + 7, 3 * W + 2]
    n_max = max(seq)
    steps = 2 * W + 6
    xk = rng.standard_normal((B, H, n_max, d)).astype(np.float16)
    xk[:, :, :, 5] *= 10  # an outlier channel
    xv = rng.standard_normal((B, H, n_max, d)).astype(np.float16)
    cap = n_max + steps
    Kc = mf.CompressedCache(B, H, d, sk, cap)
    Vc = mf.CompressedCache(B, H, d, sv, cap)
    win = mf.DenseWindow(B, H, d, W)
    mf.mustafar_window_prefill(win, Kc, Vc, torch.from_numpy(xk).cuda(), torch.from_numpy(xv).cuda(),
                               seq)
    o = WindowOracle(B, H, d, W, sk, sv)
    o.prefill(xk, xv, seq)
    _check_state(o, win, Kc, Vc, B, H, W)
    q = torch.from_numpy(rng.standard_normal((B, H * G, d)).astype(np.float16)).cuda()
    for s in range(steps):
        act = np.array([1, (s % 3) != 1, 1, (s % 2) == 0, 1], dtype=np.int32)
        if s == 0:
            act[:] = 1
        kn = rng.standard_normal((B, H, d)).astype(np.float16)
        vn = rng.standard_normal((B, H, d)).astype(np.float16)
        mf.mustafar_window_step(win, Kc, Vc, torch.from_numpy(kn).cuda(), torch.from_numpy(vn).cuda(),
                                torch.from_numpy(act).cuda())
        o.step(kn, vn, act)
        if s in (0, W - 1, steps - 1):
            _check_state(o, win, Kc, Vc, B, H, W)
            _check_attention(o, win, Kc, Vc, q, B, G, f"W={W} G={G} step {s + 1}")


def test_window_step_without_mask_and_long_prefill_splits():
    """Every entry active, a prefill long enough for several split-K segments."""
    import torch
    announce("window lifecycle long prefill")
    rng = np.random.default_rng(7)
    B, H, d, W, G = 2, 2, 128, 32, 1
    seq = [700, 300]
    xk = rng.standard_normal((B, H, 700, d)).astype(np.float16)
    xv = rng.standard_normal((B, H, 700, d)).astype(np.float16)
    Kc = mf.CompressedCache(B, H, d, 0.5, 800)
    Vc = mf.CompressedCache(B, H, d, 0.7, 800)
    win = mf.DenseWindow(B, H, d, W)
    mf.mustafar_window_prefill(win, Kc, Vc, torch.from_numpy(xk).cuda(), torch.from_numpy(xv).cuda(),
                               seq)
    o = WindowOracle(B, H, d, W, 0.5, 0.7)
    o.prefill(xk, xv, seq)
    q = torch.from_numpy(rng.standard_normal((B, H * G, d)).astype(np.float16)).cuda()
    for s in range(3):
        kn = rng.standard_normal((B, H, d)).astype(np.float16)
        vn = rng.standard_normal((B, H, d)).astype(np.float16)
        mf.mustafar_window_step(win, Kc, Vc, torch.from_numpy(kn).cuda(), torch.from_numpy(vn).cuda())
        o.step(kn, vn)
    _check_state(o, win, Kc, Vc, B, H, W)
    out = mf.mustafar_window_decode_attn(q, Kc, Vc, win, n_splits=4).cpu().numpy()
    err = max(attn_error(out[b], o.attention(q.cpu().numpy()[b], b)) for b in range(B))
    announce(f"window long prefill: attention error {err:.2e}")
    assert err <= ATTN_TOL


@pytest.mark.parametrize("W,G,d", [(32, 1, 128), (48, 4, 128), (40, 2, 64), (32, 8, 256)])
def test_window_lifecycle_output_aware_keys(W, G, d):
    """The lifecycle with output-aware keys (Sec. 2): mustafar_window_key_weights
    after every step's attention, mustafar_window_step_weighted for the step. The
    key weights of every window slot equal the oracle's, bit for bit (fp32 adds in
    the same order), and so do the caches; attention within the tolerance."""
    import torch
    announce(f"window lifecycle output-aware keys W={W} G={G} d={d}")
    rng = np.random.default_rng(300 + W + G + d)
    B, H = 3, 2
    seq = [1, 20, W + 30]
    n_max = max(seq)
    steps = W + 50
    xk = rng.standard_normal((B, H, n_max, d)).astype(np.float16)
    xv = rng.standard_normal((B, H, n_max, d)).astype(np.float16)
    cap = n_max + steps
    Kc = mf.CompressedCache(B, H, d, 0.5, cap)
    Vc = mf.CompressedCache(B, H, d, 0.7, cap)
    win = mf.DenseWindow(B, H, d, W)
    kacc = torch.zeros((B, H, W, d), dtype=torch.float32, device="cuda")
    mf.mustafar_window_prefill(win, Kc, Vc, torch.from_numpy(xk).cuda(), torch.from_numpy(xv).cuda(),
                               seq)
    o = WindowOracle(B, H, d, W, 0.5, 0.7, output_aware_keys=True)
    o.prefill(xk, xv, seq)
    graduated = 0
    for s in range(steps):
        act = np.array([1, (s % 4) != 2, 1], dtype=np.int32)
        kn = rng.standard_normal((B, H, d)).astype(np.float16)
        vn = rng.standard_normal((B, H, d)).astype(np.float16)
        mf.mustafar_window_step_weighted(win, Kc, Vc, torch.from_numpy(kn).cuda(),
                                         torch.from_numpy(vn).cuda(), kacc,
                                         torch.from_numpy(act).cuda())
        o.step(kn, vn, act)
        q = torch.from_numpy(rng.standard_normal((B, H * G, d)).astype(np.float16)).cuda()
        if s % 10 == 9 or s == steps - 1:
            _check_state(o, win, Kc, Vc, B, H, W)
            _check_attention(o, win, Kc, Vc, q, B, G, f"output-aware keys W={W} G={G} step {s + 1}")
        before = kacc.clone() if not act.all() else None
        mf.mustafar_window_key_weights(q, win, kacc, active=torch.from_numpy(act).cuda())
        o.accumulate_key_weights(q.cpu().numpy(), act)
        if before is not None:   # an entry that sits the step out gathers nothing
            idle = torch.from_numpy(act == 0).cuda()
            assert torch.equal(kacc[idle], before[idle]), s
        if s % 10 == 9 or s == steps - 1:
            torch.cuda.synchronize()
            a = kacc.cpu().numpy()
            lens, heads = win.len.cpu().numpy(), win.head.cpu().numpy()
            for b in range(B):
                n = o.n_comp(b)
                for p in range(int(lens[b])):
                    slot = (int(heads[b]) + p) % W
                    assert np.array_equal(a[b, :, slot], o.key_weights(b, n + p)), (s, b, p)
            graduated = sum(o.n_comp(b) - o.n_prefill[b] for b in range(B))
    assert graduated >= 40
