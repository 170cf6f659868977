"""Parity at the benchmark workloads' full sizes, in the launch configuration the
benchmark times: inputs drawn on the GPU by synth.make_kv_torch, the library's
default split count, a 32-token dense window.

Per workload:
  * every stream: each token keeps exactly n_keep channels, and the tile
    offsets are the exclusive prefix sum of the padded tile counts ending at
    stream_len (Sec. 3 and Sec. 4.3) -- checked on the GPU with integer ops;
  * sampled streams (all of them for the smaller workloads): bitmaps, offsets,
    stream_len and packed values equal the oracle's, bit for bit, on the same
    dense tokens copied back to the host;
  * attention output of the sampled (batch, kv-head) groups within the 2e-3
    tolerance of the oracle's Algorithm 1.
The 128K-context workload also runs its 256 decode steps (append the token that
leaves the 32-token window, attend) with a sliding window, and is checked after
the first and the last step.
"""
import numpy as np
import pytest

import oracle
import paper_2505_22913_amd as mf
from paper_2505_22913_amd import synth
from tests.gpu_common import ATTN_TOL, announce, attn_error, compare_format

pytestmark = pytest.mark.gpu

SEED = 11
WINDOW = synth.WINDOW


def _popc_table(device):
    import torch
    t = torch.tensor([bin(i).count("1") for i in range(256)], dtype=torch.uint8, device=device)
    return t


def _check_properties(cache, n_tokens: int) -> None:
    """All streams: n_keep bits per token; offsets = exclusive scan of pad8(popcount)."""
    import torch
    B, H, d = cache.shape
    T = d // 64
    bm = cache.bitmaps[:, :, :n_tokens].contiguous()                  # int64 [B][H][n][T]
    cnt = _popc_table(bm.device)[bm.view(torch.uint8).long()].view(B, H, n_tokens, T, 8)
    cnt = cnt.to(torch.int32).sum(-1)                                 # [B][H][n][T]
    per_token = cnt.sum(-1)
    bad = (per_token != cache.n_keep).nonzero()
    assert bad.numel() == 0, f"token with {int(per_token[tuple(bad[0])])} kept at {bad[0].tolist()}"
    padded = ((cnt + 7) // 8) * 8
    flat = padded.view(B, H, n_tokens * T).to(torch.int64)
    excl = torch.cumsum(flat, dim=-1) - flat
    offs = cache.offsets[:, :, :n_tokens].contiguous().view(B, H, n_tokens * T).to(torch.int64)
    assert torch.equal(offs, excl), "tile offsets are not the exclusive scan of padded counts"
    total = flat.sum(-1)
    assert torch.equal(cache.stream_len.to(torch.int64), total), "stream_len mismatch"


def _read_streams(cache, picks, n_tokens: int) -> dict:
    """Host copies of the sampled streams, shaped [S][1][...] like the oracle's output."""
    import torch
    torch.cuda.synchronize()
    B, H, _ = cache.shape
    bi = [p // H for p in picks]
    hi = [p % H for p in picks]
    lens = cache.stream_len[bi, hi].cpu().numpy().view(np.uint32)
    vmax = int(lens.max()) if len(lens) else 0
    return {
        "bitmaps": cache.bitmaps[bi, hi, :n_tokens].cpu().numpy().view(np.uint64)[:, None],
        "offsets": cache.offsets[bi, hi, :n_tokens].cpu().numpy().view(np.uint32)[:, None],
        "values": cache.values[bi, hi, :vmax].cpu().numpy().view(np.uint16)[:, None],
        "stream_len": lens[:, None],
    }


def _host(x, picks, H):
    return np.stack([x[p // H, p % H].cpu().numpy() for p in picks])[:, None]


def _picks(BH: int, n: int):
    if n >= BH:
        return list(range(BH))
    return sorted(set(np.linspace(0, BH - 1, n).round().astype(int).tolist()))


def _run_workload(name: str, n_sample: int):
    import torch
    w = synth.WORKLOADS[name]
    announce(f"full-size {name}")
    steps = w.decode_steps
    K, V = synth.make_kv_torch(w.B, w.Hkv, w.N + WINDOW + steps, w.d, seed=SEED)
    gq = torch.Generator(device="cuda")
    gq.manual_seed(SEED)
    q = torch.randn((w.B, w.Hq, w.d), generator=gq, device="cuda").half()
    cap = w.N + steps
    Kc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sK, cap)
    Vc = mf.CompressedCache(w.B, w.Hkv, w.d, w.sV, cap)
    mf.mustafar_prune_compress(Kc, K[:, :, :w.N].contiguous())
    mf.mustafar_prune_compress(Vc, V[:, :, :w.N].contiguous())
    BH = w.B * w.Hkv
    picks = _picks(BH, n_sample)
    G = w.G

    def attend_and_check(n_comp: int, label: str):
        kt = K[:, :, n_comp:n_comp + WINDOW].contiguous()
        vt = V[:, :, n_comp:n_comp + WINDOW].contiguous()
        out = mf.mustafar_sparse_decode_attn(q, Kc, Vc, kt, vt)
        torch.cuda.synchronize()
        Ks = _host(K[:, :, :n_comp], picks, w.Hkv)
        Vs = _host(V[:, :, :n_comp], picks, w.Hkv)
        ek = oracle.compress(Ks, w.sK, threads=16)
        ev = oracle.compress(Vs, w.sV, threads=16)
        compare_format(_read_streams(Kc, picks, n_comp), ek, n_comp,
                       [((i, 0), (i, 0)) for i in range(len(picks))])
        compare_format(_read_streams(Vc, picks, n_comp), ev, n_comp,
                       [((i, 0), (i, 0)) for i in range(len(picks))])
        qs = np.stack([q[p // w.Hkv, (p % w.Hkv) * G:(p % w.Hkv + 1) * G].cpu().numpy()
                       for p in picks])
        ref = oracle.sparse_decode_attention(qs, ek, ev, _host(kt, picks, w.Hkv),
                                             _host(vt, picks, w.Hkv), threads=16)
        got = np.stack([out[p // w.Hkv, (p % w.Hkv) * G:(p % w.Hkv + 1) * G].cpu().numpy()
                        for p in picks])
        err = attn_error(got, ref)
        announce(f"{name} {label}: {len(picks)} of {BH} streams, attention error {err:.2e}")
        assert err <= ATTN_TOL, (label, err)

    _check_properties(Kc, w.N)
    _check_properties(Vc, w.N)
    if steps == 0:
        attend_and_check(w.N, "prefill")
        return
    # Decode: at step s the token N+s leaves the window [N+s, N+s+32) and is
    # appended; attention then covers compressed [0, N+s+1) and window [N+s+1, N+s+33).
    for s in range(steps):
        mf.mustafar_append(Kc, K[:, :, w.N + s].contiguous())
        mf.mustafar_append(Vc, V[:, :, w.N + s].contiguous())
        if s == 0:
            attend_and_check(w.N + 1, "after decode step 1")
        else:
            kt = K[:, :, w.N + s + 1:w.N + s + 1 + WINDOW].contiguous()
            vt = V[:, :, w.N + s + 1:w.N + s + 1 + WINDOW].contiguous()
            mf.mustafar_sparse_decode_attn(q, Kc, Vc, kt, vt)
    _check_properties(Kc, w.N + steps)
    _check_properties(Vc, w.N + steps)
    attend_and_check(w.N + steps, f"after decode step {steps}")


@pytest.mark.parametrize("name,n_sample", [
    ("tiny-mha-1k", 10 ** 9),
    ("llama2-7b-4k", 10 ** 9),
    ("llama3-8b-gqa-16k", 10 ** 9),
    ("mha-b16-32k", 6),
    ("gqa-128k-decode", 10 ** 9),
])
def test_full_size_workload(name, n_sample):
    _run_workload(name, n_sample)
