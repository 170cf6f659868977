"""The bulk compressor's bounded look-back wait, forced to give up from the host.

mustafar_prune_compress_bounded with max_polls = 0 lets no chunk but the first
of a stream read its predecessors' totals, so every stream of more than one
chunk gives up; every kernel still finishes. Checked: the call reports the
give-up in the workspace's status word, the streams are poisoned
(stream_len = MUSTAFAR_STREAM_POISONED), later compressions and appends write
nothing to them, and the decode attention treats their compressed part as
empty (the output equals the oracle's attention over the window alone), while
a healthy cache in the same calls stays bit-exact against the oracle. A
one-chunk compression under the same bound gives up nowhere.
"""
import numpy as np
import pytest

import oracle
import paper_2505_22913_amd as mf
from paper_2505_22913_amd import synth
from tests.gpu_common import ATTN_TOL, all_pairs, announce, attn_error, compare_format, read_cache, to_dev

pytestmark = pytest.mark.gpu


def test_give_up_poisons_the_stream_and_later_calls_skip_it():
    import torch
    announce("look-back give-up forced from the host")
    B, H, d, N, n_more, Nd = 1, 4, 128, 5000, 64, 32
    K, V = synth.make_kv(B, H, N + n_more + 1, d, seed=91)
    KL, VL = synth.make_tail(B, H, Nd, d, seed=91)
    q = synth.make_q(B, H, d, seed=91)
    Kc = mf.CompressedCache(B, H, d, 0.5, N + n_more + 1)
    Vc = mf.CompressedCache(B, H, d, 0.7, N + n_more + 1)
    ws = torch.empty(mf.mustafar_compress_workspace_bytes(B, H, N), dtype=torch.uint8, device="cuda")
    mf.mustafar_prune_compress_bounded(Kc, to_dev(np.ascontiguousarray(K[:, :, :N])), 0, ws=ws)
    assert mf.compress_status(ws) != 0
    lens = read_cache(Kc)["stream_len"]
    assert (lens == mf.STREAM_POISONED).all(), lens
    # the value cache, compressed with the default bound through the same workspace
    mf.mustafar_prune_compress(Vc, to_dev(np.ascontiguousarray(V[:, :, :N])), ws=ws)
    assert mf.compress_status(ws) == 0

    # later calls: a bulk compression and an append write nothing to the poisoned streams
    mf.mustafar_prune_compress(Kc, to_dev(np.ascontiguousarray(K[:, :, N:N + n_more])), ws=ws)
    mf.mustafar_prune_compress(Vc, to_dev(np.ascontiguousarray(V[:, :, N:N + n_more])), ws=ws)
    n = N + n_more
    mf.mustafar_append_kv(Kc, Vc, to_dev(np.ascontiguousarray(K[:, :, n])),
                          to_dev(np.ascontiguousarray(V[:, :, n])))
    n += 1
    got_k, got_v = read_cache(Kc), read_cache(Vc)
    assert (got_k["stream_len"] == mf.STREAM_POISONED).all()
    compare_format(got_v, oracle.compress(np.ascontiguousarray(V[:, :, :n]), 0.7), n, all_pairs(B, H))

    # attention: the poisoned key streams contribute nothing, the window does
    out = mf.mustafar_sparse_decode_attn(to_dev(q), Kc, Vc, to_dev(KL), to_dev(VL))
    empty = np.zeros((B, H, 0, d), np.float16)
    ref = oracle.decode_attention(q, empty, empty, KL, VL)
    err = attn_error(out.cpu().numpy(), ref)
    announce(f"look-back give-up: window-only attention error {err:.2e}")
    assert err <= ATTN_TOL
    # with no window either, every part of the softmax is empty: the output is 0
    out0 = mf.mustafar_sparse_decode_attn(to_dev(q), Kc, Vc, None, None)
    assert not out0.cpu().numpy().any()


@pytest.mark.parametrize("d", [64, 128])
def test_one_chunk_needs_no_look_back(d):
    import torch
    announce(f"look-back bound 0 on one chunk d={d}")
    B, H, N = 2, 3, 64
    K, _ = synth.make_kv(B, H, N, d, seed=92)
    Kc = mf.CompressedCache(B, H, d, 0.5, N)
    ws = torch.empty(mf.mustafar_compress_workspace_bytes(B, H, N), dtype=torch.uint8, device="cuda")
    mf.mustafar_prune_compress_bounded(Kc, to_dev(K), 0, ws=ws)
    assert mf.compress_status(ws) == 0
    compare_format(read_cache(Kc), oracle.compress(K, 0.5), N, all_pairs(B, H))
