"""The decode entry point that allocates nothing (mustafar_sparse_decode_attn_static).

Two calls in a row through the C ABI, the second with a smaller input, each
against mustafar_sparse_decode_attn with a caller workspace and the same split
count: the same kernels, so the outputs are equal bit for bit; both within the
2e-3 bound of the oracle. A request whose partials exceed the static buffer is
refused on the host (ESCRATCH) before anything is launched.
"""
import numpy as np
import pytest

import oracle
import paper_2505_22913_amd as mf
from paper_2505_22913_amd import synth
from tests.gpu_common import ATTN_TOL, announce, attn_error, to_dev


@pytest.mark.gpu
def test_static_scratch_decode_equals_the_workspace_call():
    import torch
    cases = [(2, 4, 4, 3000, 32, 0.7, 0.7, 0), (1, 2, 1, 500, 7, 0.5, 0.7, 3)]   # larger, then smaller
    for B, Hkv, G, N, Nd, sK, sV, splits in cases:
        announce(f"static-scratch decode B={B} Hkv={Hkv} G={G} N={N} Nd={Nd} splits={splits}")
        K, V = synth.make_kv(B, Hkv, N, 128, seed=N + G)
        KL, VL = synth.make_tail(B, Hkv, Nd, 128, seed=N + G)
        q = synth.make_q(B, Hkv * G, 128, seed=N + G)
        Kc = mf.CompressedCache(B, Hkv, 128, sK, N)
        Vc = mf.CompressedCache(B, Hkv, 128, sV, N)
        mf.mustafar_prune_compress(Kc, to_dev(K))
        mf.mustafar_prune_compress(Vc, to_dev(V))
        qd, kl, vl = to_dev(q), to_dev(KL), to_dev(VL)
        got = mf.mustafar_sparse_decode_attn_static(qd, Kc, Vc, kl, vl, n_splits=splits)
        want = mf.mustafar_sparse_decode_attn(qd, Kc, Vc, kl, vl, n_splits=splits)
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int16), want.view(torch.int16))
        ref = oracle.sparse_decode_attention(q, oracle.compress(K, sK), oracle.compress(V, sV), KL, VL)
        assert attn_error(got.cpu().numpy(), ref) <= ATTN_TOL


@pytest.mark.gpu
def test_static_scratch_refuses_what_does_not_fit():
    Kc = mf.CompressedCache(16, 32, 128, 0.5, 64)
    Vc = mf.CompressedCache(16, 32, 128, 0.5, 64)
    Kc.desc.n_tokens = Vc.desc.n_tokens = 64
    import torch
    q = torch.zeros((16, 256, 128), dtype=torch.float16, device="cuda")
    need = mf.mustafar_attn_workspace_bytes(16, 256, 32, 128, 64, 2000)
    assert need > mf.STATIC_SCRATCH_BYTES
    with pytest.raises(mf.MustafarError) as e:
        mf.mustafar_sparse_decode_attn_static(q, Kc, Vc, n_splits=2000)
    assert e.value.status == mf.ESCRATCH
