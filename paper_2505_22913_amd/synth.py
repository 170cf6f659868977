"""Seeded synthetic inputs for the MUSTAFAR hot path (shared by tests and bench).

This module generates data only; it holds none of the method's arithmetic.

The paper drives its kernels with the KV caches of Llama-2-7B / Llama-3-8B on
LongBench prompts (Sec. 4) and RULER at 64K (Appendix A.3). Neither weights nor
datasets are used here. The synthetic caches copy the structure the paper
reports instead (Sec. 2, Fig. "kv_visualization"): the Key cache has a few
outlier channels of much larger magnitude, persistent across tokens, while the
Value cache has no preferred direction.

Recipe (all fp32 draws, then cast to fp16 with round-to-nearest-even):
  K[b, h, j, c] ~ N(0, 1), times 10 on 4 outlier channels per kv-head h
                  (the same channels for every batch entry and token)
  V[b, h, j, c] ~ N(0, 1)
  q[b, h, c]    ~ N(0, 1)
  window tokens (dense tail) drawn like K and V.

Two generators with identical distributions:
  * numpy (``np.random.PCG64`` seeded by ``SeedSequence([seed, tensor, b, h])``)
    so that any (batch, head) slice can be regenerated on its own -- used for
    sizes the CPU oracle handles;
  * torch on the GPU (Philox, one seeded ``torch.Generator`` per tensor) for the
    multi-GB workloads. Its bits differ from numpy's; full-size parity checks
    copy sampled slices of the generated device tensors back to the host.
Outlier channels always come from numpy so both generators agree on them.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

N_OUTLIERS = 4
OUTLIER_SCALE = 10.0
WINDOW = 32  # dense local window in tokens (Sec. 2 and Sec. 3)

# tensor ids for the seed sequences
_K, _V, _Q, _KT, _VT, _OUT = 0, 1, 2, 3, 4, 9


@dataclass(frozen=True)
class Workload:
    """One synthetic decode workload (sizes of a Llama-class attention layer)."""
    name: str
    B: int
    Hq: int
    Hkv: int
    N: int            # compressed context tokens per stream
    d: int
    sK: float         # Key-cache sparsity
    sV: float         # Value-cache sparsity
    n_tail: int = WINDOW
    decode_steps: int = 0  # append+attend steps after the prefill compression

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def dense_kv_bytes(self) -> int:
        return 2 * 2 * self.B * self.Hkv * self.N * self.d


WORKLOADS = {
    "tiny-mha-1k": Workload("tiny-mha-1k", B=1, Hq=8, Hkv=8, N=1024, d=128, sK=0.5, sV=0.5),
    "llama2-7b-4k": Workload("llama2-7b-4k", B=1, Hq=32, Hkv=32, N=4096, d=128, sK=0.5, sV=0.5),
    "llama3-8b-gqa-16k": Workload("llama3-8b-gqa-16k", B=4, Hq=32, Hkv=8, N=16384, d=128,
                                  sK=0.7, sV=0.7),
    "mha-b16-32k": Workload("mha-b16-32k", B=16, Hq=32, Hkv=32, N=32768, d=128, sK=0.5, sV=0.7),
    "gqa-128k-decode": Workload("gqa-128k-decode", B=1, Hq=32, Hkv=8, N=131072, d=128,
                                sK=0.7, sV=0.7, decode_steps=256),
    # Group-size points around the Llama-3-8B shape (32 streams of 16K tokens,
    # 70/70) with 2 and 8 query heads per kv-head, for comparing the kernels.
    "gqa2-b4-16k": Workload("gqa2-b4-16k", B=4, Hq=16, Hkv=8, N=16384, d=128, sK=0.7, sV=0.7),
    "gqa8-b4-16k": Workload("gqa8-b4-16k", B=4, Hq=64, Hkv=8, N=16384, d=128, sK=0.7, sV=0.7),
}


def _rng(seed: int, *keys: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, *keys])))


def outlier_channels(seed: int, h: int, d: int) -> np.ndarray:
    """The N_OUTLIERS distinct Key outlier channels of kv-head h."""
    return np.sort(_rng(seed, _OUT, h).choice(d, N_OUTLIERS, replace=False))


def key_slice(seed: int, b: int, h: int, n: int, d: int, tensor: int = _K) -> np.ndarray:
    """K[b, h] (or the K window when tensor=_KT) as fp16 [n][d]."""
    x = _rng(seed, tensor, b, h).standard_normal((n, d), dtype=np.float32)
    x[:, outlier_channels(seed, h, d)] *= OUTLIER_SCALE
    return x.astype(np.float16)


def value_slice(seed: int, b: int, h: int, n: int, d: int, tensor: int = _V) -> np.ndarray:
    """V[b, h] (or the V window when tensor=_VT) as fp16 [n][d]."""
    return _rng(seed, tensor, b, h).standard_normal((n, d), dtype=np.float32).astype(np.float16)


def make_kv(B: int, H: int, N: int, d: int, seed: int):
    """numpy K, V fp16 [B][H][N][d]."""
    K = np.empty((B, H, N, d), dtype=np.float16)
    V = np.empty((B, H, N, d), dtype=np.float16)
    for b in range(B):
        for h in range(H):
            K[b, h] = key_slice(seed, b, h, N, d)
            V[b, h] = value_slice(seed, b, h, N, d)
    return K, V


def make_tail(B: int, H: int, n_tail: int, d: int, seed: int):
    """numpy dense window K_L, V_L fp16 [B][H][n_tail][d]."""
    K = np.empty((B, H, n_tail, d), dtype=np.float16)
    V = np.empty((B, H, n_tail, d), dtype=np.float16)
    for b in range(B):
        for h in range(H):
            K[b, h] = key_slice(seed, b, h, n_tail, d, tensor=_KT)
            V[b, h] = value_slice(seed, b, h, n_tail, d, tensor=_VT)
    return K, V


def make_q(B: int, Hq: int, d: int, seed: int) -> np.ndarray:
    """numpy q fp16 [B][Hq][d]."""
    return _rng(seed, _Q).standard_normal((B, Hq, d), dtype=np.float32).astype(np.float16)


def make_kv_torch(B: int, H: int, N: int, d: int, seed: int, device="cuda", chunk_tokens=4096):
    """Device K, V fp16 [B][H][N][d] drawn with torch's GPU generator (same recipe)."""
    import torch

    K = torch.empty((B, H, N, d), dtype=torch.float16, device=device)
    V = torch.empty((B, H, N, d), dtype=torch.float16, device=device)
    gk = torch.Generator(device=device)
    gk.manual_seed(seed * 1000003 + 11)
    gv = torch.Generator(device=device)
    gv.manual_seed(seed * 1000003 + 17)
    scale = torch.ones((H, 1, d), dtype=torch.float32, device=device)
    for h in range(H):
        scale[h, 0, torch.as_tensor(outlier_channels(seed, h, d), device=device)] = OUTLIER_SCALE
    for b in range(B):
        for j0 in range(0, N, chunk_tokens):
            n = min(chunk_tokens, N - j0)
            kb = torch.randn((H, n, d), generator=gk, device=device, dtype=torch.float32)
            K[b, :, j0:j0 + n] = (kb * scale).to(torch.float16)
            vb = torch.randn((H, n, d), generator=gv, device=device, dtype=torch.float32)
            V[b, :, j0:j0 + n] = vb.to(torch.float16)
    return K, V
