"""Oracle of the dense local window's lifecycle (Sec. 3; Algorithm 1's dense part).

TEST INFRASTRUCTURE, like the rest of ``oracle/``: only the test suite may use it,
and it shares no code with the GPU library.

The method keeps the most recent tokens of every stream dense and unpruned;
a token that leaves that window is pruned and compressed, and decode attention
runs over the compressed tokens plus the window (Algorithm 1). With a window of
W tokens this fixes, for a batch entry that has received t tokens so far:

* the window holds its last min(t, W) tokens;
* every earlier token is in the compressed caches, in arrival order, pruned
  exactly as a one-shot compression of those tokens would prune them.

This oracle keeps the plain arrival history of every batch entry and derives
both parts from it on demand; how a GPU stores the window (a ring of W slots)
is not modelled. Batch entries are independent and may have received different
numbers of tokens (ragged batches: prompts of different lengths, entries that
skip decode steps).
"""
from __future__ import annotations

import numpy as np

from . import compress, decode_attention, prune_token, sparse_decode_attention


class WindowOracle:
    """Token history of a batch of B entries with H kv-heads of dimension d.

    ``sk`` and ``sv`` are the K and V sparsities, ``W`` the window length.
    """

    def __init__(self, B: int, H: int, d: int, W: int, sk: float, sv: float):
        self.B, self.H, self.d, self.W = B, H, d, W
        self.sk, self.sv = sk, sv
        # hist_k[b] is a list of [H][d] uint16 arrays, one per arrived token.
        self.hist_k = [[] for _ in range(B)]
        self.hist_v = [[] for _ in range(B)]

    # ---- arrivals ------------------------------------------------------------------------
    def prefill(self, xk, xv, seq_len) -> None:
        """Entry b receives the first seq_len[b] tokens of xk, xv [B][H][n_max][d]."""
        xk = np.asarray(xk).view(np.uint16)
        xv = np.asarray(xv).view(np.uint16)
        for b in range(self.B):
            for j in range(int(seq_len[b])):
                self.hist_k[b].append(np.array(xk[b, :, j]))
                self.hist_v[b].append(np.array(xv[b, :, j]))

    def step(self, k_new, v_new, active=None) -> None:
        """Active entries receive one token each: k_new, v_new [B][H][d]."""
        k_new = np.asarray(k_new).view(np.uint16)
        v_new = np.asarray(v_new).view(np.uint16)
        for b in range(self.B):
            if active is None or active[b]:
                self.hist_k[b].append(np.array(k_new[b]))
                self.hist_v[b].append(np.array(v_new[b]))

    # ---- derived state -------------------------------------------------------------------
    def arrived(self, b: int) -> int:
        return len(self.hist_k[b])

    def window_len(self, b: int) -> int:
        return min(self.arrived(b), self.W)

    def n_comp(self, b: int) -> int:
        return self.arrived(b) - self.window_len(b)

    def _tokens(self, hist, b: int, lo: int, hi: int) -> np.ndarray:
        """Tokens lo..hi-1 of entry b as [H][hi-lo][d] uint16."""
        if hi <= lo:
            return np.zeros((self.H, 0, self.d), dtype=np.uint16)
        return np.stack(hist[b][lo:hi], axis=1)

    def window(self, b: int):
        """(K, V) of entry b's window, oldest first: [H][len][d] uint16 each."""
        lo, hi = self.n_comp(b), self.arrived(b)
        return self._tokens(self.hist_k, b, lo, hi), self._tokens(self.hist_v, b, lo, hi)

    def compressed(self, b: int):
        """(K, V) compressed streams of entry b in the oracle's format (B = 1)."""
        n = self.n_comp(b)
        k = self._tokens(self.hist_k, b, 0, n)[None]
        v = self._tokens(self.hist_v, b, 0, n)[None]
        return compress(k, self.sk), compress(v, self.sv)

    # ---- attention -----------------------------------------------------------------------
    def attention(self, q, b: int, scale: float = 0.0) -> np.ndarray:
        """Algorithm 1 for entry b: q [Hq][d] over its compressed tokens and window.
        float64 [Hq][d]."""
        q = np.asarray(q).view(np.uint16)[None]
        enc_k, enc_v = self.compressed(b)
        wk, wv = self.window(b)
        return sparse_decode_attention(q, enc_k, enc_v, wk[None], wv[None], scale)[0]

    def attention_direct(self, q, b: int, scale: float = 0.0) -> np.ndarray:
        """The same attention without the compressed format: the tokens before the
        window are pruned with ``prune_token`` (zeros where dropped) and every
        token enters ``decode_attention`` as a dense row."""
        q = np.asarray(q).view(np.uint16)[None]
        n = self.n_comp(b)
        kk = np.ascontiguousarray(self._tokens(self.hist_k, b, 0, self.arrived(b)))
        vv = np.ascontiguousarray(self._tokens(self.hist_v, b, 0, self.arrived(b)))
        kk, vv = kk.copy(), vv.copy()
        kkeep = _keep_count(self.d, self.sk)
        vkeep = _keep_count(self.d, self.sv)
        for h in range(self.H):
            for j in range(n):
                kk[h, j][~prune_token(kk[h, j], kkeep)] = 0
                vv[h, j][~prune_token(vv[h, j], vkeep)] = 0
        return decode_attention(q, kk[None], vv[None], None, None, scale)[0]


def _keep_count(d: int, sparsity: float) -> int:
    from . import keep_count
    return keep_count(d, sparsity)
