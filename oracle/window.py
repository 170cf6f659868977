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

from . import (GROUP, attention_probs, compress, decode_attention, decompress, encode,
               keep_count, prune_channel_group, prune_token, prune_token_scored,
               sparse_decode_attention)

# Output-aware keys: a key's weights sum the query at its position and the 31
# after it (Sec. 2).
KEY_WEIGHT_STEPS = 32


class WindowOracle:
    """Token history of a batch of B entries with H kv-heads of dimension d.

    ``sk`` and ``sv`` are the K and V sparsities, ``W`` the window length.

    With ``output_aware_keys`` the keys that leave the window are pruned by the
    output-aware score of Sec. 2 instead of by magnitude: every call of
    ``accumulate_key_weights`` (one per decode step, with that step's queries
    and activity mask) adds, for every entry active in the step, |q| of each
    query head of a kv-head, one head after the other in float32, to the
    channel weights of each of the entry's newest 32 window tokens, and a key
    leaves with channels ranked by fl32(|k_c| * w_c). An entry that sits a step
    out has no query of its own in it and gathers nothing. A token that leaves
    the window thus carries the sum over the queries of its own entry in the
    step it arrived and the entry's 31 active steps after it, as
    ``query_lookahead`` adds them over that entry's query sequence. The tokens
    a prefill compresses at once have no decode queries and are pruned by
    magnitude.
    """

    def __init__(self, B: int, H: int, d: int, W: int, sk: float, sv: float,
                 output_aware_keys: bool = False):
        self.B, self.H, self.d, self.W = B, H, d, W
        self.sk, self.sv = sk, sv
        # hist_k[b] is a list of [H][d] uint16 arrays, one per arrived token.
        self.hist_k = [[] for _ in range(B)]
        self.hist_v = [[] for _ in range(B)]
        self.output_aware_keys = output_aware_keys
        self.key_w = [dict() for _ in range(B)]   # token index -> float32 [H][d]
        self.n_prefill = [0] * B                  # tokens the prefill compressed

    # ---- arrivals ------------------------------------------------------------------------
    def prefill(self, xk, xv, seq_len) -> None:
        """Entry b receives the first seq_len[b] tokens of xk, xv [B][H][n_max][d]."""
        xk = np.asarray(xk).view(np.uint16)
        xv = np.asarray(xv).view(np.uint16)
        for b in range(self.B):
            for j in range(int(seq_len[b])):
                self.hist_k[b].append(np.array(xk[b, :, j]))
                self.hist_v[b].append(np.array(xv[b, :, j]))
            self.n_prefill[b] = self.n_comp(b)

    def accumulate_key_weights(self, q, active=None) -> None:
        """One decode step's queries q [B][Hq][d] (fp16) into the key weights of the
        newest KEY_WEIGHT_STEPS window tokens of every entry active in the step."""
        qa = np.abs(np.asarray(q).view(np.float16).astype(np.float32))
        G = qa.shape[1] // self.H
        for b in range(self.B):
            if active is not None and not active[b]:
                continue
            n, L = self.n_comp(b), self.window_len(b)
            for p in range(max(0, L - KEY_WEIGHT_STEPS), L):
                w = self.key_w[b].setdefault(n + p, np.zeros((self.H, self.d), dtype=np.float32))
                for h in range(self.H):
                    for g in range(G):
                        w[h] = w[h] + qa[b, h * G + g]

    def key_weights(self, b: int, j: int) -> np.ndarray:
        """float32 [H][d] weights of token j of entry b (zeros if it has none)."""
        return self.key_w[b].get(j, np.zeros((self.H, self.d), dtype=np.float32))

    def _key_keep(self, b: int, j: int, h: int) -> np.ndarray:
        x = self.hist_k[b][j][h]
        k = _keep_count(self.d, self.sk)
        if self.output_aware_keys and j >= self.n_prefill[b]:
            return prune_token_scored(x, self.key_weights(b, j)[h], k)
        return prune_token(x, k)

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
        if not self.output_aware_keys:
            return compress(k, self.sk), compress(v, self.sv)
        keep = np.zeros((1, self.H, n, self.d), dtype=bool)
        for j in range(n):
            for h in range(self.H):
                keep[0, h, j] = self._key_keep(b, j, h)
        return encode(k, keep), compress(v, self.sv)

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
        vkeep = _keep_count(self.d, self.sv)
        for h in range(self.H):
            for j in range(n):
                kk[h, j][~self._key_keep(b, j, h)] = 0
                vv[h, j][~prune_token(vv[h, j], vkeep)] = 0
        return decode_attention(q, kk[None], vv[None], None, None, scale)[0]


def _keep_count(d: int, sparsity: float) -> int:
    from . import keep_count
    return keep_count(d, sparsity)


class GroupedWindowOracle:
    """The window lifecycle of per-channel value pruning in groups of 32 tokens
    (Sec. 2, value-cache study), for B entries with H kv-heads of dimension d.

    An entry's compressed prefix is always whole groups. A prefill of n tokens
    compresses the first 32 * floor((n - 1) / 32) (values by per-channel
    magnitude) and keeps the rest, 1 to 32 tokens, dense. A decode step first
    lets a full window (W tokens) hand its oldest 32 tokens over as one group,
    then appends the new token. Keys are pruned per token (magnitude, sk);
    values per channel within each group (keep_count(32, sv) tokens per channel),
    by magnitude or, when the step is given that group's token weights, by the
    fp32 key |v| * w_j. The window a token sits in is thus at least 32 steps
    old when it leaves, and the output-aware weight of a token is the sum of
    the attention probabilities it received (over the query heads of its
    kv-head) in the step it arrived and the 31 after: ``score_increments``
    gives a step's contributions.
    """

    def __init__(self, B: int, H: int, d: int, W: int, sk: float, sv: float):
        assert W >= 2 * GROUP and W % GROUP == 0
        self.B, self.H, self.d, self.W = B, H, d, W
        self.sk, self.sv = sk, sv
        self.hist_k = [[] for _ in range(B)]
        self.hist_v = [[] for _ in range(B)]
        self.ncomp = [0] * B
        # per entry, one entry per compressed group: None (magnitude) or float32 [H][32]
        self.group_w = [[] for _ in range(B)]

    def prefill(self, xk, xv, seq_len) -> None:
        xk = np.asarray(xk).view(np.uint16)
        xv = np.asarray(xv).view(np.uint16)
        for b in range(self.B):
            n = int(seq_len[b])
            for j in range(n):
                self.hist_k[b].append(np.array(xk[b, :, j]))
                self.hist_v[b].append(np.array(xv[b, :, j]))
            self.ncomp[b] = 0 if n == 0 else (n - 1) // GROUP * GROUP
            self.group_w[b] = [None] * (self.ncomp[b] // GROUP)

    def step(self, k_new, v_new, active=None, weights=None) -> None:
        """weights: None, or a dict {b: float32 [H][32] or None} with the token
        weights of the group entry b hands over in this step (if any)."""
        k_new = np.asarray(k_new).view(np.uint16)
        v_new = np.asarray(v_new).view(np.uint16)
        for b in range(self.B):
            if active is not None and not active[b]:
                continue
            if self.window_len(b) == self.W:
                self.ncomp[b] += GROUP
                w = None if weights is None else weights.get(b)
                self.group_w[b].append(None if w is None else np.asarray(w, dtype=np.float32))
            self.hist_k[b].append(np.array(k_new[b]))
            self.hist_v[b].append(np.array(v_new[b]))

    def arrived(self, b: int) -> int:
        return len(self.hist_k[b])

    def n_comp(self, b: int) -> int:
        return self.ncomp[b]

    def window_len(self, b: int) -> int:
        return self.arrived(b) - self.ncomp[b]

    def _tokens(self, hist, b: int, lo: int, hi: int) -> np.ndarray:
        if hi <= lo:
            return np.zeros((self.H, 0, self.d), dtype=np.uint16)
        return np.stack(hist[b][lo:hi], axis=1)

    def window(self, b: int):
        lo, hi = self.ncomp[b], self.arrived(b)
        return self._tokens(self.hist_k, b, lo, hi), self._tokens(self.hist_v, b, lo, hi)

    def compressed(self, b: int):
        """(K, V) compressed streams of entry b in the oracle's format (B = 1)."""
        n = self.ncomp[b]
        k = self._tokens(self.hist_k, b, 0, n)[None]
        v = self._tokens(self.hist_v, b, 0, n)[None]
        enc_k = compress(k, self.sk)
        gk = keep_count(GROUP, self.sv)
        keep = np.zeros((1, self.H, n, self.d), dtype=bool)
        for g, w in enumerate(self.group_w[b]):
            for h in range(self.H):
                keep[0, h, g * GROUP:(g + 1) * GROUP] = prune_channel_group(
                    v[0, h, g * GROUP:(g + 1) * GROUP], gk, None if w is None else w[h])
        return enc_k, encode(v, keep)

    def attention(self, q, b: int, scale: float = 0.0) -> np.ndarray:
        q = np.asarray(q).view(np.uint16)[None]
        enc_k, enc_v = self.compressed(b)
        wk, wv = self.window(b)
        return sparse_decode_attention(q, enc_k, enc_v, wk[None], wv[None], scale)[0]

    def score_increments(self, q, b: int, scale: float = 0.0) -> np.ndarray:
        """float64 [H][len]: for every window token of entry b younger than 32
        of its steps (the newest 32), the attention probability it receives from
        q [Hq][d], summed over the query heads of each kv-head; 0 for older ones.
        Only a step in which entry b is active adds these to its tokens' scores."""
        q = np.asarray(q).view(np.uint16)[None]
        enc_k, _ = self.compressed(b)
        wk, _ = self.window(b)
        p = attention_probs(q, decompress(enc_k), wk[None], scale)[0]
        n, L = self.ncomp[b], self.window_len(b)
        G = q.shape[1] // self.H
        out = np.zeros((self.H, L), dtype=np.float64)
        for h in range(self.H):
            tot = p[h * G:(h + 1) * G, n:].sum(axis=0)
            young = np.arange(L) >= L - GROUP
            out[h] = np.where(young, tot, 0.0)
        return out
