"""Oracle: FOCUS streaming decode, one token per step -- TEST INFRASTRUCTURE.

What is computed (Appendix A.2 "Streaming with controlled memory"; the summary
layout of Section 3.2 / Appendix A): a sequence is extended one augmented token
at a time.  The state is

  cache   retained KV of every summary token produced so far
  window  KV of the ordinary (base) tokens of the current window
  counters  bases in the current window and in the currently open k-mer

Each step
  1. decides the token's kind from the layout rule: it is a summary when the
     open k-mer holds k bases, or when the window holds W bases and a partial
     k-mer is open; otherwise it is a base;
  2. appends the token's K/V to the cache (summary) or to the window (base);
  3. attends from the token's query over [cache ; window], every row visible
     (the token's visible set C(t): all retained summaries of earlier windows,
     the current window's tokens so far, itself included -- the current
     window's own summaries are reached through the cache, where they already
     sit);
  4. when the token closes the window, drops the window's ordinary KV.

With k = 0 no summary is ever produced and the window simply ends at its W-th
base.  State arrays keep the input dtype's exact values; arithmetic is float64.
"""

from __future__ import annotations

import numpy as np

from .attention import attend, default_scale
from .layout import BASE, SUMMARY


class DecodeSequence:
    """Decode state of one sequence (see module docstring)."""

    def __init__(self, window_nt: int, kmer, cache_k, cache_v, win_k, win_v,
                 bases_in_window: int, bases_in_kmer: int):
        """kmer: one cadence for every window, or the cadences of the current
        window and of the windows after it (the last entry repeats), as the
        layout allows one k_w per window."""
        self.W = int(window_nt)
        self.cadences = [int(kmer)] if np.ndim(kmer) == 0 else [int(x) for x in kmer]
        self.win_index = 0      # windows closed since the start
        self.cache_k = [np.asarray(r) for r in cache_k]
        self.cache_v = [np.asarray(r) for r in cache_v]
        self.win_k = [np.asarray(r) for r in win_k]
        self.win_v = [np.asarray(r) for r in win_v]
        self.bases_in_window = int(bases_in_window)
        self.bases_in_kmer = int(bases_in_kmer)

    @property
    def k(self) -> int:
        """Cadence of the current window."""
        return self.cadences[min(self.win_index, len(self.cadences) - 1)]

    @staticmethod
    def replay_counters(window_nt: int, kmer: int, n_tokens: int):
        """Walk the first n_tokens augmented tokens of a window with the layout
        rule; return (bases, summaries, bases_in_open_kmer)."""
        bases = summaries = open_kmer = 0
        for _ in range(n_tokens):
            if kmer > 0 and (open_kmer == kmer or (bases == window_nt and open_kmer > 0)):
                summaries += 1
                open_kmer = 0
            else:
                bases += 1
                open_kmer += 1
        return bases, summaries, open_kmer

    def next_kind(self) -> int:
        k, W = self.k, self.W
        if k > 0 and (self.bases_in_kmer == k or (self.bases_in_window == W and self.bases_in_kmer > 0)):
            return SUMMARY
        return BASE

    def step(self, q, k_new, v_new, scale=None, compute=True):
        """Advance by one token.  q [H, D]; k_new, v_new [H_kv, D].

        Returns (O [H, D] or None, LSE [H] or None, kind, window_end)."""
        kind = self.next_kind()
        if kind == SUMMARY:
            self.cache_k.append(np.asarray(k_new))
            self.cache_v.append(np.asarray(v_new))
            self.bases_in_kmer = 0
            window_end = self.bases_in_window == self.W
        else:
            self.win_k.append(np.asarray(k_new))
            self.win_v.append(np.asarray(v_new))
            self.bases_in_window += 1
            self.bases_in_kmer += 1
            window_end = self.k == 0 and self.bases_in_window == self.W
        o = lse = None
        if compute:
            o, lse = self.attend(q, scale)
        if window_end:
            self.win_k, self.win_v = [], []
            self.bases_in_window = 0
            self.bases_in_kmer = 0
            self.win_index += 1
        return o, lse, kind, window_end

    def attend(self, q, scale=None):
        """Attention of q [H, D] over [cache ; window], all rows visible."""
        q = np.asarray(q, np.float64)
        H, D = q.shape
        if scale is None:
            scale = default_scale(D)
        keys = np.asarray(self.cache_k + self.win_k, np.float64)    # [N, H_kv, D]
        vals = np.asarray(self.cache_v + self.win_v, np.float64)
        Hkv = keys.shape[1]
        o = np.empty((H, D), np.float64)
        lse = np.empty(H, np.float64)
        vis = np.ones((1, keys.shape[0]), bool)
        for h in range(H):
            g = h // (H // Hkv)
            oh, lh, _ = attend(q[h][None, :], keys[:, g], vals[:, g], vis, scale)
            o[h], lse[h] = oh[0], lh[0]
        return o, lse

    @property
    def cache_len(self) -> int:
        return len(self.cache_k)

    @property
    def win_len(self) -> int:
        return len(self.win_k)
