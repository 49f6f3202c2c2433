"""Oracle: FOCUS window attention and retained-KV compaction -- TEST INFRASTRUCTURE.

What is computed, in float64:

* Compaction (Appendix A "KV compression and budget"; A.2 "Streaming with
  controlled memory"): after window w, the KV of its ordinary tokens is dropped
  and the KV of its B_w summary tokens is appended to the sequence's retained
  cache.  The cache of a sequence is therefore the rows of its summary tokens,
  in stream order.

* Window attention (Appendix A eq. focus-attn and A.1 "Objective and
  visibility"): token t of window w attends, by causal softmax attention, to the
  set C(t) made of every earlier-or-equal position inside its own window plus
  the retained summary KV of all earlier windows of its sequence -- never to an
  ordinary token of an earlier window.  Scores are scale * <q, k>, with
  scale = 1/sqrt(D) unless given; LSE is the natural-log normaliser.

  Two constructions of the same thing are provided, as the paper states they
  are equivalent (A.1 "Cross-window consistency"):
    prefill_sequential     windows in order; each sees [cache ; own window]
    prefill_masked_parallel  the whole augmented sequence under the C(t) mask

* dense_causal: textbook causal attention, to which FOCUS attention reduces
  with no summary tokens and a single window.

* The k-mer-local rule of Section 3.2 ("Visibility and summarization rule"),
  the paper's other visibility statement: a base token sees the earlier tokens
  of its own k-mer and the summary tokens before it in its window, including
  the boundary summary carried over from the previous window; a summary token
  sees its own k-mer, the earlier summaries of its window and that carried
  boundary.  Nothing else of earlier windows is visible.  Readings taken where
  the section is silent: the carried boundary is the last summary token of the
  previous window of the same sequence (the last retained cache row); a token
  sees itself; a window with k_w = 0 has no summaries and is a single k-mer
  (plain causal attention inside it, plus the carried boundary).
  kmer_local_stream_visibility states the rule over a whole augmented sequence
  (masked-parallel form); kmer_local_window_visibility states it over one
  window's [cache ; window] keys, the form the kernels take.

All matrix products are NumPy float64 matmuls; masking is an explicit boolean
matrix; the softmax is the definition (shift by the row max, exponentiate,
normalise).  Inputs are float arrays holding the exact values the kernels
read (bf16 inputs are upcast exactly).
"""

from __future__ import annotations

import math

import numpy as np

from .layout import SUMMARY


def attend(q, keys, values, visible, scale):
    """Masked softmax attention of rows q [T, D] over keys/values [N, D].

    visible[i, j] (bool [T, N]) says whether key j is in query i's visible set.
    Returns (O [T, D], LSE [T], P [T, N]).  Every row must see >= 1 key.
    """
    q = np.asarray(q, np.float64)
    keys = np.asarray(keys, np.float64)
    values = np.asarray(values, np.float64)
    s = scale * (q @ keys.T)
    s = np.where(visible, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    l = e.sum(axis=1, keepdims=True)
    p = e / l
    o = p @ values
    lse = (m + np.log(l))[:, 0]
    return o, lse, p


def window_visibility(n_queries: int, n_cache: int):
    """C(t) for one window: key j of [cache (n_cache rows) ; window rows] is
    visible to window query i iff it is a retained cache row or an earlier-or-
    equal window row."""
    i = np.arange(n_queries)[:, None]
    j = np.arange(n_cache + n_queries)[None, :]
    return (j < n_cache) | ((j - n_cache) <= i)


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)


def window_attention(q_win, k_win, v_win, cache_k, cache_v, scale=None):
    """One window, all heads.

    q_win [T, H, D]; k_win, v_win [T, H_kv, D]; cache_k, cache_v [C, H_kv, D].
    Query head h reads KV head h // (H / H_kv).
    Returns O [T, H, D] and LSE [T, H] (float64).
    """
    T, H, D = q_win.shape
    Hkv = k_win.shape[1]
    if H % Hkv:
        raise ValueError("heads must be a multiple of kv heads")
    if scale is None:
        scale = default_scale(D)
    C = cache_k.shape[0]
    vis = window_visibility(T, C)
    o = np.empty((T, H, D), np.float64)
    lse = np.empty((T, H), np.float64)
    for h in range(H):
        g = h // (H // Hkv)
        keys = np.concatenate([cache_k[:, g, :], k_win[:, g, :]], axis=0)
        vals = np.concatenate([cache_v[:, g, :], v_win[:, g, :]], axis=0)
        o[:, h, :], lse[:, h], _ = attend(q_win[:, h, :], keys, vals, vis, scale)
    return o, lse


def cache_token_indices(layout, w: int) -> np.ndarray:
    """Global token indices of the retained rows window w sees, in cache-row
    order: the summary tokens of the earlier windows of its sequence."""
    b = int(layout["win_seq"][w])
    first = int(layout["cu_summaries"][b])
    return layout["sum_tok"][first:first + int(layout["win_cache_off"][w])]


def compact(layout, k, v, b: int):
    """Retained cache of sequence b after all its windows: K and V rows of its
    summary tokens in stream order ([n_b, H_kv, D] each).  k and v are indexed
    by global token."""
    idx = layout["sum_tok"][layout["cu_summaries"][b]:layout["cu_summaries"][b + 1]]
    return np.asarray(k)[idx], np.asarray(v)[idx]


def prefill_window(layout, w: int, q, k, v, scale=None):
    """Attention outputs of window w from arrays indexed by global token."""
    t0 = int(layout["win_tok_off"][w])
    T = int(layout["win_ntok"][w])
    idx = cache_token_indices(layout, w)
    q, k, v = np.asarray(q), np.asarray(k), np.asarray(v)
    return window_attention(q[t0:t0 + T], k[t0:t0 + T], v[t0:t0 + T], k[idx], v[idx], scale)


def prefill_sequential(layout, q, k, v, scale=None):
    """Sequential windowed inference (A.1 (i), A.2): process each sequence's
    windows in order; before a window, the cache holds exactly the summary KV
    the earlier windows retained; after it, the window's summary rows are
    appended and its ordinary rows dropped.  Returns O [NT, H, D], LSE [NT, H]."""
    q, k, v = np.asarray(q), np.asarray(k), np.asarray(v)
    NT, H, D = q.shape
    o = np.empty((NT, H, D), np.float64)
    lse = np.empty((NT, H), np.float64)
    for b in range(len(layout["cu_windows"]) - 1):
        cache_k = np.zeros((0,) + k.shape[1:], k.dtype)
        cache_v = np.zeros((0,) + v.shape[1:], v.dtype)
        for w in range(layout["cu_windows"][b], layout["cu_windows"][b + 1]):
            t0 = int(layout["win_tok_off"][w])
            t1 = t0 + int(layout["win_ntok"][w])
            o[t0:t1], lse[t0:t1] = window_attention(q[t0:t1], k[t0:t1], v[t0:t1],
                                                    cache_k, cache_v, scale)
            keep = np.nonzero(layout["tok_kind"][t0:t1] == SUMMARY)[0] + t0
            cache_k = np.concatenate([cache_k, k[keep]], axis=0)
            cache_v = np.concatenate([cache_v, v[keep]], axis=0)
    return o, lse


def masked_parallel_visibility(layout, b: int):
    """C(t) over the whole augmented stream of sequence b: u is visible to t iff
    u <= t and (u is in t's window, or u is a summary token)."""
    t0, t1 = int(layout["cu_tokens"][b]), int(layout["cu_tokens"][b + 1])
    win = layout["tok_win"][t0:t1]
    is_sum = layout["tok_kind"][t0:t1] == SUMMARY
    n = t1 - t0
    t = np.arange(n)[:, None]
    u = np.arange(n)[None, :]
    return (u <= t) & ((win[None, :] == win[:, None]) | is_sum[None, :])


def prefill_masked_parallel(layout, q, k, v, b: int, scale=None):
    """Masked-parallel form (A.1 (ii)) for sequence b: one attention over the
    whole augmented sequence under the C(t) mask.  Returns O, LSE of its tokens."""
    t0, t1 = int(layout["cu_tokens"][b]), int(layout["cu_tokens"][b + 1])
    q, k, v = np.asarray(q)[t0:t1], np.asarray(k)[t0:t1], np.asarray(v)[t0:t1]
    n, H, D = q.shape
    Hkv = k.shape[1]
    if scale is None:
        scale = default_scale(D)
    vis = masked_parallel_visibility(layout, b)
    o = np.empty((n, H, D), np.float64)
    lse = np.empty((n, H), np.float64)
    for h in range(H):
        g = h // (H // Hkv)
        o[:, h], lse[:, h], _ = attend(q[:, h], k[:, g], v[:, g], vis, scale)
    return o, lse


def dense_causal(q, k, v, scale=None):
    """Textbook causal softmax attention: q [N, H, D], k, v [N, H_kv, D]."""
    q, k, v = np.asarray(q), np.asarray(k), np.asarray(v)
    n, H, D = q.shape
    Hkv = k.shape[1]
    if scale is None:
        scale = default_scale(D)
    vis = np.tril(np.ones((n, n), bool))
    o = np.empty((n, H, D), np.float64)
    lse = np.empty((n, H), np.float64)
    for h in range(H):
        g = h // (H // Hkv)
        o[:, h], lse[:, h], _ = attend(q[:, h], k[:, g], v[:, g], vis, scale)
    return o, lse


# ---------------------------------------------------------------- k-mer-local

def kmer_local_stream_visibility(layout, b: int):
    """Section 3.2 rule over the augmented stream of sequence b: u is visible to
    t iff u <= t and u lies in t's window and (u is in t's k-mer or u is a
    summary token), or u is the carried boundary of t's window (the last summary
    token of the previous window of the sequence).  The k-mer of a token is the
    one its closing summary ends (tok_kmer); k_w = 0 makes the window one k-mer."""
    t0, t1 = int(layout["cu_tokens"][b]), int(layout["cu_tokens"][b + 1])
    n = t1 - t0
    win = layout["tok_win"][t0:t1]
    kmer = layout["tok_kmer"][t0:t1]
    is_sum = layout["tok_kind"][t0:t1] == SUMMARY
    vis = np.zeros((n, n), bool)
    for t in range(n):
        # the carried boundary: the last summary token of an earlier window
        boundary = -1
        for u in range(t):
            if win[u] != win[t] and is_sum[u]:
                boundary = u
        for u in range(t + 1):
            if win[u] == win[t]:
                vis[t, u] = kmer[u] == kmer[t] or is_sum[u]
            elif u == boundary:
                vis[t, u] = True
    return vis


def kmer_local_window_visibility(layout, w: int):
    """The same rule for window w over keys [cache rows 0..C_w-1 ; window rows]:
    cache row r is visible only if it is the last one (r = C_w - 1, the carried
    boundary); window row u is visible to window query i iff u <= i and (u is in
    i's k-mer or u is a summary)."""
    t0 = int(layout["win_tok_off"][w])
    T = int(layout["win_ntok"][w])
    C = int(layout["win_cache_off"][w])
    kmer = layout["tok_kmer"][t0:t0 + T]
    is_sum = layout["tok_kind"][t0:t0 + T] == SUMMARY
    vis = np.zeros((T, C + T), bool)
    if C > 0:
        vis[:, C - 1] = True
    i = np.arange(T)[:, None]
    u = np.arange(T)[None, :]
    vis[:, C:] = (u <= i) & ((kmer[None, :] == kmer[:, None]) | is_sum[None, :])
    return vis


def window_attention_masked(q_win, k_win, v_win, cache_k, cache_v, visible, scale=None):
    """window_attention with an explicit visibility matrix over [cache ; window]."""
    T, H, D = q_win.shape
    Hkv = k_win.shape[1]
    if H % Hkv:
        raise ValueError("heads must be a multiple of kv heads")
    if scale is None:
        scale = default_scale(D)
    o = np.empty((T, H, D), np.float64)
    lse = np.empty((T, H), np.float64)
    for h in range(H):
        g = h // (H // Hkv)
        keys = np.concatenate([cache_k[:, g, :], k_win[:, g, :]], axis=0)
        vals = np.concatenate([cache_v[:, g, :], v_win[:, g, :]], axis=0)
        o[:, h, :], lse[:, h], _ = attend(q_win[:, h, :], keys, vals, visible, scale)
    return o, lse


def kmer_local_window(layout, w: int, q, k, v, scale=None):
    """k-mer-local attention outputs of window w from arrays indexed by global
    token (cache rows are the earlier windows' summary tokens, as in C(t))."""
    t0 = int(layout["win_tok_off"][w])
    T = int(layout["win_ntok"][w])
    idx = cache_token_indices(layout, w)
    q, k, v = np.asarray(q), np.asarray(k), np.asarray(v)
    return window_attention_masked(q[t0:t0 + T], k[t0:t0 + T], v[t0:t0 + T], k[idx], v[idx],
                                   kmer_local_window_visibility(layout, w), scale)


def kmer_local_masked_parallel(layout, q, k, v, b: int, scale=None):
    """k-mer-local attention over the whole augmented sequence b under the
    stream-domain rule.  Returns O, LSE of its tokens."""
    t0, t1 = int(layout["cu_tokens"][b]), int(layout["cu_tokens"][b + 1])
    q, k, v = np.asarray(q)[t0:t1], np.asarray(k)[t0:t1], np.asarray(v)[t0:t1]
    n, H, D = q.shape
    Hkv = k.shape[1]
    if scale is None:
        scale = default_scale(D)
    vis = kmer_local_stream_visibility(layout, b)
    o = np.empty((n, H, D), np.float64)
    lse = np.empty((n, H), np.float64)
    for h in range(H):
        g = h // (H // Hkv)
        o[:, h], lse[:, h], _ = attend(q[:, h], k[:, g], v[:, g], vis, scale)
    return o, lse
