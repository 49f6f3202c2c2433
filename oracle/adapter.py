"""Oracle: the FOCUS adapter (summary-token attention) -- TEST INFRASTRUCTURE.

What is computed (Appendix A eq. focus-compress and eq. focus-attn), in float64:

* At an adapter layer, every summary token b of window w is updated by masked
  multi-head attention in which b is the only query: Q = h_b W_Q, and the keys
  and values are H W_K, H W_V over b's visible set.  The hidden states H are
  those of the layer's input, for base and summary tokens alike.
* The visible set is the one the main attention uses for b's row: C(t)
  (App. A: past positions of b's window and the retained summaries of earlier
  windows) or the k-mer-local rule of Section 3.2 (b's own k-mer, the earlier
  summaries of b's window and the carried boundary).
* The heads are concatenated and mapped back by W_O (reading: standard
  multi-head attention, whose output projection is part of the O(d^2) adapter
  the section describes).

adapter_attention takes already projected Q (summary rows only) and K / V (all
tokens) and returns the per-head attention outputs; adapter_layer does the
whole update from hidden states and the four weight matrices.  With
store_bf16, the layer keeps its intermediates (Q, K, V and the attention
output) as bfloat16, rounded to nearest even, as a bf16 model stores its
activations; the arithmetic stays float64.
"""

from __future__ import annotations

import numpy as np

from . import attention as A


def _visibility(layout, w, mask):
    if mask == "ct":
        T = int(layout["win_ntok"][w])
        return A.window_visibility(T, int(layout["win_cache_off"][w]))
    if mask == "kmer_local":
        return A.kmer_local_window_visibility(layout, w)
    raise ValueError(mask)


def adapter_attention(layout, q_sum, k, v, mask="ct", scale=None, windows=None):
    """q_sum [n_summaries, H, D] (summary order), k, v [n_tokens, H_kv, D]
    (global token order).  Returns O [n_summaries, H, D], LSE [n_summaries, H].
    windows: compute only the summaries of these windows (the other rows are
    left NaN)."""
    q_sum, k, v = np.asarray(q_sum), np.asarray(k), np.asarray(v)
    n_sum, H, D = q_sum.shape
    Hkv = k.shape[1]
    if scale is None:
        scale = A.default_scale(D)
    o = np.full((n_sum, H, D), np.nan)
    lse = np.full((n_sum, H), np.nan)
    for w in (range(layout["n_windows"]) if windows is None else windows):
        s0, B = int(layout["win_sum_off"][w]), int(layout["win_nsum"][w])
        if B == 0:
            continue
        t0, T = int(layout["win_tok_off"][w]), int(layout["win_ntok"][w])
        rows = layout["sum_tok"][s0:s0 + B] - t0          # the summaries' window rows
        idx = A.cache_token_indices(layout, w)
        vis = _visibility(layout, w, mask)[rows]
        for h in range(H):
            g = h // (H // Hkv)
            keys = np.concatenate([k[idx, g], k[t0:t0 + T, g]], axis=0)
            vals = np.concatenate([v[idx, g], v[t0:t0 + T, g]], axis=0)
            o[s0:s0 + B, h], lse[s0:s0 + B, h], _ = A.attend(q_sum[s0:s0 + B, h], keys, vals, vis, scale)
    return o, lse


def round_bf16(x):
    """Round to the nearest bfloat16 value (ties to even), returned as float64:
    the float32 image's low 16 bits are rounded away."""
    b = np.asarray(x, np.float64).astype(np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16 << 16
    return (b & 0xFFFFFFFF).astype(np.uint32).view(np.float32).astype(np.float64)


def adapter_layer(layout, hidden, w_q, w_k, w_v, w_o, n_heads, n_kv_heads, mask="ct", scale=None,
                  store_bf16=False, windows=None):
    """Updated hidden states of the summary tokens ([n_summaries, d_model]).

    hidden [n_tokens, d_model] (a callable row -> rows of hidden is accepted
    too, to fetch only what the listed windows read); w_q [d_model, H D];
    w_k, w_v [d_model, H_kv D]; w_o [H D, d_model].  windows: update only the
    summaries of these windows (other rows NaN); only the rows they read are
    projected."""
    get = hidden if callable(hidden) else (lambda r: np.asarray(hidden, np.float64)[r])
    st = round_bf16 if store_bf16 else (lambda x: x)
    n_tok, n_sum = int(layout["n_tokens"]), int(layout["n_summaries"])
    D = np.asarray(w_q).shape[1] // n_heads
    if windows is None:
        rows = np.arange(n_tok)
    else:
        need = []
        for w in windows:
            t0, T = int(layout["win_tok_off"][w]), int(layout["win_ntok"][w])
            need += [A.cache_token_indices(layout, w), np.arange(t0, t0 + T)]
        rows = np.unique(np.concatenate(need)) if need else np.zeros(0, np.int64)
    h_rows = np.asarray(get(rows), np.float64)
    k = np.zeros((n_tok, n_kv_heads, D))
    v = np.zeros((n_tok, n_kv_heads, D))
    k[rows] = st(h_rows @ w_k).reshape(-1, n_kv_heads, D)
    v[rows] = st(h_rows @ w_v).reshape(-1, n_kv_heads, D)
    q_sum = np.zeros((n_sum, n_heads, D))
    pos = {int(t): i for i, t in enumerate(rows)}
    sums = [s for s in range(n_sum) if int(layout["sum_tok"][s]) in pos]
    q_sum[sums] = st(h_rows[[pos[int(layout["sum_tok"][s])] for s in sums]] @ w_q).reshape(-1, n_heads, D)
    o, _ = adapter_attention(layout, q_sum, k, v, mask, scale, windows)
    return st(o.reshape(n_sum, n_heads * D)) @ w_o
