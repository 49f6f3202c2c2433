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
whole update from hidden states and the four weight matrices.
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


def adapter_attention(layout, q_sum, k, v, mask="ct", scale=None):
    """q_sum [n_summaries, H, D] (summary order), k, v [n_tokens, H_kv, D]
    (global token order).  Returns O [n_summaries, H, D], LSE [n_summaries, H]."""
    q_sum, k, v = np.asarray(q_sum), np.asarray(k), np.asarray(v)
    n_sum, H, D = q_sum.shape
    Hkv = k.shape[1]
    if scale is None:
        scale = A.default_scale(D)
    o = np.empty((n_sum, H, D), np.float64)
    lse = np.empty((n_sum, H), np.float64)
    for w in range(layout["n_windows"]):
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


def adapter_layer(layout, hidden, w_q, w_k, w_v, w_o, n_heads, n_kv_heads, mask="ct", scale=None):
    """Updated hidden states of the summary tokens ([n_summaries, d_model]).

    hidden [n_tokens, d_model]; w_q [d_model, H D]; w_k, w_v [d_model, H_kv D];
    w_o [H D, d_model]."""
    hidden = np.asarray(hidden, np.float64)
    D = np.asarray(w_q).shape[1] // n_heads
    q_sum = (hidden[layout["sum_tok"]] @ w_q).reshape(-1, n_heads, D)
    k = (hidden @ w_k).reshape(-1, n_kv_heads, D)
    v = (hidden @ w_v).reshape(-1, n_kv_heads, D)
    o, _ = adapter_attention(layout, q_sum, k, v, mask, scale)
    return o.reshape(len(q_sum), n_heads * D) @ w_o
