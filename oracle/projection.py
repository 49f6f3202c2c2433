"""Oracle: the layer's Q/K/V projection with FOCUS-aware rotary positions and
the retained-KV cache it feeds -- TEST INFRASTRUCTURE.

What is computed, in float64:

* [Q | K | V] = hidden W_qkv, the columns of W_qkv being the query heads, then
  the key heads, then the value heads.
* Rotary position embedding on Q and K (reading: the paper inserts summary
  tokens that occupy real sequence positions, Sec. 3.2 / App. A "occupies a
  real sequence position", so the position of a token is its index in its
  sequence's augmented stream): inside each head the pairs (2i, 2i + 1) are
  rotated by the angle pos * theta^(-2i/D).  The interleaved pairing is one
  fixed permutation of the head dimension away from the half-split pairing,
  which a trained W_qkv absorbs.
* The retained cache of a sequence: the rotated K (and V) rows of its summary
  tokens in stream order (App. A "KV compression and budget"), as
  attention.compact builds it.
* store_bf16: Q, K, V rounded to bfloat16 after the rotation, as the device
  stores them.
"""

from __future__ import annotations

import numpy as np

from .adapter import round_bf16


def rope(x, pos, theta):
    """Rotate pairs (2i, 2i + 1) of the last axis of x [T, H, D] by
    pos[t] * theta^(-2i / D)."""
    x = np.asarray(x, np.float64)
    D = x.shape[-1]
    i = np.arange(D // 2)
    ang = np.asarray(pos, np.float64)[:, None] * theta ** (-2.0 * i / D)      # [T, D/2]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    e, o = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = e * c - o * s
    out[..., 1::2] = e * s + o * c
    return out


def qkv_project(layout, hidden, w_qkv, n_heads, n_kv_heads, theta=10000.0, store_bf16=False, rows=None):
    """Q [T, H, D], K, V [T, H_kv, D] of the tokens `rows` (default: all) of
    the layout, from hidden [n_tokens, d_model] (or a callable rows -> hidden
    rows).  theta <= 0: no rotation."""
    rows = np.arange(layout["n_tokens"]) if rows is None else np.asarray(rows, np.int64)
    h = np.asarray(hidden(rows) if callable(hidden) else np.asarray(hidden, np.float64)[rows], np.float64)
    w = np.asarray(w_qkv, np.float64)
    D = w.shape[1] // (n_heads + 2 * n_kv_heads)
    y = h @ w
    q = y[:, :n_heads * D].reshape(-1, n_heads, D)
    k = y[:, n_heads * D:(n_heads + n_kv_heads) * D].reshape(-1, n_kv_heads, D)
    v = y[:, (n_heads + n_kv_heads) * D:].reshape(-1, n_kv_heads, D)
    if theta > 0:
        pos = layout["tok_pos"][rows]
        q, k = rope(q, pos, theta), rope(k, pos, theta)
    if store_bf16:
        q, k, v = round_bf16(q), round_bf16(k), round_bf16(v)
    return q, k, v
