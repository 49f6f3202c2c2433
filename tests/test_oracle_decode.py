"""Pins for the decode oracle: decoding a stream one token at a time must give
the same rows as windowed prefill over the same augmented stream (Appendix A.2:
streaming inference carries the retained summary KV as history), whatever the
starting point inside a window; the cache grows by exactly one row per summary
and the window buffer empties at each window end."""

import numpy as np
import pytest

from oracle import attention as A
from oracle.decode import DecodeSequence
from oracle.layout import BASE, SUMMARY, build_layout


def _stream(seed, L, W, k, H=2, Hkv=1, D=4):
    rng = np.random.default_rng(seed)
    lay = build_layout([L], W, k)
    NT = lay["n_tokens"]
    q = rng.standard_normal((NT, H, D))
    kk = rng.standard_normal((NT, Hkv, D))
    v = rng.standard_normal((NT, Hkv, D))
    return lay, q, kk, v


@pytest.mark.parametrize("L,W,k", [(37, 10, 3), (30, 10, 5), (25, 7, 7), (18, 6, 0), (41, 12, 5)])
def test_decode_from_empty_equals_prefill(L, W, k):
    lay, q, kk, v = _stream(L * 7 + k, L, W, k)
    o_ref, l_ref = A.prefill_sequential(lay, q, kk, v)
    st = DecodeSequence(W, k, [], [], [], [], 0, 0)
    # Generation has no sequence end: a truncated last window closes with a
    # summary in the prefill layout, where decoding would go on with a base.
    n_cmp = lay["n_tokens"] - (1 if (L % W and k) else 0)
    for t in range(n_cmp):
        o, lse, kind, end = st.step(q[t], kk[t], v[t])
        assert kind == lay["tok_kind"][t]
        w = lay["tok_win"][t]
        assert end == (t == lay["win_tok_off"][w] + lay["win_ntok"][w] - 1)
        np.testing.assert_allclose(o, o_ref[t], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(lse, l_ref[t], rtol=1e-12, atol=1e-13)
    assert st.cache_len == lay["n_summaries"] - (n_cmp < lay["n_tokens"])


@pytest.mark.parametrize("start", [1, 4, 11, 20])
def test_decode_mid_window_start_equals_prefill(start):
    """Start with a window already `start` tokens in (its summaries in the
    cache, its bases in the window buffer), as the batch-16 decode workload
    does, and keep decoding across a window boundary."""
    L, W, k = 60, 20, 6
    lay, q, kk, v = _stream(3, L, W, k)
    o_ref, l_ref = A.prefill_sequential(lay, q, kk, v)
    w = 1
    t0 = lay["win_tok_off"][w]
    n_bases, n_sum, open_kmer = DecodeSequence.replay_counters(W, k, start)
    toks = np.arange(t0, t0 + start)
    kinds = lay["tok_kind"][toks]
    assert (kinds == BASE).sum() == n_bases and (kinds == SUMMARY).sum() == n_sum
    cache_idx = list(A.cache_token_indices(lay, w)) + list(toks[kinds == SUMMARY])
    win_idx = list(toks[kinds == BASE])
    st = DecodeSequence(W, k, kk[cache_idx], v[cache_idx], kk[win_idx], v[win_idx],
                        n_bases, open_kmer)
    for t in range(t0 + start, lay["n_tokens"]):
        o, lse, kind, _ = st.step(q[t], kk[t], v[t])
        assert kind == lay["tok_kind"][t]
        np.testing.assert_allclose(o, o_ref[t], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(lse, l_ref[t], rtol=1e-12, atol=1e-13)


def test_cache_growth_and_window_reset():
    W, k = 10, 4
    st = DecodeSequence(W, k, [], [], [], [], 0, 0)
    z = np.zeros((1, 2))
    kinds, ends, cache, win = [], [], [], []
    for _ in range(3 * 13):       # three windows of 10 bases + 3 summaries
        _, _, kind, end = st.step(np.zeros((1, 2)), z, z, compute=False)
        kinds.append(kind)
        ends.append(end)
        cache.append(st.cache_len)
        win.append(st.win_len)
    one = "bbbbSbbbbSbbS"
    assert "".join("S" if x == SUMMARY else "b" for x in kinds) == one * 3
    assert [i for i, e in enumerate(ends) if e] == [12, 25, 38]
    assert cache[-1] == 9 and win[12] == 0 and win[11] == 10


@pytest.mark.parametrize("seed", range(4))
def test_per_window_cadence_equals_prefill(seed):
    """Windows with their own cadence k_w (the layout allows one per window):
    decoding from empty through several windows, the cadence switching at each
    window end, gives the prefill rows of the same per-window layout."""
    rng = np.random.default_rng(50 + seed)
    W = int(rng.integers(5, 12))
    L = 4 * W
    km = rng.choice([1, 2, 3, 5, 50], 4).astype(np.int32)
    lay = build_layout([L], W, km)
    NT = lay["n_tokens"]
    q = rng.standard_normal((NT, 2, 4))
    kk = rng.standard_normal((NT, 1, 4))
    v = rng.standard_normal((NT, 1, 4))
    o_ref, l_ref = A.prefill_sequential(lay, q, kk, v)
    st = DecodeSequence(W, km, [], [], [], [], 0, 0)
    for t in range(NT):
        o, lse, kind, end = st.step(q[t], kk[t], v[t])
        w = lay["tok_win"][t]
        assert kind == lay["tok_kind"][t]
        assert end == (t == lay["win_tok_off"][w] + lay["win_ntok"][w] - 1)
        np.testing.assert_allclose(o, o_ref[t], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(lse, l_ref[t], rtol=1e-12, atol=1e-13)
    assert st.cache_len == lay["n_summaries"] and st.win_index == 4
