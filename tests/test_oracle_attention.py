"""Pins for the attention/compaction oracle against facts the paper and the
mathematics fix:

* with no summary tokens and one window FOCUS attention is dense causal
  attention, checked against a pure-Python brute force (scalar loops and
  math.exp) that shares nothing with the oracle's matrix form;
* softmax rows sum to one and vanish outside the visible set;
* closed forms: K = 0 gives the mean of the visible values, and with one-hot
  values this spells out the visible set C(t) exactly (all earlier-window
  summaries plus the window's own rows up to t, Appendix A.1); constant values
  give that constant; the first token of the first window returns its own value;
* invariances: permuting the retained cache rows, perturbing an earlier
  window's ordinary KV (discarded after its window, Appendix A) or a later
  token (strict causality) leaves the outputs unchanged;
* the sequential and masked-parallel forms agree (A.1 "Cross-window consistency");
* compaction keeps exactly the summary rows, and the cache length is the
  summed summary count.
"""

import math

import numpy as np
import pytest

from oracle import attention as A
from oracle.layout import BASE, SUMMARY, build_layout


def brute_force_causal(q, k, v, scale):
    """Scalar-loop causal attention for one head: q, k, v lists of D-vectors."""
    n, D = len(q), len(q[0])
    out, lses = [], []
    for i in range(n):
        s = [scale * sum(q[i][d] * k[j][d] for d in range(D)) for j in range(i + 1)]
        mx = max(s)
        e = [math.exp(x - mx) for x in s]
        tot = sum(e)
        out.append([sum(e[j] * v[j][d] for j in range(i + 1)) / tot for d in range(D)])
        lses.append(mx + math.log(tot))
    return np.array(out), np.array(lses)


def rand(rng, *shape):
    return rng.standard_normal(shape)


@pytest.mark.parametrize("seed", range(6))
def test_zero_summaries_one_window_is_dense_causal(seed):
    rng = np.random.default_rng(seed)
    n, H, D = int(rng.integers(1, 12)), 2, 5
    q, k, v = rand(rng, n, H, D), rand(rng, n, H, D), rand(rng, n, H, D)
    scale = 0.37
    lay = build_layout([n], n, 0)               # one window, no summaries
    o, lse = A.prefill_sequential(lay, q, k, v, scale)
    o2, lse2 = A.dense_causal(q, k, v, scale)
    for h in range(H):
        bo, bl = brute_force_causal(q[:, h].tolist(), k[:, h].tolist(), v[:, h].tolist(), scale)
        np.testing.assert_allclose(o[:, h], bo, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse[:, h], bl, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(o2[:, h], bo, rtol=1e-12, atol=1e-12)


def test_window_attention_matches_brute_force_with_cache():
    """[cache ; window] attention equals a scalar brute force over the explicit
    visible set (cache rows, then window rows up to and including i)."""
    rng = np.random.default_rng(7)
    C, T, D = 4, 6, 3
    q, kw, vw = rand(rng, T, 1, D), rand(rng, T, 1, D), rand(rng, T, 1, D)
    kc, vc = rand(rng, C, 1, D), rand(rng, C, 1, D)
    scale = 0.5
    o, lse = A.window_attention(q, kw, vw, kc, vc, scale)
    for i in range(T):
        keys = [kc[j, 0] for j in range(C)] + [kw[u, 0] for u in range(i + 1)]
        vals = [vc[j, 0] for j in range(C)] + [vw[u, 0] for u in range(i + 1)]
        s = [scale * float(np.dot(q[i, 0], kk)) for kk in keys]
        mx = max(s)
        e = [math.exp(x - mx) for x in s]
        ref = sum(ee * vv for ee, vv in zip(e, vals)) / sum(e)
        np.testing.assert_allclose(o[i, 0], ref, rtol=1e-12, atol=1e-13)
        assert abs(lse[i, 0] - (mx + math.log(sum(e)))) < 1e-12


def test_rows_sum_to_one_and_respect_mask():
    rng = np.random.default_rng(3)
    C, T, D = 5, 7, 4
    vis = A.window_visibility(T, C)
    _, lse, p = A.attend(rand(rng, T, D), rand(rng, C + T, D), rand(rng, C + T, D), vis, 0.3)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    assert (p[~vis] == 0).all() and (p[vis] > 0).all()


@pytest.mark.parametrize("seed", range(5))
def test_zero_keys_give_mean_of_visible_values_one_hot(seed):
    """K = 0 makes every visible score equal, so O_i is the mean of the visible
    values; one-hot values make O_i the indicator of C(t) / |C(t)|."""
    rng = np.random.default_rng(seed)
    L, W, k = int(rng.integers(5, 40)), int(rng.integers(3, 12)), int(rng.integers(1, 5))
    lay = build_layout([L], W, k)
    NT = lay["n_tokens"]
    q = rand(rng, NT, 1, NT)
    kk = np.zeros((NT, 1, NT))
    v = np.eye(NT)[:, None, :]                        # V_u = e_u
    o, _ = A.prefill_sequential(lay, q, kk, v)
    kind, win = lay["tok_kind"], lay["tok_win"]
    for t in range(NT):
        visible = [u for u in range(t + 1) if win[u] == win[t] or kind[u] == SUMMARY]
        expect = np.zeros(NT)
        expect[visible] = 1.0 / len(visible)
        np.testing.assert_allclose(o[t, 0], expect, rtol=0, atol=1e-14)
        # |C(t)| = C_w + (index of t inside its window) + 1
        w = win[t]
        assert len(visible) == lay["win_cache_off"][w] + (t - lay["win_tok_off"][w]) + 1


def test_constant_values_and_first_token():
    rng = np.random.default_rng(11)
    lay = build_layout([23], 7, 3)
    NT = lay["n_tokens"]
    q, k = rand(rng, NT, 2, 4), rand(rng, NT, 2, 4)
    c = rand(rng, 4)
    v = np.broadcast_to(c, (NT, 2, 4)).copy()
    o, _ = A.prefill_sequential(lay, q, k, v)
    np.testing.assert_allclose(o, np.broadcast_to(c, o.shape), rtol=1e-13, atol=1e-13)
    v = rand(rng, NT, 2, 4)
    o, lse = A.prefill_sequential(lay, q, k, v)
    np.testing.assert_allclose(o[0], v[0], rtol=0, atol=1e-15)      # sees only itself
    np.testing.assert_allclose(lse[0], np.einsum("hd,hd->h", q[0], k[0]) / 2.0, atol=1e-14)


def test_cache_row_permutation_invariance():
    rng = np.random.default_rng(5)
    C, T, D = 9, 5, 4
    q, kw, vw = rand(rng, T, 2, D), rand(rng, T, 2, D), rand(rng, T, 2, D)
    kc, vc = rand(rng, C, 2, D), rand(rng, C, 2, D)
    perm = rng.permutation(C)
    o1, l1 = A.window_attention(q, kw, vw, kc, vc)
    o2, l2 = A.window_attention(q, kw, vw, kc[perm], vc[perm])
    np.testing.assert_allclose(o1, o2, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=1e-13, atol=1e-14)


def test_discarded_ordinary_kv_is_invisible_but_summaries_are_not():
    rng = np.random.default_rng(9)
    lay = build_layout([30], 10, 4)
    NT = lay["n_tokens"]
    q, k, v = rand(rng, NT, 1, 3), rand(rng, NT, 1, 3), rand(rng, NT, 1, 3)
    o, _ = A.prefill_sequential(lay, q, k, v)
    w1 = np.nonzero(lay["tok_win"] == 1)[0]
    w0 = np.nonzero(lay["tok_win"] == 0)[0]
    base0 = w0[lay["tok_kind"][w0] == BASE]
    k2, v2 = k.copy(), v.copy()
    k2[base0] += 5.0
    v2[base0] -= 3.0
    o2, _ = A.prefill_sequential(lay, q, k2, v2)
    np.testing.assert_array_equal(o[w1], o2[w1])
    np.testing.assert_array_equal(o[lay["tok_win"] == 2], o2[lay["tok_win"] == 2])
    sum0 = w0[lay["tok_kind"][w0] == SUMMARY][0]
    v3 = v.copy()
    v3[sum0] += 1.0
    o3, _ = A.prefill_sequential(lay, q, k, v3)
    assert np.abs(o3[w1] - o[w1]).max() > 1e-3


def test_strict_causality():
    rng = np.random.default_rng(13)
    lay = build_layout([25], 25, 5)
    NT = lay["n_tokens"]
    q, k, v = rand(rng, NT, 1, 3), rand(rng, NT, 1, 3), rand(rng, NT, 1, 3)
    o, _ = A.prefill_sequential(lay, q, k, v)
    u = 17
    k2, v2 = k.copy(), v.copy()
    k2[u] += 2.0
    v2[u] += 2.0
    o2, _ = A.prefill_sequential(lay, q, k2, v2)
    np.testing.assert_array_equal(o[:u], o2[:u])
    assert np.abs(o2[u:] - o[u:]).max(axis=(1, 2)).min() > 0


@pytest.mark.parametrize("seed", range(6))
def test_sequential_equals_masked_parallel(seed):
    rng = np.random.default_rng(40 + seed)
    B = 2
    seq = [int(x) for x in rng.integers(1, 50, B)]
    W = int(rng.integers(2, 15))
    nw = sum(-(-L // W) for L in seq)
    kmer = rng.integers(0, 6, nw)
    lay = build_layout(seq, W, kmer)
    NT = lay["n_tokens"]
    q, k, v = rand(rng, NT, 4, 3), rand(rng, NT, 2, 3), rand(rng, NT, 2, 3)
    o, lse = A.prefill_sequential(lay, q, k, v)
    for b in range(B):
        t0, t1 = lay["cu_tokens"][b], lay["cu_tokens"][b + 1]
        om, lm = A.prefill_masked_parallel(lay, q, k, v, b)
        np.testing.assert_allclose(o[t0:t1], om, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(lse[t0:t1], lm, rtol=1e-12, atol=1e-13)
    for w in range(lay["n_windows"]):
        t0 = lay["win_tok_off"][w]
        ow, lw = A.prefill_window(lay, w, q, k, v)
        np.testing.assert_allclose(o[t0:t0 + lay["win_ntok"][w]], ow, rtol=1e-12, atol=1e-13)


def test_grouped_kv_heads_equal_repeated_heads():
    """Query head h reads KV head h // (H/H_kv): same as repeating KV heads."""
    rng = np.random.default_rng(21)
    lay = build_layout([40], 9, 3)
    NT = lay["n_tokens"]
    q, k, v = rand(rng, NT, 6, 4), rand(rng, NT, 2, 4), rand(rng, NT, 2, 4)
    o, lse = A.prefill_sequential(lay, q, k, v)
    o2, lse2 = A.prefill_sequential(lay, q, np.repeat(k, 3, axis=1), np.repeat(v, 3, axis=1))
    np.testing.assert_allclose(o, o2, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(lse, lse2, rtol=1e-13, atol=1e-14)


def test_scale_enters_only_through_scores():
    rng = np.random.default_rng(22)
    lay = build_layout([20], 6, 2)
    NT = lay["n_tokens"]
    q, k, v = rand(rng, NT, 1, 4), rand(rng, NT, 1, 4), rand(rng, NT, 1, 4)
    o1, l1 = A.prefill_sequential(lay, q, k, v, scale=0.25)
    o2, l2 = A.prefill_sequential(lay, 0.25 * q, k, v, scale=1.0)
    np.testing.assert_allclose(o1, o2, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=1e-13, atol=1e-14)
    o3, _ = A.prefill_sequential(lay, q, k, v)           # default 1/sqrt(D)
    o4, _ = A.prefill_sequential(lay, q, k, v, scale=0.5)
    np.testing.assert_allclose(o3, o4, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("seed", range(4))
def test_compaction_keeps_summary_rows_in_order(seed):
    rng = np.random.default_rng(60 + seed)
    seq = [int(x) for x in rng.integers(0, 70, 3)]
    W = int(rng.integers(3, 20))
    nw = sum(-(-L // W) for L in seq)
    lay = build_layout(seq, W, rng.integers(1, 7, nw))
    NT = lay["n_tokens"]
    k = np.arange(NT, dtype=np.float64)[:, None, None] * np.ones((1, 2, 3))
    v = -k
    for b in range(3):
        ck, cv = A.compact(lay, k, v, b)
        t0, t1 = lay["cu_tokens"][b], lay["cu_tokens"][b + 1]
        expect = [t for t in range(t0, t1) if lay["tok_kind"][t] == SUMMARY]
        assert ck[:, 0, 0].tolist() == expect and cv[:, 1, 2].tolist() == [-x for x in expect]
        n_rows = sum(lay["win_nsum"][lay["win_seq"] == b])
        assert len(ck) == n_rows
        for w in np.nonzero(lay["win_seq"] == b)[0]:
            idx = A.cache_token_indices(lay, w)
            assert idx.tolist() == expect[:lay["win_cache_off"][w]]
