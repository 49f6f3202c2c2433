"""Pins for the k-mer-local visibility oracle (Section 3.2, "Visibility and
summarization rule") against facts the rule fixes:

* two independent statements of the rule agree: the stream-domain walk over a
  whole augmented sequence (masked-parallel form) and the per-window form over
  [cache ; window] keys;
* closed form of the visible set, spelled out with K = 0 and one-hot values: a
  base at offset p of k-mer j of a window sees p + 1 tokens of its k-mer, the j
  summaries before it in the window and, after the first window, the carried
  boundary; summary j sees its n_j bases, itself, the j earlier summaries and the
  boundary;
* with one k-mer per window the rule is causal attention inside the window plus
  the boundary row only;
* invariances: an earlier window's rows other than the boundary, and the bases
  of other k-mers of the same window, never change an output;
* the first k-mer of the first window is textbook causal attention (the pure-
  Python brute force shared with the C(t) pins);
* k = 0 with one window is dense causal attention.
"""

import numpy as np
import pytest

from oracle import attention as A
from oracle.layout import SUMMARY, build_layout
from test_oracle_attention import brute_force_causal


def _random_layout(rng, max_seq=3):
    B = int(rng.integers(1, max_seq + 1))
    seq = [int(x) for x in rng.integers(1, 40, B)]
    W = int(rng.integers(3, 16))
    nw = sum(-(-L // W) for L in seq)
    kmer = rng.integers(0, 7, nw).astype(np.int32)
    return seq, W, kmer, build_layout(seq, W, kmer)


@pytest.mark.parametrize("seed", range(8))
def test_stream_form_equals_window_form(seed):
    rng = np.random.default_rng(seed)
    seq, W, kmer, lay = _random_layout(rng)
    H, Hkv, D = 2, 1, 4
    n = lay["n_tokens"]
    q, k, v = rng.standard_normal((n, H, D)), rng.standard_normal((n, Hkv, D)), rng.standard_normal((n, Hkv, D))
    for b in range(len(seq)):
        o_s, l_s = A.kmer_local_masked_parallel(lay, q, k, v, b, scale=0.41)
        t_b = int(lay["cu_tokens"][b])
        for w in range(int(lay["cu_windows"][b]), int(lay["cu_windows"][b + 1])):
            t0, T = int(lay["win_tok_off"][w]), int(lay["win_ntok"][w])
            o_w, l_w = A.kmer_local_window(lay, w, q, k, v, scale=0.41)
            np.testing.assert_allclose(o_w, o_s[t0 - t_b:t0 - t_b + T], rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(l_w, l_s[t0 - t_b:t0 - t_b + T], rtol=1e-12, atol=1e-12)


def _expected_visible(lay, w):
    """The visible key set of every query of window w, from the closed form:
    key ids are ("c", cache row) or ("w", window row)."""
    t0, T, C = int(lay["win_tok_off"][w]), int(lay["win_ntok"][w]), int(lay["win_cache_off"][w])
    k = int(lay["window_kmer"][w])
    out = []
    for i in range(T):
        g = i // (k + 1) if k > 0 else 0           # k-mer index inside the window
        start = g * (k + 1) if k > 0 else 0          # first row of that k-mer
        keys = set(("w", u) for u in range(start, i + 1))
        keys |= set(("w", (s + 1) * (k + 1) - 1) for s in range(g)) if k > 0 else set()
        if C > 0:
            keys.add(("c", C - 1))
        out.append(keys)
    return out


@pytest.mark.parametrize("seed", range(6))
def test_zero_keys_one_hot_values_spell_out_the_visible_set(seed):
    rng = np.random.default_rng(100 + seed)
    seq, W, kmer, lay = _random_layout(rng, max_seq=2)
    for w in range(lay["n_windows"]):
        T, C = int(lay["win_ntok"][w]), int(lay["win_cache_off"][w])
        n_keys = C + T
        q = rng.standard_normal((T, 1, n_keys))
        kw, kc = np.zeros((T, 1, n_keys)), np.zeros((C, 1, n_keys))
        eye = np.eye(n_keys)
        vc, vw = eye[:C, None, :], eye[C:, None, :]
        o, _ = A.window_attention_masked(q, kw, vw, kc, vc, A.kmer_local_window_visibility(lay, w))
        exp = _expected_visible(lay, w)
        for i in range(T):
            cols = sorted(C + u if s == "w" else u for s, u in exp[i])
            want = np.zeros(n_keys)
            want[cols] = 1.0 / len(cols)
            np.testing.assert_allclose(o[i, 0], want, atol=1e-14)
            # the count in words: bases of the own k-mer so far + earlier summaries + boundary
            t0 = int(lay["win_tok_off"][w])
            kind = lay["tok_kind"][t0 + i]
            k = int(lay["window_kmer"][w])
            g = i // (k + 1) if k > 0 else 0
            p = i - g * (k + 1) if k > 0 else i
            assert len(cols) == p + 1 + g + (1 if C > 0 else 0), (w, i, kind)


@pytest.mark.parametrize("seed", range(4))
def test_one_kmer_per_window_is_causal_plus_boundary(seed):
    rng = np.random.default_rng(200 + seed)
    L, W = int(rng.integers(10, 60)), int(rng.integers(3, 12))
    lay = build_layout([L], W, W)               # k = W: one k-mer per window
    for w in range(lay["n_windows"]):
        T, C = int(lay["win_ntok"][w]), int(lay["win_cache_off"][w])
        ct = A.window_visibility(T, C)
        ct[:, :max(C - 1, 0)] = False           # only the last cache row survives
        np.testing.assert_array_equal(A.kmer_local_window_visibility(lay, w), ct)


@pytest.mark.parametrize("seed", range(4))
def test_earlier_rows_and_other_kmer_bases_are_invisible(seed):
    rng = np.random.default_rng(300 + seed)
    seq, W, kmer, lay = _random_layout(rng, max_seq=1)
    n, H, D = lay["n_tokens"], 2, 3
    q, k, v = rng.standard_normal((n, H, D)), rng.standard_normal((n, H, D)), rng.standard_normal((n, H, D))
    o, lse = A.kmer_local_masked_parallel(lay, q, k, v, 0)
    kind, win, km = lay["tok_kind"], lay["tok_win"], lay["tok_kmer"]
    for t in range(n):
        # every token this one must not see: earlier-window rows other than the
        # carried boundary, same-window bases of other k-mers, later tokens
        sums_before = [u for u in range(t) if win[u] != win[t] and kind[u] == SUMMARY]
        boundary = sums_before[-1] if sums_before else -1
        hidden = [u for u in range(n) if u > t or (u != boundary and win[u] != win[t])
                  or (win[u] == win[t] and kind[u] != SUMMARY and km[u] != km[t])]
        if not hidden:
            continue
        k2, v2 = k.copy(), v.copy()
        k2[hidden] += rng.standard_normal((len(hidden), H, D)) * 3
        v2[hidden] += rng.standard_normal((len(hidden), H, D)) * 3
        o2, lse2 = A.kmer_local_masked_parallel(lay, q, k2, v2, 0)
        np.testing.assert_allclose(o2[t], o[t], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse2[t], lse[t], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_first_kmer_is_textbook_causal(seed):
    rng = np.random.default_rng(400 + seed)
    kk = int(rng.integers(2, 9))
    L = int(rng.integers(kk + 1, 4 * kk))
    lay = build_layout([L], L, kk)              # one window, several k-mers
    n, D = lay["n_tokens"], 4
    q, k, v = rng.standard_normal((n, 1, D)), rng.standard_normal((n, 1, D)), rng.standard_normal((n, 1, D))
    o, lse = A.kmer_local_window(lay, 0, q, k, v, scale=0.3)
    m = kk + 1                                  # first k-mer: kk bases and its summary
    bo, bl = brute_force_causal(q[:m, 0].tolist(), k[:m, 0].tolist(), v[:m, 0].tolist(), 0.3)
    np.testing.assert_allclose(o[:m, 0], bo, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse[:m, 0], bl, rtol=1e-12, atol=1e-12)


def test_zero_kmer_single_window_is_dense_causal():
    rng = np.random.default_rng(5)
    n = 13
    lay = build_layout([n], n, 0)
    q, k, v = rng.standard_normal((n, 2, 3)), rng.standard_normal((n, 2, 3)), rng.standard_normal((n, 2, 3))
    o, lse = A.kmer_local_window(lay, 0, q, k, v)
    o2, lse2 = A.dense_causal(q, k, v)
    np.testing.assert_allclose(o, o2, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, lse2, rtol=1e-12, atol=1e-12)
