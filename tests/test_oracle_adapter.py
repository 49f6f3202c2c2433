"""Pins for the FOCUS adapter oracle (Appendix A eq. focus-attn):

* a summary query's output is the main attention's output at the summary's
  row when the summary's query is that row's query, under both visibility
  rules (the adapter is the same masked attention, restricted to summary
  queries);
* closed form with zero keys and one-hot values: each summary sees exactly
  C_w + i + 1 keys under C(t) (i its window row), and its own k-mer, the
  earlier summaries of its window and the boundary under the k-mer-local rule;
* the layer with identity projections is the attention itself; the layer is
  linear in W_O and in W_V (for fixed Q and K); with one KV head, the H query
  heads read the same keys (grouped heads equal repeated heads);
* a window with no summaries contributes no rows, and a later token never
  changes an earlier summary's update (strict causality).
"""

import numpy as np
import pytest

from oracle import adapter as AD
from oracle import attention as A
from oracle.layout import build_layout


def _layout(rng):
    seq = [int(x) for x in rng.integers(1, 60, int(rng.integers(1, 3)))]
    W = int(rng.integers(4, 20))
    nw = sum(-(-L // W) for L in seq)
    kmer = rng.integers(0, 6, nw).astype(np.int32)
    return build_layout(seq, W, kmer)


@pytest.mark.parametrize("mask", ["ct", "kmer_local"])
@pytest.mark.parametrize("seed", range(5))
def test_summary_rows_of_the_main_attention(mask, seed):
    rng = np.random.default_rng(seed)
    lay = _layout(rng)
    n, H, Hkv, D = lay["n_tokens"], 2, 1, 4
    q, k, v = rng.standard_normal((n, H, D)), rng.standard_normal((n, Hkv, D)), rng.standard_normal((n, Hkv, D))
    o, lse = AD.adapter_attention(lay, q[lay["sum_tok"]], k, v, mask, scale=0.7)
    for w in range(lay["n_windows"]):
        t0, T = int(lay["win_tok_off"][w]), int(lay["win_ntok"][w])
        s0, B = int(lay["win_sum_off"][w]), int(lay["win_nsum"][w])
        if mask == "ct":
            ow, lw = A.prefill_window(lay, w, q, k, v, scale=0.7)
        else:
            ow, lw = A.kmer_local_window(lay, w, q, k, v, scale=0.7)
        rows = lay["sum_tok"][s0:s0 + B] - t0
        np.testing.assert_allclose(o[s0:s0 + B], ow[rows], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse[s0:s0 + B], lw[rows], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_zero_keys_one_hot_values_count_the_visible_set(seed):
    rng = np.random.default_rng(50 + seed)
    lay = _layout(rng)
    n = lay["n_tokens"]
    D = n                                          # one-hot value per token
    k = np.zeros((n, 1, D))
    v = np.eye(n)[:, None, :]
    q_sum = rng.standard_normal((lay["n_summaries"], 1, D))
    o_ct, _ = AD.adapter_attention(lay, q_sum, k, v, "ct")
    o_kl, _ = AD.adapter_attention(lay, q_sum, k, v, "kmer_local")
    for w in range(lay["n_windows"]):
        t0, C = int(lay["win_tok_off"][w]), int(lay["win_cache_off"][w])
        kw = int(lay["window_kmer"][w])
        cache_tok = A.cache_token_indices(lay, w)
        for j in range(int(lay["win_nsum"][w])):
            s = int(lay["win_sum_off"][w]) + j
            t = int(lay["sum_tok"][s])
            i = t - t0
            want = np.zeros(n)
            ct = list(cache_tok) + list(range(t0, t + 1))
            want[ct] = 1.0 / (C + i + 1)
            np.testing.assert_allclose(o_ct[s, 0], want, atol=1e-14)
            start = t0 + j * (kw + 1)              # the summary's own k-mer
            kl = list(range(start, t + 1)) + [t0 + (r + 1) * (kw + 1) - 1 for r in range(j)]
            if C > 0:
                kl.append(int(cache_tok[-1]))
            want = np.zeros(n)
            want[kl] = 1.0 / len(kl)
            np.testing.assert_allclose(o_kl[s, 0], want, atol=1e-14)


def test_identity_projections_give_the_attention():
    rng = np.random.default_rng(7)
    lay = _layout(rng)
    n, H, D = lay["n_tokens"], 2, 3
    hid = rng.standard_normal((n, H * D))
    eye = np.eye(H * D)
    h_new = AD.adapter_layer(lay, hid, eye, eye, eye, eye, H, H)
    x = hid.reshape(n, H, D)
    o, _ = AD.adapter_attention(lay, x[lay["sum_tok"]], x, x)
    np.testing.assert_allclose(h_new, o.reshape(-1, H * D), rtol=1e-12, atol=1e-12)


def test_linear_in_output_and_value_weights():
    rng = np.random.default_rng(8)
    lay = _layout(rng)
    n, d, H, D = lay["n_tokens"], 8, 2, 4
    hid = rng.standard_normal((n, d))
    wq, wk = rng.standard_normal((d, H * D)), rng.standard_normal((d, H * D))
    wv1, wv2 = rng.standard_normal((d, H * D)), rng.standard_normal((d, H * D))
    wo1, wo2 = rng.standard_normal((H * D, d)), rng.standard_normal((H * D, d))
    f = lambda wv, wo: AD.adapter_layer(lay, hid, wq, wk, wv, wo, H, H)   # noqa: E731
    np.testing.assert_allclose(f(wv1, wo1 + wo2), f(wv1, wo1) + f(wv1, wo2), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(f(wv1 + wv2, wo1), f(wv1, wo1) + f(wv2, wo1), rtol=1e-10, atol=1e-10)


def test_grouped_kv_heads_equal_repeated_heads():
    rng = np.random.default_rng(9)
    lay = _layout(rng)
    n, H, D = lay["n_tokens"], 4, 3
    q = rng.standard_normal((lay["n_summaries"], H, D))
    k, v = rng.standard_normal((n, 1, D)), rng.standard_normal((n, 1, D))
    o1, l1 = AD.adapter_attention(lay, q, k, v)
    o2, l2 = AD.adapter_attention(lay, q, np.repeat(k, H, 1), np.repeat(v, H, 1))
    np.testing.assert_allclose(o1, o2, rtol=1e-13)
    np.testing.assert_allclose(l1, l2, rtol=1e-13)


@pytest.mark.parametrize("mask", ["ct", "kmer_local"])
def test_causality_and_windows_without_summaries(mask):
    rng = np.random.default_rng(10)
    lay = build_layout([60], 20, np.array([6, 0, 4], np.int32))   # middle window: no summaries
    n, d, H, D = lay["n_tokens"], 6, 2, 3
    hid = rng.standard_normal((n, d))
    w = [rng.standard_normal((d, H * D)) for _ in range(3)] + [rng.standard_normal((H * D, d))]
    out = AD.adapter_layer(lay, hid, *w, H, H, mask)
    assert out.shape == (lay["n_summaries"], d) == (4 + 0 + 5, d)
    # a later token never changes an earlier summary's update
    for s in range(lay["n_summaries"]):
        t = int(lay["sum_tok"][s])
        if t + 1 >= n:
            continue
        hid2 = hid.copy()
        hid2[t + 1:] += rng.standard_normal((n - t - 1, d))
        out2 = AD.adapter_layer(lay, hid2, *w, H, H, mask)
        np.testing.assert_allclose(out2[:s + 1], out[:s + 1], rtol=1e-12, atol=1e-12)


def test_round_bf16_matches_torch():
    import torch
    rng = np.random.default_rng(11)
    x = np.concatenate([rng.standard_normal(10000) * 10.0 ** rng.integers(-8, 8, 10000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.01171875, 65504.0, 3e38]])
    want = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(AD.round_bf16(x), want)
