"""Pins for the projection / rotary-position oracle:

* the rotation preserves each pair's norm and is the identity at position 0;
* for D = 2 the angle is the position itself (checked against math.cos/sin);
* relative positions: <rope(q, m), rope(k, n)> is unchanged when both positions
  shift by the same amount (the property rotary embeddings exist for);
* the projection without rotation is the matrix product split into heads;
* positions are the augmented-stream indices: a summary token's position is
  one past its k-mer's last base;
* store_bf16 equals rounding the float64 result with torch's bf16 conversion;
* D = 4: the second pair turns by pos / sqrt(theta); through the projection,
  token t of a single sequence turns by exactly t.
"""

import math

import numpy as np
import pytest

from oracle import projection as P
from oracle.layout import SUMMARY, build_layout


def test_norm_and_identity():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((50, 3, 8))
    pos = rng.integers(0, 10 ** 6, 50)
    y = P.rope(x, pos, 10000.0)
    np.testing.assert_allclose(np.hypot(y[..., 0::2], y[..., 1::2]), np.hypot(x[..., 0::2], x[..., 1::2]), rtol=1e-12)
    np.testing.assert_array_equal(P.rope(x, np.zeros(50), 10000.0), x)


def test_two_dims_angle_is_the_position():
    for p in (1, 7, 12345):
        y = P.rope(np.array([[[1.0, 0.0]]]), [p], 500.0)
        assert math.isclose(y[0, 0, 0], math.cos(p), abs_tol=1e-12)
        assert math.isclose(y[0, 0, 1], math.sin(p), abs_tol=1e-12)


@pytest.mark.parametrize("shift", [1, 100, 99999])
def test_relative_positions(shift):
    rng = np.random.default_rng(shift)
    q, k = rng.standard_normal((20, 1, 16)), rng.standard_normal((20, 1, 16))
    m, n = rng.integers(0, 5000, 20), rng.integers(0, 5000, 20)
    a = (P.rope(q, m, 10000.0) * P.rope(k, n, 10000.0)).sum(-1)
    b = (P.rope(q, m + shift, 10000.0) * P.rope(k, n + shift, 10000.0)).sum(-1)
    np.testing.assert_allclose(a, b, rtol=1e-9, atol=1e-9)


def test_projection_without_rotation_and_positions():
    rng = np.random.default_rng(1)
    lay = build_layout([37], 20, 6)
    n, d, H, Hkv, D = lay["n_tokens"], 8, 2, 1, 4
    hid = rng.standard_normal((n, d))
    w = rng.standard_normal((d, (H + 2 * Hkv) * D))
    q, k, v = P.qkv_project(lay, hid, w, H, Hkv, theta=0.0)
    y = hid @ w
    np.testing.assert_allclose(q.reshape(n, -1), y[:, :H * D], rtol=1e-12)
    np.testing.assert_allclose(v.reshape(n, -1), y[:, (H + Hkv) * D:], rtol=1e-12)
    # a summary's position is one past its k-mer's last base
    s = np.nonzero(lay["tok_kind"] == SUMMARY)[0]
    assert (lay["tok_pos"][s] == lay["tok_pos"][s - 1] + 1).all()
    assert lay["tok_pos"][s[0]] == 6


def test_store_bf16_matches_torch():
    import torch
    rng = np.random.default_rng(2)
    lay = build_layout([30], 30, 5)
    hid = rng.standard_normal((lay["n_tokens"], 8))
    w = rng.standard_normal((8, 4 * 4))
    q, _, _ = P.qkv_project(lay, hid, w, 2, 1, store_bf16=True)
    q64, _, _ = P.qkv_project(lay, hid, w, 2, 1)
    want = torch.from_numpy(q64.astype(np.float32)).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(q, want)


def test_second_pair_frequency():
    # D = 4: pair 1 turns by pos * theta^(-2/4) = pos / sqrt(theta)
    theta = 400.0
    for p in (3, 50, 777):
        y = P.rope(np.array([[[0.0, 0.0, 1.0, 0.0]]]), [p], theta)
        assert math.isclose(y[0, 0, 2], math.cos(p / 20.0), abs_tol=1e-12)
        assert math.isclose(y[0, 0, 3], math.sin(p / 20.0), abs_tol=1e-12)


def test_projection_rotates_at_the_stream_position():
    lay = build_layout([23], 10, 4)
    n = lay["n_tokens"]
    hid = np.ones((n, 1))
    w = np.array([[1.0, 0.0, 1.0, 0.0, 5.0, 6.0]])      # q = k = (1, 0) before rotation, D = 2
    q, k, v = P.qkv_project(lay, hid, w, 1, 1, theta=10000.0)
    for t in range(n):
        p = int(lay["tok_pos"][t])
        assert p == t                                  # one sequence: stream index
        np.testing.assert_allclose(q[t, 0], [math.cos(p), math.sin(p)], atol=1e-12)
        np.testing.assert_allclose(k[t, 0], [math.cos(p), math.sin(p)], atol=1e-12)
        np.testing.assert_allclose(v[t, 0], [5.0, 6.0])
