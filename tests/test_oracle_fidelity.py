"""Pins for the fidelity-metric oracle (Appendix "Metrics"):

* library routines: SciPy's Jensen-Shannon distance (squared) and relative
  entropy, NumPy's norms, on the clipped and renormalised inputs;
* the two Hellinger forms the appendix prints agree;
* closed forms: identical inputs give zero everywhere; two point masses on
  different categories (after the 1e-12 clip) give L1 = 2(1-c)/(1+c),
  L2 = sqrt 2 (1-c)/(1+c), KL = (1-c)/(1+c) log(1/c) with c = 1e-12, JS and
  Hellinger from their definitions written out for two categories; a point
  mass against the uniform distribution gives L1 = 2(1 - 1/V);
* bounds and symmetry: 0 <= H <= 1, 0 <= JS <= log 2, L1 <= 2, KL >= 0;
  L1, L2, H, JS symmetric;
* softmax: invariant to a shift of the logits, uniform logits give 1/V;
* clipping: rows sum to one and no entry is below the clip after it.
"""

import math

import numpy as np
import pytest
from scipy.spatial.distance import jensenshannon
from scipy.stats import entropy

from oracle import fidelity as FD

C = 1e-12


def _dists(rng, n, V, peaky=False):
    x = rng.standard_normal((n, V)) * (6.0 if peaky else 1.0)
    return FD.softmax(x)


@pytest.mark.parametrize("V", [2, 4, 17, 512])
def test_against_library_routines(V):
    rng = np.random.default_rng(V)
    p, q = _dists(rng, 50, V), _dists(rng, 50, V, peaky=True)
    m = FD.metrics(p, q)
    pc, qc = FD.clip_renormalise(p), FD.clip_renormalise(q)
    for i in range(len(p)):
        assert math.isclose(m[i, 0], np.linalg.norm(pc[i] - qc[i], 1), rel_tol=1e-12)
        assert math.isclose(m[i, 1], np.linalg.norm(pc[i] - qc[i], 2), rel_tol=1e-12)
        assert math.isclose(m[i, 3], jensenshannon(pc[i], qc[i]) ** 2, rel_tol=1e-9, abs_tol=1e-15)
        assert math.isclose(m[i, 4], entropy(pc[i], qc[i]), rel_tol=1e-12, abs_tol=1e-15)


def test_hellinger_forms_agree():
    rng = np.random.default_rng(1)
    p, q = _dists(rng, 100, 9), _dists(rng, 100, 9, peaky=True)
    pc, qc = FD.clip_renormalise(p), FD.clip_renormalise(q)
    other = np.sqrt(1.0 - np.sqrt(pc * qc).sum(axis=1))
    np.testing.assert_allclose(FD.metrics(p, q)[:, 2], other, rtol=1e-9, atol=1e-12)


def test_identical_inputs_are_zero():
    rng = np.random.default_rng(2)
    p = _dists(rng, 20, 6)
    np.testing.assert_allclose(FD.metrics(p, p), 0.0, atol=1e-15)


def test_point_masses_closed_forms():
    p, q = np.array([[1.0, 0.0]]), np.array([[0.0, 1.0]])
    a, b = 1 / (1 + C), C / (1 + C)                 # clipped, renormalised masses
    m = FD.metrics(p, q)[0]
    assert math.isclose(m[0], 2 * (1 - C) / (1 + C), rel_tol=1e-14)
    assert math.isclose(m[1], math.sqrt(2) * (1 - C) / (1 + C), rel_tol=1e-14)
    assert math.isclose(m[4], (1 - C) / (1 + C) * math.log(1 / C), rel_tol=1e-12)
    assert math.isclose(m[2], math.sqrt(((math.sqrt(a) - math.sqrt(b)) ** 2) * 2 / 2), rel_tol=1e-12)
    half = (a + b) / 2
    js = 0.5 * (a * math.log(a / half) + b * math.log(b / half)) * 2
    assert math.isclose(m[3], js, rel_tol=1e-12)
    assert abs(m[3] - math.log(2)) < 1e-9


@pytest.mark.parametrize("V", [2, 4, 64])
def test_point_mass_against_uniform(V):
    p = np.zeros((1, V))
    p[0, 0] = 1.0
    q = np.full((1, V), 1.0 / V)
    assert math.isclose(FD.metrics(p, q)[0, 0], 2 * (1 - 1 / V), rel_tol=1e-9)


def test_bounds_and_symmetry():
    rng = np.random.default_rng(3)
    p, q = _dists(rng, 200, 5, peaky=True), _dists(rng, 200, 5, peaky=True)
    m, mt = FD.metrics(p, q), FD.metrics(q, p)
    assert (m[:, 0] <= 2 + 1e-12).all() and (m[:, 2] >= 0).all() and (m[:, 2] <= 1 + 1e-12).all()
    assert (m[:, 3] >= -1e-15).all() and (m[:, 3] <= math.log(2) + 1e-12).all()
    assert (m[:, 4] >= -1e-15).all()
    np.testing.assert_allclose(m[:, :4], mt[:, :4], rtol=1e-12, atol=1e-15)


def test_softmax_and_clipping():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((10, 7))
    np.testing.assert_allclose(FD.softmax(x), FD.softmax(x + 123.0), rtol=1e-12)
    np.testing.assert_allclose(FD.softmax(np.zeros((3, 5))), 0.2)
    p = np.array([[0.5, 0.5, 0.0, 0.0]])
    pc = FD.clip_renormalise(p)
    assert math.isclose(pc.sum(), 1.0, rel_tol=1e-15) and pc.min() >= C / (1 + 2 * C) * 0.999


def test_sequence_means():
    rng = np.random.default_rng(5)
    per = rng.random((10, 5))
    cu = [0, 3, 3, 10]
    got = FD.sequence_means(per, cu)
    np.testing.assert_allclose(got[0], per[:3].mean(0))
    np.testing.assert_allclose(got[1], 0.0)
    np.testing.assert_allclose(got[2], per[3:].mean(0))
