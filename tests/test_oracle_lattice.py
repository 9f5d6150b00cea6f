"""Pins of the oracle's lattice quantiser and field map (Section 3.2).

Brute force: for either coset, every D8 point within {-1, 0, 1}^8 of the
coordinate-wise rounding is enumerated.  That neighbourhood holds a nearest
point: if a nearest D8 point had a coordinate more than 1 away from y, moving
that coordinate by 2 towards y keeps the parity and strictly shortens the
distance.
"""
import itertools

import numpy as np
import pytest

OFFS = np.array(list(itertools.product((-1, 0, 1), repeat=8)), dtype=np.float64)


def brute_nearest_e8_dist(y):
    best = np.inf
    for shift in (0.0, 0.5):
        base = np.round(y - shift)
        cand = base[None, :] + OFFS
        cand = cand[(cand.sum(axis=1) % 2) == 0] + shift
        d = ((cand - y[None, :]) ** 2).sum(axis=1).min()
        best = min(best, d)
    return best


@pytest.mark.parametrize("scale", [0.3, 1.0, 3.0, 25.0])
def test_nearest_e8_matches_brute_force(oracle, scale):
    rng = np.random.default_rng(100 + int(scale * 10))
    y = rng.standard_normal((150, 8)) * scale
    tp, c = oracle.nearest_e8(y)
    for v in range(y.shape[0]):
        p = tp[v] / 2.0
        d = ((p - y[v]) ** 2).sum()
        assert d <= brute_nearest_e8_dist(y[v]) + 1e-12, (v, y[v], p)


def test_points_lie_on_e8(oracle):
    rng = np.random.default_rng(7)
    y = rng.standard_normal((5000, 8)) * rng.uniform(0.1, 40, size=(5000, 1))
    tp, c = oracle.nearest_e8(y)
    par = tp & 1
    # all coordinates integers (even 2p) or all half-integers (odd 2p), matching the coset
    assert np.all(par == c[:, None])
    # even coordinate sum on both cosets: sum(2p) = 2 sum(p) with sum(p) even
    assert np.all(tp.sum(axis=1) % 4 == 0)


def test_d8_tie_conventions(oracle):
    # coordinate ties round to even
    z = oracle.nearest_d8(np.array([0.5, 1.5, 2.5, -0.5, -1.5, 0, 0, 0]))
    assert z.tolist() == [[0, 2, 2, 0, -2, 0, 0, 0]]
    # odd sum, equal residuals: the first coordinate is moved
    z = oracle.nearest_d8(np.array([0.3, 0.3, 0, 0, 0, 0, 0, 1.0]))
    assert z.tolist() == [[1, 0, 0, 0, 0, 0, 0, 1]]
    # odd sum with zero residuals everywhere: first coordinate, sign(0) = +1
    z = oracle.nearest_d8(np.array([0, 0, 0, 0, 0, 0, 0, 1.0]))
    assert z.tolist() == [[1, 0, 0, 0, 0, 0, 0, 1]]
    # negative residual moves down
    z = oracle.nearest_d8(np.array([0, -0.4, 0, 0, 0, 0, 0, 1.0]))
    assert z.tolist() == [[0, -1, 0, 0, 0, 0, 0, 1]]


def test_coset_tie_prefers_integer_coset(oracle):
    # (1/4)^8 is at squared distance 1/2 from both 0 and (1/2)^8
    tp, c = oracle.nearest_e8(np.full(8, 0.25))
    assert c.tolist() == [0] and tp.tolist() == [[0] * 8]
    # just past the midpoint the half-integer coset wins
    tp, c = oracle.nearest_e8(np.full(8, 0.2500001))
    assert c.tolist() == [1] and tp.tolist() == [[1] * 8]


def test_field_map_round_trip(oracle):
    rng = np.random.default_rng(11)
    y = rng.standard_normal((20000, 8)) * rng.uniform(0.05, 200, size=(20000, 1))
    tp, c = oracle.nearest_e8(y)
    f = oracle.fields(tp)
    assert np.array_equal(f[:, 0], c)
    assert np.array_equal(oracle.points(f), tp)


def test_field_map_on_every_point_of_a_box(oracle):
    # every E8 point with coordinates in [-1.5, 1.5]
    pts = []
    for shift in (0.0, 0.5):
        vals = np.arange(-2, 3) + shift
        vals = vals[np.abs(vals) <= 1.5]
        for cand in itertools.product(vals, repeat=8):
            if sum(np.array(cand) - shift) % 2 == 0:
                pts.append(cand)
    tp = (2 * np.array(pts)).astype(np.int32)
    f = oracle.fields(tp)
    assert np.array_equal(oracle.points(f), tp)
    # z_i = p_i - c/2 for i <= 7 and m = (z8 - pi)/2 with pi = sum z_1..7 mod 2
    c = f[:, 0]
    z = (tp - c[:, None]) // 2
    assert np.array_equal(f[:, 1:8], z[:, :7])
    pi = z[:, :7].sum(axis=1) % 2
    assert np.array_equal(2 * f[:, 8] + pi, z[:, 7])
