"""Pins of the oracle's canonical fp32 arithmetic (oracle/carith.c) against
facts fixed outside it: exact results on exactly representable cases,
hand-derived consequences of the stated reduction order, the IEEE
single-rounding property of FMA, and standard floating-point error bounds."""
import math

import numpy as np
import pytest

from oracle import carith

U32 = 2.0 ** -24    # unit roundoff of binary32


def gamma(n):
    return n * U32 / (1 - n * U32)


# ------------------------------------------------------------------ cexp ---
def test_cexp_ulp_bound_dense_sweep():
    x = np.linspace(-86.0, 88.0, 3_000_001, dtype=np.float32)
    y = carith.cexp(x).astype(np.float64)
    ref = np.exp(x.astype(np.float64))
    ulp = np.spacing(ref.astype(np.float32)).astype(np.float64)
    err = np.abs(y - ref) / ulp
    assert err.max() <= 2.0, err.max()


def test_cexp_special_values():
    assert carith.cexp(0.0)[0] == 1.0
    # near multiples of ln 2 (range-reduction boundaries): within 2 ulp
    for n in range(-124, 127):
        for off in (-1, 0, 1):
            x = np.nextafter(np.float32(n * math.log(2)), np.float32(off * 1e9)) \
                if off else np.float32(n * math.log(2))
            v = float(carith.cexp(x)[0])
            ref = math.exp(float(x))
            assert abs(v - ref) <= 2 * float(np.spacing(np.float32(ref)))
    # clamp to [-86, 88]
    assert carith.cexp(-1000.0)[0] == carith.cexp(-86.0)[0]
    assert carith.cexp(1000.0)[0] == carith.cexp(88.0)[0]
    assert np.isfinite(carith.cexp(88.0)[0])
    assert carith.cexp(-86.0)[0] >= np.finfo(np.float32).tiny


def test_cexp_monotone_on_grid():
    x = np.linspace(-20, 20, 400_001, dtype=np.float32)
    y = carith.cexp(x)
    assert np.all(np.diff(y) >= 0)


# ------------------------------------------------------------------ cdot ---
@pytest.mark.parametrize("d", [256, 2048, 4096])
def test_cdot_exact_on_small_integers(d):
    g = np.random.default_rng(d)
    p = g.integers(-8, 9, d).astype(np.float32)
    q = g.integers(-8, 9, d).astype(np.float32)
    # every partial sum is an integer below 2^24: no rounding anywhere
    assert float(carith.cdot(p, q)) == float(p.astype(np.int64) @ q.astype(np.int64))


def test_cdot_one_hot_picks_element():
    g = np.random.default_rng(3)
    q = g.standard_normal(2048).astype(np.float32)
    for k in [0, 1, 5, 255, 256, 1000, 2047]:
        p = np.zeros(2048, np.float32)
        p[k] = 1.0
        assert carith.cdot(p, q) == q[k]


def test_cdot_tree_pairs_lane_j_with_lane_j_plus_32_first():
    # element k belongs to partial sum (k mod 256) // 4.
    p = np.zeros(256, np.float32)
    q = np.ones(256, np.float32)
    p[0] = 2.0 ** 24      # partial 0
    p[4] = 1.0            # partial 1
    p[128] = -2.0 ** 24   # partial 32
    # step h=32: s0 = 2^24 + (-2^24) = 0, s1 = 1 ; final 0 + 1 = 1.
    # (a left-to-right sum would give (2^24 + 1) - 2^24 = 0)
    assert carith.cdot(p, q) == 1.0


def test_cdot_tree_adds_lane_one_last():
    p = np.zeros(256, np.float32)
    q = np.ones(256, np.float32)
    p[0] = 2.0 ** 24      # partial 0
    p[128] = 1.0          # partial 32
    p[4] = -2.0 ** 24     # partial 1
    # h=32: s0 = 2^24 + 1 -> 2^24 (tie to even), s1 = -2^24;
    # h=16..2 add zeros; h=1: s0 = 2^24 - 2^24 = 0.
    # (pairing adjacent partials first would give 0 + 1 = 1)
    assert carith.cdot(p, q) == 0.0


def test_cdot_partial_owns_groups_of_four_strided_by_256():
    p = np.zeros(512, np.float32)
    q = np.ones(512, np.float32)
    p[3] = 2.0 ** 24      # partial 0 (k=3)
    p[256] = 1.0          # partial 0 again (k=256): 2^24 + 1 -> 2^24
    p[4] = 1.0            # partial 1
    # partial 0 = 2^24 after its chain; partial 1 = 1; result 2^24 + 1 -> 2^24
    assert carith.cdot(p, q) == 2.0 ** 24
    p[4] = 0.0
    p[7] = 1.0            # still partial 1 (k=7)
    assert carith.cdot(p, q) == 2.0 ** 24
    p[7] = 0.0
    p[8] = 3.0            # partial 2: tree gives (2^24) + 3 at h=2 -> exact
    assert carith.cdot(p, q) == 2.0 ** 24 + 4.0  # 2^24+3 rounds to even


def test_cdot_uses_single_rounding_fma():
    a = np.float32(1.0 + 2.0 ** -12)
    p = np.zeros(256, np.float32)
    q = np.zeros(256, np.float32)
    p[0], q[0] = a, a         # acc = fl(a*a) = 1 + 2^-11 (tie to even)
    p[1], q[1] = -a, a        # fused: fl(acc - a*a) = -2^-24 ; unfused: 0
    assert carith.cdot(p, q) == np.float32(-2.0 ** -24)


@pytest.mark.parametrize("d", [256, 2048])
def test_cdot_error_bound(d):
    g = np.random.default_rng(11)
    P = g.standard_normal((64, d)).astype(np.float32)
    Q = g.standard_normal((64, d)).astype(np.float32)
    got = carith.cdot_matrix(P, Q).astype(np.float64)
    exact = P.astype(np.float64) @ Q.astype(np.float64).T
    absd = np.abs(P.astype(np.float64)) @ np.abs(Q.astype(np.float64)).T
    bound = gamma(d // 64 + 6) * absd
    assert np.all(np.abs(got - exact) <= bound)


def test_cdot_is_order_sensitive():
    # negative control: reordering the elements changes low bits on some
    # inputs, so bit-exact comparisons against this order are meaningful.
    g = np.random.default_rng(5)
    diff = 0
    for _ in range(50):
        p = g.standard_normal(2048).astype(np.float32)
        q = g.standard_normal(2048).astype(np.float32)
        perm = g.permutation(2048)
        diff += carith.cdot(p, q) != carith.cdot(p[perm], q[perm])
    assert diff > 0


def test_cdot_matrix_equals_single_calls():
    g = np.random.default_rng(2)
    P = g.standard_normal((3, 512)).astype(np.float32)
    Q = g.standard_normal((4, 512)).astype(np.float32)
    M = carith.cdot_matrix(P, Q)
    for i in range(3):
        for e in range(4):
            assert M[i, e] == carith.cdot(P[i], Q[e])
