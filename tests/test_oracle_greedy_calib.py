"""Pins of two oracle functions against results fixed independently of
them: the greedy cross-term-aware selection (Sec. 3.3) against a
hand-derived case and the exhaustive search at n = 1, and the calibration
statistics (Sec. 3.4 target; App. A streaming statistics) against the
drop-the-expert identity and an expert with a closed-form output."""
import json
import math
import os

import numpy as np

import workloads as W
from oracle import calib, method

HERE = os.path.dirname(os.path.abspath(__file__))


def greedy_fixture():
    with open(os.path.join(HERE, "golden", "greedy_cross_example.json")) as f:
        g = json.load(f)
    ids = np.array(g["ids"], np.int32)
    w = np.array(g["w"], np.float64)
    eo = np.array(g["eo"], np.float64)
    return g, ids, w, eo


def test_greedy_cross_hand_derived_case():
    g, ids, w, eo = greedy_fixture()
    exp = g["expected"]
    for n in (1, 2, 3):
        A = method.greedy_cross(g["candidates"], n, ids, w, eo)
        assert A == exp["greedy"][n - 1], n                       # order of addition too
        err = method.exact_error64(ids, w, eo, A)
        assert abs(err - exp["greedy_error"][n - 1]) < 1e-12, n
        best, val = method.bruteforce_best(
            g["candidates"], n, lambda S: method.exact_error64(ids, w, eo, S))
        assert list(best) == exp["optimum"][n - 1] and abs(val - exp["optimum_error"][n - 1]) < 1e-12
    # the greedy set is not the additive one at any n here
    D = np.zeros(4)
    for t in range(ids.shape[0]):
        for k in range(ids.shape[1]):
            D[ids[t, k]] += (w[t, k] ** 2) * float(eo[t, k] @ eo[t, k])
    for n in (1, 2, 3):
        add = sorted(np.lexsort((np.arange(4), -D))[:n].tolist())
        assert add == exp["additive"][n - 1]
        assert sorted(exp["greedy"][n - 1]) != add


def rand_case(seed, B=5, E=7, K=3, d=6):
    g = np.random.default_rng(seed)
    ids = np.array([g.choice(E, K, replace=False) for _ in range(B)], np.int32)
    w = g.random((B, K))
    eo = g.standard_normal((B, K, d))
    return ids, w, eo


def test_greedy_cross_first_step_is_the_exhaustive_best_single_expert():
    """With n = 1 the greedy step is an exhaustive search over one expert,
    so it must equal the brute-force minimiser (ties: lower index)."""
    for seed in range(20):
        ids, w, eo = rand_case(seed)
        U = sorted(set(ids.ravel().tolist()))
        A = method.greedy_cross(U, 1, ids, w, eo)
        best, _ = method.bruteforce_best(U, 1, lambda S: method.exact_error64(ids, w, eo, S))
        assert A == list(best), seed


def test_greedy_cross_each_step_is_the_best_extension():
    """Step j adds the expert with the smallest exact error of the extended
    set among those not yet chosen (checked against an explicit scan)."""
    for seed in range(10):
        ids, w, eo = rand_case(100 + seed, B=6, E=9, K=4)
        U = sorted(set(ids.ravel().tolist()))
        n = len(U) - 2
        A = method.greedy_cross(U, n, ids, w, eo)
        for j in range(1, n + 1):
            prefix, nxt = A[:j - 1], A[j - 1]
            errs = {u: method.exact_error64(ids, w, eo, prefix + [u])
                    for u in U if u not in prefix}
            assert errs[nxt] == min(errs.values()), (seed, j)


# ------------------------------------------------------ calibration targets --
def expected_stats(z, w_router, b_router, K, experts, E):
    """Per expert: n, sum y, sum y^2, sum z_bar, sum z_bar y, with y taken
    from the drop-the-expert removal error: y = log(r / w^2 + eps), r the
    squared change of the MoE output when u is removed with weights fixed
    (Sec. 3.2, 3.4)."""
    _, ids, w = method.route64(z, w_router, b_router, K)
    r, _ = method.removal_error64(z, ids, w, experts)
    d = z.shape[1]
    out = {u: dict(n=0, sy=0.0, syy=0.0, sz=np.zeros(d), q=np.zeros(d)) for u in range(E)}
    for t in range(z.shape[0]):
        zb = z[t] / np.linalg.norm(z[t])
        for k in range(K):
            u = int(ids[t, k])
            y = math.log(r[t, k] / w[t, k] ** 2 + calib.EPS)
            e = out[u]
            e["n"] += 1
            e["sy"] += y
            e["syy"] += y * y
            e["sz"] += zb
            e["q"] += zb * y
    return out


def test_collect_stats_targets_follow_the_removal_error():
    """fp32 tiny layer, 300 calibration tokens in batches of 128 (ragged
    last batch): every expert's pair count equals the routed count, its
    target sums equal those of log(r / w^2 + eps) with r the true removal
    error, and the inputs are unit-norm rows (trace of the Gram = n)."""
    inp = W.layer_inputs("tiny")
    sh = inp["shape"]
    ex = method.Experts(inp["w13"], inp["w2"], False)
    z = W.calibration_tokens(sh, n=300).astype(np.float64)
    stats = calib.collect_stats(z, inp["w_router"], inp["b_router"], sh.K, ex, batch=128)
    ref = expected_stats(z, inp["w_router"], inp["b_router"], sh.K, ex, sh.E)
    _, ids, _ = method.route64(z, inp["w_router"], inp["b_router"], sh.K)
    counts = np.bincount(ids.ravel(), minlength=sh.E)
    assert np.linalg.norm(z, axis=1).min() > 2.0     # z_bar differs from z here
    for u in range(sh.E):
        st, e = stats[u], ref[u]
        assert st.n == e["n"] == counts[u], u
        if st.n == 0:
            continue
        scale = max(1.0, abs(e["sy"]))
        assert abs(st.sy - e["sy"]) <= 1e-9 * scale, u
        assert abs(st.syy - e["syy"]) <= 1e-9 * max(1.0, e["syy"]), u
        np.testing.assert_allclose(st.sz, e["sz"], rtol=1e-10, atol=1e-10)
        np.testing.assert_allclose(st.q, e["q"], rtol=1e-9, atol=1e-9 * scale)
        assert abs(float(np.trace(st.G.astype(np.float64))) - st.n) <= 1e-5 * st.n, u


def test_collect_stats_closed_form_expert():
    """Two experts, both routed by every token (K = E = 2), d = 4, I = 1.
    Expert 0 has gate row, up row and down column all e1, so
    E_0(z) = silu(z1) z1 e1 and y = log((z1^2 / (1 + exp(-z1)))^2 + eps);
    expert 1 is zero, so y = log(eps).  Evaluating the expert on z_bar
    instead of z, or mixing up the tokens, changes these values."""
    d, E = 4, 2
    w13 = np.zeros((E, 2, d), np.float32)
    w2 = np.zeros((E, d, 1), np.float32)
    w13[0, 0, 0] = w13[0, 1, 0] = 1.0
    w2[0, 0, 0] = 1.0
    ex = method.Experts(w13, w2, False)
    w_router = np.array([[0.1, 0.0, 0.0, 0.0], [0.0, 0.2, 0.0, 0.0]], np.float32)
    z = np.array([[2.0, 1.0, 0.0, 0.0], [-1.0, 0.0, 3.0, 0.0],
                  [0.5, 0.0, 0.0, 4.0], [3.0, 4.0, 0.0, 0.0], [0.0, 2.0, 2.0, 1.0]])
    stats = calib.collect_stats(z, w_router, None, 2, ex, batch=2)
    y0 = [math.log((s * s / (1.0 + math.exp(-s))) ** 2 + 1e-12) for s in z[:, 0]]
    zb = z / np.linalg.norm(z, axis=1, keepdims=True)
    assert stats[0].n == stats[1].n == 5
    assert abs(stats[0].sy - sum(y0)) < 1e-12
    assert abs(stats[0].syy - sum(v * v for v in y0)) < 1e-9
    np.testing.assert_allclose(stats[0].q, zb.T @ np.array(y0), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(stats[0].sz, zb.sum(axis=0), rtol=1e-12, atol=1e-14)
    assert abs(stats[1].sy - 5 * math.log(1e-12)) < 1e-9
    # the token with z1 = 0 has zero output energy: its target is log(eps)
    assert abs(y0[4] - math.log(1e-12)) < 1e-12
