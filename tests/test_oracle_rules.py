"""Selection-rule variants of the oracle (App. selection-rule ablation):
pins of each rule's per-pair score and ranking against closed forms, and
the energy-retained / brute-force quality harness on a synthetic layer
(CPU only)."""
import numpy as np
import pytest

import workloads as W
from oracle import calib, carith, method

U32 = 2.0 ** -24
RULES = method.SCORE_RULES


def route_and_scores(inp, rule, budget, pred_b=None, pred_a=None):
    sh = inp["shape"]
    A = inp["pred_a"] if pred_a is None else pred_a
    b = inp["pred_b"] if pred_b is None else pred_b
    return method.decode_layer_c(inp["x"], inp["w_router"], inp["b_router"], A, b,
                                 sh.K, budget, score_rule=rule)


@pytest.fixture(scope="module")
def qwen():
    return W.layer_inputs("qwen3_b64", with_experts=False)


def test_top1_rule_keeps_the_top1_union(qwen):
    """Budget = |top-1 union| keeps exactly the experts some token ranks
    first; a larger budget puts every member first (index order), then the
    other routed experts by index."""
    o = route_and_scores(qwen, method.SCORE_TOP1, 1)
    top1 = sorted(set(o["topk_ids"][:, 0].tolist()))
    o = route_and_scores(qwen, method.SCORE_TOP1, len(top1))
    assert sorted(o["sel_ids"][:o["n_sel"]].tolist()) == top1
    assert list(o["sel_ids"][:o["n_sel"]]) == top1          # ties: index asc
    # D_u counts the tokens whose first route is u
    cnt = np.bincount(o["topk_ids"][:, 0], minlength=qwen["shape"].E)
    assert np.array_equal(o["scores"], cnt.astype(np.float32))
    big = len(top1) + 10
    o = route_and_scores(qwen, method.SCORE_TOP1, big)
    sel = o["sel_ids"][:o["n_sel"]].tolist()
    assert sel[:len(top1)] == top1
    rest = sel[len(top1):]
    assert rest == sorted(rest) and not set(rest) & set(top1)
    assert all(o["counts"][u] > 0 for u in rest)


def test_weight_rules_match_fp64_sums(qwen):
    """WEIGHT and WEIGHT_SQ batch scores are the sums of w and w^2 over the
    routing tokens, within the rounding of a B-term fp32 sum; with top-K
    normalised weights the WEIGHT scores add up to B."""
    B, E = qwen["x"].shape[0], qwen["shape"].E
    for rule, f in ((method.SCORE_WEIGHT, lambda w: w), (method.SCORE_WEIGHT_SQ, lambda w: w * w)):
        o = route_and_scores(qwen, rule, 8)
        w64 = o["topk_w"].astype(np.float64)
        D64 = np.zeros(E)
        np.add.at(D64, o["topk_ids"].ravel(), f(w64).ravel())
        assert np.all(np.abs(o["scores"] - D64) <= (B + 2) * U32 * np.abs(D64) + 1e-30)
        if rule == method.SCORE_WEIGHT:
            assert abs(o["scores"].astype(np.float64).sum() - B) < 1e-4
        # the ranking is the fp64 one wherever the fp64 gaps exceed the rounding
        srt = np.sort(D64[D64 > 0])[::-1]
        kth = srt[7]
        if srt[7] - srt[8] > 4 * (B + 2) * U32 * kth:
            assert set(o["sel_ids"][:8]) == set(np.argsort(-D64, kind="stable")[:8])


def test_static_rule_is_base_with_a_zero_slope(qwen):
    """STATIC scores w^2 exp(b_u) equal the predictor's canonical sequence
    with a_u = 0 bit for bit, and the fp64 definition within exp's error."""
    E, d = qwen["shape"].E, qwen["x"].shape[1]
    g = np.random.default_rng(3)
    logmu = (g.standard_normal(E) * 0.7 + 2.0).astype(np.float32)
    st = route_and_scores(qwen, method.SCORE_STATIC, 16, pred_b=logmu)
    base0 = route_and_scores(qwen, method.SCORE_BASE, 16, pred_b=logmu,
                             pred_a=np.zeros((E, d), np.float32))
    for f in ("cost", "scores", "sel_ids", "slot_of_expert", "exec_ids", "exec_gates"):
        assert np.array_equal(st[f], base0[f]), f
    c64 = method.pair_scores64(method.SCORE_STATIC, qwen["x"], None, logmu,
                               st["topk_ids"], st["topk_w"].astype(np.float64))
    assert np.max(np.abs(st["cost"] - c64) / c64) < 2e-6


def test_rules_share_routing_and_union(qwen):
    """Every rule routes the same way and keeps a subset of the same batch
    union; a budget covering the union keeps all of it under every rule."""
    outs = {r: route_and_scores(qwen, r, 200) for r in RULES}
    for r in RULES:
        assert np.array_equal(outs[r]["topk_ids"], outs[0]["topk_ids"])
        assert np.array_equal(outs[r]["counts"], outs[0]["counts"])
        assert set(outs[r]["sel_ids"][:outs[r]["n_sel"]]) == set(np.nonzero(outs[0]["counts"])[0])


@pytest.fixture(scope="module")
def harness():
    L = W.rules_layer()
    ex = method.Experts(L["w13"], L["w2"], False)
    A, b, _ = calib.fit_predictor(L["calib"], L["w_router"], L["b_router"], L["K"], ex)
    # static energy: each expert's mean output energy over the calibration
    # tokens that route it
    _, idz, _ = method.route64(L["calib"], L["w_router"], L["b_router"], L["K"])
    E = L["w_router"].shape[0]
    mu = np.array([np.mean(np.sum(ex.forward(u, L["calib"][np.any(idz == u, axis=1)]) ** 2,
                                  axis=1)) for u in range(E)])
    return L, ex, A, b, np.log(mu).astype(np.float32)


def test_energy_retained_by_rule(harness):
    """App. F: with the budget matched to the top-1 union, the fraction of
    the oracle-energy set's energy each rule keeps.  Every value lies in
    [0, 1]; ranking by the oracle energy itself keeps 1; on this layer the
    rules that see expert output energy (BASE, STATIC) keep clearly more
    than the router-only rules, the order the paper's ablation reports."""
    L, ex, A, b, logmu = harness
    K, E = L["K"], L["w_router"].shape[0]
    er = {r: [] for r in RULES}
    for x in L["batches"]:
        logits, ids, w = carith.route(x, L["w_router"], L["b_router"], K)
        eo = method.expert_outputs(ex, x, ids)
        Dstar = method.oracle_scores64(ids, w.astype(np.float64), np.sum(eo ** 2, axis=2), E)
        n = len(set(ids[:, 0].tolist()))
        ostar, _, _ = method.select(Dstar, np.bincount(ids.ravel(), minlength=E), n)
        assert method.energy_retained(Dstar, [u for u in ostar if u >= 0], n) == 1.0
        for r in RULES:
            o = method.decode_layer_c(x, L["w_router"], L["b_router"], A,
                                      logmu if r == method.SCORE_STATIC else b, K, n,
                                      score_rule=r)
            v = method.energy_retained(Dstar, [u for u in o["sel_ids"] if u >= 0], n)
            assert 0.0 <= v <= 1.0 + 1e-12
            er[r].append(v)
    m = {r: float(np.mean(v)) for r, v in er.items()}
    print("mean energy retained by rule:", {r: round(v, 4) for r, v in m.items()})
    router_only = max(m[method.SCORE_TOP1], m[method.SCORE_WEIGHT], m[method.SCORE_WEIGHT_SQ])
    assert m[method.SCORE_BASE] > router_only + 0.05
    assert m[method.SCORE_STATIC] > router_only + 0.05


def test_rule_sets_against_bruteforce(harness):
    """Exact batch error (eq. error_decomposition) of each rule's kept set
    never beats the brute-force optimum over all sets of that size."""
    L, ex, A, b, logmu = harness
    K, E = L["K"], L["w_router"].shape[0]
    for x in L["batches"][:4]:
        x = x[:6]
        logits, ids, w = carith.route(x, L["w_router"], L["b_router"], K)
        eo = method.expert_outputs(ex, x, ids)
        U = sorted(set(ids.ravel().tolist()))
        n = max(1, len(U) - 4)
        _, best = method.bruteforce_best(
            U, n, lambda S: method.exact_error64(ids, w.astype(np.float64), eo, S))
        for r in RULES:
            o = method.decode_layer_c(x, L["w_router"], L["b_router"], A,
                                      logmu if r == method.SCORE_STATIC else b, K, n,
                                      score_rule=r)
            S = [u for u in o["sel_ids"] if u >= 0]
            assert method.exact_error64(ids, w.astype(np.float64), eo, S) >= best - 1e-12
