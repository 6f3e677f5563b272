"""Pins of the oracle's method-level functions against the paper's
definitions, closed forms, invariants and brute force (CPU only)."""
import numpy as np
import pytest

import workloads as W
from oracle import carith, method, calib

U32 = 2.0 ** -24


def gamma(n):
    return n * U32 / (1 - n * U32)


def tiny(data_seed=0):
    inp = W.layer_inputs("tiny", data_seed=data_seed)
    ex = method.Experts(inp["w13"], inp["w2"], False)
    return inp, ex


@pytest.fixture(scope="module")
def tiny_fit():
    inp, ex = tiny()
    sh = inp["shape"]
    z = W.calibration_tokens(sh)
    A, b, info = calib.fit_predictor(z, inp["w_router"], inp["b_router"],
                                     sh.K, ex)
    return A, b


def rand_layer(seed, B=16, d=256, E=12, K=3, I=64):
    g = np.random.default_rng(seed)
    x = g.standard_normal((B, d)).astype(np.float32)
    wr = (g.standard_normal((E, d)) * 0.1).astype(np.float32)
    br = (g.standard_normal(E) * 0.3).astype(np.float32)
    w13 = (g.standard_normal((E, 2 * I, d)) / np.sqrt(d)).astype(np.float32)
    w2 = (g.standard_normal((E, d, I)) / np.sqrt(I)).astype(np.float32)
    return x, wr, br, method.Experts(w13, w2, False)


# ---------------------------------------------------------------- router ---
def test_route_c_matches_fp64_outside_error_bound():
    inp = W.layer_inputs("qwen3_b64", with_experts=False)
    x, wr, br = inp["x"], inp["w_router"], inp["b_router"]
    K = inp["shape"].K
    lc, idc, wc = carith.route(x, wr, br, K)
    l64, id64, w64 = method.route64(x, wr, br, K)
    bound = (gamma(2048 // 64 + 6) * (np.abs(x.astype(np.float64))
             @ np.abs(wr.astype(np.float64)).T) + 2 * U32 * np.abs(l64))
    assert np.all(np.abs(lc - l64) <= bound + 1e-30)
    checked = 0
    for t in range(x.shape[0]):
        srt = np.sort(l64[t])[::-1]
        gap = srt[K - 1] - srt[K]
        if gap > 2 * bound[t].max():
            checked += 1
            assert list(idc[t]) == list(id64[t])
    assert checked >= x.shape[0] - 2
    np.testing.assert_allclose(wc, w64, rtol=1e-5)


def test_route_weights_sum_to_one_and_descend():
    inp = W.layer_inputs("olmoe", with_experts=False)
    _, ids, w = carith.route(inp["x"], inp["w_router"], inp["b_router"], 8)
    s = w.astype(np.float64).sum(axis=1)
    assert np.all(np.abs(s - 1.0) <= 8 * 2 * U32 * 2)
    assert np.all(np.diff(w, axis=1) <= 0)
    assert all(len(set(r)) == 8 for r in ids)


def test_route_tie_break_lower_index():
    d, E = 256, 6
    x = np.ones((1, d), np.float32)
    wr = np.zeros((E, d), np.float32)   # all logits equal to the bias
    br = np.array([0.0, 1.0, 1.0, 0.5, 1.0, 0.5], np.float32)
    l, ids, w = carith.route(x, wr, br, 4)
    assert list(ids[0]) == [1, 2, 4, 3]
    assert w[0, 0] == w[0, 1] == w[0, 2]


def test_route_raw_softmax_mode():
    g = np.random.default_rng(4)
    x = g.standard_normal((5, 256)).astype(np.float32)
    wr = (g.standard_normal((70, 256)) * 0.1).astype(np.float32)
    _, ids, w0 = carith.route(x, wr, None, 4, norm_topk=0)
    _, _, w064 = method.route64(x, wr, None, 4, norm_topk=0)
    np.testing.assert_allclose(w0, w064, rtol=2e-6)
    assert np.all(w0.sum(axis=1) < 1.0)


# ------------------------------------------------------------- predictor ---
def _cost_bound(x, A, b, ids):
    """Relative error bound of the fp32 cost against its fp64 definition:
    the dot bounds (gamma_{d/64+6}) propagated through z_bar, s_hat = a.z_bar
    + b, exp (<= 2 ulp) and the two products."""
    x = np.asarray(x, np.float64)
    d = x.shape[1]
    gd = gamma(d // 64 + 6)
    nrm = np.linalg.norm(x, axis=1)
    absdot = np.einsum("td,tkd->tk", np.abs(x), np.abs(np.asarray(A, np.float64))[ids])
    dot = np.einsum("td,tkd->tk", x, np.asarray(A, np.float64)[ids])
    # |d(a.z)| <= gd*sum|x a|/|x| + |a.z| * (gd + 3u)   (||x|| via sqrt, 1/)
    ds = (gd * absdot / nrm[:, None] + np.abs(dot) / nrm[:, None] * (gd + 3 * U32)
          + 2 * U32 * (np.abs(dot) / nrm[:, None] + np.abs(np.asarray(b))[ids]))
    return np.expm1(ds) + 6 * U32


def test_predict_c_matches_fp64(tiny_fit):
    A, b = tiny_fit
    inp, _ = tiny()
    _, ids, w = carith.route(inp["x"], inp["w_router"], inp["b_router"], 2)
    c = carith.predict(inp["x"], A, b, ids, w)
    c64 = method.predict64(inp["x"], A, b, ids, w.astype(np.float64))
    assert np.all(np.abs(c - c64) <= _cost_bound(inp["x"], A, b, ids) * c64)


def test_predict_large_layer_relative_error():
    inp = W.layer_inputs("qwen3_b256", with_experts=False)
    _, ids, w = carith.route(inp["x"][:64], inp["w_router"], inp["b_router"], 8)
    c = carith.predict(inp["x"][:64], inp["pred_a"], inp["pred_b"], ids, w)
    c64 = method.predict64(inp["x"][:64], inp["pred_a"], inp["pred_b"], ids,
                           w.astype(np.float64))
    bound = _cost_bound(inp["x"][:64], inp["pred_a"], inp["pred_b"], ids)
    assert np.all(np.abs(c - c64) <= bound * c64)
    assert np.max(np.abs(c - c64) / c64) < 1e-4


def test_predict_zero_hidden_state_uses_bias_only():
    d, E = 256, 4
    x = np.zeros((1, d), np.float32)
    A = np.ones((E, d), np.float32)
    b = np.array([0.0, 1.0, -1.0, 2.0], np.float32)
    ids = np.array([[3, 1]], np.int32)
    w = np.array([[0.75, 0.25]], np.float32)
    c = carith.predict(x, A, b, ids, w)
    assert c[0, 0] == np.float32(0.5625) * carith.cexp(2.0)[0]
    assert c[0, 1] == np.float32(0.0625) * carith.cexp(1.0)[0]


def test_predict_depends_on_direction_only():
    g = np.random.default_rng(9)
    x = g.standard_normal((1, 512)).astype(np.float32)
    A = g.standard_normal((3, 512)).astype(np.float32) * 0.1
    b = np.zeros(3, np.float32)
    ids = np.array([[0, 2]], np.int32)
    w = np.array([[0.6, 0.4]], np.float32)
    c1 = carith.predict(x, A, b, ids, w)
    c2 = carith.predict(x * np.float32(4.0), A, b, ids, w)  # exact scaling
    assert np.array_equal(c1, c2)   # every step scales by a power of two


# ------------------------------------------------------------- aggregate ---
def test_aggregate_chunk_tree_order():
    B, K, E = 192, 1, 3
    ids = np.zeros((B, K), np.int32)
    ids[:, 0] = 2          # other tokens route expert 2 (cost 0 for them)
    cost = np.zeros((B, K), np.float32)
    # expert 0: chunk 0 holds 2^24 (pos 0), 1 (pos 1), 1 (pos 33)
    for t, v in [(0, 2.0 ** 24), (1, 1.0), (33, 1.0)]:
        ids[t, 0] = 0
        cost[t, 0] = v
    # expert 1: chunk sums 2^24, 1, 1 -> ((2^24 + 1) + 1) = 2^24
    for t, v in [(5, 2.0 ** 24), (64 + 7, 1.0), (128 + 9, 1.0)]:
        ids[t, 0] = 1
        cost[t, 0] = v
    scores, counts = carith.aggregate(ids, cost, E)
    # tree inside chunk 0: h=32 gives s1 = 1 + 1 = 2, then s0 + 2 at h=1
    assert scores[0] == 2.0 ** 24 + 2.0
    # sequential over chunks: each +1 is a tie rounded to even
    assert scores[1] == 2.0 ** 24
    assert list(counts) == [3, 3, B - 6]


def test_aggregate_matches_fp64_and_counts():
    inp = W.layer_inputs("qwen3_b256", with_experts=False)
    x = inp["x"]
    _, ids, w = carith.route(x, inp["w_router"], inp["b_router"], 8)
    c = carith.predict(x, inp["pred_a"], inp["pred_b"], ids, w)
    s, n = carith.aggregate(ids, c, 128)
    s64, n64 = method.aggregate64(ids, c, 128)
    assert list(n) == list(n64)
    assert np.all(np.abs(s - s64) <= gamma(256 // 64 + 6) * s64 + 1e-30)


# ------------------------------------------------------------- selection ---
def test_select_additive_optimum_by_bruteforce():
    g = np.random.default_rng(0)
    for trial in range(20):
        E = 9
        D = g.random(E)
        counts = (g.random(E) < 0.8).astype(np.int32)
        counts[0] = 1
        for budget in [1, 3, 5, 12]:
            sel, n_sel, slot = method.select(D, counts, budget)
            U = [u for u in range(E) if counts[u] > 0]
            assert n_sel == min(budget, len(U))
            best, _ = method.bruteforce_best(
                U, n_sel, lambda A: method.additive_error64(
                    np.where(counts > 0, D, 0.0), A))
            assert sorted(sel[:n_sel]) == list(best)
            assert all(counts[u] > 0 for u in sel[:n_sel])
            assert np.all(sel[n_sel:] == -1)
            for r, u in enumerate(sel[:n_sel]):
                assert slot[u] == r
            assert (slot >= 0).sum() == n_sel


def test_select_ties_go_to_lower_index():
    D = np.array([1.0, 2.0, 2.0, 0.5, 2.0], np.float32)
    counts = np.ones(5, np.int32)
    sel, n, _ = method.select(D, counts, 3)
    assert list(sel) == [1, 2, 4]


# --------------------------------------------------------------- backfill ---
def _check_backfill(logits, ids, slot, n_sel, K, ex, n_ex):
    for t in range(len(ids)):
        X = list(ex[t, :n_ex[t]])
        assert n_ex[t] == min(K, n_sel)
        assert all(slot[u] >= 0 for u in X)
        kept = [u for u in ids[t] if slot[u] >= 0]
        assert X[:len(kept)] == kept          # retained routes come first
        # everything executed ranks above every retained, unexecuted expert
        rest = [u for u in range(len(slot)) if slot[u] >= 0 and u not in X]
        for u in X:
            for v in rest:
                assert (logits[t, u] > logits[t, v]) or (
                    logits[t, u] == logits[t, v] and u < v)


@pytest.mark.parametrize("budget", [1, 2, 3, 5, 8])
def test_backfill_invariants(budget):
    x, wr, br, ex_ = rand_layer(1)
    l, ids, w = carith.route(x, wr, br, 3)
    g = np.random.default_rng(budget)
    D = g.random(12).astype(np.float32)
    _, counts = carith.aggregate(ids, np.ones_like(w), 12)
    sel, n_sel, slot = method.select(D, counts, budget)
    ex, n_ex = method.backfill(l, ids, slot, n_sel, 3)
    _check_backfill(l, ids, slot, n_sel, 3, ex, n_ex)


def test_drop_mode_keeps_only_retained_routes():
    x, wr, br, _ = rand_layer(2)
    l, ids, w = carith.route(x, wr, br, 3)
    _, counts = carith.aggregate(ids, np.ones_like(w), 12)
    sel, n_sel, slot = method.select(np.arange(12, 0, -1.0), counts, 4)
    ex, n_ex = method.backfill(l, ids, slot, n_sel, 3, method.FILL_DROP)
    for t in range(len(ids)):
        assert list(ex[t, :n_ex[t]]) == [u for u in ids[t] if slot[u] >= 0]


def test_paper_gates_equal_router_weights_and_sum_below_one():
    x, wr, br, _ = rand_layer(3)
    l, ids, w = carith.route(x, wr, br, 3)
    _, counts = carith.aggregate(ids, np.ones_like(w), 12)
    sel, n_sel, slot = method.select(np.arange(12, 0, -1.0), counts, 5)
    ex, n_ex = method.backfill(l, ids, slot, n_sel, 3)
    gt = method.gates_c(l, ids, ex, n_ex)
    for t in range(len(ids)):
        for j in range(n_ex[t]):
            u = ex[t, j]
            if u in ids[t]:
                assert gt[t, j] == w[t, list(ids[t]).index(u)]   # bit-exact
        s = float(gt[t, :n_ex[t]].astype(np.float64).sum())
        if set(ex[t, :n_ex[t]]) == set(ids[t]):
            assert abs(s - 1.0) < 1e-6
        else:
            assert s < 1.0
    gr = method.gates_c(l, ids, ex, n_ex, flags=method.GATE_RENORM)
    assert np.all(np.abs(gr.astype(np.float64).sum(axis=1) - 1.0) < 1e-6)
    g64 = method.gates64(l, ids, ex, n_ex)
    np.testing.assert_allclose(gt, g64, rtol=2e-6)


def test_dense_equivalence_when_budget_covers_union():
    x, wr, br, ex_ = rand_layer(4)
    A = np.zeros((12, 256), np.float32)
    b = np.zeros(12, np.float32)
    out = method.decode_layer_c(x, wr, br, A, b, 3, 12, ex_)
    assert out["n_sel"] == int((out["counts"] > 0).sum())
    assert np.array_equal(out["exec_ids"], out["topk_ids"])
    assert np.array_equal(out["exec_gates"], out["topk_w"])
    y_dense = method.moe_dense64(x, out["topk_ids"], out["topk_w"], ex_)
    np.testing.assert_allclose(out["y"], y_dense, rtol=1e-12, atol=1e-12)


def test_compaction_is_counting_sort():
    x, wr, br, _ = rand_layer(5, B=40)
    l, ids, w = carith.route(x, wr, br, 3)
    _, counts = carith.aggregate(ids, np.ones_like(w), 12)
    sel, n_sel, slot = method.select(np.arange(12.0), counts, 6)
    ex, n_ex = method.backfill(l, ids, slot, n_sel, 3)
    g = method.gates_c(l, ids, ex, n_ex)
    off, ptok, pg, pof = method.compact(ex, n_ex, slot, g, 6)
    assert off[0] == 0 and off[-1] == n_ex.sum()
    assert np.all(np.diff(off) >= 0)
    for s in range(6):
        toks = list(ptok[off[s]:off[s + 1]])
        assert toks == sorted(toks)
        expect = [t for t in range(40) if sel[s] >= 0 and sel[s] in ex[t, :n_ex[t]]]
        assert toks == expect
    for t in range(40):
        for j in range(3):
            p = pof[t, j]
            if j < n_ex[t]:
                assert ptok[p] == t and pg[p] == g[t, j]
                assert off[slot[ex[t, j]]] <= p < off[slot[ex[t, j]] + 1]
            else:
                assert p == -1


# --------------------------------------------------- removal error, errors ---
def test_removal_error_equals_weighted_energy():
    x, wr, br, ex_ = rand_layer(6)
    _, ids, w = method.route64(x, wr, br, 3)
    r, energy = method.removal_error64(x, ids, w, ex_)
    np.testing.assert_allclose(r, w ** 2 * energy, rtol=1e-12)


def test_exact_error_bruteforce_and_greedy_and_additive():
    for seed in range(6):
        x, wr, br, ex_ = rand_layer(10 + seed, B=6, E=8, K=3)
        _, ids, w = method.route64(x, wr, br, 3)
        eo = method.expert_outputs(ex_, x, ids)
        r, energy = method.removal_error64(x, ids, w, ex_, eo)
        D = method.oracle_scores64(ids, w, energy, 8)
        U = sorted(set(ids.ravel().tolist()))
        n = max(1, len(U) - 3)
        Astar, Estar = method.bruteforce_best(
            U, n, lambda A: method.exact_error64(ids, w, eo, A))
        sel, n_sel, _ = method.select(D, np.bincount(ids.ravel(), minlength=8), n)
        A_add = list(sel[:n_sel])
        A_gr = method.greedy_cross(U, n, ids, w, eo)
        E_add = method.exact_error64(ids, w, eo, A_add)
        E_gr = method.exact_error64(ids, w, eo, A_gr)
        assert Estar <= E_add + 1e-12 and Estar <= E_gr + 1e-12
        # additive error identity: cross terms are what separates the two
        assert abs(method.additive_error64(D, A_add)
                   - sum(D[u] for u in U if u not in A_add)) < 1e-12
        # budget covering the union: zero error
        assert method.exact_error64(ids, w, eo, U) == 0.0


def test_drop_mode_output_error_equals_exact_error():
    x, wr, br, ex_ = rand_layer(7, B=10)
    A_ = np.zeros((12, 256), np.float32)
    b_ = np.zeros(12, np.float32)
    out = method.decode_layer_c(x, wr, br, A_, b_, 3, 4, ex_,
                                flags=method.FILL_DROP)
    ids, w = out["topk_ids"], out["topk_w"].astype(np.float64)
    y_dense = method.moe_dense64(x, ids, w, ex_)
    eo = method.expert_outputs(ex_, x, ids)
    A = [u for u in out["sel_ids"] if u >= 0]
    err = float(np.sum((out["y"] - y_dense) ** 2))
    assert abs(err - method.exact_error64(ids, w, eo, A)) <= 1e-9 * max(1.0, err)


def test_crossterm_identity():
    g = np.random.default_rng(8)
    for m in range(1, 8):
        for _ in range(20):
            a = g.standard_normal((m, 32)) * g.random((m, 1)) * 3
            rho, cbar, ueff = method.crossterm_stats(a)
            assert abs((rho - 1) - cbar * (ueff - 1)) < 1e-10
            assert 1 - 1e-12 <= ueff <= m + 1e-12
            if m == 1:
                assert abs(rho - 1) < 1e-15
    # equal magnitudes: |U|_eff = |U|; orthogonal: rho = 1
    a = np.eye(5) * 2.0
    rho, cbar, ueff = method.crossterm_stats(a)
    assert abs(ueff - 5) < 1e-12 and abs(rho - 1) < 1e-12 and abs(cbar) < 1e-12


def test_energy_retained_bounds():
    g = np.random.default_rng(12)
    D = g.random(20)
    order = sorted(range(20), key=lambda u: -D[u])
    assert method.energy_retained(D, order[:7], 7) == 1.0
    for _ in range(20):
        A = g.choice(20, 7, replace=False)
        er = method.energy_retained(D, A, 7)
        assert 0.0 <= er <= 1.0


# ----------------------------------------------------------------- experts ---
def test_swiglu_expert_closed_form():
    d, I = 4, 2
    w13 = np.zeros((2 * I, d), np.float32)
    w13[0, 0] = 1.0     # gate_0 = z0
    w13[2, 1] = 1.0     # up_0 = z1
    w2 = np.zeros((d, I), np.float32)
    w2[3, 0] = 2.0      # out_3 = 2 * h_0
    z = np.array([[1.5, -2.0, 0.0, 0.0]])
    out = method.expert_forward64(z, w13, w2)
    h0 = 1.5 / (1 + np.exp(-1.5)) * -2.0
    np.testing.assert_allclose(out[0], [0, 0, 0, 2 * h0], rtol=1e-15)


def test_bf16_rounding_ties_to_even():
    v = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5],
                 np.float32)
    r = method.bf16_round(v)
    assert list(r) == [1.0, 1.0 + 2 ** -6, 1.0, -2.5]
