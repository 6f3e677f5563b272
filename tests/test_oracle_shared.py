"""Shared experts in the oracle (always active, outside the budget; the
paper leaves them out of its notation, Sec. 3.1): the compaction layout,
the sigmoid gate, the cut of a wide shared expert into experts of the
routed width, and the layer output (CPU only)."""
import numpy as np

import workloads as W
from oracle import carith, method

U32 = 2.0 ** -24


def small(seed=0, B=12, d=256, E=8, K=2, I=64, S=2):
    g = np.random.default_rng(seed)
    x = g.standard_normal((B, d)).astype(np.float32)
    wr = (g.standard_normal((E, d)) * 0.1).astype(np.float32)
    w13 = (g.standard_normal((E, 2 * I, d)) / np.sqrt(d)).astype(np.float32)
    w2 = (g.standard_normal((E, d, I)) / np.sqrt(I)).astype(np.float32)
    s13 = (g.standard_normal((S, 2 * I, d)) / np.sqrt(d)).astype(np.float32)
    s2 = (g.standard_normal((S, d, I)) / np.sqrt(I)).astype(np.float32)
    gate = (g.standard_normal(d) / np.sqrt(d)).astype(np.float32)
    A = np.zeros((E, d), np.float32)
    b = np.zeros(E, np.float32)
    return x, wr, A, b, method.Experts(w13, w2, False), method.Experts(s13, s2, False), gate


def test_compaction_appends_shared_slots():
    x, wr, A, b, ex, sh, gate = small()
    B, K, budget = x.shape[0], 2, 3
    base = method.decode_layer_c(x, wr, None, A, b, K, budget)
    out = method.decode_layer_c(x, wr, None, A, b, K, budget,
                                shared=dict(experts=sh, gate=gate))
    # the routed plan is unchanged
    for f in ("sel_ids", "exec_ids", "exec_gates"):
        assert np.array_equal(out[f], base[f])
    P = int(base["offsets"][-1])
    assert np.array_equal(out["offsets"][:budget + 1], base["offsets"])
    assert list(out["offsets"][budget:]) == [P, P + B, P + 2 * B]
    assert np.array_equal(out["pair_tok"][:P], base["pair_tok"])
    for i in range(2):
        seg = slice(P + i * B, P + (i + 1) * B)
        assert np.array_equal(out["pair_tok"][seg], np.arange(B))
        assert np.array_equal(out["pair_gate"][seg], out["shared_gate"])
        assert np.array_equal(out["pair_of"][:, K + i], np.arange(P + i * B, P + (i + 1) * B))
    assert np.array_equal(out["pair_of"][:, :K], base["pair_of"])


def test_shared_gate_matches_fp64_sigmoid():
    inp = W.layer_inputs("qwen15_moe", with_experts=False)
    g = np.random.default_rng(4)
    gate = (g.standard_normal(2048) / np.sqrt(2048)).astype(np.float32)
    gc = method.shared_gate_c(inp["x"], gate)
    g64 = method.shared_gate64(inp["x"], gate)
    # dot product error (64-partial order) plus exp, add and divide rounding
    assert np.max(np.abs(gc - g64) / g64) < 1e-5
    assert np.all((gc > 0) & (gc < 1))


def test_wide_shared_expert_equals_its_cut():
    """A shared expert of intermediate size m I equals the sum of the m
    experts of width I cut from its gate rows, up rows and down columns
    (SwiGLU is separable over the intermediate index)."""
    g = np.random.default_rng(9)
    d, I, m = 256, 64, 4
    Wg = g.standard_normal((m * I, d)) / np.sqrt(d)
    Wu = g.standard_normal((m * I, d)) / np.sqrt(d)
    Wd = g.standard_normal((d, m * I)) / np.sqrt(m * I)
    z = g.standard_normal((5, d))
    wide = method.expert_forward64(z, np.concatenate([Wg, Wu]), Wd)
    parts = sum(method.expert_forward64(
        z, np.concatenate([Wg[i * I:(i + 1) * I], Wu[i * I:(i + 1) * I]]),
        Wd[:, i * I:(i + 1) * I]) for i in range(m))
    assert np.max(np.abs(wide - parts)) < 1e-12


def test_shared_output_adds_to_the_routed_output():
    x, wr, A, b, ex, sh, gate = small(3)
    K, budget = 2, 8
    r = np.random.default_rng(1).standard_normal(x.shape).astype(np.float32)
    base = method.decode_layer_c(x, wr, None, A, b, K, budget, ex, residual=r)
    for gv in (None, gate):
        out = method.decode_layer_c(x, wr, None, A, b, K, budget, ex, residual=r,
                                    shared=dict(experts=sh, gate=gv))
        gexp = np.ones(x.shape[0]) if gv is None else method.shared_gate64(x, gv)
        extra = sum(gexp[:, None] * method.expert_forward64(
            x.astype(np.float64), sh.w13(i), sh.w2(i)) for i in range(2))
        assert np.max(np.abs(out["y"] - base["y"] - extra)) < 1e-5
    # a budget covering the union: the dense MoE plus the shared experts
    out = method.decode_layer_c(x, wr, None, A, b, K, 8, ex, norm_topk=0,
                                shared=dict(experts=sh, gate=None))
    l64, ids, w = method.route64(x, wr, None, K, norm_topk=0)
    dense = method.moe_dense64(x, ids, w, ex)
    extra = sum(method.expert_forward64(x.astype(np.float64), sh.w13(i), sh.w2(i))
                for i in range(2))
    assert np.max(np.abs(out["y"] - dense - extra)) < 1e-5
