"""GPU parity of the HIP path (called through the C ABI) against the CPU
oracle on the same seeded inputs.

Bar: route logits / ids / weights, predicted costs, batch scores, counts,
the kept set, slots, executed experts, gates and the compaction are
bit-exact with the oracle's canonical fp32 level; costs are also within
1e-4 relative of the fp64 definition; the layer output is within 2e-2
max-abs (bf16) or 1e-5 (fp32) of the oracle's fp64 restricted MoE.
"""
import numpy as np
import pytest

import workloads as W
from oracle import calib, carith, method

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

Y_TOL = {True: 2e-2, False: 1e-5}


def _flush(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module")
def gu(gpu):
    import gpu_util
    return gpu_util


_TINY_PRED = {}


def tiny_predictor(inp):
    if "p" not in _TINY_PRED:
        ex = method.Experts(inp["w13"], inp["w2"], False)
        z = W.calibration_tokens(inp["shape"])
        A, b, _ = calib.fit_predictor(z, inp["w_router"], inp["b_router"],
                                      inp["shape"].K, ex)
        _TINY_PRED["p"] = (A, b)
    return _TINY_PRED["p"]


def named(name, data_seed=0, with_experts=True):
    inp = W.layer_inputs(name, data_seed=data_seed, with_experts=with_experts)
    if name == "tiny":
        inp["pred_a"], inp["pred_b"] = tiny_predictor(inp)
    return inp


def oracle_layer(inp, budget, flags=0, norm_topk=1, residual=None,
                 with_y=True, score_rule=0):
    sh = inp["shape"]
    ex = method.Experts(inp["w13"], inp["w2"], sh.bf16) if with_y else None
    shared = None
    if inp.get("w13_shared") is not None:
        shared = dict(experts=method.Experts(inp["w13_shared"], inp["w2_shared"], True),
                      gate=inp.get("shared_gate"))
    return method.decode_layer_c(inp["x"], inp["w_router"], inp["b_router"],
                                 inp["pred_a"], inp["pred_b"], sh.K, budget,
                                 ex, norm_topk, flags, residual, score_rule, shared)


def check_scoring(gl, inp, ref, B, budget, score_rule=0):
    """Staged route / predict / select against the oracle, bit for bit."""
    x = gl.x(inp["x"])
    logits, ids, w = gl.route(x, B)
    assert np.array_equal(logits.cpu().numpy(), ref["logits"])
    assert np.array_equal(ids.cpu().numpy(), ref["topk_ids"])
    assert np.array_equal(w.cpu().numpy(), ref["topk_w"])
    cost = gl.predict(x, B, ids, w)
    c = cost.cpu().numpy()
    assert np.array_equal(c, ref["cost"])
    c64 = method.pair_scores64(score_rule, inp["x"], inp["pred_a"], inp["pred_b"],
                               ref["topk_ids"], ref["topk_w"].astype(np.float64))
    assert np.max(np.abs(c - c64) / np.where(c64 > 0, c64, 1.0)) < 1e-4
    scores, counts, sel, nsel, slot = gl.select(B, ids, cost, budget)
    assert np.array_equal(scores.cpu().numpy(), ref["scores"])
    assert np.array_equal(counts.cpu().numpy(), ref["counts"])
    assert int(nsel.item()) == ref["n_sel"]
    assert np.array_equal(sel.cpu().numpy(), ref["sel_ids"])
    assert np.array_equal(slot.cpu().numpy(), ref["slot_of_expert"])
    return x, logits, ids, w, cost, sel, nsel, slot


def check_plan(got, ref):
    assert np.array_equal(got["exec_ids"], ref["exec_ids"])
    assert np.array_equal(got["exec_gates"], ref["exec_gates"])
    assert np.array_equal(got["offsets"], ref["offsets"])
    assert np.array_equal(got["pair_tok"], ref["pair_tok"])
    assert np.array_equal(got["pair_gate"], ref["pair_gate"])
    assert np.array_equal(got["pair_of"], ref["pair_of"])


def run_case(gu, inp, budget, flags=0, norm_topk=1, with_residual=False,
             check_y=True, score_rule=0):
    sh = inp["shape"]
    B = inp["x"].shape[0]
    _flush(f"case {sh.name} B={B} budget={budget} flags={flags} "
           f"norm_topk={norm_topk} residual={with_residual} rule={score_rule}")
    residual = None
    if with_residual:
        g = np.random.default_rng(7)
        residual = g.standard_normal((B, sh.d)).astype(np.float32)
        if sh.bf16:
            residual = W.bf16_bits_to_f32(W.f32_to_bf16_bits(residual))
    ref = oracle_layer(inp, budget, flags, norm_topk, residual, check_y, score_rule)
    gl = gu.GpuLayer(inp, norm_topk=norm_topk, score_rule=score_rule)
    x, logits, ids, w, cost, sel, nsel, slot = check_scoring(gl, inp, ref, B,
                                                              budget, score_rule)
    res_d = None if residual is None else gl.x(residual)
    # staged forward
    ws = gl.workspace(B, budget)
    y = gl.y_like(B)
    from paper_2609_36222_amd import binding as bd
    plan = bd.base_moe_forward(gl.desc, x, B, logits, ids, sel, nsel, slot,
                               budget, flags, res_d, y, ws)
    torch.cuda.synchronize()
    got = gu.plan_arrays(plan, ws, B, sh.K, sh.E, budget, full=False, ns=gl.ns)
    check_plan(got, ref)
    y_staged = gu.to_np_f32(y)
    if check_y:
        err = np.max(np.abs(y_staged.astype(np.float64) - ref["y"]))
        _flush(f"y max-abs error {err:.3e} (bar {Y_TOL[sh.bf16]:.0e}, "
               f"max |y| {np.max(np.abs(ref['y'])):.3e})")
        assert err <= Y_TOL[sh.bf16], err
    # fused layer: bit-identical to the staged calls
    ws2 = gl.workspace(B, budget)
    y2 = gl.y_like(B)
    plan2 = bd.base_decode_layer(gl.desc, x, B, budget, flags, res_d, y2, ws2)
    torch.cuda.synchronize()
    got2 = gu.plan_arrays(plan2, ws2, B, sh.K, sh.E, budget, full=True, ns=gl.ns)
    check_plan(got2, ref)
    for f in ("logits", "topk_ids", "topk_w", "cost", "scores", "counts",
              "sel_ids", "slot_of_expert"):
        assert np.array_equal(got2[f], ref[f]), f
    assert got2["n_sel"] == ref["n_sel"]
    assert np.array_equal(gu.to_np_f32(y2), y_staged)
    if sh.bf16:
        # packed expert layout: same values, same arithmetic, same bits
        glp = gu.GpuLayer(inp, norm_topk=norm_topk, packed=True, score_rule=score_rule)
        ws3 = glp.workspace(B, budget)
        y3 = glp.y_like(B)
        bd.base_decode_layer(glp.desc, x, B, budget, flags, res_d, y3, ws3)
        torch.cuda.synchronize()
        assert np.array_equal(gu.to_np_f32(y3), y_staged)
    return ref, y_staged


# ------------------------------------------------------------ named layers --
@pytest.mark.parametrize("name,budget", [
    ("tiny", 6), ("olmoe", 16), ("olmoe", 32), ("qwen3_b64", 16),
    ("qwen3_b64", 32), ("qwen3_b64", 64)])
def test_named_layer(gu, name, budget):
    run_case(gu, named(name), budget)


@pytest.mark.parametrize("seed", [1, 2, 3, 5, 8])
def test_tiny_seeds_with_large_union(gu, seed):
    inp = named("tiny", data_seed=seed)
    run_case(gu, inp, 6)
    run_case(gu, inp, 2, flags=2)


@pytest.fixture(scope="module")
def qwen3_b256():
    return named("qwen3_b256")


@pytest.mark.parametrize("budget", [4, 8, 32, 64, 128])
def test_qwen3_b256_full_size(gu, qwen3_b256, budget):
    """The batch-256 layer in full: 4 and 8 kept experts take the tables cut
    over the dies (gate/up units of four row-pair tiles, down's instance for
    few slots), 32 to 128 the slots dealt whole."""
    ref, _ = run_case(gu, qwen3_b256, budget)
    if budget == 128:   # covers the whole union: dense top-K
        assert np.array_equal(ref["exec_ids"], ref["topk_ids"])


@pytest.mark.parametrize("rule", [1, 2, 3, 4], ids=["top1", "weight", "weight_sq", "static"])
@pytest.mark.parametrize("name,budget", [("tiny", 3), ("olmoe", 16), ("qwen3_b64", 16)])
def test_selection_rules(gu, name, budget, rule):
    """The selection-rule variants (App. selection-rule ablation): per-pair
    scores, ranking, kept set and everything after it bit for bit with the
    oracle, fused == staged, packed == row-major."""
    run_case(gu, named(name), budget, score_rule=rule)


@pytest.mark.parametrize("name,budget", [("deepseek_v2_lite", 8), ("deepseek_v2_lite", 32),
                                         ("qwen15_moe", 8), ("qwen15_moe", 16)])
def test_shared_experts(gu, name, budget):
    """Layers with always-active shared experts (DeepSeek-V2-Lite- and
    Qwen1.5-MoE-shaped, raw-softmax router weights; the latter's wide shared
    expert given as 4 of the routed width behind a sigmoid gate): the
    routed plan and the shared slots bit for bit, y in full."""
    run_case(gu, named(name), budget, norm_topk=0)
    run_case(gu, named(name), budget, norm_topk=0, flags=2, with_residual=True)


@pytest.mark.parametrize("rule", [1, 4], ids=["top1", "static"])
def test_selection_rules_full_size(gu, qwen3_b256, rule):
    run_case(gu, qwen3_b256, 32, score_rule=rule)


def test_qwen3_b256_flags(gu, qwen3_b256):
    run_case(gu, qwen3_b256, 32, flags=1, with_residual=True)
    run_case(gu, qwen3_b256, 32, flags=2)
    run_case(gu, qwen3_b256, 32, flags=3)


# -------------------------------------------------------------- edge cases --
EDGE = [
    # (d, E, K, I, B, bf16, kwargs, budget)
    (256, 8, 2, 128, 1, True, {}, 4),          # one token
    (512, 20, 3, 128, 65, True, {}, 7),        # ragged tiles everywhere
    (256, 16, 4, 64, 130, False, {}, 5),       # fp32, ragged batch
    (256, 8, 2, 192, 33, True, {}, 1),         # budget 1 < K
    (256, 12, 4, 64, 40, True, {}, 50),        # budget above E (clamped)
    (256, 32, 8, 64, 77, True, {"identical_tokens": True}, 3),  # |U| = K
    (768, 64, 6, 128, 100, True, {"zero_token": True}, 12),     # x = 0 row
    (256, 256, 16, 64, 200, True, {}, 40),     # E and K at their maxima
    (1024, 60, 4, 320, 1024, True, {}, 14),    # B at its maximum
    (256, 32, 8, 64, 1000, True, {}, 20),      # 8000 routed pairs: 8 per compaction thread
    (256, 64, 16, 64, 1024, True, {}, 40),     # B and K at their maxima: 16384 pairs
    (16384, 8, 2, 128, 16, True, {}, 4),       # d at its maximum (512 k-steps of gate/up)
    (256, 4, 1, 32768, 8, True, {}, 2),        # I at its maximum (the deep down instance)
]


@pytest.mark.parametrize("case", EDGE, ids=[f"edge{i}" for i in range(len(EDGE))])
def test_edge_shapes(gu, case):
    d, E, K, I, B, bf16, kw, budget = case
    inp = W.custom_layer(d, E, K, I, B, bf16=bf16, seed=len(kw) + d + E, **kw)
    run_case(gu, inp, budget)


def _random_cases(n, seed=2609):
    """Seeded random layer shapes inside the ABI's limits (d a multiple of
    256, I of 64, K <= E <= 256, K <= 16, B <= 1024; most batches small),
    with random budget, gate / fill flags, router normalisation, selection
    rule and (on some bf16 layers) shared experts."""
    g = np.random.default_rng(seed)
    cases = []
    for i in range(n):
        K = int(g.integers(1, 17))
        E = int(g.integers(K, 257))
        d = int(g.choice([256, 512, 768]))
        I = 64 * int(g.integers(1, 6))
        B = int(g.integers(1, 301)) if g.random() < 0.75 else int(g.integers(301, 1025))
        bf16 = bool(g.random() < 0.8)
        budget = int(g.integers(1, E + 4))
        flags = int(g.integers(0, 4))
        norm_topk = int(g.integers(0, 2))
        rule = int(g.integers(0, 5))
        # shared experts (bf16 layers only): 1 .. 8, gated or not
        ns = int(g.integers(1, 9)) if bf16 and g.random() < 0.3 else 0
        sg = bool(ns and g.random() < 0.5)
        cases.append((d, E, K, I, B, bf16, budget, flags, norm_topk, rule, ns, sg, 1000 + i))
    return cases


RANDOM = _random_cases(64)


@pytest.mark.parametrize("case", RANDOM, ids=[f"rand{i}" for i in range(len(RANDOM))])
def test_random_shapes(gu, case):
    """Seeded random shapes, budgets, options and shared experts: every plan
    array bit for bit, y within tolerance, fused == staged, packed ==
    row-major."""
    d, E, K, I, B, bf16, budget, flags, norm_topk, rule, ns, sg, seed = case
    inp = W.custom_layer(d, E, K, I, B, bf16=bf16, seed=seed, n_shared=ns, shared_gate=sg)
    run_case(gu, inp, budget, flags=flags, norm_topk=norm_topk, score_rule=rule)


def test_raw_softmax_weights(gu):
    inp = W.custom_layer(512, 40, 4, 128, 50, seed=3)
    run_case(gu, inp, 9, norm_topk=0)
    run_case(gu, inp, 9, flags=1, norm_topk=0)


def test_no_router_bias(gu):
    inp = W.custom_layer(256, 16, 2, 64, 20, seed=4)
    inp["b_router"] = None
    run_case(gu, inp, 5)


@pytest.mark.parametrize("flags", [0, 2], ids=["backfill", "drop"])
def test_repeated_route_ids(gu, flags):
    """Routes given to base_select / base_moe_forward in which some tokens
    name one expert twice (not what base_route produces, but allowed by the
    ABI): the aggregation keeps the last cost and counts both, the drop
    rule executes both copies, and the compaction gives each copy its own
    pair in (slot, token, rank) order -- all bit for bit with the oracle."""
    from paper_2609_36222_amd import binding as bd
    inp = W.custom_layer(512, 24, 4, 128, 70, seed=11)
    sh = inp["shape"]
    B, K, E, budget = inp["x"].shape[0], sh.K, sh.E, 9
    logits, ids, w = carith.route(inp["x"], inp["w_router"], inp["b_router"], K, 1)
    ids = ids.copy()
    g = np.random.default_rng(5)
    dup = g.choice(B, size=B // 3, replace=False)
    ids[dup, K - 1] = ids[dup, 0]                 # rank K-1 repeats rank 0
    ids[dup[: B // 6], 2] = ids[dup[: B // 6], 1]  # and some repeat rank 1 too
    cost = method.pair_scores_c(0, inp["x"], inp["pred_a"], inp["pred_b"], ids, w)
    scores, counts = carith.aggregate(ids, cost, E)
    sel, n_sel, slot = method.select(scores, counts, budget)
    ex, n_ex = method.backfill(logits, ids, slot, n_sel, K, flags)
    gates = method.gates_c(logits, ids, ex, n_ex, 1, flags)
    offsets, pair_tok, pair_gate, pair_of = method.compact(ex, n_ex, slot, gates, budget)
    y_ref = method.moe_restricted64(inp["x"], ex, n_ex, gates,
                                    method.Experts(inp["w13"], inp["w2"], sh.bf16))
    _flush(f"case repeated ids flags={flags} B={B} dup={len(dup)}")
    gl = gu.GpuLayer(inp)
    x = gl.x(inp["x"])
    ids_d = torch.from_numpy(ids.astype(np.int32)).cuda()
    cost_d = gu.dev_f32(cost)
    s_d, c_d, sel_d, nsel_d, slot_d = gl.select(B, ids_d, cost_d, budget)
    assert np.array_equal(s_d.cpu().numpy(), scores)
    assert np.array_equal(c_d.cpu().numpy(), counts)
    assert int(nsel_d.item()) == n_sel
    assert np.array_equal(sel_d.cpu().numpy(), sel)
    assert np.array_equal(slot_d.cpu().numpy(), slot)
    ws = gl.workspace(B, budget)
    y = gl.y_like(B)
    plan = bd.base_moe_forward(gl.desc, x, B, gu.dev_f32(logits), ids_d, sel_d, nsel_d,
                               slot_d, budget, flags, None, y, ws)
    torch.cuda.synchronize()
    got = gu.plan_arrays(plan, ws, B, K, E, budget, full=False)
    check_plan(got, dict(exec_ids=ex, exec_gates=gates, offsets=offsets, pair_tok=pair_tok,
                         pair_gate=pair_gate, pair_of=pair_of))
    if flags & 2:   # the drop rule executes both copies of a repeated route
        assert int((np.sum(got["pair_of"] >= 0, axis=1) > np.array(
            [len(set(r.tolist())) for r in ids])).sum()) > 0
    err = np.max(np.abs(gu.to_np_f32(y).astype(np.float64) - y_ref))
    assert err <= Y_TOL[sh.bf16], err


def test_repeat_runs_are_bit_identical(gu, qwen3_b256):
    from paper_2609_36222_amd import binding as bd
    gl = gu.GpuLayer(qwen3_b256)
    x = gl.x(qwen3_b256["x"])
    B = x.shape[0]
    ws = gl.workspace(B, 32)
    outs = []
    for _ in range(5):
        y = gl.y_like(B)
        bd.base_decode_layer(gl.desc, x, B, 32, 0, None, y, ws)
        outs.append(y.view(torch.int16).cpu().numpy())
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])


def test_packed_layout_matches_its_definition(gu):
    """base_pack_experts against the layout stated in base.h, rebuilt here
    with numpy from the row-major arrays."""
    from paper_2609_36222_amd import binding as bd
    inp = W.custom_layer(512, 6, 2, 192, 4, seed=21)
    gl = gu.GpuLayer(inp, packed=True)
    E, d, I = 6, 512, 192
    got13 = gl.layer.tensors[4].view(torch.int16).cpu().numpy().view(np.uint16)
    got2 = gl.layer.tensors[5].view(torch.int16).cpu().numpy().view(np.uint16)

    def pack(w, rows_of_tile, groups, kdim):
        E_ = w.shape[0]
        out = np.empty((E_, groups, kdim // 32, 4, 64, 8), np.uint16)
        lanes = np.arange(64)
        for g in range(groups):
            for t in range(4):
                rows = rows_of_tile(g, t) + (lanes % 16)
                for ks in range(kdim // 32):
                    cols = 32 * ks + 8 * (lanes // 16)
                    idx = cols[:, None] + np.arange(8)[None, :]
                    out[:, g, ks, t] = w[:, rows[:, None], idx]
        return out.reshape(-1)
    exp13 = pack(inp["w13"], lambda g, t: (0 if t < 2 else I) + 32 * g + 16 * (t % 2),
                 I // 32, d)
    exp2 = pack(inp["w2"], lambda g, t: 64 * g + 16 * t, d // 64, I)
    assert np.array_equal(got13.reshape(-1), exp13)
    assert np.array_equal(got2.reshape(-1), exp2)


def test_graph_replay_matches_eager(gu):
    """base_decode_layer captured once in a HIP graph (through torch's stream
    capture) and replayed with new tokens and a new residual copied in
    between replays, the workspace and output overwritten with junk by
    eager kernels before each replay: every replay equals an eager call on
    the same inputs bit for bit (all plan arrays and y), and the plan equals
    the oracle's."""
    from paper_2609_36222_amd import binding as bd
    inp = named("qwen3_b64")
    sh = inp["shape"]
    B, budget, flags = sh.B, 32, 1
    gl = gu.GpuLayer(inp, packed=True)
    g = np.random.default_rng(11)
    xs, rs = [], []
    for s in range(3):
        xs.append(W.decode_tokens(sh, data_seed=s + 1))
        rs.append(W.bf16_bits_to_f32(W.f32_to_bf16_bits(
            g.standard_normal((B, sh.d)).astype(np.float32))))
    x = gl.x(xs[0])
    res = gl.x(rs[0])
    ws = gl.workspace(B, budget)
    y = gl.y_like(B)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        bd.base_decode_layer(gl.desc, x, B, budget, flags, res, y, ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        plan = bd.base_decode_layer(gl.desc, x, B, budget, flags, res, y, ws)
    torch.cuda.synchronize()
    for rep in range(5):
        k = rep % 3
        _flush(f"graph replay {rep} tokens seed {k + 1}")
        xk, rk = gl.x(xs[k]), gl.x(rs[k])
        ws_e, y_e = gl.workspace(B, budget), gl.y_like(B)
        plan_e = bd.base_decode_layer(gl.desc, xk, B, budget, flags, rk, y_e, ws_e)
        torch.cuda.synchronize()
        want = gu.plan_arrays(plan_e, ws_e, B, sh.K, sh.E, budget, full=True)
        x.copy_(xk)
        res.copy_(rk)
        ws.fill_(0xA5)
        y.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = gu.plan_arrays(plan, ws, B, sh.K, sh.E, budget, full=True)
        for f, v in want.items():
            if isinstance(v, np.ndarray):
                assert np.array_equal(got[f], v), (rep, f)
            else:
                assert got[f] == v, (rep, f)
        assert np.array_equal(y.view(torch.int16).cpu().numpy(),
                              y_e.view(torch.int16).cpu().numpy()), rep
        if rep < 3:
            ref = method.decode_layer_c(xs[k], inp["w_router"], inp["b_router"],
                                        inp["pred_a"], inp["pred_b"], sh.K, budget,
                                        None, 1, flags, rs[k])
            check_plan(got, ref)
            assert got["n_sel"] == ref["n_sel"]


def test_stage_events_ignored_under_capture(gu):
    """Stage events set while base_decode_layer is captured: the captured
    call records none of them (the capture succeeds and its replay equals an
    eager call bit for bit), and an eager call made afterwards with the same
    setting still times every kernel stage."""
    import ctypes
    import re
    from paper_2609_36222_amd import binding as bd
    maps = open("/proc/self/maps").read()
    hip = ctypes.CDLL(sorted(set(re.findall(r"(/\S*libamdhip64\.so[.\d]*)", maps)))[0])
    hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float),
                                        ctypes.c_void_p, ctypes.c_void_p]
    hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
    evs = []
    for _ in range(2 * bd.N_STAGES):
        e = ctypes.c_void_p()
        assert hip.hipEventCreate(ctypes.byref(e)) == 0
        evs.append(e.value)
    inp = named("qwen3_b64")
    sh = inp["shape"]
    B, budget, flags = sh.B, 32, 0
    gl = gu.GpuLayer(inp, packed=True)
    x = gl.x(W.decode_tokens(sh, data_seed=5))
    ws, y = gl.workspace(B, budget), gl.y_like(B)
    ws_e, y_e = gl.workspace(B, budget), gl.y_like(B)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        bd.base_decode_layer(gl.desc, x, B, budget, flags, None, y, ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    keep = bd.base_set_stage_events(evs)
    try:
        _flush("capture with stage events set")
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            bd.base_decode_layer(gl.desc, x, B, budget, flags, None, y, ws)
        torch.cuda.synchronize()
        _flush("eager call with stage events set")
        bd.base_decode_layer(gl.desc, x, B, budget, flags, None, y_e, ws_e)
        torch.cuda.synchronize()
    finally:
        bd.base_set_stage_events(None)
    del keep
    ms = ctypes.c_float()
    # every stage with a kernel of its own in base_decode_layer (3 and 5
    # record their pairs back to back)
    for s in (0, 1, 2, 4, 6, 7, 8):
        assert hip.hipEventElapsedTime(ctypes.byref(ms), evs[2 * s], evs[2 * s + 1]) == 0, s
        assert ms.value > 0.0, s
    y.fill_(float("nan"))
    torch.cuda.synchronize()
    _flush("replay of the graph captured with stage events set")
    graph.replay()
    torch.cuda.synchronize()
    assert np.array_equal(y.view(torch.int16).cpu().numpy(),
                          y_e.view(torch.int16).cpu().numpy())
    for e in evs:
        hip.hipEventDestroy(e)


# ------------------------------------------------- few large experts, stack --
@pytest.mark.timeout(600)
def test_mixtral_full_size(gu):
    """Mixtral-shaped layer (d=4096, E=8, top-2, I=14336) at batch 128 with
    B_e=4: the whole batch, every plan array bit for bit, y in full."""
    run_case(gu, named("mixtral"), 4)


def _y_tol_bf16(y_ref):
    """The bf16 bar plus the output format's own rounding: y carries the
    residual stream, whose magnitude grows with depth, and rounding it to
    bf16 moves it by up to 2^-8 of its size."""
    return Y_TOL[True] + np.abs(y_ref) * 2.0 ** -8


@pytest.mark.timeout(1200)
def test_qwen3_stack48_residual_carried(gu):
    """48 Qwen3-shaped layers at batch 128, B_e=24, pre-norm with the
    residual carried: layer l takes x_l = RMSNorm(h_l) (bf16) and outputs
    h_{l+1} = h_l + MoE_l(x_l), all on the GPU.  At every layer the oracle
    takes the GPU's own x_l and h_l (teacher forcing, so no error
    accumulates between the two sides) and every plan array must match bit
    for bit; y is checked on 8 sampled tokens per layer against the fp64
    restricted MoE plus residual, and the same layer's MoE output alone (a
    second call without the residual) against the plain 2e-2 bar."""
    from paper_2609_36222_amd import binding as bd
    name = "qwen3_stack48"
    sh = W.WORKLOADS[name]
    B, budget = sh.B, sh.budgets[0]
    h_np = W.layer_inputs(name, layer=0, with_experts=False)["x"]
    h = gu.act_to_dev(h_np, True)
    sample = np.sort(np.random.default_rng(48).choice(B, 8, replace=False))
    for layer in range(sh.layers):
        inp = W.layer_inputs(name, layer=layer)
        x_np = h_np if layer == 0 else W.stack_layer_input(h_np)
        x = gu.act_to_dev(x_np, True)
        gl = gu.GpuLayer(inp, packed=True)
        ws, y = gl.workspace(B, budget), gl.y_like(B)
        plan = bd.base_decode_layer(gl.desc, x, B, budget, 0, h, y, ws)
        torch.cuda.synchronize()
        got = gu.plan_arrays(plan, ws, B, sh.K, sh.E, budget, full=True)
        ref = method.decode_layer_c(x_np, inp["w_router"], inp["b_router"],
                                    inp["pred_a"], inp["pred_b"], sh.K, budget)
        for f in ("logits", "topk_ids", "topk_w", "cost", "scores", "counts",
                  "sel_ids", "slot_of_expert"):
            assert np.array_equal(got[f], ref[f]), (layer, f)
        assert got["n_sel"] == ref["n_sel"], layer
        check_plan(got, ref)
        ex = method.Experts(inp["w13"], inp["w2"], True)
        y_ref = method.moe_restricted64(
            x_np[sample], ref["exec_ids"][sample], ref["n_exec"][sample],
            ref["exec_gates"][sample], ex, residual=h_np[sample])
        y_np = gu.to_np_f32(y)
        err = np.abs(y_np[sample].astype(np.float64) - y_ref)
        union = int((ref["counts"] > 0).sum())
        # the MoE output alone (no residual: |y| small) at the plain bar
        y_moe = gl.y_like(B)
        bd.base_decode_layer(gl.desc, x, B, budget, 0, None, y_moe, ws)
        torch.cuda.synchronize()
        m_ref = method.moe_restricted64(
            x_np[sample], ref["exec_ids"][sample], ref["n_exec"][sample],
            ref["exec_gates"][sample], ex)
        m_err = np.abs(gu.to_np_f32(y_moe)[sample].astype(np.float64) - m_ref)
        _flush(f"stack layer {layer}: |U|={union} n_sel={ref['n_sel']} "
               f"rms(h)={float(np.sqrt(np.mean(y_np.astype(np.float64) ** 2))):.3f} "
               f"max|h|={np.abs(y_np).max():.3f} max err={err.max():.4f} "
               f"MoE alone max err={m_err.max():.4f}")
        assert np.all(err <= _y_tol_bf16(y_ref)), (layer, float(err.max()))
        assert np.all(m_err <= Y_TOL[True]), (layer, float(m_err.max()))
        h_np, h = y_np, y
        del y_moe
        del gl, ws, inp, ex, x
