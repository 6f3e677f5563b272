"""Exact ties on the GPU (Sec. 3.5 ranks a token's experts and the batch's
experts; ties go to the lower expert index, keys compared as fp32 so that
-0 equals +0): equal router logits, equal batch scores and a -0 / +0 pair,
bit for bit with the oracle through the staged calls, the fused layer and
the packed weight layout."""
import numpy as np
import pytest

import workloads as W
from oracle import carith

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def gu(gpu):
    import gpu_util
    return gpu_util


def _run(gu, inp, budget, **kw):
    import test_gpu_parity as P
    return P.run_case(gu, inp, budget, **kw)


def _tie_router(inp, groups, rest_bias=None, rest_scale=1.0):
    """Router rows set to zero (logit = bias exactly) for the experts of
    each group, all given the group's bias; the other rows scaled."""
    wr = inp["w_router"].copy() * np.float32(rest_scale)
    br = inp["b_router"].copy()
    if rest_bias is not None:
        br[:] = np.float32(rest_bias)
    for experts, bias in groups:
        for e in experts:
            wr[e] = 0.0
            br[e] = np.float32(bias)
    inp["w_router"], inp["b_router"] = wr, br
    return inp


def test_equal_logits_at_the_top_k_boundary(gu):
    """Eight experts with identical logits (zero rows, equal bias) whose
    value falls at most tokens' top-K boundary: the routed set, weights,
    costs, selection and backfill order all follow the lower index."""
    inp = _tie_router(W.custom_layer(512, 32, 4, 128, 96, seed=31), [(range(5, 13), -1.0)])
    logits, ids, _ = carith.route(inp["x"], inp["w_router"], inp["b_router"], 4, 1)
    tied = (ids >= 5) & (ids < 13)
    # ties really decide: tokens keep 1 to 3 of the tied group, lowest first
    n_tied = tied.sum(axis=1)
    assert np.sum((n_tied > 0) & (n_tied < 4)) > 40
    for t in range(ids.shape[0]):
        got = [e for e in ids[t] if 5 <= e < 13]
        assert got == list(range(5, 5 + len(got)))
    _run(gu, inp, 7)
    _run(gu, inp, 7, flags=2)


def test_negative_and_positive_zero_logits_tie(gu):
    """Router logits of exactly +0 (zero rows with bias +0 and -0: x . 0 is
    +0, and +0 + -0 = +0) tie with one another and rank by index; four
    experts rank above them with one shared logit, the rest far below."""
    inp = W.custom_layer(256, 16, 6, 64, 40, seed=32)
    br_signs = [(range(0, 4), 1.0), ([4], -0.0), ([5], 0.0), ([6], -0.0), ([7], 0.0)]
    inp = _tie_router(inp, br_signs, rest_bias=-6.0, rest_scale=0.01)
    assert np.signbit(inp["b_router"][4]) and not np.signbit(inp["b_router"][5])
    logits, ids, _ = carith.route(inp["x"], inp["w_router"], inp["b_router"], 6, 1)
    assert np.all(ids == np.array([0, 1, 2, 3, 4, 5], np.int32))
    assert np.all(logits[:, 4:8] == 0.0)
    _run(gu, inp, 5)
    _run(gu, inp, 5, flags=3)


def test_equal_batch_scores_under_the_weight_rule(gu):
    """Identical tokens with pairwise-equal logits (two tied groups): under
    the router-weight-sum rule the batch scores D_u tie exactly, so the kept
    set is decided by index alone."""
    inp = W.custom_layer(256, 24, 6, 64, 50, seed=33, identical_tokens=True)
    inp = _tie_router(inp, [(range(2, 6), 1.5), (range(10, 14), 1.0)])
    ref, _ = _run(gu, inp, 5, score_rule=2)
    s = ref["scores"]
    # every token routes 2, 3, 4, 5 (tied at the top) and 10, 11 (of the
    # second tied group, cut at the top-K boundary)
    assert s[2] == s[3] == s[4] == s[5] and s[10] == s[11] > 0 and s[12] == s[13] == 0
    assert list(ref["sel_ids"][:ref["n_sel"]]) == sorted(ref["sel_ids"][:ref["n_sel"]],
                                                         key=lambda u: (-s[u], u))
    # a budget that cuts the first tied group keeps its lowest indices
    ref2, _ = _run(gu, inp, 2, score_rule=2)
    assert list(ref2["sel_ids"][:2]) == [2, 3]
