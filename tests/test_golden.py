"""The hand-built five-token example of the paper's Figure teaser (Sec. 3.2),
with expected values derived by hand in the fixture."""
import json
import os

import numpy as np

from oracle import carith, method

HERE = os.path.dirname(os.path.abspath(__file__))


def load():
    with open(os.path.join(HERE, "golden", "teaser_example.json")) as f:
        return json.load(f)


def test_teaser_example_selection_backfill_compaction():
    g = load()
    ids = np.array(g["topk_ids"], np.int32)
    cost = np.array(g["cost"], np.float32)
    logits = np.array(g["logits"], np.float32)
    K, E, M = g["K"], g["E"], g["budget"]
    exp = g["expected"]
    scores, counts = carith.aggregate(ids, cost, E)
    assert list(scores) == exp["scores"]
    assert list(counts) == exp["counts"]
    assert sorted(set(ids[:, 0].tolist())) == exp["top1_union"]
    sel, n_sel, slot = method.select(scores, counts, M)
    assert list(sel) == exp["sel_ids"] and n_sel == exp["n_sel"]
    # an expert nobody ranks first is kept; two top-1 experts are not
    assert 2 in sel and 2 not in ids[:, 0]
    assert 4 not in sel and 7 not in sel
    ex, n_ex = method.backfill(logits, ids, slot, n_sel, K)
    exd = np.where(np.arange(K)[None, :] < n_ex[:, None], ex, -1)
    assert exd.tolist() == exp["exec_ids_backfill"]
    ex_d, n_d = method.backfill(logits, ids, slot, n_sel, K, method.FILL_DROP)
    assert ex_d.tolist() == exp["exec_ids_drop"]
    gt = method.gates_c(logits, ids, ex, n_ex)
    np.testing.assert_allclose(gt[3], exp["gates_backfill_t4"], rtol=2e-7)
    np.testing.assert_allclose(gt[4], exp["gates_backfill_t5"], rtol=2e-7)
    off, ptok, _, _ = method.compact(ex, n_ex, slot, gt, M)
    assert off.tolist() == exp["offsets"]
    assert ptok.tolist() == exp["pair_tok"]
