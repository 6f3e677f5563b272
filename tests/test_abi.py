"""The C-ABI library loads and exports every symbol include/base.h declares;
host-side validation returns its status codes before anything is enqueued
(so these run without a GPU: no call here reaches a launch)."""
import ctypes
import os
import re

import pytest

from paper_2609_36222_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

OK, NULL, SHAPE, BUDGET, DTYPE, ALIGN, WS, HIP, FLAGS = 0, -1, -2, -3, -4, -5, -6, -7, -8
FAKE = 1 << 32          # a 256-byte aligned stand-in address, never touched


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(bd.LIB_PATH):
        from paper_2609_36222_amd import build
        build.build()
    return bd.load()


def header_functions():
    with open(os.path.join(ROOT, "include", "base.h")) as f:
        src = f.read()
    return sorted(set(re.findall(r"^\s*(?:size_t|base_status|const char)\s*\*?\s*(base_\w+)\(",
                                 src, re.M)))


def test_header_and_binding_agree(lib):
    fns = header_functions()
    assert fns == sorted(bd.EXPORTS)
    for f in fns:
        assert hasattr(lib, f), f


def test_exported_symbols_in_dynamic_table(lib):
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", bd.LIB_PATH],
                         capture_output=True, text=True).stdout
    syms = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for f in header_functions():
        assert f in syms, f


def layer(**kw):
    v = dict(d=2048, E=128, K=8, I=768, dtype=1, norm_topk=1, w_layout=0,
             score_rule=0, w_router=FAKE, b_router=FAKE, pred_a=FAKE, pred_b=FAKE,
             w13=FAKE, w2=FAKE, n_shared=0, w13_shared=None, w2_shared=None,
             shared_gate=None)
    v.update(kw)
    return bd.base_layer(v["d"], v["E"], v["K"], v["I"], v["dtype"],
                         v["norm_topk"], v["w_layout"], v["score_rule"], v["w_router"],
                         v["b_router"], v["pred_a"], v["pred_b"], v["w13"],
                         v["w2"], v["n_shared"], v["w13_shared"], v["w2_shared"],
                         v["shared_gate"])


def route(lib, L, x=FAKE, B=16, lg=FAKE, ids=FAKE, w=FAKE):
    return lib.base_route(ctypes.byref(L), x, B, lg, ids, w, None)


def decode(lib, L, B=16, budget=4, flags=0, x=FAKE, y=FAKE, ws=FAKE,
           nbytes=None, residual=None):
    if nbytes is None:
        nbytes = lib.base_workspace_bytes(ctypes.byref(L), B, budget)
    return lib.base_decode_layer(ctypes.byref(L), x, B, budget, flags,
                                 residual, y, None, ws, nbytes, None)


def test_status_strings(lib):
    for s in (OK, NULL, SHAPE, BUDGET, DTYPE, ALIGN, WS, HIP, FLAGS):
        assert bd.status_string(s)
    assert bd.status_string(-99) == "unknown status"


@pytest.mark.parametrize("kw,expect", [
    (dict(d=2000), SHAPE), (dict(d=0), SHAPE), (dict(d=16640), SHAPE),
    (dict(K=0), SHAPE), (dict(K=17, E=32), SHAPE), (dict(E=4, K=8), SHAPE),
    (dict(E=257), SHAPE), (dict(I=100), SHAPE), (dict(I=0), SHAPE),
    (dict(dtype=7), DTYPE), (dict(norm_topk=2), SHAPE),
    (dict(w_layout=2), SHAPE), (dict(w_layout=1, dtype=0), DTYPE),
    (dict(w_router=0), NULL), (dict(w_router=FAKE + 4), ALIGN),
    (dict(b_router=FAKE + 2), ALIGN), (dict(score_rule=5), FLAGS),
    (dict(score_rule=-1), FLAGS)])
def test_route_layer_validation(lib, kw, expect):
    assert route(lib, layer(**kw)) == expect


@pytest.mark.parametrize("B", [0, -1, 1025])
def test_batch_limits(lib, B):
    assert route(lib, layer(), B=B) == SHAPE
    assert lib.base_workspace_bytes(ctypes.byref(layer()), B, 4) == 0


def test_route_pointer_validation(lib):
    L = layer()
    assert route(lib, L, x=0) == NULL
    assert route(lib, L, x=FAKE + 8) == ALIGN
    assert route(lib, L, lg=0) == NULL
    assert route(lib, L, ids=FAKE + 2) == ALIGN
    assert route(lib, L, w=0) == NULL


def test_predict_validation(lib):
    L = layer(pred_a=0)
    assert lib.base_predict_cost(ctypes.byref(L), FAKE, 4, FAKE, FAKE, FAKE, None) == NULL
    L = layer(pred_a=FAKE + 4)
    assert lib.base_predict_cost(ctypes.byref(L), FAKE, 4, FAKE, FAKE, FAKE, None) == ALIGN
    L = layer()
    assert lib.base_predict_cost(ctypes.byref(L), FAKE, 4, FAKE, FAKE, 0, None) == NULL


def test_select_validation(lib):
    L = layer()
    f = lambda budget, **p: lib.base_select(
        ctypes.byref(L), 16, p.get("ids", FAKE), FAKE, budget, FAKE, FAKE,
        p.get("sel", FAKE), FAKE, FAKE, None)
    assert f(0) == BUDGET
    assert f(-5) == BUDGET
    assert f(4, ids=0) == NULL
    assert f(4, sel=FAKE + 1) == ALIGN


def test_moe_forward_validation(lib):
    L = layer()
    nb = lib.base_workspace_bytes(ctypes.byref(L), 16, 4)

    def f(budget=4, flags=0, ws=FAKE, n=nb, w13=FAKE, residual=None):
        LL = layer(w13=w13)
        return lib.base_moe_forward(ctypes.byref(LL), FAKE, 16, FAKE, FAKE,
                                    FAKE, FAKE, FAKE, budget, flags, residual,
                                    FAKE, None, ws, n, None)
    assert f(budget=0) == BUDGET
    assert f(flags=4) == FLAGS
    assert f(w13=0) == NULL
    assert f(w13=FAKE + 8) == ALIGN
    assert f(ws=0) == NULL
    assert f(ws=FAKE + 128) == ALIGN
    assert f(n=nb - 1) == WS
    assert f(residual=FAKE + 4) == ALIGN


def test_decode_layer_validation(lib):
    L = layer()
    assert decode(lib, L, budget=0) == BUDGET
    assert decode(lib, L, flags=8) == FLAGS
    assert decode(lib, L, x=0) == NULL
    assert decode(lib, L, y=FAKE + 4) == ALIGN
    assert decode(lib, L, nbytes=100) == WS
    assert decode(lib, layer(pred_b=0)) == NULL
    assert decode(lib, layer(w2=0)) == NULL


def test_score_rules_read_only_their_parameters(lib):
    """BASE needs pred_a and pred_b, STATIC pred_b only, the router-only
    rules neither (their calls pass validation up to the workspace check)."""
    for rule in (bd.SCORE_TOP1, bd.SCORE_WEIGHT, bd.SCORE_WEIGHT_SQ):
        assert decode(lib, layer(score_rule=rule, pred_a=0, pred_b=0), nbytes=100) == WS
    assert decode(lib, layer(score_rule=bd.SCORE_STATIC, pred_a=0), nbytes=100) == WS
    assert decode(lib, layer(score_rule=bd.SCORE_STATIC, pred_b=0)) == NULL
    assert decode(lib, layer(score_rule=bd.SCORE_BASE, pred_a=0)) == NULL
    L = layer(score_rule=bd.SCORE_STATIC, pred_a=0)
    assert lib.base_predict_cost(ctypes.byref(L), FAKE, 4, FAKE, FAKE, 0, None) == NULL
    assert lib.base_predict_cost(ctypes.byref(layer(score_rule=9)), FAKE, 4, FAKE, FAKE,
                                 FAKE, None) == FLAGS


def test_shared_expert_validation(lib):
    """Shared experts: at most 8, bf16 layers only, their weights required
    (and 16-B aligned) where the experts are read, the gate 16-B aligned;
    they enlarge the workspace."""
    sh = dict(w13_shared=FAKE, w2_shared=FAKE)
    assert route(lib, layer(n_shared=9, **sh)) == SHAPE
    assert route(lib, layer(n_shared=-1, **sh)) == SHAPE
    assert route(lib, layer(n_shared=1, dtype=0, **sh)) == DTYPE
    assert route(lib, layer(n_shared=1, shared_gate=FAKE + 4, **sh)) == ALIGN
    assert decode(lib, layer(n_shared=2, w13_shared=None, w2_shared=FAKE)) == NULL
    assert decode(lib, layer(n_shared=2, w13_shared=FAKE + 8, w2_shared=FAKE)) == ALIGN
    a = lib.base_workspace_bytes(ctypes.byref(layer()), 64, 16)
    b = lib.base_workspace_bytes(ctypes.byref(layer(n_shared=2, **sh)), 64, 16)
    assert b > a
    # packing shared experts: a descriptor with E = n_shared (K not read)
    P = layer(E=2, K=8, n_shared=0)
    assert lib.base_pack_experts(ctypes.byref(P), 0, FAKE, None) == NULL


def test_workspace_grows_with_shape_and_clamps_budget(lib):
    L = layer()
    a = lib.base_workspace_bytes(ctypes.byref(L), 64, 16)
    b = lib.base_workspace_bytes(ctypes.byref(L), 256, 16)
    assert 0 < a < b
    assert lib.base_workspace_bytes(ctypes.byref(L), 64, 128) == \
        lib.base_workspace_bytes(ctypes.byref(L), 64, 1000)
    assert lib.base_workspace_bytes(ctypes.byref(L), 64, 0) == 0
    assert lib.base_workspace_bytes(None, 64, 4) == 0


def test_pack_validation(lib):
    f = lambda L, a=FAKE, b=FAKE: lib.base_pack_experts(ctypes.byref(L), a, b, None)
    assert lib.base_pack_experts(None, FAKE, FAKE, None) == NULL
    assert f(layer(dtype=0)) == DTYPE
    assert f(layer(w_layout=1)) == SHAPE
    assert f(layer(), a=0) == NULL
    assert f(layer(), b=FAKE + 8) == ALIGN
    assert f(layer(w13=0)) == NULL
    assert f(layer(I=100)) == SHAPE


def test_stage_events_validation(lib):
    arr = (ctypes.c_void_p * (2 * bd.N_STAGES))(*([FAKE] * (2 * bd.N_STAGES)))
    assert lib.base_set_stage_events(arr, 2 * bd.N_STAGES - 1) == SHAPE
    assert lib.base_set_stage_events(arr, bd.N_STAGES + 1) == SHAPE
    arr[3] = None
    assert lib.base_set_stage_events(arr, 2 * bd.N_STAGES) == NULL
    assert lib.base_set_stage_events(None, 0) == OK
    assert len(bd.STAGES) == bd.N_STAGES
    with open(os.path.join(ROOT, "include", "base.h")) as f:
        assert re.search(r"#define BASE_N_STAGES %d\b" % bd.N_STAGES, f.read())


def test_stream_read_probe_library():
    """The benchmark's streaming-read probe sits in a library of its own
    (not part of the method's ABI); bad arguments are refused before any
    launch with hipErrorInvalidValue (1)."""
    import subprocess
    from paper_2609_36222_amd import build
    if not os.path.exists(build.PROBE_LIB):
        build.build()
    out = subprocess.run(["nm", "-D", "--defined-only", build.PROBE_LIB],
                         capture_output=True, text=True).stdout
    syms = {line.split()[-1] for line in out.splitlines() if line.strip()}
    assert "base_probe_stream_read" in syms
    assert not any(s.startswith("base_") and s != "base_probe_stream_read" for s in syms)
    f = ctypes.CDLL(build.PROBE_LIB).base_probe_stream_read
    f.argtypes = [ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    f.restype = ctypes.c_int
    assert f(FAKE, 8, 6, 0, FAKE, None, None, None) == 1       # steps not a multiple of 4
    assert f(FAKE, 0, 16, 0, FAKE, None, None, None) == 1      # no waves
    assert f(None, 8, 16, 0, FAKE, None, None, None) == 1      # no buffer
    assert f(FAKE, 8, 16, 0, None, None, None, None) == 1      # no sink
    assert f(FAKE, 8, 1 << 19, 0, FAKE, None, None, None) == 1  # share of 2 GiB


def test_calibration_validation(lib):
    """Calibration statistics: size of the documented layout, and host-side
    refusals before anything is enqueued (the fit library's too)."""
    L = layer(d=256, E=16, K=2, I=512, dtype=0)
    up = lambda v: (v + 255) // 256 * 256
    assert lib.base_calib_stats_bytes(ctypes.byref(L)) == \
        up(16 * 4 * 8) + 2 * up(16 * 256 * 8) + up(16 * 256 * 256 * 4)
    assert lib.base_calib_stats_bytes(ctypes.byref(layer(d=300))) == 0
    assert lib.base_calib_ws_bytes(ctypes.byref(L), 64) > lib.base_workspace_bytes(ctypes.byref(L), 64, 16)
    assert lib.base_calib_reset(ctypes.byref(L), None, None) == NULL
    assert lib.base_calib_reset(ctypes.byref(L), FAKE + 64, None) == ALIGN
    nb = lib.base_calib_ws_bytes(ctypes.byref(L), 64)
    acc = lambda **k: lib.base_calib_accumulate(
        ctypes.byref(k.get("L", L)), k.get("z", FAKE), 64, k.get("st", FAKE), k.get("ws", FAKE),
        k.get("n", nb), None)
    assert acc(z=0) == NULL
    assert acc(st=FAKE + 8) == ALIGN
    assert acc(n=nb - 1) == WS
    assert acc(L=layer(d=256, E=16, K=2, I=512, dtype=0, w_router=0)) == NULL
    cal = bd.load_calib()
    lam = (ctypes.c_double * 3)(1e-3, 1e-1, 1.0)
    fit = lambda **k: cal.base_calib_fit(ctypes.byref(L), k.get("st", FAKE), k.get("n", 3),
                                         k.get("lam", lam), k.get("a", FAKE), FAKE, None, None)
    assert fit(st=None) == NULL
    assert fit(n=0) == SHAPE
    assert fit(n=65) == SHAPE
    assert fit(lam=(ctypes.c_double * 3)(1e-3, 0.0, 1.0)) == SHAPE
    assert fit(st=FAKE + 8) == ALIGN
    assert fit(a=FAKE + 2) == ALIGN


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    """Without the built library the binding raises: there is no CPU
    fallback for any entry point."""
    from paper_2609_36222_amd import binding as bd
    monkeypatch.setattr(bd, "_lib", None)
    with pytest.raises(ImportError, match="no CPU fallback"):
        bd.load(str(tmp_path / "libbase.so"))


def test_noalloc_validation(lib):
    """base_decode_layer_noalloc checks like base_decode_layer, and rejects
    a layer whose workspace exceeds its scratch array, before it touches the
    device (these calls return without a GPU)."""
    def na(L, B=16, budget=4, flags=0, x=FAKE, y=FAKE, residual=None):
        return lib.base_decode_layer_noalloc(ctypes.byref(L), x, B, budget, flags,
                                             residual, y, None, None)
    L = layer()
    assert na(L, budget=0) == BUDGET
    assert na(L, flags=8) == FLAGS
    assert na(L, x=0) == NULL
    assert na(L, y=FAKE + 4) == ALIGN
    assert na(L, residual=FAKE + 8) == ALIGN
    assert na(layer(pred_b=0)) == NULL
    assert na(L, B=2048) == SHAPE
    big = layer(E=256, K=16)
    assert lib.base_workspace_bytes(ctypes.byref(big), 1024, 256) > bd.NOALLOC_SCRATCH_BYTES
    assert na(big, B=1024, budget=256) == WS
