"""base_decode_layer_noalloc (the whole layer on the library's own scratch
array, no workspace argument) against base_decode_layer with a caller
workspace: two calls in a row on the same GPU, the second with a smaller
batch and budget, every plan array and y bit for bit."""
import ctypes

import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def gu(gpu):
    import gpu_util
    return gpu_util


def _hip():
    lib = ctypes.CDLL("libamdhip64.so")
    lib.hipMemcpy.restype = ctypes.c_int
    lib.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    return lib


def read_device(hip, ptr, count, dtype):
    """count elements of a device array the library owns (device to host)."""
    out = np.empty(count, dtype)
    torch.cuda.synchronize()
    assert hip.hipMemcpy(out.ctypes.data, ptr, out.nbytes, 2) == 0   # device to host
    return out


PLAN_FIELDS = (("logits", "E", np.float32), ("topk_ids", "K", np.int32),
               ("topk_w", "K", np.float32), ("cost", "K", np.float32),
               ("exec_ids", "K", np.int32), ("exec_gates", "K", np.float32),
               ("pair_of", "K", np.int32))


def plan_dict(hip, plan, B, K, E, budget):
    bc = min(budget, E)
    per = {"E": E, "K": K}
    out = {f: read_device(hip, getattr(plan, f), B * per[n], dt) for f, n, dt in PLAN_FIELDS}
    out["scores"] = read_device(hip, plan.scores, E, np.float32)
    out["counts"] = read_device(hip, plan.counts, E, np.int32)
    out["sel_ids"] = read_device(hip, plan.sel_ids, bc, np.int32)
    out["n_sel"] = read_device(hip, plan.n_sel, 1, np.int32)
    out["slot_of_expert"] = read_device(hip, plan.slot_of_expert, E, np.int32)
    out["offsets"] = read_device(hip, plan.offsets, bc + 1, np.int32)
    P = int(out["offsets"][-1])
    out["pair_tok"] = read_device(hip, plan.pair_tok, P, np.int32)
    out["pair_gate"] = read_device(hip, plan.pair_gate, P, np.float32)
    return out


def run_both(gu, gl, x, B, budget, hip):
    from paper_2609_36222_amd import binding as bd
    ws = gl.workspace(B, budget)
    y_ref, y_na = gl.y_like(B), gl.y_like(B)
    p_ref = bd.base_decode_layer(gl.desc, x, B, budget, 0, None, y_ref, ws)
    p_na = bd.base_decode_layer_noalloc(gl.desc, x, B, budget, 0, None, y_na)
    torch.cuda.synchronize()
    # the no-allocation call's plan lives outside the caller's workspace
    lo, hi = ws.data_ptr(), ws.data_ptr() + ws.numel()
    assert not (lo <= p_na.exec_ids < hi)
    ref = plan_dict(hip, p_ref, B, gl.K, gl.E, budget)
    got = plan_dict(hip, p_na, B, gl.K, gl.E, budget)
    for f in ref:
        assert np.array_equal(got[f].view(np.uint32) if got[f].dtype == np.float32 else got[f],
                              ref[f].view(np.uint32) if ref[f].dtype == np.float32 else ref[f]), f
    assert torch.equal(y_na.view(torch.int16), y_ref.view(torch.int16))
    return int(ref["n_sel"][0])


def test_noalloc_matches_workspace_call_twice(gu):
    """Qwen3-shaped layer (d=2048, E=128, top-8, I=768, packed bf16): batch
    256 at budget 32, then the first 100 tokens at budget 8 on the same
    scratch array."""
    print("no-alloc: qwen3_b256, B=256 budget 32, then B=100 budget 8", flush=True)
    hip = _hip()
    inp = W.layer_inputs("qwen3_b256")
    gl = gu.GpuLayer(inp, packed=True)
    x = gl.x(inp["x"])
    assert run_both(gu, gl, x, 256, 32, hip) == 32
    x2 = x[:100].contiguous()
    assert run_both(gu, gl, x2, 100, 8, hip) == 8


def test_noalloc_rejects_a_workspace_beyond_its_scratch(gu):
    """B = 1024 with K = 16 of 256 experts needs more than the 64 MiB array:
    BASE_ERR_WORKSPACE, before anything is enqueued."""
    from paper_2609_36222_amd import binding as bd
    inp = W.custom_layer(2048, 256, 16, 768, 8, seed=3)
    gl = gu.GpuLayer(inp)
    assert bd.base_workspace_bytes(gl.desc, 1024, 256) > bd.NOALLOC_SCRATCH_BYTES
    x = torch.zeros(1024, 2048, dtype=torch.bfloat16, device="cuda")
    y = torch.empty_like(x)
    with pytest.raises(bd.BaseError) as e:
        bd.base_decode_layer_noalloc(gl.desc, x, 1024, 256, 0, None, y)
    assert e.value.status == -6
