"""GPU calibration (App. A) against the oracle: the streaming statistics
(base_calib_accumulate) on the routes the GPU takes, and the fit
(base_calib_fit) against the oracle's ridge on the same statistics."""
import numpy as np
import pytest

import workloads as W
from oracle import calib, carith, method

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def gu(gpu):
    import gpu_util
    return gpu_util


def up(v):
    return (v + 255) // 256 * 256


def read_stats(stats, E, d):
    b = stats.cpu().numpy()
    o1 = up(E * 32)
    o2 = o1 + up(E * d * 8)
    o3 = o2 + up(E * d * 8)
    head = b[:E * 32].view(np.float64).reshape(E, 4)
    sz = b[o1:o1 + E * d * 8].view(np.float64).reshape(E, d)
    q = b[o2:o2 + E * d * 8].view(np.float64).reshape(E, d)
    G = b[o3:o3 + E * d * d * 4].view(np.float32).reshape(E, d, d)
    return head, sz, q, G


def oracle_stats(z_batches, inp, bf16):
    """The oracle's statistics on the canonical fp32 routes (the routes the
    GPU takes), expert outputs in fp64 (h rounded to bf16 for bf16 layers)."""
    sh = inp["shape"]
    ex = method.Experts(inp["w13"], inp["w2"], bf16)
    stats = [calib.ExpertStats(sh.d) for _ in range(sh.E)]
    for z in z_batches:
        _, ids, _ = carith.route(z, inp["w_router"], inp["b_router"], sh.K)
        z64 = z.astype(np.float64)
        nrm = np.linalg.norm(z64, axis=1, keepdims=True)
        zb = np.divide(z64, nrm, out=np.zeros_like(z64), where=nrm > 0)
        for u in np.unique(ids):
            tt = np.nonzero((ids == u).any(axis=1))[0]
            out = ex.forward(int(u), z64[tt])
            y = np.log(np.sum(out ** 2, axis=1) + calib.EPS)
            stats[u].update(zb[tt], y)
    return stats


def to_expert_stats(head, sz, q, G):
    E, d = sz.shape
    out = []
    for u in range(E):
        st = calib.ExpertStats(d)
        st.n = int(round(head[u, 0]))
        st.sy, st.syy = float(head[u, 1]), float(head[u, 2])
        st.sz, st.q, st.G = sz[u].copy(), q[u].copy(), G[u].copy()
        out.append(st)
    return out


def run_gpu_stats(gu, inp, batches):
    from paper_2609_36222_amd import binding as bd
    gl = gu.GpuLayer(inp)
    stats = bd.calib_stats(gl.desc)
    ws = None
    for z in batches:
        ws = bd.calib_accumulate(gl.desc, gl.x(z), z.shape[0], stats, ws)
    torch.cuda.synchronize()
    return gl, stats


CASES = {
    # fp32 tiny layer, its 2048 calibration tokens in batches of 256
    "tiny": lambda: (W.layer_inputs("tiny"), 256, 2048, 2e-5),
    # a bf16 layer, 1024 tokens in batches of 128 (and a ragged last one)
    "bf16": lambda: (W.custom_layer(512, 16, 4, 128, 8, seed=5), 128, 1000, 2e-3),
    # wider tokens, K = 16 of 48, batches of 97 (ragged throughout)
    "k16": lambda: (W.custom_layer(768, 48, 16, 64, 8, seed=22), 97, 700, 2e-3),
    # 120 tokens over 128 experts, top-2: many experts see 0, 1 or 2 tokens
    "sparse": lambda: (W.custom_layer(256, 128, 2, 64, 8, seed=23), 64, 120, 2e-3),
}


@pytest.mark.parametrize("case", list(CASES))
def test_calibration_statistics(gu, case):
    inp, bsz, ntok, ytol = CASES[case]()
    sh = inp["shape"]
    z = W.calibration_tokens(sh, n=ntok)
    batches = [z[i:i + bsz] for i in range(0, ntok, bsz)]
    print(f"calibration statistics {case}: {ntok} tokens", flush=True)
    gl, stats = run_gpu_stats(gu, inp, batches)
    head, sz, q, G = read_stats(stats, sh.E, sh.d)
    ref = oracle_stats(batches, inp, sh.bf16)
    for u in range(sh.E):
        r = ref[u]
        assert int(head[u, 0]) == r.n, u                       # the same routed pairs
        if r.n == 0:
            assert not np.any(sz[u]) and not np.any(G[u])
            continue
        assert abs(head[u, 1] - r.sy) <= ytol * r.n, u          # sum y
        assert abs(head[u, 2] - r.syy) <= 3 * ytol * r.n * (1 + abs(r.sy) / r.n), u
        assert np.max(np.abs(sz[u] - r.sz)) <= 1e-12 * r.n + 1e-12
        assert np.max(np.abs(q[u] - r.q)) <= ytol * r.n
        scale = max(1.0, float(np.max(np.abs(r.G))))
        assert np.max(np.abs(G[u] - r.G)) <= 1e-5 * scale, u    # fp32 Gram


@pytest.mark.parametrize("case", list(CASES))
def test_calibration_fit(gu, case):
    """base_calib_fit against the oracle's ridge (eigendecomposition, 25
    lambdas, evidence, bias correction) on the same statistics."""
    from paper_2609_36222_amd import binding as bd
    inp, bsz, ntok, _ = CASES[case]()
    sh = inp["shape"]
    z = W.calibration_tokens(sh, n=ntok)
    batches = [z[i:i + bsz] for i in range(0, ntok, bsz)]
    gl, stats = run_gpu_stats(gu, inp, batches)
    pa = torch.empty(sh.E, sh.d, dtype=torch.float32, device="cuda")
    pb = torch.empty(sh.E, dtype=torch.float32, device="cuda")
    lam = torch.empty(sh.E, dtype=torch.float32, device="cuda")
    bd.calib_fit(gl.desc, stats, calib.LAMBDAS, pa, pb, lam)
    pa, pb, lam = pa.cpu().numpy(), pb.cpu().numpy(), lam.cpu().numpy()
    for u, st in enumerate(to_expert_stats(*read_stats(stats, sh.E, sh.d))):
        f = calib.ridge_fit(st)
        if st.n == 0:
            assert not np.any(pa[u]) and pb[u] == 0.0
            continue
        assert lam[u] == np.float32(f["lam"]), u
        scale = max(1e-6, float(np.max(np.abs(f["a"]))))
        assert np.max(np.abs(pa[u] - f["a"])) <= 1e-4 * scale, u
        assert abs(pb[u] - f["b"]) <= 1e-4 * max(1.0, abs(f["b"])), u


def test_calibration_qwen3_shape(gu):
    """The Qwen3-shaped layer (d=2048, E=128, top-8, I=768, bf16), 768
    calibration tokens in 3 batches of 256 (App. A): head, sum z_bar and
    sum z_bar y of every expert in full; the fp32 Gram matrices (2048 x 2048
    each) and the fit's lambda, a and b on sampled experts (the most and
    least used, and two others)."""
    from paper_2609_36222_amd import binding as bd
    inp = W.layer_inputs("qwen3_b64")
    sh = inp["shape"]
    assert (sh.d, sh.E, sh.K, sh.I) == (2048, 128, 8, 768)
    z = W.calibration_tokens(sh, n=768)
    batches = [z[i:i + 256] for i in range(0, 768, 256)]
    print("calibration statistics qwen3: 768 tokens", flush=True)
    gl, stats = run_gpu_stats(gu, inp, batches)
    head, sz, q, G = read_stats(stats, sh.E, sh.d)
    # the oracle's statistics, the Gram only for the sampled experts
    ex = method.Experts(inp["w13"], inp["w2"], True)
    n = np.zeros(sh.E, np.int64)
    sy, syy = np.zeros(sh.E), np.zeros(sh.E)
    szr, qr = np.zeros((sh.E, sh.d)), np.zeros((sh.E, sh.d))
    rows = {u: [] for u in range(sh.E)}
    for zb_tok in batches:
        _, ids, _ = carith.route(zb_tok, inp["w_router"], inp["b_router"], sh.K)
        z64 = zb_tok.astype(np.float64)
        zbar = z64 / np.linalg.norm(z64, axis=1, keepdims=True)
        for u in np.unique(ids):
            tt = np.nonzero((ids == u).any(axis=1))[0]
            out = ex.forward(int(u), z64[tt])
            y = np.log(np.sum(out ** 2, axis=1) + calib.EPS)
            n[u] += len(tt)
            sy[u] += y.sum()
            syy[u] += y @ y
            szr[u] += zbar[tt].sum(axis=0)
            qr[u] += zbar[tt].T @ y
            rows[int(u)].append(zbar[tt])
    ytol = 2e-3
    for u in range(sh.E):
        assert int(head[u, 0]) == n[u], u
        if n[u] == 0:
            continue
        assert abs(head[u, 1] - sy[u]) <= ytol * n[u], u
        assert abs(head[u, 2] - syy[u]) <= 3 * ytol * n[u] * (1 + abs(sy[u]) / n[u]), u
        assert np.max(np.abs(sz[u] - szr[u])) <= 1e-12 * n[u] + 1e-12, u
        assert np.max(np.abs(q[u] - qr[u])) <= ytol * n[u], u
    used = [u for u in range(sh.E) if n[u] > 0]
    sample = sorted({int(max(used, key=lambda u: n[u])), int(min(used, key=lambda u: n[u])),
                     used[len(used) // 3], used[2 * len(used) // 3]})
    for u in sample:
        Zu = np.concatenate(rows[u])
        Gr = (Zu.T @ Zu)
        scale = max(1.0, float(np.max(np.abs(Gr))))
        assert np.max(np.abs(G[u] - Gr)) <= 1e-5 * scale, u
    # the fit on the device against the oracle's ridge on the same statistics
    pa = torch.empty(sh.E, sh.d, dtype=torch.float32, device="cuda")
    pb = torch.empty(sh.E, dtype=torch.float32, device="cuda")
    lam = torch.empty(sh.E, dtype=torch.float32, device="cuda")
    bd.calib_fit(gl.desc, stats, calib.LAMBDAS, pa, pb, lam)
    pa, pb, lam = pa.cpu().numpy(), pb.cpu().numpy(), lam.cpu().numpy()
    for u in sample:
        st = calib.ExpertStats(sh.d)
        st.n = int(round(head[u, 0]))
        st.sy, st.syy = float(head[u, 1]), float(head[u, 2])
        st.sz, st.q, st.G = sz[u].copy(), q[u].copy(), G[u].copy()
        f = calib.ridge_fit(st)
        assert lam[u] == np.float32(f["lam"]), u
        a_scale = max(1e-6, float(np.max(np.abs(f["a"]))))
        assert np.max(np.abs(pa[u] - f["a"])) <= 1e-4 * a_scale, u
        assert abs(pb[u] - f["b"]) <= 1e-4 * max(1.0, abs(f["b"])), u
