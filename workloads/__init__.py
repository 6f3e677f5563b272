"""Seeded synthetic inputs for the BASE decode hot path.

This module only draws random inputs. It holds none of the method's
arithmetic: no routing, no expert evaluation, no prediction, no selection.
Both the CPU oracle (``oracle/``) and the HIP path (``paper_2609_36222_amd``)
take their inputs from here, and neither imports the other.

The paper evaluates on real checkpoints (Qwen3-30B-A3B, DeepSeek-V2-Lite,
Qwen1.5-MoE-A2.7B) with FineWeb-Edu calibration text (Sec. 4 setup;
App. A "Calibration Details").  None of that is available here, so every
input is synthetic with the shapes of those models' MoE layers:

* hidden states: i.i.d. N(0,1) rows passed through RMSNorm (unit gain,
  eps 1e-6), computed in fp32 and stored bf16 (fp32 for the tiny layer);
* the batch-256 Qwen3-shaped layer mixes 128 rows drawn around 4 shared
  Gaussian centres (centre + 0.1 N(0,I)) with 128 i.i.d. rows, interleaved
  by a seeded shuffle, to vary the size of the batch union;
* router weights N(0, 0.075) with a per-expert bias log(p_e), p_e
  proportional to rank^-1.1 over a seeded permutation (a Zipf(1.1)
  popularity law; with this scale a Qwen3-shaped router at batch 16 gives a
  mean top-1 union near the 13.34 experts the paper reports in App. F);
* SwiGLU expert weights with std 1/sqrt(fan_in), stored bf16;
* a synthetic linear predictor (a_u, b_u) for the large layers (the tiny
  layer's predictor is fitted by the oracle on its calibration tokens).

bf16 tensors are returned as ``uint16`` bit patterns (round-to-nearest-even
from the fp32 draw).  Generation is chunked over child seeds so the values
do not depend on the number of threads used.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os

import numpy as np

SEED_ROOT = 2609

# stream ids inside a layer's seed sequence
_S_ROUTER, _S_BIAS, _S_CALIB, _S_EXPERT, _S_TOKENS, _S_PRED = 0, 1, 2, 3, 4, 5
_S_SHARED, _S_SHARED_GATE = 6, 7


@dataclasses.dataclass(frozen=True)
class LayerShape:
    name: str
    index: int          # position in the workload table (enters the seed)
    d: int              # hidden size
    E: int              # routed experts
    K: int              # experts per token (top-K)
    I: int              # SwiGLU intermediate size
    B: int              # decode batch (one token per sequence)
    budgets: tuple      # expert budgets B_e evaluated on this layer
    bf16: bool          # bf16 activations and expert weights (else fp32)
    layers: int = 1     # stacked MoE layers (residual carried)
    clustered: bool = False
    router_std: float = 0.075
    bias_kind: str = "zipf"   # "zipf" or "normal"
    bias_std: float = 0.5
    rmsnorm: bool = True
    calib_tokens: int = 8192
    norm_topk: int = 1      # 1: top-K weights renormalised; 0: raw softmax
    n_shared: int = 0       # always-active shared experts (the routed shape)
    shared_gate: bool = False   # sigmoid gate on the shared experts' sum


WORKLOADS = {
    # d=256, E=16, top-2, I=512, batch 8, B_e=6, everything fp32,
    # router N(0,0.02) plus bias N(0,0.5), experts N(0,1/sqrt(d)),
    # predictor fitted on 2048 calibration tokens.
    "tiny": LayerShape("tiny", 0, 256, 16, 2, 512, 8, (6,), False,
                       router_std=0.02, bias_kind="normal", rmsnorm=False,
                       calib_tokens=2048),
    # OLMoE-shaped: d=2048, E=64, top-8, I=1024, batch 32.
    "olmoe": LayerShape("olmoe", 1, 2048, 64, 8, 1024, 32, (16, 32), True),
    # Qwen3-30B-A3B-shaped layer at batch 64.
    "qwen3_b64": LayerShape("qwen3_b64", 2, 2048, 128, 8, 768, 64,
                            (16, 32, 64), True),
    # Same layer at batch 256, half the batch clustered.
    "qwen3_b256": LayerShape("qwen3_b256", 3, 2048, 128, 8, 768, 256,
                             (32, 64, 128), True, clustered=True),
    # 48 stacked Qwen3-shaped MoE layers, batch 128, B_e=24 per layer.
    "qwen3_stack48": LayerShape("qwen3_stack48", 4, 2048, 128, 8, 768, 128,
                                (24,), True, layers=48),
    # Mixtral-shaped: few large experts.
    "mixtral": LayerShape("mixtral", 5, 4096, 8, 2, 14336, 128, (4,), True),
    # DeepSeek-V2-Lite-shaped: 64 routed experts, top-6, I=1408, raw softmax
    # weights, 2 shared experts without a gate.
    "deepseek_v2_lite": LayerShape("deepseek_v2_lite", 6, 2048, 64, 6, 1408, 64,
                                   (8, 16, 32), True, norm_topk=0, n_shared=2),
    # Qwen1.5-MoE-A2.7B-shaped: 60 routed experts, top-4, I=1408, raw softmax
    # weights, one shared expert of intermediate size 5632 given as 4 of
    # width 1408, with a sigmoid gate.
    "qwen15_moe": LayerShape("qwen15_moe", 7, 2048, 60, 4, 1408, 64, (8, 16), True,
                             norm_topk=0, n_shared=4, shared_gate=True),
}


def seed_seq(shape: LayerShape, layer: int, stream: int, data_seed: int = 0):
    return np.random.SeedSequence([SEED_ROOT, shape.index, layer, stream,
                                   data_seed])


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round finite fp32 values to bf16 (nearest, ties to even); return
    uint16 bits.  (No finite value overflows the 32-bit sum.)"""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u >> 16) & np.uint32(1)
    r += u
    r += np.uint32(0x7FFF)
    r >>= 16
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32)
            << 16).view(np.float32)


def _normal_chunked(ss: np.random.SeedSequence, n: int, std: float,
                    chunk: int = 1 << 22, bf16: bool = False) -> np.ndarray:
    """n draws of N(0, std^2) in fp32, chunk i from child seed i; returned
    as bf16 bits (uint16) when bf16 is set."""
    out = np.empty(n, dtype=np.uint16 if bf16 else np.float32)
    nchunks = max(1, (n + chunk - 1) // chunk)
    children = ss.spawn(nchunks)

    def fill(i):
        lo, hi = i * chunk, min(n, (i + 1) * chunk)
        g = np.random.Generator(np.random.PCG64(children[i]))
        v = g.standard_normal(hi - lo, dtype=np.float32)
        if std != 1.0:
            v *= np.float32(std)
        out[lo:hi] = f32_to_bf16_bits(v) if bf16 else v

    workers = min(16, os.cpu_count() or 1, nchunks)
    if workers <= 1:
        for i in range(nchunks):
            fill(i)
    else:
        with _cf.ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill, range(nchunks)))
    return out


def _rmsnorm_rows(z: np.ndarray, eps: float = 1e-6) -> np.ndarray:
    """RMSNorm with unit gain, in fp32 (part of the input recipe)."""
    z = z.astype(np.float32)
    ms = np.mean(z.astype(np.float64) ** 2, axis=1, keepdims=True)
    return (z / np.sqrt(ms + eps)).astype(np.float32)


def hidden_states(shape: LayerShape, n: int, layer: int = 0,
                  stream: int = _S_TOKENS, data_seed: int = 0,
                  clustered=None) -> np.ndarray:
    """n hidden-state rows [n, d] as fp32 values (bf16-representable when
    the layer is bf16)."""
    ss = seed_seq(shape, layer, stream, data_seed)
    g = np.random.Generator(np.random.PCG64(ss))
    d = shape.d
    clustered = shape.clustered if clustered is None else clustered
    z = g.standard_normal((n, d), dtype=np.float32)
    if clustered and n >= 2:
        nc = n // 2
        centres = g.standard_normal((4, d), dtype=np.float32)
        cid = g.integers(0, 4, size=nc)
        zc = centres[cid] + np.float32(0.1) * g.standard_normal(
            (nc, d), dtype=np.float32)
        z[:nc] = zc
        z = z[g.permutation(n)]
    if shape.rmsnorm:
        z = _rmsnorm_rows(z)
    if shape.bf16:
        z = bf16_bits_to_f32(f32_to_bf16_bits(z))
    return np.ascontiguousarray(z, dtype=np.float32)


def router(shape: LayerShape, layer: int = 0):
    """Router weight [E, d] fp32 and bias [E] fp32."""
    g = np.random.Generator(np.random.PCG64(seed_seq(shape, layer, _S_ROUTER)))
    w = (g.standard_normal((shape.E, shape.d), dtype=np.float32)
         * np.float32(shape.router_std))
    gb = np.random.Generator(np.random.PCG64(seed_seq(shape, layer, _S_BIAS)))
    if shape.bias_kind == "zipf":
        perm = gb.permutation(shape.E)
        rank = np.empty(shape.E, dtype=np.float64)
        rank[perm] = np.arange(1, shape.E + 1, dtype=np.float64)
        p = rank ** -1.1
        p /= p.sum()
        b = np.log(p).astype(np.float32)
    else:
        b = gb.standard_normal(shape.E, dtype=np.float32) * np.float32(
            shape.bias_std)
    return np.ascontiguousarray(w), np.ascontiguousarray(b)


def experts(shape: LayerShape, layer: int = 0):
    """SwiGLU expert weights.

    Returns (w13, w2): w13 [E, 2I, d] (rows 0..I-1 gate, I..2I-1 up),
    w2 [E, d, I].  uint16 bf16 bits for bf16 layers, fp32 otherwise.
    Tiny layer: all three matrices std 1/sqrt(d).  Others: std 1/sqrt(fan_in).
    """
    E, d, I = shape.E, shape.d, shape.I
    ss = seed_seq(shape, layer, _S_EXPERT)
    s13, s2 = ss.spawn(2)
    std13 = 1.0 / np.sqrt(d)
    std2 = 1.0 / np.sqrt(d) if not shape.bf16 else 1.0 / np.sqrt(I)
    w13 = _normal_chunked(s13, E * 2 * I * d, std13, bf16=shape.bf16)
    w2 = _normal_chunked(s2, E * d * I, std2, bf16=shape.bf16)
    return w13.reshape(E, 2 * I, d), w2.reshape(E, d, I)


def shared_experts(shape: LayerShape, layer: int = 0):
    """The shared experts, with the routed experts' recipe and shape:
    (w13 [S, 2I, d], w2 [S, d, I]) as bf16 bits, and the gate vector [d]
    fp32 (N(0, 1/d), so x . gate is about N(0, 1)) or None."""
    S, d, I = shape.n_shared, shape.d, shape.I
    ss = seed_seq(shape, layer, _S_SHARED)
    s13, s2 = ss.spawn(2)
    w13 = _normal_chunked(s13, S * 2 * I * d, 1.0 / np.sqrt(d), bf16=shape.bf16)
    w2 = _normal_chunked(s2, S * d * I, 1.0 / np.sqrt(I), bf16=shape.bf16)
    gate = None
    if shape.shared_gate:
        g = np.random.Generator(np.random.PCG64(seed_seq(shape, layer, _S_SHARED_GATE)))
        gate = (g.standard_normal(d) / np.sqrt(d)).astype(np.float32)
    return w13.reshape(S, 2 * I, d), w2.reshape(S, d, I), gate


def synthetic_predictor(shape: LayerShape, layer: int = 0):
    """A synthetic log-energy predictor (a [E,d] fp32, b [E] fp32).

    Stands in for a calibrated one on the large layers: a_u has i.i.d.
    N(0, (0.3)^2) entries, so a_u.z_bar varies with std 0.3 over unit
    vectors; b_u = log(d * 0.18) + N(0, 0.25^2), roughly the log output
    energy of a random SwiGLU expert with this module's weight scales.
    """
    g = np.random.Generator(np.random.PCG64(seed_seq(shape, layer, _S_PRED)))
    a = g.standard_normal((shape.E, shape.d), dtype=np.float32) * np.float32(0.3)
    b = (np.float32(np.log(shape.d * 0.18))
         + g.standard_normal(shape.E, dtype=np.float32) * np.float32(0.25))
    return np.ascontiguousarray(a), np.ascontiguousarray(b.astype(np.float32))


def calibration_tokens(shape: LayerShape, layer: int = 0, n=None):
    n = shape.calib_tokens if n is None else n
    return hidden_states(shape, n, layer=layer, stream=_S_CALIB,
                         clustered=False)


def decode_tokens(shape: LayerShape, layer: int = 0, data_seed: int = 0,
                  B=None):
    return hidden_states(shape, shape.B if B is None else B, layer=layer,
                         stream=_S_TOKENS, data_seed=data_seed)


def stack_layer_input(h: np.ndarray, bf16: bool = True) -> np.ndarray:
    """Input of a stacked layer from the residual stream h [B, d]: the
    unit-gain RMSNorm a pre-norm decoder block applies before its MoE, in
    fp32, rounded to bf16 for bf16 layers.  The layer then adds its MoE
    output to h itself (the residual), so the stream grows slowly with depth
    instead of compounding the experts' gain."""
    z = _rmsnorm_rows(h)
    if bf16:
        z = bf16_bits_to_f32(f32_to_bf16_bits(z))
    return np.ascontiguousarray(z, dtype=np.float32)


def layer_inputs(name: str, layer: int = 0, data_seed: int = 0,
                 with_experts: bool = True, B=None):
    """Everything one decode layer consumes, as numpy arrays."""
    shape = WORKLOADS[name]
    wr, br = router(shape, layer)
    out = dict(shape=shape, x=decode_tokens(shape, layer, data_seed, B),
               w_router=wr, b_router=br)
    pa, pb = synthetic_predictor(shape, layer)
    out["pred_a"], out["pred_b"] = pa, pb
    if with_experts:
        out["w13"], out["w2"] = experts(shape, layer)
        if shape.n_shared:
            out["w13_shared"], out["w2_shared"], out["shared_gate"] = shared_experts(shape, layer)
    return out


def rules_layer(seed=0, d=256, E=32, K=4, I=128, B=16, n_calib=4096):
    """A small fp32 layer for comparing selection rules, whose experts
    differ in output energy in two ways the rules can see or miss: a
    per-expert output scale (log-normal, sigma 0.5) and a preferred input
    direction (the gate rows of expert u lean along a unit vector v_u, so
    its energy grows with z . v_u).  Returns the router, the row-major fp32
    experts, calibration tokens and decode batches (RMS-normalised N(0, I)
    rows); the seeds are this function's own."""
    g = np.random.default_rng(np.random.SeedSequence([SEED_ROOT, 77, seed]))
    wr = (g.standard_normal((E, d)) * 0.08).astype(np.float32)
    br = (g.standard_normal(E) * 0.3).astype(np.float32)
    w13 = (g.standard_normal((E, 2 * I, d)) / np.sqrt(d)).astype(np.float32)
    scale = np.exp(g.standard_normal(E) * 0.5)
    w2 = (g.standard_normal((E, d, I)) / np.sqrt(I) * scale[:, None, None]).astype(np.float32)
    v = g.standard_normal((E, d))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    w13[:, :I, :] += (8.0 * v[:, None, :] * g.standard_normal((E, I, 1)) / np.sqrt(d)).astype(np.float32)

    def rows(n):
        z = g.standard_normal((n, d))
        return _rmsnorm_rows(z)

    calib = rows(n_calib)
    batches = [rows(B) for _ in range(24)]
    return dict(w_router=wr, b_router=br, w13=w13, w2=w2, calib=calib,
                batches=batches, K=K)


def custom_layer(d, E, K, I, B, bf16=True, seed=0, router_std=0.075,
                 zipf_bias=True, rmsnorm=True, identical_tokens=False,
                 zero_token=False, n_shared=0, shared_gate=False):
    """A seeded layer of arbitrary shape for edge cases (same recipe as the
    named workloads; index 99 keeps its seeds apart from theirs), with
    n_shared always-active shared experts (bf16) when asked."""
    shape = LayerShape(f"custom_d{d}_E{E}_K{K}_I{I}_B{B}_S{n_shared}", 99, d, E, K, I, B,
                       (1,), bf16, router_std=router_std,
                       bias_kind="zipf" if zipf_bias else "normal",
                       rmsnorm=rmsnorm, n_shared=n_shared, shared_gate=shared_gate)
    wr, br = router(shape, seed)
    pa, pb = synthetic_predictor(shape, seed)
    x = decode_tokens(shape, seed)
    if identical_tokens:
        x[:] = x[0]
    if zero_token:
        x[0] = 0.0
    w13, w2 = experts(shape, seed)
    out = dict(shape=shape, x=x, w_router=wr, b_router=br, pred_a=pa,
               pred_b=pb, w13=w13, w2=w2)
    if n_shared:
        out["w13_shared"], out["w2_shared"], out["shared_gate"] = shared_experts(shape, seed)
    return out
