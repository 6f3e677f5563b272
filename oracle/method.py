"""TEST INFRASTRUCTURE ONLY -- the CPU oracle of BASE's decode hot path.

Plain NumPy, written from the paper ("BASE: Batch-Aware Selection of Experts
Using Predicted Removal Error for Efficient MoE Decoding").  Two levels:

* definition level, float64: the paper's formulas as written (``*64``
  functions): router (Sec. 3.1), SwiGLU experts, dense top-K MoE (Sec. 3.1),
  removal error by actually dropping an expert (Sec. 3.2, eq.
  individual_expert_damage), exact and additive batch error (eq.
  error_decomposition), predictor (eq. log_energy_predictor), restricted
  MoE after backfill (Sec. 3.5), cross-term statistics (App. B, eqs.
  weighted_mean_cosine .. crossterm_exact_identity), greedy cross-term-aware
  selection (Sec. 3.3), oracle-energy score and energy retained (App. F,
  eqs. oracle_expert_score, energy_retained);
* canonical fp32 level: the fixed-order single-precision sequence of the
  scoring path (``carith``), whose integer decisions (top-K ids, selected
  set, executed experts, compaction) a GPU implementation must reproduce
  bit for bit.

The integer logic (selection, backfill, compaction) takes its keys in
whatever precision it is given and is shared by both levels.

This package shares no code with the HIP library and is never imported by
it.  Only tests, the smoke check and the benchmark's CPU-baseline leg use it.
"""
from __future__ import annotations

import itertools

import numpy as np

from . import carith

GATE_PAPER, GATE_RENORM = 0, 1      # flags bit 0
FILL_BACKFILL, FILL_DROP = 0, 2     # flags bit 1

# Selection rules (App. selection-rule ablation): the per-pair score whose
# batch sum D_u ranks the experts.  SCORE_BASE is the method.
SCORE_BASE, SCORE_TOP1, SCORE_WEIGHT, SCORE_WEIGHT_SQ, SCORE_STATIC = 0, 1, 2, 3, 4
SCORE_RULES = (SCORE_BASE, SCORE_TOP1, SCORE_WEIGHT, SCORE_WEIGHT_SQ, SCORE_STATIC)


# ------------------------------------------------------------ bf16 helpers --
def bf16_round(a):
    """Round to the nearest bf16 value (ties to even), returned as fp32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32)


def bf16_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32)
            << 16).view(np.float32)


# ------------------------------------------------------ router, fp64 level --
def route64(x, w_router, b_router, K, norm_topk=1):
    """Sec. 3.1: logits l = x W_r^T + beta; R_t = top-K of the softmax
    (order: logit desc, expert index asc); w_{t,u} = p_{t,u} / sum_{R_t} p
    (norm_topk=1) or the raw softmax probability (norm_topk=0)."""
    x = np.asarray(x, np.float64)
    l = x @ np.asarray(w_router, np.float64).T
    if b_router is not None:
        l = l + np.asarray(b_router, np.float64)
    B, E = l.shape
    ids = np.empty((B, K), np.int32)
    w = np.empty((B, K), np.float64)
    for t in range(B):
        order = np.lexsort((np.arange(E), -l[t]))
        ids[t] = order[:K]
        p = np.exp(l[t] - l[t].max())
        den = p[ids[t]].sum() if norm_topk else p.sum()
        w[t] = p[ids[t]] / den
    return l, ids, w


# ------------------------------------------------------------- experts ------
def silu(a):
    return a / (1.0 + np.exp(-a))


def expert_forward64(z, w13_u, w2_u, round_h_bf16=False, dtype=np.float64):
    """E_u(z) = W_d (silu(W_g z) * (W_u z)) for rows z [n, d], fp64.

    w13_u [2I, d] (gate rows then up rows), w2_u [d, I], given as fp32
    arrays holding the stored values.  round_h_bf16 rounds the SwiGLU
    activation to bf16 before the down projection, the precision at which a
    bf16 serving stack feeds it to the second matrix product.  dtype: the
    arithmetic (fp64, the definition every check uses; fp32 only for the
    timed CPU baseline of the benchmark)."""
    z = np.asarray(z, dtype)
    I = w2_u.shape[1]
    gu = z @ np.asarray(w13_u, dtype).T
    h = silu(gu[:, :I]) * gu[:, I:]
    if round_h_bf16:
        h = bf16_round(h.astype(np.float32)).astype(dtype)
    return h @ np.asarray(w2_u, dtype).T


class Experts:
    """Expert weights as fp32 values (bf16 bit patterns widened exactly).

    dtype: the FFN arithmetic (fp64 for every check; see widened())."""

    def __init__(self, w13, w2, bf16, dtype=np.float64):
        self.bf16 = bf16
        self._w13, self._w2 = w13, w2
        self._widened = False
        self.dtype = dtype
        self.E = w13.shape[0]
        self.I = w2.shape[2]
        self.d = w2.shape[1]

    def widened(self, dtype):
        """The same experts with the FFN computed in dtype on weights widened
        to dtype once, on an expert's first use, and kept (the benchmark's CPU
        baseline: fp32 BLAS on weights converted before its timed region)."""
        out = Experts(self._w13, self._w2, self.bf16, dtype)
        out._widened = {}
        return out

    def _weights(self, u, which):
        if self._widened is not False:
            key = (u, which)
            if key not in self._widened:
                a = (self._w13 if which == 0 else self._w2)[u]
                a = bf16_to_f32(a) if self.bf16 else np.asarray(a, np.float32)
                self._widened[key] = np.ascontiguousarray(a, self.dtype)
            return self._widened[key]
        a = (self._w13 if which == 0 else self._w2)[u]
        return bf16_to_f32(a) if self.bf16 else np.asarray(a, np.float32)

    def w13(self, u):
        return self._weights(u, 0)

    def w2(self, u):
        return self._weights(u, 1)

    def forward(self, u, z, round_h_bf16=None):
        rh = self.bf16 if round_h_bf16 is None else round_h_bf16
        return expert_forward64(z, self.w13(u), self.w2(u), rh, self.dtype)


def expert_outputs(experts, x, ids, round_h_bf16=False):
    """out[t, k] = E_{ids[t,k]}(x_t) for every routed pair, [B, K, d]."""
    B, K = ids.shape
    out = np.zeros((B, K, experts.d), np.float64)
    for u in np.unique(ids):
        tt, kk = np.nonzero(ids == u)
        out[tt, kk] = experts.forward(int(u), x[tt], round_h_bf16)
    return out


def moe_dense64(x, ids, w, experts, round_h_bf16=False):
    """Sec. 3.1: y_t = sum_{u in R_t} w_{t,u} E_u(z_t)."""
    eo = expert_outputs(experts, x, ids, round_h_bf16)
    return np.einsum("tk,tkd->td", np.asarray(w, np.float64), eo)


def removal_error64(x, ids, w, experts, eo=None):
    """True removal error by actually dropping each routed expert with the
    weights fixed: r[t,k] = ||y_t - y_t^(-u)||^2 (Sec. 3.2, 'individual
    damage'); returns (r, energy) with energy[t,k] = ||E_u(z_t)||^2."""
    if eo is None:
        eo = expert_outputs(experts, x, ids)
    w = np.asarray(w, np.float64)
    y = np.einsum("tk,tkd->td", w, eo)
    B, K = ids.shape
    r = np.empty((B, K))
    for k in range(K):
        keep = [q for q in range(K) if q != k]
        y_minus = np.einsum("tk,tkd->td", w[:, keep], eo[:, keep])
        r[:, k] = np.sum((y - y_minus) ** 2, axis=1)
    energy = np.sum(eo ** 2, axis=2)
    return r, energy


def oracle_scores64(ids, w, energy, E):
    """App. F eq. oracle_expert_score: D*_u = sum_t w^2 ||E_u(z_t)||^2
    (equal to eq. individual_expert_damage's D_u)."""
    D = np.zeros(E)
    np.add.at(D, ids.ravel(), (np.asarray(w, np.float64) ** 2 * energy).ravel())
    return D


def exact_error64(ids, w, eo, A):
    """eq. error_decomposition: sum_t || sum_{u in R_t \\ A} w E_u(z_t) ||^2."""
    A = set(int(a) for a in A)
    mask = np.array([[int(u) not in A for u in row] for row in ids], float)
    miss = np.einsum("tk,tkd->td", np.asarray(w, np.float64) * mask, eo)
    return float(np.sum(miss ** 2))


def additive_error64(D, A):
    """E_add(A) = sum_{u not in A} D_u."""
    A = set(int(a) for a in A)
    return float(sum(D[u] for u in range(len(D)) if u not in A))


# ----------------------------------------------------- predictor, fp64 -----
def predict64(x, pred_a, pred_b, ids, w):
    """eq. log_energy_predictor: s_hat = a_u^T z_bar + b_u, e_hat = exp(s_hat),
    per-pair cost w^2 e_hat, with z_bar = z / ||z||."""
    x = np.asarray(x, np.float64)
    nrm = np.linalg.norm(x, axis=1, keepdims=True)
    zb = np.divide(x, nrm, out=np.zeros_like(x), where=nrm > 0)
    A = np.asarray(pred_a, np.float64)
    s = np.einsum("td,tkd->tk", zb, A[ids]) + np.asarray(pred_b, np.float64)[ids]
    return np.asarray(w, np.float64) ** 2 * np.exp(s)


def pair_scores64(rule, x, pred_a, pred_b, ids, w):
    """Per routed pair score of each selection rule, fp64 (App.
    selection-rule ablation): BASE w^2 exp(a_u . z_bar + b_u); TOP1 1 for
    the token's first-ranked route and 0 for the others (so that D_u > 0
    exactly when u is some token's top-1); WEIGHT w; WEIGHT_SQ w^2; STATIC
    w^2 mu_u, the expert's mean calibration energy, with mu_u = exp(b_u)
    (pred_b holds log mu_u)."""
    w = np.asarray(w, np.float64)
    if rule == SCORE_BASE:
        return predict64(x, pred_a, pred_b, ids, w)
    if rule == SCORE_TOP1:
        c = np.zeros(w.shape)
        c[:, 0] = 1.0
        return c
    if rule == SCORE_WEIGHT:
        return w.copy()
    if rule == SCORE_WEIGHT_SQ:
        return w ** 2
    if rule == SCORE_STATIC:
        return w ** 2 * np.exp(np.asarray(pred_b, np.float64)[ids])
    raise ValueError(rule)


def pair_scores_c(rule, x, pred_a, pred_b, ids, w):
    """The same scores at the canonical fp32 level: BASE is carith.predict;
    WEIGHT_SQ is one fp32 product w * w; STATIC is (w * w) * cexp(b_u), the
    predictor's sequence with a_u . z_bar = 0; TOP1 and WEIGHT are exact."""
    w = np.asarray(w, np.float32)
    if rule == SCORE_BASE:
        return carith.predict(x, pred_a, pred_b, ids, w)
    if rule == SCORE_TOP1:
        c = np.zeros(w.shape, np.float32)
        c[:, 0] = np.float32(1.0)
        return c
    if rule == SCORE_WEIGHT:
        return w.copy()
    if rule == SCORE_WEIGHT_SQ:
        return (w * w).astype(np.float32)
    if rule == SCORE_STATIC:
        e = carith.cexp(np.asarray(pred_b, np.float32)[ids])
        return ((w * w) * e).astype(np.float32)
    raise ValueError(rule)


def aggregate64(ids, cost, E):
    """D_hat_u = sum_{t: u in R_t} cost(t,u); counts of routing tokens."""
    D = np.zeros(E)
    np.add.at(D, ids.ravel(), np.asarray(cost, np.float64).ravel())
    counts = np.bincount(ids.ravel(), minlength=E).astype(np.int32)
    return D, counts


# -------------------------------------------------------------- selection ---
def select(scores, counts, budget, binary=False):
    """Sec. 3.4/3.5: keep the n_sel = min(budget, |U|) experts of the batch
    union U = {u : count_u > 0} that come first in the order (score desc,
    index asc).  With `binary` (the top-1-union rule) the order uses only
    whether the score is positive (union membership), then the index.
    Returns sel_ids [budget] (rank order, -1 padded), n_sel,
    slot_of_expert [E] (rank, or -1 when not retained)."""
    E = len(scores)
    U = [u for u in range(E) if counts[u] > 0]
    if binary:
        U.sort(key=lambda u: (-(1.0 if scores[u] > 0 else 0.0), u))
    else:
        U.sort(key=lambda u: (-scores[u], u))
    n_sel = min(budget, len(U))
    sel = np.full(budget, -1, np.int32)
    slot = np.full(E, -1, np.int32)
    for r, u in enumerate(U[:n_sel]):
        sel[r] = u
        slot[u] = r
    return sel, n_sel, slot


def token_order(l_t):
    """The token's full router ranking: logit desc, expert index asc."""
    E = len(l_t)
    return np.lexsort((np.arange(E), -np.asarray(l_t)))


def backfill(logits, ids, slot_of, n_sel, K, flags=0):
    """Sec. 3.5: each token executes its K highest-ranked experts inside the
    active set (backfill), or only its routed experts that are retained
    (drop, App. fill-rule ablation).  Returns exec_ids [B,K] (-1 padded) and
    the number executed per token."""
    B = logits.shape[0]
    ex = np.full((B, K), -1, np.int32)
    n = np.zeros(B, np.int32)
    drop = bool(flags & FILL_DROP)
    for t in range(B):
        if drop:
            lst = [int(u) for u in ids[t] if slot_of[u] >= 0]
        else:
            order = token_order(logits[t])
            lst = [int(u) for u in order if slot_of[u] >= 0][:min(K, n_sel)]
        ex[t, :len(lst)] = lst
        n[t] = len(lst)
    return ex, n


def gates_c(logits, ids, exec_ids, n_exec, norm_topk=1, flags=0):
    """Canonical fp32 gates (Sec. 3.5): original router scores over the
    original top-K denominator, or renormalised over the executed experts."""
    B, K = exec_ids.shape
    g = np.zeros((B, K), np.float32)
    for t in range(B):
        m = int(n_exec[t])
        if m:
            g[t, :m] = carith.gates(logits[t], ids[t], exec_ids[t, :m],
                                    norm_topk, bool(flags & GATE_RENORM))
    return g


def gates64(logits, ids, exec_ids, n_exec, norm_topk=1, flags=0):
    B, K = exec_ids.shape
    g = np.zeros((B, K))
    for t in range(B):
        lt = np.asarray(logits[t], np.float64)
        p = np.exp(lt - lt[ids[t, 0]])
        m = int(n_exec[t])
        if not m:
            continue
        num = p[exec_ids[t, :m]]
        if flags & GATE_RENORM:
            den = num.sum()
        else:
            den = p[ids[t]].sum() if norm_topk else p.sum()
        g[t, :m] = num / den
    return g


def compact(exec_ids, n_exec, slot_of, gates, budget, n_shared=0, shared_gates=None):
    """Token-to-expert compaction: the executed pairs (t, j) sorted by
    (slot, token).  offsets[s] = first pair of slot s (offsets[budget] = P),
    pair_tok/pair_gate per pair, pair_of[t, j] = pair index (or -1).  With
    n_shared shared experts, shared expert i follows as B more pairs (every
    token in order, gate shared_gates[t] or 1): offsets[budget + i] is its
    first pair, offsets[budget + n_shared] the total, and pair_of gets
    columns K + i."""
    B, K = exec_ids.shape
    pairs = []
    for t in range(B):
        for j in range(int(n_exec[t])):
            pairs.append((int(slot_of[exec_ids[t, j]]), t, j))
    pairs.sort()
    P = len(pairs)
    offsets = np.full(budget + 1, P, np.int32)
    pair_tok = np.zeros(max(P, 1), np.int32)[:P]
    pair_gate = np.zeros(P, np.float32)
    pair_of = np.full((B, K), -1, np.int32)
    seen = set()
    for p, (s, t, j) in enumerate(pairs):
        if s not in seen:
            offsets[s] = p
            seen.add(s)
        pair_tok[p] = t
        pair_gate[p] = gates[t, j]
        pair_of[t, j] = p
    # slots without pairs start where the next populated slot starts
    for s in range(budget - 1, -1, -1):
        if s not in seen:
            offsets[s] = offsets[s + 1]
    if n_shared:
        g = np.ones(B, np.float32) if shared_gates is None else np.asarray(shared_gates, np.float32)
        offsets = np.concatenate([offsets, P + B * np.arange(1, n_shared + 1)]).astype(np.int32)
        pair_tok = np.concatenate([pair_tok] + [np.arange(B, dtype=np.int32)] * n_shared)
        pair_gate = np.concatenate([pair_gate] + [g] * n_shared).astype(np.float32)
        pair_of = np.concatenate(
            [pair_of] + [(P + i * B + np.arange(B, dtype=np.int32))[:, None]
                         for i in range(n_shared)], axis=1).astype(np.int32)
    return offsets, pair_tok, pair_gate, pair_of


def shared_gate_c(x, gate):
    """The shared experts' gate at the canonical fp32 level: s = x . gate in
    the fixed dot-product order, g = 1 / (1 + exp(-s)) (one fp32 operation at
    a time, exp as cexp)."""
    s = carith.cdot_matrix(np.asarray(x, np.float32), np.asarray(gate, np.float32)[None, :])[:, 0]
    e = carith.cexp((-s).astype(np.float32))
    den = (np.float32(1.0) + e).astype(np.float32)
    return (np.float32(1.0) / den).astype(np.float32)


def shared_gate64(x, gate):
    s = np.asarray(x, np.float64) @ np.asarray(gate, np.float64)
    return 1.0 / (1.0 + np.exp(-s))


def moe_restricted64(x, exec_ids, n_exec, gates, experts, residual=None,
                     round_h_bf16=None):
    """Sec. 3.5: y_t = sum_{v in X_t} g_{t,v} E_v(z_t) (+ residual), fp64."""
    B, K = exec_ids.shape
    y = np.zeros((B, experts.d))
    if residual is not None:
        y += np.asarray(residual, np.float64)
    g = np.asarray(gates, np.float64)
    for u in np.unique(exec_ids[exec_ids >= 0]):
        tt, jj = np.nonzero(exec_ids == u)
        out = experts.forward(int(u), np.asarray(x)[tt], round_h_bf16)
        np.add.at(y, tt, g[tt, jj][:, None] * out)
    return y


# ------------------------------------------------ canonical fp32 pipeline --
def decode_layer_c(x, w_router, b_router, pred_a, pred_b, K, budget,
                   experts=None, norm_topk=1, flags=0, residual=None,
                   score_rule=SCORE_BASE, shared=None):
    """The whole hot path at the canonical fp32 level (ids, gates and plan)
    with the expert FFN in fp64 on the same plan.  shared: None or a dict
    with the always-active shared experts ("experts": Experts, "gate": [d]
    or None): they run on every token, outside the budget, and add
    g_t S_i(x_t) to y (g_t = sigmoid(x_t . gate) or 1)."""
    logits, ids, w = carith.route(x, w_router, b_router, K, norm_topk)
    cost = pair_scores_c(score_rule, x, pred_a, pred_b, ids, w)
    E = logits.shape[1]
    scores, counts = carith.aggregate(ids, cost, E)
    budget_c = min(budget, E)
    sel, n_sel, slot = select(scores, counts, budget_c,
                              binary=score_rule == SCORE_TOP1)
    ex, n_ex = backfill(logits, ids, slot, n_sel, K, flags)
    g = gates_c(logits, ids, ex, n_ex, norm_topk, flags)
    ns = 0 if shared is None else shared["experts"].E
    sg = None
    if ns and shared.get("gate") is not None:
        sg = shared_gate_c(x, shared["gate"])
    offsets, pair_tok, pair_gate, pair_of = compact(ex, n_ex, slot, g,
                                                    budget_c, ns, sg)
    out = dict(logits=logits, topk_ids=ids, topk_w=w, cost=cost,
               scores=scores, counts=counts, sel_ids=sel, n_sel=n_sel,
               slot_of_expert=slot, exec_ids=ex, n_exec=n_ex, exec_gates=g,
               offsets=offsets, pair_tok=pair_tok, pair_gate=pair_gate,
               pair_of=pair_of)
    if ns:
        out["shared_gate"] = np.ones(x.shape[0], np.float32) if sg is None else sg
    if experts is not None:
        y = moe_restricted64(x, ex, n_ex, g, experts, residual)
        for i in range(ns):
            y += (np.asarray(out["shared_gate"], np.float64)[:, None]
                  * shared["experts"].forward(i, np.asarray(x)))
        out["y"] = y
    return out


# ---------------------------------------------------------- diagnostics -----
def bruteforce_best(candidates, n, objective):
    """argmin of objective(A) over all size-n subsets A of candidates
    (ties: lexicographically first subset)."""
    best, best_val = None, None
    for A in itertools.combinations(sorted(candidates), n):
        v = objective(A)
        if best_val is None or v < best_val:
            best, best_val = A, v
    return best, best_val


def greedy_cross(candidates, n, ids, w, eo):
    """Sec. 3.3: A^cross built greedily, each step adding the expert with the
    largest reduction of the exact error."""
    A = []
    rest = sorted(candidates)
    for _ in range(n):
        vals = [(exact_error64(ids, w, eo, A + [u]), u) for u in rest]
        v, u = min(vals)
        A.append(u)
        rest.remove(u)
    return A


def crossterm_stats(a):
    """App. B for one token's omitted contributions a [m, d] (m >= 1):
    rho (eq. exact_additive_ratio), c_bar (eq. weighted_mean_cosine) and
    |U|_eff (eq. effective_omitted_count)."""
    a = np.asarray(a, np.float64)
    mag = np.linalg.norm(a, axis=1)
    exact = float(np.sum(a.sum(axis=0) ** 2))
    add = float(np.sum(mag ** 2))
    rho = exact / add
    ueff = float(mag.sum() ** 2 / add)
    m = len(a)
    num = den = 0.0
    for u in range(m):
        for v in range(m):
            if u != v:
                c = float(a[u] @ a[v]) / (mag[u] * mag[v])
                num += mag[u] * mag[v] * c
                den += mag[u] * mag[v]
    cbar = num / den if den > 0 else 0.0
    return rho, cbar, ueff


def energy_retained(D_star, A_method, n):
    """App. F eq. energy_retained with A* = top-n experts by D*."""
    order = sorted(range(len(D_star)), key=lambda u: (-D_star[u], u))
    top = sum(D_star[u] for u in order[:n])
    return float(sum(D_star[u] for u in A_method) / top) if top > 0 else 1.0
