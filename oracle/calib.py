"""TEST INFRASTRUCTURE ONLY -- offline calibration of the log-energy
predictor (paper Sec. 3.4 and App. A "Calibration Details"), in NumPy.

For every routed expert u the calibration target is the log output energy
y = log(||E_u(z)||^2 + eps) and the input is z_bar = z / ||z||.  Per expert,
streaming sufficient statistics are accumulated batch by batch (count,
first moments, Gram matrix, input-target cross-moment; App. A keeps the
Gram in fp32 and the vectors and scalars in fp64); the per-token
activations are dropped after each batch.  The fit is the centred
closed-form ridge

    a(lam) = (G_c + lam I)^-1 q_c,      b(lam) = y_mean - a(lam)^T z_mean

evaluated for 25 values of lam log-spaced over [1e-4, 1e2] from one
eigendecomposition of G_c, with lam chosen per expert by marginal
likelihood, and a bias correction for exponentiating a log-space fit folded
into b (App. A).

Readings where App. A leaves details open:
* G_c and q_c are the centred sums (X_c^T X_c, X_c^T y_c), i.e. lam weights
  ||a||^2 against the residual sum of squares;
* the marginal likelihood is the Bayesian-ridge evidence with the noise
  variance profiled out:
      log p(y | lam) = -(n/2) log(RSS + lam ||a||^2)
                       + 1/2 sum_i log(lam / (sigma_i + lam)) + const,
  sigma_i the eigenvalues of G_c; ties go to the smaller lam;
* the bias correction is the log-normal one, b += s^2 / 2 with
  s^2 = RSS(lam*) / n, which the streaming statistics determine (they
  include the scalar sum of y^2 for this purpose);
* eps = 1e-12.
"""
from __future__ import annotations

import numpy as np

from . import method

LAMBDAS = np.logspace(-4, 2, 25)
EPS = 1e-12


class ExpertStats:
    """Streaming sufficient statistics of one expert's routed pairs."""

    def __init__(self, d):
        self.n = 0
        self.sz = np.zeros(d, np.float64)       # sum z_bar
        self.sy = 0.0                           # sum y
        self.syy = 0.0                          # sum y^2
        self.G = np.zeros((d, d), np.float32)   # sum z_bar z_bar^T (fp32)
        self.q = np.zeros(d, np.float64)        # sum z_bar y

    def update(self, zb, y):
        zb = np.asarray(zb, np.float64)
        y = np.asarray(y, np.float64)
        self.n += len(y)
        self.sz += zb.sum(axis=0)
        self.sy += float(y.sum())
        self.syy += float(y @ y)
        self.G += (zb.T @ zb).astype(np.float32)
        self.q += zb.T @ y


def ridge_fit(st: ExpertStats, lambdas=LAMBDAS):
    """Closed-form centred ridge with evidence-chosen lambda.

    Returns dict(a, b, lam, b_raw, rss, evidence[list])."""
    n = st.n
    d = st.sz.shape[0]
    if n == 0:
        return dict(a=np.zeros(d), b=0.0, lam=float(lambdas[0]), b_raw=0.0,
                    rss=0.0, evidence=[])
    zm = st.sz / n
    ym = st.sy / n
    Gc = st.G.astype(np.float64) - n * np.outer(zm, zm)
    Gc = 0.5 * (Gc + Gc.T)
    qc = st.q - n * zm * ym
    yyc = st.syy - n * ym * ym
    sig, V = np.linalg.eigh(Gc)
    sig = np.maximum(sig, 0.0)
    qv = V.T @ qc
    best = None
    ev = []
    for lam in lambdas:
        av = qv / (sig + lam)
        a = V @ av
        # RSS = y_c^T y_c - 2 a^T q_c + a^T G_c a
        rss = yyc - 2.0 * float(av @ qv) + float(np.sum(sig * av * av))
        rss = max(rss, 0.0)
        quad = rss + lam * float(av @ av)
        e = -0.5 * n * np.log(max(quad, 1e-300)) + 0.5 * float(
            np.sum(np.log(lam / (sig + lam))))
        ev.append(e)
        if best is None or e > best[0]:
            best = (e, lam, a, rss)
    _, lam, a, rss = best
    b_raw = ym - float(a @ zm)
    b = b_raw + 0.5 * rss / n
    return dict(a=a, b=b, lam=float(lam), b_raw=b_raw, rss=rss, evidence=ev)


def ridge_direct(st: ExpertStats, lam):
    """The same estimate by a direct linear solve (no eigendecomposition)."""
    n = st.n
    zm = st.sz / n
    ym = st.sy / n
    Gc = st.G.astype(np.float64) - n * np.outer(zm, zm)
    qc = st.q - n * zm * ym
    a = np.linalg.solve(Gc + lam * np.eye(len(zm)), qc)
    return a, ym - float(a @ zm)


def collect_stats(z, w_router, b_router, K, experts, norm_topk=1,
                  batch=256):
    """Route calibration tokens (fp64 definition), evaluate every routed
    expert and accumulate per-expert statistics batch by batch."""
    E, d = w_router.shape
    stats = [ExpertStats(d) for _ in range(E)]
    for lo in range(0, len(z), batch):
        zb_tok = np.asarray(z[lo:lo + batch], np.float64)
        _, ids, _ = method.route64(zb_tok, w_router, b_router, K, norm_topk)
        nrm = np.linalg.norm(zb_tok, axis=1, keepdims=True)
        zbar = np.divide(zb_tok, nrm, out=np.zeros_like(zb_tok),
                         where=nrm > 0)
        for u in np.unique(ids):
            tt = np.nonzero((ids == u).any(axis=1))[0]
            out = experts.forward(int(u), zb_tok[tt])
            y = np.log(np.sum(out ** 2, axis=1) + EPS)
            stats[u].update(zbar[tt], y)
    return stats


def fit_predictor(z, w_router, b_router, K, experts, norm_topk=1,
                  batch=256):
    """Fitted predictor (A [E,d] fp32, b [E] fp32) plus per-expert info."""
    stats = collect_stats(z, w_router, b_router, K, experts, norm_topk, batch)
    E, d = w_router.shape
    A = np.zeros((E, d), np.float32)
    b = np.zeros(E, np.float32)
    info = []
    for u, st in enumerate(stats):
        f = ridge_fit(st)
        A[u] = f["a"].astype(np.float32)
        b[u] = np.float32(f["b"])
        info.append(dict(n=st.n, lam=f["lam"], rss=f["rss"]))
    return A, b, info
