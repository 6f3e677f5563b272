// Router logits, predictor dot products and the per-token tail of the
// scoring path (Sec. 3.1 router; Sec. 3.4, eq. log_energy_predictor).
//
// k_scores  every dot product the scoring path needs for a batch, as a tiled
//           batch x rows product: rows are the router matrix (logit
//           l[t][e] = x_t . W_r[e] + beta_e) and the predictor matrix
//           (q[t][e] = x_t . a_e, for every expert: the dense product costs
//           about as much as the router and does not wait for top-K), plus
//           ||x_t||^2.
// k_tail    one wavefront per token: top-K by exact ranks, router weights,
//           then the cost of each routed pair, cost = w^2 exp(q[t][u] /
//           ||x_t|| + b_u), one lane per pair (or another selection rule's
//           per-pair score: App. selection-rule ablation).
//
// Fixed fp32 order of every dot product of length d: partial j (0..63) owns
// the elements 256m + 4j + r (r = 0..3) and accumulates them in ascending
// element order with single-rounding FMA from +0; the 64 partials are then
// joined by the halving tree "s[j] = s[j] + s[j + h], j < h" for h = 32 ..
// 1.  Here lane j of a wavefront holds partial j of up to 72 dot products at
// once; the trees run through LDS (a transpose), one dot product per lane.
// The operands of a workgroup's 16 x 16 tile pass through LDS chunk by
// chunk, so each is read from L2 once per workgroup.
#include "common.hpp"
#include "internal.hpp"

namespace basek {

constexpr int SC_T = 8;        // tokens per wavefront tile
constexpr int SC_R = 4;        // matrix rows per wavefront tile
constexpr int SC_WT = 2;       // wavefronts of a workgroup along tokens
constexpr int SC_WR = 4;       // wavefronts of a workgroup along rows
constexpr int SC_WAVES = SC_WT * SC_WR;
constexpr int SC_TB = SC_T * SC_WT;           // tokens per workgroup
constexpr int SC_RB = SC_R * SC_WR;           // rows per workgroup
constexpr int SC_CH = 256;                    // elements per chunk
constexpr int SC_PF = 2;                      // chunks requested ahead (register stages)
constexpr int SC_DOTS = SC_T * SC_R + SC_T;   // + ||x||^2 of the tile's tokens
constexpr int SC_PAD = WAVE + 1;              // LDS row of one dot's partials

// The halving tree over 64 values held by one lane.
__device__ __forceinline__ float tree64(float (&s)[WAVE]) {
#pragma unroll
  for (int h = WAVE / 2; h >= 1; h >>= 1)
#pragma unroll
    for (int j = 0; j < h; ++j) s[j] = s[j] + s[j + h];
  return s[0];
}

// Lane i: the tree of row i of P (64 partials of one dot product).
__device__ __forceinline__ float lds_tree(const float *P, int i) {
  float s[WAVE];
#pragma unroll
  for (int j = 0; j < WAVE; ++j) s[j] = P[i * SC_PAD + j];
  return tree64(s);
}

template <typename XT> struct XChunk;
template <> struct XChunk<uint16_t> {
  u32x2 v;
  __device__ __forceinline__ void load(const uint16_t *p) { v = *reinterpret_cast<const u32x2 *>(p); }
  __device__ __forceinline__ float at(int r) const {
    const uint32_t w = (r < 2) ? v.x : v.y;
    return __uint_as_float((r & 1) ? (w & 0xFFFF0000u) : (w << 16));
  }
};
template <> struct XChunk<float> {
  float4 v;
  __device__ __forceinline__ void load(const float *p) { v = *reinterpret_cast<const float4 *>(p); }
  __device__ __forceinline__ float at(int r) const {
    return r == 0 ? v.x : r == 1 ? v.y : r == 2 ? v.z : v.w;
  }
};

// Staging of one 256-element chunk of the workgroup's SC_TB token rows and
// SC_RB matrix rows: 16-byte pieces, XP of them for the tokens and WP for
// the rows per thread.
template <typename XT>
struct ScStage {
  static constexpr int XB = SC_TB * SC_CH * (int)sizeof(XT) / 16;   // x pieces
  static constexpr int WB = SC_RB * SC_CH * 4 / 16;                  // row pieces
  static constexpr int XP = XB / (SC_WAVES * WAVE), WP = WB / (SC_WAVES * WAVE);
  static constexpr int XS = SC_CH * (int)sizeof(XT) / 16;            // pieces per token row
  static constexpr int WS = SC_CH * 4 / 16;                          // pieces per matrix row
  static_assert(XB % (SC_WAVES * WAVE) == 0 && WB % (SC_WAVES * WAVE) == 0,
                "staging pieces per thread");
  u32x4 xv[XP], wv[WP];
};

// The workgroup's LDS: two chunk buffers while streaming, then the
// wavefronts' partials for the trees.
template <typename XT>
union ScLds {
  struct {
    u32x4 x[2][ScStage<XT>::XB];
    u32x4 w[2][ScStage<XT>::WB];
  } ch;
  float P[SC_WAVES][SC_DOTS * SC_PAD];
};

// rows r < n_router: W_r (logits, + beta); n_router <= r < n_router + n_pred:
// the predictor matrix A (q); with G != nullptr one more row, the shared
// experts' gate vector (gdot).  With ss != nullptr the wavefronts of row
// tile 0 also produce ||x_t||^2.  A workgroup covers 16 tokens x 16 rows
// (2 x 4 wavefronts of 8 x 4); each 256-element chunk of its rows is staged
// once in LDS, the next chunk's loads in flight meanwhile.  Grid
// (ceil(B / 16), ceil(rows / 16)).
template <typename XT>
__global__ __launch_bounds__(SC_WAVES * WAVE, 2)
void k_scores(const XT *__restrict__ x, int B, int d,
              const float *__restrict__ Wr, const float *__restrict__ beta,
              int n_router, const float *__restrict__ A, int n_pred,
              const float *__restrict__ G, float *__restrict__ logits,
              float *__restrict__ q, float *__restrict__ gdot,
              float *__restrict__ ss) {
  using St = ScStage<XT>;
  __shared__ ScLds<XT> lds;
  const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
  const int tw = wv % SC_WT, rw = wv / SC_WT;
  const int rows = n_router + n_pred + (G ? 1 : 0);
  const int tb0 = blockIdx.x * SC_TB, rb0 = blockIdx.y * SC_RB;
  const bool do_ss = ss != nullptr && rb0 == 0 && rw == 0;

  // the thread's staging pieces: token row / matrix row and 16-byte column
  const XT *xsrc[St::XP];
  const float *wsrc[St::WP];
#pragma unroll
  for (int i = 0; i < St::XP; ++i) {
    const int c = tid + i * SC_WAVES * WAVE;
    xsrc[i] = x + (size_t)min(tb0 + c / St::XS, B - 1) * d + (c % St::XS) * (16 / sizeof(XT));
  }
#pragma unroll
  for (int i = 0; i < St::WP; ++i) {
    const int c = tid + i * SC_WAVES * WAVE;
    const int r = min(rb0 + c / St::WS, rows - 1);
    wsrc[i] = (r < n_router            ? Wr + (size_t)r * d
               : r < n_router + n_pred ? A + (size_t)(r - n_router) * d
                                       : G) +
              (c % St::WS) * 4;
  }
  St st[SC_PF];
  auto fetch = [&](St &sg, int m) {
#pragma unroll
    for (int i = 0; i < St::XP; ++i) sg.xv[i] = *reinterpret_cast<const u32x4 *>(xsrc[i] + m);
#pragma unroll
    for (int i = 0; i < St::WP; ++i) sg.wv[i] = *reinterpret_cast<const u32x4 *>(wsrc[i] + m);
  };
  auto put = [&](const St &sg, int b) {
#pragma unroll
    for (int i = 0; i < St::XP; ++i) lds.ch.x[b][tid + i * SC_WAVES * WAVE] = sg.xv[i];
#pragma unroll
    for (int i = 0; i < St::WP; ++i) lds.ch.w[b][tid + i * SC_WAVES * WAVE] = sg.wv[i];
  };

  float acc[SC_T][SC_R], sacc[SC_T];
#pragma unroll
  for (int a = 0; a < SC_T; ++a) {
    sacc[a] = 0.0f;
#pragma unroll
    for (int b = 0; b < SC_R; ++b) acc[a][b] = 0.0f;
  }
  const int nch = d / SC_CH;
  // register stage q holds the chunks m = q (mod SC_PF); chunk m + 1 goes
  // to LDS while chunk m is used, chunk m + SC_PF is requested meanwhile
#pragma unroll
  for (int q = 0; q < SC_PF; ++q) {
    if (q < nch) fetch(st[q], q * SC_CH);
    __builtin_amdgcn_sched_barrier(0);
  }
  put(st[0], 0);
  lds_barrier();
  for (int m0 = 0; m0 < nch; m0 += SC_PF) {
#pragma unroll
    for (int q = 0; q < SC_PF; ++q) {
      const int m = m0 + q;
      if (m < nch) {
        const int buf = m & 1;
        // this lane's elements 4 lane .. 4 lane + 3 of the chunk
        const XT *xl = reinterpret_cast<const XT *>(lds.ch.x[buf]) + 4 * lane;
        const float *wl = reinterpret_cast<const float *>(lds.ch.w[buf]) + 4 * lane;
        XChunk<XT> xc[SC_T];
        float4 wc[SC_R];
#pragma unroll
        for (int a = 0; a < SC_T; ++a) xc[a].load(xl + (tw * SC_T + a) * SC_CH);
#pragma unroll
        for (int b = 0; b < SC_R; ++b)
          wc[b] = *reinterpret_cast<const float4 *>(wl + (rw * SC_R + b) * SC_CH);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
#pragma unroll
          for (int a = 0; a < SC_T; ++a) {
            const float xv = xc[a].at(r);
#pragma unroll
            for (int b = 0; b < SC_R; ++b) {
              const float4 w4 = wc[b];
              const float wv4 = r == 0 ? w4.x : r == 1 ? w4.y : r == 2 ? w4.z : w4.w;
              acc[a][b] = __builtin_fmaf(xv, wv4, acc[a][b]);
            }
            if (do_ss) sacc[a] = __builtin_fmaf(xv, xv, sacc[a]);
          }
        }
        if (m + 1 < nch) {
          // buffer buf ^ 1 was last read for chunk m - 1, before the
          // previous barrier
          put(st[(q + 1) % SC_PF], buf ^ 1);
          lds_barrier();
        }
        __builtin_amdgcn_sched_barrier(0);
        if (m + SC_PF < nch) fetch(st[q], (m + SC_PF) * SC_CH);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  __syncthreads();          // the chunk buffers become the partials

  float *Pw = lds.P[wv];
#pragma unroll
  for (int a = 0; a < SC_T; ++a) {
#pragma unroll
    for (int b = 0; b < SC_R; ++b) Pw[(a * SC_R + b) * SC_PAD + lane] = acc[a][b];
    Pw[(SC_T * SC_R + a) * SC_PAD + lane] = sacc[a];
  }
  __syncthreads();
  if (lane < SC_T * SC_R) {
    const float v = lds_tree(Pw, lane);          // dot product `lane` of the tile
    const int t = tb0 + tw * SC_T + lane / SC_R, r = rb0 + rw * SC_R + lane % SC_R;
    if (t < B && r < rows) {
      if (r < n_router)
        logits[(size_t)t * n_router + r] = beta ? v + beta[r] : v;
      else if (r < n_router + n_pred)
        q[(size_t)t * n_pred + (r - n_router)] = v;
      else
        gdot[t] = v;
    }
  }
  if (do_ss && lane < SC_T) {
    const float v = lds_tree(Pw, SC_T * SC_R + lane);
    const int t = tb0 + tw * SC_T + lane;
    if (t < B) ss[t] = v;
  }
}

constexpr int TL_WAVES = 1;    // tokens (wavefronts) per workgroup
constexpr int TL_NI = MAX_E / WAVE;

// mode bit 0: route (top-K and weights from the logits into ids / w)
// mode bit 1: per-pair scores of the routed pairs (ids / w, read back when
//             bit 0 is off) under `rule`: SCORE_BASE w^2 exp(q / ||x|| + b_u)
//             from q and ss; SCORE_TOP1 1 for the first route, else 0;
//             SCORE_WEIGHT w; SCORE_WEIGHT_SQ w * w; SCORE_STATIC
//             (w * w) * exp(b_u)
// One wavefront per token.  Every global load is issued first, with clamped
// indices: the token's logits, its whole predictor row q[t][*], b and ||x||^2
// (the routed experts are not known yet, so a pair's q and b are then read
// from LDS rather than from memory); the kernel waits on memory once.
__global__ __launch_bounds__(TL_WAVES * WAVE)
void k_tail(int B, int E, int K, int norm_topk, const float *__restrict__ logits,
            const float *__restrict__ q, const float *__restrict__ ss,
            const float *__restrict__ bp, int32_t *__restrict__ ids_io,
            float *__restrict__ w_io, float *__restrict__ cost, int mode, int rule) {
  __shared__ float lrow[TL_WAVES][MAX_E];
  __shared__ float qrow[TL_WAVES][MAX_E];
  __shared__ float brow[TL_WAVES][MAX_E];
  __shared__ float eps_s[TL_WAVES][MAX_K];
  const int lane = lane_id(), wv = wave_id();
  const int t = blockIdx.x * TL_WAVES + wv;
  const int tc = min(t, B - 1);            // every wavefront takes part in the barriers
  const bool live = t < B;
  const bool need_q = (mode & 2) && rule == SCORE_BASE;
  const bool need_b = (mode & 2) && (rule == SCORE_BASE || rule == SCORE_STATIC);

  float lv[TL_NI], qv[TL_NI], bv[TL_NI];
#pragma unroll
  for (int i = 0; i < TL_NI; ++i) {
    const int ec = min(lane + WAVE * i, E - 1);
    lv[i] = (mode & 1) ? logits[(size_t)tc * E + ec] : 0.0f;
    qv[i] = need_q ? q[(size_t)tc * E + ec] : 0.0f;
    bv[i] = need_b ? bp[ec] : 0.0f;
  }
  const float s2 = need_q ? ss[tc] : 0.0f;
  int my_id = 0;       // lane k < K: routed expert k
  float my_w = 0.0f;   // and its weight
  if (!(mode & 1)) {
    my_id = ids_io[(size_t)tc * K + min(lane, K - 1)];
    my_w = w_io[(size_t)tc * K + min(lane, K - 1)];
  }
#pragma unroll
  for (int i = 0; i < TL_NI; ++i) {
    const int e = lane + WAVE * i;
    if (e < E) {
      lrow[wv][e] = lv[i];
      qrow[wv][e] = qv[i];
      brow[wv][e] = bv[i];
    }
  }

  if (mode & 1) {
    uint64_t kv[TL_NI];
#pragma unroll
    for (int i = 0; i < TL_NI; ++i) {
      const int e = lane + WAVE * i;
      kv[i] = (e < E) ? rank_key(lv[i], e) : 0;    // 0 ranks after every expert
    }
    // the top K in the order (logit desc, index asc): K successive wave
    // maxima of the keys, each winner removed by the lane holding it (keys
    // are distinct); lane k keeps route k
    int top0 = 0;
    for (int k = 0; k < K; ++k) {
      uint64_t best = 0;
#pragma unroll
      for (int i = 0; i < TL_NI; ++i) best = kv[i] > best ? kv[i] : best;
      const uint64_t win = wave_max_key(best);
      const int e = (int)(0xFFFFFFFFu - (uint32_t)win);
      if (k == 0) top0 = e;
      if (lane == k) my_id = e;
#pragma unroll
      for (int i = 0; i < TL_NI; ++i)
        if (kv[i] == win) kv[i] = 0;
    }
    __syncthreads();
    const float lmax = lrow[wv][top0];
    if (lane < K) eps_s[wv][lane] = base_exp(lrow[wv][my_id] - lmax);
    __syncthreads();
    float S;
    if (norm_topk) {
      S = 0.0f;
      for (int k = 0; k < K; ++k) S = S + eps_s[wv][k];
    } else {
      float part = 0.0f;
#pragma unroll
      for (int i = 0; i < TL_NI; ++i) {
        const int e = lane + WAVE * i;
        if (e < E) part = part + base_exp(lv[i] - lmax);
      }
      S = wave_tree_sum(part);
    }
    if (lane < K) {
      my_w = eps_s[wv][lane] / S;
      if (live) {
        ids_io[(size_t)t * K + lane] = my_id;
        w_io[(size_t)t * K + lane] = my_w;
      }
    }
  } else {
    __syncthreads();   // the rows written above
  }

  if ((mode & 2) && live && lane < K) {
    const int u = (my_id >= 0 && my_id < E) ? my_id : 0;   // out-of-range ids read row 0
    float c;
    if (rule == SCORE_BASE) {
      float inv = 0.0f;
      if (s2 > 0.0f) {
        const float rt = sqrtf(s2);
        inv = 1.0f / rt;
      }
      float s = qrow[wv][u] * inv;
      s = s + brow[wv][u];
      const float w2 = my_w * my_w;
      c = w2 * base_exp(s);
    } else if (rule == SCORE_TOP1) {
      c = lane == 0 ? 1.0f : 0.0f;
    } else if (rule == SCORE_WEIGHT) {
      c = my_w;
    } else if (rule == SCORE_WEIGHT_SQ) {
      c = my_w * my_w;
    } else {   // SCORE_STATIC
      const float w2 = my_w * my_w;
      c = w2 * base_exp(brow[wv][u]);
    }
    cost[(size_t)t * K + lane] = c;
  }
}

template <typename XT>
static void launch_scores_t(const XT *x, int B, int d, const float *Wr,
                            const float *beta, int n_router, const float *A,
                            int n_pred, const float *G, float *logits, float *q,
                            float *gdot, float *ss, hipStream_t st) {
  const int rows = n_router + n_pred + (G ? 1 : 0);
  dim3 grid((B + SC_TB - 1) / SC_TB, (rows + SC_RB - 1) / SC_RB);
  launch_k(k_scores<XT>, grid, dim3(SC_WAVES * WAVE), 0, st, x, B, d,
                     Wr, beta, n_router, A, n_pred, G, logits, q, gdot, ss);
}

hipError_t launch_scores(bool bf16, const void *x, int B, int d, const float *Wr,
                         const float *beta, int n_router, const float *A,
                         int n_pred, const float *G, float *logits, float *q,
                         float *gdot, float *ss, hipStream_t st) {
  if (bf16)
    launch_scores_t((const uint16_t *)x, B, d, Wr, beta, n_router, A, n_pred,
                    G, logits, q, gdot, ss, st);
  else
    launch_scores_t((const float *)x, B, d, Wr, beta, n_router, A, n_pred,
                    G, logits, q, gdot, ss, st);
  return hipGetLastError();
}

hipError_t launch_tail(int B, int E, int K, int norm_topk, const float *logits,
                       const float *q, const float *ss, const float *bp,
                       int32_t *ids, float *w, float *cost, int mode, int rule,
                       hipStream_t st) {
  launch_k(k_tail, dim3((B + TL_WAVES - 1) / TL_WAVES),
                     dim3(TL_WAVES * WAVE), 0, st, B, E, K, norm_topk, logits,
                     q, ss, bp, ids, w, cost, mode, rule);
  return hipGetLastError();
}

}  // namespace basek
