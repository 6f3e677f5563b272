// Router logits and the per-token tail of the scoring path (Sec. 3.1
// router; Sec. 3.4, eq. log_energy_predictor).
//
// k_scores  the router's dot products for a batch, as a tiled batch x rows
//           product: logit l[t][e] = x_t . W_r[e] + beta_e (and, with shared
//           experts gated by a vector, gdot[t] = x_t . g).
// k_tail    one workgroup per token: top-K by exact ranks, router weights,
//           then the score of each routed pair.  For the method's own rule
//           the pair's predicted removal cost w^2 exp(q / ||x|| + b_u),
//           q = a_u . x_t, is computed here for the K routed experts only
//           (App. "Custom GPU Kernels": the token is normalised once and
//           reused across its K experts), wavefront w taking routes 2w and
//           2w + 1; the other rules need only the routes.
//
// Fixed fp32 order of every dot product of length d: partial j (0..63) owns
// the elements 256m + 4j + r (r = 0..3) and accumulates them in ascending
// element order with single-rounding FMA from +0; the 64 partials are then
// joined by the halving tree "s[j] = s[j] + s[j + h], j < h" for h = 32 ..
// 1.  Lane j of a wavefront holds partial j.  A halving-tree level is a
// lane exchange over distance h, so the tree runs on lane shuffles (see
// tree16 and wave_tree_sum: any lane holding partial j^m of the same dot at
// each level gives the same sums).
#include "common.hpp"
#include "internal.hpp"

namespace basek {

constexpr int SC_T = 4;        // tokens per wavefront tile
constexpr int SC_R = 4;        // matrix rows per wavefront tile
constexpr int SC_WT = 4;       // wavefronts of a workgroup along tokens
constexpr int SC_WR = 2;       // wavefronts of a workgroup along rows
constexpr int SC_WAVES = SC_WT * SC_WR;
constexpr int SC_TB = SC_T * SC_WT;           // tokens per workgroup
constexpr int SC_RB = SC_R * SC_WR;           // rows per workgroup
constexpr int SC_CH = 256;                    // elements per chunk
constexpr int SC_PF = 2;                      // chunks requested ahead (register stages)
static_assert(SC_T * SC_R == 16, "tree16 joins 16 dot products");
static_assert(SC_TB == TOK_GROUP, "a workgroup's tokens are one group");

// The halving trees of 16 dot products at once, v[i] holding lane j's
// partial of dot i.  At the level of distance h the 2c values still held
// are paired (i, i + c): a lane whose bit h is clear keeps dot i and sends
// dot i + c, its partner (lane j ^ h) keeps i + c and sends i, and each adds
// what it receives -- every lane then holds, for its dot, s[j] + s[j ^ h]
// of that level.  After the levels 32, 16, 8, 4 lane j holds one dot,
// number j / 4, and the levels 2 and 1 finish it in all four lanes of its
// group.
template <int C, int H>
__device__ __forceinline__ void tree_level(float (&v)[16], int lane) {
  const bool hi = (lane & H) != 0;
#pragma unroll
  for (int i = 0; i < C; ++i) {
    const float keep = hi ? v[i + C] : v[i];
    const float send = hi ? v[i] : v[i + C];
    v[i] = keep + xor_lane<H>(send);
  }
}
__device__ __forceinline__ float tree16(float (&v)[16]) {
  const int lane = lane_id();
  tree_level<8, 32>(v, lane);
  tree_level<4, 16>(v, lane);
  tree_level<2, 8>(v, lane);
  tree_level<1, 4>(v, lane);
  float s = v[0];
  s = s + xor_lane<2>(s);
  s = s + xor_lane<1>(s);
  return s;
}

// Four consecutive elements of a token row as loaded (bf16 bits or fp32),
// widened only where used, so that holding a request does not wait for it.
template <typename XT> struct Raw4;
template <> struct Raw4<uint16_t> {
  u32x2 v;
  __device__ __forceinline__ void load(const uint16_t *p) { v = *reinterpret_cast<const u32x2 *>(p); }
  __device__ __forceinline__ float at(int r) const {
    const uint32_t h = (r < 2) ? v.x : v.y;
    return __uint_as_float((r & 1) ? (h & 0xFFFF0000u) : (h << 16));
  }
};
template <> struct Raw4<float> {
  float4 v;
  __device__ __forceinline__ void load(const float *p) { v = *reinterpret_cast<const float4 *>(p); }
  __device__ __forceinline__ float at(int r) const {
    return r == 0 ? v.x : r == 1 ? v.y : r == 2 ? v.z : v.w;
  }
};

template <typename XT> struct XPiece;
// 8 bf16 elements, widened to fp32 on their way into LDS
template <> struct XPiece<uint16_t> {
  static constexpr int ELEMS = 8;
  u32x4 v;
  __device__ __forceinline__ void load(const uint16_t *p) { v = *reinterpret_cast<const u32x4 *>(p); }
  __device__ __forceinline__ void put(float *dst) const {
    *reinterpret_cast<float4 *>(dst) =
        float4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xFFFF0000u),
               __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xFFFF0000u)};
    *reinterpret_cast<float4 *>(dst + 4) =
        float4{__uint_as_float(v.z << 16), __uint_as_float(v.z & 0xFFFF0000u),
               __uint_as_float(v.w << 16), __uint_as_float(v.w & 0xFFFF0000u)};
  }
};
template <> struct XPiece<float> {
  static constexpr int ELEMS = 4;
  float4 v;
  __device__ __forceinline__ void load(const float *p) { v = *reinterpret_cast<const float4 *>(p); }
  __device__ __forceinline__ void put(float *dst) const { *reinterpret_cast<float4 *>(dst) = v; }
};

// Staging of one 256-element chunk of the workgroup's SC_TB token rows and
// SC_RB matrix rows: XP token pieces and WP row pieces (16 bytes each) per
// thread.
template <typename XT>
struct ScStage {
  static constexpr int XE = XPiece<XT>::ELEMS;
  static constexpr int XB = SC_TB * SC_CH / XE;    // token pieces
  static constexpr int WB = SC_RB * SC_CH / 4;     // row pieces
  static constexpr int XP = XB / (SC_WAVES * WAVE), WP = WB / (SC_WAVES * WAVE);
  static_assert(XB % (SC_WAVES * WAVE) == 0 && WB % (SC_WAVES * WAVE) == 0,
                "staging pieces per thread");
  XPiece<XT> xv[XP];
  float4 wv[WP];
};

// rows r < n_router: W_r (logits, + beta); with G != nullptr one more row,
// the shared experts' gate vector (gdot).  A workgroup covers one token
// group (16 tokens) x 8 rows (4 x 2 wavefronts of 4 x 4), every row group of
// token group g on die g % N_XCD (xcd_group); each 256-element chunk of its
// rows is staged once in LDS (tokens widened to fp32), the next chunk's
// loads in flight meanwhile.  Grid xcd_grid(ceil(B / 16), ceil(rows / 8)).
template <typename XT>
__global__ __launch_bounds__(SC_WAVES * WAVE, 2)
void k_scores(const XT *__restrict__ x, int B, int d,
              const float *__restrict__ Wr, const float *__restrict__ beta,
              int n_router, const float *__restrict__ G, float *__restrict__ logits,
              float *__restrict__ gdot) {
  using St = ScStage<XT>;
  constexpr int XE = St::XE;
  __shared__ __attribute__((aligned(16))) float xs[2][SC_TB][SC_CH];
  __shared__ __attribute__((aligned(16))) float wsh[2][SC_RB][SC_CH];
  const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
  const int tw = wv % SC_WT, rw = wv / SC_WT;
  const int rows = n_router + (G ? 1 : 0);
  int tg, rg;
  xcd_group(blockIdx.x, (rows + SC_RB - 1) / SC_RB, tg, rg);
  if (tg * SC_TB >= B) return;
  const int tb0 = tg * SC_TB, rb0 = rg * SC_RB;

  // the thread's staging pieces: token row / matrix row and column
  const XT *xsrc[St::XP];
  const float *wsrc[St::WP];
  int xt[St::XP], xc[St::XP], wr[St::WP], wc[St::WP];
#pragma unroll
  for (int i = 0; i < St::XP; ++i) {
    const int c = tid + i * SC_WAVES * WAVE;
    xt[i] = c / (SC_CH / XE);
    xc[i] = (c % (SC_CH / XE)) * XE;
    xsrc[i] = x + (size_t)min(tb0 + xt[i], B - 1) * d + xc[i];
  }
#pragma unroll
  for (int i = 0; i < St::WP; ++i) {
    const int c = tid + i * SC_WAVES * WAVE;
    wr[i] = c / (SC_CH / 4);
    wc[i] = (c % (SC_CH / 4)) * 4;
    const int r = min(rb0 + wr[i], rows - 1);
    wsrc[i] = (r < n_router ? Wr + (size_t)r * d : G) + wc[i];
  }
  St st[SC_PF];
  auto fetch = [&](St &sg, int m) {
#pragma unroll
    for (int i = 0; i < St::XP; ++i) sg.xv[i].load(xsrc[i] + m);
#pragma unroll
    for (int i = 0; i < St::WP; ++i) sg.wv[i] = *reinterpret_cast<const float4 *>(wsrc[i] + m);
  };
  auto put = [&](const St &sg, int b) {
#pragma unroll
    for (int i = 0; i < St::XP; ++i) sg.xv[i].put(&xs[b][xt[i]][xc[i]]);
#pragma unroll
    for (int i = 0; i < St::WP; ++i) *reinterpret_cast<float4 *>(&wsh[b][wr[i]][wc[i]]) = sg.wv[i];
  };

  float acc[SC_T * SC_R];
#pragma unroll
  for (int i = 0; i < SC_T * SC_R; ++i) acc[i] = 0.0f;
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
        float4 xv[SC_T], wv4[SC_R];
#pragma unroll
        for (int a = 0; a < SC_T; ++a)
          xv[a] = *reinterpret_cast<const float4 *>(&xs[buf][tw * SC_T + a][4 * lane]);
#pragma unroll
        for (int b = 0; b < SC_R; ++b)
          wv4[b] = *reinterpret_cast<const float4 *>(&wsh[buf][rw * SC_R + b][4 * lane]);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
#pragma unroll
          for (int a = 0; a < SC_T; ++a) {
            const float xe = r == 0 ? xv[a].x : r == 1 ? xv[a].y : r == 2 ? xv[a].z : xv[a].w;
#pragma unroll
            for (int b = 0; b < SC_R; ++b) {
              const float we = r == 0 ? wv4[b].x : r == 1 ? wv4[b].y : r == 2 ? wv4[b].z : wv4[b].w;
              acc[a * SC_R + b] = __builtin_fmaf(xe, we, acc[a * SC_R + b]);
            }
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

  // dot i of the tile (token a = i / SC_R, row b = i % SC_R) ends in the
  // lanes 4i .. 4i + 3
  const float v = tree16(acc);
  const int i = lane >> 2;
  const int t = tb0 + tw * SC_T + i / SC_R, r = rb0 + rw * SC_R + i % SC_R;
  if ((lane & 3) == 0 && t < B && r < rows) {
    if (r < n_router)
      logits[(size_t)t * n_router + r] = beta ? v + beta[r] : v;
    else
      gdot[t] = v;
  }
}

constexpr int TL_NI = MAX_E / WAVE;
constexpr int TL_RANK = 256;                  // lanes that rank the logits
constexpr int TL_MAXW = (MAX_K + 1) / 2 > TL_RANK / WAVE ? (MAX_K + 1) / 2 : TL_RANK / WAVE;

// Wavefronts of a k_tail workgroup: the TL_RANK ranking lanes, and with the
// method's predictor one wavefront per two routes.
__host__ __device__ inline int tail_waves(int K, bool pred) {
  const int wp = pred ? (K + 1) / 2 : 0;
  return wp > TL_RANK / WAVE ? wp : TL_RANK / WAVE;
}

// mode bit 0: route (top-K and weights from the logits into ids / w)
// mode bit 1: per-pair scores of the routed pairs (ids / w, read back when
//             bit 0 is off) under `rule`: SCORE_BASE w^2 exp(q / ||x|| + b_u)
//             with q = a_u . x_t and ||x_t||^2 computed here in the fixed
//             order; SCORE_TOP1 1 for the first route, else 0; SCORE_WEIGHT
//             w; SCORE_WEIGHT_SQ w * w; SCORE_STATIC (w * w) * exp(b_u)
// One workgroup of tail_waves(K, pred) wavefronts per token, token group g on
// die g % N_XCD as in k_scores (xcd_group).  Top-K in the
// order (logit desc, index asc) of rank_key: the token's keys go to LDS and
// the first TL_RANK lanes count, for every expert, the keys that rank before
// its own -- lane g counts for expert g % E2 over stretch g / E2 of the C
// equal stretches of the keys (E2 the power of two >= E, C = min(TL_RANK /
// E2, E2)); route k is the expert of rank k.  Every wavefront then takes the
// routes and weights from LDS; wavefront w computes the predictor of routes
// 2w and 2w + 1.
template <typename XT>
__global__ __launch_bounds__(TL_MAXW * WAVE)
void k_tail(int B, int E, int K, int d, int norm_topk, const float *__restrict__ logits,
            const XT *__restrict__ x, const float *__restrict__ A,
            const float *__restrict__ bp, int32_t *__restrict__ ids_io,
            float *__restrict__ w_io, float *__restrict__ cost, int mode, int rule,
            uint8_t *__restrict__ order, float *__restrict__ ex, float *__restrict__ den) {
  __shared__ __attribute__((aligned(16))) uint64_t keys[MAX_E];
  __shared__ float lrow[MAX_E];
  __shared__ int part[TL_RANK];
  __shared__ int route[MAX_K];
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id_u();
  int tg, ti;
  xcd_group(blockIdx.x, TOK_GROUP, tg, ti);
  const int t = tg * TOK_GROUP + ti;   // on the die that wrote its logits
  if (t >= B) return;
  const bool pred = (mode & 2) && rule == SCORE_BASE;
  // the logits row (clamped, no branches, so that the loads are in flight
  // together); the method's predictor's first pass of the token row is
  // requested once the routing's inputs have arrived (it does not depend on
  // the routing, which then runs while it is in flight)
  float lv[TL_NI];
  if ((mode & 1) && w == 0) {
#pragma unroll
    for (int i = 0; i < TL_NI; ++i) lv[i] = logits[(size_t)t * E + min(lane + WAVE * i, E - 1)];
  }
  constexpr int GC = 8;   // chunks of 256 elements per pass, loads issued together
  const XT *xr = x + (size_t)t * d + 4 * lane;
  Raw4<XT> xv[GC];
  auto prefetch_x = [&]() {
    if (pred && 2 * w < K) {
#pragma unroll
      for (int c = 0; c < GC; ++c) xv[c].load(xr + min(c * 256, d - 256));
    }
  };

  int my_id = 0;       // lane k < K: routed expert k
  float my_w = 0.0f;   // and its weight
  if (!(mode & 1)) {
    my_id = ids_io[(size_t)t * K + min(lane, K - 1)];
    my_w = w_io[(size_t)t * K + min(lane, K - 1)];
    prefetch_x();
  } else {
    int E2 = 1;
    while (E2 < E) E2 <<= 1;
    if (w == 0) {
#pragma unroll
      for (int i = 0; i < TL_NI; ++i) {
        const int e = lane + WAVE * i;
        if (e < E2) {
          keys[e] = e < E ? rank_key(lv[i], e) : 0;   // 0 ranks after every expert
          lrow[e] = lv[i];
        }
      }
    }
    prefetch_x();
    __syncthreads();
    const int C = min(TL_RANK / E2, E2), len = E2 / C;
    if (tid < C * E2) {
      const int i = tid & (E2 - 1), j0 = (tid / E2) * len;
      const uint64_t ku = keys[i];
      int r = 0;
      if (len < 16) {
        for (int j = j0; j < j0 + len; ++j) r += keys[j] > ku;
      } else {
        // 16 keys per step, their LDS reads issued together
        for (int j = j0; j < j0 + len; j += 16) {
          u32x4 o[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) o[q] = *reinterpret_cast<const u32x4 *>(&keys[j + 2 * q]);
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            r += (((uint64_t)o[q].y << 32 | o[q].x) > ku);
            r += (((uint64_t)o[q].w << 32 | o[q].z) > ku);
          }
        }
      }
      part[tid] = r;
    }
    __syncthreads();
    int my_rank = 0;   // thread tid < E: the rank of expert tid
    if (tid < E) {
      for (int c = 0; c < C; ++c) my_rank += part[c * E2 + tid];
      if (my_rank < K) route[my_rank] = tid;
    }
    __syncthreads();
    my_id = route[min(lane, K - 1)];
    const float lmax = lrow[route[0]];
    const float eps = base_exp(lrow[my_id] - lmax);
    float S;
    if (norm_topk) {
      S = 0.0f;
      for (int k = 0; k < K; ++k)
        S = S + __builtin_bit_cast(float, __builtin_amdgcn_readlane(__float_as_int(eps), k));
    } else {
      float pt = 0.0f;
#pragma unroll
      for (int i = 0; i < TL_NI; ++i)
        if (lane + WAVE * i < E) pt = pt + base_exp(lrow[lane + WAVE * i] - lmax);
      S = wave_tree_sum(pt);
    }
    my_w = eps / S;
    if (w == 0 && lane < K) {
      ids_io[(size_t)t * K + lane] = my_id;
      w_io[(size_t)t * K + lane] = my_w;
    }
    if (order) {
      // for the fused layer's backfill: the experts in rank order, their
      // exp(l - l_max) in rank order, and the router's denominator S
      if (tid < E) {
        order[(size_t)t * E + my_rank] = (uint8_t)tid;
        ex[(size_t)t * E + my_rank] = base_exp(lrow[tid] - lmax);
      }
      if (tid == 0) den[t] = S;
    }
  }
  if (!(mode & 2)) return;

  const int u = (lane < K && my_id >= 0 && my_id < E) ? my_id : 0;   // out-of-range ids read row 0
  if (!pred) {
    if (w == 0 && lane < K) {
      float c;
      if (rule == SCORE_TOP1) {
        c = lane == 0 ? 1.0f : 0.0f;
      } else if (rule == SCORE_WEIGHT) {
        c = my_w;
      } else if (rule == SCORE_WEIGHT_SQ) {
        c = my_w * my_w;
      } else {   // SCORE_STATIC
        const float w2 = my_w * my_w;
        c = w2 * base_exp(bp[u]);
      }
      cost[(size_t)t * K + lane] = c;
    }
    return;
  }

  // this wavefront's routes k0 = 2w, k1 = 2w + 1: ||x_t||^2, q0, q1 in the
  // fixed order
  const int k0 = 2 * w, k1 = 2 * w + 1;
  if (k0 >= K) return;
  const bool has1 = k1 < K;
  const int u0 = __builtin_amdgcn_readlane(u, k0);
  const int u1 = __builtin_amdgcn_readlane(u, has1 ? k1 : k0);
  const float b_my = (lane == k0 || lane == k1) ? bp[u] : 0.0f;
  const float *a0 = A + (size_t)u0 * d + 4 * lane;
  const float *a1 = A + (size_t)u1 * d + 4 * lane;
  float ss = 0.0f, q0 = 0.0f, q1 = 0.0f;
  for (int m0 = 0; m0 < d; m0 += GC * 256) {
    float av0[GC][4], av1[GC][4];
#pragma unroll
    for (int c = 0; c < GC; ++c) {
      const int m = min(m0 + c * 256, d - 256);
      if (m0 > 0) xv[c].load(xr + m);
      load4(a0 + m, av0[c]);
      if (has1) load4(a1 + m, av1[c]);
    }
#pragma unroll
    for (int c = 0; c < GC; ++c) {
      if (m0 + c * 256 < d) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float xe = xv[c].at(r);
          ss = __builtin_fmaf(xe, xe, ss);
          q0 = __builtin_fmaf(xe, av0[c][r], q0);
          if (has1) q1 = __builtin_fmaf(xe, av1[c][r], q1);
        }
      }
    }
  }
  ss = wave_tree_sum(ss);
  q0 = wave_tree_sum(q0);
  if (has1) q1 = wave_tree_sum(q1);
  float inv = 0.0f;
  if (ss > 0.0f) {
    const float rt = sqrtf(ss);
    inv = 1.0f / rt;
  }
  if (lane == k0 || (has1 && lane == k1)) {
    float s = (lane == k0 ? q0 : q1) * inv;
    s = s + b_my;
    const float w2 = my_w * my_w;
    cost[(size_t)t * K + lane] = w2 * base_exp(s);
  }
}

template <typename XT>
static void launch_scores_t(const XT *x, int B, int d, const float *Wr, const float *beta,
                            int n_router, const float *G, float *logits, float *gdot,
                            hipStream_t st) {
  const int rows = n_router + (G ? 1 : 0);
  const dim3 grid(xcd_grid((B + SC_TB - 1) / SC_TB, (rows + SC_RB - 1) / SC_RB));
  launch_k(k_scores<XT>, grid, dim3(SC_WAVES * WAVE), 0, st, x, B, d, Wr, beta, n_router, G,
           logits, gdot);
}

hipError_t launch_scores(bool bf16, const void *x, int B, int d, const float *Wr,
                         const float *beta, int n_router, const float *G, float *logits,
                         float *gdot, hipStream_t st) {
  if (bf16)
    launch_scores_t((const uint16_t *)x, B, d, Wr, beta, n_router, G, logits, gdot, st);
  else
    launch_scores_t((const float *)x, B, d, Wr, beta, n_router, G, logits, gdot, st);
  return hipGetLastError();
}

hipError_t launch_tail(bool bf16, int B, int E, int K, int d, int norm_topk,
                       const float *logits, const void *x, const float *A, const float *bp,
                       int32_t *ids, float *w, float *cost, int mode, int rule,
                       hipStream_t st, uint8_t *order, float *ex, float *den) {
  const dim3 block(tail_waves(K, (mode & 2) && rule == SCORE_BASE) * WAVE);
  const dim3 grid(xcd_grid((B + TOK_GROUP - 1) / TOK_GROUP, TOK_GROUP));
  if (bf16)
    launch_k(k_tail<uint16_t>, grid, block, 0, st, B, E, K, d, norm_topk, logits,
             (const uint16_t *)x, A, bp, ids, w, cost, mode, rule, order, ex, den);
  else
    launch_k(k_tail<float>, grid, block, 0, st, B, E, K, d, norm_topk, logits,
             (const float *)x, A, bp, ids, w, cost, mode, rule, order, ex, den);
  return hipGetLastError();
}

}  // namespace basek
