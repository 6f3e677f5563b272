// Router and removal-cost predictor (K1).
//
// k_route_logits : l[t][e] = dot(x_t, W_r[e]) + beta_e for a tile of tokens
//                  and experts.  Router of Sec. 3.1.
// k_token        : one wavefront per token.  Top-K over the token's logits
//                  and the router weights (Sec. 3.1), then the predicted
//                  removal cost of each routed pair,
//                  cost = w^2 exp(a_u . x/||x|| + b_u)   (Sec. 3.4, eq.
//                  log_energy_predictor; App. "Custom GPU Kernels": the
//                  token is normalised once and reused across its K
//                  experts).
//
// Every dot product of length d uses one fixed order: lane j of a wavefront
// owns elements 256m + 4j + r (r = 0..3), accumulates them in ascending
// element order with single-rounding FMA from +0, and the 64 lane partials
// are joined by the halving tree (wave_tree_sum).  The same order is used
// for the router, for ||x||^2 and for a_u . x, so every fp32 value here is
// reproducible bit for bit.
#include "common.hpp"
#include "internal.hpp"

namespace basek {

constexpr int RT_TOK = 2;      // tokens per wavefront tile
constexpr int RT_EXP = 4;      // experts per wavefront tile
constexpr int RT_WAVES = 4;    // wavefronts per workgroup (expert direction)

template <typename XT>
__global__ __launch_bounds__(RT_WAVES * WAVE)
void k_route_logits(const XT *__restrict__ x, int B, int d,
                    const float *__restrict__ W, const float *__restrict__ beta,
                    int E, float *__restrict__ logits) {
  const int lane = lane_id();
  const int t0 = blockIdx.x * RT_TOK;
  const int e0 = (blockIdx.y * RT_WAVES + wave_id()) * RT_EXP;
  if (e0 >= E) return;   // whole wavefront leaves together
  float acc[RT_TOK][RT_EXP];
#pragma unroll
  for (int a = 0; a < RT_TOK; ++a)
#pragma unroll
    for (int b = 0; b < RT_EXP; ++b) acc[a][b] = 0.0f;

  const XT *xr[RT_TOK];
  bool tv[RT_TOK];
#pragma unroll
  for (int a = 0; a < RT_TOK; ++a) {
    tv[a] = (t0 + a) < B;
    xr[a] = x + (size_t)(tv[a] ? t0 + a : 0) * d;
  }
  const float *wr[RT_EXP];
  bool ev[RT_EXP];
#pragma unroll
  for (int b = 0; b < RT_EXP; ++b) {
    ev[b] = (e0 + b) < E;
    wr[b] = W + (size_t)(ev[b] ? e0 + b : 0) * d;
  }

  for (int m = 0; m < d; m += 256) {
    const int k = m + 4 * lane;
    float xv[RT_TOK][4], wv[RT_EXP][4];
#pragma unroll
    for (int a = 0; a < RT_TOK; ++a) load4(xr[a] + k, xv[a]);
#pragma unroll
    for (int b = 0; b < RT_EXP; ++b) load4(wr[b] + k, wv[b]);
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int a = 0; a < RT_TOK; ++a)
#pragma unroll
        for (int b = 0; b < RT_EXP; ++b)
          acc[a][b] = __builtin_fmaf(xv[a][r], wv[b][r], acc[a][b]);
  }
#pragma unroll
  for (int a = 0; a < RT_TOK; ++a)
#pragma unroll
    for (int b = 0; b < RT_EXP; ++b) {
      float v = wave_tree_sum(acc[a][b]);
      if (lane == 0 && tv[a] && ev[b]) {
        if (beta) v = v + beta[e0 + b];
        logits[(size_t)(t0 + a) * E + e0 + b] = v;
      }
    }
}

constexpr int TOK_WAVES = 4;   // tokens (wavefronts) per workgroup

// mode bit 0: route (top-K + weights from logits, written to ids/w)
// mode bit 1: predict (costs from ids/w, which are read when bit 0 is off)
template <typename XT>
__global__ __launch_bounds__(TOK_WAVES * WAVE)
void k_token(const XT *__restrict__ x, int B, int d, int E, int K,
             int norm_topk, const float *__restrict__ logits,
             int32_t *__restrict__ ids_io, float *__restrict__ w_io,
             const float *__restrict__ A, const float *__restrict__ bp,
             float *__restrict__ cost, int mode) {
  const int lane = lane_id();
  const int t = blockIdx.x * TOK_WAVES + wave_id();
  if (t >= B) return;

  int ids[MAX_K];
  float w[MAX_K];
#pragma unroll
  for (int k = 0; k < MAX_K; ++k) { ids[k] = 0; w[k] = 0.0f; }

  if (mode & 1) {
    float lv[4];
    bool cand[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = lane + WAVE * i;
      cand[i] = e < E;
      lv[i] = cand[i] ? logits[(size_t)t * E + e] : 0.0f;
    }
    float lmax = 0.0f;
#pragma unroll
    for (int k = 0; k < MAX_K; ++k) {
      if (k < K) {
        float bv = -INFINITY;
        int bi = 0x7FFFFFFF;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e = lane + WAVE * i;
          if (cand[i] && ranks_before(lv[i], e, bv, bi)) { bv = lv[i]; bi = e; }
        }
        wave_argbest(bv, bi);
        ids[k] = bi;
        if (k == 0) lmax = bv;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (lane + WAVE * i == bi) cand[i] = false;
      }
    }
    float eps[MAX_K];
#pragma unroll
    for (int k = 0; k < MAX_K; ++k)
      eps[k] = (k < K) ? base_exp(logits[(size_t)t * E + ids[k]] - lmax) : 0.0f;
    float S;
    if (norm_topk) {
      S = 0.0f;
#pragma unroll
      for (int k = 0; k < MAX_K; ++k)
        if (k < K) S = S + eps[k];
    } else {
      float part = 0.0f;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = lane + WAVE * i;
        if (e < E) part = part + base_exp(logits[(size_t)t * E + e] - lmax);
      }
      S = wave_tree_sum(part);
    }
#pragma unroll
    for (int k = 0; k < MAX_K; ++k) {
      if (k < K) {
        w[k] = eps[k] / S;
        if (lane == k) {
          ids_io[(size_t)t * K + k] = ids[k];
          w_io[(size_t)t * K + k] = w[k];
        }
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < MAX_K; ++k)
      if (k < K) {
        ids[k] = ids_io[(size_t)t * K + k];
        w[k] = w_io[(size_t)t * K + k];
      }
  }

  if (!(mode & 2)) return;

  // K + 1 dot products that share the token row: ||x||^2 and a_u . x.
  const XT *xr = x + (size_t)t * d;
  float ss = 0.0f;
  float acc[MAX_K];
  const float *ar[MAX_K];
  int uk[MAX_K];
#pragma unroll
  for (int k = 0; k < MAX_K; ++k) {
    acc[k] = 0.0f;
    int u = (k < K) ? ids[k] : 0;
    uk[k] = (u >= 0 && u < E) ? u : 0;   // out-of-range ids read row 0
    ar[k] = A + (size_t)uk[k] * d;
  }
  for (int m = 0; m < d; m += 256) {
    const int kk = m + 4 * lane;
    float xv[4];
    load4(xr + kk, xv);
#pragma unroll
    for (int r = 0; r < 4; ++r) ss = __builtin_fmaf(xv[r], xv[r], ss);
#pragma unroll
    for (int k = 0; k < MAX_K; ++k) {
      if (k < K) {
        float av[4];
        load4(ar[k] + kk, av);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[k] = __builtin_fmaf(xv[r], av[r], acc[k]);
      }
    }
  }
  ss = wave_tree_sum(ss);
  float inv = 0.0f;
  if (ss > 0.0f) {
    float rt = sqrtf(ss);
    inv = 1.0f / rt;
  }
#pragma unroll
  for (int k = 0; k < MAX_K; ++k) {
    if (k < K) {
      float dk = wave_tree_sum(acc[k]);
      if (lane == k) {
        float s = dk * inv;
        s = s + bp[uk[k]];
        float w2 = w[k] * w[k];
        cost[(size_t)t * K + k] = w2 * base_exp(s);
      }
    }
  }
}

template <typename XT>
static hipError_t launch_route_t(const XT *x, int B, int d, const float *W,
                                 const float *beta, int E, float *logits,
                                 hipStream_t st) {
  dim3 grid((B + RT_TOK - 1) / RT_TOK,
            (E + RT_WAVES * RT_EXP - 1) / (RT_WAVES * RT_EXP));
  hipLaunchKernelGGL(k_route_logits<XT>, grid, dim3(RT_WAVES * WAVE), 0, st,
                     x, B, d, W, beta, E, logits);
  return hipGetLastError();
}

hipError_t launch_route_logits(bool bf16, const void *x, int B, int d,
                               const float *W, const float *beta, int E,
                               float *logits, hipStream_t st) {
  return bf16 ? launch_route_t((const uint16_t *)x, B, d, W, beta, E, logits, st)
              : launch_route_t((const float *)x, B, d, W, beta, E, logits, st);
}

hipError_t launch_token(bool bf16, const void *x, int B, int d, int E, int K,
                        int norm_topk, const float *logits, int32_t *ids,
                        float *w, const float *A, const float *bp, float *cost,
                        int mode, hipStream_t st) {
  dim3 grid((B + TOK_WAVES - 1) / TOK_WAVES);
  if (bf16)
    hipLaunchKernelGGL(k_token<uint16_t>, grid, dim3(TOK_WAVES * WAVE), 0, st,
                       (const uint16_t *)x, B, d, E, K, norm_topk, logits, ids,
                       w, A, bp, cost, mode);
  else
    hipLaunchKernelGGL(k_token<float>, grid, dim3(TOK_WAVES * WAVE), 0, st,
                       (const float *)x, B, d, E, K, norm_topk, logits, ids, w,
                       A, bp, cost, mode);
  return hipGetLastError();
}

}  // namespace basek
