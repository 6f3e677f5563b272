// The staged removal-cost predictor (Sec. 3.4, eq. log_energy_predictor;
// App. "Custom GPU Kernels": the token is normalised once and reused
// across its K experts).
//
// k_token : one wavefront per token: cost = w^2 exp(a_u . x/||x|| + b_u) for
//           the routed pairs it is given.
//
// Every dot product of length d uses one fixed order: lane j of a wavefront
// owns elements 256m + 4j + r (r = 0..3), accumulates them in ascending
// element order with single-rounding FMA from +0, and the 64 lane partials
// are joined by the halving tree (wave_tree_sum).  It is the order of
// k_scores too, so both predictors give the same bits.
#include "common.hpp"
#include "internal.hpp"

namespace basek {

constexpr int TOK_WAVES = 4;   // tokens (wavefronts) per workgroup

// The predicted cost of the routed pairs given in ids / w, one wavefront
// per token (the staged predictor; the fused layer gets the same values
// from k_scores and k_tail).
template <typename XT>
__global__ __launch_bounds__(TOK_WAVES * WAVE)
void k_token(const XT *__restrict__ x, int B, int d, int E, int K,
             const int32_t *__restrict__ ids_in, const float *__restrict__ w_in,
             const float *__restrict__ A, const float *__restrict__ bp,
             float *__restrict__ cost) {
  const int lane = lane_id();
  const int t = blockIdx.x * TOK_WAVES + wave_id();
  if (t >= B) return;

  int ids[MAX_K];
  float w[MAX_K];
#pragma unroll
  for (int k = 0; k < MAX_K; ++k) {
    ids[k] = (k < K) ? ids_in[(size_t)t * K + k] : 0;
    w[k] = (k < K) ? w_in[(size_t)t * K + k] : 0.0f;
  }

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

hipError_t launch_predict(bool bf16, const void *x, int B, int d, int E, int K,
                          const int32_t *ids, const float *w, const float *A,
                          const float *bp, float *cost, hipStream_t st) {
  dim3 grid((B + TOK_WAVES - 1) / TOK_WAVES);
  if (bf16)
    launch_k(k_token<uint16_t>, grid, dim3(TOK_WAVES * WAVE), 0, st,
                       (const uint16_t *)x, B, d, E, K, ids, w, A, bp, cost);
  else
    launch_k(k_token<float>, grid, dim3(TOK_WAVES * WAVE), 0, st,
                       (const float *)x, B, d, E, K, ids, w, A, bp, cost);
  return hipGetLastError();
}

}  // namespace basek
