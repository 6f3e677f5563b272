// Streaming calibration statistics of the log-energy predictor (Sec. 3.4;
// App. A "Calibration Details"): for every routed pair (t, u) of a batch of
// calibration tokens, the target y = log(||E_u(z_t)||^2 + eps) and the
// input z_bar = z_t / ||z_t||, accumulated per expert into
//   n, sum y, sum y^2 (fp64), sum z_bar and sum z_bar y (fp64 vectors) and
//   the Gram matrix sum z_bar z_bar^T (fp32, as App. A keeps it).
// The expert outputs come from the layer's own FFN run with every routed
// expert kept and unit gates, so one batch costs one dense routed MoE pass.
//
// k_calib_norm     inv[t] = 1 / ||x_t|| (0 for x = 0), fp64
// k_calib_pairs    y[p] = log(sum_c out_p[c]^2 + eps), fp64, one workgroup per pair
// k_calib_moments  per (kept slot, 256 columns): the fp64 sums, pairs in order
// k_calib_gram     per (kept slot, 64 rows, 256 columns): G += sum_p z_i z_j
//                  (fp32 products and sums over the slot's pairs, then one add)
// Every statistic has a single writer and a fixed summation order: the
// results are deterministic.
#include "common.hpp"
#include "internal.hpp"

namespace basek {

constexpr int CAL_THREADS = 256;
constexpr double CAL_EPS = 1e-12;

__device__ __forceinline__ double act(const void *x, bool bf16, size_t i) {
  return bf16 ? (double)bf16_to_f32(((const uint16_t *)x)[i]) : (double)((const float *)x)[i];
}

// Fixed-order fp64 tree over the workgroup's CAL_THREADS values.
__device__ __forceinline__ double block_sum(double v, double *sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int h = CAL_THREADS / 2; h >= 1; h >>= 1) {
    if ((int)threadIdx.x < h) sh[threadIdx.x] = sh[threadIdx.x] + sh[threadIdx.x + h];
    __syncthreads();
  }
  const double r = sh[0];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(CAL_THREADS)
void k_calib_norm(const void *__restrict__ x, int bf16, int B, int d, double *__restrict__ inv) {
  __shared__ double sh[CAL_THREADS];
  const int t = blockIdx.x;
  if (t >= B) return;
  double s = 0.0;
  for (int c = threadIdx.x; c < d; c += CAL_THREADS) {
    const double v = act(x, bf16, (size_t)t * d + c);
    s = fma(v, v, s);
  }
  s = block_sum(s, sh);
  if (threadIdx.x == 0) inv[t] = s > 0.0 ? 1.0 / sqrt(s) : 0.0;
}

// pairs p < offsets[n_slots] (the routed pairs of the kept slots)
__global__ __launch_bounds__(CAL_THREADS)
void k_calib_pairs(const float *__restrict__ out, int d, const int32_t *__restrict__ offsets,
                   int n_slots, double *__restrict__ y) {
  __shared__ double sh[CAL_THREADS];
  const int p = blockIdx.x;
  if (p >= offsets[n_slots]) return;
  double s = 0.0;
  for (int c = threadIdx.x; c < d; c += CAL_THREADS) {
    const double v = (double)out[(size_t)p * d + c];
    s = fma(v, v, s);
  }
  s = block_sum(s, sh);
  if (threadIdx.x == 0) y[p] = log(s + CAL_EPS);
}

__global__ __launch_bounds__(CAL_THREADS)
void k_calib_moments(const void *__restrict__ x, int bf16, int d, const double *__restrict__ inv,
                     const int32_t *__restrict__ n_sel, const int32_t *__restrict__ sel_ids,
                     const int32_t *__restrict__ offsets, const int32_t *__restrict__ pair_tok,
                     const double *__restrict__ y, CalibStats st) {
  const int s = blockIdx.x;
  if (s >= *n_sel) return;
  const int u = sel_ids[s];
  const int p0 = offsets[s], p1 = offsets[s + 1];
  const int j = blockIdx.y * CAL_THREADS + threadIdx.x;
  if (j < d) {
    double sz = 0.0, q = 0.0;
    for (int p = p0; p < p1; ++p) {
      const int t = pair_tok[p];
      const double z = act(x, bf16, (size_t)t * d + j) * inv[t];
      sz = sz + z;
      q = fma(z, y[p], q);
    }
    st.sz[(size_t)u * d + j] += sz;
    st.q[(size_t)u * d + j] += q;
  }
  if (blockIdx.y == 0 && threadIdx.x == 0) {
    double sy = 0.0, syy = 0.0;
    for (int p = p0; p < p1; ++p) {
      sy = sy + y[p];
      syy = fma(y[p], y[p], syy);
    }
    st.head[(size_t)u * 4 + 0] += (double)(p1 - p0);
    st.head[(size_t)u * 4 + 1] += sy;
    st.head[(size_t)u * 4 + 2] += syy;
  }
}

constexpr int GR_ROWS = 64;   // rows of G per workgroup
constexpr int GR_STAGE = 16;  // pairs whose row values are staged at a time

__global__ __launch_bounds__(CAL_THREADS)
void k_calib_gram(const void *__restrict__ x, int bf16, int d, const double *__restrict__ inv,
                  const int32_t *__restrict__ n_sel, const int32_t *__restrict__ sel_ids,
                  const int32_t *__restrict__ offsets, const int32_t *__restrict__ pair_tok,
                  float *__restrict__ G) {
  __shared__ float zr[GR_STAGE][GR_ROWS];
  const int s = blockIdx.x;
  if (s >= *n_sel) return;
  const int u = sel_ids[s];
  const int p0 = offsets[s], p1 = offsets[s + 1];
  const int i0 = blockIdx.y * GR_ROWS;
  const int j = blockIdx.z * CAL_THREADS + threadIdx.x;
  float acc[GR_ROWS];
#pragma unroll
  for (int r = 0; r < GR_ROWS; ++r) acc[r] = 0.0f;
  for (int pb = p0; pb < p1; pb += GR_STAGE) {
    const int np = min(GR_STAGE, p1 - pb);
    // stage the row values of up to GR_STAGE pairs
    for (int k = threadIdx.x; k < np * GR_ROWS; k += CAL_THREADS) {
      const int pp = k / GR_ROWS, r = k % GR_ROWS;
      const int t = pair_tok[pb + pp];
      zr[pp][r] = (i0 + r < d) ? (float)(act(x, bf16, (size_t)t * d + i0 + r) * inv[t]) : 0.0f;
    }
    __syncthreads();
    if (j < d) {
      for (int pp = 0; pp < np; ++pp) {
        const int t = pair_tok[pb + pp];
        const float zj = (float)(act(x, bf16, (size_t)t * d + j) * inv[t]);
#pragma unroll
        for (int r = 0; r < GR_ROWS; ++r) acc[r] = fmaf(zr[pp][r], zj, acc[r]);
      }
    }
    __syncthreads();
  }
  if (j < d && p1 > p0) {
    float *g = G + (size_t)u * d * d;
#pragma unroll
    for (int r = 0; r < GR_ROWS; ++r)
      if (i0 + r < d) g[(size_t)(i0 + r) * d + j] += acc[r];
  }
}

__global__ __launch_bounds__(CAL_THREADS)
void k_fill_zero(uint32_t *__restrict__ p, size_t n) {
  for (size_t i = blockIdx.x * (size_t)CAL_THREADS + threadIdx.x; i < n;
       i += (size_t)gridDim.x * CAL_THREADS)
    p[i] = 0u;
}

hipError_t launch_calib_zero(void *stats, size_t bytes, hipStream_t st) {
  const size_t n = bytes / 4;
  const size_t nb = (n + CAL_THREADS - 1) / CAL_THREADS;
  const unsigned blocks = (unsigned)(nb < 65536 ? nb : 65536);
  launch_k(k_fill_zero, dim3(blocks), dim3(CAL_THREADS), 0, st, (uint32_t *)stats, n);
  return hipGetLastError();
}

hipError_t launch_calib_stats(const void *x, bool bf16, int B, int d, int E, int K,
                              const float *pairbuf, const int32_t *n_sel,
                              const int32_t *sel_ids, const int32_t *offsets,
                              const int32_t *pair_tok, double *inv, double *y,
                              CalibStats st, hipStream_t s) {
  launch_k(k_calib_norm, dim3(B), dim3(CAL_THREADS), 0, s, x, (int)bf16, B, d, inv);
  launch_k(k_calib_pairs, dim3(B * K), dim3(CAL_THREADS), 0, s, pairbuf, d, offsets, E, y);
  launch_k(k_calib_moments, dim3(E, (d + CAL_THREADS - 1) / CAL_THREADS), dim3(CAL_THREADS), 0,
           s, x, (int)bf16, d, (const double *)inv, n_sel, sel_ids, offsets, pair_tok,
           (const double *)y, st);
  launch_k(k_calib_gram,
           dim3(E, (d + GR_ROWS - 1) / GR_ROWS, (d + CAL_THREADS - 1) / CAL_THREADS),
           dim3(CAL_THREADS), 0, s, x, (int)bf16, d, (const double *)inv, n_sel, sel_ids,
           offsets, pair_tok, st.G);
  return hipGetLastError();
}

}  // namespace basek
