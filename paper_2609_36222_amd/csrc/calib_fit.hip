// The log-energy predictor's fit from the calibration statistics (Sec. 3.4;
// App. A "Calibration Details"): per expert a centred closed-form ridge,
//   a(lam) = (G_c + lam I)^-1 q_c,   b(lam) = y_mean - a(lam) . z_mean,
// for every lam of a list from one eigendecomposition of G_c (rocSOLVER,
// fp64), the lam of largest marginal likelihood (the Bayesian-ridge
// evidence with the noise variance profiled out), and the log-normal bias
// correction b += RSS / (2 n).  Built into its own library (it links
// rocSOLVER); an offline step.
//
// k_fit_build  G_c = G - n z_mean z_mean^T in fp64, symmetrised, into the
//              eigensolver's input (one workgroup per 256 entries of a row)
// k_fit_solve  one workgroup per expert: q_c, V^T q_c, the evidence of each
//              lam (fixed-order fp64 reductions), a = V (V^T q_c / (s + lam)),
//              b; writes pred_a, pred_b and the chosen lam
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver.h>
#include <stdint.h>

#include "../../include/base.h"
#include "../../include/base_calib.h"
#include "internal.hpp"

namespace {

using namespace basek;

constexpr int FT = 256;           // threads of k_fit_build
constexpr int FS = 1024;          // threads of k_fit_solve
constexpr int FIT_CHUNK = 8;      // experts per eigensolver batch
constexpr int MAX_LAMBDA = 64;

__global__ __launch_bounds__(FT)
void k_fit_build(CalibStats st, int d, int u0, int nu, double *__restrict__ A) {
  const int e = blockIdx.z, i = blockIdx.y, j = blockIdx.x * FT + threadIdx.x;
  if (e >= nu || j >= d) return;
  const int u = u0 + e;
  const double n = st.head[(size_t)u * 4];
  const double *sz = st.sz + (size_t)u * d;
  const float *G = st.G + (size_t)u * d * d;
  const double zi = n > 0 ? sz[i] / n : 0.0, zj = n > 0 ? sz[j] / n : 0.0;
  const double gij = (double)G[(size_t)i * d + j] - n * zi * zj;
  const double gji = (double)G[(size_t)j * d + i] - n * zj * zi;
  A[(size_t)e * d * d + (size_t)i * d + j] = 0.5 * (gij + gji);
}

// Fixed-order fp64 sum over the workgroup (FS threads).
__device__ __forceinline__ double fit_sum(double v, double *sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int h = FS / 2; h >= 1; h >>= 1) {
    if ((int)threadIdx.x < h) sh[threadIdx.x] = sh[threadIdx.x] + sh[threadIdx.x + h];
    __syncthreads();
  }
  const double r = sh[0];
  __syncthreads();
  return r;
}

// V: the eigenvectors of expert e in column-major order (column k =
// eigenvector k, eigenvalue D[k]); qv and av: scratch [d] fp64.
__global__ __launch_bounds__(FS)
void k_fit_solve(CalibStats st, int d, int u0, int nu, const double *__restrict__ V,
                 const double *__restrict__ D, const double *__restrict__ lams, int n_lam,
                 double *__restrict__ qv_s, double *__restrict__ av_s,
                 float *__restrict__ pred_a, float *__restrict__ pred_b,
                 float *__restrict__ lam_out) {
  __shared__ double sh[FS];
  const int e = blockIdx.x;
  if (e >= nu) return;
  const int u = u0 + e;
  const int tid = threadIdx.x;
  const double n = st.head[(size_t)u * 4 + 0];
  if (n <= 0) {   // an expert no calibration token routes
    for (int i = tid; i < d; i += FS) pred_a[(size_t)u * d + i] = 0.0f;
    if (tid == 0) {
      pred_b[u] = 0.0f;
      if (lam_out) lam_out[u] = (float)lams[0];
    }
    return;
  }
  const double *sz = st.sz + (size_t)u * d, *q = st.q + (size_t)u * d;
  const double ym = st.head[(size_t)u * 4 + 1] / n;
  const double yyc = st.head[(size_t)u * 4 + 2] - n * ym * ym;
  const double *Ve = V + (size_t)e * d * d, *De = D + (size_t)e * d;
  double *qv = qv_s + (size_t)e * d, *av = av_s + (size_t)e * d;
  // qv = V^T q_c, q_c = q - n z_mean y_mean
  for (int k = tid; k < d; k += FS) {
    double s = 0.0;
    for (int i = 0; i < d; ++i) s = fma(Ve[(size_t)k * d + i], q[i] - n * (sz[i] / n) * ym, s);
    qv[k] = s;
  }
  __syncthreads();
  double best_e = 0.0, best_lam = lams[0], best_rss = 0.0;
  for (int l = 0; l < n_lam; ++l) {
    const double lam = lams[l];
    double s1 = 0.0, s2 = 0.0, s3 = 0.0, s4 = 0.0;
    for (int k = tid; k < d; k += FS) {
      const double sg = De[k] > 0.0 ? De[k] : 0.0;
      const double a = qv[k] / (sg + lam);
      s1 += a * qv[k];
      s2 += sg * a * a;
      s3 += a * a;
      s4 += log(lam / (sg + lam));
    }
    s1 = fit_sum(s1, sh);
    s2 = fit_sum(s2, sh);
    s3 = fit_sum(s3, sh);
    s4 = fit_sum(s4, sh);
    double rss = yyc - 2.0 * s1 + s2;
    rss = rss > 0.0 ? rss : 0.0;
    const double quad = rss + lam * s3;
    const double ev = -0.5 * n * log(quad > 1e-300 ? quad : 1e-300) + 0.5 * s4;
    if (l == 0 || ev > best_e) {   // ties keep the smaller lam
      best_e = ev;
      best_lam = lam;
      best_rss = rss;
    }
  }
  for (int k = tid; k < d; k += FS) {
    const double sg = De[k] > 0.0 ? De[k] : 0.0;
    av[k] = qv[k] / (sg + best_lam);
  }
  __syncthreads();
  // a = V av; a . z_mean for b
  double az = 0.0;
  for (int i = tid; i < d; i += FS) {
    double a = 0.0;
    for (int k = 0; k < d; ++k) a = fma(Ve[(size_t)k * d + i], av[k], a);
    pred_a[(size_t)u * d + i] = (float)a;
    az += a * (sz[i] / n);
  }
  az = fit_sum(az, sh);
  if (tid == 0) {
    pred_b[u] = (float)(ym - az + 0.5 * best_rss / n);
    if (lam_out) lam_out[u] = (float)best_lam;
  }
}

}  // namespace

extern "C" {

base_status base_calib_fit(const base_layer *L, const void *stats, int32_t n_lambda,
                           const double *lambdas, float *pred_a, float *pred_b, float *lam_out,
                           void *stream) {
  if (!L || !stats || !lambdas || !pred_a || !pred_b) return BASE_ERR_NULL;
  if (L->E < 1 || L->E > MAX_E || L->d < 256 || L->d > 16384 || L->d % 256) return BASE_ERR_SHAPE;
  if (n_lambda < 1 || n_lambda > MAX_LAMBDA) return BASE_ERR_SHAPE;
  for (int l = 0; l < n_lambda; ++l)
    if (!(lambdas[l] > 0.0)) return BASE_ERR_SHAPE;
  if ((uintptr_t)stats % 256 || (uintptr_t)pred_a % 4 || (uintptr_t)pred_b % 4)
    return BASE_ERR_ALIGN;
  const int E = L->E, d = L->d;
  hipStream_t st = (hipStream_t)stream;
  const CalibStats cs = calib_stats_at(const_cast<void *>(stats), E, d);
  const int chunk = E < FIT_CHUNK ? E : FIT_CHUNK;
  double *A = nullptr, *D = nullptr, *Ew = nullptr, *qv = nullptr, *av = nullptr, *lam_d = nullptr;
  rocblas_int *info = nullptr;
  rocblas_handle h = nullptr;
  base_status ret = BASE_OK;
  auto fail = [&](base_status s) { if (ret == BASE_OK) ret = s; };
  if (hipMalloc(&A, (size_t)chunk * d * d * 8) != hipSuccess ||
      hipMalloc(&D, (size_t)chunk * d * 8) != hipSuccess ||
      hipMalloc(&Ew, (size_t)chunk * d * 8) != hipSuccess ||
      hipMalloc(&qv, (size_t)chunk * d * 8) != hipSuccess ||
      hipMalloc(&av, (size_t)chunk * d * 8) != hipSuccess ||
      hipMalloc(&lam_d, (size_t)n_lambda * 8) != hipSuccess ||
      hipMalloc(&info, (size_t)chunk * sizeof(rocblas_int)) != hipSuccess)
    fail(BASE_ERR_HIP);
  if (ret == BASE_OK && (rocblas_create_handle(&h) != rocblas_status_success ||
                         rocblas_set_stream(h, st) != rocblas_status_success))
    fail(BASE_ERR_HIP);
  if (ret == BASE_OK &&
      hipMemcpyAsync(lam_d, lambdas, (size_t)n_lambda * 8, hipMemcpyHostToDevice, st) != hipSuccess)
    fail(BASE_ERR_HIP);
  for (int u0 = 0; ret == BASE_OK && u0 < E; u0 += chunk) {
    const int nu = E - u0 < chunk ? E - u0 : chunk;
    hipLaunchKernelGGL(k_fit_build, dim3((d + FT - 1) / FT, d, nu), dim3(FT), 0, st, cs, d, u0,
                       nu, A);
    if (hipGetLastError() != hipSuccess) { fail(BASE_ERR_HIP); break; }
    if (rocsolver_dsyevd_strided_batched(h, rocblas_evect_original, rocblas_fill_upper, d, A, d,
                                         (rocblas_stride)d * d, D, d, Ew, d, info, nu) !=
        rocblas_status_success) {
      fail(BASE_ERR_HIP);
      break;
    }
    hipLaunchKernelGGL(k_fit_solve, dim3(nu), dim3(FS), 0, st, cs, d, u0, nu, A, D, lam_d,
                       n_lambda, qv, av, pred_a, pred_b, lam_out);
    if (hipGetLastError() != hipSuccess) fail(BASE_ERR_HIP);
  }
  // the scratch is freed only once the stream has finished with it
  if (hipStreamSynchronize(st) != hipSuccess) fail(BASE_ERR_HIP);
  if (h) rocblas_destroy_handle(h);
  hipFree(A);
  hipFree(D);
  hipFree(Ew);
  hipFree(qv);
  hipFree(av);
  hipFree(lam_d);
  hipFree(info);
  return ret;
}

}  // extern "C"
