// Streaming calibration statistics of the log-energy predictor (Sec. 3.4;
// App. A "Calibration Details"): for every routed pair (t, u) of a batch of
// calibration tokens, the target y = log(||E_u(z_t)||^2 + eps) and the
// input z_bar = z_t / ||z_t||, accumulated per expert into
//   n, sum y, sum y^2 (fp64), sum z_bar and sum z_bar y (fp64 vectors) and
//   the Gram matrix sum z_bar z_bar^T (fp32, as App. A keeps it).
// The expert outputs come from the layer's own FFN run with every routed
// expert kept and unit gates, so one batch costs one dense routed MoE pass.
//
// k_calib_norm     inv[t] = 1 / ||x_t|| (0 for x = 0), fp64, and the rows
//                  z_bar_t = fp32(x_t inv[t]) the Gram reads (plus a zero row)
// k_calib_pairs    y[p] = log(sum_c out_p[c]^2 + eps), fp64, one workgroup per pair
// k_calib_moments  per (kept slot, 256 columns): the fp64 sums, pairs in order
// k_calib_gram     per (kept slot, 128 x 128 block of the upper triangle):
//                  G += sum_p z_i z_j on the matrix cores (fp32 products and
//                  sums over the slot's pairs, then one add), mirrored
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
void k_calib_norm(const void *__restrict__ x, int bf16, int B, int d, double *__restrict__ inv,
                  float *__restrict__ zbuf) {
  __shared__ double sh[CAL_THREADS];
  const int t = blockIdx.x;
  if (t >= B) return;
  double s = 0.0;
  for (int c = threadIdx.x; c < d; c += CAL_THREADS) {
    const double v = act(x, bf16, (size_t)t * d + c);
    s = fma(v, v, s);
  }
  s = block_sum(s, sh);
  const double iv = s > 0.0 ? 1.0 / sqrt(s) : 0.0;
  if (threadIdx.x == 0) inv[t] = iv;
  for (int c = threadIdx.x; c < d; c += CAL_THREADS)
    zbuf[(size_t)t * d + c] = (float)(act(x, bf16, (size_t)t * d + c) * iv);
  if (t == 0)   // the zero row B
    for (int c = threadIdx.x; c < d; c += CAL_THREADS) zbuf[(size_t)B * d + c] = 0.0f;
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

// The Gram matrices on the matrix cores (v_mfma_f32_16x16x4_f32: fp32
// operands, products and sums).  A workgroup owns one 128 x 128 block (I, J),
// I <= J, of one kept slot's G_u, and each of its four wavefronts a 64 x 64
// quarter (rows rb.., columns cb..) as 4 x 4 instruction tiles.  Tile (a, b)
// takes rows rb + 4 i + a and columns cb + 4 j + b (i, j = 0..15), so that a
// lane's four A values (and four B values) are one 16-byte load: lane l
// supplies A[l % 16][l / 16] = z_p[rb + 4 (l % 16) + a] and B[l / 16][l % 16]
// = z_p[cb + 4 (l % 16) + b] with p = the step's first pair + l / 16, and
// holds C[4 (l / 16) + r][l % 16], r = 0..3, i.e. row rb + 16 (l / 16) + 4 r
// + a, column cb + 4 (l % 16) + b: for each (r, a) a 16-byte piece of a row.
// The contraction runs over the slot's pairs in order, four per step, in
// chunks of 64 pairs whose tokens the lanes hold (one each) and pass round
// by lane exchange; operands are requested three steps ahead; pairs past
// the slot's end read zbuf's zero row B.  The batch's sums start from zero
// and are added to G once.  Only blocks I <= J are computed: the new
// values of (I, J) are also written, transposed, to (J, I), so G_u stays
// exactly symmetric and the lower blocks are never read.  Workgroup b runs
// on die b mod 8 and the blocks of slot s go to die s mod 8, so that the
// slot's operand rows stay in one L2.  zbuf [B + 1][d] (fp32) holds the
// rows z_bar_t = fp32(x_t inv[t]) and a zero row (k_calib_norm).
constexpr int GM_TILE = 128;
constexpr int GM_WAVES = 4;
constexpr int GM_AHEAD = 3;   // steps of operands in flight (ring of 4)

__device__ __forceinline__ f32x4 mfma_f32_4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__global__ __launch_bounds__(GM_WAVES * WAVE, 2)
void k_calib_gram(const float *__restrict__ zbuf, int B, int d, int n_blk, int slots_per_die,
                  const int32_t *__restrict__ n_sel, const int32_t *__restrict__ sel_ids,
                  const int32_t *__restrict__ offsets, const int32_t *__restrict__ pair_tok,
                  float *__restrict__ G) {
  const int x = blockIdx.x % N_XCD, i = blockIdx.x / N_XCD;
  const int s = x + N_XCD * (i / n_blk);
  int k = i % n_blk;
  if (i / n_blk >= slots_per_die || s >= *n_sel) return;
  const int p0 = offsets[s], p1 = offsets[s + 1];
  if (p1 <= p0) return;
  // block k of the upper triangle, row by row
  const int T = d / GM_TILE;
  int I = 0;
  while (k >= T - I) { k -= T - I; ++I; }
  const int J = I + k;
  const int lane = threadIdx.x % WAVE, w = threadIdx.x / WAVE;
  const int m = lane & 15, kk = lane >> 4;
  const int rb = I * GM_TILE + (w >> 1) * 64, cb = J * GM_TILE + (w & 1) * 64;
  float *g = G + (size_t)sel_ids[s] * d * d;

  auto toks = [&](int pc) { return pc + lane < p1 ? pair_tok[pc + lane] : B; };
  f32x4 ra[GM_AHEAD + 1], rbv[GM_AHEAD + 1];
  auto load = [&](int slot, int t) {
    const float *zr = zbuf + (size_t)t * d;
    ra[slot] = *(const f32x4 *)(zr + rb + 4 * m);
    rbv[slot] = *(const f32x4 *)(zr + cb + 4 * m);
  };
  int tcur = toks(p0), tnext = toks(p0 + WAVE);
#pragma unroll
  for (int q = 0; q < GM_AHEAD; ++q) load(q, __shfl(tcur, 4 * q + kk));
  // the block's old values (rows rb + 16 kk + 4 r + a, 16 bytes at cb + 4 m)
  f32x4 old[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int a = 0; a < 4; ++a)
      old[r][a] = *(const f32x4 *)(g + (size_t)(rb + 16 * kk + 4 * r + a) * d + cb + 4 * m);

  f32x4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int pc = p0; pc < p1; pc += WAVE) {
#pragma unroll
    for (int st = 0; st < WAVE / 4; ++st) {
      if (pc + 4 * st >= p1) break;
      const int ahead = st + GM_AHEAD;
      load(ahead % (GM_AHEAD + 1),
           ahead < WAVE / 4 ? __shfl(tcur, 4 * ahead + kk) : __shfl(tnext, 4 * (ahead - WAVE / 4) + kk));
      const f32x4 za = ra[st % (GM_AHEAD + 1)], zb = rbv[st % (GM_AHEAD + 1)];
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = mfma_f32_4(za[a], zb[b], acc[a][b]);
    }
    tcur = tnext;
    tnext = toks(pc + 2 * WAVE);
  }

#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const f32x4 v = old[r][a] + f32x4{acc[a][0][r], acc[a][1][r], acc[a][2][r], acc[a][3][r]};
      *(f32x4 *)(g + (size_t)(rb + 16 * kk + 4 * r + a) * d + cb + 4 * m) = v;
      old[r][a] = v;
    }
  if (I != J) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int b = 0; b < 4; ++b)
        *(f32x4 *)(g + (size_t)(cb + 4 * m + b) * d + rb + 16 * kk + 4 * r) =
            f32x4{old[r][0][b], old[r][1][b], old[r][2][b], old[r][3][b]};
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
                              const int32_t *pair_tok, double *inv, double *y, float *zbuf,
                              CalibStats st, hipStream_t s) {
  launch_k(k_calib_norm, dim3(B), dim3(CAL_THREADS), 0, s, x, (int)bf16, B, d, inv, zbuf);
  launch_k(k_calib_pairs, dim3(B * K), dim3(CAL_THREADS), 0, s, pairbuf, d, offsets, E, y);
  launch_k(k_calib_moments, dim3(E, (d + CAL_THREADS - 1) / CAL_THREADS), dim3(CAL_THREADS), 0,
           s, x, (int)bf16, d, (const double *)inv, n_sel, sel_ids, offsets, pair_tok,
           (const double *)y, st);
  const int T = d / GM_TILE, n_blk = T * (T + 1) / 2;
  const int per_die = (E + N_XCD - 1) / N_XCD;
  launch_k(k_calib_gram, dim3((unsigned)(N_XCD * per_die * n_blk)), dim3(GM_WAVES * WAVE), 0, s,
           (const float *)zbuf, B, d, n_blk, per_die, n_sel, sel_ids, offsets, pair_tok, st.G);
  return hipGetLastError();
}

}  // namespace basek
