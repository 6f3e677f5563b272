// Grouped SwiGLU expert FFN over the kept experts only, and the combine
// (K3, K4, K5).  Sec. 3.5: tokens execute only experts of the kept set, so
// only those experts' weights are read; Sec. 3.1: y_t = sum_v g_{t,v} E_v(z_t)
// with E_v(z) = W_d (silu(W_g z) * (W_u z)).
//
// k_gateup (slot s, 64-row tile of I): H[p][i] = bf16(silu(g) * u) for the
//   pairs p of slot s, g = x . W_g[i], u = x . W_u[i], fp32 accumulation on
//   MFMA 16x16x32 bf16 (16 weight rows x 16 tokens x 32 k per instruction,
//   tokens padded to 16).  Each workgroup streams its 64 gate rows and 64
//   up rows of the expert once.
// k_down (slot s, 64-row tile of d): pairbuf[p][c] = gate_p * (H[p] . W_d[c]).
// k_combine: y_t = residual_t + sum_j pairbuf[pair_of[t][j]] in j order.
//
// MFMA operand layout used here (v_mfma_f32_16x16x32_bf16): lane l supplies
// row (l % 16) of A and column (l % 16) of B with the 8 contraction
// elements 8*(l/16) .. 8*(l/16)+7 of a 32-wide k step; the result holds
// D[4*(l/16) + r][l % 16] in register r.
#include "common.hpp"
#include "internal.hpp"

namespace basek {

constexpr int FF_WAVES = 4;          // wavefronts per workgroup
constexpr int FF_ROWS = 16 * FF_WAVES;  // weight rows per workgroup tile
constexpr int FF_TG = 8;             // token tiles (of 16) per pass

__device__ __forceinline__ bf16x8 ld_bf16x8(const uint16_t *p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

__global__ __launch_bounds__(FF_WAVES * WAVE)
void k_gateup_bf16(const uint16_t *__restrict__ x, int d, int I, int E,
                   const uint16_t *__restrict__ w13,
                   const int32_t *__restrict__ sel_ids,
                   const int32_t *__restrict__ n_sel_p,
                   const int32_t *__restrict__ offsets,
                   const int32_t *__restrict__ pair_tok,
                   uint16_t *__restrict__ H) {
  const int s = blockIdx.x;
  if (s >= *n_sel_p) return;
  const int u = sel_ids[s];
  if (u < 0 || u >= E) return;   // only for a plan not made by base_select
  const int p0 = offsets[s];
  const int n = offsets[s + 1] - p0;
  const int lane = lane_id(), row = lane & 15, kq = (lane >> 4) * 8;
  const int i0 = blockIdx.y * FF_ROWS + wave_id() * 16;
  const uint16_t *wg = w13 + ((size_t)u * 2 * I + i0 + row) * d + kq;
  const uint16_t *wu = w13 + ((size_t)u * 2 * I + I + i0 + row) * d + kq;
  const bf16x8 zero = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});

  for (int pass = 0; pass < n; pass += 16 * FF_TG) {
    const int nt = min(FF_TG, (n - pass + 15) / 16);
    const uint16_t *xp[FF_TG];
    bool tv[FF_TG];
#pragma unroll
    for (int j = 0; j < FF_TG; ++j) {
      const int tk = pass + 16 * j + row;
      tv[j] = (j < nt) && tk < n;
      xp[j] = x + (size_t)(tv[j] ? pair_tok[p0 + tk] : 0) * d + kq;
    }
    f32x4 ag[FF_TG], au[FF_TG];
#pragma unroll
    for (int j = 0; j < FF_TG; ++j) { ag[j] = f32x4{0, 0, 0, 0}; au[j] = ag[j]; }

    for (int k0 = 0; k0 < d; k0 += 32) {
      const bf16x8 a_g = ld_bf16x8(wg + k0);
      const bf16x8 a_u = ld_bf16x8(wu + k0);
#pragma unroll
      for (int j = 0; j < FF_TG; ++j) {
        if (j < nt) {
          const bf16x8 b = tv[j] ? ld_bf16x8(xp[j] + k0) : zero;
          ag[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_g, b, ag[j], 0, 0, 0);
          au[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_u, b, au[j], 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < FF_TG; ++j) {
      const int tk = pass + 16 * j + row;
      if (j < nt && tk < n) {
        uint16_t h[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) h[r] = f32_to_bf16(silu(ag[j][r]) * au[j][r]);
        u32x2 pk = {(uint32_t)h[0] | ((uint32_t)h[1] << 16),
                    (uint32_t)h[2] | ((uint32_t)h[3] << 16)};
        *reinterpret_cast<u32x2 *>(H + (size_t)(p0 + tk) * I + i0 + 4 * (lane >> 4)) = pk;
      }
    }
  }
}

__global__ __launch_bounds__(FF_WAVES * WAVE)
void k_down_bf16(int d, int I, int E, const uint16_t *__restrict__ w2,
                 const int32_t *__restrict__ sel_ids,
                 const int32_t *__restrict__ n_sel_p,
                 const int32_t *__restrict__ offsets,
                 const float *__restrict__ pair_gate,
                 const uint16_t *__restrict__ H, float *__restrict__ pairbuf) {
  const int s = blockIdx.x;
  if (s >= *n_sel_p) return;
  const int u = sel_ids[s];
  if (u < 0 || u >= E) return;   // only for a plan not made by base_select
  const int p0 = offsets[s];
  const int n = offsets[s + 1] - p0;
  const int lane = lane_id(), row = lane & 15, kq = (lane >> 4) * 8;
  const int c0 = blockIdx.y * FF_ROWS + wave_id() * 16;
  const uint16_t *wd = w2 + ((size_t)u * d + c0 + row) * I + kq;
  const bf16x8 zero = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});

  for (int pass = 0; pass < n; pass += 16 * FF_TG) {
    const int nt = min(FF_TG, (n - pass + 15) / 16);
    const uint16_t *hp[FF_TG];
    bool tv[FF_TG];
#pragma unroll
    for (int j = 0; j < FF_TG; ++j) {
      const int tk = pass + 16 * j + row;
      tv[j] = (j < nt) && tk < n;
      hp[j] = H + (size_t)(p0 + (tv[j] ? tk : 0)) * I + kq;
    }
    f32x4 acc[FF_TG];
#pragma unroll
    for (int j = 0; j < FF_TG; ++j) acc[j] = f32x4{0, 0, 0, 0};
    for (int k0 = 0; k0 < I; k0 += 32) {
      const bf16x8 a = ld_bf16x8(wd + k0);
#pragma unroll
      for (int j = 0; j < FF_TG; ++j) {
        if (j < nt) {
          const bf16x8 b = tv[j] ? ld_bf16x8(hp[j] + k0) : zero;
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[j], 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < FF_TG; ++j) {
      const int tk = pass + 16 * j + row;
      if (j < nt && tk < n) {
        const float g = pair_gate[p0 + tk];
        float4 o = {g * acc[j][0], g * acc[j][1], g * acc[j][2], g * acc[j][3]};
        *reinterpret_cast<float4 *>(pairbuf + (size_t)(p0 + tk) * d + c0 + 4 * (lane >> 4)) = o;
      }
    }
  }
}

// fp32 experts (small layers): one thread per (intermediate row, token
// group), plain sequential dot products.
constexpr int F32_ROWS = 64;
constexpr int F32_TG = 4;

__global__ __launch_bounds__(F32_ROWS * F32_TG)
void k_gateup_f32(const float *__restrict__ x, int d, int I, int E,
                  const float *__restrict__ w13,
                  const int32_t *__restrict__ sel_ids,
                  const int32_t *__restrict__ n_sel_p,
                  const int32_t *__restrict__ offsets,
                  const int32_t *__restrict__ pair_tok, float *__restrict__ H) {
  const int s = blockIdx.x;
  if (s >= *n_sel_p) return;
  const int u = sel_ids[s];
  if (u < 0 || u >= E) return;   // only for a plan not made by base_select
  const int p0 = offsets[s];
  const int n = offsets[s + 1] - p0;
  const int i = blockIdx.y * F32_ROWS + (threadIdx.x % F32_ROWS);
  const int tg = threadIdx.x / F32_ROWS;
  if (i >= I) return;
  const float *wg = w13 + ((size_t)u * 2 * I + i) * d;
  const float *wu = w13 + ((size_t)u * 2 * I + I + i) * d;
  for (int tk = tg; tk < n; tk += F32_TG) {
    const float *xr = x + (size_t)pair_tok[p0 + tk] * d;
    float g = 0.0f, v = 0.0f;
    for (int k = 0; k < d; ++k) {
      g = __builtin_fmaf(xr[k], wg[k], g);
      v = __builtin_fmaf(xr[k], wu[k], v);
    }
    H[(size_t)(p0 + tk) * I + i] = silu(g) * v;
  }
}

__global__ __launch_bounds__(F32_ROWS * F32_TG)
void k_down_f32(int d, int I, int E, const float *__restrict__ w2,
                const int32_t *__restrict__ sel_ids,
                const int32_t *__restrict__ n_sel_p,
                const int32_t *__restrict__ offsets,
                const float *__restrict__ pair_gate,
                const float *__restrict__ H, float *__restrict__ pairbuf) {
  const int s = blockIdx.x;
  if (s >= *n_sel_p) return;
  const int u = sel_ids[s];
  if (u < 0 || u >= E) return;   // only for a plan not made by base_select
  const int p0 = offsets[s];
  const int n = offsets[s + 1] - p0;
  const int c = blockIdx.y * F32_ROWS + (threadIdx.x % F32_ROWS);
  const int tg = threadIdx.x / F32_ROWS;
  if (c >= d) return;
  const float *wd = w2 + ((size_t)u * d + c) * I;
  for (int tk = tg; tk < n; tk += F32_TG) {
    const float *hr = H + (size_t)(p0 + tk) * I;
    float o = 0.0f;
    for (int k = 0; k < I; ++k) o = __builtin_fmaf(hr[k], wd[k], o);
    pairbuf[(size_t)(p0 + tk) * d + c] = pair_gate[p0 + tk] * o;
  }
}

constexpr int CB_THREADS = 256;

template <bool BF16>
__global__ __launch_bounds__(CB_THREADS)
void k_combine(int B, int d, int K, const int32_t *__restrict__ pair_of,
               const float *__restrict__ pairbuf, const void *__restrict__ res,
               void *__restrict__ y) {
  const int t = blockIdx.x;
  const int c = (blockIdx.y * CB_THREADS + threadIdx.x) * 4;
  if (t >= B || c >= d) return;
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (res) {
    if (BF16) load4((const uint16_t *)res + (size_t)t * d + c, acc);
    else load4((const float *)res + (size_t)t * d + c, acc);
  }
  for (int j = 0; j < K; ++j) {
    const int p = pair_of[(size_t)t * K + j];
    if (p < 0) break;
    const float4 v = *reinterpret_cast<const float4 *>(pairbuf + (size_t)p * d + c);
    acc[0] = acc[0] + v.x; acc[1] = acc[1] + v.y;
    acc[2] = acc[2] + v.z; acc[3] = acc[3] + v.w;
  }
  if (BF16) {
    u32x2 pk = {(uint32_t)f32_to_bf16(acc[0]) | ((uint32_t)f32_to_bf16(acc[1]) << 16),
                (uint32_t)f32_to_bf16(acc[2]) | ((uint32_t)f32_to_bf16(acc[3]) << 16)};
    *reinterpret_cast<u32x2 *>((uint16_t *)y + (size_t)t * d + c) = pk;
  } else {
    *reinterpret_cast<float4 *>((float *)y + (size_t)t * d + c) =
        float4{acc[0], acc[1], acc[2], acc[3]};
  }
}

hipError_t launch_ffn(bool bf16, const void *x, int B, int d, int I, int K,
                      int E, int budget, const void *w13, const void *w2,
                      const int32_t *sel_ids, const int32_t *n_sel,
                      const int32_t *offsets, const int32_t *pair_tok,
                      const float *pair_gate, void *H, float *pairbuf,
                      hipStream_t st) {
  (void)B; (void)K;
  if (bf16) {
    hipLaunchKernelGGL(k_gateup_bf16, dim3(budget, I / FF_ROWS),
                       dim3(FF_WAVES * WAVE), 0, st, (const uint16_t *)x, d, I, E,
                       (const uint16_t *)w13, sel_ids, n_sel, offsets, pair_tok,
                       (uint16_t *)H);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_down_bf16, dim3(budget, d / FF_ROWS),
                       dim3(FF_WAVES * WAVE), 0, st, d, I, E, (const uint16_t *)w2,
                       sel_ids, n_sel, offsets, pair_gate, (const uint16_t *)H,
                       pairbuf);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_gateup_f32, dim3(budget, (I + F32_ROWS - 1) / F32_ROWS),
                     dim3(F32_ROWS * F32_TG), 0, st, (const float *)x, d, I, E,
                     (const float *)w13, sel_ids, n_sel, offsets, pair_tok,
                     (float *)H);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_down_f32, dim3(budget, (d + F32_ROWS - 1) / F32_ROWS),
                     dim3(F32_ROWS * F32_TG), 0, st, d, I, E, (const float *)w2,
                     sel_ids, n_sel, offsets, pair_gate, (const float *)H,
                     pairbuf);
  return hipGetLastError();
}

hipError_t launch_combine(bool bf16, int B, int d, int K,
                          const int32_t *pair_of, const float *pairbuf,
                          const void *residual, void *y, hipStream_t st) {
  dim3 grid(B, (d + CB_THREADS * 4 - 1) / (CB_THREADS * 4));
  if (bf16)
    hipLaunchKernelGGL(k_combine<true>, grid, dim3(CB_THREADS), 0, st, B, d, K,
                       pair_of, pairbuf, residual, y);
  else
    hipLaunchKernelGGL(k_combine<false>, grid, dim3(CB_THREADS), 0, st, B, d, K,
                       pair_of, pairbuf, residual, y);
  return hipGetLastError();
}

}  // namespace basek
