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
constexpr int FF_TG = 8;             // token tiles (of 16) per pass
constexpr int FF_Q = 4;              // k-steps (of 32) per pipeline chunk
constexpr int FRAG = 64 * 16;        // bytes of one MFMA operand fragment
constexpr int FF_LDS = 2 * FF_TG * FF_Q * FRAG;   // double-buffered chunk

__device__ __forceinline__ bf16x8 ld_bf16x8(const uint16_t *p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Pipeline over chunks of Q k-steps.  Token fragments (the MFMA B operand,
// shared by the workgroup's wavefronts) pass through a double-buffered LDS
// area in MFMA lane order: fragment (tile j, k-step q) holds lane l's 16
// bytes at l * 16, so reads are conflict-free.  Wavefront w fetches k-step
// q = w of every tile.  Step c: store chunk c's token registers to LDS half
// (c & 1), barrier, request chunk c + 1 (tokens into registers, weights into
// the other weight register set), multiply chunk c.  Loads are issued in
// the order tokens, then weights, so waiting for a chunk's tokens never
// waits for the weights requested after them.
template <int NT, int Q>
__device__ __forceinline__ void load_tokens(bf16x8 (&tok)[FF_TG],
                                            const uint16_t *const *trow, int c) {
  static_assert(Q == 2 || Q == 4, "chunk depth");
  const int w = wave_id();
  if constexpr (Q == 4) {          // wavefront w: k-step w of every tile
#pragma unroll
    for (int j = 0; j < NT; ++j) tok[j] = ld_bf16x8(trow[j] + (c * Q + w) * 32);
  } else {                         // tiles 2m + (w >= 2), k-step w % 2
#pragma unroll
    for (int m = 0; m < (NT + 1) / 2; ++m) {
      const uint16_t *row = trow[2 * m];
      if (2 * m + 1 < NT && w >= 2) row = trow[2 * m + 1];
      if (2 * m + (w >= 2) < NT) tok[m] = ld_bf16x8(row + (c * Q + (w & 1)) * 32);
    }
  }
}

template <int RT, int Q>
__device__ __forceinline__ void load_weights(bf16x8 (&wdst)[RT][Q],
                                             const uint16_t *const *wr, int c) {
#pragma unroll
  for (int q = 0; q < Q; ++q)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
      wdst[rt][q] = ld_bf16x8(wr[rt] + (c * Q + q) * 32);
}

template <int NT, int RT, int Q>
__device__ __forceinline__ void mul_chunk(const bf16x8 (&wc)[RT][Q],
                                          const char *buf, f32x4 (&acc)[RT][FF_TG]) {
  const int lane = lane_id();
#pragma unroll
  for (int q = 0; q < Q; ++q) {
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const bf16x8 t = *reinterpret_cast<const bf16x8 *>(
          buf + (j * Q + q) * FRAG + lane * 16);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) acc[rt][j] = mfma16(wc[rt][q], t, acc[rt][j]);
    }
  }
}

// Step c of the pipeline: store chunk c's token registers to LDS half
// (c & 1); barrier; request chunk c + 1 (tokens into the token registers,
// weights into the other weight register set); multiply chunk c.  Issue
// order tokens-then-weights keeps each wait from covering loads requested
// after the data it needs.
template <int NT, int RT, int Q>
__device__ __forceinline__ void pipe_step(int c, bool more, bf16x8 (&tok)[FF_TG],
                                          const bf16x8 (&wc)[RT][Q],
                                          bf16x8 (&wn)[RT][Q],
                                          const uint16_t *const *wr,
                                          const uint16_t *const *trow, char *lds,
                                          f32x4 (&acc)[RT][FF_TG]) {
  const int w = wave_id(), lane = lane_id();
  char *buf = lds + (c & 1) * (FF_LDS / 2);
  if constexpr (Q == 4) {
#pragma unroll
    for (int j = 0; j < NT; ++j)
      *reinterpret_cast<bf16x8 *>(buf + (j * Q + w) * FRAG + lane * 16) = tok[j];
  } else {
#pragma unroll
    for (int m = 0; m < (NT + 1) / 2; ++m) {
      const int j = 2 * m + (w >= 2);
      if (j < NT)
        *reinterpret_cast<bf16x8 *>(buf + (j * Q + (w & 1)) * FRAG + lane * 16) = tok[m];
    }
  }
  __syncthreads();
  // issue chunk c + 1's loads before chunk c's MFMAs (scheduling fences
  // keep the compiler from sinking them next to their uses)
  __builtin_amdgcn_sched_barrier(0);
  if (more) {
    load_tokens<NT, Q>(tok, trow, c + 1);
    load_weights<RT, Q>(wn, wr, c + 1);
  }
  __builtin_amdgcn_sched_barrier(0);
  mul_chunk<NT, RT, Q>(wc, buf, acc);
  __builtin_amdgcn_sched_barrier(0);
}

// kl must be a multiple of 32 * Q
template <int NT, int RT, int Q>
__device__ __forceinline__ void stream_rows_q(const uint16_t *const *wr,
                                              const uint16_t *const *trow, int kl,
                                              char *lds, f32x4 (&acc)[RT][FF_TG]) {
  const int nchunks = kl / (32 * Q);
  bf16x8 tok[FF_TG], wa[RT][Q], wb[RT][Q];
  load_tokens<NT, Q>(tok, trow, 0);
  load_weights<RT, Q>(wa, wr, 0);
  int c = 0;
  for (; c + 2 < nchunks; c += 2) {
    pipe_step<NT, RT, Q>(c, true, tok, wa, wb, wr, trow, lds, acc);
    pipe_step<NT, RT, Q>(c + 1, true, tok, wb, wa, wr, trow, lds, acc);
  }
  if (nchunks - c == 2) {
    pipe_step<NT, RT, Q>(c, true, tok, wa, wb, wr, trow, lds, acc);
    pipe_step<NT, RT, Q>(c + 1, false, tok, wb, wa, wr, trow, lds, acc);
  } else {
    pipe_step<NT, RT, Q>(c, false, tok, wa, wb, wr, trow, lds, acc);
  }
  __syncthreads();   // LDS free for the next pass
}

template <int NT, int RT, int Q>
__device__ __forceinline__ void stream_rows(const uint16_t *const *wr,
                                            const uint16_t *const *trow, int kl,
                                            char *lds, f32x4 (&acc)[RT][FF_TG]) {
  stream_rows_q<NT, RT, Q>(wr, trow, kl, lds, acc);
}

// Token row pointers of this lane for the NT tiles of a pass: tile j, lane
// l covers token 16 j + (l % 16) at k offset 8 (l / 16).  Padded slots point
// at a real row; their output columns are discarded.
__device__ __forceinline__ void token_rows(const uint16_t *base, size_t stride,
                                           const int32_t *rows, int pass, int n,
                                           const uint16_t **trow) {
  const int lane = lane_id();
#pragma unroll
  for (int j = 0; j < FF_TG; ++j) {
    const int tk = min(pass + 16 * j + (lane & 15), n - 1);
    const size_t r = rows ? (size_t)rows[tk] : (size_t)tk;
    trow[j] = base + r * stride + (lane >> 4) * 8;
  }
}

__global__ __launch_bounds__(FF_WAVES * WAVE, 2)
void k_gateup_bf16(const uint16_t *__restrict__ x, int d, int I, int E,
                   const uint16_t *__restrict__ w13,
                   const int32_t *__restrict__ sel_ids,
                   const int32_t *__restrict__ n_sel_p,
                   const int32_t *__restrict__ offsets,
                   const int32_t *__restrict__ pair_tok,
                   uint16_t *__restrict__ H) {
  __shared__ __attribute__((aligned(1024))) char lds[FF_LDS];
  const int s = blockIdx.x;
  if (s >= *n_sel_p) return;
  const int u = sel_ids[s];
  if (u < 0 || u >= E) return;   // only for a plan not made by base_select
  const int p0 = offsets[s];
  const int n = offsets[s + 1] - p0;
  if (n <= 0) return;
  const int lane = lane_id(), row = lane & 15, kq = (lane >> 4) * 8;
  const int i0 = blockIdx.y * (16 * FF_WAVES) + wave_id() * 16;
  const uint16_t *wr[2] = {w13 + ((size_t)u * 2 * I + i0 + row) * d + kq,
                           w13 + ((size_t)u * 2 * I + I + i0 + row) * d + kq};

  for (int pass = 0; pass < n; pass += 16 * FF_TG) {
    const int nt = min(FF_TG, (n - pass + 15) / 16);
    const uint16_t *trow[FF_TG];
    token_rows(x, (size_t)d, pair_tok + p0, pass, n, trow);
    f32x4 acc[2][FF_TG];
#pragma unroll
    for (int j = 0; j < FF_TG; ++j) acc[0][j] = acc[1][j] = f32x4{0, 0, 0, 0};
    switch (nt) {
      case 1: stream_rows<1, 2, 4>(wr, trow, d, lds, acc); break;
      case 2: stream_rows<2, 2, 4>(wr, trow, d, lds, acc); break;
      case 3: stream_rows<3, 2, 4>(wr, trow, d, lds, acc); break;
      case 4: stream_rows<4, 2, 4>(wr, trow, d, lds, acc); break;
      case 5: stream_rows<5, 2, 4>(wr, trow, d, lds, acc); break;
      case 6: stream_rows<6, 2, 4>(wr, trow, d, lds, acc); break;
      case 7: stream_rows<7, 2, 4>(wr, trow, d, lds, acc); break;
      default: stream_rows<8, 2, 4>(wr, trow, d, lds, acc); break;
    }
#pragma unroll
    for (int j = 0; j < FF_TG; ++j) {
      const int tk = pass + 16 * j + row;
      if (j < nt && tk < n) {
        uint16_t h[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) h[r] = f32_to_bf16(silu(acc[0][j][r]) * acc[1][j][r]);
        u32x2 pk = {(uint32_t)h[0] | ((uint32_t)h[1] << 16),
                    (uint32_t)h[2] | ((uint32_t)h[3] << 16)};
        *reinterpret_cast<u32x2 *>(H + (size_t)(p0 + tk) * I + i0 + 4 * (lane >> 4)) = pk;
      }
    }
  }
}

constexpr int DN_RT = 2;   // row tiles of W_d per wavefront in k_down

template <int Q>
__global__ __launch_bounds__(FF_WAVES * WAVE, 2)
void k_down_bf16(int d, int I, int E, const uint16_t *__restrict__ w2,
                 const int32_t *__restrict__ sel_ids,
                 const int32_t *__restrict__ n_sel_p,
                 const int32_t *__restrict__ offsets,
                 const float *__restrict__ pair_gate,
                 const uint16_t *__restrict__ H, float *__restrict__ pairbuf) {
  __shared__ __attribute__((aligned(1024))) char lds[FF_LDS];
  const int s = blockIdx.x;
  if (s >= *n_sel_p) return;
  const int u = sel_ids[s];
  if (u < 0 || u >= E) return;   // only for a plan not made by base_select
  const int p0 = offsets[s];
  const int n = offsets[s + 1] - p0;
  if (n <= 0) return;
  const int lane = lane_id(), row = lane & 15, kq = (lane >> 4) * 8;
  const int c0 = blockIdx.y * (16 * DN_RT * FF_WAVES) + wave_id() * 16 * DN_RT;
  const uint16_t *wr[DN_RT];
#pragma unroll
  for (int rt = 0; rt < DN_RT; ++rt)
    wr[rt] = w2 + ((size_t)u * d + c0 + 16 * rt + row) * I + kq;

  for (int pass = 0; pass < n; pass += 16 * FF_TG) {
    const int nt = min(FF_TG, (n - pass + 15) / 16);
    const uint16_t *trow[FF_TG];
    token_rows(H + (size_t)p0 * I, (size_t)I, nullptr, pass, n, trow);
    f32x4 acc[DN_RT][FF_TG];
#pragma unroll
    for (int j = 0; j < FF_TG; ++j)
#pragma unroll
      for (int rt = 0; rt < DN_RT; ++rt) acc[rt][j] = f32x4{0, 0, 0, 0};
    switch (nt) {
      case 1: stream_rows<1, DN_RT, Q>(wr, trow, I, lds, acc); break;
      case 2: stream_rows<2, DN_RT, Q>(wr, trow, I, lds, acc); break;
      case 3: stream_rows<3, DN_RT, Q>(wr, trow, I, lds, acc); break;
      case 4: stream_rows<4, DN_RT, Q>(wr, trow, I, lds, acc); break;
      case 5: stream_rows<5, DN_RT, Q>(wr, trow, I, lds, acc); break;
      case 6: stream_rows<6, DN_RT, Q>(wr, trow, I, lds, acc); break;
      case 7: stream_rows<7, DN_RT, Q>(wr, trow, I, lds, acc); break;
      default: stream_rows<8, DN_RT, Q>(wr, trow, I, lds, acc); break;
    }
#pragma unroll
    for (int j = 0; j < FF_TG; ++j) {
      const int tk = pass + 16 * j + row;
      if (j < nt && tk < n) {
        const float g = pair_gate[p0 + tk];
#pragma unroll
        for (int rt = 0; rt < DN_RT; ++rt) {
          float4 o = {g * acc[rt][j][0], g * acc[rt][j][1], g * acc[rt][j][2],
                      g * acc[rt][j][3]};
          *reinterpret_cast<float4 *>(pairbuf + (size_t)(p0 + tk) * d + c0 +
                                      16 * rt + 4 * (lane >> 4)) = o;
        }
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

hipError_t launch_gateup(bool bf16, const void *x, int d, int I, int E,
                         int budget, const void *w13, const int32_t *sel_ids,
                         const int32_t *n_sel, const int32_t *offsets,
                         const int32_t *pair_tok, void *H, hipStream_t st) {
  if (bf16)
    hipLaunchKernelGGL(k_gateup_bf16, dim3(budget, I / (16 * FF_WAVES)),
                       dim3(FF_WAVES * WAVE), 0, st, (const uint16_t *)x, d, I,
                       E, (const uint16_t *)w13, sel_ids, n_sel, offsets,
                       pair_tok, (uint16_t *)H);
  else
    hipLaunchKernelGGL(k_gateup_f32, dim3(budget, (I + F32_ROWS - 1) / F32_ROWS),
                       dim3(F32_ROWS * F32_TG), 0, st, (const float *)x, d, I,
                       E, (const float *)w13, sel_ids, n_sel, offsets, pair_tok,
                       (float *)H);
  return hipGetLastError();
}

hipError_t launch_down(bool bf16, int d, int I, int E, int budget,
                       const void *w2, const int32_t *sel_ids,
                       const int32_t *n_sel, const int32_t *offsets,
                       const float *pair_gate, const void *H, float *pairbuf,
                       hipStream_t st) {
  if (bf16)
    hipLaunchKernelGGL(I % 128 == 0 ? k_down_bf16<4> : k_down_bf16<2>,
                       dim3(budget, d / (16 * DN_RT * FF_WAVES)),
                       dim3(FF_WAVES * WAVE), 0, st, d, I, E,
                       (const uint16_t *)w2, sel_ids, n_sel, offsets, pair_gate,
                       (const uint16_t *)H, pairbuf);
  else
    hipLaunchKernelGGL(k_down_f32, dim3(budget, (d + F32_ROWS - 1) / F32_ROWS),
                       dim3(F32_ROWS * F32_TG), 0, st, d, I, E,
                       (const float *)w2, sel_ids, n_sel, offsets, pair_gate,
                       (const float *)H, pairbuf);
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
