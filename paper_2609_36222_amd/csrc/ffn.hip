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
// k_combine: y_t = residual_t + sum_j pairbuf[pair_of[t][j]] in j order
//   (the K routed ranks, then the shared experts).
//
// MFMA operand layout used here (v_mfma_f32_16x16x32_bf16): lane l supplies
// row (l % 16) of A and column (l % 16) of B with the 8 contraction
// elements 8*(l/16) .. 8*(l/16)+7 of a 32-wide k step; the result holds
// D[4*(l/16) + r][l % 16] in register r.
#include "common.hpp"
#include "internal.hpp"

namespace basek {

constexpr int GU_SPLIT = 4;      // gate/up: wavefronts per workgroup = contraction shares
constexpr int DN_SPLIT = 1;      // down: one wavefront per unit
constexpr int FF_RT = 4;         // 16-row weight tiles per wavefront
constexpr int FF_NT = 4;         // 16-token tiles per wavefront (64 tokens)
constexpr int FF_TOK = 16 * FF_NT;
static_assert(FF_TOK == FFN_PART, "FFN token part");

__device__ __forceinline__ bf16x8 ld_bf16x8(const uint16_t *p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Buffer loads: a wave-uniform resource (base, size) in scalar registers,
// a 32-bit per-lane offset, a uniform scalar offset and an immediate.  Reads
// past the resource's size return zero instead of touching memory.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int RSRC_CFG = 0x00020000;

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes, RSRC_CFG);
}

__device__ __forceinline__ bf16x8 bload(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(bf16x8,
                            __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0));
}

// The weight operand of one wavefront: FF_RT tiles of 16 rows.
//  packed:    one resource over the row group's stream; tile t of k-step ks
//             at lane * 16 + t * 1024 + ks * 4096 bytes
//  row-major: one resource per tile (its 16 rows); k-step ks of lane l at
//             (l % 16) * rowbytes + (l / 16) * 16 + ks * 64 bytes
struct WeightSrc {
  rsrc_t r[FF_RT];
  uint32_t voff;
};

template <bool PACKED>
__device__ __forceinline__ bf16x8 wload(const WeightSrc &w, int t, int ks) {
  if (PACKED) return bload(w.r[0], w.voff + t * 1024, (uint32_t)ks * 4096u);
  return bload(w.r[t], w.voff, (uint32_t)ks * 64u);
}

// Token operands in fragment order.  The pairs of kept slot s occupy
// consecutive 16-pair tiles (its i-th tile holds its pairs 16 i .. 16 i +
// 15, the last one padded); a part's tiles start at its tile0.
// For a contraction of `ks` k-steps a tile is ks fragments of 1 KiB:
// fragment (tile, k-step) = 64 lanes x 8 elements, lane l holding pair
// 16 i' + l % 16, elements 32 k-step + 8 (l / 16) .. +7.  So every operand
// load of the FFN reads one contiguous 1 KiB block.
//   xp: the hidden states of the pairs (contraction d), written by the
//       compaction launch (k_compact)
//   hp: the SwiGLU activations (contraction I), written by k_gateup
// Padding rows are never written; they only meet discarded output columns.

// Work units: one per workgroup, unit b of a launch at units[b], written by
// the compaction launch (see k_compact for their order and their XCD runs).
// A gate/up unit is (slot, row group of 32 gate + 32 up rows, 64-token
// part), a down unit (slot, row group of 64 rows of d, part); the
// workgroup's wavefronts (GU_SPLIT, DN_SPLIT) each take an equal share of
// the contraction and their partial sums are added through LDS in a fixed
// order.
struct Unit {
  int u, p0, n, tile0, g;
};

// Every value here is uniform over the workgroup, and is said to be so
// (readfirstlane), so that the addresses derived from it stay in scalar
// registers: a buffer resource held in vector registers would turn each
// load into a loop over the lanes.
__device__ __forceinline__ bool load_unit(const UnitRec *units, Unit &w) {
  const UnitRec r = units[blockIdx.x];
  w.u = __builtin_amdgcn_readfirstlane(r.u);
  w.g = __builtin_amdgcn_readfirstlane(r.g);
  w.p0 = __builtin_amdgcn_readfirstlane(r.p0);
  w.n = __builtin_amdgcn_readfirstlane(r.n);
  w.tile0 = __builtin_amdgcn_readfirstlane(r.tile0);
  return w.u >= 0;
}

// One wavefront: FF_RT row tiles against NT token tiles over k-steps
// k0 .. k0 + cnt - 1 (cnt a multiple of D).  Token fragment (j, ks) at
// byte j * tstride + ks * 1024 + lane * 16 of resource rt.  Weights and
// tokens are requested D k-steps ahead of their MFMAs, both at the same
// distance: loads complete in issue order, so waiting for the oldest
// k-step's data never waits for anything requested after it.
template <int NT, int D, bool PACKED>
__device__ __forceinline__ void stream_wave(const WeightSrc &ws, rsrc_t rt,
                                            uint32_t tstride, int k0, int cnt,
                                            f32x4 (&acc)[FF_RT][FF_NT]) {
  const uint32_t tl = lane_id() * 16;
  const int kend = k0 + cnt;
  bf16x8 wb[D][FF_RT], xb[D][NT];
#pragma unroll
  for (int p = 0; p < D; ++p) {
#pragma unroll
    for (int t = 0; t < FF_RT; ++t) wb[p][t] = wload<PACKED>(ws, t, k0 + p);
#pragma unroll
    for (int j = 0; j < NT; ++j)
      xb[p][j] = bload(rt, tl + j * tstride, (uint32_t)(k0 + p) * 1024u);
  }
  int ks = k0;
  for (; ks + D < kend; ks += D) {
#pragma unroll
    for (int p = 0; p < D; ++p) {
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int t = 0; t < FF_RT; ++t) acc[t][j] = mfma16(wb[p][t], xb[p][j], acc[t][j]);
      const int kn = ks + D + p;
#pragma unroll
      for (int t = 0; t < FF_RT; ++t) wb[p][t] = wload<PACKED>(ws, t, kn);
#pragma unroll
      for (int j = 0; j < NT; ++j) xb[p][j] = bload(rt, tl + j * tstride, (uint32_t)kn * 1024u);
      // keep this k-step's refill here: sunk to the end of the loop, the
      // refills of all D k-steps would wait for nearly every load in flight
      __builtin_amdgcn_sched_barrier(0);
    }
  }
#pragma unroll
  for (int p = 0; p < D; ++p)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int t = 0; t < FF_RT; ++t) acc[t][j] = mfma16(wb[p][t], xb[p][j], acc[t][j]);
}

template <int NT, bool PACKED>
__device__ __forceinline__ void stream_wave_d(const WeightSrc &ws, rsrc_t rt,
                                              uint32_t tstride, int k0, int cnt,
                                              f32x4 (&acc)[FF_RT][FF_NT]) {
  if (cnt % 4 == 0) stream_wave<NT, 4, PACKED>(ws, rt, tstride, k0, cnt, acc);
  else if (cnt % 2 == 0) stream_wave<NT, 2, PACKED>(ws, rt, tstride, k0, cnt, acc);
  else stream_wave<NT, 1, PACKED>(ws, rt, tstride, k0, cnt, acc);
}

// This wavefront's share of a unit's contraction (ksteps k-steps of 32)
// when S wavefronts split it: k-steps [w ksteps / S, (w + 1) ksteps / S);
// possibly empty.
template <int S, bool PACKED>
__device__ __forceinline__ void stream_share(int nt, const WeightSrc &ws, rsrc_t rt,
                                             uint32_t tstride, int ksteps,
                                             f32x4 (&acc)[FF_RT][FF_NT]) {
#pragma unroll
  for (int t = 0; t < FF_RT; ++t)
#pragma unroll
    for (int j = 0; j < FF_NT; ++j) acc[t][j] = f32x4{0, 0, 0, 0};
  const int w = wave_id();
  const int k0 = __builtin_amdgcn_readfirstlane(ksteps * w / S);
  const int cnt = __builtin_amdgcn_readfirstlane(ksteps * (w + 1) / S) - k0;
  if (cnt <= 0) return;
  switch (nt) {
    case 1: stream_wave_d<1, PACKED>(ws, rt, tstride, k0, cnt, acc); break;
    case 2: stream_wave_d<2, PACKED>(ws, rt, tstride, k0, cnt, acc); break;
    case 3: stream_wave_d<3, PACKED>(ws, rt, tstride, k0, cnt, acc); break;
    default: stream_wave_d<4, PACKED>(ws, rt, tstride, k0, cnt, acc); break;
  }
}

// Partial sums of the S wavefronts: [wave][row tile][token tile][lane]
template <int S>
struct Partials {
  f32x4 v[S][FF_RT][FF_NT][WAVE];
};

// The gate/up exchange as a reduce-scatter: wavefront W finishes gate tile
// W % 2 with its up tile for the token tiles j = W / 2 (mod 2); it keeps
// those partial sums in registers and writes only the other twelve tiles.
// Every sum still runs over the wavefronts in order 0 .. 3.
template <int W>
__device__ __forceinline__ bool rs_own(int t, int j) {
  return (t % 2) == (W % 2) && (j % 2) == (W / 2);
}
template <int W>
__device__ __forceinline__ void put_partials_rs(Partials<GU_SPLIT> &sh, int nt,
                                                const f32x4 (&acc)[FF_RT][FF_NT]) {
  const int l = lane_id();
#pragma unroll
  for (int t = 0; t < FF_RT; ++t)
#pragma unroll
    for (int j = 0; j < FF_NT; ++j)
      if (j < nt && !rs_own<W>(t, j)) sh.v[W][t][j][l] = acc[t][j];
}
template <int W>
__device__ __forceinline__ f32x4 sum_rs(const Partials<GU_SPLIT> &sh, const f32x4 &own,
                                        int t, int j) {
  const int l = lane_id();
  f32x4 r = W == 0 ? own : sh.v[0][t][j][l];
#pragma unroll
  for (int w = 1; w < GU_SPLIT; ++w) r += (w == W) ? own : sh.v[w][t][j][l];
  return r;
}
template <int W>
__device__ __forceinline__ void gu_epilogue(const Partials<GU_SPLIT> &sh,
                                            const f32x4 (&acc)[FF_RT][FF_NT], int nt, int n,
                                            int I, int g, int tile0, uint16_t *hp) {
  const int lane = lane_id(), row = lane & 15;
  constexpr int t = W % 2;
#pragma unroll
  for (int jj = 0; jj < FF_NT * 2 / GU_SPLIT; ++jj) {
    const int j = W / 2 + (GU_SPLIT / 2) * jj;
    const int tk = 16 * j + row;
    if (j < nt && tk < n) {
      const f32x4 ga = sum_rs<W>(sh, acc[t][j], t, j), up = sum_rs<W>(sh, acc[t + 2][j], t + 2, j);
      uint16_t h[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) h[r] = f32_to_bf16(silu_bf16(ga[r]) * up[r]);
      u32x2 pk = {(uint32_t)h[0] | ((uint32_t)h[1] << 16),
                  (uint32_t)h[2] | ((uint32_t)h[3] << 16)};
      uint16_t *frag = hp + (((size_t)(tile0 + j) * (I / 32) + g) * WAVE) * 8;
      const int l2 = row + 16 * (2 * t + (lane >> 5));
      *reinterpret_cast<u32x2 *>(frag + l2 * 8 + 4 * ((lane >> 4) & 1)) = pk;
    }
  }
}

// gate/up: row group g = gate rows 32 g .. 32 g + 31 (tiles 0, 1) and up
// rows I + 32 g .. I + 32 g + 31 (tiles 2, 3).  Writes H in fragment order:
// SwiGLU column i = 32 g + 16 t + 4 (l / 16) + r of pair tk sits in
// fragment (tile of tk, k-step g), lane tk % 16 + 16 (2 t + (l / 16) / 2),
// element 4 ((l / 16) % 2) + r.  After the partial sums are exchanged,
// every wavefront finishes a share of the (gate tile, token tile) pairs.
template <bool PACKED>
__global__ __launch_bounds__(GU_SPLIT * WAVE, 2)
void k_gateup_bf16(int d, int I, int E, int ns, const uint16_t *__restrict__ w13r,
                   const uint16_t *__restrict__ w13s,
                   const UnitRec *__restrict__ units,
                   const uint16_t *__restrict__ xp, uint16_t *__restrict__ hp) {
  __shared__ Partials<GU_SPLIT> sh;
  const int groups = I / 32;
  Unit un;
  if (!load_unit(units, un)) return;
  if (un.u < 0 || un.u >= E + ns) return;   // only for a plan not made by base_select
  // experts E .. E + ns - 1 are the shared ones
  const uint16_t *w13 = un.u < E ? w13r : w13s;
  const int u = un.u < E ? un.u : un.u - E, n = un.n, tile0 = un.tile0;
  const int nt = (n + 15) / 16;
  const int lane = lane_id(), row = lane & 15, g = un.g;
  WeightSrc ws;
  if (PACKED) {
    const uint32_t bytes = (uint32_t)(d / 32) * 4096u;
    ws.r[0] = make_rsrc(w13 + ((size_t)u * groups + g) * (size_t)bytes / 2, bytes);
    ws.voff = lane * 16;
  } else {
#pragma unroll
    for (int t = 0; t < FF_RT; ++t)
      ws.r[t] = make_rsrc(w13 + ((size_t)u * 2 * I + (t < 2 ? 0 : I) + 32 * g + 16 * (t & 1)) * d,
                          (uint32_t)(16 * d * 2));
    ws.voff = (uint32_t)row * (uint32_t)(d * 2) + (uint32_t)(lane >> 4) * 16u;
  }
  const uint32_t tstride = (uint32_t)(d / 32) * 1024u;        // one tile
  const rsrc_t rt = make_rsrc(xp + (size_t)tile0 * (d / 32) * 512, (uint32_t)nt * tstride);
  f32x4 acc[FF_RT][FF_NT];
  stream_share<GU_SPLIT, PACKED>(nt, ws, rt, tstride, d / 32, acc);
  // the SwiGLU of the 2 gate tiles x FF_NT token tiles, spread over the
  // wavefronts (template argument: the wavefront, so that the tiles it
  // keeps are fixed registers)
  static_assert(GU_SPLIT == 4, "reduce-scatter exchange");
  switch (wave_id()) {
    case 0: put_partials_rs<0>(sh, nt, acc); break;
    case 1: put_partials_rs<1>(sh, nt, acc); break;
    case 2: put_partials_rs<2>(sh, nt, acc); break;
    default: put_partials_rs<3>(sh, nt, acc); break;
  }
  __syncthreads();
  switch (wave_id()) {
    case 0: gu_epilogue<0>(sh, acc, nt, n, I, g, tile0, hp); break;
    case 1: gu_epilogue<1>(sh, acc, nt, n, I, g, tile0, hp); break;
    case 2: gu_epilogue<2>(sh, acc, nt, n, I, g, tile0, hp); break;
    default: gu_epilogue<3>(sh, acc, nt, n, I, g, tile0, hp); break;
  }
}

// down: row group g = rows 64 g .. 64 g + 63 of W_d (tiles 0..3); tokens
// are the SwiGLU activations in fragment order.  One wavefront per unit.
template <bool PACKED>
__global__ __launch_bounds__(DN_SPLIT * WAVE, 2)
void k_down_bf16(int d, int I, int E, int ns, const uint16_t *__restrict__ w2r,
                 const uint16_t *__restrict__ w2s,
                 const UnitRec *__restrict__ units,
                 const float *__restrict__ pair_gate,
                 const uint16_t *__restrict__ hp, float *__restrict__ pairbuf) {
  static_assert(DN_SPLIT == 1, "the down epilogue takes the accumulators as they are");
  const int groups = d / 64;
  Unit un;
  if (!load_unit(units, un)) return;
  if (un.u < 0 || un.u >= E + ns) return;   // only for a plan not made by base_select
  const uint16_t *w2 = un.u < E ? w2r : w2s;
  const int u = un.u < E ? un.u : un.u - E, n = un.n, tile0 = un.tile0, p0 = un.p0;
  const int nt = (n + 15) / 16;
  const int lane = lane_id(), row = lane & 15, g = un.g;
  WeightSrc ws;
  if (PACKED) {
    const uint32_t bytes = (uint32_t)(I / 32) * 4096u;
    ws.r[0] = make_rsrc(w2 + ((size_t)u * groups + g) * (size_t)bytes / 2, bytes);
    ws.voff = lane * 16;
  } else {
#pragma unroll
    for (int t = 0; t < FF_RT; ++t)
      ws.r[t] = make_rsrc(w2 + ((size_t)u * d + 64 * g + 16 * t) * I, (uint32_t)(16 * I * 2));
    ws.voff = (uint32_t)row * (uint32_t)(I * 2) + (uint32_t)(lane >> 4) * 16u;
  }
  // the gates first: loaded after the contraction, each would sit behind
  // the previous tile's stores in the memory counter
  float gt[FF_NT];
#pragma unroll
  for (int j = 0; j < FF_NT; ++j) gt[j] = pair_gate[p0 + min(16 * j + row, n - 1)];
  const uint32_t tstride = (uint32_t)(I / 32) * 1024u;
  const rsrc_t rt = make_rsrc(hp + (size_t)tile0 * (I / 32) * 512, (uint32_t)nt * tstride);
  f32x4 acc[FF_RT][FF_NT];
  stream_share<DN_SPLIT, PACKED>(nt, ws, rt, tstride, I / 32, acc);
  // one wavefront per unit: its accumulators are the sums
#pragma unroll
  for (int t = 0; t < FF_RT; ++t)
#pragma unroll
  for (int j = 0; j < FF_NT; ++j) {
    const int tk = 16 * j + row;
    if (j < nt && tk < n) {
      const f32x4 o = acc[t][j];
      float4 v = {gt[j] * o[0], gt[j] * o[1], gt[j] * o[2], gt[j] * o[3]};
      *reinterpret_cast<float4 *>(pairbuf + (size_t)(p0 + tk) * d + 64 * g + 16 * t +
                                  4 * (lane >> 4)) = v;
    }
  }
}

// fp32 experts (small layers): one wavefront per (kept slot, output row).
// The lanes split the contraction (lane l takes elements l, l + 64, ..., so
// every load of a row is contiguous across the wavefront) and each token's
// dot product is summed across the lanes by the butterfly of
// wave_tree_sum.  The slot's tokens are taken one after another; the row
// stays in L1 between them.
constexpr int F32_WAVES = 4;   // rows per workgroup

__global__ __launch_bounds__(F32_WAVES * WAVE)
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
  const int i = blockIdx.y * F32_WAVES + wave_id(), lane = lane_id();
  if (i >= I) return;
  const float *wg = w13 + ((size_t)u * 2 * I + i) * d;
  const float *wu = w13 + ((size_t)u * 2 * I + I + i) * d;
  for (int tk = 0; tk < n; ++tk) {
    const float *xr = x + (size_t)pair_tok[p0 + tk] * d;
    float g = 0.0f, v = 0.0f;
    for (int k = lane; k < d; k += WAVE) {
      const float xv = xr[k];
      g = __builtin_fmaf(xv, wg[k], g);
      v = __builtin_fmaf(xv, wu[k], v);
    }
    g = wave_tree_sum(g);
    v = wave_tree_sum(v);
    if (lane == 0) H[(size_t)(p0 + tk) * I + i] = silu(g) * v;
  }
}

__global__ __launch_bounds__(F32_WAVES * WAVE)
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
  const int c = blockIdx.y * F32_WAVES + wave_id(), lane = lane_id();
  if (c >= d) return;
  const float *wd = w2 + ((size_t)u * d + c) * I;
  for (int tk = 0; tk < n; ++tk) {
    const float *hr = H + (size_t)(p0 + tk) * I;
    float o = 0.0f;
    for (int k = lane; k < I; k += WAVE) o = __builtin_fmaf(hr[k], wd[k], o);
    o = wave_tree_sum(o);
    if (lane == 0) pairbuf[(size_t)(p0 + tk) * d + c] = pair_gate[p0 + tk] * o;
  }
}

constexpr int CB_THREADS = 256;
constexpr int CB_GROUP = 4;   // ranks whose rows are in flight together

template <bool BF16>
__global__ __launch_bounds__(CB_THREADS)
void k_combine(int B, int d, int kc, const int32_t *__restrict__ pair_of,
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
  // CB_GROUP ranks at a time: their pair indices, then their rows, all
  // requested before the first is added (the adds stay in rank order)
  for (int j0 = 0; j0 < kc; j0 += CB_GROUP) {
    int p[CB_GROUP];
#pragma unroll
    for (int i = 0; i < CB_GROUP; ++i)
      p[i] = (j0 + i < kc) ? pair_of[(size_t)t * kc + j0 + i] : -1;
    float4 v[CB_GROUP];
#pragma unroll
    for (int i = 0; i < CB_GROUP; ++i)
      if (p[i] >= 0) v[i] = *reinterpret_cast<const float4 *>(pairbuf + (size_t)p[i] * d + c);
#pragma unroll
    for (int i = 0; i < CB_GROUP; ++i) {
      if (p[i] < 0) continue;   // a routed rank the token does not execute
      acc[0] = acc[0] + v[i].x; acc[1] = acc[1] + v[i].y;
      acc[2] = acc[2] + v[i].z; acc[3] = acc[3] + v[i].w;
    }
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

hipError_t launch_gateup(bool bf16, bool packed, const void *x, int B, int d,
                         int I, int E, int K, int budget, int ns, const void *w13,
                         const void *w13s, const int32_t *sel_ids, const int32_t *n_sel,
                         const int32_t *offsets, const int32_t *pair_tok,
                         const UnitRec *units, const void *xp, void *H, hipStream_t st) {
  if (bf16) {
    launch_k(packed ? k_gateup_bf16<true> : k_gateup_bf16<false>,
                       dim3(ffn_gu_blocks(B, K, budget, ns, I)), dim3(GU_SPLIT * WAVE), 0, st,
                       d, I, E, ns, (const uint16_t *)w13, (const uint16_t *)w13s, units,
                       (const uint16_t *)xp, (uint16_t *)H);
  } else {
    launch_k(k_gateup_f32, dim3(budget, (I + F32_WAVES - 1) / F32_WAVES),
                       dim3(F32_WAVES * WAVE), 0, st, (const float *)x, d, I,
                       E, (const float *)w13, sel_ids, n_sel, offsets, pair_tok,
                       (float *)H);
  }
  return hipGetLastError();
}

hipError_t launch_down(bool bf16, bool packed, int B, int d, int I, int E, int K,
                       int budget, int ns, const void *w2, const void *w2s,
                       const int32_t *sel_ids,
                       const int32_t *n_sel, const int32_t *offsets,
                       const UnitRec *units, const float *pair_gate, const void *H,
                       float *pairbuf, hipStream_t st) {
  if (bf16) {
    launch_k(packed ? k_down_bf16<true> : k_down_bf16<false>,
                       dim3(ffn_dn_blocks(B, K, budget, ns, d)), dim3(DN_SPLIT * WAVE), 0, st,
                       d, I, E, ns, (const uint16_t *)w2, (const uint16_t *)w2s, units,
                       pair_gate, (const uint16_t *)H, pairbuf);
  } else {
    launch_k(k_down_f32, dim3(budget, (d + F32_WAVES - 1) / F32_WAVES),
                       dim3(F32_WAVES * WAVE), 0, st, d, I, E,
                       (const float *)w2, sel_ids, n_sel, offsets, pair_gate,
                       (const float *)H, pairbuf);
  }
  return hipGetLastError();
}

hipError_t launch_combine(bool bf16, int B, int d, int kc,
                          const int32_t *pair_of, const float *pairbuf,
                          const void *residual, void *y, hipStream_t st) {
  dim3 grid(B, (d + CB_THREADS * 4 - 1) / (CB_THREADS * 4));
  if (bf16)
    launch_k(k_combine<true>, grid, dim3(CB_THREADS), 0, st, B, d, kc,
                       pair_of, pairbuf, residual, y);
  else
    launch_k(k_combine<false>, grid, dim3(CB_THREADS), 0, st, B, d, kc,
                       pair_of, pairbuf, residual, y);
  return hipGetLastError();
}

}  // namespace basek
