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

constexpr int FF_WAVES = 1;      // wavefronts per workgroup
constexpr int N_XCD = 8;         // accelerator dies, one L2 each
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

// Token operands in fragment order.  The tokens of kept slot s occupy the
// 16-pair tiles tile_base[s] .. tile_base[s+1]-1 (tile i holds the slot's
// pairs 16 i' .. 16 i' + 15, i' = i - tile_base[s]; the last tile padded).
// For a contraction of `ks` k-steps a tile is ks fragments of 1 KiB:
// fragment (tile, k-step) = 64 lanes x 8 elements, lane l holding pair
// 16 i' + l % 16, elements 32 k-step + 8 (l / 16) .. +7.  So every operand
// load of the FFN reads one contiguous 1 KiB block.
//   xp: the hidden states of the pairs (contraction d), built by k_gather
//   hp: the SwiGLU activations (contraction I), written by k_gateup
// Padding rows are never written; they only meet discarded output columns.

// One wavefront per (tile, k-step): gather 1 KiB of hidden states.
__global__ __launch_bounds__(256)
void k_gather(const uint16_t *__restrict__ x, int d, int budget,
              const int32_t *__restrict__ n_sel_p,
              const int32_t *__restrict__ offsets,
              const int32_t *__restrict__ pair_tok,
              const int32_t *__restrict__ tile_base,
              uint16_t *__restrict__ xp) {
  const int ksteps = d / 32;
  const int v = blockIdx.x * (blockDim.x / WAVE) + wave_id();
  const int n_sel = min(max(*n_sel_p, 0), budget);
  const int tile = v / ksteps, ks = v % ksteps;
  if (tile >= tile_base[n_sel]) return;
  int lo = 0, hi = n_sel - 1;      // last slot with tile_base[s] <= tile
  while (lo < hi) {
    const int mid = (lo + hi + 1) / 2;
    if (tile_base[mid] <= tile) lo = mid; else hi = mid - 1;
  }
  const int s = lo, lane = lane_id();
  const int p = offsets[s] + 16 * (tile - tile_base[s]) + (lane & 15);
  u32x4 v4 = {0u, 0u, 0u, 0u};
  if (p < offsets[s + 1])
    v4 = *reinterpret_cast<const u32x4 *>(x + (size_t)pair_tok[p] * d + 32 * ks +
                                          8 * (lane >> 4));
  *reinterpret_cast<u32x4 *>(xp + (((size_t)tile * ksteps + ks) * WAVE + lane) * 8) = v4;
}

// Flat work assignment: wavefront v of the grid takes unit v of the list
// (slot s, row group g, token part ts) ordered by slot, then group, then
// part (a slot has parts = ceil(n_s / 64) token parts of 64 and `groups`
// row groups of 64 weight rows; part_base[s] is the prefix of parts).  The
// parts of one row group are neighbours, so they usually run in one
// workgroup on one CU and fetch the group's weights from HBM once.
struct Unit {
  int s, g, ts;
};

// The dispatcher deals the workgroups of a launch round-robin over the
// XCDs (workgroup b runs on XCD b % 8).  The unit list is cut into 8
// contiguous runs, run x for XCD x, so the units that read one slot's
// tokens or one row group's weights mostly share an L2.  Returns the unit
// of the calling wavefront, or -1.
__device__ __forceinline__ int xcd_unit(int units) {
  const int per = (units + N_XCD * FF_WAVES - 1) / (N_XCD * FF_WAVES);
  const int local = blockIdx.x / N_XCD;
  if (local >= per) return -1;
  // wave-uniform by construction; said so, so that every address derived
  // from it stays scalar (a buffer resource held in vector registers would
  // turn each load into a loop over the lanes)
  return __builtin_amdgcn_readfirstlane(((blockIdx.x % N_XCD) * per + local) * FF_WAVES +
                                        wave_id());
}

__device__ __forceinline__ bool find_unit(int groups, int n_sel,
                                          const int32_t *part_base, Unit &w) {
  const int v = xcd_unit(groups * part_base[n_sel]);
  if (v < 0 || v >= groups * part_base[n_sel]) return false;
  int lo = 0, hi = n_sel - 1;      // last slot with groups * part_base[s] <= v
  while (lo < hi) {
    const int mid = (lo + hi + 1) / 2;
    if (groups * part_base[mid] <= v) lo = mid; else hi = mid - 1;
  }
  const int parts = __builtin_amdgcn_readfirstlane(part_base[lo + 1] - part_base[lo]);
  const int r = v - groups * __builtin_amdgcn_readfirstlane(part_base[lo]);
  w.s = __builtin_amdgcn_readfirstlane(lo);
  w.g = r / parts;
  w.ts = r % parts;
  return true;
}

// Workgroups for up to `units` units: a multiple of N_XCD, so that every
// XCD's run of xcd_unit has all its workgroups.
inline unsigned ffn_grid(long long units) {
  const long long per = (units + N_XCD * FF_WAVES - 1) / (N_XCD * FF_WAVES);
  return (unsigned)(per * N_XCD);
}

// One wavefront: FF_RT row tiles against NT token tiles, `ksteps` k-steps
// of 32.  Token fragment (j, ks) at byte j * tstride + ks * 1024 + lane * 16
// of resource rt.  Weights and tokens are requested D k-steps ahead of
// their MFMAs, both at the same distance, so waiting for the oldest
// k-step's data never waits for anything requested after it.
template <int NT, int D, bool PACKED>
__device__ __forceinline__ void stream_wave(const WeightSrc &ws, rsrc_t rt,
                                            uint32_t tstride, int ksteps,
                                            f32x4 (&acc)[FF_RT][FF_NT]) {
  const uint32_t tl = lane_id() * 16;
  bf16x8 wb[D][FF_RT], xb[D][NT];
#pragma unroll
  for (int p = 0; p < D; ++p) {
#pragma unroll
    for (int t = 0; t < FF_RT; ++t) wb[p][t] = wload<PACKED>(ws, t, p);
#pragma unroll
    for (int j = 0; j < NT; ++j) xb[p][j] = bload(rt, tl + j * tstride, (uint32_t)p * 1024u);
  }
  int ks = 0;
  for (; ks + D < ksteps; ks += D) {
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
                                              uint32_t tstride, int ksteps,
                                              f32x4 (&acc)[FF_RT][FF_NT]) {
  if (ksteps % 4 == 0) stream_wave<NT, 4, PACKED>(ws, rt, tstride, ksteps, acc);
  else stream_wave<NT, 2, PACKED>(ws, rt, tstride, ksteps, acc);
}

template <bool PACKED>
__device__ __forceinline__ void stream_wave_nt(int nt, const WeightSrc &ws, rsrc_t rt,
                                               uint32_t tstride, int ksteps,
                                               f32x4 (&acc)[FF_RT][FF_NT]) {
  switch (nt) {
    case 1: stream_wave_d<1, PACKED>(ws, rt, tstride, ksteps, acc); break;
    case 2: stream_wave_d<2, PACKED>(ws, rt, tstride, ksteps, acc); break;
    case 3: stream_wave_d<3, PACKED>(ws, rt, tstride, ksteps, acc); break;
    default: stream_wave_d<4, PACKED>(ws, rt, tstride, ksteps, acc); break;
  }
}

__device__ __forceinline__ void zero_acc(f32x4 (&acc)[FF_RT][FF_NT]) {
#pragma unroll
  for (int t = 0; t < FF_RT; ++t)
#pragma unroll
    for (int j = 0; j < FF_NT; ++j) acc[t][j] = f32x4{0, 0, 0, 0};
}

// gate/up: row group g = gate rows 32 g .. 32 g + 31 (tiles 0, 1) and up
// rows I + 32 g .. I + 32 g + 31 (tiles 2, 3).  Writes H in fragment order:
// SwiGLU column i = 32 g + 16 t + 4 (l / 16) + r of pair tk sits in
// fragment (tile of tk, k-step g), lane tk % 16 + 16 (2 t + (l / 16) / 2),
// element 4 ((l / 16) % 2) + r.
template <bool PACKED>
__global__ __launch_bounds__(FF_WAVES * WAVE, 2)
void k_gateup_bf16(int d, int I, int E, int budget, const uint16_t *__restrict__ w13,
                   const int32_t *__restrict__ sel_ids,
                   const int32_t *__restrict__ n_sel_p,
                   const int32_t *__restrict__ offsets,
                   const int32_t *__restrict__ tile_base,
                   const int32_t *__restrict__ part_base,
                   const uint16_t *__restrict__ xp, uint16_t *__restrict__ hp) {
  const int groups = I / 32;
  const int n_sel = min(max(*n_sel_p, 0), budget);
  Unit un;
  if (!find_unit(groups, n_sel, part_base, un)) return;
  const int u = __builtin_amdgcn_readfirstlane(sel_ids[un.s]);
  if (u < 0 || u >= E) return;   // only for a plan not made by base_select
  const int n = __builtin_amdgcn_readfirstlane(offsets[un.s + 1] - offsets[un.s]);
  const int tbeg = FF_TOK * un.ts;
  const int nt = min(FF_NT, (n - tbeg + 15) / 16);
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
  const int tile0 = __builtin_amdgcn_readfirstlane(tile_base[un.s]) + tbeg / 16;
  const uint32_t tstride = (uint32_t)(d / 32) * 1024u;        // one tile
  const rsrc_t rt = make_rsrc(xp + (size_t)tile0 * (d / 32) * 512, (uint32_t)nt * tstride);
  f32x4 acc[FF_RT][FF_NT];
  zero_acc(acc);
  stream_wave_nt<PACKED>(nt, ws, rt, tstride, d / 32, acc);
#pragma unroll
  for (int j = 0; j < FF_NT; ++j) {
    const int tk = tbeg + 16 * j + row;
    if (j < nt && tk < n) {
      uint16_t *frag = hp + (((size_t)(tile0 + j) * (I / 32) + g) * WAVE) * 8;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        uint16_t h[4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
          h[r] = f32_to_bf16(silu(acc[t][j][r]) * acc[t + 2][j][r]);
        u32x2 pk = {(uint32_t)h[0] | ((uint32_t)h[1] << 16),
                    (uint32_t)h[2] | ((uint32_t)h[3] << 16)};
        const int l2 = row + 16 * (2 * t + (lane >> 5));
        *reinterpret_cast<u32x2 *>(frag + l2 * 8 + 4 * ((lane >> 4) & 1)) = pk;
      }
    }
  }
}

// down: row group g = rows 64 g .. 64 g + 63 of W_d (tiles 0..3); tokens
// are the SwiGLU activations in fragment order.
template <bool PACKED>
__global__ __launch_bounds__(FF_WAVES * WAVE, 2)
void k_down_bf16(int d, int I, int E, int budget, const uint16_t *__restrict__ w2,
                 const int32_t *__restrict__ sel_ids,
                 const int32_t *__restrict__ n_sel_p,
                 const int32_t *__restrict__ offsets,
                 const int32_t *__restrict__ tile_base,
                 const int32_t *__restrict__ part_base,
                 const float *__restrict__ pair_gate,
                 const uint16_t *__restrict__ hp, float *__restrict__ pairbuf) {
  const int groups = d / 64;
  const int n_sel = min(max(*n_sel_p, 0), budget);
  Unit un;
  if (!find_unit(groups, n_sel, part_base, un)) return;
  const int u = __builtin_amdgcn_readfirstlane(sel_ids[un.s]);
  if (u < 0 || u >= E) return;   // only for a plan not made by base_select
  const int p0 = __builtin_amdgcn_readfirstlane(offsets[un.s]);
  const int n = __builtin_amdgcn_readfirstlane(offsets[un.s + 1]) - p0;
  const int tbeg = FF_TOK * un.ts;
  const int nt = min(FF_NT, (n - tbeg + 15) / 16);
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
  const int tile0 = __builtin_amdgcn_readfirstlane(tile_base[un.s]) + tbeg / 16;
  const uint32_t tstride = (uint32_t)(I / 32) * 1024u;
  const rsrc_t rt = make_rsrc(hp + (size_t)tile0 * (I / 32) * 512, (uint32_t)nt * tstride);
  f32x4 acc[FF_RT][FF_NT];
  zero_acc(acc);
  stream_wave_nt<PACKED>(nt, ws, rt, tstride, I / 32, acc);
#pragma unroll
  for (int j = 0; j < FF_NT; ++j) {
    const int tk = tbeg + 16 * j + row;
    if (j < nt && tk < n) {
      const float gt = pair_gate[p0 + tk];
#pragma unroll
      for (int t = 0; t < FF_RT; ++t) {
        float4 o = {gt * acc[t][j][0], gt * acc[t][j][1], gt * acc[t][j][2],
                    gt * acc[t][j][3]};
        *reinterpret_cast<float4 *>(pairbuf + (size_t)(p0 + tk) * d + 64 * g + 16 * t +
                                    4 * (lane >> 4)) = o;
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

hipError_t launch_gather(const void *x, int B, int d, int K, int budget,
                         const int32_t *n_sel, const int32_t *offsets,
                         const int32_t *pair_tok, const int32_t *tile_base,
                         void *xp, hipStream_t st) {
  const long long waves = (long long)ffn_max_tiles(B, K, budget) * (d / 32);
  hipLaunchKernelGGL(k_gather, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, st,
                     (const uint16_t *)x, d, budget, n_sel, offsets, pair_tok,
                     tile_base, (uint16_t *)xp);
  return hipGetLastError();
}

hipError_t launch_gateup(bool bf16, bool packed, const void *x, int B, int d,
                         int I, int E, int K, int budget, const void *w13,
                         const int32_t *sel_ids, const int32_t *n_sel,
                         const int32_t *offsets, const int32_t *pair_tok,
                         const int32_t *tile_base, const int32_t *part_base,
                         const void *xp, void *H, hipStream_t st) {
  if (bf16) {
    const long long units = (long long)ffn_max_parts(B, K, budget) * (I / 32);
    hipLaunchKernelGGL(packed ? k_gateup_bf16<true> : k_gateup_bf16<false>,
                       dim3(ffn_grid(units)),
                       dim3(FF_WAVES * WAVE), 0, st, d, I, E, budget,
                       (const uint16_t *)w13, sel_ids, n_sel, offsets, tile_base,
                       part_base, (const uint16_t *)xp, (uint16_t *)H);
  } else {
    hipLaunchKernelGGL(k_gateup_f32, dim3(budget, (I + F32_ROWS - 1) / F32_ROWS),
                       dim3(F32_ROWS * F32_TG), 0, st, (const float *)x, d, I,
                       E, (const float *)w13, sel_ids, n_sel, offsets, pair_tok,
                       (float *)H);
  }
  return hipGetLastError();
}

hipError_t launch_down(bool bf16, bool packed, int B, int d, int I, int E, int K,
                       int budget, const void *w2, const int32_t *sel_ids,
                       const int32_t *n_sel, const int32_t *offsets,
                       const int32_t *tile_base, const int32_t *part_base,
                       const float *pair_gate, const void *H, float *pairbuf,
                       hipStream_t st) {
  if (bf16) {
    const long long units = (long long)ffn_max_parts(B, K, budget) * (d / 64);
    hipLaunchKernelGGL(packed ? k_down_bf16<true> : k_down_bf16<false>,
                       dim3(ffn_grid(units)),
                       dim3(FF_WAVES * WAVE), 0, st, d, I, E, budget,
                       (const uint16_t *)w2, sel_ids, n_sel, offsets, tile_base,
                       part_base, pair_gate, (const uint16_t *)H, pairbuf);
  } else {
    hipLaunchKernelGGL(k_down_f32, dim3(budget, (d + F32_ROWS - 1) / F32_ROWS),
                       dim3(F32_ROWS * F32_TG), 0, st, d, I, E,
                       (const float *)w2, sel_ids, n_sel, offsets, pair_gate,
                       (const float *)H, pairbuf);
  }
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
