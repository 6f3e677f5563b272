// Grouped SwiGLU expert FFN over the kept experts only, and the combine
// (K3, K4, K5).  Sec. 3.5: tokens execute only experts of the kept set, so
// only those experts' weights are read; Sec. 3.1: y_t = sum_v g_{t,v} E_v(z_t)
// with E_v(z) = W_d (silu(W_g z) * (W_u z)).
//
// k_gateup_bf16 (part of a kept slot's pairs, row-pair tiles of I):
//   H[p][i] = bf16(silu(g) * u), g = x . W_g[i], u = x . W_u[i], fp32
//   accumulation on MFMA 16x16x32 bf16 (16 weight rows x 16 tokens x 32 k
//   per instruction, tokens padded to 16).
// k_down_bf16 (part, row tiles of d): pairbuf[p][c] = gate_p * (H[p] . W_d[c]).
// Each unit streams its weight rows once; see "Grouped bf16 FFN" below.
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

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Buffer loads: a wave-uniform resource (base, size) in scalar registers,
// a 32-bit per-lane offset and a uniform scalar offset.  Reads past the
// resource's size return zero without touching memory.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef __attribute__((address_space(3))) void *lds_ptr_t;
constexpr int RSRC_CFG = 0x00020000;
constexpr uint32_t OOB = 0x40000000u;   // a scalar offset past every resource used here

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes, RSRC_CFG);
}

__device__ __forceinline__ bf16x8 bload(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(bf16x8,
                            __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0));
}

// 16 bytes per lane from a buffer straight into LDS: lane l's bytes land at
// lds + 16 l (lds: uniform over the wavefront).  Counted by vmcnt like any
// buffer load; the compiler does not track these writes, so every reader
// waits for them explicitly (wait_vm, then a barrier).
__device__ __forceinline__ void load_lds(rsrc_t r, void *lds, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)lds, 16, voff, soff, 0, 0);
}

// Wait until at most N vector-memory operations of this wavefront are in
// flight (they complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

// ----------------------------------------------------------------------------
// Grouped bf16 FFN (K3, K4).  Work is cut by the compaction launch into
// parts: a kept (or shared) slot's pairs, as 16-pair tiles, split into parts
// of at most FFN_GU_PT (gate/up) or FFN_DN_PT (down) tiles of balanced size.
// A unit is (part, row group).  The launch's units are numbered slot by slot
// and, within a slot, row group by row group, and cut into one run of equal
// length per die (FfnUnit records and per-die headers, written by
// k_compact): a row group's weights are read through one L2 by all the parts
// that need them, and every die has the same number of units, whether the
// kept slots are many or few.  The units of die x are taken by the
// workgroups that run on die x (workgroup b runs on die b % N_XCD),
// workgroup b taking units b / N_XCD, b / N_XCD + gridDim.x / N_XCD, ... of
// its die's run.
//
// Inside a unit every wavefront owns its rows over the whole contraction (so
// it finishes its outputs alone, in one fixed order: k ascending), and the
// unit's token operand is shared: for each 32-wide k-step the part's token
// fragments (1 KiB each, fragment order, see below) are loaded once into an
// LDS ring of DT + 1 k-steps, DT k-steps ahead (FFN_GU_DT, FFN_DN_DT), by
// the wavefronts in turn; each wavefront requests its own weight fragments FFN_GU_DW or
// FFN_DN_DW k-steps ahead into registers.  Per k-step: wait for this wavefront's share of the
// k-step's token loads, meet the other wavefronts (the barrier also tells
// every wavefront that the ring slot about to be refilled has been read),
// read the fragments from LDS (gate/up: all of the step's at once, so that
// one LDS round trip per step is exposed, not one per tile; down: one ahead
// of the MFMAs), then request the next k-steps.  Waves without rows in a unit (a short last row group) read past
// their resource (zero, no memory access) and skip the MFMAs, but still take
// their share of the token loads.
//
// Token operands: the pairs of slot s occupy consecutive 16-pair tiles (its
// i-th tile holds its pairs 16 i .. 16 i + 15); the fragment of (tile,
// k-step) is 64 lanes x 8 elements, lane l holding pair 16 i' + l % 16,
// elements 32 k-step + 8 (l / 16) .. +7 -- the MFMA B-operand layout.
//   gate/up (contraction d): gathered from the hidden states x by a buffer
//       load per lane into the LDS ring, 64 contiguous bytes of a token row
//       per 16 lanes (x stays in L2: every kept expert's pairs read it);
//       padding rows read zero
//   hp: the SwiGLU activations (contraction I), written by k_gateup_bf16 in
//       fragment order (1 KiB per fragment, tile-major); its padding rows are
//       never written (they meet only the discarded output columns of
//       padding pairs)

// The weight operand of one wavefront: one 16-row tile (two for gate/up:
// the gate rows and their up rows).
//  packed:    one resource over the row group's stream; the tile's fragment
//             of k-step ks at lane * 16 + tile * 1024 + ks * 4096 bytes
//  row-major: one resource per tile (its 16 rows); k-step ks of lane l at
//             (l % 16) * rowbytes + (l / 16) * 16 + ks * 64 bytes
struct TileSrc {
  rsrc_t r0, r1;       // gate/up: gate tile, up tile; down: r0 only
  uint32_t v0, v1;     // lane offsets
  uint32_t kstride;    // bytes per k-step (4096 packed, 64 row-major)
};

__device__ __forceinline__ uint32_t ksoff(const TileSrc &s, int ks, int KS) {
  return ks < KS ? (uint32_t)ks * s.kstride : OOB;
}

// Every value here is uniform over the workgroup and is said to be so, so
// that the addresses derived from it stay in scalar registers (a buffer
// resource held in vector registers would turn each load into a loop).
struct PartU {
  int u, tile0, nt, p0, n, rg;
};
__device__ __forceinline__ PartU load_unit(const FfnUnit *p) {
  const FfnUnit r = *p;
  return {__builtin_amdgcn_readfirstlane(r.u), __builtin_amdgcn_readfirstlane(r.tile0),
          __builtin_amdgcn_readfirstlane(r.nt), __builtin_amdgcn_readfirstlane(r.p0),
          __builtin_amdgcn_readfirstlane(r.n), __builtin_amdgcn_readfirstlane(r.rg)};
}
// This workgroup's die's run of a unit table, [u0, u1), and its first unit
// and stride (workgroup b runs on die b % N_XCD).
struct Run {
  int k0, k1, step;
};
__device__ __forceinline__ Run die_run(const int32_t &u0, const int32_t &u1) {
  return {__builtin_amdgcn_readfirstlane(u0) + (int)(blockIdx.x / N_XCD),
          __builtin_amdgcn_readfirstlane(u1), (int)(gridDim.x / N_XCD)};
}

// One unit of gate/up: wavefront w owns row-pair tile r = rp0 + w (gate rows
// 16 r .. 16 r + 15 and their up rows I + 16 r ..), if w < nrp.  NT: the
// part's tile count.  The loop advances two k-steps at a time (a step: 64
// contraction elements, one 128-byte line of every token row).  The token
// fragments come straight from the hidden states (resource rx over x):
// wavefront w < NT loads tile w's pairs 0..7 (half 0) and 8..15 (half 1), one
// line each per step, lane l taking row l / 8 of its half and 16-byte
// segment (l % 8) ^ (l / 8) of the line (tv0, tv1: that row's byte offset
// in x plus 16 times the segment; past the part's pairs at least
// FFN_TOK_PAD, beyond rx: zero).  Lane l's bytes land at 16 l of the half's
// 1 KiB in the ring, so the fragment of k-step e (0, 1) of the step, lane m
// (pair n = m % 16, elements 8 (m / 16) ..), is read at half n / 8, position
// 8 (n % 8) + ((4 e + m / 16) ^ (n % 8)): the swizzle keeps the eight lanes
// of a read pass on distinct bank groups, and every token line is fetched
// whole by one load.  Writes H = bf16(silu(g) * u) in fragment order: column
// i = 16 r + 4 (l / 16) + q of pair tk sits in fragment (tile of tk, k-step
// r / 2), lane tk % 16 + 16 (2 (r % 2) + (l / 16) / 2), element
// 4 ((l / 16) % 2) + q.
template <int NT, bool PACKED>
__device__ __forceinline__ void gateup_unit(uint8_t *ring, uint8_t *dummy, int d, int I,
                                            const uint16_t *__restrict__ w13, const PartU &pt,
                                            int rp0, int nrp, rsrc_t rx, uint32_t tv0,
                                            uint32_t tv1, uint16_t *__restrict__ hp) {
  constexpr int W = FFN_WAVES, DW = FFN_GU_DW, DT = FFN_GU_DT;
  constexpr int SLOT = NT * 2048;       // one step's token lines in the ring
  constexpr int LPS = 6;                // loads per step and wavefront
  static_assert(NT <= W, "one token tile per wavefront");
  static_assert(DW % 2 == 0 && DT == DW / 2 + 1, "tokens requested before the step's weights");
  const int w = wave_id_u(), lane = lane_id();
  const int KS = d / 32, NS = KS / 2;
  const bool active = w < nrp;
  const int r = rp0 + (active ? w : 0);
  TileSrc ws;
  if (PACKED) {
    const uint32_t gbytes = (uint32_t)KS * 4096u;
    ws.r0 = make_rsrc(w13 + ((size_t)pt.u * (I / 32) + (r >> 1)) * (gbytes / 2),
                      active ? gbytes : 0u);
    ws.r1 = ws.r0;
    ws.v0 = lane * 16 + (r & 1) * 1024;
    ws.v1 = ws.v0 + 2048;
    ws.kstride = 4096;
  } else {
    const uint32_t tb = (uint32_t)(16 * d * 2);
    ws.r0 = make_rsrc(w13 + ((size_t)pt.u * 2 * I + 16 * r) * d, active ? tb : 0u);
    ws.r1 = make_rsrc(w13 + ((size_t)pt.u * 2 * I + I + 16 * r) * d, active ? tb : 0u);
    ws.v0 = ws.v1 = (uint32_t)(lane & 15) * (uint32_t)(d * 2) + (uint32_t)(lane >> 4) * 16u;
    ws.kstride = 64;
  }
  // the step offset goes into the lane offset, so that the range check
  // alone keeps every load inside x
  auto tok_load = [&](int st) {
    uint8_t *slot = ring + (st % (DT + 1)) * SLOT;
    const uint32_t o = (uint32_t)st * 128u;
    if (w < NT) {
      load_lds(rx, slot + w * 2048, st < NS ? tv0 + o : FFN_TOK_PAD, 0);
      load_lds(rx, slot + w * 2048 + 1024, st < NS ? tv1 + o : FFN_TOK_PAD, 0);
    } else {
      load_lds(rx, dummy + w * 1024, FFN_TOK_PAD, 0);
      load_lds(rx, dummy + w * 1024, FFN_TOK_PAD, 0);
    }
  };
  // this lane's fragment positions in a step's tile (k-step e = 0, 1)
  const int n = lane & 15, n8 = n & 7;
  const int rb0 = (n >> 3) * 1024 + (8 * n8 + ((lane >> 4) ^ n8)) * 16;
  const int rb1 = (n >> 3) * 1024 + (8 * n8 + ((4 + (lane >> 4)) ^ n8)) * 16;
  f32x4 ag[NT], au[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) { ag[j] = f32x4{0, 0, 0, 0}; au[j] = f32x4{0, 0, 0, 0}; }
  // Loads go out in groups, one per step: the token lines of step st + DT
  // (DT = DW / 2 + 1) and then the weights of step st + DW / 2.  A step's
  // tokens are thus requested one group before its weights, so the wait for
  // the weights (at most DW / 2 - 1 younger groups in flight) covers the
  // tokens too and never waits for weights still ahead; vmcnt counts in
  // issue order.  The prologue issues groups -DT .. -1 the same way.
  bf16x8 wg[DW], wu[DW];
#pragma unroll
  for (int j = 0; j < DT; ++j) {
    tok_load(j);
    if (j >= DT - DW / 2) {
      const int q = 2 * (j - (DT - DW / 2));
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        wg[q + e] = bload(ws.r0, ws.v0, ksoff(ws, q + e, KS));
        wu[q + e] = bload(ws.r1, ws.v1, ksoff(ws, q + e, KS));
      }
    }
  }
  for (int k0 = 0; k0 < KS; k0 += DW) {
#pragma unroll
    for (int p = 0; p < DW; p += 2) {
      const int ks = k0 + p, st = ks / 2;
      // this wavefront's loads of step st are done: at most the DW / 2 - 1
      // later groups are in flight; after the barrier the ring slot of step
      // st - 1 is free for the tokens of step st + DT (issued before the
      // MFMAs), and each k-step's weight registers are refilled as soon as
      // its MFMAs have read them
      wait_vm<(DW / 2 - 1) * LPS>();
      wg_barrier();
      __builtin_amdgcn_sched_barrier(0);
      tok_load(st + DT);
      __builtin_amdgcn_sched_barrier(0);
      const uint8_t *sb = ring + (st % (DT + 1)) * SLOT;
      // both k-steps' fragments of the step in one batch of LDS reads
      bf16x8 xf[2][NT];
      if (active) {
#pragma unroll
        for (int e = 0; e < 2; ++e)
#pragma unroll
          for (int j = 0; j < NT; ++j)
            xf[e][j] = *reinterpret_cast<const bf16x8 *>(sb + (e == 0 ? rb0 : rb1) + j * 2048);
      }
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        if (active) {
#pragma unroll
          for (int j = 0; j < NT; ++j) {
            ag[j] = mfma16(wg[p + e], xf[e][j], ag[j]);
            au[j] = mfma16(wu[p + e], xf[e][j], au[j]);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        wg[p + e] = bload(ws.r0, ws.v0, ksoff(ws, ks + e + DW, KS));
        wu[p + e] = bload(ws.r1, ws.v1, ksoff(ws, ks + e + DW, KS));
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  wait_vm<0>();
  if (!active) return;
  const int row = lane & 15, g = r >> 1, t = r & 1;
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int tk = 16 * j + row;
    if (tk < pt.n) {
      uint16_t h[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) h[q] = f32_to_bf16(silu_bf16(ag[j][q]) * au[j][q]);
      const u32x2 pk = {(uint32_t)h[0] | ((uint32_t)h[1] << 16),
                        (uint32_t)h[2] | ((uint32_t)h[3] << 16)};
      uint16_t *frag = hp + (((size_t)(pt.tile0 + j) * (I / 32) + g) * WAVE) * 8;
      const int l2 = row + 16 * (2 * t + (lane >> 5));
      *reinterpret_cast<u32x2 *>(frag + l2 * 8 + 4 * ((lane >> 4) & 1)) = pk;
    }
  }
}

// Down's token depth: FFN_DN_DT k-steps, or for the deeper instances one
// k-step beyond their weights.
constexpr int dn_token_depth(int dw) { return dw > FFN_DN_DW ? dw + 1 : FFN_DN_DT; }

// One unit of down: wavefront w owns row tile rt = rt0 + w (rows 16 rt ..
// 16 rt + 15 of W_d), if w < nrt; the tokens are the part's SwiGLU
// activations.  pairbuf[p][c] = gate_p * (H[p] . W_d[c]).
template <int NT, bool PACKED, int DW>
__device__ __forceinline__ void down_unit(uint8_t *ring, uint8_t *dummy, int d, int I,
                                          const uint16_t *__restrict__ w2, const PartU &pt,
                                          int rt0, int nrt, const float *__restrict__ pair_gate,
                                          const uint16_t *__restrict__ hp,
                                          float *__restrict__ pairbuf) {
  // the deeper instances request tokens one k-step before their weights
  constexpr bool TA = DW > FFN_DN_DW;
  constexpr int W = FFN_WAVES, DT = dn_token_depth(DW);
  constexpr int NTK = (NT + W - 1) / W;
  const int w = wave_id_u(), lane = lane_id();
  const int KS = I / 32;
  const bool active = w < nrt;
  const int rtile = rt0 + (active ? w : 0);
  TileSrc ws;
  if (PACKED) {
    const uint32_t gbytes = (uint32_t)KS * 4096u;
    ws.r0 = make_rsrc(w2 + ((size_t)pt.u * (d / 64) + (rtile >> 2)) * (gbytes / 2),
                      active ? gbytes : 0u);
    ws.v0 = lane * 16 + (rtile & 3) * 1024;
    ws.kstride = 4096;
  } else {
    ws.r0 = make_rsrc(w2 + ((size_t)pt.u * d + 16 * rtile) * I,
                      active ? (uint32_t)(16 * I * 2) : 0u);
    ws.v0 = (uint32_t)(lane & 15) * (uint32_t)(I * 2) + (uint32_t)(lane >> 4) * 16u;
    ws.kstride = 64;
  }
  ws.r1 = ws.r0;
  ws.v1 = ws.v0;
  const uint32_t tbytes = (uint32_t)KS * 1024u;
  const rsrc_t rt = make_rsrc(hp + (size_t)pt.tile0 * (tbytes / 2), (uint32_t)pt.nt * tbytes);
  const uint32_t vl = lane * 16;
  const int row = lane & 15;
  // the gates first: loaded after the contraction, each would wait behind
  // the previous tile's stores
  float gt[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) gt[j] = pair_gate[pt.p0 + min(16 * j + row, pt.n - 1)];
  auto tok_load = [&](int ks) {
    uint8_t *slot = ring + (ks % (DT + 1)) * (NT * 1024);
#pragma unroll
    for (int q = 0; q < NTK; ++q) {
      const int j = w + W * q;
      if (j < NT)
        load_lds(rt, slot + j * 1024, vl,
                 ks < KS ? (uint32_t)j * tbytes + (uint32_t)ks * 1024u : OOB);
      else
        load_lds(rt, dummy + w * 1024, vl, OOB);
    }
  };
  f32x4 acc[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) acc[j] = f32x4{0, 0, 0, 0};
  bf16x8 wb[DW];
  // token loads next, then the weights; the gate loads are older still, so
  // the first k-step's wait also covers them (their L2 round trip overlaps
  // the first weights' HBM one).  The deeper instances issue their loads in
  // groups as gate/up does (the tokens of k-step ks + DT, then the weights
  // of ks + DW, DT = DW + 1), so that the wait for a k-step's weights
  // covers that k-step's tokens and leaves the later weights in flight; the
  // short one waits for the tokens of DT = DW k-steps back, which with two
  // k-steps of weights in flight measured faster.
  if (TA) {
#pragma unroll
    for (int j = 0; j < DT; ++j) {
      tok_load(j);
      if (j >= DT - DW) wb[j - (DT - DW)] = bload(ws.r0, ws.v0, ksoff(ws, j - (DT - DW), KS));
    }
  } else {
#pragma unroll
    for (int p = 0; p < DT; ++p) tok_load(p);
#pragma unroll
    for (int p = 0; p < DW; ++p) wb[p] = bload(ws.r0, ws.v0, ksoff(ws, p, KS));
  }
  for (int k0 = 0; k0 < KS; k0 += DW) {
#pragma unroll
    for (int p = 0; p < DW; ++p) {
      const int ks = k0 + p;
      wait_vm<(TA ? DW - 1 : DT - 1) * (1 + NTK)>();
      wg_barrier();
      __builtin_amdgcn_sched_barrier(0);
      if (TA) tok_load(ks + DT);
      __builtin_amdgcn_sched_barrier(0);
      if (active) {
        const uint8_t *sb = ring + (ks % (DT + 1)) * (NT * 1024) + lane * 16;
        bf16x8 xc = *reinterpret_cast<const bf16x8 *>(sb);
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          bf16x8 xn = xc;
          if (j + 1 < NT) xn = *reinterpret_cast<const bf16x8 *>(sb + (j + 1) * 1024);
          acc[j] = mfma16(wb[p], xc, acc[j]);
          __builtin_amdgcn_sched_barrier(0);
          xc = xn;
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      wb[p] = bload(ws.r0, ws.v0, ksoff(ws, ks + DW, KS));
      if (!TA) tok_load(ks + DT);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  wait_vm<0>();
  if (!active) return;
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const int tk = 16 * j + row;
    if (tk < pt.n) {
      const f32x4 o = acc[j];
      const float4 v = {gt[j] * o[0], gt[j] * o[1], gt[j] * o[2], gt[j] * o[3]};
      *reinterpret_cast<float4 *>(pairbuf + (size_t)(pt.p0 + tk) * d + 16 * rtile +
                                  4 * (lane >> 4)) = v;
    }
  }
}

// gate/up: up to FFN_WAVES row-pair tiles per unit (hdr->rp_gu, chosen by
// the compaction launch), the part's tiles shared through the LDS ring.
template <bool PACKED>
__global__ __launch_bounds__(FFN_WAVES * WAVE)
void k_gateup_bf16(int d, int I, int E, int ns, const uint16_t *__restrict__ w13r,
                   const uint16_t *__restrict__ w13s, const FfnHdr *__restrict__ hdr,
                   const FfnUnit *__restrict__ units, const uint16_t *__restrict__ x, int B,
                   const uint32_t *__restrict__ tokoff, uint16_t *__restrict__ hp) {
  __shared__ __attribute__((aligned(16))) uint8_t ring[(FFN_GU_DT + 1) * FFN_GU_PT * 2048];
  __shared__ __attribute__((aligned(16))) uint8_t dummy[FFN_WAVES * 1024];
  // this die's header and run (written by the compaction workgroup that
  // ran on the same die)
  hdr += blockIdx.x % N_XCD;
  const int RP = __builtin_amdgcn_readfirstlane(hdr->rp_gu);
  const int T = I / 16;                    // row-pair tiles per expert
  if (RP < 1 || RP > FFN_WAVES) return;    // only for a plan not made by k_compact
  const Run run = die_run(hdr->gu0, hdr->gu1);
  const rsrc_t rx = make_rsrc(x, (uint32_t)B * (uint32_t)d * 2u);
  const int w = wave_id_u(), lane = lane_id();
  for (int k = run.k0; k < run.k1; k += run.step) {
    // the unit and this wavefront's token rows (row l / 8 of each half of
    // its tile), loaded together
    const uint32_t *tr = tokoff + (size_t)k * FFN_GU_TOK + 16 * w + (lane >> 3);
    const uint32_t tk0 = w < FFN_GU_PT ? tr[0] : FFN_TOK_PAD;
    const uint32_t tk1 = w < FFN_GU_PT ? tr[8] : FFN_TOK_PAD;
    const PartU pt = load_unit(units + k);
    if (pt.u < 0 || pt.u >= E + ns || pt.nt < 1 || pt.nt > FFN_GU_PT) continue;
    const uint16_t *w13 = pt.u < E ? w13r : w13s;
    PartU q = pt;
    q.u = pt.u < E ? pt.u : pt.u - E;   // experts E .. E + ns - 1: the shared ones
    const int rp0 = pt.rg * RP, nrp = min(RP, T - rp0);
    if (nrp < 1) continue;
    wg_barrier();   // every wavefront is done with the previous unit's ring
    // entries past the part's pairs are not written: those lanes read zero
    const uint32_t seg = 16u * (uint32_t)((lane & 7) ^ (lane >> 3));
    const uint32_t tv0 = 16 * w + (lane >> 3) < q.n ? tk0 + seg : FFN_TOK_PAD;
    const uint32_t tv1 = 16 * w + 8 + (lane >> 3) < q.n ? tk1 + seg : FFN_TOK_PAD;
#define BASE_GU(N) case N: gateup_unit<N, PACKED>(ring, dummy, d, I, w13, q, rp0, nrp, rx, tv0, tv1, hp); break;
    switch (q.nt) { BASE_GU(1) BASE_GU(2) BASE_GU(3) BASE_GU(4) BASE_GU(5) default: BASE_GU(6) }
#undef BASE_GU
  }
}
static_assert(FFN_GU_PT == 6, "gate/up tile-count cases");

// down: hdr.rt_dn row tiles of 16 rows of d per unit (FFN_WAVES, fewer for
// a long contraction when the units would not fill the workgroups), DW
// k-steps of weights in flight; registers for WPE wavefronts per SIMD.
// Three instances (ffn_dn_kind): FFN_DN_WPE / FFN_DN_DW for launches with
// many kept slots, FFN_DN_WPE_MID / FFN_DN_DW_MID for few, FFN_DN_WPE_LONG
// / FFN_DN_DW_LONG for long contractions, whose few units each stream many
// k-steps.
template <bool PACKED, int DW, int WPE>
__global__ __launch_bounds__(FFN_WAVES * WAVE, WPE)
void k_down_bf16(int d, int I, int E, int ns, const uint16_t *__restrict__ w2r,
                 const uint16_t *__restrict__ w2s, const FfnHdr *__restrict__ hdr,
                 const FfnUnit *__restrict__ units, const float *__restrict__ pair_gate,
                 const uint16_t *__restrict__ hp, float *__restrict__ pairbuf) {
  __shared__ __attribute__((aligned(16))) uint8_t ring[(dn_token_depth(DW) + 1) * FFN_DN_PT * 1024];
  __shared__ __attribute__((aligned(16))) uint8_t dummy[FFN_WAVES * 1024];
  hdr += blockIdx.x % N_XCD;   // this die's header and run
  const int T = d / 16;          // row tiles per expert
  const int RD = __builtin_amdgcn_readfirstlane(hdr->rt_dn);
  if (RD < 1 || RD > FFN_WAVES) return;
  const Run run = die_run(hdr->dn0, hdr->dn1);
  for (int k = run.k0; k < run.k1; k += run.step) {
    const PartU pt = load_unit(units + k);
    if (pt.u < 0 || pt.u >= E + ns || pt.nt < 1 || pt.nt > FFN_DN_PT) continue;
    const uint16_t *w2 = pt.u < E ? w2r : w2s;
    PartU q = pt;
    q.u = pt.u < E ? pt.u : pt.u - E;
    const int rt0 = pt.rg * RD, nrt = min(RD, T - rt0);
    if (nrt < 1) continue;
    wg_barrier();
#define BASE_DN(N) case N: down_unit<N, PACKED, DW>(ring, dummy, d, I, w2, q, rt0, nrt, pair_gate, hp, pairbuf); break;
    switch (q.nt) { BASE_DN(1) BASE_DN(2) BASE_DN(3) BASE_DN(4) BASE_DN(5) BASE_DN(6) BASE_DN(7) default: BASE_DN(8) }
#undef BASE_DN
  }
}
static_assert(FFN_DN_PT == 8, "down tile-count cases");

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
                         const FfnHdr *hdr, const FfnUnit *units, int n_cu,
                         const uint32_t *tokoff, void *H, hipStream_t st) {
  if (bf16) {
    launch_k(packed ? k_gateup_bf16<true> : k_gateup_bf16<false>, dim3(ffn_gu_grid(n_cu)),
             dim3(FFN_WAVES * WAVE), 0, st, d, I, E, ns, (const uint16_t *)w13,
             (const uint16_t *)w13s, hdr, units, (const uint16_t *)x, B, tokoff, (uint16_t *)H);
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
                       const FfnHdr *hdr, const FfnUnit *units, int n_cu,
                       const float *pair_gate, const void *H, float *pairbuf, hipStream_t st) {
  if (bf16) {
    const int kind = ffn_dn_kind(budget, ns, I);
    const auto kern =
        kind == 2 ? (packed ? k_down_bf16<true, FFN_DN_DW_LONG, FFN_DN_WPE_LONG>
                            : k_down_bf16<false, FFN_DN_DW_LONG, FFN_DN_WPE_LONG>)
        : kind == 1 ? (packed ? k_down_bf16<true, FFN_DN_DW_MID, FFN_DN_WPE_MID>
                              : k_down_bf16<false, FFN_DN_DW_MID, FFN_DN_WPE_MID>)
                    : (packed ? k_down_bf16<true, FFN_DN_DW, FFN_DN_WPE>
                              : k_down_bf16<false, FFN_DN_DW, FFN_DN_WPE>);
    launch_k(kern, dim3(ffn_dn_grid(n_cu, kind)), dim3(FFN_WAVES * WAVE), 0, st, d, I, E, ns,
             (const uint16_t *)w2,
             (const uint16_t *)w2s, hdr, units, pair_gate, (const uint16_t *)H, pairbuf);
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
