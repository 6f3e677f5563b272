// Launchers of the BASE kernels, called by the C ABI layer (api.hip).
// Each enqueues on `st` and returns hipGetLastError() of its launch.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>

namespace basek {

constexpr int MAX_K = 16;     // experts per token
constexpr int MAX_E = 256;    // experts per layer
constexpr int MAX_B = 1024;   // tokens per batch

// Events attached to the next kernel launch (per host thread): when set,
// launch_k hands them to the dispatch itself, which records `start` as the
// kernel begins and `stop` as it ends, then clears them.
struct KernelEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
KernelEvents &kernel_events();

template <typename F, typename... Args>
inline void launch_k(F kernel, dim3 grid, dim3 block, uint32_t shm, hipStream_t st,
                     Args... args) {
  KernelEvents &ev = kernel_events();
  if (ev.start || ev.stop) {
    hipExtLaunchKernelGGL(kernel, grid, block, shm, st, ev.start, ev.stop, 0, args...);
    ev.start = ev.stop = nullptr;
  } else {
    // the ordinary launch: the form a stream capture records as a graph node
    hipLaunchKernelGGL(kernel, grid, block, shm, st, args...);
  }
}

constexpr int N_XCD = 8;   // accelerator dies, one L2 each

// Token groups on dies.  The scoring launches keep a group of TOK_GROUP
// consecutive tokens on one die, g on die g % N_XCD, so that a token's
// logits are read where they were written (in that die's L2).  Workgroup b
// of such a launch runs on die b % N_XCD; with `per` workgroups per group it
// takes group g = b % N_XCD + N_XCD * (q / per) and share q % per of it (q =
// b / N_XCD).  The launch has xcd_grid(groups, per) workgroups; those past
// the last group have nothing to do.
constexpr int TOK_GROUP = 16;
__host__ __device__ inline int xcd_grid(int groups, int per) {
  return N_XCD * ((groups + N_XCD - 1) / N_XCD) * per;
}
__device__ inline void xcd_group(int b, int per, int &g, int &share) {
  const int q = b / N_XCD;
  g = b % N_XCD + N_XCD * (q / per);
  share = q % per;
}

constexpr int MAX_SHARED = 8;               // shared experts per layer
constexpr int MAX_SLOTS = MAX_E + MAX_SHARED;  // kept slots + shared slots

// Upper bound (host-known) of the FFN's 16-pair tiles for a batch over all
// kept slots and the ns shared slots (B pairs each).
inline int ffn_max_tiles(int B, int K, int budget, int ns) {
  return (B * K + 15) / 16 + budget + ns * ((B + 15) / 16);
}

// The grouped bf16 FFN (see "Grouped bf16 FFN" in ffn.hip).  A part is at
// most FFN_GU_PT (gate/up) or FFN_DN_PT (down) 16-pair tiles of one kept or
// shared slot; a unit of work is (part, row group), one per workgroup of
// FFN_WAVES wavefronts at a time, each wavefront owning 16-row tiles over the
// whole contraction with weights requested FFN_GU_DW (gate/up) or FFN_DN_DW
// (down) k-steps ahead and token fragments FFN_GU_DT steps (two k-steps each,
// one step further ahead than the weights) or FFN_DN_DT k-steps ahead (the
// deep down instance: one k-step further ahead than its weights).
constexpr int FFN_WAVES = 8;
constexpr int FFN_GU_DW = 8;
constexpr int FFN_GU_DT = FFN_GU_DW / 2 + 1;
constexpr int FFN_DN_DW = 2;
constexpr int FFN_DN_DT = 2;
// wavefronts per SIMD the down kernel's registers allow: three workgroups
// per CU, so that a die's down units mostly run in one round
constexpr int FFN_DN_WPE = 6;
// down with a long contraction (more than FFN_DN_LONG_KS k-steps of I): few
// units that each stream many k-steps, so more weights in flight per
// wavefront and one workgroup per CU
constexpr int FFN_DN_LONG_KS = 64;
constexpr int FFN_DN_DW_LONG = 8;
constexpr int FFN_DN_WPE_LONG = 2;
__host__ __device__ inline bool ffn_dn_long(int I) { return I / 32 > FFN_DN_LONG_KS; }
// down for launches with few kept slots (fewer than 4 per die, so that the
// compaction cuts each slot's row groups over the dies): fewer units, so
// four k-steps of weights in flight and two workgroups per CU
constexpr int FFN_DN_DW_MID = 4;
constexpr int FFN_DN_WPE_MID = 4;
// down's instance: 2 long contraction, 1 few slots (budget + shared ones),
// 0 otherwise
__host__ __device__ inline int ffn_dn_kind(int budget, int ns, int I) {
  return ffn_dn_long(I) ? 2 : (budget + ns < 4 * N_XCD ? 1 : 0);
}
constexpr int FFN_GU_PT = 6;
constexpr int FFN_DN_PT = 8;
// gate/up reads its token rows straight from the hidden states: entry i of
// gate/up unit k's row is the byte offset of the row of its part's pair i,
// tokoff[k * FFN_GU_TOK + i] = t * d * 2 (written for the part's pairs only)
constexpr int FFN_GU_TOK = FFN_GU_PT * 16;
constexpr uint32_t FFN_TOK_PAD = 0x80000000u;   // past every x: a buffer load returns zero
static_assert(FFN_GU_PT <= FFN_WAVES, "one token tile per gate/up wavefront");
static_assert((size_t)MAX_B * 16384 * 2 < FFN_TOK_PAD, "token row offsets below the pad mark");

// A unit: expert u (u >= E: shared expert u - E), the part's first 16-pair
// tile, its tile count, its first pair in the compacted order and its pair
// count, and the unit's row group (gate/up: hdr.rp_gu row-pair tiles;
// down: hdr.rt_dn row tiles).
struct alignas(32) FfnUnit {
  int32_t u, tile0, nt, p0, n, rg, pad0, pad1;
};
// Die x's header, written by the compaction workgroup that ran on die x:
// gate/up's row group (rp_gu row-pair tiles), down's (rt_dn row tiles) and
// die x's runs of units, [gu0, gu1) of the gate/up table and [dn0, dn1) of
// the down table.
struct alignas(32) FfnHdr {
  int32_t rp_gu, gu0, gu1, dn0, dn1, rt_dn, pad1, pad2;
};

// Upper bound of the parts of a launch with at most pt tiles per part: the
// sum over slots of ceil(tiles / pt) is below tiles / pt + slots.
inline int ffn_parts_bound(int B, int K, int budget, int ns, int pt) {
  return ffn_max_tiles(B, K, budget, ns) / pt + budget + ns + 1;
}
// Upper bounds of the units: every part times its row groups (gate/up: at
// least FFN_WAVES / 2 row-pair tiles per group; down: at least 2 row tiles).
inline int ffn_units_bound_gu(int B, int K, int budget, int ns, int I) {
  return ffn_parts_bound(B, K, budget, ns, FFN_GU_PT) * ((I / 16 + FFN_WAVES / 2 - 1) / (FFN_WAVES / 2));
}
inline int ffn_units_bound_dn(int B, int K, int budget, int ns, int d) {
  return ffn_parts_bound(B, K, budget, ns, FFN_DN_PT) * ((d / 16 + 1) / 2);
}
// Workgroups of the FFN launches: a multiple of N_XCD, from the device's
// compute units -- gate/up one per CU (its registers allow no second), down
// FFN_DN_WPE / 2 (FFN_DN_WPE_MID / 2, FFN_DN_WPE_LONG / 2) per CU: a
// workgroup of FFN_WAVES wavefronts puts two on each SIMD.
__host__ __device__ inline unsigned ffn_cu_grid(int n_cu) { return (unsigned)(((n_cu + N_XCD - 1) / N_XCD) * N_XCD); }
__host__ __device__ inline unsigned ffn_gu_grid(int n_cu) { return ffn_cu_grid(n_cu); }
__host__ __device__ inline unsigned ffn_dn_grid(int n_cu, int kind) {
  const int wpe = kind == 2 ? FFN_DN_WPE_LONG : kind == 1 ? FFN_DN_WPE_MID : FFN_DN_WPE;
  return (unsigned)(wpe / 2) * ffn_cu_grid(n_cu);
}

// rows: n_router of Wr (logits, + beta), then the vector G when given (gdot)
hipError_t launch_scores(bool bf16, const void *x, int B, int d, const float *Wr,
                         const float *beta, int n_router, const float *G, float *logits,
                         float *gdot, hipStream_t st);
// Selection rules (the values of BASE_SCORE_* in base.h): the per-pair
// score k_tail writes as the cost
constexpr int SCORE_BASE = 0, SCORE_TOP1 = 1, SCORE_WEIGHT = 2, SCORE_WEIGHT_SQ = 3,
              SCORE_STATIC = 4;
// mode bit 0: top-K + weights from logits; bit 1: per-pair scores of `rule`
// (SCORE_BASE: the predictor a_u . x / ||x|| from x (rows of d) and A)
// order / ex / den (optional, route mode): per token the experts in rank
// order [B][E] (bytes), exp(l - l_max) in rank order [B][E] and the router's
// softmax denominator S [B], for the fused layer's backfill
hipError_t launch_tail(bool bf16, int B, int E, int K, int d, int norm_topk,
                       const float *logits, const void *x, const float *A, const float *bp,
                       int32_t *ids, float *w, float *cost, int mode, int rule,
                       hipStream_t st, uint8_t *order = nullptr, float *ex = nullptr,
                       float *den = nullptr);
// binary: rank by (score > 0) instead of the score (the top-1-union rule)
hipError_t launch_select(int B, int K, int E, const int32_t *ids,
                         const float *cost, int budget, bool binary, float *scores,
                         int32_t *counts, int32_t *sel_ids, int32_t *n_sel,
                         int32_t *slot_of, hipStream_t st);
// selection and backfill in one launch (same results as the two launches)
// (order / ex / den: k_tail's rank rows and denominators of the batch)
hipError_t launch_select_backfill(int B, int K, int E, const int32_t *ids, const float *cost,
                                  int budget, bool binary, int flags, const uint8_t *order,
                                  const float *ex, const float *den, float *scores,
                                  int32_t *counts, int32_t *sel_ids, int32_t *n_sel,
                                  int32_t *slot_of, int32_t *exec_ids, float *exec_gates,
                                  hipStream_t st);
hipError_t launch_backfill(int B, int E, int K, int norm_topk, int flags,
                           const float *logits, const int32_t *ids,
                           const int32_t *slot_of, const int32_t *n_sel,
                           int32_t *exec_ids, float *exec_gates,
                           hipStream_t st);
// ns shared slots follow the kept ones (expert E + i, every token, gate
// sigmoid(gdot[t]) or 1 when gdot is null).  With `tables` (bf16 layers)
// the same launch also writes the FFN's unit tables (units_gu, units_dn, of
// at most ffn_units_bound_gu / _dn rows), the per-die headers and gate/up's
// token row offsets (tokoff, FFN_GU_TOK per gate/up unit; d: the hidden
// size); n_cu: the device's compute units (the FFN launches' sizes follow
// from it).
hipError_t launch_compact(int B, int K, int E, int budget, int ns, const int32_t *exec_ids,
                          const float *exec_gates, const int32_t *slot_of,
                          const int32_t *n_sel, const float *gdot, int32_t *offsets,
                          int32_t *pair_tok, float *pair_gate,
                          int32_t *pair_of, const int32_t *sel_ids, bool tables, int d,
                          int I, uint32_t *tokoff, FfnHdr *hdr, FfnUnit *units_gu,
                          FfnUnit *units_dn, int n_cu, hipStream_t st);
hipError_t launch_pack(const void *w13, const void *w2, void *w13p, void *w2p,
                       int E, int d, int I, hipStream_t st);
// parts of expert u >= E read the shared experts' weights (w13s / w2s, u - E)
hipError_t launch_gateup(bool bf16, bool packed, const void *x, int B, int d,
                         int I, int E, int K, int budget, int ns, const void *w13,
                         const void *w13s,
                         const int32_t *sel_ids, const int32_t *n_sel,
                         const int32_t *offsets, const int32_t *pair_tok,
                         const FfnHdr *hdr, const FfnUnit *units, int n_cu,
                         const uint32_t *tokoff, void *H, hipStream_t st);
hipError_t launch_down(bool bf16, bool packed, int B, int d, int I, int E, int K,
                       int budget, int ns, const void *w2, const void *w2s,
                       const int32_t *sel_ids,
                       const int32_t *n_sel, const int32_t *offsets,
                       const FfnHdr *hdr, const FfnUnit *units, int n_cu,
                       const float *pair_gate, const void *H, float *pairbuf, hipStream_t st);
// kc: columns of pair_of (K routed + the shared experts)
hipError_t launch_combine(bool bf16, int B, int d, int kc,
                          const int32_t *pair_of, const float *pairbuf,
                          const void *residual, void *y, hipStream_t st);

// Calibration statistics (per expert u): head[u] = (n, sum y, sum y^2, 0)
// fp64, sz[u][d] and q[u][d] fp64, G[u][d][d] fp32; each array 256-byte
// aligned in the caller's buffer, in this order.
struct CalibStats {
  double *head, *sz, *q;
  float *G;
};
inline size_t calib_up256(size_t v) { return (v + 255) & ~(size_t)255; }
inline size_t calib_stats_bytes(int E, int d) {
  return calib_up256((size_t)E * 4 * 8) + 2 * calib_up256((size_t)E * d * 8) +
         calib_up256((size_t)E * d * d * 4);
}
inline CalibStats calib_stats_at(void *base, int E, int d) {
  char *p = static_cast<char *>(base);
  CalibStats s;
  s.head = reinterpret_cast<double *>(p);
  p += calib_up256((size_t)E * 4 * 8);
  s.sz = reinterpret_cast<double *>(p);
  p += calib_up256((size_t)E * d * 8);
  s.q = reinterpret_cast<double *>(p);
  p += calib_up256((size_t)E * d * 8);
  s.G = reinterpret_cast<float *>(p);
  return s;
}
hipError_t launch_calib_zero(void *stats, size_t bytes, hipStream_t st);
hipError_t launch_calib_stats(const void *x, bool bf16, int B, int d, int E, int K,
                              const float *pairbuf, const int32_t *n_sel,
                              const int32_t *sel_ids, const int32_t *offsets,
                              const int32_t *pair_tok, double *inv, double *y, float *zbuf,
                              CalibStats st, hipStream_t s);

// internal flags bit of the backfill: unit gates (calibration runs the
// experts' own outputs)
constexpr int FLAG_UNIT_GATES = 4;

}  // namespace basek
