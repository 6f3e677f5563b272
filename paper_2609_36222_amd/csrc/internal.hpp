// Launchers of the BASE kernels, called by the C ABI layer (api.hip).
// Each enqueues on `st` and returns hipGetLastError() of its launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace basek {

constexpr int MAX_K = 16;     // experts per token
constexpr int MAX_E = 256;    // experts per layer
constexpr int MAX_B = 1024;   // tokens per batch
constexpr int FFN_PART = 64;  // tokens of one FFN wavefront (4 MFMA tiles)

// Upper bounds (host-known) of the FFN token tiling for a batch: 16-pair
// tiles and 64-token parts over all kept slots.
inline int ffn_max_tiles(int B, int K, int budget) { return (B * K + 15) / 16 + budget; }
inline int ffn_max_parts(int B, int K, int budget) {
  return (B * K + FFN_PART - 1) / FFN_PART + budget;
}

hipError_t launch_route_logits(bool bf16, const void *x, int B, int d,
                               const float *W, const float *beta, int E,
                               float *logits, hipStream_t st);
hipError_t launch_token(bool bf16, const void *x, int B, int d, int E, int K,
                        int norm_topk, const float *logits, int32_t *ids,
                        float *w, const float *A, const float *bp, float *cost,
                        int mode, hipStream_t st);
hipError_t launch_select(int B, int K, int E, const int32_t *ids,
                         const float *cost, int budget, float *scores,
                         int32_t *counts, int32_t *sel_ids, int32_t *n_sel,
                         int32_t *slot_of, hipStream_t st);
hipError_t launch_backfill(int B, int E, int K, int norm_topk, int flags,
                           const float *logits, const int32_t *ids,
                           const int32_t *slot_of, const int32_t *n_sel,
                           int32_t *exec_ids, float *exec_gates,
                           hipStream_t st);
hipError_t launch_compact(int B, int K, int budget, const int32_t *exec_ids,
                          const float *exec_gates, const int32_t *slot_of,
                          const int32_t *n_sel, int32_t *offsets,
                          int32_t *pair_tok, float *pair_gate,
                          int32_t *pair_of, int32_t *tile_base,
                          int32_t *part_base, hipStream_t st);
hipError_t launch_gather(const void *x, int B, int d, int K, int budget,
                         const int32_t *n_sel, const int32_t *offsets,
                         const int32_t *pair_tok, const int32_t *tile_base,
                         void *xp, hipStream_t st);
hipError_t launch_pack(const void *w13, const void *w2, void *w13p, void *w2p,
                       int E, int d, int I, hipStream_t st);
hipError_t launch_gateup(bool bf16, bool packed, const void *x, int B, int d,
                         int I, int E, int K, int budget, const void *w13,
                         const int32_t *sel_ids, const int32_t *n_sel,
                         const int32_t *offsets, const int32_t *pair_tok,
                         const int32_t *tile_base, const int32_t *part_base,
                         const void *xp, void *H, hipStream_t st);
hipError_t launch_down(bool bf16, bool packed, int B, int d, int I, int E, int K,
                       int budget, const void *w2, const int32_t *sel_ids,
                       const int32_t *n_sel, const int32_t *offsets,
                       const int32_t *tile_base, const int32_t *part_base,
                       const float *pair_gate, const void *H, float *pairbuf,
                       hipStream_t st);
hipError_t launch_combine(bool bf16, int B, int d, int K,
                          const int32_t *pair_of, const float *pairbuf,
                          const void *residual, void *y, hipStream_t st);

}  // namespace basek
