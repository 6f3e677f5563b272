// Batch aggregation, budgeted selection, backfill and compaction (K2).
//
// k_select   one workgroup.  D_hat_u = sum over tokens routing u of their
//            predicted cost (Sec. 3.4, eq. log_energy_predictor), summed
//            per 64-token chunk by the halving tree and chunk by chunk in
//            ascending order; then the kept set: the min(budget, |union|)
//            experts of the batch union first in the order (D_hat desc,
//            index asc) (Sec. 3.4; App. "Custom GPU Kernels": one kernel
//            selects the highest-scoring experts for the whole batch).
// k_backfill one wavefront per token: the experts it executes -- its K
//            highest-ranked experts inside the kept set, or only its kept
//            routes under the drop rule -- and their gates (Sec. 3.5).
// k_compact  one workgroup: counting sort of the executed (token, rank)
//            pairs by (kept slot, token), the token lists of the grouped FFN.
#include "common.hpp"
#include "internal.hpp"

namespace basek {

constexpr int SEL_THREADS = 1024;

__global__ __launch_bounds__(SEL_THREADS)
void k_select(int B, int K, int E, const int32_t *__restrict__ ids,
              const float *__restrict__ cost, int budget,
              float *__restrict__ scores, int32_t *__restrict__ counts,
              int32_t *__restrict__ sel_ids, int32_t *__restrict__ n_sel_out,
              int32_t *__restrict__ slot_of) {
  __shared__ float V[MAX_E * WAVE];   // chunk matrix: expert x token-in-chunk
  __shared__ float D[MAX_E];
  __shared__ int cnt[MAX_E];
  __shared__ int n_union;
  const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
  const int nwaves = SEL_THREADS / WAVE;

  for (int u = tid; u < E; u += SEL_THREADS) { cnt[u] = 0; D[u] = 0.0f; }
  if (tid == 0) n_union = 0;
  __syncthreads();
  for (int p = tid; p < B * K; p += SEL_THREADS) {
    const int u = ids[p];
    if (u >= 0 && u < E) atomicAdd(&cnt[u], 1);
  }

  const int nchunks = (B + WAVE - 1) / WAVE;
  for (int c = 0; c < nchunks; ++c) {
    for (int i = tid; i < E * WAVE; i += SEL_THREADS) V[i] = 0.0f;
    __syncthreads();
    for (int q = tid; q < WAVE * K; q += SEL_THREADS) {
      const int t = c * WAVE + q / K;
      if (t < B) {
        const int u = ids[(size_t)t * K + q % K];
        if (u >= 0 && u < E) V[u * WAVE + (t - c * WAVE)] = cost[(size_t)t * K + q % K];
      }
    }
    __syncthreads();
    // row u always belongs to the same wavefront, so chunks are added to
    // D[u] in ascending order
    for (int u = wave; u < E; u += nwaves) {
      const float s = wave_tree_sum(V[u * WAVE + lane]);
      if (lane == 0) D[u] = (c == 0) ? s : D[u] + s;
    }
    __syncthreads();
  }

  for (int u = tid; u < E; u += SEL_THREADS)
    if (cnt[u] > 0) atomicAdd(&n_union, 1);
  __syncthreads();
  const int n_sel = min(budget, n_union);
  for (int u = tid; u < E; u += SEL_THREADS) {
    int slot = -1;
    if (cnt[u] > 0) {
      const float du = D[u];
      int r = 0;
      for (int v = 0; v < E; ++v)
        r += (cnt[v] > 0) && ranks_before(D[v], v, du, u);
      if (r < n_sel) { slot = r; sel_ids[r] = u; }
    }
    slot_of[u] = slot;
    scores[u] = D[u];
    counts[u] = cnt[u];
  }
  for (int r = n_sel + tid; r < budget; r += SEL_THREADS) sel_ids[r] = -1;
  if (tid == 0) *n_sel_out = n_sel;
}

constexpr int BF_WAVES = 4;

__global__ __launch_bounds__(BF_WAVES * WAVE)
void k_backfill(int B, int E, int K, int norm_topk, int flags,
                const float *__restrict__ logits, const int32_t *__restrict__ ids,
                const int32_t *__restrict__ slot_of,
                const int32_t *__restrict__ n_sel_p,
                int32_t *__restrict__ exec_ids, float *__restrict__ exec_gates) {
  const int lane = lane_id();
  const int t = blockIdx.x * BF_WAVES + wave_id();
  if (t >= B) return;
  const int n_sel = *n_sel_p;
  const float *lt = logits + (size_t)t * E;

  int R[MAX_K];
#pragma unroll
  for (int k = 0; k < MAX_K; ++k) {
    int u = (k < K) ? ids[(size_t)t * K + k] : 0;
    R[k] = (u >= 0 && u < E) ? u : 0;
  }
  const float lmax = lt[R[0]];

  int X[MAX_K];
  int nx = 0;
#pragma unroll
  for (int k = 0; k < MAX_K; ++k) X[k] = -1;

  if (flags & 2) {   // drop: the routed experts that were kept, rank order
#pragma unroll
    for (int k = 0; k < MAX_K; ++k)
      if (k < K && slot_of[R[k]] >= 0) {
#pragma unroll
        for (int q = 0; q < MAX_K; ++q)
          if (q == nx) X[q] = R[k];
        ++nx;
      }
  } else {           // backfill: first min(K, n_sel) kept experts in rank order
    float lv[4];
    bool cand[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = lane + WAVE * i;
      cand[i] = (e < E) && slot_of[e] >= 0;
      lv[i] = (e < E) ? lt[e] : 0.0f;
    }
    const int kp = min(K, n_sel);
#pragma unroll
    for (int k = 0; k < MAX_K; ++k) {
      if (k < kp && nx == k) {
        float bv = -INFINITY;
        int bi = 0x7FFFFFFF;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e = lane + WAVE * i;
          if (cand[i] && ranks_before(lv[i], e, bv, bi)) { bv = lv[i]; bi = e; }
        }
        wave_argbest(bv, bi);
        if (bi < E) {   // a kept expert was left (always, for a consistent plan)
          X[k] = bi;
          nx = k + 1;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (lane + WAVE * i == bi) cand[i] = false;
      }
    }
  }

  // gates: numerators exp(l_v - l_max); denominator per flags
  float num[MAX_K];
#pragma unroll
  for (int j = 0; j < MAX_K; ++j)
    num[j] = (j < nx) ? base_exp(lt[X[j]] - lmax) : 0.0f;
  float S;
  if (flags & 1) {
    S = 0.0f;
#pragma unroll
    for (int j = 0; j < MAX_K; ++j)
      if (j < nx) S = S + num[j];
  } else if (norm_topk) {
    S = 0.0f;
#pragma unroll
    for (int k = 0; k < MAX_K; ++k)
      if (k < K) S = S + base_exp(lt[R[k]] - lmax);
  } else {
    float part = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = lane + WAVE * i;
      if (e < E) part = part + base_exp(lt[e] - lmax);
    }
    S = wave_tree_sum(part);
  }
#pragma unroll
  for (int j = 0; j < MAX_K; ++j) {
    if (j < K && lane == j) {
      exec_ids[(size_t)t * K + j] = (j < nx) ? X[j] : -1;
      exec_gates[(size_t)t * K + j] = (j < nx) ? num[j] / S : 0.0f;
    }
  }
}

// Exclusive prefix over slots s < n of ceil(cnt[s] / unit) by one
// wavefront (4 slots per lane); out[MAX_E] receives the total.
__device__ __forceinline__ void wave_scan_slots(const int *cnt, int n, int unit,
                                                int *out) {
  const int lane = lane_id();
  int local[MAX_E / WAVE];
  int sum = 0;
#pragma unroll
  for (int q = 0; q < MAX_E / WAVE; ++q) {
    const int s = lane * (MAX_E / WAVE) + q;
    local[q] = (s < n) ? (cnt[s] + unit - 1) / unit : 0;
    sum += local[q];
  }
  int incl = sum;
#pragma unroll
  for (int h = 1; h < WAVE; h <<= 1) {
    const int o = __shfl_up(incl, h, WAVE);
    if (lane >= h) incl += o;
  }
  int run = incl - sum;
#pragma unroll
  for (int q = 0; q < MAX_E / WAVE; ++q) {
    out[lane * (MAX_E / WAVE) + q] = run;
    run += local[q];
  }
  if (lane == WAVE - 1) out[MAX_E] = incl;
}

constexpr int CP_THREADS = 1024;
constexpr int CP_WORDS = MAX_B / 32;

__global__ __launch_bounds__(CP_THREADS)
void k_compact(int B, int K, int budget, const int32_t *__restrict__ exec_ids,
               const float *__restrict__ exec_gates,
               const int32_t *__restrict__ slot_of,
               const int32_t *__restrict__ n_sel_p,
               int32_t *__restrict__ offsets, int32_t *__restrict__ pair_tok,
               float *__restrict__ pair_gate, int32_t *__restrict__ pair_of,
               int32_t *__restrict__ tile_base, int32_t *__restrict__ part_base) {
  // bits[s][w]: bit (t & 31) of word w = t >> 5 is set when token t runs slot s
  __shared__ uint32_t bits[MAX_E * CP_WORDS];
  __shared__ int pre[MAX_E * CP_WORDS];
  __shared__ int cnt[MAX_E];
  __shared__ int off[MAX_E + 1];
  __shared__ int tb[MAX_E + 1];
  __shared__ int pb[MAX_E + 1];
  const int tid = threadIdx.x, lane = lane_id();
  const int n_sel = min(max(*n_sel_p, 0), budget);
  const int nwords = (B + 31) / 32;

  for (int i = tid; i < n_sel * CP_WORDS; i += CP_THREADS) bits[i] = 0u;
  __syncthreads();
  const int t = tid;
  int s_of[MAX_K];
#pragma unroll
  for (int j = 0; j < MAX_K; ++j) {
    int s = -1;
    if (t < B && j < K) {
      const int u = exec_ids[(size_t)t * K + j];
      if (u >= 0) s = slot_of[u];
    }
    s_of[j] = (s >= 0 && s < n_sel) ? s : -1;
    if (s_of[j] >= 0) atomicOr(&bits[s_of[j] * CP_WORDS + (t >> 5)], 1u << (t & 31));
  }
  __syncthreads();
  for (int s = tid; s < n_sel; s += CP_THREADS) {
    int run = 0;
    for (int w = 0; w < nwords; ++w) {
      pre[s * CP_WORDS + w] = run;
      run += __popc(bits[s * CP_WORDS + w]);
    }
    cnt[s] = run;
  }
  __syncthreads();
  if (tid < WAVE) {   // exclusive scans over slots by one wavefront:
    wave_scan_slots(cnt, n_sel, 1, off);          // pairs
    wave_scan_slots(cnt, n_sel, 16, tb);          // 16-pair tiles
    wave_scan_slots(cnt, n_sel, FFN_PART, pb);    // FFN token parts
  }
  __syncthreads();
  for (int s = tid; s <= budget; s += CP_THREADS) {
    tile_base[s] = (s < n_sel) ? tb[s] : tb[MAX_E];
    part_base[s] = (s < n_sel) ? pb[s] : pb[MAX_E];
  }
  const int total = off[MAX_E];
  for (int s = tid; s <= budget; s += CP_THREADS)
    offsets[s] = (s < n_sel) ? off[s] : total;
  if (t < B) {
#pragma unroll
    for (int j = 0; j < MAX_K; ++j) {
      if (j < K) {
        int p = -1;
        const int s = s_of[j];
        if (s >= 0) {
          const uint32_t below = bits[s * CP_WORDS + (t >> 5)] & ((1u << (t & 31)) - 1u);
          p = off[s] + pre[s * CP_WORDS + (t >> 5)] + __popc(below);
          pair_tok[p] = t;
          pair_gate[p] = exec_gates[(size_t)t * K + j];
        }
        pair_of[(size_t)t * K + j] = p;
      }
    }
  }
}

hipError_t launch_select(int B, int K, int E, const int32_t *ids,
                         const float *cost, int budget, float *scores,
                         int32_t *counts, int32_t *sel_ids, int32_t *n_sel,
                         int32_t *slot_of, hipStream_t st) {
  hipLaunchKernelGGL(k_select, dim3(1), dim3(SEL_THREADS), 0, st, B, K, E, ids,
                     cost, budget, scores, counts, sel_ids, n_sel, slot_of);
  return hipGetLastError();
}

hipError_t launch_backfill(int B, int E, int K, int norm_topk, int flags,
                           const float *logits, const int32_t *ids,
                           const int32_t *slot_of, const int32_t *n_sel,
                           int32_t *exec_ids, float *exec_gates,
                           hipStream_t st) {
  hipLaunchKernelGGL(k_backfill, dim3((B + BF_WAVES - 1) / BF_WAVES),
                     dim3(BF_WAVES * WAVE), 0, st, B, E, K, norm_topk, flags,
                     logits, ids, slot_of, n_sel, exec_ids, exec_gates);
  return hipGetLastError();
}

hipError_t launch_compact(int B, int K, int budget, const int32_t *exec_ids,
                          const float *exec_gates, const int32_t *slot_of,
                          const int32_t *n_sel, int32_t *offsets,
                          int32_t *pair_tok, float *pair_gate,
                          int32_t *pair_of, int32_t *tile_base,
                          int32_t *part_base, hipStream_t st) {
  hipLaunchKernelGGL(k_compact, dim3(1), dim3(CP_THREADS), 0, st, B, K, budget,
                     exec_ids, exec_gates, slot_of, n_sel, offsets, pair_tok,
                     pair_gate, pair_of, tile_base, part_base);
  return hipGetLastError();
}

}  // namespace basek
