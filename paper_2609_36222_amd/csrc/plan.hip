// Batch aggregation, budgeted selection, backfill and compaction (K2).
//
// k_select   one workgroup.  D_hat_u = sum over tokens routing u of their
//            predicted cost (Sec. 3.4, eq. log_energy_predictor), summed
//            per 64-token chunk by the halving tree and chunk by chunk in
//            ascending order; then the kept set: the min(budget, |union|)
//            experts of the batch union first in the order (D_hat desc,
//            index asc) (Sec. 3.4; App. "Custom GPU Kernels": one kernel
//            selects the highest-scoring experts for the whole batch); for
//            the top-1-union rule the order (D_hat > 0 desc, index asc).
// k_backfill one wavefront per token: the experts it executes -- its K
//            highest-ranked experts inside the kept set, or only its kept
//            routes under the drop rule -- and their gates (Sec. 3.5).
// k_compact  one workgroup: stable counting sort of the executed (token,
//            rank) pairs by kept slot, the token lists of the grouped FFN.
// k_select_backfill  the first two in one launch (the fused layer): every
//            workgroup repeats the selection and backfills its own tokens.
#include <algorithm>

#include "common.hpp"
#include "internal.hpp"

namespace basek {

constexpr int SEL_THREADS = 1024;
constexpr int SEL_PAD = WAVE + 1;                 // LDS row of one chunk tree
constexpr int SEL_V = 4 * 128 * SEL_PAD;          // chunk-matrix capacity (floats)

// LDS of the selection (one workgroup of SEL_THREADS threads)
struct SelLds {
  float V[SEL_V];
  float CS[SEL_THREADS];
  float D[MAX_E];
  int cnt[MAX_E];
  __attribute__((aligned(16))) uint64_t key[MAX_E];
  int rnk[MAX_E];
  int n_union;
};

// Aggregation and selection by one workgroup of SEL_THREADS threads; thread
// t < B brings token t's routes (uk) and costs (ck).  Chunk c (tokens 64c ..
// 64c + 63) of expert u is the row V[c][u][0..63] (position j: the cost of
// token 64c + j if it routes u, else +0); one thread per (chunk, expert)
// adds its row by the halving tree, and the chunk sums are added to D_hat_u
// in ascending chunk order.  The kept set is ranked with 64-bit keys whose
// unsigned order is (D_hat desc, index asc) -- (D_hat > 0 desc, index asc)
// with `binary`.  Writes scores, counts, sel_ids, n_sel and slot_of when
// `out` is set, and slot_of into slot_lds when that is given; returns n_sel
// (every thread).
__device__ __forceinline__ int select_body(SelLds &S, int B, int K, int E, int budget,
                                           int binary, const int (&uk)[MAX_K],
                                           const float (&ck)[MAX_K], bool out,
                                           float *__restrict__ scores,
                                           int32_t *__restrict__ counts,
                                           int32_t *__restrict__ sel_ids,
                                           int32_t *__restrict__ n_sel_out,
                                           int32_t *__restrict__ slot_of, int *slot_lds) {
  const int tid = threadIdx.x, lane = lane_id();
  for (int u = tid; u < E; u += SEL_THREADS) { S.cnt[u] = 0; S.D[u] = 0.0f; }
  if (tid == 0) S.n_union = 0;
  const int nchunks = (B + WAVE - 1) / WAVE;
  // chunks per batch: bounded by V and by one thread per (chunk, expert)
  const int cb = max(1, min(min(nchunks, SEL_V / (E * SEL_PAD)), SEL_THREADS / E));
  for (int c0 = 0; c0 < nchunks; c0 += cb) {
    const int nb = min(cb, nchunks - c0);
    const int nv = min(SEL_V, (nb * E * SEL_PAD + 3) & ~3) / 4;
    for (int i = tid; i < nv; i += SEL_THREADS)
      reinterpret_cast<float4 *>(S.V)[i] = float4{0.0f, 0.0f, 0.0f, 0.0f};
    __syncthreads();
    // the routes in rank order (a repeated expert keeps its last cost, and
    // counts every time)
    const int cl = tid / WAVE - c0;
    if (tid < B && cl >= 0 && cl < nb) {
#pragma unroll
      for (int k = 0; k < MAX_K; ++k)
        if (k < K && uk[k] >= 0 && uk[k] < E) {
          S.V[(cl * E + uk[k]) * SEL_PAD + lane] = ck[k];
          atomicAdd(&S.cnt[uk[k]], 1);
        }
    }
    __syncthreads();
    if (tid < nb * E) {
      // the tree's first level as the row is read (positions q, q + 32)
      float v[WAVE / 2];
#pragma unroll
      for (int q = 0; q < WAVE / 2; ++q)
        v[q] = S.V[tid * SEL_PAD + q] + S.V[tid * SEL_PAD + q + WAVE / 2];
#pragma unroll
      for (int h = WAVE / 4; h >= 1; h >>= 1)
#pragma unroll
        for (int q = 0; q < h; ++q) v[q] = v[q] + v[q + h];
      S.CS[tid] = v[0];
    }
    __syncthreads();
    for (int u = tid; u < E; u += SEL_THREADS)
      for (int c = 0; c < nb; ++c)
        S.D[u] = (c0 + c == 0) ? S.CS[c * E + u] : S.D[u] + S.CS[c * E + u];
    __syncthreads();
  }

  // E2: the power of two >= E (at least a wavefront); keys past E are 0
  int E2 = WAVE;
  while (E2 < E) E2 <<= 1;
  for (int u = tid; u < E2; u += SEL_THREADS) {
    const bool in = u < E && S.cnt[u] > 0;
    float kv = 0.0f;
    if (u < E) kv = binary ? (S.D[u] > 0.0f ? 1.0f : 0.0f) : S.D[u];
    S.key[u] = in ? rank_key(kv, u) : 0;   // 0: ranks after every expert
    const uint64_t m = __ballot(in);
    if (lane == 0 && m) atomicAdd(&S.n_union, (int)__popcll(m));
  }
  __syncthreads();
  const int n_sel = min(budget, S.n_union);
  {
    // tpe consecutive threads per expert, thread `part` over the key pairs
    // part, part + tpe, ... (16 bytes each: the tpe threads of an expert
    // read consecutive bytes, distinct banks); the keys past E are 0 and
    // never count
    const int tpe = SEL_THREADS / E2, npair = E2 / (2 * tpe);
    const int u = tid / tpe, part = tid % tpe;
    int r = 0;
    if (u < E && S.cnt[u] > 0) {
      const uint64_t ku = S.key[u];
      // up to 8 pairs per step, their LDS reads issued together
      for (int i0 = 0; i0 < npair; i0 += 8) {
        u32x4 o[8];
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (i0 + q < npair)
            o[q] = *reinterpret_cast<const u32x4 *>(&S.key[2 * (part + tpe * (i0 + q))]);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          if (i0 + q < npair) {
            r += (((uint64_t)o[q].y << 32 | o[q].x) > ku);
            r += (((uint64_t)o[q].w << 32 | o[q].z) > ku);
          }
        }
      }
    }
    for (int h = 1; h < tpe; h <<= 1) r += __shfl_xor(r, h, WAVE);
    if (u < E && part == 0) S.rnk[u] = r;
  }
  __syncthreads();
  for (int u = tid; u < E; u += SEL_THREADS) {
    int slot = -1;
    if (S.cnt[u] > 0 && S.rnk[u] < n_sel) {
      slot = S.rnk[u];
      if (out) sel_ids[slot] = u;
    }
    if (slot_lds) slot_lds[u] = slot;
    if (out) {
      slot_of[u] = slot;
      scores[u] = S.D[u];
      counts[u] = S.cnt[u];
    }
  }
  if (out) {
    for (int r = n_sel + tid; r < budget; r += SEL_THREADS) sel_ids[r] = -1;
    if (tid == 0) *n_sel_out = n_sel;
  }
  return n_sel;
}

// Thread t < B: token t's routes and costs (-1 / 0 past K; threads t >= B
// get nothing).  The [B][K] arrays are read with contiguous loads (a
// wavefront's load covers 64 consecutive words, not 64 rows K words apart)
// into `stage` (SEL_V floats, free again on return), rows padded to an odd
// stride, and each thread then reads its token's row from LDS.
__device__ __forceinline__ void load_routes(int B, int K, const int32_t *__restrict__ ids,
                                            const float *__restrict__ cost, float *stage,
                                            int (&uk)[MAX_K], float (&ck)[MAX_K]) {
  constexpr int LG = 2;   // loads per thread and array in flight at once
  const int tid = threadIdx.x;
  const int KP = K | 1;                                   // odd row stride
  const int tpp = (SEL_V / 2) / KP;                       // tokens per pass
  const uint64_t kmul = ((1ull << 32) + (uint64_t)K - 1) / (uint64_t)K;
  int *si = reinterpret_cast<int *>(stage);
  float *sf = stage + SEL_V / 2;
#pragma unroll
  for (int k = 0; k < MAX_K; ++k) {
    uk[k] = -1;
    ck[k] = 0.0f;
  }
  for (int t0 = 0; t0 < B; t0 += tpp) {
    const int nt = min(tpp, B - t0);
    const int n = nt * K;
    const size_t q0 = (size_t)t0 * K;
    for (int g0 = 0; g0 < n; g0 += LG * SEL_THREADS) {
      int vi[LG];
      float vf[LG];
#pragma unroll
      for (int r = 0; r < LG; ++r) {
        const int ic = min(g0 + tid + r * SEL_THREADS, n - 1);
        vi[r] = ids[q0 + ic];
        vf[r] = cost[q0 + ic];
      }
#pragma unroll
      for (int r = 0; r < LG; ++r) {
        const int i = g0 + tid + r * SEL_THREADS;
        if (i < n) {
          const int tt = (int)(((uint64_t)(uint32_t)i * kmul) >> 32);
          si[tt * KP + (i - tt * K)] = vi[r];
          sf[tt * KP + (i - tt * K)] = vf[r];
        }
      }
    }
    __syncthreads();
    if (tid >= t0 && tid < t0 + nt) {
#pragma unroll
      for (int k = 0; k < MAX_K; ++k)
        if (k < K) {
          uk[k] = si[(tid - t0) * KP + k];
          ck[k] = sf[(tid - t0) * KP + k];
        }
    }
    __syncthreads();
  }
}

// One workgroup: the batch's aggregation and selection.
__global__ __launch_bounds__(SEL_THREADS)
void k_select(int B, int K, int E, const int32_t *__restrict__ ids,
              const float *__restrict__ cost, int budget, int binary,
              float *__restrict__ scores, int32_t *__restrict__ counts,
              int32_t *__restrict__ sel_ids, int32_t *__restrict__ n_sel_out,
              int32_t *__restrict__ slot_of) {
  __shared__ SelLds S;
  int uk[MAX_K];
  float ck[MAX_K];
  load_routes(B, K, ids, cost, S.V, uk, ck);
  select_body(S, B, K, E, budget, binary, uk, ck, true, scores, counts, sel_ids, n_sel_out,
              slot_of, nullptr);
}

constexpr int BF_WAVES = 4;
constexpr int SB_WAVES = SEL_THREADS / WAVE;   // wavefronts of k_select_backfill
constexpr int SB_TOK = 2;                      // its tokens per workgroup (wavefronts 0 ..)
static_assert(TOK_GROUP % SB_TOK == 0, "a token group in whole workgroups");

// Per-wavefront LDS of the backfill
template <int W>
struct BfLds {
  __attribute__((aligned(16))) uint64_t kk[W][MAX_E];
  int ke[W][MAX_E];
  int xs[W][MAX_K];
  float num_s[W][MAX_K];
  float den_s[W][MAX_K];
  int nx_s[W];
};

// One wavefront per token t (wavefront wv of a workgroup of W; every
// wavefront takes part in the barriers).  The kept experts (slot_of >= 0)
// are packed into an LDS list with their keys (logit, index) for this
// token; each is ranked among them, and the first min(K, n_sel) by rank are
// executed in rank order.  (Ranking by counting in LDS takes fewer vector
// instructions than K successive wave maxima, which matters when 16
// wavefronts share a CU.)  Under the drop rule the token executes its
// routed experts that were kept, in routing order.  Gates: exp(l_v - l_max)
// over the original denominator (its top-K, or all E for a plain softmax
// router) or, with renormalisation, over the executed experts.
// Lane k < K: routed expert k of token t as stored (lanes >= K read the
// token's last one); backfill_body maps out-of-range ids to expert 0.  The
// load has no branch and no use here, so that it is in flight with the
// kernel's other loads.
__device__ __forceinline__ int route_of(const int32_t *__restrict__ ids, int t, int K) {
  return ids[(size_t)t * K + min(lane_id(), K - 1)];
}

// lt: the token's logits row (global memory or an LDS copy); r_k: lane k <
// K's routed expert as loaded by route_of.  An inactive wavefront
// only takes part in the workgroup's barriers.
template <int W>
__device__ __forceinline__ void backfill_body(BfLds<W> &S, bool active, int t, int B, int E,
                                              int K, int norm_topk, int flags, const float *lt,
                                              int r_k, const int32_t *slot_of, int n_sel,
                                              int32_t *__restrict__ exec_ids,
                                              float *__restrict__ exec_gates) {
  const int lane = lane_id(), wv = wave_id();
  r_k = (lane < K && r_k >= 0 && r_k < E) ? r_k : 0;
  const int r0 = __shfl(r_k, 0, WAVE);
  const float lmax = active ? lt[r0] : 0.0f;

  if (flags & 2) {   // drop: the routed experts that were kept, routing order
    if (active) {
      const bool kept = lane < K && slot_of[r_k] >= 0;
      const uint64_t m = __ballot(kept);
      if (kept) S.xs[wv][__popcll(m & ((1ull << lane) - 1))] = r_k;
      if (lane == 0) S.nx_s[wv] = __popcll(m);
    }
  } else {           // backfill: first min(K, n_sel) kept experts by rank
    int n_kept = 0;
    if (active) {
#pragma unroll
      for (int i = 0; i < MAX_E / WAVE; ++i) {
        const int e = lane + WAVE * i;
        const bool kept = e < E && slot_of[e] >= 0;
        const uint64_t m = __ballot(kept);
        if (kept) {
          const int pos = n_kept + __popcll(m & ((1ull << lane) - 1));
          S.kk[wv][pos] = rank_key(lt[e], e);
          S.ke[wv][pos] = e;
        }
        n_kept += __popcll(m);
      }
      if (lane == 0) S.nx_s[wv] = min(min(K, n_sel), n_kept);
      // keys 0 (ranked after every expert) up to a multiple of 16
      if (n_kept + lane < ((n_kept + 15) & ~15)) S.kk[wv][n_kept + lane] = 0;
    }
    __syncthreads();
    const int kp = min(K, n_sel);
    for (int s = lane; s < n_kept; s += WAVE) {
      const uint64_t ks = S.kk[wv][s];
      int r = 0;
      // 16 keys per step, their LDS reads issued together
      for (int f = 0; f < n_kept; f += 16) {
        u32x4 o[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) o[q] = *reinterpret_cast<const u32x4 *>(&S.kk[wv][f + 2 * q]);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          r += (((uint64_t)o[q].y << 32 | o[q].x) > ks);
          r += (((uint64_t)o[q].w << 32 | o[q].z) > ks);
        }
      }
      if (r < kp) S.xs[wv][r] = S.ke[wv][s];
    }
  }
  __syncthreads();
  const int nx = active ? S.nx_s[wv] : 0;

  // gates: numerators exp(l_v - l_max); denominator per flags
  float num = 0.0f;
  if (lane < nx) {
    num = base_exp(lt[S.xs[wv][lane]] - lmax);
    S.num_s[wv][lane] = num;
  }
  if (active && lane < K) S.den_s[wv][lane] = base_exp(lt[r_k] - lmax);
  __syncthreads();
  if (!active) return;
  float Ssum;
  if (flags & 1) {          // renormalised over the executed experts
    Ssum = 0.0f;
    for (int j = 0; j < nx; ++j) Ssum = Ssum + S.num_s[wv][j];
  } else if (norm_topk) {   // the router's top-K denominator
    Ssum = 0.0f;
    for (int k = 0; k < K; ++k) Ssum = Ssum + S.den_s[wv][k];
  } else {                  // the router's full softmax denominator
    float part = 0.0f;
#pragma unroll
    for (int i = 0; i < MAX_E / WAVE; ++i) {
      const int e = lane + WAVE * i;
      if (e < E) part = part + base_exp(lt[e] - lmax);
    }
    Ssum = wave_tree_sum(part);
  }
  if (t < B && lane < K) {
    exec_ids[(size_t)t * K + lane] = (lane < nx) ? S.xs[wv][lane] : -1;
    exec_gates[(size_t)t * K + lane] =
        (lane < nx) ? ((flags & FLAG_UNIT_GATES) ? 1.0f : num / Ssum) : 0.0f;
  }
}

__global__ __launch_bounds__(BF_WAVES * WAVE)
void k_backfill(int B, int E, int K, int norm_topk, int flags,
                const float *__restrict__ logits, const int32_t *__restrict__ ids,
                const int32_t *__restrict__ slot_of,
                const int32_t *__restrict__ n_sel_p,
                int32_t *__restrict__ exec_ids, float *__restrict__ exec_gates) {
  __shared__ BfLds<BF_WAVES> S;
  const int t = blockIdx.x * BF_WAVES + wave_id(), tc = min(t, B - 1);
  backfill_body<BF_WAVES>(S, true, t, B, E, K, norm_topk, flags, logits + (size_t)tc * E,
                          route_of(ids, tc, K), slot_of, *n_sel_p, exec_ids, exec_gates);
}

// Selection and backfill in one launch (the fused layer): every workgroup
// makes the batch's selection itself (the same fixed-order arithmetic, so
// the same result everywhere; workgroup 0 writes it out) and then backfills
// its own SB_TOK tokens, one per wavefront, on the tokens' own die.  The
// backfill takes the token's experts in rank order (order, written by
// k_tail with exp(l - l_max) in rank order, ex, and the router's
// denominator S, den), requested before the selection: the first
// min(K, n_sel) kept ones are executed (drop: its routed experts, ranks
// 0 .. K - 1, that were kept, in routing order), each with numerator
// exp(l - l_max) and denominator S or, renormalised, the numerators' sum in
// execution order -- the values and the order of backfill_body.
template <int NCH>
__global__ __launch_bounds__(SEL_THREADS)
void k_select_backfill(int B, int K, int E, const int32_t *__restrict__ ids,
                       const float *__restrict__ cost, int budget, int binary, int flags,
                       const uint8_t *__restrict__ order, const float *__restrict__ ex,
                       const float *__restrict__ den, float *__restrict__ scores,
                       int32_t *__restrict__ counts, int32_t *__restrict__ sel_ids,
                       int32_t *__restrict__ n_sel_out, int32_t *__restrict__ slot_of,
                       int32_t *__restrict__ exec_ids, float *__restrict__ exec_gates) {
  __shared__ SelLds S;
  __shared__ int slot_s[MAX_E];
  const int lane = lane_id(), wv = wave_id();
  int tg, tq;
  xcd_group(blockIdx.x, TOK_GROUP / SB_TOK, tg, tq);
  if (tg * TOK_GROUP >= B) return;
  const bool active = wv < SB_TOK;
  // the tokens of group tg sit on die tg % N_XCD, where k_tail wrote their
  // rank rows
  const int t = tg * TOK_GROUP + tq * SB_TOK + wv, tc = min(t, B - 1);
  int ov[NCH];
  float xv[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int r = min(WAVE * c + lane, E - 1);
    ov[c] = active ? order[(size_t)tc * E + r] : 0;
    xv[c] = active ? ex[(size_t)tc * E + r] : 0.0f;
  }
  const float dv = active ? den[tc] : 1.0f;
  int uk[MAX_K];
  float ck[MAX_K];
  load_routes(B, K, ids, cost, S.V, uk, ck);
  const int n_sel = select_body(S, B, K, E, budget, binary, uk, ck, blockIdx.x == 0, scores,
                                counts, sel_ids, n_sel_out, slot_of, slot_s);
  __syncthreads();   // slot_s complete
  if (!active || t >= B) return;
  const int kp = min(K, n_sel);
  const bool drop = flags & 2, renorm = flags & 1;
  const uint64_t below = (1ull << lane) - 1ull;
  int nx = 0;
  float Ssum = 0.0f;
  int tj[NCH];   // this lane's execution position in chunk c (-1: none)
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    tj[c] = -1;
    if (drop ? c == 0 : nx < kp) {
      const int r = WAVE * c + lane;
      const int e = ov[c];
      const bool cand = (drop ? lane < K : r < E) && e < E && slot_s[e] >= 0;
      const int j = nx + __popcll(__ballot(cand) & below);
      const bool take = cand && (drop || j < kp);
      if (take) tj[c] = j;
      uint64_t mt = __ballot(take);
      nx += __popcll(mt);
      if (renorm) {
        while (mt) {
          const int b = __builtin_ctzll(mt);
          Ssum = Ssum + __builtin_bit_cast(
                            float, __builtin_amdgcn_readlane(__float_as_int(xv[c]), b));
          mt &= mt - 1;
        }
      }
    }
  }
  if (!renorm) Ssum = dv;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    if (tj[c] >= 0) {
      exec_ids[(size_t)t * K + tj[c]] = ov[c];
      exec_gates[(size_t)t * K + tj[c]] = (flags & FLAG_UNIT_GATES) ? 1.0f : xv[c] / Ssum;
    }
  }
  if (lane < K && lane >= nx) {
    exec_ids[(size_t)t * K + lane] = -1;
    exec_gates[(size_t)t * K + lane] = 0.0f;
  }
}

// Exclusive prefixes over slots s < n of cnt[s] (pairs) and ceil(cnt[s] /
// 16) (16-pair tiles), by one wavefront in one pass (SCAN_Q slots per
// lane); index SCAN_N receives each total.
constexpr int SCAN_Q = (MAX_SLOTS + WAVE - 1) / WAVE;
constexpr int SCAN_N = SCAN_Q * WAVE;
__device__ __forceinline__ void wave_scan2(const int *cnt, int n, int *off, int *tb) {
  const int lane = lane_id();
  constexpr int Q = SCAN_Q;
  int l0[Q], l1[Q];
  int s0 = 0, s1 = 0;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int s = lane * Q + q;
    const int c = (s < n) ? cnt[s] : 0;
    l0[q] = c;
    l1[q] = (c + 15) / 16;
    s0 += l0[q]; s1 += l1[q];
  }
  int i0 = s0, i1 = s1;
#pragma unroll
  for (int h = 1; h < WAVE; h <<= 1) {
    const int o0 = __shfl_up(i0, h, WAVE), o1 = __shfl_up(i1, h, WAVE);
    if (lane >= h) { i0 += o0; i1 += o1; }
  }
  int r0 = i0 - s0, r1 = i1 - s1;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int s = lane * Q + q;
    off[s] = r0; tb[s] = r1;
    r0 += l0[q]; r1 += l1[q];
  }
  if (lane == WAVE - 1) { off[SCAN_N] = i0; tb[SCAN_N] = i1; }
}

// hr[s] = slots below s with more than pt 16-pair tiles (s <= SCAN_N;
// hr[SCAN_N]: all of them), from the slots' pair counts, by one wavefront.
__device__ __forceinline__ void wave_scan_multi(const int *cnt, int nslot, int pt, int *hr) {
  const int lane = lane_id();
  constexpr int Q = SCAN_Q;
  int l[Q], s = 0;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int i = lane * Q + q;
    l[q] = (i < nslot && cnt[i] > 16 * pt) ? 1 : 0;
    s += l[q];
  }
  int inc = s;
#pragma unroll
  for (int h = 1; h < WAVE; h <<= 1) {
    const int o = __shfl_up(inc, h, WAVE);
    if (lane >= h) inc += o;
  }
  int r = inc - s;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    hr[lane * Q + q] = r;
    r += l[q];
  }
  if (lane == WAVE - 1) hr[SCAN_N] = inc;
}

// A slot of nt tiles cut into np = ceil(nt / pt) parts of balanced size:
// the first ex = nt % np parts have lo + 1 tiles, the others lo = nt / np.
struct PartSplit {
  int np, lo, ex;
};
__device__ __forceinline__ PartSplit part_split(int nt, int pt) {
  if (nt <= 0) return {0, 0, 0};
  const int np = (nt + pt - 1) / pt;   // pt is a constant: no division
  // nt / np as a multiply-high by ceil(2^16 / np): exact while nt np < 2^16
  // (a slot has at most MAX_B / 16 tiles)
  const int lo = (int)(((uint32_t)nt * ((65536u + (uint32_t)np - 1u) / (uint32_t)np)) >> 16);
  return {np, lo, nt - lo * np};
}
static_assert((MAX_B / 16) * (MAX_B / 16) < 65536, "part_split's quotient");
static_assert((MAX_B / 16) * (FFN_GU_PT + 1) < 65536, "put_tok's quotients");
// pre[j] = cnt[0] + ... + cnt[j - 1] (j <= SCAN_N; pre[SCAN_N]: the
// total), by one wavefront.
__device__ __forceinline__ void wave_scan_counts(const int *cnt, int *pre) {
  const int lane = lane_id();
  constexpr int Q = SCAN_Q;
  int l[Q], s = 0;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    l[q] = cnt[lane * Q + q];
    s += l[q];
  }
  int inc = s;
#pragma unroll
  for (int h = 1; h < WAVE; h <<= 1) {
    const int o = __shfl_up(inc, h, WAVE);
    if (lane >= h) inc += o;
  }
  int r = inc - s;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    pre[lane * Q + q] = r;
    r += l[q];
  }
  if (lane == WAVE - 1) pre[SCAN_N] = inc;
}

constexpr int CP_THREADS = 1024;
constexpr int CP_WAVES = CP_THREADS / WAVE;
constexpr int CP_STAGE = 4096;   // pair gates staged in LDS per pass
constexpr int CP_PAIRS = MAX_B * MAX_K;   // routed pairs at most

// A stable counting sort of the executed pairs by kept slot and (bf16
// layers) the FFN's part tables.  With tables there is one workgroup per
// die, each making the whole sort (the same arithmetic, so the same result
// everywhere) and writing its die's header, units and token rows, which the
// FFN's workgroups on that die then read from their own L2; workgroup 0
// alone writes the plan.  Without tables, one workgroup.
// The routed pairs are taken in flat order q = t K + j, so sorting by (slot,
// q) is sorting by (slot, token, rank).  Wavefront w owns the pairs w 64 PPT
// + r 64 + lane (r = 0 .. PPT - 1, PPT pairs per thread, PPT * CP_THREADS >=
// B K) and ranks each sub-block r without atomics: the lanes holding the same
// slot find each other by ballots over the slot's bits, the lowest of them
// adds their number to the wavefront's own counter of that slot, and every
// lane's rank is that counter's value before the add plus its peers below
// it.  The counters are then turned into prefixes over wavefronts and slots,
// and the pair lists are written through an LDS staging buffer so that the
// global stores are contiguous.  Then ns shared slots (slot n_sel + i runs
// expert E + i for every token in token order, gate sigmoid(gdot[t]) =
// 1 / (1 + exp(-s)) in fp32, or 1); offsets, the pair lists and pair_of
// [B][K + ns].
// With 16 wavefronts on one CU every per-thread instruction costs about 16
// cycles, so the per-pair work is kept short: no division (t = q / K as a
// multiply-high by kmul = ceil(2^32 / K), exact for q < 2^32 / K, far above
// B K), and every global load is issued before the first wait.
//
// The FFN's unit tables (see "Grouped bf16 FFN" in ffn.hip), gate/up's and
// down's.  Slot s (kept slots, then shared ones) has nt = tb[s + 1] - tb[s]
// tiles, cut into parts of balanced size (part_split); a unit is (part, row
// group).  The units are numbered slot by slot, and within a slot row group
// by row group (all of the slot's parts for one row group together, so that
// they read those weight rows through one L2), and the numbering is cut
// into N_XCD runs, die x taking run x.  With at least four slots per die
// the slots are dealt to the dies whole, round-robin, the slots with more
// than one gate/up part first, and numbered die by die, a slot's units part
// by part (a part's row groups together): every slot's units then fall on
// one die in both tables (down finds gate/up's activations in that die's
// L2) and the dies get equal shares as far as whole slots allow.  With
// fewer slots they are numbered in slot order, a slot's units row group by
// row group (all its parts for one row group together), and each table is
// cut into runs of equal numbers of units at row-group boundaries (down at
// the same fraction of the same slot's row groups): a slot's row groups then
// spread over several dies, so that every die has its share of the work.
// A unit's time is mostly its weight stream, so units are what is shared
// out.  Workgroup x
// of the launch writes die x's header, die x's units and gate/up's token
// rows of those units (entry i of unit k's row: the byte offset in x of the
// row of the part's pair i, tokoff[k * FFN_GU_TOK + i], for the part's
// pairs only; gate/up reads no entry at or past the part's pair count).
// Gate/up's row group (row-pair tiles per unit, FFN_WAVES down to
// FFN_WAVES / 2) is the one that gives the fewest row-pair tiles to the
// busiest workgroup when every die's units are shared by its workgroups.
template <int PPT>
__global__ __launch_bounds__(CP_THREADS)
void k_compact(int B, int K, uint64_t kmul, int E, int budget, int ns,
               const int32_t *__restrict__ exec_ids, const float *__restrict__ exec_gates,
               const int32_t *__restrict__ slot_of,
               const int32_t *__restrict__ n_sel_p, const float *__restrict__ gdot,
               int32_t *__restrict__ offsets, int32_t *__restrict__ pair_tok,
               float *__restrict__ pair_gate, int32_t *__restrict__ pair_of,
               const int32_t *__restrict__ sel_ids, int tables, int d, int I,
               uint32_t *__restrict__ tokoff, FfnHdr *__restrict__ hdr,
               FfnUnit *__restrict__ units_gu, FfnUnit *__restrict__ units_dn, int n_cu) {
  // cw[w][s]: pairs of slot s in wavefront w, then their first rank in slot s
  __shared__ int cw[CP_WAVES][MAX_E];
  __shared__ int cnt[SCAN_N];
  __shared__ int off[SCAN_N + 1];
  __shared__ int tb[SCAN_N + 1];
  __shared__ int sel_s[MAX_E];
  __shared__ int slot_s[MAX_E];
  __shared__ int stage_t[CP_PAIRS];     // token of every routed position
  __shared__ float stage_g[CP_STAGE];   // gates, CP_STAGE positions per pass
  // the tables' order: slot s at position pos_s[s] (slot_at: the inverse);
  // parts per position and their prefixes
  __shared__ int pos_s[SCAN_N], slot_at[SCAN_N];
  __shared__ int np_gu[SCAN_N], np_dn[SCAN_N];
  __shared__ int pre_gu[SCAN_N + 1], pre_dn[SCAN_N + 1];
  __shared__ int hr[SCAN_N + 1];
  __shared__ uint32_t sp_s[SCAN_N];      // slot -> its gate/up part split, packed
  __shared__ int cut_s[3][N_XCD + 1];    // die y's first gate/up unit, down unit, slot
  __shared__ uint32_t rc_s[2][SCAN_N];   // slot -> ceil(2^16 / (lo + 1)), ceil(2^16 / lo)
  const int tid = threadIdx.x, lane = lane_id(), wv = wave_id();
  const bool out = blockIdx.x == 0;     // the workgroup that writes the plan
  const int kc = K + ns;   // columns of pair_of
  const int nq = B * K;
  const int q0 = wv * WAVE * PPT + lane;
  // every global load first (clamped indices, no branches): the pairs'
  // experts and gates, the kept list, the slot map, n_sel, the token's
  // shared-expert gate
  int u_r[PPT];
  float g_r[PPT];
#pragma unroll
  for (int r = 0; r < PPT; ++r) {
    const int qc = min(q0 + r * WAVE, nq - 1);
    u_r[r] = exec_ids[qc];
    g_r[r] = exec_gates[qc];
  }
  const int sel_v = sel_ids[min(tid, budget - 1)];
  const int slot_v = slot_of[min(tid, E - 1)];
  const int n_sel = min(max(*n_sel_p, 0), budget);
  float gs = 1.0f;
  if (gdot) {
    const float e = base_exp(-gdot[min(tid, B - 1)]);
    const float den = 1.0f + e;
    gs = 1.0f / den;
  }
  if (tid < budget) sel_s[tid] = sel_v;
  if (tid < E) slot_s[tid] = slot_v;
  for (int s = lane; s < n_sel; s += WAVE) cw[wv][s] = 0;   // the wavefront's own row
  __syncthreads();
  const int nbits = n_sel > 1 ? 32 - __clz(n_sel - 1) : 0;
  const uint64_t below = (1ull << lane) - 1ull;
  int s_r[PPT], p_r[PPT];
#pragma unroll
  for (int r = 0; r < PPT; ++r) {
    const int u = u_r[r];
    int s = (q0 + r * WAVE < nq && u >= 0 && u < E) ? slot_s[u] : -1;
    s = (s >= 0 && s < n_sel) ? s : -1;
    s_r[r] = s;
    uint64_t peers = __ballot(s >= 0);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (s >> b) & 1;
      const uint64_t m = __ballot(bit);
      peers &= bit ? m : ~m;
    }
    p_r[r] = -1;
    if (s >= 0) {
      const int base = cw[wv][s];
      p_r[r] = base + __popcll(peers & below);
      if ((peers & below) == 0ull) cw[wv][s] = base + __popcll(peers);
    }
  }
  __syncthreads();
  for (int s = tid; s < n_sel; s += CP_THREADS) {
    int run = 0;
#pragma unroll
    for (int w = 0; w < CP_WAVES; ++w) {
      const int c = cw[w][s];
      cw[w][s] = run;
      run += c;
    }
    cnt[s] = run;
  }
  if (tid >= n_sel && tid < n_sel + ns) cnt[tid] = B;
  __syncthreads();
  const int nslot = n_sel + ns;
  const bool whole = nslot >= 4 * N_XCD;   // slots dealt to the dies whole
  if (wv == 0) wave_scan2(cnt, nslot, off, tb);
  if (tables) {
    if (wv == 1 && whole) wave_scan_multi(cnt, nslot, FFN_GU_PT, hr);
    for (int j = tid - 2 * WAVE; j >= 0 && j < SCAN_N; j += CP_THREADS - 2 * WAVE)
      np_gu[j] = np_dn[j] = 0;
  }
  __syncthreads();
  if (tables) {
    // each slot's position, parts and gate/up split (packed for put_tok)
    for (int s = tid; s < nslot; s += CP_THREADS) {
      int j = s;
      if (whole) {
        // deal position r (multi-part slots first) to die r % N_XCD, as its
        // slot r / N_XCD; die y holds ceil((nslot - y) / N_XCD) slots
        const bool multi = hr[s + 1] > hr[s];
        const int r = multi ? hr[s] : hr[SCAN_N] + (s - hr[s]), y = r % N_XCD;
        j = r / N_XCD;
        for (int z = 0; z < y; ++z) j += (nslot - z + N_XCD - 1) / N_XCD;
      }
      const int nt = tb[s + 1] - tb[s];
      const PartSplit sg = part_split(nt, FFN_GU_PT);
      pos_s[s] = j;
      slot_at[j] = s;
      np_gu[j] = sg.np;
      np_dn[j] = part_split(nt, FFN_DN_PT).np;
      // lo (<= FFN_GU_PT) and ex (< np <= MAX_B / 16)
      sp_s[s] = (uint32_t)sg.lo | ((uint32_t)sg.ex << 8);
      rc_s[0][s] = (65536u + (uint32_t)sg.lo) / (uint32_t)(sg.lo + 1);
      rc_s[1][s] = (65536u + (uint32_t)sg.lo - 1u) / (uint32_t)max(sg.lo, 1);
    }
  }
  const int routed = off[n_sel];   // pairs of the kept slots
  if (out && tid <= budget) offsets[tid] = (tid < n_sel) ? off[tid] : routed;
  if (out && tid < ns) offsets[budget + 1 + tid] = off[n_sel + tid + 1];
  // positions, pair_of, every routed position's token and the first pass
  // of gates
#pragma unroll
  for (int r = 0; r < PPT; ++r) {
    const int q = q0 + r * WAVE;
    const int t = (int)(((uint64_t)(uint32_t)q * kmul) >> 32);
    const int s = s_r[r];
    if (s >= 0) {
      p_r[r] += off[s] + cw[wv][s];
      stage_t[p_r[r]] = t;
      if (p_r[r] < CP_STAGE) stage_g[p_r[r]] = g_r[r];
    }
    if (out && q < nq) pair_of[(size_t)t * kc + (q - t * K)] = p_r[r];
  }
  if (tables) {
    __syncthreads();   // the positions' part counts complete
    if (wv < 2) wave_scan_counts(wv == 0 ? np_gu : np_dn, wv == 0 ? pre_gu : pre_dn);
    __syncthreads();
    // every thread derives the same row group and runs
    const int x = blockIdx.x;
    const int T = I / 16, Pg = pre_gu[SCAN_N], Pd = pre_dn[SCAN_N];
    const float per_die = (float)(ffn_gu_grid(n_cu) / N_XCD);
    // parts on the busiest die: dealt slots, or an even share
    int pmax = (Pg + N_XCD - 1) / N_XCD;
    if (whole) {
      pmax = 0;
      for (int y = 0, j = 0; y < N_XCD; ++y) {
        const int jn = j + (nslot - y + N_XCD - 1) / N_XCD;
        pmax = max(pmax, pre_gu[jn] - pre_gu[j]);
        j = jn;
      }
    }
    int rp = FFN_WAVES, best_cost = 0x7FFFFFFF;
    for (int c = FFN_WAVES; c >= FFN_WAVES / 2; --c) {
      // the busiest die's units: its dealt parts' row groups, or an equal
      // share of all of them
      const int units = whole ? pmax * ((T + c - 1) / c)
                              : (Pg * ((T + c - 1) / c) + N_XCD - 1) / N_XCD;
      // rounds = ceil(units / per_die); exact in fp32 for these small integers
      const int cost = (int)ceilf((float)units / per_die) * c;
      if (cost < best_cost) { rp = c; best_cost = cost; }
    }
    // down's row group: FFN_WAVES row tiles, or for a long contraction (one
    // workgroup per CU) fewer when that gives the busiest workgroup fewer
    const int Td = d / 16;
    int rd = FFN_WAVES;
    if (ffn_dn_long(I)) {
      int pdmax = (Pd + N_XCD - 1) / N_XCD;
      if (whole) {
        pdmax = 0;
        for (int y = 0, j = 0; y < N_XCD; ++y) {
          const int jn = j + (nslot - y + N_XCD - 1) / N_XCD;
          pdmax = max(pdmax, pre_dn[jn] - pre_dn[j]);
          j = jn;
        }
      }
      const float wgs = (float)(ffn_dn_grid(n_cu, 2) / N_XCD);
      int best = 0x7FFFFFFF;
      for (int c = FFN_WAVES; c >= 2; c /= 2) {
        const int units = whole ? pdmax * ((Td + c - 1) / c)
                                : (Pd * ((Td + c - 1) / c) + N_XCD - 1) / N_XCD;
        const int cost = (int)ceilf((float)units / wgs) * c;
        if (cost < best) { rd = c; best = cost; }
      }
    }
    const int ug = (T + rp - 1) / rp, ud = (Td + rd - 1) / rd;
    // die y's first unit in both tables and first position.  Whole slots:
    // the first position of die y.  Otherwise, from the target gate/up unit
    // Pg ug y / N_XCD at position j: the start of its row group r of ug, and
    // in down of row group r ud / ug at j (one pass: the thread of the
    // position holding a target writes its cut).
    int g0, g1, d0, d1, s0, s1;   // this die's runs; their positions lie in [s0, s1]
    if (whole) {
      // every thread finds its own die's first positions
      int j0 = 0;
      for (int z = 0; z < x; ++z) j0 += (nslot - z + N_XCD - 1) / N_XCD;
      const int j1 = j0 + (nslot - x + N_XCD - 1) / N_XCD;
      g0 = pre_gu[j0] * ug; g1 = pre_gu[j1] * ug;
      d0 = pre_dn[j0] * ud; d1 = pre_dn[j1] * ud;
      s0 = min(j0, nslot - 1); s1 = min(j1, nslot - 1);
    } else {
      for (int j = tid; j < nslot; j += CP_THREADS) {
        const int a = pre_gu[j] * ug, b = pre_gu[j + 1] * ug;
        for (int y = 1; y < N_XCD; ++y) {
          const int i = Pg * ug * y / N_XCD;
          if (i >= a && i < b) {
            const int r = (i - a) / np_gu[j];
            cut_s[0][y] = a + r * np_gu[j];
            cut_s[1][y] = pre_dn[j] * ud + (r * ud / ug) * np_dn[j];
            cut_s[2][y] = j;
          }
        }
      }
      if (tid == 0) {
        for (int y = 0; y < N_XCD && Pg == 0; ++y)   // no units: no position holds a cut
          cut_s[0][y] = cut_s[1][y] = cut_s[2][y] = 0;
        cut_s[0][0] = cut_s[1][0] = cut_s[2][0] = 0;
        cut_s[0][N_XCD] = Pg * ug;
        cut_s[1][N_XCD] = Pd * ud;
        cut_s[2][N_XCD] = max(nslot - 1, 0);
      }
      __syncthreads();
      g0 = cut_s[0][x]; g1 = cut_s[0][x + 1];
      d0 = cut_s[1][x]; d1 = cut_s[1][x + 1];
      s0 = cut_s[2][x]; s1 = cut_s[2][x + 1];
    }
    if (tid == 0) {
      FfnHdr h;
      h.rp_gu = rp;
      h.gu0 = g0; h.gu1 = g1; h.dn0 = d0; h.dn1 = d1;
      h.rt_dn = rd;
      h.pad1 = h.pad2 = 0;
      hdr[x] = h;
    }
    // unit i: its position (the first j with pre[j + 1] * upp > i) and
    // slot, then row group and part
    auto put_unit = [&](int i, int upp, const int *pre, const int *np, int pt, FfnUnit *dst) {
      int lo = s0, hi = s1;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (pre[mid + 1] * upp > i) hi = mid; else lo = mid + 1;
      }
      const int j = lo, s = slot_at[j], r = i - pre[j] * upp;
      const int rg = whole ? r % upp : r / np[j], q = whole ? r / upp : r % np[j];
      const PartSplit sp = part_split(tb[s + 1] - tb[s], pt);
      const int c = q < sp.ex ? sp.lo + 1 : sp.lo;
      const int tf = q * sp.lo + min(q, sp.ex);   // the part's first tile in its slot
      FfnUnit rec;
      rec.u = s < n_sel ? sel_s[s] : E + (s - n_sel);
      rec.tile0 = tb[s] + tf;
      rec.nt = c;
      rec.p0 = off[s] + 16 * tf;
      rec.n = min(16 * c, cnt[s] - 16 * tf);
      rec.rg = rg;
      rec.pad0 = rec.pad1 = 0;
      dst[i] = rec;
    };
    for (int i = g0 + tid; i < g1; i += CP_THREADS) put_unit(i, ug, pre_gu, np_gu, FFN_GU_PT, units_gu);
    for (int i = d0 + tid; i < d1; i += CP_THREADS) put_unit(i, ud, pre_dn, np_dn, FFN_DN_PT, units_dn);
    // gate/up's token row of pair pr of slot s (token t), in every unit of
    // its part in [g0, g1).  The
    // part of tile ti: the first ex parts have lo + 1 tiles, the others lo;
    // the quotients as multiply-highs by ceil(2^16 / divisor), exact for
    // ti < 2^16 / (FFN_GU_PT + 1) (a slot has at most MAX_B / 16 tiles).
    auto put_tok = [&](int s, int pr, int t) {
      const int j = pos_s[s];
      if (pre_gu[j + 1] * ug <= g0 || pre_gu[j] * ug >= g1) return;   // not on this die
      const uint32_t pk = sp_s[s];
      const int lo = (int)(pk & 0xFFu), ex = (int)(pk >> 8);
      const int ti = pr >> 4, big = ex * (lo + 1);
      const uint32_t a = (uint32_t)(ti < big ? ti : ti - big);
      const int qq = (int)((a * rc_s[ti < big ? 0 : 1][s]) >> 16);
      const int q = ti < big ? qq : ex + qq;
      const int tf = q * lo + min(q, ex);
      // the part's units, base + rg n (n = 1 when numbered part by part),
      // in [g0, g1)
      const int n = whole ? 1 : np_gu[j];
      const int base = pre_gu[j] * ug + (whole ? q * ug : q);
      int rg0, rg1;
      if (whole) {   // n = 1: no division
        rg0 = max(g0 - base, 0);
        rg1 = min(ug, max(g1 - base, 0));
      } else {
        rg0 = g0 > base ? (g0 - base + n - 1) / n : 0;
        rg1 = min(ug, g1 > base ? (g1 - base + n - 1) / n : 0);
      }
      const uint32_t v = (uint32_t)t * (uint32_t)d * 2u;
      for (int rg = rg0; rg < rg1; ++rg)
        tokoff[(size_t)(base + rg * n) * FFN_GU_TOK + (pr - 16 * tf)] = v;
    };
#pragma unroll
    for (int r = 0; r < PPT; ++r)
      if (s_r[r] >= 0)
        put_tok(s_r[r], p_r[r] - off[s_r[r]], (int)(((uint64_t)(uint32_t)(q0 + r * WAVE) * kmul) >> 32));
    if (tid < B)
      for (int i = 0; i < ns; ++i) put_tok(n_sel + i, tid, tid);
  }
  if (!out) return;
  __syncthreads();
  for (int i = tid; i < routed; i += CP_THREADS) pair_tok[i] = stage_t[i];
  // the gates, CP_STAGE positions per pass
  for (int c0 = 0; c0 < routed; c0 += CP_STAGE) {
    if (c0 > 0) {
#pragma unroll
      for (int r = 0; r < PPT; ++r) {
        const int i = p_r[r] - c0;
        if (s_r[r] >= 0 && i >= 0 && i < CP_STAGE) stage_g[i] = g_r[r];
      }
      __syncthreads();
    }
    const int n = min(CP_STAGE, routed - c0);
    for (int i = tid; i < n; i += CP_THREADS) pair_gate[c0 + i] = stage_g[i];
    __syncthreads();
  }
  if (tid < B) {
    for (int i = 0; i < ns; ++i) {
      const int p = off[n_sel + i] + tid;
      pair_tok[p] = tid;
      pair_gate[p] = gs;
      pair_of[(size_t)tid * kc + K + i] = p;
    }
  }
}

hipError_t launch_select(int B, int K, int E, const int32_t *ids,
                         const float *cost, int budget, bool binary, float *scores,
                         int32_t *counts, int32_t *sel_ids, int32_t *n_sel,
                         int32_t *slot_of, hipStream_t st) {
  launch_k(k_select, dim3(1), dim3(SEL_THREADS), 0, st, B, K, E, ids,
                     cost, budget, (int)binary, scores, counts, sel_ids, n_sel, slot_of);
  return hipGetLastError();
}

hipError_t launch_select_backfill(int B, int K, int E, const int32_t *ids, const float *cost,
                                  int budget, bool binary, int flags, const uint8_t *order,
                                  const float *ex, const float *den, float *scores,
                                  int32_t *counts, int32_t *sel_ids, int32_t *n_sel,
                                  int32_t *slot_of, int32_t *exec_ids, float *exec_gates,
                                  hipStream_t st) {
  const dim3 grid(xcd_grid((B + TOK_GROUP - 1) / TOK_GROUP, TOK_GROUP / SB_TOK));
#define BASE_SB(C)                                                                         \
  launch_k(k_select_backfill<C>, grid, dim3(SEL_THREADS), 0, st, B, K, E, ids, cost, budget, \
           (int)binary, flags, order, ex, den, scores, counts, sel_ids, n_sel, slot_of,     \
           exec_ids, exec_gates)
  if (E <= WAVE) BASE_SB(1);
  else if (E <= 2 * WAVE) BASE_SB(2);
  else BASE_SB(4);
#undef BASE_SB
  return hipGetLastError();
}

hipError_t launch_backfill(int B, int E, int K, int norm_topk, int flags,
                           const float *logits, const int32_t *ids,
                           const int32_t *slot_of, const int32_t *n_sel,
                           int32_t *exec_ids, float *exec_gates,
                           hipStream_t st) {
  launch_k(k_backfill, dim3((B + BF_WAVES - 1) / BF_WAVES),
                     dim3(BF_WAVES * WAVE), 0, st, B, E, K, norm_topk, flags,
                     logits, ids, slot_of, n_sel, exec_ids, exec_gates);
  return hipGetLastError();
}

hipError_t launch_compact(int B, int K, int E, int budget, int ns, const int32_t *exec_ids,
                          const float *exec_gates, const int32_t *slot_of,
                          const int32_t *n_sel, const float *gdot, int32_t *offsets,
                          int32_t *pair_tok, float *pair_gate,
                          int32_t *pair_of, const int32_t *sel_ids, bool tables, int d,
                          int I, uint32_t *tokoff, FfnHdr *hdr, FfnUnit *units_gu,
                          FfnUnit *units_dn, int n_cu, hipStream_t st) {
  const int ppt = (B * K + CP_THREADS - 1) / CP_THREADS;
  const uint64_t kmul = ((1ull << 32) + (uint64_t)K - 1) / (uint64_t)K;
  const unsigned blocks = tables ? N_XCD : 1u;   // one workgroup per die
#define BASE_COMPACT(P)                                                                    \
  launch_k(k_compact<P>, dim3(blocks), dim3(CP_THREADS), 0, st, B, K, kmul, E, budget, ns, \
           exec_ids, exec_gates, slot_of, n_sel, gdot, offsets, pair_tok, pair_gate,      \
           pair_of, sel_ids, (int)tables, d, I, tokoff, hdr, units_gu, units_dn, n_cu)
  if (ppt <= 1) BASE_COMPACT(1);
  else if (ppt <= 2) BASE_COMPACT(2);
  else if (ppt <= 4) BASE_COMPACT(4);
  else if (ppt <= 8) BASE_COMPACT(8);
  else BASE_COMPACT(16);
#undef BASE_COMPACT
  return hipGetLastError();
}

}  // namespace basek
