/*
 * base.h -- C ABI of an MI355X (gfx950) implementation of the decode hot path
 * of BASE (Batch-Aware Selection of Experts using predicted removal error).
 *
 * One MoE layer, one decode step, batch B (one token per active sequence):
 *
 *   route          l = x W_r^T + beta, top-K, router weights      (Sec. 3.1)
 *   predict_cost   c(t,u) = w^2 exp(a_u . x/||x|| + b_u)   (Sec. 3.4, eq.
 *                  log_energy_predictor; App. "Custom GPU Kernels")
 *   select         D_hat_u = sum_t c(t,u); keep the budget experts with the
 *                  largest D_hat among the batch union             (Sec. 3.4)
 *   moe_forward    backfill each token onto the kept set, compact tokens by
 *                  expert, grouped SwiGLU FFN over the kept experts only,
 *                  gate-weighted combine                     (Sec. 3.5, 3.1)
 *   decode_layer   all of the above in one call
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers named in a base_layer and every array argument are DEVICE
 *   pointers; `L`, `plan_out` and the return values are host memory.
 * - `stream` is a hipStream_t (NULL = the null stream).  Every call only
 *   enqueues work on it: no allocation, no host synchronisation, no
 *   device-to-host copy.  Outputs are valid once the stream reaches them.
 *   Kernels are launched with ordinary launches, so a call made while the
 *   stream is being captured (hipStreamBeginCapture) is recorded into the
 *   graph; replays read the buffers the captured call was given.
 * - The caller owns every buffer.  Calls that need scratch memory take a
 *   workspace `ws` of at least base_workspace_bytes(L, B, budget) bytes.
 * - Validation happens on the host before anything is enqueued; on any
 *   error the call returns a negative base_status and leaves every output
 *   untouched.  A failed launch returns BASE_ERR_HIP.
 * - Input values are not checked (NaN/Inf give unspecified results).
 * - Integer outputs (ids, selected set, executed experts, compaction) and
 *   every fp32 value of the scoring path are bit-deterministic and follow
 *   one fixed fp32 operation order: dot products of length d use 64 partial
 *   sums (partial j owns elements 256m + 4j + r, accumulated in ascending
 *   order with single-rounding FMA) joined by a halving tree; batch scores
 *   sum 64-token chunks by the same tree and chunks in ascending order;
 *   exp is a fixed Cody-Waite + degree-7 polynomial sequence; division and
 *   square root are correctly rounded.  The FFN output is deterministic
 *   run to run.
 * - Ties: wherever experts are ranked by a float key, equal keys are
 *   ordered by the lower expert index.
 *
 * Limits (else BASE_ERR_SHAPE): 1 <= B <= 1024; d a multiple of 256 with
 * d <= 16384; 1 <= K <= 16; K <= E <= 256; I a multiple of 64 with
 * I <= 32768.  budget >= 1 (else BASE_ERR_BUDGET); a budget above E is
 * clamped to E.
 */
#ifndef BASE_MI355X_BASE_H
#define BASE_MI355X_BASE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BASE_OK = 0,
    BASE_ERR_NULL = -1,       /* a required pointer is NULL */
    BASE_ERR_SHAPE = -2,      /* B, d, E, K or I outside the limits above */
    BASE_ERR_BUDGET = -3,     /* budget < 1 */
    BASE_ERR_DTYPE = -4,      /* unknown dtype */
    BASE_ERR_ALIGN = -5,      /* misaligned pointer (see base_layer) */
    BASE_ERR_WORKSPACE = -6,  /* workspace smaller than base_workspace_bytes */
    BASE_ERR_HIP = -7,        /* a HIP launch failed */
    BASE_ERR_FLAGS = -8       /* unknown bits in flags, or unknown score_rule */
} base_status;

/* Element type of x, y, residual and the expert weights w13, w2.  Router
 * and predictor parameters are always fp32. */
typedef enum { BASE_F32 = 0, BASE_BF16 = 1 } base_dtype;

/* flags of base_moe_forward / base_decode_layer */
enum {
    /* Gate of an executed expert v of token t: its original router score
     * exp(l_v - l_max) over the router's own denominator (the original
     * top-K sum), also for backfilled experts (Sec. 3.5).  Default. */
    BASE_GATE_PAPER = 0,
    /* ... or renormalised over the experts the token executes. */
    BASE_GATE_RENORM = 1,
    /* A token executes its K highest-ranked experts inside the kept set,
     * backfilling unavailable routes (Sec. 3.5).  Default. */
    BASE_FILL_BACKFILL = 0,
    /* ... or only its routed experts that were kept (fill-rule ablation,
     * Sec. 4, Table fill_rule_ablation). */
    BASE_FILL_DROP = 2
};

/* Selection rule of a layer (base_layer.score_rule): the per-pair score
 * whose sum over the batch, D_u = sum_{t: u in R_t} score(t, u), ranks the
 * experts (App. "Selection-rule ablation", Table selection_score_ablation).
 * Every rule keeps min(budget, |union|) experts of the batch union, ties to
 * the lower index, and feeds the same backfill. */
enum {
    /* predicted removal error w^2 exp(a_u . x/||x|| + b_u) (Sec. 3.4,
     * eq. log_energy_predictor).  The method; default. */
    BASE_SCORE_BASE = 0,
    /* top-1 union: 1 for the token's first route, 0 for its others; the
     * experts are ranked by membership (D_u > 0), then index, so a budget
     * equal to the union's size keeps exactly the union. */
    BASE_SCORE_TOP1 = 1,
    /* router-weight sum: w */
    BASE_SCORE_WEIGHT = 2,
    /* squared router-weight sum: w^2 (one fp32 product) */
    BASE_SCORE_WEIGHT_SQ = 3,
    /* static expert energy: w^2 mu_u with mu_u the expert's mean
     * calibration energy, given as pred_b = log mu_u; computed as the
     * predictor's sequence with a_u . x/||x|| = 0, (w * w) * exp(b_u).
     * pred_a is not read. */
    BASE_SCORE_STATIC = 4
};

/* Layout of the expert weights w13 and w2 (see base_pack_experts). */
enum {
    /* w13 [E][2I][d], w2 [E][d][I], row-major */
    BASE_W_ROWMAJOR = 0,
    /* the same values permuted by base_pack_experts so that every MFMA
     * operand fragment of the FFN is one contiguous 1 KiB block and each
     * wavefront of the FFN reads one contiguous stream (bf16 only) */
    BASE_W_PACKED = 1
};

/* One MoE layer.  Host struct holding device pointers. */
typedef struct base_layer {
    int32_t d;          /* hidden size */
    int32_t E;          /* routed experts */
    int32_t K;          /* experts per token (router top-K) */
    int32_t I;          /* SwiGLU intermediate size */
    int32_t dtype;      /* base_dtype of x, y, residual, w13, w2 */
    int32_t norm_topk;  /* 1: w = p / sum_{top-K} p ; 0: w = softmax p */
    int32_t w_layout;   /* BASE_W_ROWMAJOR or BASE_W_PACKED */
    int32_t score_rule; /* BASE_SCORE_* (0: the method's predicted error) */
    const float *w_router;  /* [E][d] fp32, 16-B aligned */
    const float *b_router;  /* [E] fp32 router bias, or NULL */
    const float *pred_a;    /* [E][d] fp32 predictor slopes a_u, 16-B
                               aligned; read by BASE_SCORE_BASE only */
    const float *pred_b;    /* [E] fp32 predictor intercepts b_u (bias
                               correction folded in, App. A), or log mu_u
                               for BASE_SCORE_STATIC; not read by the
                               router-only rules */
    const void *w13;        /* [E][2I][d]: rows 0..I-1 gate, I..2I-1 up;
                               16-B aligned */
    const void *w2;         /* [E][d][I] down projection; 16-B aligned */
    /* Shared experts: always active for every token, outside the budget
     * and the selection (the paper leaves them out of its notation, Sec.
     * 3.1; its DeepSeek-V2-Lite and Qwen1.5-MoE models have them).  bf16
     * layers only (else BASE_ERR_DTYPE).  Each has the routed experts'
     * shape; a wider shared expert (intermediate size m I) is given as m of
     * them: its gate rows, up rows and down columns cut into m consecutive
     * blocks of I. */
    int32_t n_shared;          /* 0 .. BASE_MAX_SHARED */
    const void *w13_shared;    /* [n_shared][2I][d], layout w_layout; 16-B aligned */
    const void *w2_shared;     /* [n_shared][d][I], layout w_layout; 16-B aligned */
    const float *shared_gate;  /* [d] fp32: the shared experts' outputs are
                                  scaled by sigmoid(x_t . shared_gate), or NULL:
                                  by 1 */
} base_layer;

#define BASE_MAX_SHARED 8

/* Device pointers into the caller's workspace, filled by base_moe_forward
 * and base_decode_layer when plan_out != NULL.  Arrays not produced by the
 * call are set to NULL.  Valid until the workspace is reused. */
typedef struct base_plan {
    /* produced by base_decode_layer only */
    float   *logits;          /* [B][E] */
    int32_t *topk_ids;        /* [B][K] */
    float   *topk_w;          /* [B][K] */
    float   *cost;            /* [B][K] */
    float   *scores;          /* [E] */
    int32_t *counts;          /* [E] */
    int32_t *sel_ids;         /* [budget] */
    int32_t *n_sel;           /* [1] */
    int32_t *slot_of_expert;  /* [E] */
    /* produced by both */
    int32_t *exec_ids;        /* [B][K] expert executed at rank j, -1 padded */
    float   *exec_gates;      /* [B][K] its gate, 0 padded */
    int32_t *offsets;         /* [budget+n_shared+1] first pair of each
                                 slot: kept slots 0 .. n_sel-1, then the
                                 routed pair count up to index budget, then
                                 shared expert i at budget+i (B pairs each,
                                 after every routed pair) */
    int32_t *pair_tok;        /* [B*K + n_shared*B] token of pair p (pairs
                                 sorted by (slot, token)) */
    float   *pair_gate;       /* [B*K + n_shared*B] gate of pair p */
    int32_t *pair_of;         /* [B][K+n_shared] pair index of (t, j), -1 if
                                 none; j >= K: shared expert j-K */
} base_plan;

/* Bytes of workspace base_moe_forward / base_decode_layer need for this
 * layer, batch and budget (0 if the shape is invalid).  The workspace must
 * be 256-byte aligned. */
size_t base_workspace_bytes(const base_layer *L, int32_t B, int32_t budget);

/* Router (Sec. 3.1; App. "Custom GPU Kernels": the routing stage provides
 * z_t, R_t and w_{t,u}).
 *   x         [B][d] (L->dtype), 16-B aligned
 *   logits    [B][E] fp32 out: l = x . W_r[e] + beta_e
 *   topk_ids  [B][K] int32 out: R_t, ordered by (logit desc, index asc)
 *   topk_w    [B][K] fp32 out: exp(l_u - l_max) / S, S = sum over R_t
 *             (norm_topk = 1) or over all E experts (norm_topk = 0) */
base_status base_route(const base_layer *L, const void *x, int32_t B,
                       float *logits, int32_t *topk_ids, float *topk_w,
                       void *stream);

/* Predicted removal cost of every routed pair (Sec. 3.4, eq.
 * log_energy_predictor): z_bar = x / ||x|| (0 if x = 0),
 * s_hat = a_u . z_bar + b_u, cost = w^2 exp(s_hat).  For a layer with
 * another score_rule, that rule's per-pair score (see BASE_SCORE_*; x is
 * then not read).
 *   topk_ids, topk_w  [B][K] as produced by base_route
 *   cost              [B][K] fp32 out */
base_status base_predict_cost(const base_layer *L, const void *x, int32_t B,
                              const int32_t *topk_ids, const float *topk_w,
                              float *cost, void *stream);

/* Batch aggregation and budgeted selection (Sec. 3.4; Sec. 3.5 "loads the M
 * experts with the largest scores").
 *   scores          [E] fp32 out: D_hat_u = sum of cost over tokens routing u
 *   counts          [E] int32 out: number of tokens routing u
 *   sel_ids         [budget] int32 out: the kept experts in rank order
 *                   (D_hat desc, index asc; for BASE_SCORE_TOP1 layers
 *                   (D_hat > 0) desc, index asc) among experts with
 *                   count > 0; -1 beyond n_sel
 *   n_sel           [1] int32 out: min(budget, |batch union|)
 *   slot_of_expert  [E] int32 out: rank of u in sel_ids, or -1
 * Route ids are device data and are not validated: an id outside [0, E)
 * is ignored here and read as expert 0 by moe_forward; no access goes out
 * of bounds, and the results are then unspecified. */
base_status base_select(const base_layer *L, int32_t B,
                        const int32_t *topk_ids, const float *cost,
                        int32_t budget, float *scores, int32_t *counts,
                        int32_t *sel_ids, int32_t *n_sel,
                        int32_t *slot_of_expert, void *stream);

/* Re-routing onto the kept set and the restricted MoE (Sec. 3.5; Sec. 3.1):
 * backfill (or drop) per token, gates per `flags`, compaction of the
 * executed (token, expert) pairs by kept slot, grouped SwiGLU FFN over the
 * kept experts only -- each kept expert's weights are read once -- and
 *   y_t = residual_t + sum_j gate_{t,j} E_{X_t[j]}(x_t)   (j ascending)
 *         + sum_i g_t S_i(x_t)   (shared experts, i ascending; g_t =
 *         sigmoid(x_t . shared_gate) with the dot product in the fixed
 *         order above and 1 / (1 + exp(-s)) in fp32, or 1).
 *   logits, topk_ids          from base_route
 *   sel_ids, n_sel, slot_of_expert   from base_select (same budget)
 *   residual  [B][d] (L->dtype) or NULL
 *   y         [B][d] (L->dtype) out, 16-B aligned; may not alias x
 *   plan_out  host struct, may be NULL
 *   ws        workspace, ws_bytes >= base_workspace_bytes(L, B, budget) */
base_status base_moe_forward(const base_layer *L, const void *x, int32_t B,
                             const float *logits, const int32_t *topk_ids,
                             const int32_t *sel_ids, const int32_t *n_sel,
                             const int32_t *slot_of_expert, int32_t budget,
                             int32_t flags, const void *residual, void *y,
                             base_plan *plan_out, void *ws, size_t ws_bytes,
                             void *stream);

/* The whole layer in one call: route, predict, select and moe_forward.
 * Every intermediate lives in the workspace (reported through plan_out)
 * and equals, bit for bit, what the staged calls produce. */
base_status base_decode_layer(const base_layer *L, const void *x, int32_t B,
                              int32_t budget, int32_t flags,
                              const void *residual, void *y,
                              base_plan *plan_out, void *ws, size_t ws_bytes,
                              void *stream);

/* For callers that cannot allocate device memory (code under stream
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * layer as base_decode_layer, with the workspace replaced by a fixed scratch
 * array the library holds on each GPU it runs on (BASE_NOALLOC_SCRATCH_BYTES,
 * a static device array, kept until the process ends).  The call allocates
 * nothing and calls no allocating routine; the caller still owns x, y and
 * residual.  Results are bit for bit those of base_decode_layer.
 *   Limit: a layer, batch and budget whose base_workspace_bytes exceeds
 *          BASE_NOALLOC_SCRATCH_BYTES returns BASE_ERR_WORKSPACE (64 MiB
 *          covers, e.g., d = 2048, E = 128, K = 8, I = 768 at B = 256 with
 *          any budget up to E).
 *   plan_out: pointers into the GPU's scratch array, valid until the next
 *          call on that GPU.
 *   Sharing: every call on one GPU uses that GPU's one array, which keeps
 *          the last call's contents (nothing in it needs to start at zero:
 *          every value a call reads is written by the same call first).
 *          Calls that overlap on one GPU -- from several host threads or on
 *          several streams without ordering between them -- race; the
 *          caller orders them.
 *   Errors: as base_decode_layer, checked on the host before anything is
 *          enqueued; BASE_ERR_HIP if the scratch array's address cannot be
 *          taken on the current device. */
#define BASE_NOALLOC_SCRATCH_BYTES (64u << 20)
base_status base_decode_layer_noalloc(const base_layer *L, const void *x, int32_t B,
                                      int32_t budget, int32_t flags,
                                      const void *residual, void *y,
                                      base_plan *plan_out, void *stream);

/* Packed expert weights (BASE_W_PACKED).  A one-time permutation, done when
 * a model is loaded; the values are unchanged.  The shared experts of a
 * packed layer are packed the same way, by a call whose L has E = n_shared
 * and w13, w2 = w13_shared, w2_shared (K and n_shared are not read).  With 16-row tiles and
 * 32-element k-steps, a "fragment" is 16 rows x 32 elements of one matrix,
 * stored as 64 lanes x 8 consecutive elements (lane l: row l % 16,
 * elements 8 (l / 16) .. +7 of the k-step).  Rows are grouped four tiles at
 * a time: for w13 group g (g < I/32) holds gate rows 32g..32g+31 (tiles 0,
 * 1) and up rows I+32g..I+32g+31 (tiles 2, 3); for w2 group g (g < d/64)
 * holds rows 64g..64g+63 (tiles 0..3).  Storage order:
 * [E][group][k-step][tile 0..3][fragment], so each group is one contiguous
 * stream read by one wavefront of the FFN.  Sizes equal the row-major
 * sizes.
 *   L          layer with dtype BASE_BF16 and row-major w13, w2 (inputs)
 *   w13_packed [E * 2I * d] bf16 out, 16-B aligned, may not alias L->w13
 *   w2_packed  [E * d * I] bf16 out, 16-B aligned, may not alias L->w2
 * Returns BASE_ERR_DTYPE for fp32 layers. */
base_status base_pack_experts(const base_layer *L, void *w13_packed,
                              void *w2_packed, void *stream);

/* Calibration statistics of the predictor (Sec. 3.4; App. A "Calibration
 * Details"), accumulated batch by batch on the device; the fit is
 * base_calib_fit (base_calib.h).  For a batch z [B][d] (L->dtype) of
 * calibration hidden states, every routed pair (t, u) (router top-K of
 * L's router) gets the target y = log(||E_u(z_t)||^2 + 1e-12), the expert's
 * own output (the layer's FFN with every routed expert kept, gate 1), and
 * z_bar = z_t / ||z_t|| (fp64); per expert u the statistics add
 *   n_u, sum y, sum y^2                (fp64),
 *   sum z_bar [d], sum z_bar y [d]     (fp64),
 *   G_u = sum z_bar z_bar^T [d][d]     (fp32 products and sums per batch,
 *                                       on the matrix cores, then one add).
 * G_u is kept exactly symmetric: each call reads only the blocks on and
 * above the diagonal (128 x 128 blocks) and writes the new values there and,
 * transposed, below; statistics not made by base_calib_reset and this call
 * must be symmetric too.
 * Layout of `stats` (device, 256-B aligned, base_calib_stats_bytes(L)
 * bytes; each array starts on a 256-byte boundary, in this order):
 *   double head[E][4] (n, sum y, sum y^2, unused); double sz[E][d];
 *   double q[E][d]; float G[E][d][d].
 * Every statistic has one writer and a fixed order: results are
 * deterministic.  Shared experts and score_rule are not used.
 * base_calib_reset zeroes the statistics; base_calib_accumulate needs a
 * workspace of base_calib_ws_bytes(L, B) bytes (256-B aligned).  Both only
 * enqueue work, like every call here. */
size_t base_calib_stats_bytes(const base_layer *L);
size_t base_calib_ws_bytes(const base_layer *L, int32_t B);
base_status base_calib_reset(const base_layer *L, void *stats, void *stream);
base_status base_calib_accumulate(const base_layer *L, const void *z, int32_t B,
                                  void *stats, void *ws, size_t ws_bytes,
                                  void *stream);

/* Kernel timing for profiling.  `events` holds 2 * BASE_N_STAGES hipEvent_t
 * handles created by the caller (hipEventCreate), or is NULL to switch
 * timing off (n_events is then ignored).  While set, the calls that run a
 * stage launch its kernel with events[2 i] and events[2 i + 1] attached to
 * the kernel's own dispatch (hipExtLaunchKernel): hipEventElapsedTime of
 * the pair is that kernel's execution time, with nothing added to the
 * stream between kernels.  A stage that launches no kernel (stage 5
 * always) records its pair back to back.
 * Stages: 0 scores (router logits, the shared experts' gate dots), 1 tail
 * (top-K, router weights, the routed pairs' predictor dot products, norms
 * and predicted costs), 2 aggregation + selection,
 * 3 backfill + gates, 4 compaction and the FFN's part tables, 5 (no
 * kernel: FFN gate/up gathers its own token rows), 6 FFN gate/up, 7 FFN
 * down, 8 combine.  base_route runs stages 0 and 1,
 * base_select stage 2, base_moe_forward 3 to 8 (base_predict_cost runs the
 * tail kernel in its cost mode, untimed); base_decode_layer runs all of
 * them except that one
 * kernel makes the selection and the backfill: stage 2 times it and stage 3
 * records its pair back to back.  The setting belongs
 * to the calling host thread; the caller keeps the events alive while it
 * is set.  Calls on a stream that is being captured ignore it (no event is
 * recorded into the graph).
 * Returns BASE_ERR_SHAPE if n_events != 2 * BASE_N_STAGES. */
#define BASE_N_STAGES 9
base_status base_set_stage_events(void *const *events, int32_t n_events);

/* Static description of a status code. */
const char *base_status_string(int32_t status);

#ifdef __cplusplus
}
#endif
#endif /* BASE_MI355X_BASE_H */
