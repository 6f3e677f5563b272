// C ABI of the BASE decode hot path: host-side validation, workspace
// layout and the launch sequence of every call.  Nothing here touches device
// memory; all work is enqueued on the caller's stream.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>

#include "../../include/base.h"
#include "internal.hpp"

namespace {

using namespace basek;

constexpr int FILL_DROP_BIT = BASE_FILL_DROP;
static_assert(FLAG_UNIT_GATES != BASE_GATE_RENORM && FLAG_UNIT_GATES != BASE_FILL_DROP,
              "internal flag bit");

static_assert(SCORE_BASE == BASE_SCORE_BASE && SCORE_TOP1 == BASE_SCORE_TOP1 &&
                  SCORE_WEIGHT == BASE_SCORE_WEIGHT && SCORE_WEIGHT_SQ == BASE_SCORE_WEIGHT_SQ &&
                  SCORE_STATIC == BASE_SCORE_STATIC,
              "selection rule values");

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

size_t elem_bytes(int32_t dtype) { return dtype == BASE_BF16 ? 2 : 4; }

base_status check_layer(const base_layer *L, int32_t B, bool need_router,
                        bool need_pred, bool need_experts) {
  if (L && (L->score_rule < BASE_SCORE_BASE || L->score_rule > BASE_SCORE_STATIC))
    return BASE_ERR_FLAGS;
  if (!L) return BASE_ERR_NULL;
  if (L->dtype != BASE_F32 && L->dtype != BASE_BF16) return BASE_ERR_DTYPE;
  if (B < 1 || B > MAX_B) return BASE_ERR_SHAPE;
  if (L->d < 256 || L->d > 16384 || L->d % 256) return BASE_ERR_SHAPE;
  if (L->K < 1 || L->K > MAX_K || L->E < L->K || L->E > MAX_E) return BASE_ERR_SHAPE;
  if (L->I < 64 || L->I > 32768 || L->I % 64) return BASE_ERR_SHAPE;
  if (L->norm_topk != 0 && L->norm_topk != 1) return BASE_ERR_SHAPE;
  if (L->w_layout != BASE_W_ROWMAJOR && L->w_layout != BASE_W_PACKED) return BASE_ERR_SHAPE;
  if (L->w_layout == BASE_W_PACKED && L->dtype != BASE_BF16) return BASE_ERR_DTYPE;
  if (need_router) {
    if (!L->w_router) return BASE_ERR_NULL;
    if (!aligned(L->w_router, 16)) return BASE_ERR_ALIGN;
    if (L->b_router && !aligned(L->b_router, 4)) return BASE_ERR_ALIGN;
  }
  // the predictor parameters each selection rule reads
  if (need_pred && L->score_rule == BASE_SCORE_BASE) {
    if (!L->pred_a) return BASE_ERR_NULL;
    if (!aligned(L->pred_a, 16)) return BASE_ERR_ALIGN;
  }
  if (need_pred && (L->score_rule == BASE_SCORE_BASE || L->score_rule == BASE_SCORE_STATIC)) {
    if (!L->pred_b) return BASE_ERR_NULL;
    if (!aligned(L->pred_b, 4)) return BASE_ERR_ALIGN;
  }
  if (L->n_shared < 0 || L->n_shared > BASE_MAX_SHARED) return BASE_ERR_SHAPE;
  if (L->n_shared > 0 && L->dtype != BASE_BF16) return BASE_ERR_DTYPE;
  if (L->shared_gate && !aligned(L->shared_gate, 16)) return BASE_ERR_ALIGN;
  if (need_experts) {
    if (!L->w13 || !L->w2) return BASE_ERR_NULL;
    if (!aligned(L->w13, 16) || !aligned(L->w2, 16)) return BASE_ERR_ALIGN;
    if (L->n_shared > 0) {
      if (!L->w13_shared || !L->w2_shared) return BASE_ERR_NULL;
      if (!aligned(L->w13_shared, 16) || !aligned(L->w2_shared, 16)) return BASE_ERR_ALIGN;
    }
  }
  return BASE_OK;
}

// the shared-expert gate vector (only with shared experts)
const float *shared_gate(const base_layer *L) {
  return L->n_shared > 0 ? L->shared_gate : nullptr;
}

base_status check_ptr(const void *p, size_t a) {
  if (!p) return BASE_ERR_NULL;
  return aligned(p, a) ? BASE_OK : BASE_ERR_ALIGN;
}

#define BASE_TRY(expr)                          \
  do {                                          \
    base_status _s = (expr);                    \
    if (_s != BASE_OK) return _s;               \
  } while (0)

#define HIP_TRY(expr)                           \
  do {                                          \
    if ((expr) != hipSuccess) return BASE_ERR_HIP; \
  } while (0)

// Workspace layout: every array starts on a 256-byte boundary.
struct Layout {
  size_t logits, gdot, topk_ids, topk_w, cost, scores, counts, sel_ids, n_sel,
      slot_of, exec_ids, exec_gates, offsets, pair_tok, pair_gate, pair_of, order, ex,
      den, hdr, units_gu, units_dn, tokoff, H, pairbuf, total;
};

size_t up256(size_t v) { return (v + 255) & ~(size_t)255; }

Layout layout(const base_layer *L, int32_t B, int32_t bc) {
  Layout o;
  size_t at = 0;
  auto take = [&](size_t bytes) {
    size_t here = at;
    at = up256(at + bytes);
    return here;
  };
  const size_t BK = (size_t)B * L->K;
  const int ns = L->n_shared;
  const size_t P = BK + (size_t)ns * B;   // routed pairs + shared pairs
  o.logits = take((size_t)B * L->E * 4);
  o.gdot = take((size_t)B * 4);
  o.topk_ids = take(BK * 4);
  o.topk_w = take(BK * 4);
  o.cost = take(BK * 4);
  o.scores = take((size_t)L->E * 4);
  o.counts = take((size_t)L->E * 4);
  o.sel_ids = take((size_t)bc * 4);
  o.n_sel = take(4);
  o.slot_of = take((size_t)L->E * 4);
  o.exec_ids = take(BK * 4);
  o.exec_gates = take(BK * 4);
  o.offsets = take(((size_t)bc + ns + 1) * 4);
  o.pair_tok = take(P * 4);
  o.pair_gate = take(P * 4);
  o.pair_of = take((size_t)B * (L->K + ns) * 4);
  // k_tail's rank order, exp(l - l_max) in rank order and denominators,
  // for the fused layer's backfill
  o.order = take((size_t)B * L->E);
  o.ex = take((size_t)B * L->E * 4);
  o.den = take((size_t)B * 4);
  // the FFN's part tables and their header (bf16)
  const bool bf = L->dtype == BASE_BF16;
  // (one header per die; every die's run of units written on that die)
  const size_t ug = bf ? (size_t)ffn_units_bound_gu(B, L->K, bc, ns, L->I) : 0;
  const size_t ud = bf ? (size_t)ffn_units_bound_dn(B, L->K, bc, ns, L->d) : 0;
  o.hdr = take(bf ? N_XCD * sizeof(FfnHdr) : 0);
  o.units_gu = take(ug * sizeof(FfnUnit));
  o.units_dn = take(ud * sizeof(FfnUnit));
  o.tokoff = take(ug * FFN_GU_TOK * 4);
  if (L->dtype == BASE_BF16) {
    // fragment-ordered SwiGLU activations (16-pair tiles)
    const size_t tiles = (size_t)ffn_max_tiles(B, L->K, bc, ns);
    o.H = take(tiles * 16 * (size_t)L->I * 2);
  } else {
    o.H = take(BK * L->I * 4);
  }
  o.pairbuf = take(P * L->d * 4);
  o.total = at;
  return o;
}

// kernel timing (base_set_stage_events), per host thread
thread_local void *const *g_stage_events = nullptr;
thread_local KernelEvents g_next;

// the events of stage i go to the next kernel launched on st; on a stream
// that is being captured the setting is ignored, so that no event of the
// calling thread's timing set is recorded into a graph
void stage(int i, hipStream_t st) {
  if (!g_stage_events) return;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(st, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return;
  g_next = {(hipEvent_t)g_stage_events[2 * i], (hipEvent_t)g_stage_events[2 * i + 1]};
}

// a stage that launched no kernel records its pair back to back
void stage_end(hipStream_t st) {
  if (g_next.start) {
    (void)hipEventRecord(g_next.start, st);
    (void)hipEventRecord(g_next.stop, st);
    g_next = {};
  }
}

// Compute units of the current device (queried once per device): the FFN
// launches are sized from it.
int device_cus() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) dev = 0;
  const int slot = dev < 64 ? dev : 63;
  int n = cache[slot].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n <= 0)
      n = 256;
    if (dev < 64) cache[slot].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Scratch of base_decode_layer_noalloc: one array of
// BASE_NOALLOC_SCRATCH_BYTES per GPU, held by the library until the process
// ends.  In host code `scratch` names a host-side stand-in, not device
// memory: its device address on the current GPU comes from
// hipGetSymbolAddress, taken once per device (with that device current) on
// the entry point's first call there, and only that address is used.
static __device__ __align__(256) unsigned char scratch[BASE_NOALLOC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::atomic<void *> g_scratch_ptr[MAX_DEVICES];

base_status scratch_of_current_device(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return BASE_ERR_HIP;
  void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    // two threads racing here both store the same address
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return BASE_ERR_HIP;
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return BASE_OK;
}

template <typename T>
T *at(void *ws, size_t off) {
  return reinterpret_cast<T *>(static_cast<char *>(ws) + off);
}

// backfill (unless done with the selection) + compaction + FFN + combine,
// on plan arrays already in place
base_status run_forward(const base_layer *L, const void *x, int32_t B,
                        const float *logits, const int32_t *ids,
                        const int32_t *sel_ids, const int32_t *n_sel,
                        const int32_t *slot_of, int32_t bc, int32_t flags,
                        const void *residual, void *y, void *ws,
                        const Layout &o, hipStream_t st, bool backfilled = false) {
  const bool bf16 = L->dtype == BASE_BF16;
  int32_t *exec_ids = at<int32_t>(ws, o.exec_ids);
  float *exec_gates = at<float>(ws, o.exec_gates);
  int32_t *offsets = at<int32_t>(ws, o.offsets);
  int32_t *pair_tok = at<int32_t>(ws, o.pair_tok);
  float *pair_gate = at<float>(ws, o.pair_gate);
  int32_t *pair_of = at<int32_t>(ws, o.pair_of);
  stage(3, st);
  if (!backfilled)
    HIP_TRY(launch_backfill(B, L->E, L->K, L->norm_topk, flags, logits, ids,
                            slot_of, n_sel, exec_ids, exec_gates, st));
  stage_end(st);
  stage(4, st);
  const int ns = L->n_shared;
  const int n_cu = device_cus();
  FfnHdr *hdr = at<FfnHdr>(ws, o.hdr);
  FfnUnit *units_gu = at<FfnUnit>(ws, o.units_gu), *units_dn = at<FfnUnit>(ws, o.units_dn);
  uint32_t *tokoff = at<uint32_t>(ws, o.tokoff);
  // the same launch lists the FFN's parts and gate/up's token rows (bf16)
  HIP_TRY(launch_compact(B, L->K, L->E, bc, ns, exec_ids, exec_gates, slot_of, n_sel,
                         shared_gate(L) ? at<float>(ws, o.gdot) : nullptr, offsets,
                         pair_tok, pair_gate, pair_of, sel_ids, bf16, L->d, L->I, tokoff,
                         hdr, units_gu, units_dn, n_cu, st));
  stage_end(st);
  stage(5, st);   // no launch of its own: gate/up gathers its tokens itself
  stage_end(st);
  stage(6, st);
  const bool packed = L->w_layout == BASE_W_PACKED;
  HIP_TRY(launch_gateup(bf16, packed, x, B, L->d, L->I, L->E, L->K, bc, ns, L->w13,
                        L->w13_shared, sel_ids, n_sel, offsets, pair_tok, hdr, units_gu, n_cu,
                        tokoff, at<void>(ws, o.H), st));
  stage_end(st);
  stage(7, st);
  HIP_TRY(launch_down(bf16, packed, B, L->d, L->I, L->E, L->K, bc, ns, L->w2,
                      L->w2_shared, sel_ids, n_sel, offsets, hdr, units_dn, n_cu, pair_gate,
                      at<void>(ws, o.H), at<float>(ws, o.pairbuf), st));
  stage_end(st);
  stage(8, st);
  HIP_TRY(launch_combine(bf16, B, L->d, L->K + ns, pair_of, at<float>(ws, o.pairbuf),
                         residual, y, st));
  stage_end(st);
  return BASE_OK;
}

void fill_plan(base_plan *P, void *ws, const Layout &o, bool full) {
  if (!P) return;
  P->logits = full ? at<float>(ws, o.logits) : nullptr;
  P->topk_ids = full ? at<int32_t>(ws, o.topk_ids) : nullptr;
  P->topk_w = full ? at<float>(ws, o.topk_w) : nullptr;
  P->cost = full ? at<float>(ws, o.cost) : nullptr;
  P->scores = full ? at<float>(ws, o.scores) : nullptr;
  P->counts = full ? at<int32_t>(ws, o.counts) : nullptr;
  P->sel_ids = full ? at<int32_t>(ws, o.sel_ids) : nullptr;
  P->n_sel = full ? at<int32_t>(ws, o.n_sel) : nullptr;
  P->slot_of_expert = full ? at<int32_t>(ws, o.slot_of) : nullptr;
  P->exec_ids = at<int32_t>(ws, o.exec_ids);
  P->exec_gates = at<float>(ws, o.exec_gates);
  P->offsets = at<int32_t>(ws, o.offsets);
  P->pair_tok = at<int32_t>(ws, o.pair_tok);
  P->pair_gate = at<float>(ws, o.pair_gate);
  P->pair_of = at<int32_t>(ws, o.pair_of);
}

base_status check_ws(const base_layer *L, int32_t B, int32_t bc, void *ws,
                     size_t ws_bytes) {
  if (!ws) return BASE_ERR_NULL;
  if (!aligned(ws, 256)) return BASE_ERR_ALIGN;
  if (ws_bytes < layout(L, B, bc).total) return BASE_ERR_WORKSPACE;
  return BASE_OK;
}

}  // namespace

namespace basek {
KernelEvents &kernel_events() { return g_next; }
}  // namespace basek

extern "C" {

size_t base_workspace_bytes(const base_layer *L, int32_t B, int32_t budget) {
  if (check_layer(L, B, false, false, false) != BASE_OK || budget < 1) return 0;
  return layout(L, B, budget < L->E ? budget : L->E).total;
}

base_status base_route(const base_layer *L, const void *x, int32_t B,
                       float *logits, int32_t *topk_ids, float *topk_w,
                       void *stream) {
  BASE_TRY(check_layer(L, B, true, false, false));
  BASE_TRY(check_ptr(x, 16));
  BASE_TRY(check_ptr(logits, 4));
  BASE_TRY(check_ptr(topk_ids, 4));
  BASE_TRY(check_ptr(topk_w, 4));
  hipStream_t st = (hipStream_t)stream;
  const bool bf16 = L->dtype == BASE_BF16;
  stage(0, st);
  HIP_TRY(launch_scores(bf16, x, B, L->d, L->w_router, L->b_router, L->E, nullptr, logits,
                        nullptr, st));
  stage_end(st);
  stage(1, st);
  HIP_TRY(launch_tail(bf16, B, L->E, L->K, L->d, L->norm_topk, logits, nullptr, nullptr,
                      nullptr, topk_ids, topk_w, nullptr, 1, BASE_SCORE_BASE, st));
  stage_end(st);
  return BASE_OK;
}

base_status base_predict_cost(const base_layer *L, const void *x, int32_t B,
                              const int32_t *topk_ids, const float *topk_w,
                              float *cost, void *stream) {
  BASE_TRY(check_layer(L, B, false, true, false));
  BASE_TRY(check_ptr(x, 16));
  BASE_TRY(check_ptr(topk_ids, 4));
  BASE_TRY(check_ptr(topk_w, 4));
  BASE_TRY(check_ptr(cost, 4));
  // the method's rule computes the predictor's dot products of the routed
  // pairs; the other rules' scores need only the routes (and pred_b)
  HIP_TRY(launch_tail(L->dtype == BASE_BF16, B, L->E, L->K, L->d, L->norm_topk, nullptr, x,
                      L->pred_a, L->pred_b, const_cast<int32_t *>(topk_ids),
                      const_cast<float *>(topk_w), cost, 2, L->score_rule,
                      (hipStream_t)stream));
  return BASE_OK;
}

base_status base_select(const base_layer *L, int32_t B, const int32_t *topk_ids,
                        const float *cost, int32_t budget, float *scores,
                        int32_t *counts, int32_t *sel_ids, int32_t *n_sel,
                        int32_t *slot_of_expert, void *stream) {
  BASE_TRY(check_layer(L, B, false, false, false));
  if (budget < 1) return BASE_ERR_BUDGET;
  BASE_TRY(check_ptr(topk_ids, 4));
  BASE_TRY(check_ptr(cost, 4));
  BASE_TRY(check_ptr(scores, 4));
  BASE_TRY(check_ptr(counts, 4));
  BASE_TRY(check_ptr(sel_ids, 4));
  BASE_TRY(check_ptr(n_sel, 4));
  BASE_TRY(check_ptr(slot_of_expert, 4));
  const int32_t bc = budget < L->E ? budget : L->E;
  stage(2, (hipStream_t)stream);
  HIP_TRY(launch_select(B, L->K, L->E, topk_ids, cost, bc,
                        L->score_rule == BASE_SCORE_TOP1, scores, counts, sel_ids,
                        n_sel, slot_of_expert, (hipStream_t)stream));
  stage_end((hipStream_t)stream);
  return BASE_OK;
}

base_status base_moe_forward(const base_layer *L, const void *x, int32_t B,
                             const float *logits, const int32_t *topk_ids,
                             const int32_t *sel_ids, const int32_t *n_sel,
                             const int32_t *slot_of_expert, int32_t budget,
                             int32_t flags, const void *residual, void *y,
                             base_plan *plan_out, void *ws, size_t ws_bytes,
                             void *stream) {
  BASE_TRY(check_layer(L, B, false, false, true));
  if (budget < 1) return BASE_ERR_BUDGET;
  if (flags & ~3) return BASE_ERR_FLAGS;
  BASE_TRY(check_ptr(x, 16));
  BASE_TRY(check_ptr(logits, 4));
  BASE_TRY(check_ptr(topk_ids, 4));
  BASE_TRY(check_ptr(sel_ids, 4));
  BASE_TRY(check_ptr(n_sel, 4));
  BASE_TRY(check_ptr(slot_of_expert, 4));
  BASE_TRY(check_ptr(y, 16));
  if (residual && !aligned(residual, 16)) return BASE_ERR_ALIGN;
  const int32_t bc = budget < L->E ? budget : L->E;
  BASE_TRY(check_ws(L, B, bc, ws, ws_bytes));
  const Layout o = layout(L, B, bc);
  if (shared_gate(L))   // the shared experts' gate: its own dot-product launch
    HIP_TRY(launch_scores(L->dtype == BASE_BF16, x, B, L->d, nullptr, nullptr, 0,
                          shared_gate(L), nullptr, at<float>(ws, o.gdot), (hipStream_t)stream));
  BASE_TRY(run_forward(L, x, B, logits, topk_ids, sel_ids, n_sel,
                       slot_of_expert, bc, flags, residual, y, ws, o,
                       (hipStream_t)stream));
  fill_plan(plan_out, ws, o, false);
  return BASE_OK;
}

base_status base_decode_layer(const base_layer *L, const void *x, int32_t B,
                              int32_t budget, int32_t flags,
                              const void *residual, void *y,
                              base_plan *plan_out, void *ws, size_t ws_bytes,
                              void *stream) {
  BASE_TRY(check_layer(L, B, true, true, true));
  if (budget < 1) return BASE_ERR_BUDGET;
  if (flags & ~3) return BASE_ERR_FLAGS;
  BASE_TRY(check_ptr(x, 16));
  BASE_TRY(check_ptr(y, 16));
  if (residual && !aligned(residual, 16)) return BASE_ERR_ALIGN;
  const int32_t bc = budget < L->E ? budget : L->E;
  BASE_TRY(check_ws(L, B, bc, ws, ws_bytes));
  const Layout o = layout(L, B, bc);
  hipStream_t st = (hipStream_t)stream;
  const bool bf16 = L->dtype == BASE_BF16;
  float *logits = at<float>(ws, o.logits);
  int32_t *ids = at<int32_t>(ws, o.topk_ids);
  float *w = at<float>(ws, o.topk_w);
  float *cost = at<float>(ws, o.cost);
  int32_t *sel = at<int32_t>(ws, o.sel_ids);
  int32_t *nsel = at<int32_t>(ws, o.n_sel);
  int32_t *slot = at<int32_t>(ws, o.slot_of);
  stage(0, st);
  HIP_TRY(launch_scores(bf16, x, B, L->d, L->w_router, L->b_router, L->E, shared_gate(L),
                        logits, at<float>(ws, o.gdot), st));
  stage_end(st);
  uint8_t *order = at<uint8_t>(ws, o.order);
  float *ex = at<float>(ws, o.ex), *den = at<float>(ws, o.den);
  stage(1, st);   // top-K, weights, (the method's rule) the routed pairs' predictor,
              // and each token's experts in rank order for the backfill
  HIP_TRY(launch_tail(bf16, B, L->E, L->K, L->d, L->norm_topk, logits, x, L->pred_a,
                      L->pred_b, ids, w, cost, 3, L->score_rule, st, order, ex, den));
  stage_end(st);
  stage(2, st);   // selection and backfill in one launch
  HIP_TRY(launch_select_backfill(B, L->K, L->E, ids, cost, bc,
                                 L->score_rule == BASE_SCORE_TOP1, flags, order, ex, den,
                                 at<float>(ws, o.scores), at<int32_t>(ws, o.counts), sel, nsel,
                                 slot, at<int32_t>(ws, o.exec_ids), at<float>(ws, o.exec_gates),
                                 st));
  stage_end(st);
  BASE_TRY(run_forward(L, x, B, logits, ids, sel, nsel, slot, bc, flags,
                       residual, y, ws, o, st, true));
  fill_plan(plan_out, ws, o, true);
  return BASE_OK;
}

base_status base_decode_layer_noalloc(const base_layer *L, const void *x, int32_t B,
                                      int32_t budget, int32_t flags, const void *residual,
                                      void *y, base_plan *plan_out, void *stream) {
  // the checks base_decode_layer makes, then the size limit, all before the
  // device is touched
  BASE_TRY(check_layer(L, B, true, true, true));
  if (budget < 1) return BASE_ERR_BUDGET;
  if (flags & ~3) return BASE_ERR_FLAGS;
  BASE_TRY(check_ptr(x, 16));
  BASE_TRY(check_ptr(y, 16));
  if (residual && !aligned(residual, 16)) return BASE_ERR_ALIGN;
  const int32_t bc = budget < L->E ? budget : L->E;
  if (layout(L, B, bc).total > (size_t)BASE_NOALLOC_SCRATCH_BYTES) return BASE_ERR_WORKSPACE;
  void *ws = nullptr;
  BASE_TRY(scratch_of_current_device(&ws));
  return base_decode_layer(L, x, B, budget, flags, residual, y, plan_out, ws,
                           (size_t)BASE_NOALLOC_SCRATCH_BYTES, stream);
}

// ------------------------------------------------------------ calibration --
size_t base_calib_stats_bytes(const base_layer *L) {
  if (!L || L->E < 1 || L->E > MAX_E || L->d < 256 || L->d > 16384 || L->d % 256) return 0;
  return calib_stats_bytes(L->E, L->d);
}

// the routed layer the calibration runs (no shared experts, its own rule)
static base_layer calib_layer(const base_layer *L) {
  base_layer C = *L;
  C.n_shared = 0;
  C.score_rule = BASE_SCORE_WEIGHT;
  return C;
}

size_t base_calib_ws_bytes(const base_layer *L, int32_t B) {
  if (!L) return 0;
  const base_layer C = calib_layer(L);
  if (check_layer(&C, B, false, false, false) != BASE_OK) return 0;
  return layout(&C, B, C.E).total + up256((size_t)B * 8) + up256((size_t)B * C.K * 8) +
         up256((size_t)(B + 1) * C.d * 4);
}

base_status base_calib_reset(const base_layer *L, void *stats, void *stream) {
  const size_t n = base_calib_stats_bytes(L);
  if (n == 0) return BASE_ERR_SHAPE;
  BASE_TRY(check_ptr(stats, 256));
  HIP_TRY(launch_calib_zero(stats, n, (hipStream_t)stream));
  return BASE_OK;
}

base_status base_calib_accumulate(const base_layer *L, const void *z, int32_t B, void *stats,
                                  void *ws, size_t ws_bytes, void *stream) {
  if (!L) return BASE_ERR_NULL;
  const base_layer C = calib_layer(L);
  BASE_TRY(check_layer(&C, B, true, false, true));
  BASE_TRY(check_ptr(z, 16));
  BASE_TRY(check_ptr(stats, 256));
  if (!ws) return BASE_ERR_NULL;
  if (!aligned(ws, 256)) return BASE_ERR_ALIGN;
  if (ws_bytes < base_calib_ws_bytes(L, B)) return BASE_ERR_WORKSPACE;
  const int32_t bc = C.E;   // keep every routed expert
  const Layout o = layout(&C, B, bc);
  hipStream_t st = (hipStream_t)stream;
  const bool bf16 = C.dtype == BASE_BF16;
  float *logits = at<float>(ws, o.logits);
  int32_t *ids = at<int32_t>(ws, o.topk_ids);
  float *w = at<float>(ws, o.topk_w);
  int32_t *sel = at<int32_t>(ws, o.sel_ids);
  int32_t *nsel = at<int32_t>(ws, o.n_sel);
  int32_t *slot = at<int32_t>(ws, o.slot_of);
  HIP_TRY(launch_scores(bf16, z, B, C.d, C.w_router, C.b_router, C.E, nullptr, logits,
                        nullptr, st));
  HIP_TRY(launch_tail(bf16, B, C.E, C.K, C.d, C.norm_topk, logits, nullptr, nullptr, nullptr,
                      ids, w, nullptr, 1, BASE_SCORE_BASE, st));
  // the budget E keeps the whole batch union (any positive scores do)
  HIP_TRY(launch_select(B, C.K, C.E, ids, w, bc, false, at<float>(ws, o.scores),
                        at<int32_t>(ws, o.counts), sel, nsel, slot, st));
  // every routed expert executed, with gate 1: the FFN writes E_u(z_t)
  HIP_TRY(launch_backfill(B, C.E, C.K, C.norm_topk, FILL_DROP_BIT | FLAG_UNIT_GATES, logits,
                          ids, slot, nsel, at<int32_t>(ws, o.exec_ids),
                          at<float>(ws, o.exec_gates), st));
  int32_t *offsets = at<int32_t>(ws, o.offsets);
  int32_t *pair_tok = at<int32_t>(ws, o.pair_tok);
  const int n_cu = device_cus();
  FfnHdr *hdr = at<FfnHdr>(ws, o.hdr);
  FfnUnit *units_gu = at<FfnUnit>(ws, o.units_gu), *units_dn = at<FfnUnit>(ws, o.units_dn);
  HIP_TRY(launch_compact(B, C.K, C.E, bc, 0, at<int32_t>(ws, o.exec_ids),
                         at<float>(ws, o.exec_gates), slot, nsel, nullptr, offsets, pair_tok,
                         at<float>(ws, o.pair_gate), at<int32_t>(ws, o.pair_of), sel,
                         bf16, C.d, C.I, at<uint32_t>(ws, o.tokoff), hdr, units_gu, units_dn,
                         n_cu, st));
  const bool packed = C.w_layout == BASE_W_PACKED;
  HIP_TRY(launch_gateup(bf16, packed, z, B, C.d, C.I, C.E, C.K, bc, 0, C.w13, nullptr, sel,
                        nsel, offsets, pair_tok, hdr, units_gu, n_cu, at<uint32_t>(ws, o.tokoff),
                        at<void>(ws, o.H), st));
  HIP_TRY(launch_down(bf16, packed, B, C.d, C.I, C.E, C.K, bc, 0, C.w2, nullptr, sel, nsel,
                      offsets, hdr, units_dn, n_cu, at<float>(ws, o.pair_gate),
                      at<void>(ws, o.H), at<float>(ws, o.pairbuf), st));
  double *inv = at<double>(ws, o.total);
  double *y = at<double>(ws, o.total + up256((size_t)B * 8));
  float *zbuf = at<float>(ws, o.total + up256((size_t)B * 8) + up256((size_t)B * C.K * 8));
  HIP_TRY(launch_calib_stats(z, bf16, B, C.d, C.E, C.K, at<float>(ws, o.pairbuf), nsel, sel,
                             offsets, pair_tok, inv, y, zbuf, calib_stats_at(stats, C.E, C.d),
                             st));
  return BASE_OK;
}

base_status base_pack_experts(const base_layer *L, void *w13_packed,
                              void *w2_packed, void *stream) {
  if (!L) return BASE_ERR_NULL;
  if (L->dtype != BASE_BF16) return BASE_ERR_DTYPE;
  if (L->w_layout != BASE_W_ROWMAJOR) return BASE_ERR_SHAPE;
  // only the expert matrices' shape matters here (E experts of [2I][d] and
  // [d][I]; the shared experts are packed by a call with E = n_shared)
  base_layer C = *L;
  C.K = 1;
  C.n_shared = 0;
  BASE_TRY(check_layer(&C, 1, false, false, true));
  BASE_TRY(check_ptr(w13_packed, 16));
  BASE_TRY(check_ptr(w2_packed, 16));
  HIP_TRY(launch_pack(L->w13, L->w2, w13_packed, w2_packed, L->E, L->d, L->I,
                      (hipStream_t)stream));
  return BASE_OK;
}

base_status base_set_stage_events(void *const *events, int32_t n_events) {
  if (!events) {
    g_stage_events = nullptr;
    return BASE_OK;
  }
  if (n_events != 2 * BASE_N_STAGES) return BASE_ERR_SHAPE;
  for (int i = 0; i < n_events; ++i)
    if (!events[i]) return BASE_ERR_NULL;
  g_stage_events = events;
  return BASE_OK;
}

const char *base_status_string(int32_t status) {
  switch (status) {
    case BASE_OK: return "ok";
    case BASE_ERR_NULL: return "a required pointer is NULL";
    case BASE_ERR_SHAPE: return "shape outside the supported limits";
    case BASE_ERR_BUDGET: return "budget must be at least 1";
    case BASE_ERR_DTYPE: return "unknown dtype";
    case BASE_ERR_ALIGN: return "misaligned pointer";
    case BASE_ERR_WORKSPACE: return "workspace too small";
    case BASE_ERR_HIP: return "HIP launch failed";
    case BASE_ERR_FLAGS: return "unknown flag bits or score rule";
    default: return "unknown status";
  }
}

}  // extern "C"
