// mita_api.hip - the C ABI (include/mita.h): validation, workspace carving and
// the launch sequence of the forward pass (Algorithm 1 order).
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>
#include <vector>

#include "check.hpp"
#include "kernels.hpp"

using namespace mita;

namespace {

thread_local std::string g_err;

int set_err(int status, const std::string &msg) {
  g_err = msg;
  return status;
}

int hip_status(hipError_t e, const char *what) {
  if (e == hipSuccess) return MITA_OK;
  return set_err(MITA_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

int validate(const mita_cfg_t *c) {
  std::string msg;
  const int st = check_cfg(c, &msg);
  if (st != MITA_OK) return set_err(st, msg);
  return MITA_OK;
}

int need_ptr(const void *p, const char *name) {
  if (!p) return set_err(MITA_ERR_INVALID_ARG, std::string(name) + " is NULL");
  if (!aligned16(p)) return set_err(MITA_ERR_INVALID_ARG, std::string(name) + " is not 16-byte aligned");
  return MITA_OK;
}

int need_ws(const mita_cfg_t *c, int which, const void *ws, size_t ws_bytes) {
  const size_t need = workspace_size(c, which);
  if (need == 0) return MITA_OK;
  if (!ws || ws_bytes < need)
    return set_err(MITA_ERR_WORKSPACE, "workspace needs " + std::to_string(need) + " bytes, got " +
                                           std::to_string(ws ? ws_bytes : 0));
  if (((uintptr_t)ws & (WS_ALIGN - 1)) != 0) return set_err(MITA_ERR_INVALID_ARG, "workspace is not 256-byte aligned");
  return MITA_OK;
}

#define TRY(x)                   \
  do {                           \
    const int _s = (x);          \
    if (_s != MITA_OK) return _s; \
  } while (0)

size_t tensor_bytes(const mita_cfg_t *c) { return (size_t)BH(*c) * c->N * c->d * elem_bytes(*c); }

}  // namespace

// Event slots of a timed forward: one event before its first launch and one
// behind each launch, with the launch's kernel name and stage.
struct mita_timer {
  int max_calls = 0;
  int used = 0;
  std::vector<hipEvent_t> ev;       // max_calls * (MITA_MAX_LAUNCHES + 1)
  std::vector<const char *> name;   // max_calls * MITA_MAX_LAUNCHES
  std::vector<int32_t> stage;       // max_calls * MITA_MAX_LAUNCHES
  std::vector<int32_t> nlaunch;     // max_calls
};

namespace {

// The timed forward being enqueued on this thread, if any.
struct Recording {
  mita_timer *t;
  int call;
  int stage;
  hipError_t err;
};
thread_local Recording *g_rec = nullptr;

}  // namespace

hipError_t mita::launched(const char *kernel, hipStream_t st) {
  const hipError_t e = hipGetLastError();
  Recording *r = g_rec;
  if (!r || e != hipSuccess) return e;
  mita_timer *t = r->t;
  int &n = t->nlaunch[r->call];
  if (n >= MITA_MAX_LAUNCHES) return e;  // cannot happen: a forward or backward launches fewer kernels
  const size_t slot = (size_t)r->call * MITA_MAX_LAUNCHES + n;
  t->name[slot] = kernel;
  t->stage[slot] = r->stage;
  const hipError_t er = hipEventRecord(t->ev[(size_t)r->call * (MITA_MAX_LAUNCHES + 1) + n + 1], st);
  if (er != hipSuccess && r->err == hipSuccess) r->err = er;
  ++n;
  return e;
}

namespace {

// q_lm_in: caller-supplied landmark queries (mita_forward_lm), or NULL to pool them.
int forward_impl(const mita_cfg_t *c, const void *q, const void *k, const void *v, void *o, void *ws,
                 size_t ws_bytes, hipStream_t st, mita_timer *timer, const void *q_lm_in = nullptr) {
  TRY(validate(c));
  TRY(need_ptr(q, "q"));
  TRY(need_ptr(k, "k"));
  TRY(need_ptr(v, "v"));
  TRY(need_ptr(o, "o"));
  const size_t tb = tensor_bytes(c);
  if (overlaps(o, tb, q, tb) || overlaps(o, tb, k, tb) || overlaps(o, tb, v, tb))
    return set_err(MITA_ERR_INVALID_ARG, "o overlaps an input");
  if (q_lm_in && overlaps(o, tb, q_lm_in, (size_t)BH(*c) * c->M * c->d * elem_bytes(*c)))
    return set_err(MITA_ERR_INVALID_ARG, "o overlaps q_lm");
  TRY(need_ws(c, MITA_WS_FORWARD, ws, ws_bytes));
  Recording rec{timer, 0, 0, hipSuccess};
  if (timer) {
    if (timer->used >= timer->max_calls) return set_err(MITA_ERR_INVALID_ARG, "timer is full");
    rec.call = timer->used++;
    timer->nlaunch[rec.call] = 0;
    TRY(hip_status(hipEventRecord(timer->ev[(size_t)rec.call * (MITA_MAX_LAUNCHES + 1)], st), "hipEventRecord"));
  }
  // launches are attributed to the stage set last (a launch that does the
  // work of two stages counts under the later one)
  struct Scope {
    Recording *prev;
    explicit Scope(Recording *r) : prev(g_rec) { g_rec = r->t ? r : nullptr; }
    ~Scope() { g_rec = prev; }
  } scope(&rec);
  auto mark = [&](int stage) -> int {
    rec.stage = stage;
    return MITA_OK;
  };

  const FwdLayout L = forward_layout(*c);
  char *w = (char *)ws;
  void *q_lm_ws = w + L.q_lm;
  const void *q_lm = q_lm_in ? q_lm_in : q_lm_ws;
  void *v_lm = c->use_shared ? (void *)(w + L.v_lm) : nullptr;
  float *S = c->use_routed ? (float *)(w + L.scores) : nullptr;
  int32_t *idx = (int32_t *)(w + L.idx);
  const bool staged = c->use_routed && (c->flags & MITA_FLAG_STAGED_GATHER);
  void *kx = w + L.kx, *vx = w + L.vx;
  int32_t *expert = (int32_t *)(w + L.expert), *perm = (int32_t *)(w + L.perm);
  int32_t *offsets = (int32_t *)(w + L.offsets), *tile_cnt = (int32_t *)(w + L.tile_cnt);
  int32_t *tile_base = (int32_t *)(w + L.tile_base), *tile_start = (int32_t *)(w + L.tile_start);
  int32_t *counts = (int32_t *)(w + L.counts);
  const bool fused = fused_select(*c);
  SelectBufs sel{};
  if (fused) {
    sel.plo = (uint32_t *)(w + L.plo);
    sel.ccnt = (uint32_t *)(w + L.ccnt);
    sel.cand = (uint2 *)(w + L.cand);
    sel.fail_cnt = (uint32_t *)(w + L.fail);
    sel.fail_list = (int32_t *)(w + L.fail) + 1;
    sel.ns = sel_ns(*c);
    sel.cap = sel_cap(*c);
    sel.rank = sel_rank(*c);
    sel.idx = sel.ns == c->N ? idx : nullptr;  // the sample is the row: the pivot launch writes the sets
  }
  const bool direct = fused && sel.idx;

  // with the fused selection and in-place gather, the selection's finish
  // shares launches with the routing (the "route" stage then includes it),
  // whose placement cursors (in the tile_base buffer) start at zero
  // s > 1 routes through its own launches (stable grouping of the pairs)
  const bool multi = multi_route(*c);
  const bool sel_in_route = fused && c->use_routed && !staged && !multi;
  int32_t *group = multi ? (int32_t *)(w + L.group) : nullptr;
  float *pair_o = multi ? (float *)(w + L.pair_o) : nullptr;
  float *pair_lse = multi ? (float *)(w + L.pair_lse) : nullptr;
  TRY(mark(0));
  int32_t *zero_counts = c->use_routed && !multi ? counts : nullptr;
  int32_t *zero_cursor = sel_in_route ? tile_base : nullptr;
  if (q_lm_in) {
    TRY(hip_status(launch_zero2(zero_counts, zero_counts ? BH(*c) * c->M : 0, zero_cursor,
                                zero_cursor ? BH(*c) * c->M : 0, st),
                   "landmarks"));
  } else {
    TRY(hip_status(launch_pool(*c, q, q_lm_ws, zero_counts, zero_cursor, st), "landmarks"));
  }
  TRY(mark(1));
  // bf16: the routing logits are formed beside the sampled scores (they
  // depend on the landmarks only), in the same launch
  const bool logits_early = sel_in_route && !direct && pivots_with_logits(*c, sel);
  if (logits_early)
    TRY(hip_status(launch_pivots_logits(*c, q, q_lm, k, sel, expert, counts, st), "select pivots"));
  else if (fused)
    TRY(hip_status(launch_select_pivots(*c, q_lm, k, sel, st), "select pivots"));
  // (direct selection: the score pass forms the landmark values only)
  TRY(hip_status(launch_scores(*c, q_lm, k, v, fused ? nullptr : S, v_lm, w + L.partial,
                               fused && !direct ? &sel : nullptr, st),
                 "scores"));
  TRY(mark(2));
  if (fused && !sel_in_route)
    TRY(hip_status(launch_select_finish(*c, q_lm, k, sel, S, idx, w + L.partial, v_lm, st), "topk"));
  else if (!fused && c->use_routed)
    TRY(hip_status(launch_topk(*c, S, idx, st), "topk"));
  TRY(mark(3));
  if (staged) TRY(hip_status(launch_gather(*c, k, v, idx, kx, vx, st), "gather"));
  TRY(mark(4));
  if (sel_in_route)
    TRY(hip_status(launch_select_route(*c, q, q_lm, k, sel, S, idx, w + L.partial, v_lm, expert, perm, offsets,
                                       tile_cnt, tile_base, counts, tile_start, logits_early, st),
                   "route"));
  else if (c->use_routed)
    TRY(hip_status(
        launch_route(*c, q, q_lm, expert, perm, offsets, tile_cnt, tile_base, counts, tile_start, group, st),
        "route"));
  TRY(mark(5));
  TRY(hip_status(launch_attend(*c, q, q_lm, v_lm, staged ? kx : k, staged ? vx : v, staged ? nullptr : idx, perm,
                               offsets, tile_start, o, pair_o, pair_lse, st),
                 "attend"));
  if (rec.err != hipSuccess) return hip_status(rec.err, "hipEventRecord");
  return MITA_OK;
}

// The backward pass: the forward's landmarks, selection and routing
// recomputed into the workspace, then the gradient kernels.
int backward_impl(const mita_cfg_t *c, const void *q, const void *k, const void *v, const void *o, const void *dO,
                  void *dq, void *dk, void *dv, void *ws, size_t ws_bytes, hipStream_t st, mita_timer *timer) {
  TRY(validate(c));
  if (c->use_routed && c->s != 1) return set_err(MITA_ERR_UNSUPPORTED, "the backward pass supports s = 1 only");
  for (auto pr : {std::make_pair(q, "q"), std::make_pair(k, "k"), std::make_pair(v, "v"), std::make_pair(o, "o"),
                  std::make_pair(dO, "dO")})
    TRY(need_ptr(pr.first, pr.second));
  TRY(need_ptr(dq, "dq"));
  TRY(need_ptr(dk, "dk"));
  TRY(need_ptr(dv, "dv"));
  const size_t tb = tensor_bytes(c);
  for (const void *out : {(const void *)dq, (const void *)dk, (const void *)dv}) {
    for (const void *in : {q, k, v, o, dO})
      if (overlaps(out, tb, in, tb)) return set_err(MITA_ERR_INVALID_ARG, "a gradient output overlaps an input");
  }
  if (overlaps(dq, tb, dk, tb) || overlaps(dq, tb, dv, tb) || overlaps(dk, tb, dv, tb))
    return set_err(MITA_ERR_INVALID_ARG, "the gradient outputs overlap");
  TRY(need_ws(c, MITA_WS_BACKWARD, ws, ws_bytes));
  Recording rec{timer, 0, 0, hipSuccess};
  if (timer) {
    if (timer->used >= timer->max_calls) return set_err(MITA_ERR_INVALID_ARG, "timer is full");
    rec.call = timer->used++;
    timer->nlaunch[rec.call] = 0;
    TRY(hip_status(hipEventRecord(timer->ev[(size_t)rec.call * (MITA_MAX_LAUNCHES + 1)], st), "hipEventRecord"));
  }
  struct Scope {
    Recording *prev;
    explicit Scope(Recording *r) : prev(g_rec) { g_rec = r->t ? r : nullptr; }
    ~Scope() { g_rec = prev; }
  } scope(&rec);

  const BwdLayout BL = backward_layout(*c);
  const FwdLayout &L = BL.f;
  char *w = (char *)ws;
  void *q_lm = w + L.q_lm;
  void *v_lm = c->use_shared ? (void *)(w + L.v_lm) : nullptr;
  float *S = c->use_routed ? (float *)(w + L.scores) : nullptr;
  int32_t *idx = (int32_t *)(w + L.idx);
  int32_t *expert = (int32_t *)(w + L.expert), *perm = (int32_t *)(w + L.perm);
  int32_t *offsets = (int32_t *)(w + L.offsets), *tile_cnt = (int32_t *)(w + L.tile_cnt);
  int32_t *tile_base = (int32_t *)(w + L.tile_base), *tile_start = (int32_t *)(w + L.tile_start);
  int32_t *counts = (int32_t *)(w + L.counts);
  const bool fused = fused_select(*c);
  SelectBufs sel{};
  if (fused) {
    sel.plo = (uint32_t *)(w + L.plo);
    sel.ccnt = (uint32_t *)(w + L.ccnt);
    sel.cand = (uint2 *)(w + L.cand);
    sel.fail_cnt = (uint32_t *)(w + L.fail);
    sel.fail_list = (int32_t *)(w + L.fail) + 1;
    sel.ns = sel_ns(*c);
    sel.cap = sel_cap(*c);
    sel.rank = sel_rank(*c);
    sel.idx = sel.ns == c->N ? idx : nullptr;  // the sample is the row: the pivot launch writes the sets
  }
  // recomputation (stages 0 to 4)
  rec.stage = 0;
  TRY(hip_status(launch_pool(*c, q, q_lm, c->use_routed ? counts : nullptr, nullptr, st), "landmarks"));
  rec.stage = 1;
  if (c->use_routed) {
    if (fused) {
      TRY(hip_status(launch_select_pivots(*c, q_lm, k, sel, st), "select pivots"));
      TRY(hip_status(launch_scores(*c, q_lm, k, v, nullptr, v_lm, w + L.partial, sel.idx ? nullptr : &sel, st),
                     "scores"));
      rec.stage = 2;
      TRY(hip_status(launch_select_finish(*c, q_lm, k, sel, S, idx, w + L.partial, v_lm, st), "topk"));
    } else {
      TRY(hip_status(launch_scores(*c, q_lm, k, v, S, v_lm, w + L.partial, nullptr, st), "scores"));
      rec.stage = 2;
      TRY(hip_status(launch_topk(*c, S, idx, st), "topk"));
    }
    rec.stage = 4;
    TRY(hip_status(launch_route(*c, q, q_lm, expert, perm, offsets, tile_cnt, tile_base, counts, tile_start, nullptr,
                                st),
                   "route"));
  } else {
    TRY(hip_status(launch_scores(*c, q_lm, k, v, nullptr, v_lm, w + L.partial, nullptr, st), "scores"));
  }
  // gradients (stage 5)
  rec.stage = 5;
  const int64_t nd = BH(*c) * c->N * c->d, md = BH(*c) * c->M * c->d;
  if (!c->use_routed) {  // with routing, the routed keys' gather writes dk_acc and dv_acc first
    TRY(hip_status(launch_zero2((int32_t *)(w + BL.dk_acc), nd, (int32_t *)(w + BL.dv_acc), nd, st), "backward"));
  }
  TRY(hip_status(launch_zero2((int32_t *)(w + BL.dq_lm_acc), md, (int32_t *)(w + BL.dv_lm_acc), md, st),
                 "backward"));
  BwdBufs b{};
  b.q = q;
  b.k = k;
  b.v = v;
  b.o = o;
  b.dO = dO;
  b.q_lm = q_lm;
  b.v_lm = v_lm;
  b.idx = idx;
  b.perm = perm;
  b.offsets = offsets;
  b.tile_start = tile_start;
  b.part_ml = w + L.partial;
  b.lse_lm = (float *)(w + BL.lse_lm);
  b.dq_direct = (float *)(w + BL.dq_direct);
  b.dk_acc = (float *)(w + BL.dk_acc);
  b.dv_acc = (float *)(w + BL.dv_acc);
  b.dq_lm_acc = (float *)(w + BL.dq_lm_acc);
  b.dv_lm_acc = (float *)(w + BL.dv_lm_acc);
  b.q_lse = (float *)(w + BL.q_lse);
  b.q_D = (float *)(w + BL.q_D);
  b.stage_k = (float *)(w + BL.stage_k);
  b.stage_v = (float *)(w + BL.stage_v);
  b.inv_start = (int32_t *)(w + BL.inv_start);
  b.inv_slot = (int32_t *)(w + BL.inv_slot);
  b.dv_lm16 = w + BL.dv_lm16;
  b.D_lm = (float *)(w + BL.D_lm);
  b.dq = dq;
  b.dk = dk;
  b.dv = dv;
  TRY(hip_status(launch_backward(*c, b, st), "backward"));
  if (rec.err != hipSuccess) return hip_status(rec.err, "hipEventRecord");
  return MITA_OK;
}

}  // namespace

// Workspace of mita_forward_noalloc, for callers that cannot allocate: one
// static device array per GPU the library runs on (held until the process
// ends). In host code `scratch` is only a stand-in for the symbol; its device
// address on the current GPU comes from hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[MITA_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[MAX_DEVICES] = {};

// The device address of `scratch` on the current device, looked up once per
// device (with that device current).
int scratch_address(void **out) {
  int dev = -1;
  TRY(hip_status(hipGetDevice(&dev), "hipGetDevice"));
  if (dev < 0 || dev >= MAX_DEVICES) return set_err(MITA_ERR_HIP, "device index out of range for the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    TRY(hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)"));
    if (!p) return set_err(MITA_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MITA_OK;
}

}  // namespace

extern "C" {

int mita_forward_noalloc(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, void *o,
                         mita_stream_t stream) {
  g_err.clear();
  TRY(validate(cfg));
  const size_t need = workspace_size(cfg, MITA_WS_FORWARD);
  if (need > MITA_NOALLOC_SCRATCH_BYTES)
    return set_err(MITA_ERR_WORKSPACE, "the forward needs " + std::to_string(need) +
                                           " bytes of workspace; the static scratch of mita_forward_noalloc holds " +
                                           std::to_string((size_t)MITA_NOALLOC_SCRATCH_BYTES));
  void *ws = nullptr;
  TRY(scratch_address(&ws));
  return forward_impl(cfg, q, k, v, o, ws, MITA_NOALLOC_SCRATCH_BYTES, (hipStream_t)stream, nullptr);
}

int mita_check(const mita_cfg_t *cfg) { return validate(cfg); }

size_t mita_workspace_size(const mita_cfg_t *cfg, int which) { return workspace_size(cfg, which); }

const char *mita_status_string(int status) {
  switch (status) {
    case MITA_OK: return "ok";
    case MITA_ERR_INVALID_ARG: return "invalid argument";
    case MITA_ERR_UNSUPPORTED: return "unsupported configuration";
    case MITA_ERR_WORKSPACE: return "workspace too small";
    case MITA_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char *mita_last_error(void) { return g_err.c_str(); }

int mita_forward(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, void *o, void *ws,
                 size_t ws_bytes, mita_stream_t stream) {
  g_err.clear();
  return forward_impl(cfg, q, k, v, o, ws, ws_bytes, (hipStream_t)stream, nullptr);
}

int mita_forward_timed(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, void *o, void *ws,
                       size_t ws_bytes, mita_stream_t stream, mita_timer_t *timer) {
  g_err.clear();
  if (!timer) return set_err(MITA_ERR_INVALID_ARG, "timer is NULL");
  return forward_impl(cfg, q, k, v, o, ws, ws_bytes, (hipStream_t)stream, timer);
}

int mita_backward(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, const void *o, const void *dO,
                  void *dq, void *dk, void *dv, void *ws, size_t ws_bytes, mita_stream_t stream) {
  g_err.clear();
  return backward_impl(cfg, q, k, v, o, dO, dq, dk, dv, ws, ws_bytes, (hipStream_t)stream, nullptr);
}

int mita_backward_timed(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, const void *o,
                        const void *dO, void *dq, void *dk, void *dv, void *ws, size_t ws_bytes,
                        mita_stream_t stream, mita_timer_t *timer) {
  g_err.clear();
  if (!timer) return set_err(MITA_ERR_INVALID_ARG, "timer is NULL");
  return backward_impl(cfg, q, k, v, o, dO, dq, dk, dv, ws, ws_bytes, (hipStream_t)stream, timer);
}

int mita_forward_lm_timed(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, const void *q_lm,
                          void *o, void *ws, size_t ws_bytes, mita_stream_t stream, mita_timer_t *timer) {
  g_err.clear();
  TRY(validate(cfg));
  TRY(need_ptr(q_lm, "q_lm"));
  if (!timer) return set_err(MITA_ERR_INVALID_ARG, "timer is NULL");
  return forward_impl(cfg, q, k, v, o, ws, ws_bytes, (hipStream_t)stream, timer, q_lm);
}

int mita_forward_fallbacks(const mita_cfg_t *cfg, const void *ws, size_t ws_bytes, int64_t *count,
                           mita_stream_t stream) {
  g_err.clear();
  TRY(validate(cfg));
  if (!count) return set_err(MITA_ERR_INVALID_ARG, "count is NULL");
  TRY(need_ws(cfg, MITA_WS_FORWARD, ws, ws_bytes));
  hipStream_t st = (hipStream_t)stream;
  *count = 0;
  TRY(hip_status(hipStreamSynchronize(st), "hipStreamSynchronize"));
  if (!fused_select(*cfg)) return MITA_OK;
  uint32_t n = 0;
  TRY(hip_status(hipMemcpy(&n, (const char *)ws + forward_layout(*cfg).fail, sizeof n, hipMemcpyDeviceToHost),
                 "hipMemcpy"));
  *count = n;
  return MITA_OK;
}

int mita_select_plan(const mita_cfg_t *cfg, int32_t *fused, int32_t *ns, int32_t *rank, int32_t *cap) {
  g_err.clear();
  TRY(validate(cfg));
  const bool f = fused_select(*cfg);
  const SelPlan p = sel_plan(*cfg);
  if (fused) *fused = f ? 1 : 0;
  if (ns) *ns = f ? p.ns : 0;
  if (rank) *rank = f ? p.rank : 0;
  if (cap) *cap = f ? p.cap : 0;
  return MITA_OK;
}

int mita_landmarks(const mita_cfg_t *cfg, const void *q, void *q_lm, mita_stream_t stream) {
  g_err.clear();
  TRY(validate(cfg));
  TRY(need_ptr(q, "q"));
  TRY(need_ptr(q_lm, "q_lm"));
  return hip_status(launch_pool(*cfg, q, q_lm, nullptr, nullptr, (hipStream_t)stream), "landmarks");
}

int mita_landmarks_select(const mita_cfg_t *cfg, const void *q, const int32_t *sel, void *q_lm,
                          mita_stream_t stream) {
  g_err.clear();
  TRY(validate(cfg));
  TRY(need_ptr(q, "q"));
  TRY(need_ptr(sel, "sel"));
  TRY(need_ptr(q_lm, "q_lm"));
  return hip_status(launch_select_landmarks(*cfg, q, sel, q_lm, (hipStream_t)stream), "landmarks");
}

int mita_landmarks_tome(const mita_cfg_t *cfg, const void *q, void *q_lm, int32_t *assign, void *ws, size_t ws_bytes,
                        mita_stream_t stream) {
  g_err.clear();
  TRY(validate(cfg));
  TRY(need_ptr(q, "q"));
  TRY(need_ptr(q_lm, "q_lm"));
  if (assign) TRY(need_ptr(assign, "assign"));
  TRY(need_ws(cfg, MITA_WS_TOME, ws, ws_bytes));
  const TomeLayout L = tome_layout(*cfg);
  char *w = (char *)ws;
  TomeBufs b{};
  b.S[0] = (int64_t *)(w + L.S0);
  b.S[1] = (int64_t *)(w + L.S1);
  b.cnt[0] = (int32_t *)(w + L.cnt0);
  b.cnt[1] = (int32_t *)(w + L.cnt1);
  b.rep[0] = (int32_t *)(w + L.rep0);
  b.rep[1] = (int32_t *)(w + L.rep1);
  b.X = (float *)(w + L.X);
  b.score = (float *)(w + L.score);
  b.match = (int32_t *)(w + L.match);
  b.sel = (int32_t *)(w + L.sel);
  b.merged = (int32_t *)(w + L.merged);
  b.alive = (int32_t *)(w + L.alive);
  b.pos = (int32_t *)(w + L.pos);
  return hip_status(launch_tome(*cfg, q, q_lm, assign, b, (hipStream_t)stream), "landmarks (token merging)");
}

int mita_forward_lm(const mita_cfg_t *cfg, const void *q, const void *k, const void *v, const void *q_lm, void *o,
                    void *ws, size_t ws_bytes, mita_stream_t stream) {
  g_err.clear();
  TRY(validate(cfg));
  TRY(need_ptr(q_lm, "q_lm"));
  return forward_impl(cfg, q, k, v, o, ws, ws_bytes, (hipStream_t)stream, nullptr, q_lm);
}

int mita_scores(const mita_cfg_t *cfg, const void *q_lm, const void *k, const void *v, float *scores, void *v_lm,
                void *ws, size_t ws_bytes, mita_stream_t stream) {
  g_err.clear();
  TRY(validate(cfg));
  TRY(need_ptr(q_lm, "q_lm"));
  TRY(need_ptr(k, "k"));
  if (scores) TRY(need_ptr(scores, "scores"));
  if (v_lm) {
    TRY(need_ptr(v_lm, "v_lm"));
    TRY(need_ptr(v, "v"));
    TRY(need_ws(cfg, MITA_WS_SCORES, ws, ws_bytes));
  }
  return hip_status(launch_scores(*cfg, q_lm, k, v, scores, v_lm, ws, nullptr, (hipStream_t)stream), "scores");
}

int mita_topk(const mita_cfg_t *cfg, const float *scores, int32_t *idx, void *ws, size_t ws_bytes,
              mita_stream_t stream) {
  g_err.clear();
  (void)ws;
  (void)ws_bytes;
  TRY(validate(cfg));
  TRY(need_ptr(scores, "scores"));
  TRY(need_ptr(idx, "idx"));
  return hip_status(launch_topk(*cfg, scores, idx, (hipStream_t)stream), "topk");
}

int mita_gather(const mita_cfg_t *cfg, const void *k, const void *v, const int32_t *idx, void *k_x, void *v_x,
                mita_stream_t stream) {
  g_err.clear();
  TRY(validate(cfg));
  TRY(need_ptr(k, "k"));
  TRY(need_ptr(v, "v"));
  TRY(need_ptr(idx, "idx"));
  TRY(need_ptr(k_x, "k_x"));
  TRY(need_ptr(v_x, "v_x"));
  return hip_status(launch_gather(*cfg, k, v, idx, k_x, v_x, (hipStream_t)stream), "gather");
}

int mita_route(const mita_cfg_t *cfg, const void *q, const void *q_lm, int32_t *expert, int32_t *perm,
               int32_t *offsets, void *ws, size_t ws_bytes, mita_stream_t stream) {
  g_err.clear();
  TRY(validate(cfg));
  TRY(need_ptr(q, "q"));
  TRY(need_ptr(q_lm, "q_lm"));
  TRY(need_ptr(expert, "expert"));
  TRY(need_ptr(perm, "perm"));
  TRY(need_ptr(offsets, "offsets"));
  TRY(need_ws(cfg, MITA_WS_ROUTE, ws, ws_bytes));
  const size_t tb = route_tiles_bytes(*cfg);
  char *w = (char *)ws;
  int32_t *tile_cnt = (int32_t *)w;
  int32_t *tile_base = (int32_t *)(w + tb);
  int32_t *counts = (int32_t *)(w + 2 * tb);
  int32_t *tile_start = (int32_t *)(w + 2 * tb + route_counts_bytes(*cfg));
  int32_t *group = multi_route(*cfg)
                       ? (int32_t *)(w + 2 * tb + route_counts_bytes(*cfg) + route_start_bytes(*cfg))
                       : nullptr;
  hipStream_t st = (hipStream_t)stream;
  if (!multi_route(*cfg)) TRY(hip_status(launch_zero(counts, BH(*cfg) * cfg->M, st), "route"));
  return hip_status(
      launch_route(*cfg, q, q_lm, expert, perm, offsets, tile_cnt, tile_base, counts, tile_start, group, st),
      "route");
}

int mita_attend(const mita_cfg_t *cfg, const void *q, const void *q_lm, const void *v_lm, const void *k_x,
                const void *v_x, const int32_t *perm, const int32_t *offsets, void *o, void *ws, size_t ws_bytes,
                mita_stream_t stream) {
  g_err.clear();
  TRY(validate(cfg));
  TRY(need_ptr(q, "q"));
  TRY(need_ptr(o, "o"));
  if (cfg->use_shared) {
    TRY(need_ptr(q_lm, "q_lm"));
    TRY(need_ptr(v_lm, "v_lm"));
  }
  if (cfg->use_routed) {
    TRY(need_ptr(k_x, "k_x"));
    TRY(need_ptr(v_x, "v_x"));
    TRY(need_ptr(perm, "perm"));
    TRY(need_ptr(offsets, "offsets"));
  }
  const size_t tb = tensor_bytes(cfg);
  if (overlaps(o, tb, q, tb)) return set_err(MITA_ERR_INVALID_ARG, "o overlaps q");
  TRY(need_ws(cfg, MITA_WS_ATTEND, ws, ws_bytes));
  hipStream_t st = (hipStream_t)stream;
  char *w = (char *)ws;
  int32_t *tile_start = (int32_t *)w;
  float *pair_o = multi_route(*cfg) ? (float *)(w + route_start_bytes(*cfg)) : nullptr;
  float *pair_lse = multi_route(*cfg) ? (float *)(w + route_start_bytes(*cfg) + pair_out_bytes(*cfg)) : nullptr;
  if (cfg->use_routed) TRY(hip_status(launch_worklist(*cfg, offsets, tile_start, st), "worklist"));
  return hip_status(
      launch_attend(*cfg, q, q_lm, v_lm, k_x, v_x, nullptr, perm, offsets, tile_start, o, pair_o, pair_lse, st),
      "attend");
}

int mita_timer_create(mita_timer_t **timer, int max_calls) {
  g_err.clear();
  if (!timer || max_calls < 1) return set_err(MITA_ERR_INVALID_ARG, "bad timer arguments");
  mita_timer *t = new mita_timer();
  t->max_calls = max_calls;
  t->ev.resize((size_t)max_calls * (MITA_MAX_LAUNCHES + 1));
  t->name.assign((size_t)max_calls * MITA_MAX_LAUNCHES, nullptr);
  t->stage.assign((size_t)max_calls * MITA_MAX_LAUNCHES, 0);
  t->nlaunch.assign((size_t)max_calls, 0);
  for (size_t i = 0; i < t->ev.size(); ++i) {
    hipError_t e = hipEventCreate(&t->ev[i]);
    if (e != hipSuccess) {
      for (size_t j = 0; j < i; ++j) (void)hipEventDestroy(t->ev[j]);
      delete t;
      return hip_status(e, "hipEventCreate");
    }
  }
  *timer = t;
  return MITA_OK;
}

int mita_timer_destroy(mita_timer_t *timer) {
  if (!timer) return MITA_OK;
  for (hipEvent_t e : timer->ev) (void)hipEventDestroy(e);
  delete timer;
  return MITA_OK;
}

int mita_timer_reset(mita_timer_t *timer) {
  if (!timer) return set_err(MITA_ERR_INVALID_ARG, "timer is NULL");
  timer->used = 0;
  return MITA_OK;
}

namespace {
// Waits for the last event of the last recorded call.
int timer_wait(mita_timer *t) {
  if (t->used == 0) return MITA_OK;
  const int c = t->used - 1;
  return hip_status(hipEventSynchronize(t->ev[(size_t)c * (MITA_MAX_LAUNCHES + 1) + t->nlaunch[c]]),
                    "hipEventSynchronize");
}
}  // namespace

int mita_timer_read(mita_timer_t *timer, float *ms, int ms_len, int *n_calls) {
  g_err.clear();
  if (!timer || !ms || !n_calls) return set_err(MITA_ERR_INVALID_ARG, "NULL argument");
  if (ms_len < timer->used * MITA_NUM_STAGES) return set_err(MITA_ERR_INVALID_ARG, "ms buffer too small");
  *n_calls = timer->used;
  TRY(timer_wait(timer));
  for (int c = 0; c < timer->used; ++c) {
    for (int s = 0; s < MITA_NUM_STAGES; ++s) ms[c * MITA_NUM_STAGES + s] = 0.f;
    const hipEvent_t *ev = &timer->ev[(size_t)c * (MITA_MAX_LAUNCHES + 1)];
    for (int i = 0; i < timer->nlaunch[c]; ++i) {
      float t = 0.f;
      TRY(hip_status(hipEventElapsedTime(&t, ev[i], ev[i + 1]), "hipEventElapsedTime"));
      ms[c * MITA_NUM_STAGES + timer->stage[(size_t)c * MITA_MAX_LAUNCHES + i]] += t;
    }
  }
  return MITA_OK;
}

int mita_timer_launches(mita_timer_t *timer, int call, int cap, const char **kernels, int32_t *stages, float *ms,
                        int32_t *n_launches) {
  g_err.clear();
  if (!timer || !kernels || !stages || !ms || !n_launches) return set_err(MITA_ERR_INVALID_ARG, "NULL argument");
  if (call < 0 || call >= timer->used) return set_err(MITA_ERR_INVALID_ARG, "no such recorded call");
  const int n = timer->nlaunch[call];
  if (cap < n) return set_err(MITA_ERR_INVALID_ARG, "output arrays too small");
  TRY(timer_wait(timer));
  const hipEvent_t *ev = &timer->ev[(size_t)call * (MITA_MAX_LAUNCHES + 1)];
  for (int i = 0; i < n; ++i) {
    const size_t slot = (size_t)call * MITA_MAX_LAUNCHES + i;
    kernels[i] = timer->name[slot];
    stages[i] = timer->stage[slot];
    TRY(hip_status(hipEventElapsedTime(&ms[i], ev[i], ev[i + 1]), "hipEventElapsedTime"));
  }
  *n_launches = n;
  return MITA_OK;
}

}  // extern "C"
