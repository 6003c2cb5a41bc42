// Host side of the C ABI declared in include/omnimoe.h: argument checks, workspace carving and
// kernel launches on the caller's stream. No device memory is allocated here and there is no
// host synchronisation inside a call.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/omnimoe.h"
#include "internal.hpp"

using omnimoe::Shape;

// Workspace of omnimoe_layer_forward_noalloc: one copy on every GPU the library runs on, held
// until the process ends. Host code never uses this name as an address: the device address is
// looked up per device (noalloc_scratch below) and only that is passed to kernels.
static __device__ __align__(256) unsigned char scratch[OMNIMOE_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int64_t kIntMax = 2147483647LL;

size_t align_up(size_t v) { return (v + 255) & ~(size_t)255; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

omnimoe_status check_desc(const omnimoe_layer_desc* d, Shape* s) {
  if (!d) return OMNIMOE_ERR_INVALID_ARG;
  if (d->T < 0 || d->T > (1LL << 23)) return OMNIMOE_ERR_INVALID_ARG;
  if (d->d < 8 || d->d > 8192 || d->d % 8) return OMNIMOE_ERR_INVALID_ARG;
  if (d->n_rows < 1 || d->n_rows > 4096 || d->n_cols < 1 || d->n_cols > 4096)
    return OMNIMOE_ERR_INVALID_ARG;
  if (d->d_key < 8 || d->d_key % 8) return OMNIMOE_ERR_INVALID_ARG;
  if (d->query_mode == OMNIMOE_QUERY_SPLIT) {
    if (2LL * d->d_key > d->d) return OMNIMOE_ERR_INVALID_ARG;
  } else if (d->query_mode == OMNIMOE_QUERY_SHARED) {
    if (d->d_key > d->d) return OMNIMOE_ERR_INVALID_ARG;
  } else {
    return OMNIMOE_ERR_INVALID_ARG;
  }
  if (d->H < 1 || d->K < 1) return OMNIMOE_ERR_INVALID_ARG;
  const int64_t N = (int64_t)d->n_rows * d->n_cols;
  if (d->K > N) return OMNIMOE_ERR_INVALID_ARG;
  if (d->K > 4096) return OMNIMOE_ERR_UNSUPPORTED;
  if (d->dtype != OMNIMOE_F32 && d->dtype != OMNIMOE_BF16) return OMNIMOE_ERR_INVALID_ARG;
  if (d->dtype == OMNIMOE_F32 && d->d > 4096) return OMNIMOE_ERR_UNSUPPORTED;
  if (d->act != OMNIMOE_ACT_GELU && d->act != OMNIMOE_ACT_SILU) return OMNIMOE_ERR_INVALID_ARG;
  if (d->group_size < 1) return OMNIMOE_ERR_INVALID_ARG;
  const int64_t rows = d->T * d->H;
  if (rows * d->K >= kIntMax || rows * (d->n_rows + d->n_cols) >= kIntMax)
    return OMNIMOE_ERR_INVALID_ARG;
  s->T = d->T;
  s->d = d->d;
  s->nr = d->n_rows;
  s->nc = d->n_cols;
  s->dk = d->d_key;
  s->H = d->H;
  s->K = d->K;
  s->bf16 = d->dtype == OMNIMOE_BF16;
  s->act = d->act;
  s->col0 = d->query_mode == OMNIMOE_QUERY_SPLIT ? d->d_key : 0;
  s->N = N;
  s->rows = rows;
  s->M = rows * d->K;
  s->hk = d->H * d->K;
  s->B = d->group_size;
  return OMNIMOE_OK;
}

omnimoe_status check_ptrs(std::initializer_list<const void*> ps) {
  for (const void* p : ps) {
    if (!p) return OMNIMOE_ERR_INVALID_ARG;
    if (!aligned16(p)) return OMNIMOE_ERR_ALIGNMENT;
  }
  return OMNIMOE_OK;
}

omnimoe_status check_opt(const void* p) {
  return (p && !aligned16(p)) ? OMNIMOE_ERR_ALIGNMENT : OMNIMOE_OK;
}

omnimoe_status hip_status(hipError_t e) { return e == hipSuccess ? OMNIMOE_OK : OMNIMOE_ERR_HIP; }

size_t hs_bytes(const Shape& s) { return align_up((size_t)s.rows * (s.nr + s.nc) * 4); }
size_t m_bytes(const Shape& s) { return align_up((size_t)s.M * 4); }
size_t dense_bytes(const Shape& s) { return align_up((size_t)s.rows * (size_t)s.N * 4); }
size_t active_bytes(const Shape& s) { return align_up((size_t)(std::min(s.M, s.N) + 1) * 4); }

// The grouped expert GEMM (Eq. 14) runs for bf16 with d a multiple of 64; the layer takes it
// when the schedule's groups hold more than one expert.
bool grouped_supported(const Shape& s) { return s.bf16 && s.d % 64 == 0; }
bool layer_grouped(const Shape& s) { return s.B > 1 && grouped_supported(s); }

// Which kernels the layer runs for a shape (omnimoe_layer_path reports the same flags).
// Where the expert-major order saves no memory traffic (a decode step; at most one task per two
// experts; or a u table that fits in the MALL) the layer takes the slot-order dot and forms no
// schedule. With at least kSelectDotMinRows (token, head) rows the selection kernel forms that
// dot itself; with fewer, a wave per row would fetch its K u rows four at a time, while the
// separate dot kernel fetches all of them at once (one decoded token: 19.1 against 22.1 us).
constexpr int64_t kSelectDotMinRows = 256;
// Up to this many tasks the sort by expert is one launch, as cheap as the flag pass and scan
// that replace it above (launch_group_schedule).
constexpr int64_t kSortFreeMinTasks = 8192;
int32_t layer_path(const Shape& s) {
  const bool grouped = layer_grouped(s);
  const bool unscheduled = !grouped && omnimoe::slot_dot(s);
  int32_t f = 0;
  if (!unscheduled) f |= OMNIMOE_PATH_SCHEDULE;
  if (grouped) f |= OMNIMOE_PATH_GROUPED;
  if (unscheduled && s.rows >= kSelectDotMinRows && omnimoe::select_dot_fusable(s))
    f |= OMNIMOE_PATH_SELECT_DOT;
  if (omnimoe::dense_accumulate(s)) f |= OMNIMOE_PATH_DENSE_SUM;
  // Both products dense over all experts: no schedule and no per-task dot.
  if (omnimoe::dense_dot(s)) f = OMNIMOE_PATH_DENSE_SUM | OMNIMOE_PATH_DENSE_DOT;
  return f;
}

// Schedule workspace, followed by the grouped plan's (which reads the schedule's sorted keys).
// The routed sum y_t = sum of a_p v_e over t's tasks: one dense GEMM over all experts when
// the pairs are dense enough (Eq. 14 with a single group), else the token-major slot-order
// kernel. dense_ws holds dense_accumulate_ws_bytes(s) bytes.
hipError_t routed_sum(const Shape& s, const void* v, const int32_t* idx, const float* abuf,
                      float* y, void* dense_ws, hipStream_t st) {
  if (omnimoe::dense_accumulate(s))
    return omnimoe::launch_dense_accumulate(s, v, idx, abuf, y, dense_ws, st);
  return omnimoe::launch_accumulate(s, v, idx, abuf, y, st);
}

// Slots (group, token) of a schedule with groups of B: at most one per task, and at most one
// per token in each of the ceil(min(M, N) / B) groups.
int64_t group_rows_bound(const Shape& s) {
  const int64_t groups = (std::min(s.M, s.N) + s.B - 1) / s.B;
  return std::min(s.M, groups * s.T);
}

size_t sched_or_plan_bytes(const Shape& s) {
  const size_t sb = omnimoe::schedule_ws_bytes(s.M, s.N);
  return layer_grouped(s) ? sb + omnimoe::group_plan_ws_bytes(s) : sb;
}

size_t stage_bytes(const Shape& s, int stage) {
  switch (stage) {
    case OMNIMOE_STAGE_ROUTE: return hs_bytes(s);
    case OMNIMOE_STAGE_SELECT: return 0;
    case OMNIMOE_STAGE_SCHEDULE: return omnimoe::schedule_ws_bytes(s.M, s.N);
    case OMNIMOE_STAGE_EXPERT: return m_bytes(s) + omnimoe::dense_accumulate_ws_bytes(s);
    case OMNIMOE_STAGE_ROUTE_DENSE: return dense_bytes(s);
    case OMNIMOE_STAGE_EXPERT_BACKWARD: return omnimoe::backward_ws_bytes(s.M);
    case OMNIMOE_STAGE_ROUTE_BACKWARD: return omnimoe::route_backward_ws_bytes(s);
    case OMNIMOE_STAGE_EXPERT_SCATTER: return m_bytes(s) + align_up((size_t)s.M * s.d * 4);
    case OMNIMOE_STAGE_EXPERT_GROUP_ROWS: {
      const int64_t n = group_rows_bound(s);
      return m_bytes(s) + omnimoe::group_plan_ws_bytes(s) + align_up((size_t)n * s.d * 4) +
             omnimoe::slot_sort_ws_bytes(n, s.T);
    }
    case OMNIMOE_STAGE_EXPERT_GROUPED:  // the plan is dead once the grouped dot has run
      return m_bytes(s) + std::max(omnimoe::group_plan_ws_bytes(s),
                                   omnimoe::dense_accumulate_ws_bytes(s));
    default: {
      // idx, gates, perm, active, active_offsets, n_active, then the logits (dead after
      // selection) overlapped with the sort buffers, the a[] buffer and the dense routed sum's
      // buffers.
      size_t fixed = 3 * m_bytes(s) + 2 * active_bytes(s) + 256;
      size_t late = sched_or_plan_bytes(s) + m_bytes(s) + omnimoe::dense_accumulate_ws_bytes(s);
      // A selection kernel that forms a[] writes it while other rows' logits are still being
      // read: a[] and the dense sum's buffers then follow the logits instead of sharing them.
      if (layer_path(s) & OMNIMOE_PATH_SELECT_DOT)
        late = hs_bytes(s) + m_bytes(s) + omnimoe::dense_accumulate_ws_bytes(s);
      // Both products dense: only their buffers, after the logits are dead.
      if (layer_path(s) & OMNIMOE_PATH_DENSE_DOT) late = omnimoe::dense_dot_ws_bytes(s);
      return fixed + std::max(hs_bytes(s), late);
    }
  }
}

}  // namespace

struct omnimoe_timer {
  int capacity = 0;
  int used = 0;
  std::vector<hipEvent_t> ev;  // capacity * (OMNIMOE_KERNEL_COUNT + 1)
};

namespace {

constexpr int kEv = OMNIMOE_KERNEL_COUNT + 1;

omnimoe_status layer_impl(const omnimoe_layer_desc* desc, const void* x, const void* keys_row,
                          const void* keys_col, const void* u, const void* v, float* y,
                          int32_t* idx_out, float* gates_out, void* ws, size_t ws_bytes,
                          void* stream, omnimoe_timer* timer) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({x, keys_row, keys_col, u, v, y, ws}))) return st;
  if ((st = check_opt(idx_out)) || (st = check_opt(gates_out))) return st;
  if (ws_bytes < stage_bytes(s, OMNIMOE_STAGE_LAYER)) return OMNIMOE_ERR_WORKSPACE;
  if (timer && timer->used >= timer->capacity) return OMNIMOE_ERR_INVALID_ARG;
  hipStream_t strm = (hipStream_t)stream;
  char* w = (char*)ws;
  int32_t* idx = (int32_t*)w; w += m_bytes(s);
  float* gates = (float*)w; w += m_bytes(s);
  int32_t* perm = (int32_t*)w; w += m_bytes(s);
  int32_t* active = (int32_t*)w; w += active_bytes(s);
  int32_t* offsets = (int32_t*)w; w += active_bytes(s);
  int32_t* n_active = (int32_t*)w; w += 256;
  char* late = w;
  float* hs = (float*)late;
  void* sched_ws = late;
  const int32_t path = layer_path(s);
  // (after the logits when the selection kernel writes a[]: see stage_bytes)
  float* abuf = (float*)(late + ((path & OMNIMOE_PATH_SELECT_DOT) ? hs_bytes(s)
                                                                  : sched_or_plan_bytes(s)));
  if (idx_out) idx = idx_out;
  if (gates_out) gates = gates_out;

  hipEvent_t* ev = timer ? &timer->ev[(size_t)timer->used * kEv] : nullptr;
  auto mark = [&](int k) {
    if (ev) (void)hipEventRecord(ev[k], strm);
  };
  hipError_t e;
  mark(0);
  if ((e = omnimoe::launch_score(s, x, keys_row, keys_col, hs, strm))) return hip_status(e);
  mark(1);
  const bool unscheduled = !(path & OMNIMOE_PATH_SCHEDULE);
  const bool fused = (path & OMNIMOE_PATH_SELECT_DOT) != 0;
  if (fused) {
    if ((e = omnimoe::launch_select_dot(s, hs, idx, gates, x, u, abuf, strm)))
      return hip_status(e);
  } else if ((e = omnimoe::launch_select(s, hs, idx, gates, strm))) {
    return hip_status(e);
  }
  mark(2);
  if (path & OMNIMOE_PATH_DENSE_DOT) {
    if ((e = omnimoe::launch_select_mask(s, idx, gates, late, strm))) return hip_status(e);
    mark(3);
    if ((e = omnimoe::launch_dense_dot(s, x, u, late, strm))) return hip_status(e);
    mark(4);
    if ((e = omnimoe::launch_dense_routed_sum(s, v, y, late, strm))) return hip_status(e);
    mark(5);
    if (timer) ++timer->used;
    return OMNIMOE_OK;
  }
  const int32_t* sk = nullptr;
  const int32_t* gk = nullptr;
  if (!unscheduled) {
    // The grouped product needs the active list and the (group, task id) order but no
    // per-expert offsets, so past the single-launch sizes it skips the sort by expert.
    if ((path & OMNIMOE_PATH_GROUPED) && s.M > kSortFreeMinTasks &&
        omnimoe::group_schedule_fits(s))
      e = omnimoe::launch_group_schedule(s, idx, perm, active, n_active, sched_ws, &gk, strm);
    else
      e = omnimoe::launch_schedule(s, idx, perm, active, offsets, n_active, nullptr, sched_ws,
                                   &sk, strm, &gk);
    if (e) return hip_status(e);
  }
  mark(3);
  if (unscheduled) {
    if (!fused && (e = omnimoe::launch_slot_dot(s, x, u, idx, gates, abuf, strm)))
      return hip_status(e);
  } else if (path & OMNIMOE_PATH_GROUPED) {
    omnimoe::GroupPlan plan;
    void* plan_ws = (char*)sched_ws + omnimoe::schedule_ws_bytes(s.M, s.N);
    if ((e = omnimoe::launch_group_plan(s, perm, n_active, gk, idx, active, plan_ws, &plan,
                                        strm)))
      return hip_status(e);
    if ((e = omnimoe::launch_grouped_dot(s, x, u, gates, perm, active, n_active, plan, abuf,
                                         strm)))
      return hip_status(e);
  } else if ((e = omnimoe::launch_expert_dot(s, x, u, idx, gates, perm, sk, abuf, strm))) {
    return hip_status(e);
  }
  mark(4);
  if ((e = routed_sum(s, v, idx, abuf, y, (char*)abuf + m_bytes(s), strm))) return hip_status(e);
  mark(5);
  if (timer) ++timer->used;
  return OMNIMOE_OK;
}

// Device address of `scratch` on the calling thread's current device, looked up with that
// device current on its first use and kept per device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

omnimoe_status noalloc_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return OMNIMOE_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return OMNIMOE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return OMNIMOE_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return OMNIMOE_OK;
}

}  // namespace

extern "C" {

const char* omnimoe_status_string(int32_t status) {
  switch (status) {
    case OMNIMOE_OK: return "ok";
    case OMNIMOE_ERR_INVALID_ARG: return "invalid argument";
    case OMNIMOE_ERR_UNSUPPORTED: return "unsupported by the library";
    case OMNIMOE_ERR_ALIGNMENT: return "pointer not 16-byte aligned";
    case OMNIMOE_ERR_WORKSPACE: return "workspace too small";
    case OMNIMOE_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

omnimoe_status omnimoe_workspace_size(const omnimoe_layer_desc* desc, int32_t stage,
                                      size_t* bytes) {
  if (!bytes) return OMNIMOE_ERR_INVALID_ARG;
  if (stage < OMNIMOE_STAGE_ROUTE || stage > OMNIMOE_STAGE_EXPERT_GROUP_ROWS)
    return OMNIMOE_ERR_INVALID_ARG;
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  *bytes = stage_bytes(s, stage);
  return OMNIMOE_OK;
}

omnimoe_status omnimoe_route(const omnimoe_layer_desc* desc, const void* x, const void* keys_row,
                             const void* keys_col, int32_t* idx, float* gates, float* half_scores,
                             void* ws, size_t ws_bytes, void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({x, keys_row, keys_col, idx, gates}))) return st;
  if ((st = check_opt(half_scores))) return st;
  float* hs = half_scores;
  if (!hs) {
    if ((st = check_ptrs({ws}))) return st;
    if (ws_bytes < stage_bytes(s, OMNIMOE_STAGE_ROUTE)) return OMNIMOE_ERR_WORKSPACE;
    hs = (float*)ws;
  }
  hipStream_t strm = (hipStream_t)stream;
  hipError_t e = omnimoe::launch_score(s, x, keys_row, keys_col, hs, strm);
  if (e == hipSuccess) e = omnimoe::launch_select(s, hs, idx, gates, strm);
  return hip_status(e);
}

omnimoe_status omnimoe_route_dense(const omnimoe_layer_desc* desc, const void* x,
                                   const void* w_gate, int32_t* idx, float* gates, float* logits,
                                   void* ws, size_t ws_bytes, void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({x, w_gate, idx, gates}))) return st;
  if ((st = check_opt(logits))) return st;
  if ((int64_t)s.H * s.N >= kIntMax || s.K > 64) return OMNIMOE_ERR_UNSUPPORTED;
  float* L = logits;
  if (!L) {
    if ((st = check_ptrs({ws}))) return st;
    if (ws_bytes < stage_bytes(s, OMNIMOE_STAGE_ROUTE_DENSE)) return OMNIMOE_ERR_WORKSPACE;
    L = (float*)ws;
  }
  // The logit GEMM with one "half" holding all N gating vectors of each head over the full
  // width of x, and an empty second half.
  Shape g = s;
  g.nr = (int)s.N;
  g.nc = 0;
  g.dk = s.d;
  g.col0 = 0;
  hipStream_t strm = (hipStream_t)stream;
  hipError_t e = omnimoe::launch_score(g, x, w_gate, w_gate, L, strm);
  if (e == hipSuccess) e = omnimoe::launch_select_dense(s.rows, s.N, s.K, L, idx, gates, strm);
  return hip_status(e);
}

omnimoe_status omnimoe_select_dense(const omnimoe_layer_desc* desc, const float* logits,
                                    int32_t* idx, float* gates, void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({logits, idx, gates}))) return st;
  if (s.K > 64) return OMNIMOE_ERR_UNSUPPORTED;
  return hip_status(omnimoe::launch_select_dense(s.rows, s.N, s.K, logits, idx, gates,
                                                 (hipStream_t)stream));
}

namespace {

size_t mlp_ws_bytes(const Shape& s, int d_ff) {
  return align_up((size_t)s.T * 2 * d_ff * 4) + align_up((size_t)s.T * d_ff * (s.bf16 ? 2 : 4));
}

bool valid_d_ff(int32_t d_ff) { return d_ff >= 8 && d_ff <= 65536 && d_ff % 8 == 0; }

}  // namespace

omnimoe_status omnimoe_shared_mlp_workspace_size(const omnimoe_layer_desc* desc, int32_t d_ff,
                                                 size_t* bytes) {
  if (!bytes || !valid_d_ff(d_ff)) return OMNIMOE_ERR_INVALID_ARG;
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  *bytes = mlp_ws_bytes(s, d_ff);
  return OMNIMOE_OK;
}

omnimoe_status omnimoe_shared_mlp(const omnimoe_layer_desc* desc, int32_t d_ff, const void* x,
                                  const void* w_gu, const void* w_down, float* y, void* ws,
                                  size_t ws_bytes, void* stream) {
  if (!valid_d_ff(d_ff)) return OMNIMOE_ERR_INVALID_ARG;
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({x, w_gu, w_down, y, ws}))) return st;
  if (ws_bytes < mlp_ws_bytes(s, d_ff)) return OMNIMOE_ERR_WORKSPACE;
  float* h = (float*)ws;
  void* act = (char*)ws + align_up((size_t)s.T * 2 * d_ff * 4);
  hipStream_t strm = (hipStream_t)stream;
  // gate and up projections: h [T, 2 d_ff] = x w_gu^T
  Shape g = s;
  g.H = 1;
  g.nr = 2 * d_ff;
  g.nc = 0;
  g.dk = s.d;
  g.col0 = 0;
  hipError_t e = omnimoe::launch_score(g, x, w_gu, w_gu, h, strm);
  if (e == hipSuccess) e = omnimoe::launch_swiglu(s.T, d_ff, s.bf16, h, act, strm);
  // down projection added into y: y [T, d] += act w_down^T
  Shape dn = s;
  dn.H = 1;
  dn.d = d_ff;
  dn.dk = d_ff;
  dn.nr = s.d;
  dn.nc = 0;
  dn.col0 = 0;
  if (e == hipSuccess) e = omnimoe::launch_score(dn, act, w_down, w_down, y, strm, true);
  return hip_status(e);
}

omnimoe_status omnimoe_select(const omnimoe_layer_desc* desc, const float* half_scores,
                              int32_t* idx, float* gates, void* ws, size_t ws_bytes,
                              void* stream) {
  (void)ws;
  (void)ws_bytes;
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({half_scores, idx, gates}))) return st;
  return hip_status(omnimoe::launch_select(s, half_scores, idx, gates, (hipStream_t)stream));
}

omnimoe_status omnimoe_schedule(const omnimoe_layer_desc* desc, const int32_t* idx,
                                int32_t* perm, int32_t* active, int32_t* active_offsets,
                                int32_t* n_active, int32_t* dense_offsets, void* ws,
                                size_t ws_bytes, void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if ((st = check_ptrs({active_offsets, n_active}))) return st;
  if ((st = check_opt(dense_offsets))) return st;
  hipStream_t strm = (hipStream_t)stream;
  if (s.T == 0) {
    // No tasks: an empty schedule.
    hipError_t e = omnimoe::launch_fill_i32(n_active, 1, 0, strm);
    if (e == hipSuccess) e = omnimoe::launch_fill_i32(active_offsets, 1, 0, strm);
    if (e == hipSuccess && dense_offsets)
      e = omnimoe::launch_fill_i32(dense_offsets, s.N + 1, 0, strm);
    return hip_status(e);
  }
  if ((st = check_ptrs({idx, perm, active, ws}))) return st;
  if (ws_bytes < stage_bytes(s, OMNIMOE_STAGE_SCHEDULE)) return OMNIMOE_ERR_WORKSPACE;
  const int32_t* sk = nullptr;
  return hip_status(omnimoe::launch_schedule(s, idx, perm, active, active_offsets, n_active,
                                             dense_offsets, ws, &sk, strm));
}

omnimoe_status omnimoe_expert_forward(const omnimoe_layer_desc* desc, const void* x,
                                      const void* u, const void* v, const int32_t* idx,
                                      const float* gates, const int32_t* perm, float* y,
                                      void* ws, size_t ws_bytes, void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({x, u, v, idx, gates, perm, y, ws}))) return st;
  if (ws_bytes < stage_bytes(s, OMNIMOE_STAGE_EXPERT)) return OMNIMOE_ERR_WORKSPACE;
  hipStream_t strm = (hipStream_t)stream;
  float* abuf = (float*)ws;
  hipError_t e = omnimoe::launch_expert_dot(s, x, u, idx, gates, perm, nullptr, abuf, strm);
  if (e == hipSuccess) e = routed_sum(s, v, idx, abuf, y, (char*)ws + m_bytes(s), strm);
  return hip_status(e);
}

omnimoe_status omnimoe_expert_forward_grouped(const omnimoe_layer_desc* desc, const void* x,
                                              const void* u, const void* v, const int32_t* idx,
                                              const float* gates, const int32_t* perm,
                                              const int32_t* active, const int32_t* n_active,
                                              float* y, void* ws, size_t ws_bytes,
                                              void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({x, u, v, idx, gates, perm, active, n_active, y, ws}))) return st;
  if (!grouped_supported(s)) return OMNIMOE_ERR_UNSUPPORTED;
  if (ws_bytes < stage_bytes(s, OMNIMOE_STAGE_EXPERT_GROUPED)) return OMNIMOE_ERR_WORKSPACE;
  hipStream_t strm = (hipStream_t)stream;
  float* abuf = (float*)ws;
  omnimoe::GroupPlan plan;
  hipError_t e = omnimoe::launch_group_plan(s, perm, n_active, nullptr, idx, active,
                                            (char*)ws + m_bytes(s), &plan, strm);
  if (e == hipSuccess)
    e = omnimoe::launch_grouped_dot(s, x, u, gates, perm, active, n_active, plan, abuf, strm);
  if (e == hipSuccess) e = routed_sum(s, v, idx, abuf, y, (char*)ws + m_bytes(s), strm);
  return hip_status(e);
}

omnimoe_status omnimoe_expert_forward_group_rows(const omnimoe_layer_desc* desc, const void* x,
                                                 const void* u, const void* v,
                                                 const int32_t* idx, const float* gates,
                                                 const int32_t* perm, const int32_t* active,
                                                 const int32_t* n_active, float* y, void* ws,
                                                 size_t ws_bytes, void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({x, u, v, idx, gates, perm, active, n_active, y, ws}))) return st;
  if (!grouped_supported(s)) return OMNIMOE_ERR_UNSUPPORTED;
  if (ws_bytes < stage_bytes(s, OMNIMOE_STAGE_EXPERT_GROUP_ROWS)) return OMNIMOE_ERR_WORKSPACE;
  hipStream_t strm = (hipStream_t)stream;
  const int64_t n = group_rows_bound(s);
  char* w = (char*)ws;
  float* abuf = (float*)w; w += m_bytes(s);
  void* plan_ws = w; w += omnimoe::group_plan_ws_bytes(s);
  float* rows = (float*)w; w += align_up((size_t)n * s.d * 4);
  void* sort_ws = w;
  omnimoe::GroupPlan plan;
  omnimoe::SlotOrder order;
  hipError_t e = omnimoe::launch_group_plan(s, perm, n_active, nullptr, idx, active, plan_ws,
                                            &plan, strm);
  if (e == hipSuccess)
    e = omnimoe::launch_grouped_dot(s, x, u, gates, perm, active, n_active, plan, abuf, strm);
  if (e == hipSuccess) e = omnimoe::launch_slot_sort(plan, n, s.T, sort_ws, &order, strm);
  if (e == hipSuccess)
    e = omnimoe::launch_group_rows(s, v, idx, perm, abuf, plan, order, rows, n, y, strm);
  return hip_status(e);
}

omnimoe_status omnimoe_expert_forward_scatter(const omnimoe_layer_desc* desc, const void* x,
                                              const void* u, const void* v, const int32_t* idx,
                                              const float* gates, const int32_t* perm, float* y,
                                              void* ws, size_t ws_bytes, void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({x, u, v, idx, gates, perm, y, ws}))) return st;
  if (ws_bytes < stage_bytes(s, OMNIMOE_STAGE_EXPERT_SCATTER)) return OMNIMOE_ERR_WORKSPACE;
  float* abuf = (float*)ws;
  float* cbuf = (float*)((char*)ws + m_bytes(s));
  return hip_status(omnimoe::launch_expert_contrib(s, x, u, v, idx, gates, perm, abuf, cbuf, y,
                                                   (hipStream_t)stream));
}

omnimoe_status omnimoe_expert_forward_token_centric(const omnimoe_layer_desc* desc,
                                                   const void* x, const void* u, const void* v,
                                                   const int32_t* idx, const float* gates,
                                                   float* y, void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({x, u, v, idx, gates, y}))) return st;
  return hip_status(omnimoe::launch_token_centric(s, x, u, v, idx, gates, y,
                                                  (hipStream_t)stream));
}

omnimoe_status omnimoe_expert_backward(const omnimoe_layer_desc* desc, const void* x,
                                       const void* u, const void* v, const int32_t* idx,
                                       const float* gates, const int32_t* perm,
                                       const int32_t* active_offsets, const int32_t* n_active,
                                       const float* dy, float* dx, float* du_rows,
                                       float* dv_rows, float* dgates, float* dscores, void* ws,
                                       size_t ws_bytes, void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if (s.d > (s.bf16 ? 4096 : 2048)) return OMNIMOE_ERR_UNSUPPORTED;
  if ((st = check_ptrs({x, u, v, idx, gates, perm, active_offsets, n_active, dy, dx, du_rows,
                        dv_rows, dgates, dscores, ws})))
    return st;
  if (ws_bytes < stage_bytes(s, OMNIMOE_STAGE_EXPERT_BACKWARD)) return OMNIMOE_ERR_WORKSPACE;
  return hip_status(omnimoe::launch_expert_backward(s, x, u, v, idx, gates, perm, active_offsets,
                                                    n_active, dy, dx, du_rows, dv_rows, dgates,
                                                    dscores, ws, (hipStream_t)stream));
}

omnimoe_status omnimoe_route_backward(const omnimoe_layer_desc* desc, const void* x,
                                      const void* keys_row, const void* keys_col,
                                      const int32_t* idx, const float* dscores, float* dx,
                                      float* dkeys_row, float* dkeys_col, void* ws,
                                      size_t ws_bytes, void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if (s.dk > (s.bf16 ? 4096 : 2048)) return OMNIMOE_ERR_UNSUPPORTED;
  if ((st = check_ptrs({x, keys_row, keys_col, idx, dscores, dx, dkeys_row, dkeys_col, ws})))
    return st;
  if (ws_bytes < stage_bytes(s, OMNIMOE_STAGE_ROUTE_BACKWARD)) return OMNIMOE_ERR_WORKSPACE;
  return hip_status(omnimoe::launch_route_backward(s, x, keys_row, keys_col, idx, dscores, dx,
                                                   dkeys_row, dkeys_col, ws,
                                                   (hipStream_t)stream));
}

omnimoe_status omnimoe_layer_forward(const omnimoe_layer_desc* desc, const void* x,
                                     const void* keys_row, const void* keys_col, const void* u,
                                     const void* v, float* y, int32_t* idx_out, float* gates_out,
                                     void* ws, size_t ws_bytes, void* stream) {
  return layer_impl(desc, x, keys_row, keys_col, u, v, y, idx_out, gates_out, ws, ws_bytes,
                    stream, nullptr);
}

omnimoe_status omnimoe_layer_path(const omnimoe_layer_desc* desc, int32_t* path) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (!path) return OMNIMOE_ERR_INVALID_ARG;
  *path = layer_path(s);
  return OMNIMOE_OK;
}

omnimoe_status omnimoe_layer_forward_noalloc(const omnimoe_layer_desc* desc, const void* x,
                                             const void* keys_row, const void* keys_col,
                                             const void* u, const void* v, float* y,
                                             int32_t* idx_out, float* gates_out, void* stream) {
  Shape s;
  omnimoe_status st = check_desc(desc, &s);
  if (st) return st;
  if (s.T == 0) return OMNIMOE_OK;
  if ((st = check_ptrs({x, keys_row, keys_col, u, v, y}))) return st;
  if ((st = check_opt(idx_out)) || (st = check_opt(gates_out))) return st;
  if (stage_bytes(s, OMNIMOE_STAGE_LAYER) > (size_t)OMNIMOE_NOALLOC_SCRATCH_BYTES)
    return OMNIMOE_ERR_WORKSPACE;
  void* ws = nullptr;
  if ((st = noalloc_scratch(&ws))) return st;
  return layer_impl(desc, x, keys_row, keys_col, u, v, y, idx_out, gates_out, ws,
                    (size_t)OMNIMOE_NOALLOC_SCRATCH_BYTES, stream, nullptr);
}

omnimoe_status omnimoe_layer_forward_timed(const omnimoe_layer_desc* desc, const void* x,
                                           const void* keys_row, const void* keys_col,
                                           const void* u, const void* v, float* y,
                                           int32_t* idx_out, float* gates_out, void* ws,
                                           size_t ws_bytes, void* stream, omnimoe_timer* timer) {
  if (!timer) return OMNIMOE_ERR_INVALID_ARG;
  return layer_impl(desc, x, keys_row, keys_col, u, v, y, idx_out, gates_out, ws, ws_bytes,
                    stream, timer);
}

omnimoe_status omnimoe_timer_create(int32_t capacity, omnimoe_timer** out) {
  if (!out || capacity < 1 || capacity > 100000) return OMNIMOE_ERR_INVALID_ARG;
  omnimoe_timer* t = new (std::nothrow) omnimoe_timer();
  if (!t) return OMNIMOE_ERR_INVALID_ARG;
  t->capacity = capacity;
  t->ev.resize((size_t)capacity * kEv, nullptr);
  for (auto& e : t->ev) {
    if (hipEventCreate(&e) != hipSuccess) {
      e = nullptr;
      omnimoe_timer_destroy(t);
      return OMNIMOE_ERR_HIP;
    }
  }
  *out = t;
  return OMNIMOE_OK;
}

omnimoe_status omnimoe_timer_destroy(omnimoe_timer* t) {
  if (!t) return OMNIMOE_ERR_INVALID_ARG;
  for (auto e : t->ev)
    if (e) (void)hipEventDestroy(e);
  delete t;
  return OMNIMOE_OK;
}

omnimoe_status omnimoe_timer_read(omnimoe_timer* t, float* ms, int32_t* n_calls) {
  if (!t || !ms) return OMNIMOE_ERR_INVALID_ARG;
  for (int k = 0; k < OMNIMOE_KERNEL_COUNT; ++k) ms[k] = 0.0f;
  for (int c = 0; c < t->used; ++c) {
    hipEvent_t* ev = &t->ev[(size_t)c * kEv];
    if (hipEventSynchronize(ev[kEv - 1]) != hipSuccess) return OMNIMOE_ERR_HIP;
    for (int k = 0; k < OMNIMOE_KERNEL_COUNT; ++k) {
      float dt = 0.0f;
      if (hipEventElapsedTime(&dt, ev[k], ev[k + 1]) != hipSuccess) return OMNIMOE_ERR_HIP;
      ms[k] += dt;
    }
  }
  if (n_calls) *n_calls = t->used;
  t->used = 0;
  return OMNIMOE_OK;
}

}  // extern "C"
