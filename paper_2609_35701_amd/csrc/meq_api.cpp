// Host side of the MeqMuon C ABI: argument validation, shape grouping, the
// workspace layout, and the launch sequence of one step for each parameter kind
// (the three branches of Algorithm "MeqMuon", and the Moonlight-Muon rule for hidden
// weights).  meq_init_kind touches no device; meq_step only enqueues.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <memory>
#include <new>
#include <utility>
#include <vector>

#include "meq.h"
#include "meq_internal.h"

#define MEQ_EXPORT extern "C" __attribute__((visibility("default")))

using namespace meq;

namespace {

constexpr size_t kAlign = 256;
constexpr int64_t kMaxDim = 65536;
constexpr int64_t kMaxAuxRows = int64_t{1} << 24;
constexpr int64_t kMaxElems = (int64_t{1} << 31) - 1;
// Every per-matrix wide buffer must stay addressable with 32-bit byte offsets.
constexpr int64_t kMaxWideBytes = (int64_t{1} << 31) - 1;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }
int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

struct MatInfo {
  int64_t m, n, s, l, S, L;
  bool tall;
  int dtype;  // param dtype == grad dtype
  int group, gidx;
  int tiles_pad_r, tiles_pad_c;  // kEwRows x kEwCols tiles over the padded matrix in its own orientation
  int tiles_upd_r, tiles_upd_c;  // kEwRows x kEwCols tiles over the real matrix
  size_t off_part, off_rrms, off_crms, off_scale;
  // aux and vector plans
  int row_blocks;
  int64_t len;
  size_t off_rscale, off_cscale, off_cpart, off_normsq;
};

struct GroupInfo {
  int64_t s, l, S, L;
  std::vector<int> mats;
  size_t off_xa, off_xb, off_a, off_p, off_rpart, off_cpart, off_fold;
  int64_t stride_x, stride_a, stride_rpart, stride_cpart;  // elements per matrix
};

struct TimedLaunch {
  int kind;
  hipEvent_t start, stop;
};

}  // namespace

struct meq_plan {
  int kind = MEQ_PARAM_HIDDEN;
  meq_hparams hp;
  std::vector<MatInfo> mats;
  std::vector<GroupInfo> groups;
  size_t off_scal = 0;
  size_t ws_bytes = 0;
  uint32_t timing_mask = 0;
  std::vector<TimedLaunch> pending;
  std::vector<hipEvent_t> event_pool;
  double total_ms[MEQ_K_COUNT] = {};
  int64_t launches[MEQ_K_COUNT] = {};
};

namespace {

bool finite(float v) { return std::isfinite(v); }

meq_status validate_hparams(const meq_hparams& hp) {
  if (!finite(hp.mu) || hp.mu < 0.f || hp.mu >= 1.f) return MEQ_ERR_INVALID_ARG;
  if (!finite(hp.rho) || hp.rho <= 0.f) return MEQ_ERR_INVALID_ARG;
  if (!finite(hp.weight_decay) || hp.weight_decay < 0.f) return MEQ_ERR_INVALID_ARG;
  if (hp.ns_steps < 1 || hp.ns_steps > 64) return MEQ_ERR_INVALID_ARG;
  if (!finite(hp.ns_a) || !finite(hp.ns_b) || !finite(hp.ns_c)) return MEQ_ERR_INVALID_ARG;
  if (!finite(hp.zero_rms_delta) || hp.zero_rms_delta < 0.f) return MEQ_ERR_INVALID_ARG;
  if (hp.nesterov != 0 && hp.nesterov != 1) return MEQ_ERR_INVALID_ARG;
  if (hp.update_rule != MEQ_RULE_MEQMUON && hp.update_rule != MEQ_RULE_MOONLIGHT) return MEQ_ERR_INVALID_ARG;
  return MEQ_OK;
}

// (param, grad) dtypes: both known, and equal.
meq_status validate_dtypes(const meq_matrix_desc& d) {
  const bool known = (d.param_dtype == MEQ_F32 || d.param_dtype == MEQ_BF16) &&
                     (d.grad_dtype == MEQ_F32 || d.grad_dtype == MEQ_BF16);
  if (!known) return MEQ_ERR_INVALID_ARG;
  if (d.param_dtype != d.grad_dtype) return MEQ_ERR_UNSUPPORTED;
  return MEQ_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

hipEvent_t take_event(meq_plan* p) {
  if (!p->event_pool.empty()) {
    hipEvent_t e = p->event_pool.back();
    p->event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Launch `fn` (which returns the launch's hipError_t), bracketed by events when
// the kind is being timed.
template <typename F>
meq_status timed_launch(meq_plan* p, int kind, hipStream_t st, F&& fn) {
  const bool timed = (p->timing_mask >> kind) & 1u;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (timed) {
    p->pending.reserve(p->pending.size() + 1);  // may throw: before anything is recorded
    e0 = take_event(p);
    e1 = take_event(p);
    if (!e0 || !e1 || hipEventRecord(e0, st) != hipSuccess) return MEQ_ERR_HIP;
  }
  if (fn() != hipSuccess) return MEQ_ERR_HIP;
  if (timed) {
    if (hipEventRecord(e1, st) != hipSuccess) return MEQ_ERR_HIP;
    p->pending.push_back({kind, e0, e1});
  }
  return MEQ_OK;
}

#define MEQ_TRY(expr)                 \
  do {                                \
    const meq_status _s = (expr);     \
    if (_s != MEQ_OK) return _s;      \
  } while (0)

// Exported calls keep C++ exceptions (host allocations) on this side of the C ABI.
template <typename F>
meq_status guarded(F&& fn) {
  try {
    return fn();
  } catch (const std::bad_alloc&) {
    return MEQ_ERR_NO_MEMORY;
  } catch (...) {
    return MEQ_ERR_INVALID_ARG;
  }
}

}  // namespace

// ======================================================================== ABI
MEQ_EXPORT void meq_default_hparams(meq_hparams* hp) {
  if (!hp) return;
  hp->mu = 0.95f;
  hp->rho = 0.2f;
  hp->weight_decay = 0.1f;
  hp->ns_steps = 5;
  hp->ns_a = 3.4445f;
  hp->ns_b = -4.7750f;
  hp->ns_c = 2.0315f;
  hp->zero_rms_delta = 1e-7f;
  hp->nesterov = 0;
  hp->update_rule = MEQ_RULE_MEQMUON;
}

MEQ_EXPORT const char* meq_status_string(meq_status s) {
  switch (s) {
    case MEQ_OK: return "ok";
    case MEQ_ERR_INVALID_ARG: return "invalid argument";
    case MEQ_ERR_UNSUPPORTED: return "unsupported dtype or size";
    case MEQ_ERR_HIP: return "HIP runtime error";
    case MEQ_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case MEQ_ERR_NO_MEMORY: return "host memory allocation failed";
  }
  return "unknown status";
}

namespace {

// Hidden 2D weights: shape groups for the Newton-Schulz launches and the workspace layout.
meq_status init_hidden(const meq_matrix_desc* mats, int32_t count, const meq_hparams* hp, meq_plan** out) {
  for (int i = 0; i < count; ++i) {
    const meq_matrix_desc& d = mats[i];
    if (d.rows < 1 || d.cols < 1 || d.rows > kMaxDim || d.cols > kMaxDim) return MEQ_ERR_INVALID_ARG;
    MEQ_TRY(validate_dtypes(d));
    const int64_t S = round_up(std::min(d.rows, d.cols), kTile), L = round_up(std::max(d.rows, d.cols), kTile);
    if (S * L * 2 > kMaxWideBytes) return MEQ_ERR_UNSUPPORTED;
  }
  meq_plan* p = new (std::nothrow) meq_plan();
  if (!p) return MEQ_ERR_NO_MEMORY;
  std::unique_ptr<meq_plan> owner(p);  // freed if an allocation below throws
  p->hp = *hp;
  p->mats.resize(count);
  std::map<std::pair<int64_t, int64_t>, int> group_of;
  for (int i = 0; i < count; ++i) {
    MatInfo& mi = p->mats[i];
    mi.m = mats[i].rows;
    mi.n = mats[i].cols;
    mi.tall = mi.m > mi.n;
    mi.s = std::min(mi.m, mi.n);
    mi.l = std::max(mi.m, mi.n);
    mi.S = round_up(mi.s, kTile);
    mi.L = round_up(mi.l, kTile);
    mi.dtype = mats[i].param_dtype;
    const int64_t pad_r = mi.tall ? mi.L : mi.S, pad_c = mi.tall ? mi.S : mi.L;
    mi.tiles_pad_r = static_cast<int>(pad_r / kEwRows);
    mi.tiles_pad_c = static_cast<int>(pad_c / kEwCols);
    mi.tiles_upd_r = static_cast<int>((mi.m + kEwRows - 1) / kEwRows);
    mi.tiles_upd_c = static_cast<int>((mi.n + kEwCols - 1) / kEwCols);
    auto key = std::make_pair(mi.s, mi.l);
    auto it = group_of.find(key);
    if (it == group_of.end()) {
      it = group_of.emplace(key, static_cast<int>(p->groups.size())).first;
      GroupInfo g{};
      g.s = mi.s;
      g.l = mi.l;
      g.S = mi.S;
      g.L = mi.L;
      p->groups.push_back(g);
    }
    mi.group = it->second;
    mi.gidx = static_cast<int>(p->groups[mi.group].mats.size());
    p->groups[mi.group].mats.push_back(i);
  }
  // Workspace layout: per-matrix scalars, then each group's NS buffers, then
  // per-matrix partials and vectors.  Every region starts 256-byte aligned.
  size_t off = 0;
  p->off_scal = off;
  off = align_up(off + sizeof(MatScalars) * static_cast<size_t>(count), kAlign);
  for (GroupInfo& g : p->groups) {
    const size_t c = g.mats.size();
    g.stride_x = g.S * g.L;
    g.stride_a = g.S * g.S;
    g.stride_rpart = (g.L / kTile) * g.S;
    g.stride_cpart = (g.S / kTile) * g.L;
    g.off_fold = off;
    off = align_up(off + 8 * c, kAlign);
    g.off_xa = off;
    off = align_up(off + 2 * c * g.stride_x, kAlign);
    g.off_xb = off;
    off = align_up(off + 2 * c * g.stride_x, kAlign);
    g.off_a = off;
    off = align_up(off + 2 * c * g.stride_a, kAlign);
    g.off_p = off;
    off = align_up(off + 2 * c * g.stride_a, kAlign);
    g.off_rpart = off;
    off = align_up(off + 4 * c * g.stride_rpart, kAlign);
    g.off_cpart = off;
    off = align_up(off + 4 * c * g.stride_cpart, kAlign);
  }
  for (MatInfo& mi : p->mats) {
    mi.off_part = off;
    off = align_up(off + 4 * static_cast<size_t>(mi.tiles_pad_r) * mi.tiles_pad_c, kAlign);
    mi.off_rrms = off;
    off = align_up(off + 8 * static_cast<size_t>(mi.m), kAlign);
    mi.off_crms = off;
    off = align_up(off + 8 * static_cast<size_t>(mi.n), kAlign);
    mi.off_scale = off;
    off = align_up(off + 4 * static_cast<size_t>(std::max(mi.m, mi.n)), kAlign);
  }
  p->ws_bytes = off;
  *out = owner.release();
  return MEQ_OK;
}

// Remaining 2D parameters (eq. "aux") and 1-D parameters (eq. "vector"): per-parameter
// vectors and partials only.
meq_status init_stream_kind(int32_t kind, const meq_matrix_desc* mats, int32_t count, const meq_hparams* hp,
                            meq_plan** out) {
  for (int i = 0; i < count; ++i) {
    const meq_matrix_desc& d = mats[i];
    if (d.rows < 1 || d.cols < 1 || d.rows > kMaxElems || d.cols > kMaxElems) return MEQ_ERR_INVALID_ARG;
    if (d.rows * d.cols > kMaxElems) return MEQ_ERR_UNSUPPORTED;
    if (kind == MEQ_PARAM_AUX && (d.rows > kMaxAuxRows || d.cols > kMaxDim)) return MEQ_ERR_UNSUPPORTED;
    MEQ_TRY(validate_dtypes(d));
  }
  meq_plan* p = new (std::nothrow) meq_plan();
  if (!p) return MEQ_ERR_NO_MEMORY;
  std::unique_ptr<meq_plan> owner(p);
  p->kind = kind;
  p->hp = *hp;
  p->mats.resize(count);
  size_t off = 0;
  for (int i = 0; i < count; ++i) {
    MatInfo& mi = p->mats[i];
    mi = MatInfo{};
    mi.m = mats[i].rows;
    mi.n = mats[i].cols;
    mi.len = mi.m * mi.n;
    mi.dtype = mats[i].param_dtype;
    if (kind == MEQ_PARAM_AUX) {
      mi.row_blocks = static_cast<int>((mi.m + kAuxColRows - 1) / kAuxColRows);
      mi.off_rrms = off;
      off = align_up(off + 8 * static_cast<size_t>(mi.m), kAlign);
      mi.off_crms = off;
      off = align_up(off + 8 * static_cast<size_t>(mi.n), kAlign);
      mi.off_rscale = off;
      off = align_up(off + 4 * static_cast<size_t>(mi.m), kAlign);
      mi.off_cscale = off;
      off = align_up(off + 4 * static_cast<size_t>(mi.n), kAlign);
      mi.off_cpart = off;
      off = align_up(off + 8 * static_cast<size_t>(mi.row_blocks) * mi.n, kAlign);
    } else {
      mi.off_normsq = off;
      off = align_up(off + 8, kAlign);
    }
  }
  p->ws_bytes = off;
  *out = owner.release();
  return MEQ_OK;
}

}  // namespace

MEQ_EXPORT meq_status meq_init_kind(int32_t kind, const meq_matrix_desc* mats, int32_t count, const meq_hparams* hp,
                                    meq_plan** out) {
  if (out) *out = nullptr;
  if (!out || !hp || count < 0 || (count > 0 && !mats)) return MEQ_ERR_INVALID_ARG;
  if (kind != MEQ_PARAM_HIDDEN && kind != MEQ_PARAM_AUX && kind != MEQ_PARAM_VECTOR) return MEQ_ERR_INVALID_ARG;
  MEQ_TRY(validate_hparams(*hp));
  if (hp->update_rule != MEQ_RULE_MEQMUON && kind != MEQ_PARAM_HIDDEN) return MEQ_ERR_INVALID_ARG;
  return guarded([&] {
    return kind == MEQ_PARAM_HIDDEN ? init_hidden(mats, count, hp, out) : init_stream_kind(kind, mats, count, hp, out);
  });
}

MEQ_EXPORT meq_status meq_init(const meq_matrix_desc* mats, int32_t count, const meq_hparams* hp, meq_plan** out) {
  return meq_init_kind(MEQ_PARAM_HIDDEN, mats, count, hp, out);
}

MEQ_EXPORT size_t meq_workspace_bytes(const meq_plan* plan) { return plan ? plan->ws_bytes : 0; }

MEQ_EXPORT int32_t meq_plan_num_groups(const meq_plan* plan) {
  return plan ? static_cast<int32_t>(plan->groups.size()) : 0;
}

MEQ_EXPORT meq_status meq_plan_group(const meq_plan* plan, int32_t g, int64_t* s, int64_t* l, int32_t* count) {
  if (!plan || g < 0 || g >= static_cast<int32_t>(plan->groups.size())) return MEQ_ERR_INVALID_ARG;
  const GroupInfo& gi = plan->groups[g];
  if (s) *s = gi.s;
  if (l) *l = gi.l;
  if (count) *count = static_cast<int32_t>(gi.mats.size());
  return MEQ_OK;
}

MEQ_EXPORT meq_status meq_debug_region(const meq_plan* plan, int32_t matrix, int32_t kind, size_t* offset,
                                       int64_t* rows, int64_t* cols, int64_t* ld) {
  if (!plan || matrix < 0 || matrix >= static_cast<int32_t>(plan->mats.size())) return MEQ_ERR_INVALID_ARG;
  const MatInfo& mi = plan->mats[matrix];
  size_t o = 0;
  int64_t r = 1, c = 1, d = 1;
  if (plan->kind != MEQ_PARAM_HIDDEN) {
    if (plan->kind == MEQ_PARAM_AUX && kind == MEQ_BUF_ROW_RMS) {
      o = mi.off_rrms;
      c = d = mi.m;
    } else if (plan->kind == MEQ_PARAM_AUX && kind == MEQ_BUF_COL_RMS) {
      o = mi.off_crms;
      c = d = mi.n;
    } else if (plan->kind == MEQ_PARAM_VECTOR && kind == MEQ_BUF_NORMSQ) {
      o = mi.off_normsq;
    } else {
      return MEQ_ERR_INVALID_ARG;
    }
    if (offset) *offset = o;
    if (rows) *rows = r;
    if (cols) *cols = c;
    if (ld) *ld = d;
    return MEQ_OK;
  }
  const GroupInfo& g = plan->groups[mi.group];
  switch (kind) {
    case MEQ_BUF_X0:
    case MEQ_BUF_U: {
      // X_0 sits in buffer a; iteration k writes buffer b when k is even, so the
      // output of K steps is in b for odd K and in a for even K.
      const bool in_b = kind == MEQ_BUF_U && (plan->hp.ns_steps % 2 == 1);
      o = (in_b ? g.off_xb : g.off_xa) + 2 * static_cast<size_t>(mi.gidx) * g.stride_x;
      r = mi.s;
      c = mi.l;
      d = g.L;
      break;
    }
    case MEQ_BUF_NORMSQ:
      o = plan->off_scal + sizeof(MatScalars) * matrix + offsetof(MatScalars, normsq);
      break;
    case MEQ_BUF_ROW_RMS:
      o = mi.off_rrms;
      c = mi.m;
      d = mi.m;
      break;
    case MEQ_BUF_COL_RMS:
      o = mi.off_crms;
      c = mi.n;
      d = mi.n;
      break;
    case MEQ_BUF_SCALE:
      o = mi.off_scale;
      c = std::max(mi.m, mi.n);
      d = c;
      break;
    default:
      return MEQ_ERR_INVALID_ARG;
  }
  if (offset) *offset = o;
  if (rows) *rows = r;
  if (cols) *cols = c;
  if (ld) *ld = d;
  return MEQ_OK;
}

namespace {

float decay_of(const meq_hparams& hp, float lr) {
  return static_cast<float>(1.0 - static_cast<double>(lr) * hp.weight_decay);
}
float step_of(const meq_hparams& hp, float lr) { return static_cast<float>(static_cast<double>(hp.rho) * lr); }

// Remaining 2D parameters, one matrix at a time: rows (momentum + r), columns (c of
// N_r(V)), write-back.
meq_status step_aux(meq_plan* p, void* const* params, const void* const* grads, float* const* momenta, float lr,
                    char* ws, hipStream_t st) {
  const meq_hparams& hp = p->hp;
  for (size_t i = 0; i < p->mats.size(); ++i) {
    const MatInfo& mi = p->mats[i];
    const bool bf = mi.dtype == MEQ_BF16;
    AuxArgs a{};
    a.m = static_cast<int>(mi.m);
    a.n = static_cast<int>(mi.n);
    a.nesterov = hp.nesterov;
    a.row_blocks = mi.row_blocks;
    a.mu = hp.mu;
    a.decay = decay_of(hp, lr);
    a.step = step_of(hp, lr);
    a.delta = static_cast<double>(hp.zero_rms_delta);
    a.g = grads[i];
    a.b = momenta[i];
    a.w = params[i];
    const size_t ea = bf ? 8 : 16;  // four elements of the parameter / gradient dtype
    a.vec = (mi.n % 4 == 0) && aligned(a.b, 16) && aligned(a.g, ea) && aligned(a.w, ea);
    a.rrms = reinterpret_cast<double*>(ws + mi.off_rrms);
    a.crms = reinterpret_cast<double*>(ws + mi.off_crms);
    a.rscale = reinterpret_cast<float*>(ws + mi.off_rscale);
    a.cscale = reinterpret_cast<float*>(ws + mi.off_cscale);
    a.cpart = reinterpret_cast<double*>(ws + mi.off_cpart);
    MEQ_TRY(timed_launch(p, MEQ_K_AUX_ROWS, st, [&] { return launch_aux_rows(a, bf, st); }));
    MEQ_TRY(timed_launch(p, MEQ_K_AUX_COLS, st, [&] { return launch_aux_cols(a, bf, st); }));
    MEQ_TRY(timed_launch(p, MEQ_K_AUX_COLS, st, [&] { return launch_aux_colfin(a, st); }));
    MEQ_TRY(timed_launch(p, MEQ_K_AUX_UPDATE, st, [&] { return launch_aux_update(a, bf, st); }));
  }
  return MEQ_OK;
}

// 1-D parameters: one block per vector, up to kMaxChunk vectors of one dtype per launch.
meq_status step_vec(meq_plan* p, void* const* params, const void* const* grads, float* const* momenta, float lr,
                    char* ws, hipStream_t st) {
  const meq_hparams& hp = p->hp;
  const int count = static_cast<int>(p->mats.size());
  for (int dt = 0; dt < 2; ++dt) {
    VecArgs a{};
    auto flush = [&]() -> meq_status {
      if (a.count == 0) return MEQ_OK;
      const VecArgs sent = a;
      a.count = 0;
      return timed_launch(p, MEQ_K_VECTOR, st, [&] { return launch_vec(sent, dt == MEQ_BF16, st); });
    };
    for (int i = 0; i < count; ++i) {
      const MatInfo& mi = p->mats[i];
      if (mi.dtype != dt) continue;
      const int k = a.count++;
      a.nesterov = hp.nesterov;
      a.mu = hp.mu;
      a.decay = decay_of(hp, lr);
      a.step = step_of(hp, lr);
      a.len[k] = mi.len;
      a.g[k] = grads[i];
      a.b[k] = momenta[i];
      a.w[k] = params[i];
      const size_t ea = dt == MEQ_BF16 ? 8 : 16;
      a.vec[k] = (mi.len % 4 == 0) && aligned(a.b[k], 16) && aligned(a.g[k], ea) && aligned(a.w[k], ea);
      a.normsq[k] = reinterpret_cast<double*>(ws + mi.off_normsq);
      if (a.count == kMaxChunk) MEQ_TRY(flush());
    }
    MEQ_TRY(flush());
  }
  return MEQ_OK;
}

}  // namespace

namespace {

// Element-wise kernels run over chunks of matrices sharing a dtype.
std::vector<std::vector<int>> dtype_chunks(const meq_plan* p) {
  const int count = static_cast<int>(p->mats.size());
  std::vector<std::vector<int>> chunks;
  for (int dt = 0; dt < 2; ++dt) {
    std::vector<int> cur;
    for (int i = 0; i < count; ++i) {
      if (p->mats[i].dtype != dt) continue;
      cur.push_back(i);
      if (static_cast<int>(cur.size()) == kMaxChunk) {
        chunks.push_back(cur);
        cur.clear();
      }
    }
    if (!cur.empty()) chunks.push_back(cur);
  }
  return chunks;
}

// Steps a1-a2: momentum (or, with momenta == nullptr, V = the given inputs), bf16 V in wide
// orientation, ||V||_F^2 and its reciprocals.
meq_status enqueue_prescale(meq_plan* p, char* ws, const void* const* grads, float* const* momenta, hipStream_t st) {
  const meq_hparams& hp = p->hp;
  const int count = static_cast<int>(p->mats.size());
  MatScalars* scal = reinterpret_cast<MatScalars*>(ws + p->off_scal);
  const auto chunks = dtype_chunks(p);
  // 1. momentum + bf16 V (wide, zero-padded) + per-tile ||V||^2 partials
  for (const auto& ch : chunks) {
    MomentumArgs a{};
    a.count = static_cast<int>(ch.size());
    a.nesterov = hp.nesterov;
    a.mu = hp.mu;
    int tiles = 0;
    for (int k = 0; k < a.count; ++k) {
      const MatInfo& mi = p->mats[ch[k]];
      const GroupInfo& g = p->groups[mi.group];
      a.tile_start[k] = tiles;
      tiles += mi.tiles_pad_r * mi.tiles_pad_c;
      a.m[k] = static_cast<int>(mi.m);
      a.n[k] = static_cast<int>(mi.n);
      a.tiles_c[k] = mi.tiles_pad_c;
      a.tall[k] = mi.tall;
      a.ldx[k] = g.L;
      a.g[k] = grads[ch[k]];
      a.b[k] = momenta ? momenta[ch[k]] : nullptr;  // none: V is the input itself
      a.vec[k] = (mi.n % 8 == 0) && aligned(a.b[k], 16) && aligned(a.g[k], 16);
      a.x[k] = reinterpret_cast<uint16_t*>(ws + g.off_xa) + mi.gidx * g.stride_x;
      a.part[k] = reinterpret_cast<float*>(ws + mi.off_part);
    }
    a.tile_start[a.count] = tiles;
    const int gbf = p->mats[ch[0]].dtype == MEQ_BF16;
    MEQ_TRY(timed_launch(p, MEQ_K_MOMENTUM, st, [&] { return launch_momentum(a, gbf, tiles, st); }));
  }
  // 2. ||V||_F^2 and its reciprocals
  for (int c0 = 0; c0 < count; c0 += kMaxChunk) {
    NormArgs a{};
    a.count = std::min(kMaxChunk, count - c0);
    for (int k = 0; k < a.count; ++k) {
      const MatInfo& mi = p->mats[c0 + k];
      a.nparts[k] = mi.tiles_pad_r * mi.tiles_pad_c;
      a.part[k] = reinterpret_cast<const float*>(ws + mi.off_part);
      a.scal[k] = scal + c0 + k;
      a.fold[k] = reinterpret_cast<float*>(ws + p->groups[mi.group].off_fold) + 2 * mi.gidx;
    }
    MEQ_TRY(timed_launch(p, MEQ_K_NORM, st, [&] { return launch_norm(a, st); }));
  }
  return MEQ_OK;
}

// Step a3, iteration k of eq. "ns": per product one launch over all shape groups (chunks of
// kMaxGemmGroups), longest K first so the long tiles start first.  Ping-pong between buffers
// a (holding X_0) and b: iteration k reads a when k is even.  With `rowcol` the apply
// product also writes the row/column sums of squares of its output (step a4's partials).
meq_status enqueue_ns_iteration(meq_plan* p, char* ws, int k, bool rowcol, hipStream_t st) {
  const meq_hparams& hp = p->hp;
  std::vector<int> order(p->groups.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = static_cast<int>(i);
  {
    const bool from_a = (k % 2) == 0;
    for (int kind = 0; kind < 3; ++kind) {
      // kind 0: Gram (K = L), 1: polynomial (K = S), 2: apply (K = S)
      std::stable_sort(order.begin(), order.end(), [&](int x, int y) {
        const GroupInfo& gx = p->groups[x];
        const GroupInfo& gy = p->groups[y];
        const int64_t kx = kind == 0 ? gx.L : gx.S, ky = kind == 0 ? gy.L : gy.S;
        return kx > ky;
      });
      for (size_t c0 = 0; c0 < order.size(); c0 += kMaxGemmGroups) {
        GemmArgs ga{};
        ga.count = static_cast<int>(std::min<size_t>(kMaxGemmGroups, order.size() - c0));
        ga.scale_kind = k == 0 ? (kind == 0 ? 2 : kind == 2 ? 1 : 0) : 0;
        // The a X term of X <- a X + P X is carried by P: the polynomial product stores
        // a I + b A + c A A, and the apply product is the plain product (a I + P) X.
        ga.alpha_e = kind == 1 ? hp.ns_b : 0.f;
        ga.alpha_acc = kind == 1 ? hp.ns_c : 1.f;
        ga.alpha_diag = kind == 1 ? hp.ns_a : 0.f;
        int start = 0;
        for (int q = 0; q < ga.count; ++q) {
          const GroupInfo& g = p->groups[order[c0 + q]];
          const int batch = static_cast<int>(g.mats.size());
          const int tm = static_cast<int>(g.S / kTile), tn = static_cast<int>(g.L / kTile);
          uint16_t* cur = reinterpret_cast<uint16_t*>(ws + (from_a ? g.off_xa : g.off_xb));
          uint16_t* nxt = reinterpret_cast<uint16_t*>(ws + (from_a ? g.off_xb : g.off_xa));
          uint16_t* am = reinterpret_cast<uint16_t*>(ws + g.off_a);
          uint16_t* pm = reinterpret_cast<uint16_t*>(ws + g.off_p);
          GemmGroup& gg = ga.grp[q];
          gg.fold = reinterpret_cast<const float*>(ws + g.off_fold);
          if (kind == 0) {  // A = X X^T
            gg.a = cur; gg.lda = static_cast<int>(g.L); gg.stride_a = g.stride_x;
            gg.b = cur; gg.ldb = static_cast<int>(g.L); gg.stride_b = g.stride_x;
            gg.c = am; gg.ldc = static_cast<int>(g.S); gg.stride_c = g.stride_a;
            gg.e = nullptr; gg.lde = 0; gg.stride_e = 0;
            gg.K = static_cast<int>(g.L);
            gg.tiles_m = tm; gg.tiles_n = tm; gg.tiles_per_mat = tm * (tm + 1) / 2;
          } else if (kind == 1) {  // P = a I + b A + c A A
            gg.a = am; gg.lda = static_cast<int>(g.S); gg.stride_a = g.stride_a;
            gg.b = am; gg.ldb = static_cast<int>(g.S); gg.stride_b = g.stride_a;
            gg.c = pm; gg.ldc = static_cast<int>(g.S); gg.stride_c = g.stride_a;
            gg.e = am; gg.lde = static_cast<int>(g.S); gg.stride_e = g.stride_a;
            gg.K = static_cast<int>(g.S);
            gg.tiles_m = tm; gg.tiles_n = tm; gg.tiles_per_mat = tm * (tm + 1) / 2;
          } else {  // X <- (a I + b A + c A A) X
            gg.a = pm; gg.lda = static_cast<int>(g.S); gg.stride_a = g.stride_a;
            gg.b = cur; gg.ldb = static_cast<int>(g.L); gg.stride_b = g.stride_x;
            gg.c = nxt; gg.ldc = static_cast<int>(g.L); gg.stride_c = g.stride_x;
            gg.e = nullptr; gg.lde = 0; gg.stride_e = 0;
            gg.K = static_cast<int>(g.S);
            gg.tiles_m = tm; gg.tiles_n = tn; gg.tiles_per_mat = tm * tn;
            if (rowcol) {
              gg.rpart = reinterpret_cast<float*>(ws + g.off_rpart);
              gg.cpart = reinterpret_cast<float*>(ws + g.off_cpart);
              gg.stride_rpart = g.stride_rpart;
              gg.stride_cpart = g.stride_cpart;
            }
          }
          gg.tiles = gg.tiles_per_mat * batch;
          ga.tile_start[q] = start;
          start += (gg.tiles + 7) / 8 * 8;
        }
        ga.tile_start[ga.count] = start;
        const int kk = kind == 0 ? MEQ_K_GRAM : kind == 1 ? MEQ_K_POLY : MEQ_K_APPLY;
        MEQ_TRY(timed_launch(p, kk, st, [&] { return launch_gemm(ga, kind, st); }));
      }
    }
  }
  return MEQ_OK;
}

// Steps a4-a5 on the Newton-Schulz output in buffer b (u_in_b) or a: row/column RMS, CVs,
// direction and scale vectors; with the Moonlight rule only the uniform scale.  With
// `sums_done` the row/column sums of squares were already written by the last apply product.
meq_status enqueue_stats(meq_plan* p, char* ws, bool u_in_b, bool moonlight, bool sums_done, hipStream_t st) {
  const meq_hparams& hp = p->hp;
  const int count = static_cast<int>(p->mats.size());
  MatScalars* scal = reinterpret_cast<MatScalars*>(ws + p->off_scal);
  // 4. row / column sums of squares of U, per shape group (MeqMuon only)
  for (size_t gi = 0; gi < p->groups.size() && !moonlight && !sums_done; ++gi) {
    const GroupInfo& g = p->groups[gi];
    const int batch = static_cast<int>(g.mats.size());
    const int tm = static_cast<int>(g.S / kTile), tn = static_cast<int>(g.L / kTile);
    uint16_t* xa = reinterpret_cast<uint16_t*>(ws + g.off_xa);
    uint16_t* xb = reinterpret_cast<uint16_t*>(ws + g.off_xb);
    RowColArgs rc{};
    rc.u = u_in_b ? xb : xa;
    rc.stride_u = g.stride_x;
    rc.S = static_cast<int>(g.S);
    rc.L = static_cast<int>(g.L);
    rc.rpart = reinterpret_cast<float*>(ws + g.off_rpart);
    rc.stride_rpart = g.stride_rpart;
    rc.cpart = reinterpret_cast<float*>(ws + g.off_cpart);
    rc.stride_cpart = g.stride_cpart;
    rc.tiles_r = tm;
    rc.tiles_c = tn;
    MEQ_TRY(timed_launch(p, MEQ_K_ROWCOL, st, [&] { return launch_rowcol(rc, batch, st); }));
  }
  // 5. row/column RMS, CVs, direction, scale vectors (Moonlight: the uniform scale)
  for (int c0 = 0; c0 < count; c0 += kMaxChunk) {
    SelectArgs a{};
    a.count = std::min(kMaxChunk, count - c0);
    a.delta = static_cast<double>(hp.zero_rms_delta);
    for (int k = 0; k < a.count; ++k) {
      const MatInfo& mi = p->mats[c0 + k];
      const GroupInfo& g = p->groups[mi.group];
      a.m[k] = static_cast<int>(mi.m);
      a.n[k] = static_cast<int>(mi.n);
      a.tall[k] = mi.tall;
      a.S[k] = static_cast<int>(g.S);
      a.L[k] = static_cast<int>(g.L);
      a.rpart[k] = reinterpret_cast<const float*>(ws + g.off_rpart) + mi.gidx * g.stride_rpart;
      a.cpart[k] = reinterpret_cast<const float*>(ws + g.off_cpart) + mi.gidx * g.stride_cpart;
      a.rrms[k] = reinterpret_cast<double*>(ws + mi.off_rrms);
      a.crms[k] = reinterpret_cast<double*>(ws + mi.off_crms);
      a.scale[k] = reinterpret_cast<float*>(ws + mi.off_scale);
      a.scal[k] = scal + c0 + k;
      a.max_lines = std::max(a.max_lines, static_cast<int>(mi.s + mi.l));
    }
    if (moonlight) {
      // U~ = sqrt(max(m, n)) U: one scale for every row, no statistics
      MEQ_TRY(timed_launch(p, MEQ_K_SELECT, st, [&] { return launch_scale_fill(a, st); }));
    } else {
      MEQ_TRY(timed_launch(p, MEQ_K_SELECT, st, [&] { return launch_rms(a, st); }));
      MEQ_TRY(timed_launch(p, MEQ_K_SELECT, st, [&] { return launch_select(a, st); }));
    }
  }
  return MEQ_OK;
}

// Step a6: decoupled weight decay and the normalized update.
meq_status enqueue_update(meq_plan* p, char* ws, void* const* params, float lr, hipStream_t st) {
  const meq_hparams& hp = p->hp;
  MatScalars* scal = reinterpret_cast<MatScalars*>(ws + p->off_scal);
  const auto chunks = dtype_chunks(p);
  // 6. write-back
  const float decay = static_cast<float>(1.0 - static_cast<double>(lr) * hp.weight_decay);
  const float stepc = static_cast<float>(static_cast<double>(hp.rho) * lr);
  for (const auto& ch : chunks) {
    UpdateArgs a{};
    a.count = static_cast<int>(ch.size());
    a.decay = decay;
    a.step = stepc;
    int tiles = 0;
    for (int k = 0; k < a.count; ++k) {
      const MatInfo& mi = p->mats[ch[k]];
      const GroupInfo& g = p->groups[mi.group];
      a.tile_start[k] = tiles;
      tiles += mi.tiles_upd_r * mi.tiles_upd_c;
      a.m[k] = static_cast<int>(mi.m);
      a.n[k] = static_cast<int>(mi.n);
      a.tiles_c[k] = mi.tiles_upd_c;
      a.tall[k] = mi.tall;
      a.ldu[k] = g.L;
      a.w[k] = params[ch[k]];
      a.vec[k] = (mi.n % 8 == 0) && aligned(a.w[k], 16);
      const size_t uoff = (hp.ns_steps % 2 == 1) ? g.off_xb : g.off_xa;
      a.u[k] = reinterpret_cast<const uint16_t*>(ws + uoff) + mi.gidx * g.stride_x;
      a.scale[k] = reinterpret_cast<const float*>(ws + mi.off_scale);
      a.scal[k] = scal + ch[k];
    }
    a.tile_start[a.count] = tiles;
    const int pbf = p->mats[ch[0]].dtype == MEQ_BF16;
    MEQ_TRY(timed_launch(p, MEQ_K_UPDATE, st, [&] { return launch_update(a, pbf, tiles, st); }));
  }
  return MEQ_OK;
}

}  // namespace

MEQ_EXPORT meq_status meq_step(meq_plan* p, void* const* params, const void* const* grads, float* const* momenta,
                               float lr, void* workspace, size_t workspace_bytes, hipStream_t st) {
  if (!p) return MEQ_ERR_INVALID_ARG;
  const int count = static_cast<int>(p->mats.size());
  if (!std::isfinite(lr) || lr < 0.f) return MEQ_ERR_INVALID_ARG;
  if (count == 0) return MEQ_OK;
  if (!params || !grads || !momenta) return MEQ_ERR_INVALID_ARG;
  for (int i = 0; i < count; ++i)
    if (!params[i] || !grads[i] || !momenta[i]) return MEQ_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < p->ws_bytes || (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return MEQ_ERR_WORKSPACE;

  char* ws = static_cast<char*>(workspace);
  return guarded([&]() -> meq_status {
    if (p->kind == MEQ_PARAM_AUX) return step_aux(p, params, grads, momenta, lr, ws, st);
    if (p->kind == MEQ_PARAM_VECTOR) return step_vec(p, params, grads, momenta, lr, ws, st);
    const meq_hparams& hp = p->hp;
    const bool moonlight = hp.update_rule == MEQ_RULE_MOONLIGHT;
    MEQ_TRY(enqueue_prescale(p, ws, grads, momenta, st));
    for (int k = 0; k < hp.ns_steps; ++k)
      MEQ_TRY(enqueue_ns_iteration(p, ws, k, !moonlight && k == hp.ns_steps - 1, st));
    MEQ_TRY(enqueue_stats(p, ws, hp.ns_steps % 2 == 1, moonlight, !moonlight, st));
    MEQ_TRY(enqueue_update(p, ws, params, lr, st));
    return MEQ_OK;
  });
}

MEQ_EXPORT meq_status meq_ns_cv_trace(meq_plan* p, const void* const* inputs, int32_t kmax, void* workspace,
                                      size_t workspace_bytes, double* gamma_r, double* gamma_c, hipStream_t st) {
  if (!p || p->kind != MEQ_PARAM_HIDDEN || kmax < 0 || kmax > 64) return MEQ_ERR_INVALID_ARG;
  const int count = static_cast<int>(p->mats.size());
  if (count == 0) return MEQ_OK;
  if (!inputs || !gamma_r || !gamma_c) return MEQ_ERR_INVALID_ARG;
  for (int i = 0; i < count; ++i)
    if (!inputs[i]) return MEQ_ERR_INVALID_ARG;
  if (!workspace || workspace_bytes < p->ws_bytes || (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return MEQ_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  return guarded([&]() -> meq_status {
    std::vector<MatScalars> host(count);
    const char* src = ws + p->off_scal;
    MEQ_TRY(enqueue_prescale(p, ws, inputs, nullptr, st));
    for (int k = 0; k <= kmax; ++k) {
      if (k > 0) MEQ_TRY(enqueue_ns_iteration(p, ws, k - 1, false, st));
      // X_0 (unscaled V: CVs are scale free) sits in buffer a; iteration k - 1 writes b for odd k
      MEQ_TRY(enqueue_stats(p, ws, k % 2 == 1, false, false, st));
      if (hipMemcpyAsync(host.data(), src, sizeof(MatScalars) * count, hipMemcpyDeviceToHost, st) != hipSuccess)
        return MEQ_ERR_HIP;
      if (hipStreamSynchronize(st) != hipSuccess) return MEQ_ERR_HIP;
      for (int i = 0; i < count; ++i) {
        gamma_r[static_cast<size_t>(i) * (kmax + 1) + k] = host[i].gamma_r;
        gamma_c[static_cast<size_t>(i) * (kmax + 1) + k] = host[i].gamma_c;
      }
    }
    return MEQ_OK;
  });
}

MEQ_EXPORT meq_status meq_get_stats(const meq_plan* plan, const void* workspace, double* gamma_r, double* gamma_c,
                                    int32_t* dir, hipStream_t st) {
  if (!plan) return MEQ_ERR_INVALID_ARG;
  if (plan->kind != MEQ_PARAM_HIDDEN || plan->hp.update_rule != MEQ_RULE_MEQMUON) return MEQ_ERR_UNSUPPORTED;
  const size_t count = plan->mats.size();
  if (count == 0) return MEQ_OK;
  if (!workspace) return MEQ_ERR_WORKSPACE;
  return guarded([&]() -> meq_status {
    std::vector<MatScalars> host(count);
    const char* src = static_cast<const char*>(workspace) + plan->off_scal;
    if (hipMemcpyAsync(host.data(), src, sizeof(MatScalars) * count, hipMemcpyDeviceToHost, st) != hipSuccess)
      return MEQ_ERR_HIP;
    if (hipStreamSynchronize(st) != hipSuccess) return MEQ_ERR_HIP;
    for (size_t i = 0; i < count; ++i) {
      if (gamma_r) gamma_r[i] = host[i].gamma_r;
      if (gamma_c) gamma_c[i] = host[i].gamma_c;
      if (dir) dir[i] = host[i].dir;
    }
    return MEQ_OK;
  });
}

MEQ_EXPORT meq_status meq_set_timing(meq_plan* plan, uint32_t kind_mask) {
  if (!plan) return MEQ_ERR_INVALID_ARG;
  plan->timing_mask = kind_mask & ((1u << MEQ_K_COUNT) - 1);
  return MEQ_OK;
}

MEQ_EXPORT meq_status meq_get_timing(meq_plan* plan, int32_t kind, double* total_ms, int64_t* launches,
                                     int32_t reset) {
  if (!plan || kind < 0 || kind >= MEQ_K_COUNT) return MEQ_ERR_INVALID_ARG;
  // Fold the finished launches into the totals; on an error the launches already folded
  // are dropped from the pending list, so a later call does not count them twice.
  size_t done = 0;
  meq_status status = guarded([&]() -> meq_status {
    for (; done < plan->pending.size(); ++done) {
      const TimedLaunch& tl = plan->pending[done];
      if (hipEventSynchronize(tl.stop) != hipSuccess) return MEQ_ERR_HIP;
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, tl.start, tl.stop) != hipSuccess) return MEQ_ERR_HIP;
      plan->event_pool.reserve(plan->event_pool.size() + 2);
      plan->total_ms[tl.kind] += ms;
      plan->launches[tl.kind] += 1;
      plan->event_pool.push_back(tl.start);
      plan->event_pool.push_back(tl.stop);
    }
    return MEQ_OK;
  });
  plan->pending.erase(plan->pending.begin(), plan->pending.begin() + static_cast<std::ptrdiff_t>(done));
  if (status != MEQ_OK) return status;
  if (total_ms) *total_ms = plan->total_ms[kind];
  if (launches) *launches = plan->launches[kind];
  if (reset) {
    for (int k = 0; k < MEQ_K_COUNT; ++k) {
      plan->total_ms[k] = 0.0;
      plan->launches[k] = 0;
    }
  }
  return MEQ_OK;
}

MEQ_EXPORT void meq_destroy(meq_plan* plan) {
  if (!plan) return;
  for (const TimedLaunch& tl : plan->pending) {
    hipEventDestroy(tl.start);
    hipEventDestroy(tl.stop);
  }
  for (hipEvent_t e : plan->event_pool) hipEventDestroy(e);
  delete plan;
}
