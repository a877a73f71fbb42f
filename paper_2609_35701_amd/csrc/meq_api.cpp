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
  int group, gidx;  // group slice (index into meq_plan::groups) and position in it
  int pass;         // hidden plans: the pass that updates this matrix
  int tiles_pad_r, tiles_pad_c;  // kEwRows x kEwCols tiles over the padded matrix in its own orientation
  int tiles_upd_r, tiles_upd_c;  // kEwRows x kEwCols tiles over the real matrix
  size_t off_part, off_rrms, off_crms, off_scale;
  // aux and vector plans
  int row_blocks;
  int64_t len;
  size_t off_rscale, off_cscale, off_cpart, off_normsq;
};

// A shape group, or the slice of one that a pass of a workspace-capped plan updates.
struct GroupInfo {
  int64_t s, l, S, L;
  std::vector<int> mats;
  std::vector<int> segs;  // Newton-Schulz schedule: steps per segment (all ones: eq. "ns" as printed)
  size_t off_xa, off_xb, off_a, off_p, off_rpart, off_cpart, off_fold;
  size_t off_p2, off_t, off_q0, off_q1;  // Gram-space segment buffers (only when a segment has >= 2 / 3 steps)
  int64_t stride_x, stride_a, stride_rpart, stride_cpart;  // elements per matrix
};

// Gram matrices A = X X^T and the Gram-space matrices are kept in fp16, whose 11-bit
// significand keeps the S x S iteration more accurate than the printed bf16 step; A and T are
// stored times kGramScale so that their entries (about 1/s on the diagonal of the first A, and
// smaller off it) stay in fp16's normal range.
constexpr float kGramScale = 8192.f;

// Whether fp16 storage is safe for the plan's coefficients.  X_0 = V/||V||_F has singular values
// in [0, 1], and a step maps [0, r] into [0, max |phi| on [0, r]] (phi(x) = a x + b x^3 + c x^5),
// so r_k bounds the singular values of X_k.  Every entry of a symmetric matrix is bounded by its
// largest eigenvalue: A_k by r_k^2, T = P A by max |p(l) l| and P = p(A) by max |p(l)| for
// l in [0, r_k^2] (p(l) = a + b l + c l^2), and a segment's Q by max |p|^3.  The bounds are taken
// over 64 steps (the CV trace's limit) by dense sampling with 2% slack, and fp16 (65504 at most)
// is used when the scaled values stay below 16384.  The paper's coefficients give r <= 1.21:
// A * kGramScale <= 1.21e4, T * kGramScale <= 1.0e4, Q <= 43.
bool gram_fp16_safe(const meq_hparams& hp) {
  const double a = hp.ns_a, b = hp.ns_b, c = hp.ns_c;
  double r = 1.0, ma = 1.0, mt = 0.0, mp = 0.0;
  constexpr int kSamples = 4096;
  for (int k = 0; k < 64; ++k) {
    double phimax = 0.0, tmax = 0.0, pmax = 0.0;
    for (int i = 0; i <= kSamples; ++i) {
      const double x = r * i / kSamples, l = x * x;
      const double pl = a + b * l + c * l * l;
      phimax = std::max(phimax, std::fabs(pl * x));
      tmax = std::max(tmax, std::fabs(pl * l));
      pmax = std::max(pmax, std::fabs(pl));
    }
    r = 1.02 * phimax;
    ma = std::max(ma, r * r);
    mt = std::max(mt, 1.02 * tmax);
    mp = std::max(mp, 1.02 * pmax);
    if (!(r < 1e3)) return false;
  }
  const double lim = 16384.0;
  return kGramScale * ma <= lim && kGramScale * mt <= lim && mp * mp * mp <= lim;
}

// Segments of the K Newton-Schulz steps of one shape group.  A segment of j steps costs, in
// s^3 units with r = L / S (symmetric products counted once): X X^T r, the j polynomials j,
// the 3 (j - 1) products P A, P T, P Q, and Q X 2 r; j single steps cost (3 r + 1) j.  With
// j >= 2 that is cheaper once r > 1; segments are used from r >= 2 on, where they save at
// least a quarter of the flops.
std::vector<int> ns_schedule(int64_t S, int64_t L, int steps, int gram_steps) {
  const int len = (gram_steps >= 2 && L >= 2 * S) ? gram_steps : 1;
  std::vector<int> segs;
  for (int left = steps; left > 0; left -= len) segs.push_back(std::min(len, left));
  return segs;
}

// The Newton-Schulz output of a group sits in buffer b after an odd number of segments
// (each segment ends with one X product that writes the other buffer).
bool u_in_b(const GroupInfo& g) { return g.segs.size() % 2 == 1; }

// One pass of a hidden plan: group slices whose Newton-Schulz buffers share the workspace's
// Newton-Schulz region, and their matrices.  An uncapped plan has one pass holding every shape
// group whole; a capped plan runs its passes one after the other, each reusing the region.
struct Pass {
  std::vector<int> groups;
  std::vector<int> mats;
};

struct TimedLaunch {
  int kind;
  hipEvent_t start, stop;
};

}  // namespace

struct meq_plan {
  int kind = MEQ_PARAM_HIDDEN;
  meq_hparams hp;
  bool gram16 = true;  // fp16 Gram and Gram-space matrices (gram_fp16_safe); else the printed bf16 iteration
  std::vector<MatInfo> mats;
  std::vector<GroupInfo> groups;
  std::vector<Pass> passes;
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
  if (hp.ns_gram_steps < 1 || hp.ns_gram_steps > 3) return MEQ_ERR_INVALID_ARG;
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
    return MEQ_ERR_INTERNAL;
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
  hp->ns_gram_steps = 3;
}

MEQ_EXPORT const char* meq_status_string(meq_status s) {
  switch (s) {
    case MEQ_OK: return "ok";
    case MEQ_ERR_INVALID_ARG: return "invalid argument";
    case MEQ_ERR_UNSUPPORTED: return "unsupported dtype or size";
    case MEQ_ERR_HIP: return "HIP runtime error";
    case MEQ_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case MEQ_ERR_NO_MEMORY: return "host memory allocation failed";
    case MEQ_ERR_INTERNAL: return "internal library error";
  }
  return "unknown status";
}

namespace {

// Bytes of one group slice's Newton-Schulz buffers for c matrices, each region 256-byte aligned:
// the 1/||V|| fold table, two ping-pong X buffers, A and P, the Gram-space buffers its schedule
// needs, and the row/column sum-of-squares partials.  With `g` the offsets are assigned from `base`.
size_t slice_layout(GroupInfo* g, int64_t S, int64_t L, size_t c, int longest, size_t base) {
  const size_t sx = static_cast<size_t>(S * L), sa = static_cast<size_t>(S * S);
  const size_t srp = static_cast<size_t>((L / kTile) * S), scp = static_cast<size_t>((S / kTile) * L);
  size_t off = base;
  auto take = [&](size_t* dst, size_t bytes) {
    if (dst) *dst = off;
    off = align_up(off + bytes, kAlign);
  };
  take(g ? &g->off_fold : nullptr, 8 * c);
  take(g ? &g->off_xa : nullptr, 2 * c * sx);
  take(g ? &g->off_xb : nullptr, 2 * c * sx);
  take(g ? &g->off_a : nullptr, 2 * c * sa);
  take(g ? &g->off_p : nullptr, 2 * c * sa);
  if (g) g->off_p2 = g->off_t = g->off_q0 = g->off_q1 = 0;
  if (longest >= 2) {
    take(g ? &g->off_p2 : nullptr, 2 * c * sa);
    take(g ? &g->off_t : nullptr, 2 * c * sa);
    take(g ? &g->off_q0 : nullptr, 2 * c * sa);
  }
  if (longest >= 3) take(g ? &g->off_q1 : nullptr, 2 * c * sa);
  take(g ? &g->off_rpart : nullptr, 4 * c * srp);
  take(g ? &g->off_cpart : nullptr, 4 * c * scp);
  return off - base;
}

// Hidden 2D weights: shape groups for the Newton-Schulz launches and the workspace layout.  The
// workspace holds the per-matrix scalars and vectors, then one Newton-Schulz region.  Without a
// cap (max_ws == 0) one pass covers every shape group; with one, the groups are cut into slices
// packed greedily into passes whose region fits the cap.
meq_status init_hidden(const meq_matrix_desc* mats, int32_t count, const meq_hparams* hp, size_t max_ws,
                       meq_plan** out) {
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
  p->gram16 = gram_fp16_safe(*hp);
  p->mats.resize(count);
  // shape groups in order of first appearance
  std::map<std::pair<int64_t, int64_t>, int> group_of;
  std::vector<GroupInfo> shapes;
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
      it = group_of.emplace(key, static_cast<int>(shapes.size())).first;
      GroupInfo g{};
      g.s = mi.s;
      g.l = mi.l;
      g.S = mi.S;
      g.L = mi.L;
      g.segs = ns_schedule(g.S, g.L, p->hp.ns_steps, p->gram16 ? p->hp.ns_gram_steps : 1);
      shapes.push_back(g);
    }
    shapes[it->second].mats.push_back(i);
  }
  // persistent part: per-matrix scalars, tile partials of ||V||^2, r, c and the scale vector
  size_t off = 0;
  p->off_scal = off;
  off = align_up(off + sizeof(MatScalars) * static_cast<size_t>(count), kAlign);
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
  const size_t off_ns = off;
  if (max_ws != 0 && off_ns > max_ws) return MEQ_ERR_WORKSPACE;
  const size_t room = max_ws == 0 ? SIZE_MAX : max_ws - off_ns;
  // group slices packed into passes
  size_t used = 0, region = 0;
  p->passes.emplace_back();
  for (const GroupInfo& sg : shapes) {
    const int longest = *std::max_element(sg.segs.begin(), sg.segs.end());
    size_t next = 0;
    while (next < sg.mats.size()) {
      const size_t left = sg.mats.size() - next;
      size_t c = left;
      while (c > 0 && used + slice_layout(nullptr, sg.S, sg.L, c, longest, 0) > room) c = c * 2 / 3;
      while (c < left && used + slice_layout(nullptr, sg.S, sg.L, c + 1, longest, 0) <= room) ++c;
      if (c == 0) {
        if (used == 0) return MEQ_ERR_WORKSPACE;  // not even one matrix of this shape fits
        p->passes.emplace_back();
        used = 0;
        continue;
      }
      GroupInfo g = sg;
      g.mats.assign(sg.mats.begin() + static_cast<std::ptrdiff_t>(next),
                    sg.mats.begin() + static_cast<std::ptrdiff_t>(next + c));
      g.stride_x = g.S * g.L;
      g.stride_a = g.S * g.S;
      g.stride_rpart = (g.L / kTile) * g.S;
      g.stride_cpart = (g.S / kTile) * g.L;
      used += slice_layout(&g, g.S, g.L, c, longest, off_ns + used);
      region = std::max(region, used);
      const int gi = static_cast<int>(p->groups.size());
      for (size_t k = 0; k < g.mats.size(); ++k) {
        MatInfo& mi = p->mats[g.mats[k]];
        mi.group = gi;
        mi.gidx = static_cast<int>(k);
        mi.pass = static_cast<int>(p->passes.size()) - 1;
        p->passes.back().mats.push_back(g.mats[k]);
      }
      p->passes.back().groups.push_back(gi);
      p->groups.push_back(std::move(g));
      next += c;
    }
  }
  if (p->passes.back().groups.empty()) p->passes.pop_back();
  // matrices of a pass in their plan order (the launch chunks follow it)
  for (Pass& ps : p->passes) std::sort(ps.mats.begin(), ps.mats.end());
  p->ws_bytes = off_ns + region;
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

namespace {

meq_status init_any(int32_t kind, const meq_matrix_desc* mats, int32_t count, const meq_hparams* hp, size_t max_ws,
                    meq_plan** out) {
  if (out) *out = nullptr;
  if (!out || !hp || count < 0 || (count > 0 && !mats)) return MEQ_ERR_INVALID_ARG;
  if (kind != MEQ_PARAM_HIDDEN && kind != MEQ_PARAM_AUX && kind != MEQ_PARAM_VECTOR) return MEQ_ERR_INVALID_ARG;
  MEQ_TRY(validate_hparams(*hp));
  if (hp->update_rule != MEQ_RULE_MEQMUON && kind != MEQ_PARAM_HIDDEN) return MEQ_ERR_INVALID_ARG;
  return guarded([&]() -> meq_status {
    if (kind == MEQ_PARAM_HIDDEN) return init_hidden(mats, count, hp, max_ws, out);
    MEQ_TRY(init_stream_kind(kind, mats, count, hp, out));
    if (max_ws != 0 && (*out)->ws_bytes > max_ws) {
      delete *out;
      *out = nullptr;
      return MEQ_ERR_WORKSPACE;
    }
    return MEQ_OK;
  });
}

}  // namespace

MEQ_EXPORT meq_status meq_init_kind(int32_t kind, const meq_matrix_desc* mats, int32_t count, const meq_hparams* hp,
                                    meq_plan** out) {
  return init_any(kind, mats, count, hp, 0, out);
}

MEQ_EXPORT meq_status meq_init_capped(int32_t kind, const meq_matrix_desc* mats, int32_t count,
                                      const meq_hparams* hp, size_t max_workspace_bytes, meq_plan** out) {
  return init_any(kind, mats, count, hp, max_workspace_bytes, out);
}

MEQ_EXPORT meq_status meq_init(const meq_matrix_desc* mats, int32_t count, const meq_hparams* hp, meq_plan** out) {
  return meq_init_kind(MEQ_PARAM_HIDDEN, mats, count, hp, out);
}

MEQ_EXPORT size_t meq_workspace_bytes(const meq_plan* plan) { return plan ? plan->ws_bytes : 0; }

MEQ_EXPORT int32_t meq_plan_num_groups(const meq_plan* plan) {
  return plan ? static_cast<int32_t>(plan->groups.size()) : 0;
}

MEQ_EXPORT int32_t meq_plan_num_passes(const meq_plan* plan) {
  return plan && plan->kind == MEQ_PARAM_HIDDEN ? static_cast<int32_t>(plan->passes.size()) : 0;
}

MEQ_EXPORT meq_status meq_plan_group(const meq_plan* plan, int32_t g, int64_t* s, int64_t* l, int32_t* count) {
  if (!plan || g < 0 || g >= static_cast<int32_t>(plan->groups.size())) return MEQ_ERR_INVALID_ARG;
  const GroupInfo& gi = plan->groups[g];
  if (s) *s = gi.s;
  if (l) *l = gi.l;
  if (count) *count = static_cast<int32_t>(gi.mats.size());
  return MEQ_OK;
}

MEQ_EXPORT meq_status meq_plan_group_schedule(const meq_plan* plan, int32_t g, int32_t* segs, int32_t max_segs,
                                              int32_t* nsegs) {
  if (!plan || g < 0 || g >= static_cast<int32_t>(plan->groups.size()) || max_segs < 0 || (max_segs > 0 && !segs))
    return MEQ_ERR_INVALID_ARG;
  const std::vector<int>& sg = plan->groups[g].segs;
  if (nsegs) *nsegs = static_cast<int32_t>(sg.size());
  for (int32_t i = 0; i < max_segs && i < static_cast<int32_t>(sg.size()); ++i) segs[i] = sg[i];
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
      // X_0 sits in buffer a; each segment's last product writes the other buffer
      const bool in_b = kind == MEQ_BUF_U && u_in_b(g);
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
std::vector<std::vector<int>> dtype_chunks(const meq_plan* p, const std::vector<int>& mats) {
  std::vector<std::vector<int>> chunks;
  for (int dt = 0; dt < 2; ++dt) {
    std::vector<int> cur;
    for (int i : mats) {
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

// Matrices of a pass in chunks of at most kMaxChunk (any dtype).
std::vector<std::vector<int>> plain_chunks(const std::vector<int>& mats) {
  std::vector<std::vector<int>> chunks;
  for (size_t c0 = 0; c0 < mats.size(); c0 += kMaxChunk)
    chunks.emplace_back(mats.begin() + static_cast<std::ptrdiff_t>(c0),
                        mats.begin() + static_cast<std::ptrdiff_t>(std::min(mats.size(), c0 + kMaxChunk)));
  return chunks;
}

// Steps a1-a2: momentum (or, with momenta == nullptr, V = the given inputs), bf16 V in wide
// orientation, ||V||_F^2 and its reciprocals.
meq_status enqueue_prescale(meq_plan* p, const Pass& ps, char* ws, const void* const* grads, float* const* momenta,
                            hipStream_t st) {
  const meq_hparams& hp = p->hp;
  MatScalars* scal = reinterpret_cast<MatScalars*>(ws + p->off_scal);
  const auto chunks = dtype_chunks(p, ps.mats);
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
  for (const auto& ch : plain_chunks(ps.mats)) {
    NormArgs a{};
    a.count = static_cast<int>(ch.size());
    for (int k = 0; k < a.count; ++k) {
      const MatInfo& mi = p->mats[ch[k]];
      a.nparts[k] = mi.tiles_pad_r * mi.tiles_pad_c;
      a.part[k] = reinterpret_cast<const float*>(ws + mi.off_part);
      a.scal[k] = scal + ch[k];
      a.fold[k] = reinterpret_cast<float*>(ws + p->groups[mi.group].off_fold) + 2 * mi.gidx;
    }
    MEQ_TRY(timed_launch(p, MEQ_K_NORM, st, [&] { return launch_norm(a, st); }));
  }
  return MEQ_OK;
}

// Step a3 as chains of products, one chain per shape group.  Four product kinds:
//   OP_GRAM   A <- X X^T                       (symmetric NT kernel, K = L)
//   OP_POLY   P <- a I + b A + c A A           (poly kernel: symmetric NT with the A tile added, K = S)
//   OP_SPROD  C <- P M for M in {A, T, Q}      (symmetric NT kernel, K = S; P and M are commuting
//                                               symmetric matrices, so P M = P M^T is symmetric)
//   OP_APPLY  X' <- P X or Q X                 (NN kernel, K = S)
enum OpKind { OP_GRAM = 0, OP_POLY = 1, OP_SPROD = 2, OP_APPLY = 3 };

struct NsOp {
  int kind;
  size_t a, b, c, e;  // workspace offsets: operands, output, added tile (OP_POLY)
  int scale_kind;     // 2: 1/||V||^2 (first X X^T of a step), 1: 1/||V|| (first X product)
  bool rowcol;        // the step's last X product also writes the row/column sums of squares
  bool with_prev;     // independent of the previous op of the chain (may share its launch)
  bool in_f16, out_f16;                  // operand and output formats (else bf16)
  float alpha_acc, alpha_e, alpha_diag;  // C = alpha_acc * (product) + alpha_e * E + alpha_diag * I
};

// One shape group's products over a schedule.  A segment of j steps is eq. "ns" regrouped:
// A = X X^T once; for each step P_i = a I + b A + c A A, then (before the segment's last
// step) A <- P_i (P_i A), since X P-updated gives (P X)(P X)^T = P A P = P P A; the
// segment's product Q = P_last ... P_first accumulates alongside; finally X <- Q X.  A
// one-step segment is exactly A = X X^T, P, X <- P X.  With gram16, A is fp16 (scaled by
// kGramScale) and a longer segment also keeps T, its P factors and Q in fp16; the matrix that
// feeds the X product (P of a one-step segment, the last Q of a longer one) is bf16, like X.
// Without it (coefficients outside the fp16 range check) every matrix is bf16 and the
// schedule has only one-step segments.  X_0 is in buffer a when x_in_a.
std::vector<NsOp> group_ops(const GroupInfo& g, const std::vector<int>& segs, bool x_in_a, bool first_fold,
                            bool rowcol, const meq_hparams& hp, bool gram16) {
  std::vector<NsOp> ops;
  size_t cur = x_in_a ? g.off_xa : g.off_xb, nxt = x_in_a ? g.off_xb : g.off_xa;
  const size_t pbuf[2] = {g.off_p, g.off_p2}, qbuf[2] = {g.off_q0, g.off_q1};
  for (size_t si = 0; si < segs.size(); ++si) {
    const bool fold = first_fold && si == 0;
    const int len = segs[si];
    const bool f16 = gram16 && len >= 2;  // P factors in fp16 (they feed fp16 products, not the X product)
    const float sc = gram16 ? kGramScale : 1.f;
    ops.push_back({OP_GRAM, cur, cur, g.off_a, 0, fold ? 2 : 0, false, false, false, gram16, sc, 0.f, 0.f});
    size_t q = 0;
    for (int j = 0; j < len; ++j) {
      const size_t pj = pbuf[j % 2];
      // P = a I + (b / sc) A' + (c / sc^2) A' A' for the scaled A' = sc A
      ops.push_back({OP_POLY, g.off_a, g.off_a, pj, g.off_a, 0, false, false, gram16, f16, hp.ns_c / (sc * sc),
                     hp.ns_b / sc, hp.ns_a});
      if (j == 0) {
        q = pj;
      } else {  // Q <- P_j Q (reads the other P buffer or a Q buffer, writes the free Q buffer)
        const size_t qn = qbuf[(j - 1) % 2];
        ops.push_back({OP_SPROD, pj, q, qn, 0, 0, false, false, true, j + 1 < len, 1.f, 0.f, 0.f});
        q = qn;
      }
      if (j + 1 < len) {
        ops.push_back({OP_SPROD, pj, g.off_a, g.off_t, 0, 0, false, j > 0, true, true, 1.f, 0.f, 0.f});  // T <- P_j A
        ops.push_back({OP_SPROD, pj, g.off_t, g.off_a, 0, 0, false, false, true, true, 1.f, 0.f, 0.f});  // A <- P_j T
      }
    }
    ops.push_back({OP_APPLY, q, cur, nxt, 0, fold ? 1 : 0, rowcol && si + 1 == segs.size(), false, false, false,
                   1.f, 0.f, 0.f});
    std::swap(cur, nxt);
  }
  return ops;
}

// Fill one launch entry for op `op` of shape group g.
void fill_gemm_group(GemmGroup& gg, const NsOp& op, const GroupInfo& g, char* ws) {
  auto buf = [&](size_t off) { return reinterpret_cast<uint16_t*>(ws + off); };
  const int tm = static_cast<int>(g.S / kTile), tn = static_cast<int>(g.L / kTile);
  const int S = static_cast<int>(g.S), L = static_cast<int>(g.L);
  gg = GemmGroup{};
  gg.fold = reinterpret_cast<const float*>(ws + g.off_fold);
  gg.scale_kind = op.scale_kind;
  gg.out_f16 = op.out_f16;
  gg.alpha_acc = op.alpha_acc;
  gg.alpha_e = op.alpha_e;
  gg.alpha_diag = op.alpha_diag;
  gg.a = buf(op.a);
  gg.c = buf(op.c);
  if (op.kind == OP_APPLY) {
    gg.lda = S; gg.stride_a = g.stride_a;
    gg.b = buf(op.b); gg.ldb = L; gg.stride_b = g.stride_x;
    gg.ldc = L; gg.stride_c = g.stride_x;
    gg.K = S;
    gg.tiles_m = tm; gg.tiles_n = tn; gg.tiles_per_mat = tm * tn;
    if (op.rowcol) {
      gg.rpart = reinterpret_cast<float*>(ws + g.off_rpart);
      gg.cpart = reinterpret_cast<float*>(ws + g.off_cpart);
      gg.stride_rpart = g.stride_rpart;
      gg.stride_cpart = g.stride_cpart;
    }
  } else {
    const bool gram = op.kind == OP_GRAM;
    gg.lda = gram ? L : S; gg.stride_a = gram ? g.stride_x : g.stride_a;
    gg.b = buf(op.b); gg.ldb = gg.lda; gg.stride_b = gg.stride_a;
    gg.ldc = S; gg.stride_c = g.stride_a;
    if (op.kind == OP_POLY) {
      gg.e = buf(op.e); gg.lde = S; gg.stride_e = g.stride_a;
    }
    gg.K = gram ? L : S;
    gg.symmetrize = op.kind == OP_SPROD;
    gg.tiles_m = tm; gg.tiles_n = tm; gg.tiles_per_mat = tm * (tm + 1) / 2;
  }
  gg.tiles = gg.tiles_per_mat * static_cast<int>(g.mats.size());
}

// Kernel instantiation of an op: template mode (0 symmetric NT, 1 poly, 2 apply) x operand format.
int mode_of(const NsOp& op) { return 2 * (op.kind == OP_POLY ? 1 : op.kind == OP_APPLY ? 2 : 0) + (op.in_f16 ? 1 : 0); }

// A run of a chain's ops that may share one launch: the op and the ops after it marked
// with_prev (same kernel, independent of each other).
struct Bundle {
  int mode;  // kernel instantiation (mode_of): one launch runs one instantiation
  std::vector<std::pair<int, const NsOp*>> ops;  // (shape group, op)
};

std::vector<Bundle> bundles_of(int gi, const std::vector<NsOp>& chain) {
  std::vector<Bundle> out;
  for (const NsOp& op : chain) {
    const int mode = mode_of(op);
    if (op.with_prev && !out.empty() && out.back().mode == mode)
      out.back().ops.push_back({gi, &op});
    else
      out.push_back({mode, {{gi, &op}}});
  }
  return out;
}

// Interleave two launch sequences into a shortest common supersequence over kernel templates:
// each output launch takes the next bundle of either sequence or, when both use the same
// kernel, of both.  Each sequence keeps its order, and different chains are independent, so
// every dependency is respected; equal sequences (groups on the same schedule) merge exactly.
std::vector<Bundle> merge_launches(const std::vector<Bundle>& a, const std::vector<Bundle>& b) {
  const size_t n = a.size(), m = b.size();
  std::vector<std::vector<int>> len(n + 1, std::vector<int>(m + 1, 0));  // SCS length of a[i:], b[j:]
  for (size_t i = n + 1; i-- > 0;)
    for (size_t j = m + 1; j-- > 0;) {
      if (i == n || j == m)
        len[i][j] = static_cast<int>((n - i) + (m - j));
      else if (a[i].mode == b[j].mode)
        len[i][j] = 1 + len[i + 1][j + 1];
      else
        len[i][j] = 1 + std::min(len[i + 1][j], len[i][j + 1]);
    }
  std::vector<Bundle> out;
  size_t i = 0, j = 0;
  while (i < n || j < m) {
    if (i < n && j < m && a[i].mode == b[j].mode) {
      Bundle x = a[i++];
      x.ops.insert(x.ops.end(), b[j].ops.begin(), b[j].ops.end());
      ++j;
      out.push_back(std::move(x));
    } else if (j == m || (i < n && len[i + 1][j] <= len[i][j + 1])) {
      out.push_back(a[i++]);
    } else {
      out.push_back(b[j++]);
    }
  }
  return out;
}

// Enqueue the chains of all groups: the heaviest chain first, the others merged into its launch
// sequence; each launch runs its entries in grouped launches of up to kMaxGemmGroups, longest K
// first so the long tiles start first.
meq_status enqueue_chains(meq_plan* p, char* ws, const std::vector<int>& gids,
                          const std::vector<std::vector<NsOp>>& chains, hipStream_t st) {
  auto chain_work = [&](size_t c) {
    const GroupInfo& g = p->groups[gids[c]];
    double w = 0.0;
    for (const NsOp& op : chains[c]) {
      const double tm = static_cast<double>(g.S / kTile);
      const double tiles = op.kind == OP_APPLY ? tm * static_cast<double>(g.L / kTile) : tm * (tm + 1) / 2;
      w += tiles * static_cast<double>(op.kind == OP_GRAM ? g.L : g.S);
    }
    return w * static_cast<double>(g.mats.size());
  };
  std::vector<int> order(chains.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = static_cast<int>(i);
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return chain_work(x) > chain_work(y); });
  std::vector<Bundle> seq;
  for (int c : order) seq = merge_launches(seq, bundles_of(gids[c], chains[c]));
  for (Bundle& launch : seq) {
    std::stable_sort(launch.ops.begin(), launch.ops.end(), [&](const auto& x, const auto& y) {
      const GroupInfo& gx = p->groups[x.first];
      const GroupInfo& gy = p->groups[y.first];
      return (x.second->kind == OP_GRAM ? gx.L : gx.S) > (y.second->kind == OP_GRAM ? gy.L : gy.S);
    });
    const int mode = launch.mode / 2, f16 = launch.mode % 2;
    const int tk = mode == 0 ? MEQ_K_GRAM : mode == 1 ? MEQ_K_POLY : MEQ_K_APPLY;
    for (size_t c0 = 0; c0 < launch.ops.size(); c0 += kMaxGemmGroups) {
      // The a X term of X <- a X + P X is carried by P: the polynomial product stores
      // a I + b A + c A A, and the X product is the plain product P X.
      GemmArgs ga{};
      ga.count = static_cast<int>(std::min<size_t>(kMaxGemmGroups, launch.ops.size() - c0));
      int start = 0;
      for (int q = 0; q < ga.count; ++q) {
        fill_gemm_group(ga.grp[q], *launch.ops[c0 + q].second, p->groups[launch.ops[c0 + q].first], ws);
        ga.tile_start[q] = start;
        start += (ga.grp[q].tiles + 7) / 8 * 8;
      }
      ga.tile_start[ga.count] = start;
      MEQ_TRY(timed_launch(p, tk, st, [&] { return launch_gemm(ga, mode, f16, st); }));
    }
  }
  return MEQ_OK;
}

// Step a3 of a full step: every group over its own schedule, X_0 in buffer a, the prescale
// folded into the first products; with `rowcol` the last X product also writes the row/column
// sums of squares of its output (step a4's partials).
meq_status enqueue_ns(meq_plan* p, const Pass& ps, char* ws, bool rowcol, hipStream_t st) {
  std::vector<std::vector<NsOp>> chains;
  for (int gi : ps.groups) {
    const GroupInfo& g = p->groups[gi];
    chains.push_back(group_ops(g, g.segs, true, true, rowcol, p->hp, p->gram16));
  }
  return enqueue_chains(p, ws, ps.groups, chains, st);
}

// One step k of eq. "ns" as printed for every group (the CV trace replays the iterates one by
// one): iteration k reads buffer a when k is even.
meq_status enqueue_ns_iteration(meq_plan* p, const Pass& ps, char* ws, int k, hipStream_t st) {
  std::vector<std::vector<NsOp>> chains;
  for (int gi : ps.groups) chains.push_back(group_ops(p->groups[gi], {1}, k % 2 == 0, k == 0, false, p->hp, p->gram16));
  return enqueue_chains(p, ws, ps.groups, chains, st);
}

// Steps a4-a5 on the Newton-Schulz output: row/column RMS, CVs, direction and scale vectors;
// with the Moonlight rule only the uniform scale.  With `sums_done` the row/column sums of
// squares were already written by the last X product.  The output sits where each group's
// schedule left it, or, for the CV trace's replayed iterates, in buffer b when trace_in_b > 0
// and a when it is 0.
meq_status enqueue_stats(meq_plan* p, const Pass& ps, char* ws, bool moonlight, bool sums_done, hipStream_t st,
                         int trace_in_b = -1) {
  const meq_hparams& hp = p->hp;
  MatScalars* scal = reinterpret_cast<MatScalars*>(ws + p->off_scal);
  // 4. row / column sums of squares of U, per shape group (MeqMuon only)
  for (size_t q = 0; q < ps.groups.size() && !moonlight && !sums_done; ++q) {
    const GroupInfo& g = p->groups[ps.groups[q]];
    const int batch = static_cast<int>(g.mats.size());
    const int tm = static_cast<int>(g.S / kTile), tn = static_cast<int>(g.L / kTile);
    uint16_t* xa = reinterpret_cast<uint16_t*>(ws + g.off_xa);
    uint16_t* xb = reinterpret_cast<uint16_t*>(ws + g.off_xb);
    RowColArgs rc{};
    rc.u = (trace_in_b >= 0 ? trace_in_b > 0 : u_in_b(g)) ? xb : xa;
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
  for (const auto& ch : plain_chunks(ps.mats)) {
    SelectArgs a{};
    a.count = static_cast<int>(ch.size());
    a.delta = static_cast<double>(hp.zero_rms_delta);
    for (int k = 0; k < a.count; ++k) {
      const MatInfo& mi = p->mats[ch[k]];
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
      a.scal[k] = scal + ch[k];
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
meq_status enqueue_update(meq_plan* p, const Pass& ps, char* ws, void* const* params, float lr, hipStream_t st) {
  const meq_hparams& hp = p->hp;
  MatScalars* scal = reinterpret_cast<MatScalars*>(ws + p->off_scal);
  const auto chunks = dtype_chunks(p, ps.mats);
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
      const size_t uoff = u_in_b(g) ? g.off_xb : g.off_xa;
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
    for (const Pass& ps : p->passes) {
      MEQ_TRY(enqueue_prescale(p, ps, ws, grads, momenta, st));
      MEQ_TRY(enqueue_ns(p, ps, ws, !moonlight, st));
      MEQ_TRY(enqueue_stats(p, ps, ws, moonlight, !moonlight, st));
      MEQ_TRY(enqueue_update(p, ps, ws, params, lr, st));
    }
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
    for (const Pass& ps : p->passes) {
      MEQ_TRY(enqueue_prescale(p, ps, ws, inputs, nullptr, st));
      for (int k = 0; k <= kmax; ++k) {
        if (k > 0) MEQ_TRY(enqueue_ns_iteration(p, ps, ws, k - 1, st));
        // X_0 (unscaled V: CVs are scale free) sits in buffer a; iteration k - 1 writes b for odd k
        MEQ_TRY(enqueue_stats(p, ps, ws, false, false, st, k % 2 == 1));
        if (hipMemcpyAsync(host.data(), src, sizeof(MatScalars) * count, hipMemcpyDeviceToHost, st) != hipSuccess)
          return MEQ_ERR_HIP;
        if (hipStreamSynchronize(st) != hipSuccess) return MEQ_ERR_HIP;
        for (int i : ps.mats) {
          gamma_r[static_cast<size_t>(i) * (kmax + 1) + k] = host[i].gamma_r;
          gamma_c[static_cast<size_t>(i) * (kmax + 1) + k] = host[i].gamma_c;
        }
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
    (void)hipEventDestroy(tl.start);
    (void)hipEventDestroy(tl.stop);
  }
  for (hipEvent_t e : plan->event_pool) (void)hipEventDestroy(e);
  delete plan;
}
