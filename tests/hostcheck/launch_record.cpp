// Test infrastructure (host only, no GPU): replacements for the kernel launchers of libmeq.so
// that record, for every launch the planner enqueues, the byte range each kernel would read or
// write.  Linked with the planner (meq_api.cpp) into a host-only library, optionally built with
// AddressSanitizer and UndefinedBehaviorSanitizer; the tests then drive meq_step with fake device
// addresses and check every recorded range against the caller's buffers and the workspace.
//
// The ranges follow each kernel's indexing: the GEMM tiles cover tiles_m x tiles_n (or the
// upper block triangle) of 256 x 256 with K in slabs of 64 and no bounds checks; the
// element-wise kernels cover their 64 x 128 tiles; the per-matrix vectors their lengths.
#include <stdint.h>

#include <algorithm>
#include <vector>

#include "meq.h"
#include "meq_internal.h"

#define HC_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

// kBound: an extent that depends on the direction chosen on the device (the scale vector has m
// entries for rows and n for columns); checked against the buffers only.
enum Access { kRead = 0, kWrite = 1, kReadWrite = 2, kBound = 3 };

struct Range {
  int launch;   // sequence number of the launch
  int kernel;   // meq_kernel_kind-like code, see kernel_code below
  int access;
  int item;     // matrix / group index within the launch
  int what;     // operand tag (for messages)
  uint64_t lo, hi;  // [lo, hi) in bytes
};

// Extent records: the rectangle a launch covers in a padded buffer (momentum's bf16 V).
struct Cover {
  int launch, item;
  uint64_t base;
  int64_t rows, cols, ld;  // wide orientation
};

std::vector<Range> g_ranges;
std::vector<Cover> g_covers;
int g_launch = 0;

// operand tags
enum What { W_G = 0, W_B, W_X, W_PART, W_SCAL, W_FOLD, W_A, W_BOP, W_C, W_E, W_RPART, W_CPART, W_U, W_RRMS,
            W_CRMS, W_SCALE, W_W, W_RSCALE, W_CSCALE, W_NORMSQ };

void add(int kernel, int access, int item, int what, const void* p, uint64_t bytes) {
  const uint64_t lo = reinterpret_cast<uintptr_t>(p);
  g_ranges.push_back({g_launch, kernel, access, item, what, lo, lo + bytes});
}

// kernel codes (the timing kinds of meq.h, plus the sub-kernels that share a kind)
enum Code { C_MOMENTUM = 0, C_NORM = 1, C_GEMM_SYM = 2, C_GEMM_POLY = 3, C_GEMM_APPLY = 4, C_ROWCOL = 5,
            C_RMS = 6, C_SELECT = 7, C_UPDATE = 8, C_AUX_ROWS = 9, C_AUX_COLS = 10, C_AUX_COLFIN = 11,
            C_AUX_UPDATE = 12, C_VEC = 13, C_SCALE_FILL = 14 };

}  // namespace

namespace meq {

hipError_t launch_momentum(const MomentumArgs& a, int grad_bf16, int total_tiles, hipStream_t) {
  const uint64_t gsz = grad_bf16 ? 2 : 4;
  if (a.count < 1 || a.count > kMaxChunk || a.tile_start[0] != 0 || a.tile_start[a.count] != total_tiles)
    return hipErrorInvalidValue;
  for (int k = 0; k < a.count; ++k) {
    const uint64_t mn = static_cast<uint64_t>(a.m[k]) * a.n[k];
    add(C_MOMENTUM, kRead, k, W_G, a.g[k], mn * gsz);
    if (a.b[k]) add(C_MOMENTUM, kReadWrite, k, W_B, a.b[k], mn * 4);
    const int tiles = a.tile_start[k + 1] - a.tile_start[k];
    const int tiles_r = tiles / a.tiles_c[k];
    if (tiles_r * a.tiles_c[k] != tiles) return hipErrorInvalidValue;
    // own orientation: tiles_r * 64 rows x tiles_c * 128 columns; the wide buffer holds it transposed
    // for tall matrices
    const int64_t own_r = static_cast<int64_t>(tiles_r) * kEwRows, own_c = static_cast<int64_t>(a.tiles_c[k]) * kEwCols;
    const int64_t wr = a.tall[k] ? own_c : own_r, wc = a.tall[k] ? own_r : own_c;
    add(C_MOMENTUM, kWrite, k, W_X, a.x[k], static_cast<uint64_t>((wr - 1) * a.ldx[k] + wc) * 2);
    g_covers.push_back({g_launch, k, reinterpret_cast<uintptr_t>(a.x[k]), wr, wc, a.ldx[k]});
    add(C_MOMENTUM, kWrite, k, W_PART, a.part[k], static_cast<uint64_t>(tiles) * 4);
  }
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_norm(const NormArgs& a, hipStream_t) {
  for (int k = 0; k < a.count; ++k) {
    add(C_NORM, kRead, k, W_PART, a.part[k], static_cast<uint64_t>(a.nparts[k]) * 4);
    add(C_NORM, kWrite, k, W_SCAL, a.scal[k], sizeof(MatScalars));
    add(C_NORM, kWrite, k, W_FOLD, a.fold[k], 8);
  }
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_gemm(const GemmArgs& a, int mode, int f16, hipStream_t) {
  if (a.count < 1 || a.count > kMaxGemmGroups || a.tile_start[0] != 0) return hipErrorInvalidValue;
  if (mode == 2 && f16) return hipErrorInvalidValue;
  const int code = mode == 0 ? C_GEMM_SYM : mode == 1 ? C_GEMM_POLY : C_GEMM_APPLY;
  for (int q = 0; q < a.count; ++q) {
    const GemmGroup& g = a.grp[q];
    if (g.tiles_per_mat <= 0 || g.tiles % g.tiles_per_mat != 0 || g.K % 256 != 0 || g.K <= 0) return hipErrorInvalidValue;
    if (a.tile_start[q + 1] - a.tile_start[q] < g.tiles || (a.tile_start[q] & 7)) return hipErrorInvalidValue;
    const int64_t batch = g.tiles / g.tiles_per_mat;
    const int64_t M = static_cast<int64_t>(g.tiles_m) * 256, N = static_cast<int64_t>(g.tiles_n) * 256;
    if (mode != 2 && (g.tiles_m != g.tiles_n || g.tiles_per_mat != g.tiles_m * (g.tiles_m + 1) / 2))
      return hipErrorInvalidValue;
    if (mode == 2 && g.tiles_per_mat != g.tiles_m * g.tiles_n) return hipErrorInvalidValue;
    // operand A: rows 0 .. M - 1, k 0 .. K - 1 (row-major, lda)
    add(code, kRead, q, W_A, g.a, static_cast<uint64_t>((batch - 1) * g.stride_a + (M - 1) * g.lda + g.K) * 2);
    if (mode == 2)  // operand B K-major: rows k 0 .. K - 1, columns 0 .. N - 1
      add(code, kRead, q, W_BOP, g.b, static_cast<uint64_t>((batch - 1) * g.stride_b + (g.K - 1) * g.ldb + N) * 2);
    else            // operand B as rows: 0 .. N - 1, k 0 .. K - 1
      add(code, kRead, q, W_BOP, g.b, static_cast<uint64_t>((batch - 1) * g.stride_b + (N - 1) * g.ldb + g.K) * 2);
    if (mode == 1)
      add(code, kRead, q, W_E, g.e, static_cast<uint64_t>((batch - 1) * g.stride_e + (M - 1) * g.lde + M) * 2);
    add(code, kWrite, q, W_C, g.c, static_cast<uint64_t>((batch - 1) * g.stride_c + (M - 1) * g.ldc + N) * 2);
    if (g.scale_kind != 0) add(code, kRead, q, W_FOLD, g.fold, static_cast<uint64_t>(batch) * 8);
    if (g.rpart) {
      add(code, kWrite, q, W_RPART, g.rpart,
          static_cast<uint64_t>((batch - 1) * g.stride_rpart + static_cast<int64_t>(g.tiles_n) * M) * 4);
      add(code, kWrite, q, W_CPART, g.cpart,
          static_cast<uint64_t>((batch - 1) * g.stride_cpart + (g.tiles_m - 1) * static_cast<int64_t>(g.ldc) + N) * 4);
    }
  }
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_rowcol(const RowColArgs& a, int batch, hipStream_t) {
  const int64_t R = static_cast<int64_t>(a.tiles_r) * kTile, C = static_cast<int64_t>(a.tiles_c) * kTile;
  add(C_ROWCOL, kRead, 0, W_U, a.u, static_cast<uint64_t>((batch - 1) * a.stride_u + (R - 1) * a.L + C) * 2);
  add(C_ROWCOL, kWrite, 0, W_RPART, a.rpart,
      static_cast<uint64_t>((batch - 1) * a.stride_rpart + (a.tiles_c - 1) * static_cast<int64_t>(a.S) + R) * 4);
  add(C_ROWCOL, kWrite, 0, W_CPART, a.cpart,
      static_cast<uint64_t>((batch - 1) * a.stride_cpart + (a.tiles_r - 1) * static_cast<int64_t>(a.L) + C) * 4);
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_rms(const SelectArgs& a, hipStream_t) {
  for (int k = 0; k < a.count; ++k) {
    const int s_dim = a.tall[k] ? a.n[k] : a.m[k], l_dim = a.tall[k] ? a.m[k] : a.n[k];
    add(C_RMS, kRead, k, W_RPART, a.rpart[k],
        static_cast<uint64_t>((a.L[k] / kTile - 1) * static_cast<int64_t>(a.S[k]) + s_dim) * 4);
    add(C_RMS, kRead, k, W_CPART, a.cpart[k],
        static_cast<uint64_t>((a.S[k] / kTile - 1) * static_cast<int64_t>(a.L[k]) + l_dim) * 4);
    add(C_RMS, kWrite, k, W_RRMS, a.rrms[k], static_cast<uint64_t>(a.m[k]) * 8);
    add(C_RMS, kWrite, k, W_CRMS, a.crms[k], static_cast<uint64_t>(a.n[k]) * 8);
  }
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_select(const SelectArgs& a, hipStream_t) {
  for (int k = 0; k < a.count; ++k) {
    add(C_SELECT, kRead, k, W_RRMS, a.rrms[k], static_cast<uint64_t>(a.m[k]) * 8);
    add(C_SELECT, kRead, k, W_CRMS, a.crms[k], static_cast<uint64_t>(a.n[k]) * 8);
    add(C_SELECT, kWrite, k, W_SCALE, a.scale[k], static_cast<uint64_t>(a.m[k]) * 4);  // row direction
    add(C_SELECT, kBound, k, W_SCALE, a.scale[k], static_cast<uint64_t>(std::max(a.m[k], a.n[k])) * 4);
    add(C_SELECT, kWrite, k, W_SCAL, a.scal[k], sizeof(MatScalars));
  }
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_scale_fill(const SelectArgs& a, hipStream_t) {
  for (int k = 0; k < a.count; ++k) {
    add(C_SCALE_FILL, kWrite, k, W_SCALE, a.scale[k], static_cast<uint64_t>(a.m[k]) * 4);
    add(C_SCALE_FILL, kWrite, k, W_SCAL, a.scal[k], sizeof(MatScalars));
  }
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_update(const UpdateArgs& a, int param_bf16, int total_tiles, hipStream_t) {
  const uint64_t psz = param_bf16 ? 2 : 4;
  if (a.count < 1 || a.count > kMaxChunk || a.tile_start[0] != 0 || a.tile_start[a.count] != total_tiles)
    return hipErrorInvalidValue;
  for (int k = 0; k < a.count; ++k) {
    const int64_t m = a.m[k], n = a.n[k];
    const int tiles = a.tile_start[k + 1] - a.tile_start[k];
    const int tiles_r = tiles / a.tiles_c[k];
    if (tiles_r * a.tiles_c[k] != tiles) return hipErrorInvalidValue;
    add(C_UPDATE, kReadWrite, k, W_W, a.w[k], static_cast<uint64_t>(m * n) * psz);
    // U in wide orientation: wide matrices read rows < m, columns < n; tall ones read whole 64 x 128
    // tiles transposed (own rows -> wide columns, own columns -> wide rows) from the padded buffer
    const int64_t own_r = static_cast<int64_t>(tiles_r) * kEwRows, own_c = static_cast<int64_t>(a.tiles_c[k]) * kEwCols;
    const uint64_t ub = a.tall[k] ? static_cast<uint64_t>((own_c - 1) * a.ldu[k] + own_r) * 2
                                  : static_cast<uint64_t>((m - 1) * a.ldu[k] + n) * 2;
    add(C_UPDATE, kRead, k, W_U, a.u[k], ub);
    add(C_UPDATE, kRead, k, W_SCALE, a.scale[k], static_cast<uint64_t>(m) * 4);  // row direction
    add(C_UPDATE, kBound, k, W_SCALE, a.scale[k], static_cast<uint64_t>(std::max(m, n)) * 4);
    add(C_UPDATE, kRead, k, W_SCAL, a.scal[k], sizeof(MatScalars));
  }
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_aux_rows(const AuxArgs& a, int grad_bf16, hipStream_t) {
  const uint64_t mn = static_cast<uint64_t>(a.m) * a.n;
  add(C_AUX_ROWS, kRead, 0, W_G, a.g, mn * (grad_bf16 ? 2 : 4));
  add(C_AUX_ROWS, kReadWrite, 0, W_B, a.b, mn * 4);
  add(C_AUX_ROWS, kWrite, 0, W_RRMS, a.rrms, static_cast<uint64_t>(a.m) * 8);
  add(C_AUX_ROWS, kWrite, 0, W_RSCALE, a.rscale, static_cast<uint64_t>(a.m) * 4);
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_aux_cols(const AuxArgs& a, int grad_bf16, hipStream_t) {
  const uint64_t mn = static_cast<uint64_t>(a.m) * a.n;
  add(C_AUX_COLS, kRead, 0, W_B, a.b, mn * 4);
  if (a.nesterov) add(C_AUX_COLS, kRead, 0, W_G, a.g, mn * (grad_bf16 ? 2 : 4));
  add(C_AUX_COLS, kRead, 0, W_RSCALE, a.rscale, static_cast<uint64_t>(a.m) * 4);
  add(C_AUX_COLS, kWrite, 0, W_CPART, a.cpart, static_cast<uint64_t>(a.row_blocks) * a.n * 8);
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_aux_colfin(const AuxArgs& a, hipStream_t) {
  add(C_AUX_COLFIN, kRead, 0, W_CPART, a.cpart, static_cast<uint64_t>(a.row_blocks) * a.n * 8);
  add(C_AUX_COLFIN, kWrite, 0, W_CRMS, a.crms, static_cast<uint64_t>(a.n) * 8);
  add(C_AUX_COLFIN, kWrite, 0, W_CSCALE, a.cscale, static_cast<uint64_t>(a.n) * 4);
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_aux_update(const AuxArgs& a, int bf16, hipStream_t) {
  const uint64_t mn = static_cast<uint64_t>(a.m) * a.n, esz = bf16 ? 2 : 4;
  add(C_AUX_UPDATE, kRead, 0, W_B, a.b, mn * 4);
  if (a.nesterov) add(C_AUX_UPDATE, kRead, 0, W_G, a.g, mn * esz);
  add(C_AUX_UPDATE, kReadWrite, 0, W_W, a.w, mn * esz);
  add(C_AUX_UPDATE, kRead, 0, W_RSCALE, a.rscale, static_cast<uint64_t>(a.m) * 4);
  add(C_AUX_UPDATE, kRead, 0, W_CSCALE, a.cscale, static_cast<uint64_t>(a.n) * 4);
  ++g_launch;
  return hipSuccess;
}

hipError_t launch_vec(const VecArgs& a, int bf16, hipStream_t) {
  const uint64_t esz = bf16 ? 2 : 4;
  for (int k = 0; k < a.count; ++k) {
    const uint64_t len = static_cast<uint64_t>(a.len[k]);
    add(C_VEC, kRead, k, W_G, a.g[k], len * esz);
    add(C_VEC, kReadWrite, k, W_B, a.b[k], len * 4);
    add(C_VEC, kReadWrite, k, W_W, a.w[k], len * esz);
    add(C_VEC, kWrite, k, W_NORMSQ, a.normsq[k], 8);
  }
  ++g_launch;
  return hipSuccess;
}

}  // namespace meq

// The no-allocation step: the library's version takes its workspace from a device array; here the
// array is a fake address range past the other fake buffers, checked like any workspace.
constexpr uintptr_t kFakeScratch = uintptr_t{5} << 44;

HC_EXPORT meq_status meq_step_static(meq_plan* plan, void* const* params, const void* const* grads,
                                     float* const* momenta, float lr, hipStream_t stream) {
  if (!plan) return MEQ_ERR_INVALID_ARG;
  const size_t need = meq_workspace_bytes(plan);
  if (need > MEQ_STATIC_SCRATCH_BYTES) return MEQ_ERR_WORKSPACE;
  if (need == 0) return meq_step(plan, params, grads, momenta, lr, nullptr, 0, stream);
  return meq_step(plan, params, grads, momenta, lr, reinterpret_cast<void*>(kFakeScratch), MEQ_STATIC_SCRATCH_BYTES,
                  stream);
}

// ------------------------------------------------------------------ queries for the tests
HC_EXPORT void meq_hc_clear(void) {
  g_ranges.clear();
  g_covers.clear();
  g_launch = 0;
}

HC_EXPORT int32_t meq_hc_num_ranges(void) { return static_cast<int32_t>(g_ranges.size()); }
HC_EXPORT int32_t meq_hc_num_launches(void) { return g_launch; }

// Range i: launch, kernel code, access (0 read, 1 write, 2 read-write, 3 bound only), item, operand
// tag, [lo, hi).
HC_EXPORT int32_t meq_hc_range(int32_t i, int32_t* out5, uint64_t* lo, uint64_t* hi) {
  if (i < 0 || i >= static_cast<int32_t>(g_ranges.size())) return -1;
  const Range& r = g_ranges[i];
  out5[0] = r.launch;
  out5[1] = r.kernel;
  out5[2] = r.access;
  out5[3] = r.item;
  out5[4] = r.what;
  *lo = r.lo;
  *hi = r.hi;
  return 0;
}

HC_EXPORT int32_t meq_hc_num_covers(void) { return static_cast<int32_t>(g_covers.size()); }

// Cover i: launch, item, base address and the written rectangle (rows x cols, leading dimension).
HC_EXPORT int32_t meq_hc_cover(int32_t i, int32_t* launch_item, uint64_t* base, int64_t* rows_cols_ld) {
  if (i < 0 || i >= static_cast<int32_t>(g_covers.size())) return -1;
  const Cover& c = g_covers[i];
  launch_item[0] = c.launch;
  launch_item[1] = c.item;
  *base = c.base;
  rows_cols_ld[0] = c.rows;
  rows_cols_ld[1] = c.cols;
  rows_cols_ld[2] = c.ld;
  return 0;
}
