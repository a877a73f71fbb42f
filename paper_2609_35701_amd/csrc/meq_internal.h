// Internal definitions shared by the host planner and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace meq {

// Every Newton-Schulz buffer is padded to multiples of this tile on both sides,
// so the GEMM kernels never need bounds checks.  Zero padding is exact for the
// iteration: zero rows/columns of X stay zero through X X^T, A A and P X.
constexpr int kTile = 256;
// The momentum and write-back kernels work on kEwRows x kEwCols tiles of the matrix's own
// orientation; each thread owns 8 consecutive columns of 4 rows.
constexpr int kEwRows = 64;
constexpr int kEwCols = 128;
// Matrices per launch of the multi-matrix element-wise kernels.  Their per-matrix pointers and
// sizes travel as kernel arguments: at most about 10 KB per launch at this count (ROCm passes
// argument blocks well beyond the traditional 4 KB; 32 KB was checked on gfx950), so the 1B
// step's 112 matrices take one launch per stage and no launch ends in a partial wave per chunk.
constexpr int kMaxChunk = 128;

// Per-matrix scalars kept at the start of the workspace.
struct MatScalars {
  double normsq;   // ||V||_F^2
  double gamma_r;  // CV of row RMS of U
  double gamma_c;  // CV of column RMS of U
  float inv_norm;  // 1 / ||V||_F  (0 for a zero matrix)
  float inv_normsq;
  int32_t dir;     // 0 row, 1 column
  int32_t pad;
};
static_assert(sizeof(MatScalars) == 40, "layout");

// ----------------------------------------------------------------- momentum + bf16 V
struct MomentumArgs {
  int count;
  int nesterov;
  float mu;
  int tile_start[kMaxChunk + 1];  // prefix sum of tiles over the padded matrix
  int m[kMaxChunk], n[kMaxChunk];
  int tiles_c[kMaxChunk];         // tile columns of the padded matrix (own orientation)
  int tall[kMaxChunk];
  int vec[kMaxChunk];             // n % 8 == 0 and aligned pointers: 8-element vector access
  int64_t ldx[kMaxChunk];         // leading dimension of the wide bf16 buffer (padded long side)
  const void* g[kMaxChunk];
  float* b[kMaxChunk];
  uint16_t* x[kMaxChunk];         // wide bf16 V, padded
  float* part[kMaxChunk];         // one sum of squares per tile
};

// --------------------------------------------------------------------- norm finalize
struct NormArgs {
  int count;
  int nparts[kMaxChunk];
  const float* part[kMaxChunk];
  MatScalars* scal[kMaxChunk];
  float* fold[kMaxChunk];  // (1/||V||, 1/||V||^2) at the matrix's slot of its shape group
};

// ------------------------------------------------------------------------ NS GEMMs
// C = s * (alpha_e * E + alpha_acc * (Aop . Bop) + alpha_diag * I) stored as bf16 or fp16, batched over
// the matrices of a shape group; one launch covers up to kMaxGemmGroups groups.  The operands
// (and E) are bf16 or, for the Gram-space products, fp16 (one format per launch).  Aop is
// M x K row-major.  Bop is N x K row-major (NT) or K x N row-major (NN).  For the
// symmetric products only tiles on or above the diagonal are computed and each
// off-diagonal tile is also stored mirrored: Aop . Bop^T must be symmetric (X X^T, or
// the product of two commuting symmetric matrices, where Bop^T = Bop).
constexpr int kMaxGemmGroups = 8;

struct GemmGroup {
  const uint16_t* a;
  const uint16_t* b;
  uint16_t* c;
  const uint16_t* e;   // null when alpha_e == 0
  const float* fold;   // per batch member: (1/||V||, 1/||V||^2)
  int64_t stride_a, stride_b, stride_c, stride_e;  // elements per matrix
  int lda, ldb, ldc, lde;
  int K;
  int tiles_m, tiles_n, tiles_per_mat;
  int tiles;           // batch * tiles_per_mat
  int scale_kind;      // 0 none, 1 scale by 1/||V||, 2 scale by 1/||V||^2 (first products of a step)
  int symmetrize;      // symmetric products of two different factors: make diagonal tiles exactly symmetric
  int out_f16;         // store C as fp16 (Gram-space matrices) instead of bf16
  float alpha_e, alpha_acc, alpha_diag;  // alpha_diag: symmetric products only
  // apply product only, when not null: sums of squares of the bf16 output per row of each
  // 256-column tile (rpart, (L/256) x S per matrix) and per column of each 256-row tile
  // (cpart, (S/256) x L per matrix), the partials of eq. "row-col-rms" for the last iteration
  float* rpart;
  float* cpart;
  int64_t stride_rpart, stride_cpart;
};

struct GemmArgs {
  int count;                             // groups in this launch
  int tile_start[kMaxGemmGroups + 1];    // workgroup ranges per group, multiples of 8
  GemmGroup grp[kMaxGemmGroups];
};

// ----------------------------------------------------------------- row/col sums of U
struct RowColArgs {
  const uint16_t* u;  // group base, wide, S x L per matrix
  int64_t stride_u;
  int S, L;
  float* rpart;  // per matrix: (L/256) x S
  int64_t stride_rpart;
  float* cpart;  // per matrix: (S/256) x L
  int64_t stride_cpart;
  int tiles_r, tiles_c;
};

// ------------------------------------------------------------------ CV + direction
// Also used by the row/column RMS finalization (one launch per chunk of matrices).
struct SelectArgs {
  int count;
  double delta;
  int max_lines;  // max over the chunk of s + l (wide rows + wide columns)
  int m[kMaxChunk], n[kMaxChunk], tall[kMaxChunk], S[kMaxChunk], L[kMaxChunk];
  const float* rpart[kMaxChunk];
  const float* cpart[kMaxChunk];
  double* rrms[kMaxChunk];
  double* crms[kMaxChunk];
  float* scale[kMaxChunk];
  MatScalars* scal[kMaxChunk];
};

// ------------------------------------------------------------------------ write-back
struct UpdateArgs {
  int count;
  float decay;  // 1 - lr * lambda
  float step;   // rho * lr
  int tile_start[kMaxChunk + 1];
  int m[kMaxChunk], n[kMaxChunk], tiles_c[kMaxChunk], tall[kMaxChunk];
  int vec[kMaxChunk];  // n % 8 == 0 and an aligned parameter pointer
  int64_t ldu[kMaxChunk];
  void* w[kMaxChunk];
  const uint16_t* u[kMaxChunk];
  const float* scale[kMaxChunk];
  const MatScalars* scal[kMaxChunk];
};

// ------------------------------------------- remaining 2D parameters (eq. "aux"), one matrix per launch
constexpr int kAuxRowsPerBlock = 4;  // row pass and write-back: one wave per row
constexpr int kAuxColRows = 128;     // rows summed by one block of the column pass
struct AuxArgs {
  int m, n;
  int nesterov;
  int vec;         // n % 4 == 0: rows start 16-byte aligned (fp32) / 8-byte aligned (bf16)
  int row_blocks;  // ceil(m / kAuxColRows)
  float mu, decay, step;
  double delta;
  const void* g;
  float* b;
  void* w;
  double* rrms;    // r of V, m entries
  double* crms;    // c of N_r(V), n entries
  float* rscale;   // 1 / r (0 at or below delta)
  float* cscale;   // 1 / c (0 at or below delta)
  double* cpart;   // row_blocks x n partial column sums of (V_ij / r_i)^2
};

// ------------------------------------------------------- 1-D parameters (eq. "vector")
struct VecArgs {
  int count;
  int nesterov;
  float mu, decay, step;
  int64_t len[kMaxChunk];
  int vec[kMaxChunk];  // length and pointers allow 4-element vector access
  const void* g[kMaxChunk];
  float* b[kMaxChunk];
  void* w[kMaxChunk];
  double* normsq[kMaxChunk];
};

// Launchers (defined in the .hip files).  Each returns the hipError_t of the launch.
hipError_t launch_momentum(const MomentumArgs& a, int grad_bf16, int total_tiles, hipStream_t st);
hipError_t launch_norm(const NormArgs& a, hipStream_t st);
// mode 0 symmetric NT, 1 poly, 2 apply; f16: fp16 operands (modes 0 and 1)
hipError_t launch_gemm(const GemmArgs& a, int mode, int f16, hipStream_t st);
hipError_t launch_rowcol(const RowColArgs& a, int batch, hipStream_t st);
hipError_t launch_rms(const SelectArgs& a, hipStream_t st);
hipError_t launch_select(const SelectArgs& a, hipStream_t st);
hipError_t launch_update(const UpdateArgs& a, int param_bf16, int total_tiles, hipStream_t st);
hipError_t launch_scale_fill(const SelectArgs& a, hipStream_t st);  // Moonlight: scale sqrt(max(m, n)), rows
hipError_t launch_aux_rows(const AuxArgs& a, int grad_bf16, hipStream_t st);
hipError_t launch_aux_cols(const AuxArgs& a, int grad_bf16, hipStream_t st);
hipError_t launch_aux_colfin(const AuxArgs& a, hipStream_t st);
hipError_t launch_aux_update(const AuxArgs& a, int bf16, hipStream_t st);
hipError_t launch_vec(const VecArgs& a, int bf16, hipStream_t st);

}  // namespace meq
