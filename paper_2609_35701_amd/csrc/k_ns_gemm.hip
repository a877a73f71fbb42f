// Newton-Schulz products on bf16 MFMA (gfx950), eq. "ns":
//   A_k = X_k X_k^T                (NT, symmetric output: upper tiles + mirrored store)
//   P_k = b A_k + c A_k A_k        (NT since A_k is symmetric; symmetric output)
//   X_{k+1} = a X_k + P_k X_k      (NN: X_k is read K-major and transposed in registers)
// X_0 = V / ||V||_F is folded in: the bf16 buffer holds V, the k = 0 Gram epilogue
// scales by 1/||V||^2 and the k = 0 apply epilogue by 1/||V||.
//
// One workgroup = 4 waves = one 256 x 256 output tile; each wave owns a 128 x 128
// quadrant as 4 x 4 blocks of v_mfma_f32_32x32x16_bf16 (fp32 accumulation).  K
// advances in slabs of 64 through double-buffered LDS (one barrier per slab);
// the next slab's global loads are in flight while the current slab's MFMAs run.
// A batch of same-shape matrices is one launch; workgroup ids are remapped so
// consecutive tiles of one matrix run on one XCD (shared L2).
#include "meq_internal.h"

namespace meq {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int BM = kTile, BN = kTile, BK = 64;
constexpr int PK = BK + 8;  // LDS row pitch (elements): 144 B rows keep 16-byte fragment reads conflict-free
constexpr int kOperandElems = BM * PK;
// Buffer resource word 3 for raw (untyped, 32-bit format) buffer access on gfx9.
constexpr int kBufferFlags = 0x00020000;

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Component q (a compile-time constant after unrolling) of a 4-dword vector.
__device__ __forceinline__ uint32_t dword(const u32x4& v, int q) { return v[q]; }

// Map a launch-order workgroup id to a logical tile so that the workgroups one
// XCD receives (ids x, x + 8, x + 16, ... are dispatched round-robin over the 8
// XCDs) form one contiguous run of logical tiles.
__device__ __forceinline__ int xcd_remap(int w, int nblk) {
  const int q = nblk >> 3, r = nblk & 7;
  const int x = w & 7, pos = w >> 3;
  return x * q + min(x, r) + pos;
}

// kMode: 0 Gram (NT, symmetric, no epilogue input), 1 polynomial (NT, symmetric,
// epilogue reads A), 2 apply (NN, epilogue reads X).
template <int kMode>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_ns_gemm(GemmArgs g) {
  constexpr bool kNN = kMode == 2;
  constexpr bool kSym = kMode != 2;
  constexpr bool kHasE = kMode != 0;
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][kOperandElems];

  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int mat = logical / g.tiles_per_mat;
  int tile = logical - mat * g.tiles_per_mat;
  int ti, tj;
  if (kSym) {
    ti = 0;
    int rowlen = g.tiles_m;
    while (tile >= rowlen) {
      tile -= rowlen;
      ++ti;
      --rowlen;
    }
    tj = ti + tile;
  } else {
    constexpr int kGroup = 8;  // tile rows per group: tiles sharing a column panel run close in time
    const int per = kGroup * g.tiles_n;
    const int gid = tile / per;
    const int first = gid * kGroup;
    const int gm = min(g.tiles_m - first, kGroup);
    const int in = tile - gid * per;
    ti = first + in % gm;
    tj = in / gm;
  }

  // Operands are read with buffer loads: a scalar resource per matrix plus a
  // 32-bit per-lane byte offset (each matrix buffer stays below 2^31 bytes).
  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(g.a + mat * g.stride_a), 0, 0x7fffffff, kBufferFlags);
  const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(g.b + mat * g.stride_b), 0, 0x7fffffff, kBufferFlags);
  const int lda = static_cast<int>(g.lda), ldb = static_cast<int>(g.ldb);

  u32x4 ra[8], rb[8];
  // NT operand slab: thread t loads rows t/8 + 32 i at k-chunk 8 (t % 8).
  // NN operand slab (K x N): lane loads k rows 8 kb .. 8 kb + 7 at n-chunk nb.
  const int kb = lane & 7, nb = (lane >> 3) + 8 * wave;
  const int va = 2 * ((ti * BM + (t >> 3)) * lda + (t & 7) * 8);
  const int vb = kNN ? 2 * ((kb * 8) * ldb + tj * BN + nb * 8) : 2 * ((tj * BN + (t >> 3)) * ldb + (t & 7) * 8);

  auto load = [&](int kt) {
    const int k0 = kt * BK;
#pragma unroll
    for (int i = 0; i < 8; ++i) ra[i] = __builtin_amdgcn_raw_buffer_load_b128(rA, va, 2 * (32 * i * lda + k0), 0);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      rb[i] = __builtin_amdgcn_raw_buffer_load_b128(rB, vb, kNN ? 2 * ((k0 + i) * ldb) : 2 * (32 * i * ldb + k0), 0);
  };

  auto store = [&](int buf) {
    uint16_t* As = lds[buf][0];
    uint16_t* Bs = lds[buf][1];
#pragma unroll
    for (int i = 0; i < 8; ++i)
      *reinterpret_cast<u32x4*>(As + ((t >> 3) + 32 * i) * PK + (t & 7) * 8) = ra[i];
    if (kNN) {
      // 8 x 8 transpose of 16-bit elements: out[c] = column c of the 8 loaded rows.
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
        const int q = c >> 1;
        u32x4 o;
        o.x = __builtin_amdgcn_perm(dword(rb[1], q), dword(rb[0], q), sel);
        o.y = __builtin_amdgcn_perm(dword(rb[3], q), dword(rb[2], q), sel);
        o.z = __builtin_amdgcn_perm(dword(rb[5], q), dword(rb[4], q), sel);
        o.w = __builtin_amdgcn_perm(dword(rb[7], q), dword(rb[6], q), sel);
        *reinterpret_cast<u32x4*>(Bs + (nb * 8 + c) * PK + kb * 8) = o;
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        *reinterpret_cast<u32x4*>(Bs + ((t >> 3) + 32 * i) * PK + (t & 7) * 8) = rb[i];
    }
  };

  floatx16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // MFMAs of one 16-deep k step use fragments loaded one step earlier, so LDS
  // latency hides behind the 16 MFMAs of the previous step.
  auto compute = [&](int buf) {
    const uint16_t* As = lds[buf][0] + (wm * 128 + (lane & 31)) * PK + (lane >> 5) * 8;
    const uint16_t* Bs = lds[buf][1] + (wn * 128 + (lane & 31)) * PK + (lane >> 5) * 8;
    bf16x8 af[2][4], bf[2][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[0][i] = *reinterpret_cast<const bf16x8*>(As + i * 32 * PK);
#pragma unroll
    for (int j = 0; j < 4; ++j) bf[0][j] = *reinterpret_cast<const bf16x8*>(Bs + j * 32 * PK);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int cur = kk & 1;
      if (kk + 1 < BK / 16) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          af[cur ^ 1][i] = *reinterpret_cast<const bf16x8*>(As + i * 32 * PK + (kk + 1) * 16);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          bf[cur ^ 1][j] = *reinterpret_cast<const bf16x8*>(Bs + j * 32 * PK + (kk + 1) * 16);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bf[cur][j], acc[i][j], 0, 0, 0);
    }
  };

  const int nk = g.K / BK;
  load(0);
  store(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load(kt + 1);
    compute(cur);
    if (kt + 1 < nk) store(cur ^ 1);
    __syncthreads();
  }

  // Epilogue: C = s * (alpha_e * E + alpha_acc * acc), bf16 round-to-nearest-even.
  float s = 1.f;
  if (g.scale_kind != 0) s = g.fold[2 * mat + (g.scale_kind - 1)];
  const float ae = g.alpha_e * s, aa = g.alpha_acc * s;
  uint16_t* __restrict__ C = g.c + mat * g.stride_c;
  const uint16_t* __restrict__ E = kHasE ? g.e + mat * g.stride_e : nullptr;
  const bool mirror = kSym && ti != tj;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = tj * BN + wn * 128 + j * 32 + (lane & 31);
#pragma unroll
      for (int vb = 0; vb < 4; ++vb) {
        const int row0 = ti * BM + wm * 128 + i * 32 + vb * 8 + (lane >> 5) * 4;
        uint16_t h[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = row0 + v;
          float val = aa * acc[i][j][vb * 4 + v];
          if (kHasE) val = fmaf(ae, bf16_to_f32(E[static_cast<int64_t>(row) * g.lde + col]), val);
          h[v] = f32_to_bf16(val);
          C[static_cast<int64_t>(row) * g.ldc + col] = h[v];
        }
        if (mirror) {
          u32x2 pk;
          pk.x = h[0] | (static_cast<uint32_t>(h[1]) << 16);
          pk.y = h[2] | (static_cast<uint32_t>(h[3]) << 16);
          *reinterpret_cast<u32x2*>(C + static_cast<int64_t>(col) * g.ldc + row0) = pk;
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, int mode, hipStream_t st) {
  const int blocks = a.tiles_per_mat * a.batch;
  switch (mode) {
    case 0: hipLaunchKernelGGL(k_ns_gemm<0>, dim3(blocks), dim3(256), 0, st, a); break;
    case 1: hipLaunchKernelGGL(k_ns_gemm<1>, dim3(blocks), dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL(k_ns_gemm<2>, dim3(blocks), dim3(256), 0, st, a); break;
  }
  return hipGetLastError();
}

}  // namespace meq
