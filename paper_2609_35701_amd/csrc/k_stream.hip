// Streaming kernels of the MeqMuon hidden-weight update (HBM-bound stages):
//   momentum + Frobenius partials + bf16 V in wide orientation   eq. "momentum", eq. "ns" (X_0)
//   ||V||_F^2 finalization                                         eq. "ns" (X_0 = H / ||H||_F)
//   row / column sums of squares of U                              eq. "row-col-rms"
//   CVs, direction and scale vector                                 eqs. "cv", "operators", "hidden"
//   decoupled weight decay + normalized update                      eq. "meqmuon-update"
// All reductions are fixed-order trees (no floating-point atomics), so results
// are bitwise reproducible run to run.
#include "meq_internal.h"

namespace meq {

namespace {

typedef uint32_t nt_u32x4 __attribute__((ext_vector_type(4)));
typedef float nt_f32x4 __attribute__((ext_vector_type(4)));
// Loads and stores marked non-temporal: the write-back reads U and W and writes W once per
// step (measured: 6% faster write-back), the momentum step reads G and writes V once (1% and 2%
// faster once its loads were hoisted; on B the hint changed nothing).
__device__ __forceinline__ uint4 ld_nt(const uint4* p) {
  const nt_u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const nt_u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float4 ld_nt(const float4* p) {
  const nt_f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const nt_f32x4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st_nt(uint4 v, uint4* p) {
  __builtin_nontemporal_store(nt_u32x4{v.x, v.y, v.z, v.w}, reinterpret_cast<nt_u32x4*>(p));
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(static_cast<uint32_t>(h) << 16); }

// float -> bfloat16, round to nearest, ties to even; NaN stays NaN (quieted).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Sum over a 256-thread block in a fixed order; every thread gets the result.
template <typename T>
__device__ __forceinline__ T block_sum256(T v, T* red /* >= 4 entries */) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  T r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

// The matrix whose tile range [tile_start[mi], tile_start[mi + 1]) holds block bid (binary
// search over the launch's prefix sums; tile_start[0] = 0 <= bid).
__device__ __forceinline__ int find_matrix(const int* tile_start, int count, int bid) {
  int lo = 0, hi = count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (bid >= tile_start[mid]) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Eight consecutive floats of a bf16 or fp32 array (16- or 32-byte access).
template <bool kBf16, bool kNT = false>
__device__ __forceinline__ void load8(const void* p, int64_t i, float (&x)[8]) {
  if (kBf16) {
    const uint4* q = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p) + i);
    const uint4 v = kNT ? ld_nt(q) : *q;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      x[2 * q] = bf16_to_f32(w[q] & 0xffffu);
      x[2 * q + 1] = bf16_to_f32(w[q] >> 16);
    }
  } else {
    const float4* q = reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
    const float4 lo = kNT ? ld_nt(q) : q[0];
    const float4 hi = kNT ? ld_nt(q + 1) : q[1];
    x[0] = lo.x; x[1] = lo.y; x[2] = lo.z; x[3] = lo.w;
    x[4] = hi.x; x[5] = hi.y; x[6] = hi.z; x[7] = hi.w;
  }
}

// Eight consecutive values as loaded (16 bytes of bf16 or 32 of fp32), unpacked to floats only
// when used, so that loads in flight hold half the registers for bf16 data.
template <bool kBf16> struct Raw8;
template <> struct Raw8<true> { uint4 v; };
template <> struct Raw8<false> { float4 lo, hi; };
template <bool kBf16, bool kNT = false>
__device__ __forceinline__ void load_raw8(const void* p, int64_t i, Raw8<kBf16>& r) {
  if constexpr (kBf16) {
    const uint4* q = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p) + i);
    r.v = kNT ? ld_nt(q) : *q;
  } else {
    const float4* q = reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
    r.lo = kNT ? ld_nt(q) : q[0];
    r.hi = kNT ? ld_nt(q + 1) : q[1];
  }
}
template <bool kBf16>
__device__ __forceinline__ void unpack8(const Raw8<kBf16>& r, float (&x)[8]) {
  if constexpr (kBf16) {
    const uint32_t w[4] = {r.v.x, r.v.y, r.v.z, r.v.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      x[2 * q] = bf16_to_f32(w[q] & 0xffffu);
      x[2 * q + 1] = bf16_to_f32(w[q] >> 16);
    }
  } else {
    x[0] = r.lo.x; x[1] = r.lo.y; x[2] = r.lo.z; x[3] = r.lo.w;
    x[4] = r.hi.x; x[5] = r.hi.y; x[6] = r.hi.z; x[7] = r.hi.w;
  }
}

__device__ __forceinline__ uint4 pack_bf16x8(const uint16_t (&h)[8]) {
  uint4 v;
  v.x = h[0] | (static_cast<uint32_t>(h[1]) << 16);
  v.y = h[2] | (static_cast<uint32_t>(h[3]) << 16);
  v.z = h[4] | (static_cast<uint32_t>(h[5]) << 16);
  v.w = h[6] | (static_cast<uint32_t>(h[7]) << 16);
  return v;
}

// --------------------------------------------------------------------------------
// Momentum B <- mu B + G, V = B (or G + mu B), per-tile sum of V^2, bf16 V written
// into the zero-padded wide buffer (transposed through LDS for tall matrices).
// Without a momentum buffer (b == nullptr) V is the input G itself.
// One block = one 64 x 128 tile of the padded matrix in its own orientation;
// thread (ty, tx) owns columns 8 tx .. 8 tx + 7 of rows ty + 16 k (wide) or of the four
// consecutive rows 4 ty + k (tall, k < 4).
// Tall tiles pass through LDS as tr[own column][own row]: a thread writes the four rows of
// one column as one 8-byte chunk, and each 128-byte row of tr holds its 8-byte chunks at
// chunk ^ 2 ((column >> 3) & 7), which spreads a wave's writes evenly over the banks and
// keeps the 16-byte pairs the read-back takes adjacent.
template <bool kGradBf16>
__global__ __launch_bounds__(256) void k_momentum(MomentumArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t tr[kEwCols][kEwRows + 8];  // tall: [own column][own row]
  __shared__ float red[4];
  const int mi = find_matrix(a.tile_start, a.count, blockIdx.x);
  const int t = blockIdx.x - a.tile_start[mi];
  const int tcols = a.tiles_c[mi];
  const int r0 = (t / tcols) * kEwRows, c0 = (t % tcols) * kEwCols;
  const int m = a.m[mi], n = a.n[mi];
  const bool tall = a.tall[mi] != 0;
  const bool vec = a.vec[mi] != 0;
  const int64_t ldx = a.ldx[mi];
  float* __restrict__ bp = a.b[mi];
  uint16_t* __restrict__ xp = a.x[mi];
  const float mu = a.mu;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float ss = 0.f;
  uint16_t hv[8][4];  // tall: column q, rows 4 ty + k
  // The end of one row: the sum of squares, bf16 V and its store (wide) or its place in the
  // LDS transpose (tall).
  auto finish = [&](int k, int row, int col, const float (&v)[8]) __attribute__((always_inline)) {
    uint16_t h[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      ss = fmaf(v[q], v[q], ss);
      h[q] = f32_to_bf16(v[q]);
    }
    if (!tall) {
      // non-temporal: 2% faster momentum in a same-machine A/B (the products read V from HBM anyway)
      st_nt(pack_bf16x8(h), reinterpret_cast<uint4*>(xp + static_cast<int64_t>(row) * ldx + col));
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) hv[q][k] = h[q];
    }
  };
  if (bp && vec && r0 + kEwRows <= m && c0 + kEwCols <= n) {
    // Interior tile with a momentum buffer (almost every tile): the four rows' loads all go out
    // before any arithmetic, four times the bytes in flight of the row-by-row loop below.
    const int col = c0 + 8 * tx;
    // G is read once per step: non-temporal loads (1% faster in a same-machine A/B), kept packed
    // until used
    Raw8<kGradBf16> gr[4];
    float bv[4][8];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t off = static_cast<int64_t>(r0 + (tall ? 4 * ty + k : ty + 16 * k)) * n + col;
      load_raw8<kGradBf16, true>(a.g[mi], off, gr[k]);
      load8<false>(bp, off, bv[k]);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = r0 + (tall ? 4 * ty + k : ty + 16 * k);
      const int64_t off = static_cast<int64_t>(row) * n + col;
      float gk[8], v[8];
      unpack8(gr[k], gk);
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        bv[k][q] = fmaf(mu, bv[k][q], gk[q]);
        v[q] = a.nesterov ? fmaf(mu, bv[k][q], gk[q]) : bv[k][q];
      }
      *reinterpret_cast<float4*>(bp + off) = make_float4(bv[k][0], bv[k][1], bv[k][2], bv[k][3]);
      *reinterpret_cast<float4*>(bp + off + 4) = make_float4(bv[k][4], bv[k][5], bv[k][6], bv[k][7]);
      finish(k, row, col, v);
    }
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = r0 + (tall ? 4 * ty + k : ty + 16 * k);
      const int col = c0 + 8 * tx;
      float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if (row < m && col < n) {
        const int64_t off = static_cast<int64_t>(row) * n + col;
        if (!bp) {
          if (vec) {
            load8<kGradBf16>(a.g[mi], off, v);
          } else {
#pragma unroll
            for (int q = 0; q < 8; ++q)
              if (col + q < n)
                v[q] = kGradBf16 ? bf16_to_f32(static_cast<const uint16_t*>(a.g[mi])[off + q])
                                 : static_cast<const float*>(a.g[mi])[off + q];
          }
        } else if (vec) {
          float g[8], b[8];
          load8<kGradBf16>(a.g[mi], off, g);
          load8<false>(bp, off, b);
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            b[q] = fmaf(mu, b[q], g[q]);
            v[q] = a.nesterov ? fmaf(mu, b[q], g[q]) : b[q];
          }
          *reinterpret_cast<float4*>(bp + off) = make_float4(b[0], b[1], b[2], b[3]);
          *reinterpret_cast<float4*>(bp + off + 4) = make_float4(b[4], b[5], b[6], b[7]);
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            if (col + q < n) {
              const float gq = kGradBf16 ? bf16_to_f32(static_cast<const uint16_t*>(a.g[mi])[off + q])
                                         : static_cast<const float*>(a.g[mi])[off + q];
              const float bq = fmaf(mu, bp[off + q], gq);
              bp[off + q] = bq;
              v[q] = a.nesterov ? fmaf(mu, bq, gq) : bq;
            }
          }
        }
      }
      finish(k, row, col, v);
    }
  }
  if (tall) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int c = 8 * tx + q;  // local own-column index; its rows 4 ty .. 4 ty + 3 form chunk ty
      uint2 w;
      w.x = hv[q][0] | (static_cast<uint32_t>(hv[q][1]) << 16);
      w.y = hv[q][2] | (static_cast<uint32_t>(hv[q][3]) << 16);
      *reinterpret_cast<uint2*>(&tr[c][4 * (ty ^ (2 * (tx & 7)))]) = w;
    }
    __syncthreads();
    // wide row = own column (128 of them), wide column = own row (64): 8 threads per wide row
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int wr = (threadIdx.x >> 3) + 32 * k;  // local own-column index
      const int j = threadIdx.x & 7;               // own rows 8 j .. 8 j + 7
      const uint4 pk = *reinterpret_cast<const uint4*>(&tr[wr][8 * (j ^ ((wr >> 3) & 7))]);
      *reinterpret_cast<uint4*>(xp + static_cast<int64_t>(c0 + wr) * ldx + r0 + 8 * j) = pk;
    }
  }
  const float tot = block_sum256(ss, red);
  if (threadIdx.x == 0) a.part[mi][t] = tot;
}

// --------------------------------------------------------------------------------
// ||V||_F^2 = sum of the tile partials (fixed order, in double), then 1/||V|| and
// 1/||V||^2 for the Newton-Schulz prescale folded into the first iteration.
__global__ __launch_bounds__(256) void k_norm(NormArgs a) {
  __shared__ double red[4];
  const int mi = blockIdx.x;
  const float* p = a.part[mi];
  double s = 0.0;
  for (int i = threadIdx.x; i < a.nparts[mi]; i += 256) s += static_cast<double>(p[i]);
  s = block_sum256(s, red);
  if (threadIdx.x == 0) {
    MatScalars* sc = a.scal[mi];
    sc->normsq = s;
    sc->inv_norm = s > 0.0 ? static_cast<float>(1.0 / sqrt(s)) : 0.f;
    sc->inv_normsq = s > 0.0 ? static_cast<float>(1.0 / s) : 0.f;
    a.fold[mi][0] = sc->inv_norm;
    a.fold[mi][1] = sc->inv_normsq;
  }
}

// --------------------------------------------------------------------------------
// Sums of squares of the bf16 U per row and per column of one 256 x 256 tile of
// the wide buffer.  Thread t owns columns 8 (t % 32) .. +7 of rows t / 32 + 8 q.
__global__ __launch_bounds__(256) void k_rowcol(RowColArgs a) {
  __shared__ float csh[8][kTile];
  const int mat = blockIdx.y;
  const int ti = blockIdx.x / a.tiles_c, tj = blockIdx.x % a.tiles_c;
  const uint16_t* __restrict__ u = a.u + mat * a.stride_u;
  const int cg = threadIdx.x & 31, rg = threadIdx.x >> 5;
  const int r0 = ti * kTile, c0 = tj * kTile;
  float csum[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  float* rp = a.rpart + mat * a.stride_rpart + static_cast<int64_t>(tj) * a.S + r0;
  for (int q0 = 0; q0 < 32; q0 += 8) {
    uint4 vv[8];  // eight rows' loads in flight
#pragma unroll
    for (int d = 0; d < 8; ++d)
      vv[d] = *reinterpret_cast<const uint4*>(u + static_cast<int64_t>(r0 + rg + 8 * (q0 + d)) * a.L + c0 + 8 * cg);
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      const int r = rg + 8 * (q0 + d);
      const uint32_t w[4] = {vv[d].x, vv[d].y, vv[d].z, vv[d].w};
      float rs = 0.f;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const float lo = bf16_to_f32(w[p] & 0xffffu), hi = bf16_to_f32(w[p] >> 16);
        csum[2 * p] = fmaf(lo, lo, csum[2 * p]);
        csum[2 * p + 1] = fmaf(hi, hi, csum[2 * p + 1]);
        rs = fmaf(lo, lo, rs);
        rs = fmaf(hi, hi, rs);
      }
#pragma unroll
      for (int off = 16; off > 0; off >>= 1) rs += __shfl_xor(rs, off, 64);
      if (cg == 0) rp[r] = rs;
    }
  }
#pragma unroll
  for (int p = 0; p < 8; ++p) csh[rg][8 * cg + p] = csum[p];
  __syncthreads();
  const int c = threadIdx.x;
  float s = 0.f;
#pragma unroll
  for (int g = 0; g < 8; ++g) s += csh[g][c];
  a.cpart[mat * a.stride_cpart + static_cast<int64_t>(ti) * a.L + c0 + c] = s;
}

// --------------------------------------------------------------------------------
// Population standard deviation over mean of the entries above delta (eq. "cv"), two
// passes with fixed-order block reductions; 0 when no entry is above delta.
__device__ double cv_of(const double* v, int len, double delta, double* red) {
  double s = 0.0, cnt = 0.0;
  for (int i = threadIdx.x; i < len; i += 256) {
    const double x = v[i];
    if (x > delta) { s += x; cnt += 1.0; }
  }
  s = block_sum256(s, red);
  cnt = block_sum256(cnt, red);
  if (cnt == 0.0) return 0.0;
  const double mean = s / cnt;
  double q = 0.0;
  for (int i = threadIdx.x; i < len; i += 256) {
    const double x = v[i];
    if (x > delta) q += (x - mean) * (x - mean);
  }
  q = block_sum256(q, red);
  return sqrt(q / cnt) / mean;
}

// r and c (eq. "row-col-rms") from the tile partials, in double: block (x, y) covers
// lines 256 x .. 256 x + 255 of matrix y, where lines 0 .. s-1 are the wide rows and
// s .. s+l-1 the wide columns.  A tall matrix's wide rows are its own columns.
__global__ __launch_bounds__(256) void k_rms(SelectArgs a) {
  const int mi = blockIdx.y;
  const int m = a.m[mi], n = a.n[mi], S = a.S[mi], L = a.L[mi];
  const bool tall = a.tall[mi] != 0;
  const int s_dim = tall ? n : m, l_dim = tall ? m : n;
  const int q = blockIdx.x * 256 + threadIdx.x;
  if (q >= s_dim + l_dim) return;
  double t = 0.0;
  if (q < s_dim) {
    const float* rp = a.rpart[mi] + q;  // (L/256) x S, one partial per wide row and column tile
    for (int k = 0; k < L / kTile; ++k) t += static_cast<double>(rp[static_cast<int64_t>(k) * S]);
    if (!tall) a.rrms[mi][q] = sqrt(t / n); else a.crms[mi][q] = sqrt(t / m);
  } else {
    const int j = q - s_dim;
    const float* cp = a.cpart[mi] + j;  // (S/256) x L, one partial per wide column and row tile
    for (int k = 0; k < S / kTile; ++k) t += static_cast<double>(cp[static_cast<int64_t>(k) * L]);
    if (!tall) a.crms[mi][j] = sqrt(t / m); else a.rrms[mi][j] = sqrt(t / n);
  }
}

// One block per matrix: CVs of r and c over entries above delta (eq. "cv", double, two
// passes), the direction (rows iff gamma_r >= gamma_c, eq. "hidden") and the scale
// vector of N_r or N_c (eq. "operators"; entries at or below delta get scale 0).
__global__ __launch_bounds__(256) void k_select(SelectArgs a) {
  __shared__ double red[4];
  const int mi = blockIdx.x;
  const int m = a.m[mi], n = a.n[mi];
  const double* rr = a.rrms[mi];
  const double* cc = a.crms[mi];
  const double gr = cv_of(rr, m, a.delta, red);
  const double gc = cv_of(cc, n, a.delta, red);
  const int dir = gr >= gc ? 0 : 1;
  float* sc = a.scale[mi];
  const double* v = dir == 0 ? rr : cc;
  const int len = dir == 0 ? m : n;
  for (int i = threadIdx.x; i < len; i += 256) {
    const double x = v[i];
    sc[i] = x > a.delta ? static_cast<float>(1.0 / x) : 0.f;
  }
  if (threadIdx.x == 0) {
    MatScalars* s = a.scal[mi];
    s->gamma_r = gr;
    s->gamma_c = gc;
    s->dir = dir;
  }
}

// --------------------------------------------------------------------------------
// W <- decay * W - step * U * scale over 64 x 128 tiles of the matrix's own orientation
// (thread (ty, tx): columns 8 tx .. 8 tx + 7 of rows ty + 16 k, or of rows 4 ty + k for tall
// matrices); U is read from the padded wide buffer (staged through LDS and transposed for
// tall matrices, in the momentum kernel's swizzled layout).
template <bool kParamBf16>
__global__ __launch_bounds__(256) void k_update(UpdateArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t tr[kEwCols][kEwRows + 8];  // tall: [own column][own row]
  const int mi = find_matrix(a.tile_start, a.count, blockIdx.x);
  const int t = blockIdx.x - a.tile_start[mi];
  const int tcols = a.tiles_c[mi];
  const int r0 = (t / tcols) * kEwRows, c0 = (t % tcols) * kEwCols;
  const int m = a.m[mi], n = a.n[mi];
  const bool tall = a.tall[mi] != 0;
  const bool vec = a.vec[mi] != 0;
  const int64_t ldu = a.ldu[mi];
  const uint16_t* __restrict__ u = a.u[mi];
  const float* __restrict__ scale = a.scale[mi];
  const int dir = a.scal[mi]->dir;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  uint2 tch[8];  // tall: own rows 4 ty .. 4 ty + 3 of column 8 tx + q
  if (tall) {
    // own rows r0.., cols c0.. = wide rows c0.., wide cols r0..  (the wide buffer is padded: no
    // bounds); the same swizzled layout as the momentum kernel's transpose
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int wr = (threadIdx.x >> 3) + 32 * k;
      const int j = threadIdx.x & 7;
      const uint4 pk = *reinterpret_cast<const uint4*>(u + static_cast<int64_t>(c0 + wr) * ldu + r0 + 8 * j);
      *reinterpret_cast<uint4*>(&tr[wr][8 * (j ^ ((wr >> 3) & 7))]) = pk;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 8; ++q) tch[q] = *reinterpret_cast<const uint2*>(&tr[8 * tx + q][4 * (ty ^ (2 * (tx & 7)))]);
  }
  const float decay = a.decay, step = a.step;
  // column scales: the same 8 for all four rows of this thread
  const int col = c0 + 8 * tx;
  float cs[8];
  if (dir != 0) {
    if (col + 8 <= n) {
      const float4 lo = *reinterpret_cast<const float4*>(scale + col);
      const float4 hi = *reinterpret_cast<const float4*>(scale + col + 4);
      cs[0] = lo.x; cs[1] = lo.y; cs[2] = lo.z; cs[3] = lo.w;
      cs[4] = hi.x; cs[5] = hi.y; cs[6] = hi.z; cs[7] = hi.w;
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) cs[q] = (col + q < n) ? scale[col + q] : 0.f;
    }
  }
  // Unpacked U of own row 4 ty + k (tall) from the transposed chunks.
  auto tall_u = [&](int k, float (&uu)[8]) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const uint32_t w = (k < 2) ? tch[q].x : tch[q].y;
      uu[q] = bf16_to_f32(static_cast<uint16_t>((k & 1) ? (w >> 16) : (w & 0xffffu)));
    }
  };
  if (vec && r0 + kEwRows <= m && c0 + kEwCols <= n) {
    // Interior tile (almost every tile): the four rows' loads of U, W and the row scales all go
    // out before any arithmetic.
    float uu[4][8], wv[4][8], sr[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = r0 + (tall ? 4 * ty + k : ty + 16 * k);
      if (!tall) load8<true, true>(u, static_cast<int64_t>(row) * ldu + col, uu[k]);
      load8<kParamBf16, true>(a.w[mi], static_cast<int64_t>(row) * n + col, wv[k]);
      if (dir == 0) sr[k] = scale[row];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = r0 + (tall ? 4 * ty + k : ty + 16 * k);
      const int64_t off = static_cast<int64_t>(row) * n + col;
      if (tall) tall_u(k, uu[k]);
      float w[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) w[q] = fmaf(decay, wv[k][q], -step * (uu[k][q] * (dir == 0 ? sr[k] : cs[q])));
      if (kParamBf16) {
        uint16_t h[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) h[q] = f32_to_bf16(w[q]);
        st_nt(pack_bf16x8(h), reinterpret_cast<uint4*>(static_cast<uint16_t*>(a.w[mi]) + off));
      } else {
        float* wp = static_cast<float*>(a.w[mi]);
        *reinterpret_cast<float4*>(wp + off) = make_float4(w[0], w[1], w[2], w[3]);
        *reinterpret_cast<float4*>(wp + off + 4) = make_float4(w[4], w[5], w[6], w[7]);
      }
    }
    return;
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int row = r0 + (tall ? 4 * ty + k : ty + 16 * k);
    if (row >= m || col >= n) continue;
    float uu[8];
    if (!tall) {
      load8<true, true>(u, static_cast<int64_t>(row) * ldu + col, uu);
    } else {
      tall_u(k, uu);
    }
    float s[8];
    if (dir == 0) {
      const float sr = scale[row];
#pragma unroll
      for (int q = 0; q < 8; ++q) s[q] = sr;
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) s[q] = cs[q];
    }
    const int64_t off = static_cast<int64_t>(row) * n + col;
    if (vec) {
      float w[8];
      load8<kParamBf16, true>(a.w[mi], off, w);
#pragma unroll
      for (int q = 0; q < 8; ++q) w[q] = fmaf(decay, w[q], -step * (uu[q] * s[q]));
      if (kParamBf16) {
        uint16_t h[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) h[q] = f32_to_bf16(w[q]);
        st_nt(pack_bf16x8(h), reinterpret_cast<uint4*>(static_cast<uint16_t*>(a.w[mi]) + off));
      } else {
        float* wp = static_cast<float*>(a.w[mi]);
        *reinterpret_cast<float4*>(wp + off) = make_float4(w[0], w[1], w[2], w[3]);
        *reinterpret_cast<float4*>(wp + off + 4) = make_float4(w[4], w[5], w[6], w[7]);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if (col + q >= n) break;
        if (kParamBf16) {
          uint16_t* wp = static_cast<uint16_t*>(a.w[mi]);
          wp[off + q] = f32_to_bf16(fmaf(decay, bf16_to_f32(wp[off + q]), -step * (uu[q] * s[q])));
        } else {
          float* wp = static_cast<float*>(a.w[mi]);
          wp[off + q] = fmaf(decay, wp[off + q], -step * (uu[q] * s[q]));
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_momentum(const MomentumArgs& a, int grad_bf16, int total_tiles, hipStream_t st) {
  if (grad_bf16)
    hipLaunchKernelGGL(k_momentum<true>, dim3(total_tiles), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(k_momentum<false>, dim3(total_tiles), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_norm(const NormArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_norm, dim3(a.count), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_rowcol(const RowColArgs& a, int batch, hipStream_t st) {
  hipLaunchKernelGGL(k_rowcol, dim3(a.tiles_r * a.tiles_c, batch), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_rms(const SelectArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_rms, dim3((a.max_lines + 255) / 256, a.count), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_select, dim3(a.count), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_update(const UpdateArgs& a, int param_bf16, int total_tiles, hipStream_t st) {
  if (param_bf16)
    hipLaunchKernelGGL(k_update<true>, dim3(total_tiles), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(k_update<false>, dim3(total_tiles), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace meq
