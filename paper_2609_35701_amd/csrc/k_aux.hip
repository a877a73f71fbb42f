// Streaming kernels of the other MeqMuon parameter kinds (Algorithm "MeqMuon") and of
// the Moonlight-Muon scale (eq. "moonlight-update").  All are HBM-bound.
//   remaining 2D parameters, U~ = N_c(N_r(V))          eq. "aux"
//     k_aux_rows    momentum B <- mu B + G, V, row RMS r of V and 1/r       (one wave per row)
//     k_aux_cols    partial column sums of (V_ij / r_i)^2 over 128-row blocks
//     k_aux_colfin  column RMS c of N_r(V) and 1/c
//     k_aux_update  W <- decay W - step V_ij / (r_i c_j)                    (one wave per row)
//   1-D parameters, U~ = V / (||V|| / sqrt(d))          eq. "vector"
//     k_vec         momentum, ||V||^2 and the write-back of one vector per block
// Rows or columns with RMS at or below delta get scale 0 (they stay zero).  Sums of
// squares accumulate in double and reduce in a fixed order, so results are bitwise
// reproducible run to run.
#include "meq_internal.h"

namespace meq {

namespace {

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// float -> bfloat16 bits, round to nearest, ties to even; NaN stays NaN (quieted).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// Four consecutive elements of a bf16 or fp32 array as floats (8- or 16-byte access).
template <bool kBf16>
__device__ __forceinline__ void load4(const void* p, int64_t i, float (&x)[4]) {
  if (kBf16) {
    const uint2 v = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(p) + i);
    x[0] = bf16_bits_to_f32(v.x & 0xffffu);
    x[1] = bf16_bits_to_f32(v.x >> 16);
    x[2] = bf16_bits_to_f32(v.y & 0xffffu);
    x[3] = bf16_bits_to_f32(v.y >> 16);
  } else {
    const float4 v = *reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
    x[0] = v.x;
    x[1] = v.y;
    x[2] = v.z;
    x[3] = v.w;
  }
}

template <bool kBf16>
__device__ __forceinline__ void store4(void* p, int64_t i, const float (&x)[4]) {
  if (kBf16) {
    uint2 v;
    v.x = f32_to_bf16_bits(x[0]) | (f32_to_bf16_bits(x[1]) << 16);
    v.y = f32_to_bf16_bits(x[2]) | (f32_to_bf16_bits(x[3]) << 16);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p) + i) = v;
  } else {
    *reinterpret_cast<float4*>(static_cast<float*>(p) + i) = make_float4(x[0], x[1], x[2], x[3]);
  }
}

template <bool kBf16>
__device__ __forceinline__ float load1(const void* p, int64_t i) {
  if (kBf16) return bf16_bits_to_f32(static_cast<const uint16_t*>(p)[i]);
  return static_cast<const float*>(p)[i];
}

template <bool kBf16>
__device__ __forceinline__ void store1(void* p, int64_t i, float x) {
  if (kBf16)
    static_cast<uint16_t*>(p)[i] = static_cast<uint16_t>(f32_to_bf16_bits(x));
  else
    static_cast<float*>(p)[i] = x;
}

// ------------------------------------------------------------------ eq. "aux", rows
template <bool kGradBf16>
__global__ __launch_bounds__(256) void k_aux_rows(AuxArgs a) {
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * kAuxRowsPerBlock + (threadIdx.x >> 6);
  if (i >= a.m) return;  // whole wave
  const int n = a.n;
  const int64_t base = static_cast<int64_t>(i) * n;
  const float mu = a.mu;
  double ss = 0.0;
  if (a.vec) {
    for (int c = 4 * lane; c < n; c += 256) {
      float g[4], b[4];
      load4<kGradBf16>(a.g, base + c, g);
      load4<false>(a.b, base + c, b);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        b[q] = fmaf(mu, b[q], g[q]);
        const float v = a.nesterov ? fmaf(mu, b[q], g[q]) : b[q];
        ss += static_cast<double>(v) * v;
      }
      store4<false>(a.b, base + c, b);
    }
  } else {
    for (int c = lane; c < n; c += 64) {
      const float g = load1<kGradBf16>(a.g, base + c);
      const float b = fmaf(mu, a.b[base + c], g);
      a.b[base + c] = b;
      const float v = a.nesterov ? fmaf(mu, b, g) : b;
      ss += static_cast<double>(v) * v;
    }
  }
  ss = wave_sum_d(ss);
  if (lane == 0) {
    const double r = sqrt(ss / n);
    a.rrms[i] = r;
    a.rscale[i] = r > a.delta ? static_cast<float>(1.0 / r) : 0.f;
  }
}

// --------------------------------------------------------------- eq. "aux", columns
// Block (x, y): columns 1024 x .. 1024 x + 1023 (4 per thread), rows kAuxColRows y .. + kAuxColRows - 1,
// eight rows' loads in flight per thread.
template <bool kGradBf16>
__global__ __launch_bounds__(256) void k_aux_cols(AuxArgs a) {
  constexpr int U = 8;
  const int n = a.n;
  const int r0 = blockIdx.y * kAuxColRows;
  const int r1 = min(a.m, r0 + kAuxColRows);
  const float mu = a.mu;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  if (a.vec) {
    const int c = blockIdx.x * 1024 + 4 * threadIdx.x;
    if (c >= n) return;
    for (int r = r0; r < r1; r += U) {
      float b[U][4], g[U][4], rs[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int rr = min(r + u, r1 - 1);  // rows past r1 are loaded again and not added
        const int64_t off = static_cast<int64_t>(rr) * n + c;
        load4<false>(a.b, off, b[u]);
        if (a.nesterov) load4<kGradBf16>(a.g, off, g[u]);
        rs[u] = a.rscale[rr];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (r + u >= r1) break;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float v = a.nesterov ? fmaf(mu, b[u][q], g[u][q]) : b[u][q];
          const float x = v * rs[u];
          acc[q] += static_cast<double>(x) * x;
        }
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) a.cpart[static_cast<int64_t>(blockIdx.y) * n + c + q] = acc[q];
  } else {
    for (int q = 0; q < 4; ++q) {
      const int c = blockIdx.x * 1024 + threadIdx.x + 256 * q;
      if (c >= n) break;
      double t = 0.0;
      for (int r = r0; r < r1; ++r) {
        const int64_t off = static_cast<int64_t>(r) * n + c;
        const float b = a.b[off];
        const float v = a.nesterov ? fmaf(mu, b, load1<kGradBf16>(a.g, off)) : b;
        const float x = v * a.rscale[r];
        t += static_cast<double>(x) * x;
      }
      a.cpart[static_cast<int64_t>(blockIdx.y) * n + c] = t;
    }
  }
}

// 16 columns per block: the 16 threads of a column each sum every 16th row block (short
// chains of loads, and enough blocks to spread over the CUs), then meet in LDS, added in a
// fixed order.
__global__ __launch_bounds__(256) void k_aux_colfin(AuxArgs a) {
  __shared__ double part[16][16];
  const int jj = threadIdx.x & 15, w = threadIdx.x >> 4;
  const int j = blockIdx.x * 16 + jj;
  double t = 0.0;
  if (j < a.n)
    for (int k = w; k < a.row_blocks; k += 16) t += a.cpart[static_cast<int64_t>(k) * a.n + j];
  part[w][jj] = t;
  __syncthreads();
  if (w == 0 && j < a.n) {
    double q4[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      q4[q] = (part[4 * q][jj] + part[4 * q + 1][jj]) + (part[4 * q + 2][jj] + part[4 * q + 3][jj]);
    const double sum = (q4[0] + q4[1]) + (q4[2] + q4[3]);
    const double c = sqrt(sum / a.m);
    a.crms[j] = c;
    a.cscale[j] = c > a.delta ? static_cast<float>(1.0 / c) : 0.f;
  }
}

// ------------------------------------------------------------ eq. "aux", write-back
template <bool kBf16>
__global__ __launch_bounds__(256) void k_aux_update(AuxArgs a) {
  const int lane = threadIdx.x & 63;
  const int i = blockIdx.x * kAuxRowsPerBlock + (threadIdx.x >> 6);
  if (i >= a.m) return;
  const int n = a.n;
  const int64_t base = static_cast<int64_t>(i) * n;
  const float mu = a.mu, decay = a.decay, step = a.step;
  const float rs = a.rscale[i];
  if (a.vec) {
    for (int c = 4 * lane; c < n; c += 256) {
      float b[4], w[4];
      load4<false>(a.b, base + c, b);
      load4<kBf16>(a.w, base + c, w);
      float g[4] = {0.f, 0.f, 0.f, 0.f};
      if (a.nesterov) load4<kBf16>(a.g, base + c, g);
      const float4 cs = *reinterpret_cast<const float4*>(a.cscale + c);
      const float css[4] = {cs.x, cs.y, cs.z, cs.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float v = a.nesterov ? fmaf(mu, b[q], g[q]) : b[q];
        w[q] = fmaf(decay, w[q], -step * ((v * rs) * css[q]));
      }
      store4<kBf16>(a.w, base + c, w);
    }
  } else {
    for (int c = lane; c < n; c += 64) {
      const float b = a.b[base + c];
      const float v = a.nesterov ? fmaf(mu, b, load1<kBf16>(a.g, base + c)) : b;
      const float w = load1<kBf16>(a.w, base + c);
      store1<kBf16>(a.w, base + c, fmaf(decay, w, -step * ((v * rs) * a.cscale[c])));
    }
  }
}

// ------------------------------------------------------------------- eq. "vector"
// One block per vector.  Both passes give each thread the same elements, so the second
// pass reads back only momenta this thread wrote itself.
template <bool kBf16>
__global__ __launch_bounds__(256) void k_vec(VecArgs a) {
  __shared__ double red[4];
  const int k = blockIdx.x;
  const int64_t len = a.len[k];
  const bool vec = a.vec[k] != 0;
  const float mu = a.mu;
  float* __restrict__ bp = a.b[k];
  double ss = 0.0;
  if (vec) {
    for (int64_t e = 4 * static_cast<int64_t>(threadIdx.x); e < len; e += 1024) {
      float g[4], b[4];
      load4<kBf16>(a.g[k], e, g);
      load4<false>(bp, e, b);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        b[q] = fmaf(mu, b[q], g[q]);
        const float v = a.nesterov ? fmaf(mu, b[q], g[q]) : b[q];
        ss += static_cast<double>(v) * v;
      }
      store4<false>(bp, e, b);
    }
  } else {
    for (int64_t e = threadIdx.x; e < len; e += 256) {
      const float g = load1<kBf16>(a.g[k], e);
      const float b = fmaf(mu, bp[e], g);
      bp[e] = b;
      const float v = a.nesterov ? fmaf(mu, b, g) : b;
      ss += static_cast<double>(v) * v;
    }
  }
  ss = wave_sum_d(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const double tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float inv = tot > 0.0 ? static_cast<float>(sqrt(static_cast<double>(len) / tot)) : 0.f;
  if (threadIdx.x == 0) *a.normsq[k] = tot;
  const float decay = a.decay, step = a.step;
  if (vec) {
    for (int64_t e = 4 * static_cast<int64_t>(threadIdx.x); e < len; e += 1024) {
      float b[4], w[4];
      load4<false>(bp, e, b);
      load4<kBf16>(a.w[k], e, w);
      float g[4] = {0.f, 0.f, 0.f, 0.f};
      if (a.nesterov) load4<kBf16>(a.g[k], e, g);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float v = a.nesterov ? fmaf(mu, b[q], g[q]) : b[q];
        w[q] = fmaf(decay, w[q], -step * (v * inv));
      }
      store4<kBf16>(a.w[k], e, w);
    }
  } else {
    for (int64_t e = threadIdx.x; e < len; e += 256) {
      const float b = bp[e];
      const float v = a.nesterov ? fmaf(mu, b, load1<kBf16>(a.g[k], e)) : b;
      store1<kBf16>(a.w[k], e, fmaf(decay, load1<kBf16>(a.w[k], e), -step * (v * inv)));
    }
  }
}

// ------------------------------------------------------- eq. "moonlight-update" scale
// Every row of U~ = sqrt(max(m, n)) U gets the same scale; direction "rows".
__global__ __launch_bounds__(256) void k_scale_fill(SelectArgs a) {
  const int mi = blockIdx.x;
  const int m = a.m[mi], n = a.n[mi];
  const float s = static_cast<float>(sqrt(static_cast<double>(max(m, n))));
  for (int i = threadIdx.x; i < m; i += 256) a.scale[mi][i] = s;
  if (threadIdx.x == 0) {
    MatScalars* sc = a.scal[mi];
    sc->gamma_r = 0.0;
    sc->gamma_c = 0.0;
    sc->dir = 0;
  }
}

}  // namespace

hipError_t launch_aux_rows(const AuxArgs& a, int grad_bf16, hipStream_t st) {
  const dim3 grid((a.m + kAuxRowsPerBlock - 1) / kAuxRowsPerBlock);
  if (grad_bf16)
    hipLaunchKernelGGL(k_aux_rows<true>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(k_aux_rows<false>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_aux_cols(const AuxArgs& a, int grad_bf16, hipStream_t st) {
  const dim3 grid((a.n + 1023) / 1024, a.row_blocks);
  if (grad_bf16)
    hipLaunchKernelGGL(k_aux_cols<true>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(k_aux_cols<false>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_aux_colfin(const AuxArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_aux_colfin, dim3((a.n + 15) / 16), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_aux_update(const AuxArgs& a, int bf16, hipStream_t st) {
  const dim3 grid((a.m + kAuxRowsPerBlock - 1) / kAuxRowsPerBlock);
  if (bf16)
    hipLaunchKernelGGL(k_aux_update<true>, grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(k_aux_update<false>, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_vec(const VecArgs& a, int bf16, hipStream_t st) {
  if (bf16)
    hipLaunchKernelGGL(k_vec<true>, dim3(a.count), dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL(k_vec<false>, dim3(a.count), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_scale_fill(const SelectArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(k_scale_fill, dim3(a.count), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace meq
