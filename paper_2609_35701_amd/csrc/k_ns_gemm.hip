// Newton-Schulz products on MFMA (gfx950), eq. "ns":
//   A_k = X_k X_k^T                (NT, symmetric: tiles on or above the diagonal + mirrored store)
//   P_k = a I + b A_k + c A_k A_k  (NT since A_k is symmetric; symmetric output)
//   X_{k+1} = P_k X_k              (NN: X_k is staged K-major and read with LDS transpose reads)
// which is a X_k + (b A_k + c A_k A_k) X_k regrouped: the a X_k term rides on the
// diagonal of P_k, so the apply epilogue reads nothing besides its accumulators.
// A Gram-space segment uses the same three kernels: the symmetric NT product also forms
// P_k A_k, P_k T and P_k Q (commuting symmetric factors), and the NN product X <- Q X.
// X_0 = V / ||V||_F is folded in: the bf16 buffer holds V, the k = 0 Gram epilogue
// scales by 1/||V||^2 and the k = 0 apply epilogue by 1/||V||.
// Formats: X and the matrix multiplying it are bf16 (v_mfma_f32_32x32x16_bf16); A and the
// other S x S matrices may be fp16 (kF16: v_mfma_f32_32x32x16_f16); each product stores its
// output as bf16 or fp16 (per shape group, GemmGroup::out_f16) with per-group coefficients.
//
// One workgroup = 4 waves = one 256 x 256 output tile; each wave owns a 128 x 128
// quadrant as 4 x 4 blocks of 32 x 32 x 16 MFMAs (fp32 accumulation in AGPRs).
// K advances in slabs of 64 through an LDS ring: operand A in 2 buffers and operand B in 3
// buffers of 32 KiB, so B is fetched a slab further ahead; that is all of the 160 KiB of
// LDS.  This measured faster for all three products than a 4-stage ring of 32-wide slabs,
// a 2-stage ring of 64-wide slabs, or 3 buffers for operand A instead.  Global ->
// LDS traffic uses buffer loads that write LDS directly (no registers, no LDS store
// instructions); 16-byte chunks are XOR-swizzled so fragment reads are free of bank
// conflicts.  The epilogue stages the output tile (and, for P, the A tile it adds) in
// LDS and writes whole rows with 16-byte stores.  Same-shape matrices form one
// launch; workgroup ids are remapped so each XCD receives a contiguous run of tiles.
// Diagonal tiles of X X^T and of the polynomial's A A (a matrix times its own transpose) take
// a path of their own that computes only the 36 needed 32 x 32 blocks from one operand.
// Every lambda is forced inline: one left outlined would pass the accumulators by reference,
// that is through scratch memory.
#include <type_traits>

#include "meq_internal.h"

namespace meq {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) uint8_t lds_u8;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) u32x2 lds_u32x2;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

// Buffer resource word 3 for raw (untyped, 32-bit format) buffer access on gfx9.
constexpr int kBufferFlags = 0x00020000;

__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }
__device__ __forceinline__ float f16_to_f32(uint32_t h) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(h)));
}

// Two floats -> packed bf16 pair (v_cvt_pk_bf16_f32: round to nearest even), lo first.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2 v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}
// Two floats -> packed fp16 pair (round to nearest even), lo first.
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  const half2 v = {static_cast<_Float16>(lo), static_cast<_Float16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

// Map a launch-order workgroup id to a logical tile so that the workgroups one
// XCD receives (ids x, x + 8, x + 16, ... are dispatched round-robin over the 8
// XCDs) form one contiguous run of logical tiles.
__device__ __forceinline__ int xcd_remap(int w, int nblk) {
  const int q = nblk >> 3, r = nblk & 7;
  const int x = w & 7, pos = w >> 3;
  return x * q + min(x, r) + pos;
}

// 16 bytes per lane from a buffer straight into LDS at dst + 16 * lane.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, lds_u8* dst, int voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)dst, 16, voff, soff, 0, 0);
}

// s_waitcnt vmcnt(n) with expcnt and lgkmcnt left at their maxima (gfx9 encoding).
template <int n>
__device__ __forceinline__ void wait_vm() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((n & 15) | ((n >> 4) << 14) | 0x0f70);
}

// LDS layouts (bytes).  Each 16-lane pass of an LDS access covers 256 bytes (64 banks).
//   NT slab (256 rows x 64 k):   row r at r * 128; 16-byte chunk c (k = 8c..8c+7) at slot c ^ ((r >> 1) & 7),
//                                so 16 consecutive rows read at one chunk fill the 256 bytes exactly.
//   NN slab (64 k x 256 n):      row k at k * 512; chunk c (n = 8c..8c+7) at slot c ^ (4 (k & 3)), so the
//                                4 rows x 4 chunks a 32-lane transpose read touches fill 256 bytes exactly.
//   staged output (256 x 256):   row r in ring buffer r / 64 at (r % 64) * 512; chunk c at slot c ^ (r & 31).
__device__ __forceinline__ int stage_byte(int rr, int c) {
  return (rr & 63) * 512 + 16 * ((c >> 3) ^ (rr & 31)) + 2 * (c & 7);
}

// Scheduling pattern of one 16-MFMA k step: kReads LDS reads (for the next step) and
// kDma LDS-bound buffer loads interleaved between the MFMAs, the loads at most one per
// two MFMAs (a load can hold up the wave's issue behind outstanding misses).
template <int kReads, int kDma>
__device__ __forceinline__ void sched_step() {
#ifndef MEQ_NO_SCHED
#define MEQ_SG(mask, n) __builtin_amdgcn_sched_group_barrier(mask, n, 0)
#define MEQ_QUAD(r, d)                    \
  if (r > 0) MEQ_SG(0x100, r);            \
  MEQ_SG(0x008, 1);                       \
  if (d > 0) MEQ_SG(0x020, (d + 1) / 2);  \
  MEQ_SG(0x008, 1);                       \
  if (r > 0) MEQ_SG(0x100, r);            \
  MEQ_SG(0x008, 1);                       \
  if (d > 1) MEQ_SG(0x020, d / 2);        \
  MEQ_SG(0x008, 1);
  constexpr int r0 = kReads / 8, r1 = kReads / 4 - kReads / 8;  // 4 (r0 + r1) reads
  constexpr int d = kDma / 4;
  MEQ_QUAD(r1, d) MEQ_QUAD(r0, d) MEQ_QUAD(r1, d) MEQ_QUAD(r0, d)
#undef MEQ_QUAD
#undef MEQ_SG
#endif
}


// Scheduling pattern of one k step of a diagonal tile: nM MFMAs with the nR LDS reads of the next
// step placed at the start, two after each of the first MFMAs (each step's fragment registers are
// free once the previous step's MFMAs are issued), and the nD LDS-bound loads spread over the step.
template <int nM, int nR, int nD, int m = 0>
__device__ __forceinline__ void dsched() {
#ifndef MEQ_NO_SCHED
  if constexpr (m < nM) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    constexpr int r = (2 * m + 2 <= nR) ? 2 : (2 * m < nR ? nR - 2 * m : 0);  // two per MFMA, from the first
    if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(0x100, r, 0);
    constexpr int d = (nD * (m + 2)) / nM - (nD * (m + 1)) / nM;
    if constexpr (d > 0) __builtin_amdgcn_sched_group_barrier(0x020, d, 0);
    dsched<nM, nR, nD, m + 1>();
  }
#endif
}

template <int kMode, bool kF16>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_ns_gemm(GemmArgs args) {
  constexpr bool kNN = kMode == 2;
  constexpr bool kSym = kMode != 2;
  constexpr bool kHasE = kMode == 1;
  // Ring geometry
  constexpr int BK = 64;               // k per slab
  constexpr int kBufBytes = 32768;     // one operand's slab
  constexpr int kRowBytes = 2 * BK;    // one NT slab row
  constexpr int kDma = 16;             // LDS-bound buffer loads per wave per slab (8 per operand)
  // Ring buffers as separate objects, so the compiler can tell the buffer being read from
  // the buffers being filled: st0, st1 hold operand A, st2, st3, st4 operand B.  The
  // epilogue stages its output in st0..st3 and the fused row and column partials in st4.
  __shared__ __attribute__((aligned(1024))) uint8_t st0_[kBufBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t st1_[kBufBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t st2_[kBufBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t st3_[kBufBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t st4_[kBufBytes];
  lds_u8* const st0 = (lds_u8*)st0_;
  lds_u8* const st1 = (lds_u8*)st1_;
  lds_u8* const st2 = (lds_u8*)st2_;
  lds_u8* const st3 = (lds_u8*)st3_;
  lds_u8* const st4 = (lds_u8*)st4_;
  // apply: per-wave column partials of the fused sums, in the ring's fifth buffer
  typedef __attribute__((address_space(3))) float lds_f32;
  lds_f32* const colsum = (lds_f32*)st4_;
  // The epilogue stages 64-row quarters of the output tile, 32 KiB each.
  auto stage_of = [&](int q) { return q == 0 ? st0 : q == 1 ? st1 : q == 2 ? st2 : st3; };

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);  // wave-uniform: scalar offsets and LDS bases
  const int wm = wave >> 1, wn = wave & 1;
  const int h = lane >> 5;

  // workgroup -> (shape group, matrix, tile).  Each group's range starts at a multiple
  // of 8, so the XCD remap runs within the group.
  int gi = 0;
  while (gi + 1 < args.count && static_cast<int>(blockIdx.x) >= args.tile_start[gi + 1]) ++gi;
  const GemmGroup& g = args.grp[gi];
  const int u = blockIdx.x - args.tile_start[gi];
  const int logical = xcd_remap(u, args.tile_start[gi + 1] - args.tile_start[gi]);
  if (logical >= g.tiles) return;  // padding slot (uniform over the workgroup)
  const int mat = logical / g.tiles_per_mat;
  int tile = logical - mat * g.tiles_per_mat;
  int ti, tj;
  if (kSym) {
    // A matrix's T diagonal tiles come after its T (T - 1) / 2 others when they take the short
    // path of a matrix times itself (the short tiles then fill the end of the launch), and
    // first when they carry the symmetrizing pass of two different factors.
    const int T = g.tiles_m, noff = T * (T - 1) / 2;
    const bool self = g.a == g.b && g.lda == g.ldb && g.stride_a == g.stride_b;
    const int dpos = self ? noff : 0;
    if (tile >= dpos && tile < dpos + T) {
      ti = tj = tile - dpos;
    } else {
      if (tile >= dpos + T) tile -= T;
      ti = 0;  // off-diagonal tiles row by row
      int rowlen = T - 1;
      while (tile >= rowlen) {
        tile -= rowlen;
        ++ti;
        --rowlen;
      }
      tj = ti + 1 + tile;
    }
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

  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(g.a + mat * g.stride_a), 0, 0x7fffffff, kBufferFlags);
  const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(g.b + mat * g.stride_b), 0, 0x7fffffff, kBufferFlags);
  const int lda = g.lda, ldb = g.ldb;
  const int rowA0 = ti * 256;
  const int rowB0 = tj * 256;  // NT: operand-B rows; NN: output columns

  // ---- global -> LDS slab loads: 8 instructions per wave per operand (1 KiB each).
  // NT: instruction I = 8 wave + i covers rows 8I .. 8I + 7; lane -> row 8I + lane / 8,
  //     slot lane % 8, which holds chunk slot ^ ((row >> 1) & 7) = slot ^ (lane >> 4) ^ 4 (I & 1).
  constexpr int kRowsPerDma = 1024 / kRowBytes;
  const int nt_r = lane >> 3;
  const int nt_c = (lane & 7) ^ (lane >> 4);
  const int vA = 2 * ((rowA0 + nt_r) * lda + 8 * nt_c);                // even I
  const int vA_odd = 2 * ((rowA0 + nt_r) * lda + 8 * (nt_c ^ 4));      // odd I
  const int vB_nt = 2 * ((rowB0 + nt_r) * ldb + 8 * nt_c);
  const int vB_nt_odd = 2 * ((rowB0 + nt_r) * ldb + 8 * (nt_c ^ 4));
  // NN: instruction I = 8 wave + i covers k rows 2I, 2I + 1; lane -> row 2I + lane/32, slot lane%32.
  const int nn_r = lane >> 5;
  const int vB_nn0 = 2 * (nn_r * ldb + rowB0 + 8 * ((lane & 31) ^ (4 * (nn_r & 3))));
  const int vB_nn1 = 2 * (nn_r * ldb + rowB0 + 8 * ((lane & 31) ^ (4 * ((2 + nn_r) & 3))));

  auto issue_half_a = [&](lds_u8* abuf, int kt, int i0 = 0, int i1 = kDma / 2) __attribute__((always_inline)) {
    const int k0 = kt * BK;
#pragma unroll
    for (int i = i0; i < i1; ++i) {
      const int I = (kDma / 2) * wave + i;
      dma16(rA, abuf + I * 1024, (i & 1) ? vA_odd : vA, 2 * (kRowsPerDma * I * lda + k0));
    }
  };
  auto issue_half_b = [&](lds_u8* bbuf, int kt, int i0 = 0, int i1 = kDma / 2) __attribute__((always_inline)) {
    const int k0 = kt * BK;
#pragma unroll
    for (int i = i0; i < i1; ++i) {
      const int I = (kDma / 2) * wave + i;
      if (kNN)
        dma16(rB, bbuf + I * 1024, (i & 1) ? vB_nn1 : vB_nn0, 2 * ((k0 + 2 * I) * ldb));
      else
        dma16(rB, bbuf + I * 1024, (i & 1) ? vB_nt_odd : vB_nt, 2 * (kRowsPerDma * I * ldb + k0));
    }
  };

  // ---- fragment addresses (bytes within a buffer)
  // NT fragment: row R = base + 32 i + lane%32 (base a multiple of 32), k chunk 2 kk + lane/32,
  // at slot chunk ^ ((R >> 1) & 7) = chunk ^ (((lane & 31) >> 1) & 7).
  const int offA = (wm * 128 + (lane & 31)) * kRowBytes;
  const int offB_nt = (wn * 128 + (lane & 31)) * kRowBytes;
  const int nt_swz = ((lane & 31) >> 1) & 7;
  int slot_kk[BK / 16];
#pragma unroll
  for (int kk = 0; kk < BK / 16; ++kk) slot_kk[kk] = 16 * ((2 * kk + h) ^ nt_swz);
  // NN fragment via ds_read_b64_tr_b16: within each 16-lane group, lane q points at
  // k row q / 4 and n columns 4 (q % 4) .. +3; afterwards lane q holds 4 consecutive k
  // of column q, so two reads give the 8 k values an MFMA operand lane needs.
  const int jq = lane & 15, grp = lane >> 4;
  const int nn_k = 8 * (grp >> 1) + (jq >> 2);                // + 16 kk + 4 t
  const int nn_n = wn * 128 + 16 * (grp & 1) + 4 * (jq & 3);  // + 32 j
  const int nn_swz = 4 * (nn_k & 3);
  // Lane part of the address of column block j.  Rows k + 16 kk + 4 t lie (16 kk + 4 t) * 512
  // bytes further with the same swizzle (it depends on k & 3 only).  One precomputed offset
  // per block keeps every read a short constant step from its stage array, which is what
  // lets the compiler tell the stages apart when it places waits for the LDS-bound loads.
  int nn_off[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = nn_n + 32 * j;
    nn_off[j] = nn_k * 512 + 16 * ((n >> 3) ^ nn_swz) + 2 * (n & 7);
  }

  // Stage E (the polynomial's A tile, the same rows and columns as OUT, which starts at row
  // out_row0 and column out_col0 of the matrix) in st0..st3: 32 instructions per stage, 2 rows each.
  auto stage_e = [&](int out_row0, int out_col0) __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rE = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(g.e + mat * g.stride_e), 0, 0x7fffffff, kBufferFlags);
    const int lde = g.lde;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      lds_u8* dst = stage_of(q);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int I = 8 * wave + i;  // rows 2I, 2I + 1 of this stage
        const int r = 64 * q + 2 * I + h;
        const int c = (lane & 31) ^ (r & 31);
        dma16(rE, dst + I * 1024, 2 * ((out_row0 + 64 * q + h) * lde + out_col0 + 8 * c), 2 * (2 * I * lde));
      }
    }
    wait_vm<0>();
    __syncthreads();
  };

  // Diagonal tile of a product of a matrix with itself (X X^T, A A): OUT is symmetric, and only the
  // lower block triangle of OUT (36 of its 64 32 x 32 blocks, the product's upper triangle) is
  // computed.  Waves 0 and 1 take the lower triangles of the two diagonal 128 x 128 quadrants (10
  // blocks each, from the 4 fragments of their own rows, which serve both factors); waves 2 and 3
  // take the two 128 x 64 halves of the off-diagonal quadrant (8 blocks each, from 2 + 4
  // fragments).  Only operand A is fetched (the same 256 rows are both factors), into a ring of
  // four 32 KiB buffers, three slabs ahead.
  const bool dfast = kSym && ti == tj && g.a == g.b && g.lda == g.ldb && g.stride_a == g.stride_b;
  if (dfast) {
    if constexpr (kSym) {
      const int nkd = g.K / BK;  // a multiple of 4
      const bool roleD = wave < 2;
      const int q = wave & 1;
      auto dbar = []() __attribute__((always_inline)) {
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
      };
      auto dmfma = [&](const bf16x8& x, const bf16x8& y, floatx16& c) __attribute__((always_inline)) {
        if constexpr (kF16)
          c = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, x), __builtin_bit_cast(half8, y), c, 0, 0, 0);
        else
          c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, c, 0, 0, 0);
      };
      floatx16 dacc[10];
#pragma unroll
      for (int n = 0; n < 10; ++n)
#pragma unroll
        for (int v = 0; v < 16; ++v) dacc[n][v] = 0.f;
      // fragment bases: role D rows 128 q + 32 i; role O A-side rows 64 q + 32 i, B-side 128 + 32 j
      const int offD = (128 * q + (lane & 31)) * kRowBytes;
      const int offOA = (64 * q + (lane & 31)) * kRowBytes;
      const int offOB = (128 + (lane & 31)) * kRowBytes;
      // slab kt's buffer is st[kt % 4]; during slab kt the loads of slab kt + 3 go into the buffer
      // slab kt - 1 used (free since slab kt - 1's barrier); at slab kt's barrier the loads of
      // slabs kt + 2 and the first 6 of kt + 3 may still be in flight.
      issue_half_a(st0, 0);
      issue_half_a(st1, 1);
      issue_half_a(st2, 2);
      wait_vm<16>();
      dbar();
      if (roleD) {
        bf16x8 f[4], gq[4];
        auto rd = [&](const lds_u8* buf, int kk, bf16x8 (&x)[4]) __attribute__((always_inline)) {
          const int o = offD + slot_kk[kk];
#pragma unroll
          for (int i = 0; i < 4; ++i) x[i] = *reinterpret_cast<const lds_bf16x8*>(buf + o + i * 32 * kRowBytes);
        };
        auto mf = [&](const bf16x8 (&x)[4]) __attribute__((always_inline)) {
          int n = 0;
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = i; j < 4; ++j) dmfma(x[i], x[j], dacc[n++]);
        };
        auto dslab = [&](const lds_u8* cur, const lds_u8* nxt, lds_u8* fr, int kt) __attribute__((always_inline)) {
          const int kl = min(kt + 3, nkd - 1);
          rd(cur, 1, gq);
          issue_half_a(fr, kl, 0, 2);
          mf(f);
          dsched<10, 4, 2>();
          rd(cur, 2, f);
          issue_half_a(fr, kl, 2, 4);
          mf(gq);
          dsched<10, 4, 2>();
          rd(cur, 3, gq);
          issue_half_a(fr, kl, 4, 6);
          mf(f);
          dsched<10, 4, 2>();
          __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
          wait_vm<14>();
          dbar();
          issue_half_a(fr, kl, 6, 8);
          rd(nxt, 0, f);
          mf(gq);
          dsched<10, 4, 2>();
        };
        rd(st0, 0, f);
        for (int kt = 0; kt < nkd; kt += 4) {
          dslab(st0, st1, st3, kt);
          dslab(st1, st2, st0, kt + 1);
          dslab(st2, st3, st1, kt + 2);
          dslab(st3, st0, st2, kt + 3);
        }
      } else {
        bf16x8 fa[2], fb[4], ga[2], gb[4];
        auto rd = [&](const lds_u8* buf, int kk, bf16x8 (&xa)[2], bf16x8 (&xb)[4]) __attribute__((always_inline)) {
#pragma unroll
          for (int i = 0; i < 2; ++i)
            xa[i] = *reinterpret_cast<const lds_bf16x8*>(buf + offOA + slot_kk[kk] + i * 32 * kRowBytes);
#pragma unroll
          for (int j = 0; j < 4; ++j)
            xb[j] = *reinterpret_cast<const lds_bf16x8*>(buf + offOB + slot_kk[kk] + j * 32 * kRowBytes);
        };
        auto mf = [&](const bf16x8 (&xa)[2], const bf16x8 (&xb)[4]) __attribute__((always_inline)) {
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) dmfma(xa[i], xb[j], dacc[4 * i + j]);
        };
        auto dslab = [&](const lds_u8* cur, const lds_u8* nxt, lds_u8* fr, int kt) __attribute__((always_inline)) {
          const int kl = min(kt + 3, nkd - 1);
          rd(cur, 1, ga, gb);
          issue_half_a(fr, kl, 0, 2);
          mf(fa, fb);
          dsched<8, 6, 2>();
          rd(cur, 2, fa, fb);
          issue_half_a(fr, kl, 2, 4);
          mf(ga, gb);
          dsched<8, 6, 2>();
          rd(cur, 3, ga, gb);
          issue_half_a(fr, kl, 4, 6);
          mf(fa, fb);
          dsched<8, 6, 2>();
          __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
          wait_vm<14>();
          dbar();
          issue_half_a(fr, kl, 6, 8);
          rd(nxt, 0, fa, fb);
          mf(ga, gb);
          dsched<8, 6, 2>();
        };
        rd(st0, 0, fa, fb);
        for (int kt = 0; kt < nkd; kt += 4) {
          dslab(st0, st1, st3, kt);
          dslab(st1, st2, st0, kt + 1);
          dslab(st2, st3, st1, kt + 2);
          dslab(st3, st0, st2, kt + 3);
        }
      }
      wait_vm<0>();
      __syncthreads();
      const int out_row0 = rowB0, out_col0 = rowA0, ldo = g.ldc;
      float s = 1.f;
      if (g.scale_kind != 0) s = g.fold[2 * mat + (g.scale_kind - 1)];
      const float ae = g.alpha_e * s, aa = g.alpha_acc * s, ad = g.alpha_diag * s;
      if (kHasE) stage_e(out_row0, out_col0);
      // block with A-side rows RA.. and B-side rows RB..: lane holds OUT[RB + lane%32][RA + 8 (v/4) + 4h + v%4]
      // Off-diagonal 32 x 32 blocks are also written transposed (OUT[c][r] = OUT[r][c]) with 2-byte
      // stores; the 8 diagonal 32 x 32 blocks keep both of their triangles as the matrix cores
      // form them, as in the general path.
      typedef __attribute__((address_space(3))) uint16_t lds_u16;
      auto emit = [&](const floatx16& a, int RA, int RB, auto out16_tag) __attribute__((always_inline)) {
        constexpr bool kOut16 = decltype(out16_tag)::value;
        const int r = RB + (lane & 31);
        lds_u8* dst = stage_of(r >> 6);
        u32x2 e[4];
        if (kHasE) {
#pragma unroll
          for (int vq = 0; vq < 4; ++vq)
            e[vq] = *reinterpret_cast<const lds_u32x2*>(dst + stage_byte(r, RA + 8 * vq + 4 * h));
        }
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) {
          const int c = RA + 8 * vq + 4 * h;
          float o[4];
#pragma unroll
          for (int qq = 0; qq < 4; ++qq) o[qq] = aa * a[4 * vq + qq];
          if (kHasE) {
            auto up = [](uint32_t x) { return kF16 ? f16_to_f32(x) : bf16_to_f32(x); };
            o[0] = fmaf(ae, up(e[vq].x & 0xffffu), o[0]);
            o[1] = fmaf(ae, up(e[vq].x >> 16), o[1]);
            o[2] = fmaf(ae, up(e[vq].y & 0xffffu), o[2]);
            o[3] = fmaf(ae, up(e[vq].y >> 16), o[3]);
          }
#pragma unroll
          for (int qq = 0; qq < 4; ++qq) o[qq] += (r == c + qq) ? ad : 0.f;
          u32x2 pk;
          pk.x = kOut16 ? pack_f16x2(o[0], o[1]) : pack_bf16x2(o[0], o[1]);
          pk.y = kOut16 ? pack_f16x2(o[2], o[3]) : pack_bf16x2(o[2], o[3]);
          *reinterpret_cast<lds_u32x2*>(dst + stage_byte(r, c)) = pk;
          if (RA != RB) {
            const uint32_t hv[4] = {pk.x & 0xffffu, pk.x >> 16, pk.y & 0xffffu, pk.y >> 16};
#pragma unroll
            for (int qq = 0; qq < 4; ++qq)
              *reinterpret_cast<lds_u16*>(stage_of((c + qq) >> 6) + stage_byte(c + qq, r)) = static_cast<uint16_t>(hv[qq]);
          }
        }
      };
      auto emit_all = [&](auto out16_tag) __attribute__((always_inline)) {
        if (roleD) {
          int n = 0;
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = i; j < 4; ++j) emit(dacc[n++], 128 * q + 32 * i, 128 * q + 32 * j, out16_tag);
        } else {
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) emit(dacc[4 * i + j], 64 * q + 32 * i, 128 + 32 * j, out16_tag);
        }
      };
      if (g.out_f16)
        emit_all(std::true_type{});
      else
        emit_all(std::false_type{});
      __syncthreads();
      // whole-row stores of OUT, as for the other tiles
      uint16_t* __restrict__ Cd = g.c + mat * g.stride_c;
#pragma unroll
      for (int qs = 0; qs < 4; ++qs) {
        const lds_u8* src = stage_of(qs);
#pragma unroll
        for (int it = 0; it < 8; ++it) {
          const int idx = it * 256 + t;
          const int rr = idx >> 5, p = idx & 31;
          const u32x4 v = *reinterpret_cast<const lds_u32x4*>(src + rr * 512 + 16 * p);
          const int r = 64 * qs + rr;
          const int c = p ^ (r & 31);
          *reinterpret_cast<u32x4*>(Cd + static_cast<int64_t>(out_row0 + r) * ldo + out_col0 + 8 * c) = v;
        }
      }
    }
    return;
  }
  floatx16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  auto load_frags = [&](const lds_u8* abuf, const lds_u8* bbuf, int kk, bf16x8 (&af)[4], bf16x8 (&bfr)[4]) __attribute__((always_inline)) {
    const int oa = offA + slot_kk[kk];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const lds_bf16x8*>(abuf + oa + i * 32 * kRowBytes);
    if (kNN) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const i16x4 lo =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(bbuf + (nn_off[j] + 8192 * kk)));
        const i16x4 hi =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(bbuf + (nn_off[j] + 2048 + 8192 * kk)));
        bfr[j] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
    } else {
      const int ob = offB_nt + slot_kk[kk];
#pragma unroll
      for (int j = 0; j < 4; ++j) bfr[j] = *reinterpret_cast<const lds_bf16x8*>(bbuf + ob + j * 32 * kRowBytes);
    }
  };

  auto mfma16 = [&](const bf16x8 (&af)[4], const bf16x8 (&bfr)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        // apply: operands swapped so each lane ends up with 4 consecutive output columns
        if constexpr (kNN)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
        else if constexpr (kF16)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(half8, af[i]),
                                                              __builtin_bit_cast(half8, bfr[j]), acc[i][j], 0, 0, 0);
        else
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
      }
  };

  // Software pipeline over slabs.  Operand A of slab s lives in buffer s % 2 of (st0, st1),
  // operand B in buffer s % 3 of (st2, st3, st4).  On entry to slab kt its first k step's
  // fragments are already in registers (fa).  Each later step's fragments are read under the
  // previous step's MFMAs.  Before the last step the wave waits for its own loads of slab
  // kt + 1 and meets the other waves: slab kt + 1 has fully landed and no wave reads slab
  // kt's buffers any more; slab kt + 1's first fragments are then read under the last step's
  // MFMAs.  Each k step also issues 4 of the 16 LDS-bound loads a slab needs per wave:
  //   step 0: the second half of operand A of slab kt + 1 (its buffer was freed a step ago),
  //   steps 1, 2: operand B of slab kt + 2, into the B buffer slab kt - 1 used,
  //   step 3 (after the barrier): the first half of operand A of slab kt + 2, into slab kt's.
  // At the barrier only operand B of slab kt + 2 may still be in flight (the waits count
  // loads in issue order).  An LDS-bound load can hold up the wave's issue while misses are
  // outstanding, so the loads go out evenly, at most one per 4 MFMAs (measured on the apply
  // product: two bursts instead of one 3% faster, spaced within the step 2% more, four even
  // parts another 2-3%); operand B's extra slab of lead time is what makes that possible.
  const int nk = g.K / BK;
  bf16x8 fa[4], fb[4], ga[4], gb[4];
  auto bar = []() __attribute__((always_inline)) {
    // A bare barrier: __syncthreads() would also wait for the newer slabs' loads.  The
    // empty asm statements keep the compiler from moving memory accesses across it.
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  constexpr int kReads = kNN ? 12 : 8;  // LDS read instructions per k step
  // ac, an: A buffers of slabs kt, kt + 1; bc, bn: B buffers of slabs kt, kt + 1; bp: the
  // B buffer of slab kt - 1, which receives slab kt + 2.  Past the end the loads are harmless
  // reloads of the last slab.
  auto slab = [&](lds_u8* ac, lds_u8* an, const lds_u8* bc, const lds_u8* bn, lds_u8* bp, int kt) __attribute__((always_inline)) {
    load_frags(ac, bc, 1, ga, gb);
    issue_half_a(an, min(kt + 1, nk - 1), 4, 8);  // second half of A of slab kt + 1
    mfma16(fa, fb);
    sched_step<kReads, 4>();
    load_frags(ac, bc, 2, fa, fb);
    issue_half_b(bp, min(kt + 2, nk - 1), 0, 4);  // B of slab kt + 2, first half
    mfma16(ga, gb);
    sched_step<kReads, 4>();
    load_frags(ac, bc, 3, ga, gb);
    issue_half_b(bp, min(kt + 2, nk - 1), 4, 8);  // second half
    mfma16(fa, fb);
    sched_step<kReads, 4>();
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave is done reading slab kt
    wait_vm<kDma / 2>();                 // all but operand B of slab kt + 2 have landed
    bar();
    issue_half_a(ac, min(kt + 2, nk - 1), 0, 4);  // first half of A of slab kt + 2
    load_frags(an, bn, 0, fa, fb);
    mfma16(ga, gb);
    sched_step<kReads, 4>();
  };

  // ---- main loop: every buffer is addressed statically.  The buffers repeat every 6 slabs
  // (2 A, 3 B), so the loop runs 6 slabs per trip; K is a multiple of 256 (zero padding),
  // so the slab count is a multiple of 4 and the tail is 0, 2 or 4 slabs.
  issue_half_a(st0, 0);
  issue_half_b(st2, 0);
  issue_half_b(st3, 1);
  issue_half_a(st1, 1, 0, 4);  // its second half goes out under slab 0's first step
  wait_vm<12>();               // slab 0 has landed
  bar();
  load_frags(st0, st2, 0, fa, fb);
  int kt = 0;
  for (; kt + 6 <= nk; kt += 6) {
    slab(st0, st1, st2, st3, st4, kt);
    slab(st1, st0, st3, st4, st2, kt + 1);
    slab(st0, st1, st4, st2, st3, kt + 2);
    slab(st1, st0, st2, st3, st4, kt + 3);
    slab(st0, st1, st3, st4, st2, kt + 4);
    slab(st1, st0, st4, st2, st3, kt + 5);
  }
  if (kt + 2 <= nk) {
    slab(st0, st1, st2, st3, st4, kt);
    slab(st1, st0, st3, st4, st2, kt + 1);
    kt += 2;
  }
  if (kt + 2 <= nk) {
    slab(st0, st1, st4, st2, st3, kt);
    slab(st1, st0, st2, st3, st4, kt + 1);
  }
  wait_vm<0>();
  __syncthreads();
  // ---- epilogue.  OUT is the 256 x 256 tile written with whole-row stores:
  //   apply:     OUT = C(ti, tj); lane holds OUT[128 wm + 32 i + lane%32][128 wn + 32 j + 8 (v/4) + 4 (lane/32) + v%4]
  //   Gram/poly: OUT = C(tj, ti) = C(ti, tj)^T; lane holds OUT[128 wn + 32 j + lane%32][128 wm + 32 i + ...]
  // OUT row r is staged in ring buffer r / 64 (st0..st3).
  const int out_row0 = kNN ? rowA0 : rowB0;
  const int out_col0 = kNN ? rowB0 : rowA0;
  float s = 1.f;
  if (g.scale_kind != 0) s = g.fold[2 * mat + (g.scale_kind - 1)];
  const float ae = g.alpha_e * s, aa = g.alpha_acc * s;
  const float ad = (kSym && ti == tj) ? g.alpha_diag * s : 0.f;  // diagonal tiles only
  const int own_row = kNN ? wm : wn;  // 128-row half holding this wave's OUT rows
  const int own_col = kNN ? wn : wm;  // 128-column half holding this wave's OUT columns
  const int ldo = g.ldc;

  if (kHasE) stage_e(out_row0, out_col0);

  // combine: each lane owns 4 consecutive OUT columns per (i, j, v/4).  Block by block
  // (fenced against the scheduler, which otherwise hoists every product at once and runs out
  // of registers), with the staged E values of the next block read while this one is
  // computed.  All staged E reads come before any staged write.
  u32x2 packed[4][4][4];
  auto e_read = [&](int i, int j, u32x2 (&e)[4]) __attribute__((always_inline)) {
    const int r = 128 * own_row + 32 * (kNN ? i : j) + (lane & 31);
    const lds_u8* src = stage_of(2 * own_row + ((kNN ? i : j) >> 1));
#pragma unroll
    for (int vq = 0; vq < 4; ++vq) {
      const int c = 128 * own_col + 32 * (kNN ? j : i) + 8 * vq + 4 * h;
      e[vq] = *reinterpret_cast<const lds_u32x2*>(src + stage_byte(r, c));
    }
  };
  // The output format is uniform over the workgroup: one copy of the loop per format.
  auto combine = [&](auto out16_tag) __attribute__((always_inline)) {
    constexpr bool kOut16 = decltype(out16_tag)::value;
    u32x2 ecur[4], enext[4];
    if (kHasE) e_read(0, 0, ecur);
#pragma unroll
    for (int b = 0; b < 16; ++b) {
      const int i = b >> 2, j = b & 3;
      if (kHasE && b < 15) e_read((b + 1) >> 2, (b + 1) & 3, enext);
      if (kHasE) __builtin_amdgcn_sched_barrier(0);
      const int r = 128 * own_row + 32 * (kNN ? i : j) + (lane & 31);
#pragma unroll
      for (int vq = 0; vq < 4; ++vq) {
        const int c = 128 * own_col + 32 * (kNN ? j : i) + 8 * vq + 4 * h;
        float o[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = aa * acc[i][j][4 * vq + q];
        if (kHasE) {
          const u32x2 e = ecur[vq];
          auto up = [](uint32_t x) { return kF16 ? f16_to_f32(x) : bf16_to_f32(x); };  // E has the operands' format
          o[0] = fmaf(ae, up(e.x & 0xffffu), o[0]);
          o[1] = fmaf(ae, up(e.x >> 16), o[1]);
          o[2] = fmaf(ae, up(e.y & 0xffffu), o[2]);
          o[3] = fmaf(ae, up(e.y >> 16), o[3]);
        }
        if (kSym) {
          // OUT is symmetric here, so OUT[r][c + q] is on the diagonal when r == c + q
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] += (r == c + q) ? ad : 0.f;
        }
        packed[i][j][vq].x = kOut16 ? pack_f16x2(o[0], o[1]) : pack_bf16x2(o[0], o[1]);
        packed[i][j][vq].y = kOut16 ? pack_f16x2(o[2], o[3]) : pack_bf16x2(o[2], o[3]);
      }
      if (kHasE) {
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) ecur[vq] = enext[vq];
      }
    }
  };
  if (kSym && g.out_f16)  // the X product always writes bf16
    combine(std::true_type{});
  else
    combine(std::false_type{});
  // x0^2 + x1^2 + acc for a packed bf16 pair (v_dot2: the bf16 products are exact in fp32)
  auto sq2 = [](uint32_t x, float acc) __attribute__((always_inline)) {
    const bf16x2 v = __builtin_bit_cast(bf16x2, x);
    return __builtin_amdgcn_fdot2_f32_bf16(v, v, acc, false);
  };
  // apply with fused sums: per-lane row partials of the bf16 output straight from the packed
  // registers (each lane holds 64 values of each of its 4 rows), one slot per (wn, h) half of
  // the row, in the ring's fifth buffer behind the column partials
  lds_f32* const rowpart = (lds_f32*)(st4_ + 8192);
  if (kNN && g.rpart) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float rs = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int vq = 0; vq < 4; ++vq) rs = sq2(packed[i][j][vq].y, sq2(packed[i][j][vq].x, rs));
      rowpart[256 * (2 * wn + h) + 128 * wm + 32 * i + (lane & 31)] = rs;
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = 128 * own_row + 32 * (kNN ? i : j) + (lane & 31);
      lds_u8* dst = stage_of(2 * own_row + ((kNN ? i : j) >> 1));
#pragma unroll
      for (int vq = 0; vq < 4; ++vq) {
        const int c = 128 * own_col + 32 * (kNN ? j : i) + 8 * vq + 4 * h;
        *reinterpret_cast<lds_u32x2*>(dst + stage_byte(r, c)) = packed[i][j][vq];
      }
    }
  __syncthreads();

  if (kSym && ti == tj && g.symmetrize) {
    // A product of two different commuting symmetric factors (P A, P T, P Q) is symmetric only
    // up to rounding, and the next product reads the stored matrix as its own transpose.  The
    // off-diagonal tiles store the upper block triangle of the product and its mirror; a
    // diagonal tile keeps the same triangle (OUT[r][c] with r >= c, the product's upper
    // triangle) and copies it onto the other half: OUT[R][C] = OUT[C][R] for R < C.  Transpose
    // reads as in the mirrored store below give each lane OUT[r0 .. r0 + 7][R]; it writes the
    // entries of row R in columns r0 .. r0 + 7 above the diagonal.  Only entries below the
    // diagonal are used and only entries above it are written, so no read waits for a write.
    const int jq16 = lane & 15, g4 = lane >> 4;
#pragma unroll 2
    for (int it = 0; it < 32; ++it) {
      const int blk = it * 4 + wave;
      const int cb = blk & 15, rb = blk >> 4;
      const int r0 = 32 * rb + 8 * g4;  // source rows = target columns r0 .. r0 + 7
      const int R = 16 * cb + jq16;     // target row = source column
      u32x4 tv;
      const lds_u8* src = stage_of(r0 >> 6);
#pragma unroll
      for (int t4 = 0; t4 < 2; ++t4) {
        const int r = r0 + 4 * t4 + (jq16 >> 2);
        const int c = 16 * cb + 4 * (jq16 & 3);
        const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(src + stage_byte(r, c)));
        const u32x2 w = __builtin_bit_cast(u32x2, v);
        tv[2 * t4] = w.x;
        tv[2 * t4 + 1] = w.y;
      }
      if (R < r0 + 7) {  // some column r0 + e lies above the diagonal of row R
        lds_u8* dst = stage_of(R >> 6) + stage_byte(R, r0);
        if (R >= r0) {   // the chunk straddles the diagonal: keep columns <= R
          const u32x4 cur = *reinterpret_cast<const lds_u32x4*>(dst);
#pragma unroll
          for (int e2 = 0; e2 < 4; ++e2) {
            const uint32_t lo = (r0 + 2 * e2 > R) ? (tv[e2] & 0xffffu) : (cur[e2] & 0xffffu);
            const uint32_t hi = (r0 + 2 * e2 + 1 > R) ? (tv[e2] & 0xffff0000u) : (cur[e2] & 0xffff0000u);
            tv[e2] = lo | hi;
          }
        }
        *reinterpret_cast<lds_u32x4*>(dst) = tv;
      }
    }
    __syncthreads();
  }

  if (kNN && g.rpart) {
    // Row and column sums of squares of this bf16 output tile, in a fixed order.  Rows: the four
    // register partials of each row.  Columns: wave w sums its own stage (rows 64 w .. 64 w + 63)
    // with transpose reads, lane q of 16-lane group g4 taking 4 consecutive rows of column
    // 16 (4 m + g4) + q per read, and the four waves meet in LDS.
    const int jq16 = lane & 15, g4 = lane >> 4;
    const lds_u8* sw = stage_of(wave);
    float cs[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int m = 0; m < 4; ++m) {
#pragma unroll 4
      for (int rb = 0; rb < 16; ++rb) {
        const int r = 64 * wave + 4 * rb + (jq16 >> 2);
        const int c = 16 * (4 * m + g4) + 4 * (jq16 & 3);
        const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(sw + stage_byte(r, c)));
        const u32x2 w2 = __builtin_bit_cast(u32x2, v);
        cs[m] = sq2(w2.y, sq2(w2.x, cs[m]));
      }
    }
#pragma unroll
    for (int m = 0; m < 4; ++m) colsum[256 * wave + 16 * (4 * m + g4) + jq16] = cs[m];
    __syncthreads();
    const float csum = (colsum[t] + colsum[256 + t]) + (colsum[512 + t] + colsum[768 + t]);
    const float rsum = (rowpart[t] + rowpart[256 + t]) + (rowpart[512 + t] + rowpart[768 + t]);
    g.rpart[mat * g.stride_rpart + static_cast<int64_t>(tj) * (g.tiles_m * 256) + rowA0 + t] = rsum;
    g.cpart[mat * g.stride_cpart + static_cast<int64_t>(ti) * g.ldc + rowB0 + t] = csum;
  }

  // whole-row stores of OUT: each wave instruction writes 2 full rows
  uint16_t* __restrict__ C = g.c + mat * g.stride_c;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const lds_u8* src = stage_of(q);
#pragma unroll
    for (int it = 0; it < 8; ++it) {
      const int idx = it * 256 + t;
      const int rr = idx >> 5, p = idx & 31;  // row within the stage, slot
      const u32x4 v = *reinterpret_cast<const lds_u32x4*>(src + rr * 512 + 16 * p);
      const int r = 64 * q + rr;
      const int c = p ^ (r & 31);
      *reinterpret_cast<u32x4*>(C + static_cast<int64_t>(out_row0 + r) * ldo + out_col0 + 8 * c) = v;
    }
  }

  if (kSym && ti != tj) {
    // Mirrored tile C(ti, tj) = OUT^T.  Transpose reads give each lane 4 consecutive OUT rows
    // of one OUT column (= 4 consecutive columns of one C(ti, tj) row); two reads make 16
    // bytes.  Per trip a 16-lane group covers 16 OUT columns x 8 OUT rows and the 4 groups
    // of a wave take consecutive 8-row blocks, so a wave writes 64 contiguous bytes in each
    // of 16 rows.
    const int jq16 = lane & 15, g4 = lane >> 4;
#pragma unroll 2
    for (int it = 0; it < 32; ++it) {
      const int blk = it * 4 + wave;  // 128 blocks: 16 column blocks x 8 row blocks
      const int cb = blk & 15, rb = blk >> 4;
      const int r0 = 32 * rb + 8 * g4;  // OUT rows r0 .. r0 + 7 (one stage)
      const int c0 = 16 * cb;
      const lds_u8* src = stage_of(r0 >> 6);
      u32x4 out;
#pragma unroll
      for (int t4 = 0; t4 < 2; ++t4) {
        const int r = r0 + 4 * t4 + (jq16 >> 2);
        const int c = c0 + 4 * (jq16 & 3);
        const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(src + stage_byte(r, c)));
        const u32x2 w = __builtin_bit_cast(u32x2, v);
        out[2 * t4] = w.x;
        out[2 * t4 + 1] = w.y;
      }
      // lane holds OUT[r0 .. r0 + 7][c0 + jq16] = C(ti, tj)[c0 + jq16][r0 .. r0 + 7]
      *reinterpret_cast<u32x4*>(C + static_cast<int64_t>(rowA0 + c0 + jq16) * ldo + rowB0 + r0) = out;
    }
  }
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, int mode, int f16, hipStream_t st) {
  const int blocks = a.tile_start[a.count];
  if (mode == 0 && f16) hipLaunchKernelGGL((k_ns_gemm<0, true>), dim3(blocks), dim3(256), 0, st, a);
  else if (mode == 0) hipLaunchKernelGGL((k_ns_gemm<0, false>), dim3(blocks), dim3(256), 0, st, a);
  else if (mode == 1 && f16) hipLaunchKernelGGL((k_ns_gemm<1, true>), dim3(blocks), dim3(256), 0, st, a);
  else if (mode == 1) hipLaunchKernelGGL((k_ns_gemm<1, false>), dim3(blocks), dim3(256), 0, st, a);
  else if (!f16) hipLaunchKernelGGL((k_ns_gemm<2, false>), dim3(blocks), dim3(256), 0, st, a);
  else return hipErrorInvalidValue;  // the X product's operands are bf16
  return hipGetLastError();
}

}  // namespace meq
