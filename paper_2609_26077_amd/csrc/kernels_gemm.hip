// fp8 sub-products with fp32 accumulation and the fused W-combine.
//
// A workgroup owns a BM x BN tile of the m' x n' grid and one outer term
// r_o; it runs the K loop of each of the R inner terms r = r_o R + r_i in turn
// (one flattened (term, k-step) pipeline), and after each term adds
// w[r_i][q] * P_r into four quadrant accumulators q = 2k + i held in
// registers.  At depth 1 the quadrants are the four blocks of C and are
// written once; at depth >= 2 they are the inner-level partial products
// Q[r_o][q], stored [batch][m'][T_o][4][n'] (the T_o 4 partials of one row
// adjacent, so that the outer combine streams one region of HBM), combined
// over r_o by outer_combine_kernel.
//
// MX path (power-of-two scales, block 32 or 128): v_mfma_scale_f32_32x32x64_f8f6f4
// applies the E8M0 block scales in hardware.  Operand layout of that
// instruction (measured): lane (r, h = lane/32) holds row r, contracted bytes
// [16h, 16h+16) in VGPRs 0-3 and [32+16h, +16) in VGPRs 4-7; VGPRs 0-3 of all
// lanes form the instruction's first 32-element scale block, VGPRs 4-7 the
// second, and lane r + 32 kb supplies the scale of block kb of row r.
//
// The fp8 dot product of those instructions aligns each group of eight
// products to the group's largest and keeps 13 bits below it (measured:
// 1 + 2^-13 survives, 1 + 2^-14 returns 1; groups are summed at fp32 grade).
//
// Exact-dot paths (FMM_FLAG_EXACT_DOT, fp32 scales or block 16): the codes are
// converted exactly to bf16 and fed to v_mfma_f32_32x32x16_bf16 (lane (r, h)
// holds row r, elements [8h, 8h+8); 23 retained bits).  With E8M0 scales on
// the tile layout (gemm_dq8_kernel) each code's conversion applies its block's
// power of two; otherwise (gemm_promote_kernel) the codes convert at scale 1,
// each block's products are summed in a temporary and scaled by sA * sB in
// fp32 -- in both, the products of the dequantized operands accumulated in fp32.
//
// Output layout of the 32x32 instructions: lane l, register j holds
// column l % 32, row 8 (j / 4) + 4 (l / 32) + j % 4.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "device.h"
#include "internal.h"
#include "lds_dma.h"

namespace fmm {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

// eight e4m3 codes (little-endian in two words) -> eight bf16, exactly
__device__ __forceinline__ v8bf e4m3x8_to_bf16(uint2 w) {
  const v2bf a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w.x, 1.0f, false);
  const v2bf b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w.x, 1.0f, true);
  const v2bf c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w.y, 1.0f, false);
  const v2bf d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w.y, 1.0f, true);
  v8bf r;
  r[0] = a[0]; r[1] = a[1]; r[2] = b[0]; r[3] = b[1];
  r[4] = c[0]; r[5] = c[1]; r[6] = d[0]; r[7] = d[1];
  return r;
}

constexpr int BM = 128, BN = 128, BK = 128;
constexpr int kThreads = 256;

struct GemmArgs {
  const uint8_t *xa, *xb;        // codes, [batch][T][rows][kp]
  const uint8_t *sa, *sb;        // scales, [batch][T][rows][kblocks]
  float *out;                    // C (depth 1) or partial products (depth >= 2)
  int64_t mp, np, kp, kblocks, T, To, M, N;
  int R, block, depth, tiles_n;
  const float *w;                // R x 4 inner decoder weights (device)
};

// LDS tile: 128 rows x 128 bytes; 16-byte chunk c of row r sits at chunk
// c ^ (r & 7) ^ ((r >> 3) & 1).  A 16-byte read is served in groups of 16
// lanes over 64 four-byte banks; the fragment rows r and r + 8 of one group
// would share banks under c ^ (r & 7) alone.
__device__ __forceinline__ int swz(int row, int chunk) {
  return row * BK + 16 * (chunk ^ (row & 7) ^ ((row >> 3) & 1));
}

// Global -> registers for one (term, k-step): each thread moves four 16-byte chunks
// of A and four of B.  Rows past the end and chunks past kp read as zero.
struct Stage {
  uint4 a[4], b[4];
};

__device__ __forceinline__ void load_stage(const GemmArgs &g, int64_t bt, int64_t r, int64_t k0,
                                           int64_t pm0, int64_t pn0, Stage &s) {
  const int t = threadIdx.x;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c = t + kThreads * j;
    const int row = c >> 3, ch = c & 7;
    const int64_t k = k0 + 16 * ch;
    const int64_t pa = pm0 + row, pb = pn0 + row;
    uint4 za = make_uint4(0, 0, 0, 0), zb = make_uint4(0, 0, 0, 0);
    if (pa < g.mp && k < g.kp)
      za = *reinterpret_cast<const uint4 *>(g.xa + ((bt * g.T + r) * g.mp + pa) * g.kp + k);
    if (pb < g.np && k < g.kp)
      zb = *reinterpret_cast<const uint4 *>(g.xb + ((bt * g.T + r) * g.np + pb) * g.kp + k);
    s.a[j] = za;
    s.b[j] = zb;
  }
}

__device__ __forceinline__ void store_stage(uint8_t *la, uint8_t *lb, const Stage &s) {
  const int t = threadIdx.x;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c = t + kThreads * j;
    const int row = c >> 3, ch = c & 7;
    *reinterpret_cast<uint4 *>(la + swz(row, ch)) = s.a[j];
    *reinterpret_cast<uint4 *>(lb + swz(row, ch)) = s.b[j];
  }
}

// E8M0 scale bytes a lane needs for one k-step: [tile i][substep s] for A, [j][s] for B.
struct MxScales {
  int a[2][2], b[2][2];
};

__device__ __forceinline__ int scale_byte(const uint8_t *base, int64_t rowid_valid, int64_t rowid,
                                          int64_t kblocks, int64_t k, int64_t kp, int block) {
  if (!rowid_valid || k >= kp) return 127;  // padding: codes are zero, scale 1.0
  return base[rowid * kblocks + k / block];
}

__device__ __forceinline__ void load_mx_scales(const GemmArgs &g, int64_t bt, int64_t r, int64_t k0,
                                               int64_t rowa0, int64_t rowb0, MxScales &sc) {
  const int lane = threadIdx.x & 63;
  const int r32 = lane & 31, h = lane >> 5;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int64_t k = k0 + 64 * s + 32 * h;
      const int64_t pa = rowa0 + 32 * i + r32;
      const int64_t pb = rowb0 + 32 * i + r32;
      sc.a[i][s] = scale_byte(g.sa, pa < g.mp, (bt * g.T + r) * g.mp + pa, g.kblocks, k, g.kp, g.block);
      sc.b[i][s] = scale_byte(g.sb, pb < g.np, (bt * g.T + r) * g.np + pb, g.kblocks, k, g.kp, g.block);
    }
}

__device__ __forceinline__ v8i frag_mx(const uint8_t *lt, int row, int s, int h) {
  const uint4 lo = *reinterpret_cast<const uint4 *>(lt + swz(row, 4 * s + h));
  const uint4 hi = *reinterpret_cast<const uint4 *>(lt + swz(row, 4 * s + 2 + h));
  v8i f;
  f[0] = (int)lo.x; f[1] = (int)lo.y; f[2] = (int)lo.z; f[3] = (int)lo.w;
  f[4] = (int)hi.x; f[5] = (int)hi.y; f[6] = (int)hi.z; f[7] = (int)hi.w;
  return f;
}

__device__ __forceinline__ void store_tile(const GemmArgs &g, int64_t bt, int64_t ro, int q,
                                           int64_t p0, int64_t c0, const v16f &v) {
  // p0/c0: first row/column of this 32x32 tile in the m' x n' grid
  const int lane = threadIdx.x & 63;
  const int64_t col = c0 + (lane & 31);
  if (col >= g.np) return;
  const int iq = q & 1, kq = q >> 1;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int64_t row = p0 + 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3);
    if (row < g.mp) {
      if (g.depth == 1) {
        g.out[bt * g.M * g.N + (iq * g.mp + row) * g.N + kq * g.np + col] = v[j];
      } else {
        g.out[(((bt * g.mp + row) * g.To + ro) * 4 + q) * g.np + col] = v[j];
      }
    }
  }
}

__global__ __launch_bounds__(kThreads, 1) void gemm_mx_kernel(GemmArgs g) {
  __shared__ uint4 lds_raw[2 * 2 * BM * BK / 16];
  uint8_t *lds = reinterpret_cast<uint8_t *>(lds_raw);
  const int t = threadIdx.x;
  const int wave = t >> 6, lane = t & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int r32 = lane & 31, h = lane >> 5;
  const int64_t tm = blockIdx.x / g.tiles_n, tn = blockIdx.x % g.tiles_n;
  const int64_t ro = blockIdx.y, bt = blockIdx.z;
  const int64_t pm0 = tm * BM, pn0 = tn * BN;
  const int64_t rowa0 = pm0 + wm * 64, rowb0 = pn0 + wn * 64;

  const int64_t nsteps = (g.kp + BK - 1) / BK;
  const int64_t total = (int64_t)g.R * nsteps;

  v16f acc[2][2];
  v16f quad[4][2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      acc[i][j] = (v16f){};
#pragma unroll
      for (int q = 0; q < 4; ++q) quad[q][i][j] = (v16f){};
    }

  Stage st;
  MxScales sc, sc_next;
  load_stage(g, bt, ro * g.R, 0, pm0, pn0, st);
  load_mx_scales(g, bt, ro * g.R, 0, rowa0, rowb0, sc);
  store_stage(lds, lds + BM * BK, st);
  __syncthreads();

  for (int64_t it = 0; it < total; ++it) {
    const int ri = (int)(it / nsteps);
    const int64_t ks = it % nsteps;
    const int buf = (int)(it & 1);
    const bool more = it + 1 < total;
    if (more) {
      const int64_t rn = ro * g.R + (it + 1) / nsteps;
      const int64_t kn = ((it + 1) % nsteps) * BK;
      load_stage(g, bt, rn, kn, pm0, pn0, st);
      load_mx_scales(g, bt, rn, kn, rowa0, rowb0, sc_next);
    }
    const uint8_t *la = lds + buf * 2 * BM * BK;
    const uint8_t *lb = la + BM * BK;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      v8i fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        fa[i] = frag_mx(la, wm * 64 + 32 * i + r32, s, h);
        fb[i] = frag_mx(lb, wn * 64 + 32 * i + r32, s, h);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
              fa[i], fb[j], acc[i][j], 0, 0, 0, sc.a[i][s], 0, sc.b[j][s]);
    }
    if (ks == nsteps - 1) {
      // end of term ri: quadrant q += w[ri][q] * P
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float wq = g.w[4 * ri + q];
        if (wq != 0.0f) {
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
              for (int e = 0; e < 16; ++e) quad[q][i][j][e] = __fmaf_rn(wq, acc[i][j][e], quad[q][i][j][e]);
        }
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = (v16f){};
    }
    if (more) {
      uint8_t *na = lds + (buf ^ 1) * 2 * BM * BK;
      store_stage(na, na + BM * BK, st);
      sc = sc_next;
    }
    __syncthreads();
  }

#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        store_tile(g, bt, ro, q, rowa0 + 32 * i, rowb0 + 32 * j, quad[q][i][j]);
}


// ---------------------------------------------------------------------------
// Fast MX path for tile-aligned shapes (m', n' and k' multiples of 128), whose
// codes and scales the encoder writes in the 128 x 128 tile layout.
//
// One workgroup of four waves owns a 128 x 128 tile of the m' x n' grid; each
// wave a 64 x 64 quarter as 2 x 2 MFMA tiles of 32 x 32.  The codes and E8M0
// scales of each 128-byte K step go from HBM straight into LDS
// (global_load_lds: no staging registers) through a four-slot ring; each wave
// issues exactly nine such transfers per step (four 1 KB of A codes, four of
// B codes, one 256 B of scales), all straight copies of the tile images, and
// waits for them with an explicit vmcnt.
// While the MFMAs of step s run on fragments already in registers, the
// fragments of step s + 1 are read from LDS into a second register set and the
// transfers of steps s + 2 and s + 3 are in flight.  LDS code rows are 128
// bytes; 16-byte chunk c of row r is stored at c ^ (r & 7) ^ ((r >> 3) & 1),
// which keeps every 16-lane group of a fragment read on distinct banks.
//
// The quadrant accumulators of the fused W-combine live in AGPRs for the
// whole kernel (the four 64 x 64 sets fill the 256 accumulation registers),
// leaving the architectural VGPRs to the MFMA accumulator, the two fragment
// sets and addressing; they are touched only through the helpers below, eight
// at a time at a term end.  The decoder weights are copied to LDS once, so the
// term-end combine never waits on vector memory (which would drain the
// transfer ring).
// ---------------------------------------------------------------------------
constexpr int FBK = 128;
constexpr int kSlot = 2 * BM * FBK + 2 * BM * 4;   // codes A, B + scale words A, B
constexpr int kSlots = 4;

using dma::copy16;
using dma::copy4;
using dma::wait_vmcnt;

__device__ __forceinline__ void agpr_zero(float &q) {
  asm volatile("v_accvgpr_write_b32 %0, 0" : "=a"(q));
}
__device__ __forceinline__ void agpr_fma(float &q, float w, float p) {
  float t;
  asm volatile(
      "v_accvgpr_read_b32 %0, %1\n\t"
      "v_fmac_f32_e32 %0, %2, %3\n\t"
      "v_accvgpr_write_b32 %1, %0"
      : "=&v"(t), "+a"(q)
      : "s"(w), "v"(p));
}
// eight of the above at once, on eight temporaries, so the reads, the
// multiply-adds and the writes each issue back to back
__device__ __forceinline__ void agpr_fma8(float *q, float w, const float *p) {
  float t0, t1, t2, t3, t4, t5, t6, t7;
  asm volatile(
      "v_accvgpr_read_b32 %0, %8\n\tv_accvgpr_read_b32 %1, %9\n\t"
      "v_accvgpr_read_b32 %2, %10\n\tv_accvgpr_read_b32 %3, %11\n\t"
      "v_accvgpr_read_b32 %4, %12\n\tv_accvgpr_read_b32 %5, %13\n\t"
      "v_accvgpr_read_b32 %6, %14\n\tv_accvgpr_read_b32 %7, %15\n\t"
      "v_fmac_f32_e32 %0, %16, %17\n\tv_fmac_f32_e32 %1, %16, %18\n\t"
      "v_fmac_f32_e32 %2, %16, %19\n\tv_fmac_f32_e32 %3, %16, %20\n\t"
      "v_fmac_f32_e32 %4, %16, %21\n\tv_fmac_f32_e32 %5, %16, %22\n\t"
      "v_fmac_f32_e32 %6, %16, %23\n\tv_fmac_f32_e32 %7, %16, %24\n\t"
      "v_accvgpr_write_b32 %8, %0\n\tv_accvgpr_write_b32 %9, %1\n\t"
      "v_accvgpr_write_b32 %10, %2\n\tv_accvgpr_write_b32 %11, %3\n\t"
      "v_accvgpr_write_b32 %12, %4\n\tv_accvgpr_write_b32 %13, %5\n\t"
      "v_accvgpr_write_b32 %14, %6\n\tv_accvgpr_write_b32 %15, %7"
      : "=&v"(t0), "=&v"(t1), "=&v"(t2), "=&v"(t3), "=&v"(t4), "=&v"(t5), "=&v"(t6), "=&v"(t7),
        "+a"(q[0]), "+a"(q[1]), "+a"(q[2]), "+a"(q[3]), "+a"(q[4]), "+a"(q[5]), "+a"(q[6]), "+a"(q[7])
      : "s"(w), "v"(p[0]), "v"(p[1]), "v"(p[2]), "v"(p[3]), "v"(p[4]), "v"(p[5]), "v"(p[6]), "v"(p[7]));
}
__device__ __forceinline__ float agpr_read(const float &q) {
  float v;
  asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v) : "a"(q));
  return v;
}

// XCD-aware tile order: workgroups are dispatched round-robin over the eight
// XCDs, so consecutive workgroups of one XCD (bid, bid + 8, ...) are given a
// contiguous range of tiles, walked in groups of eight tile-rows so that the
// workgroups resident on an XCD share A rows and B columns in its L2.
__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int &tm, int &tn) {
  const int ntiles = tiles_m * tiles_n;
  int id = bid;
  if ((ntiles & 7) == 0) id = (bid & 7) * (ntiles >> 3) + (bid >> 3);
  constexpr int GM = 8;
  const int per_group = GM * tiles_n;
  const int group = id / per_group;
  const int first_m = group * GM;
  const int gm = min(tiles_m - first_m, GM);
  const int in = id - group * per_group;
  tm = first_m + in % gm;
  tn = in / gm;
}

// The (tile, outer term, batch) item of this workgroup.  Grids whose tile
// count is not a multiple of eight (small batched products: 2 x 2 tiles of a
// 256 x 256 sub-product) would spread the tiles of one item over four XCDs,
// each fetching the item's codes into its own L2; there the linear dispatch
// index L (x fastest) is remapped, as for the large-tile kernel, so that XCD
// L mod 8 takes a contiguous range of items and all tiles of each (1024
// products of 512^3: 0.64 -> 0.54 ms).  Grids of fewer than 2048 workgroups
// (eight rounds of the 256 the chip holds) keep the plain order, which
// measured slightly faster there.
__device__ __forceinline__ void item_of(int tiles_m, int tiles_n, int &tm, int &tn, int64_t &ro, int64_t &bt) {
  const int ntiles = tiles_m * tiles_n;
  const int64_t total = (int64_t)ntiles * gridDim.y * gridDim.z;
  if ((ntiles & 7) == 0 || (total & 7) != 0 || total < 2048) {
    tile_of(blockIdx.x, tiles_m, tiles_n, tm, tn);
    ro = blockIdx.y;
    bt = blockIdx.z;
    return;
  }
  const int64_t L = blockIdx.x + (int64_t)ntiles * (blockIdx.y + (int64_t)gridDim.y * blockIdx.z);
  const int64_t id = (L & 7) * (total >> 3) + (L >> 3);
  const int64_t item = id / ntiles;
  tile_of((int)(id - item * ntiles), tiles_m, tiles_n, tm, tn);
  ro = item % gridDim.y;
  bt = item / gridDim.y;
}

// Operands of one K step for one wave: fragments [substep s][tile i] and,
// for each of its A and B row tiles, the E8M0 scale bytes of the lane's two
// blocks (byte s: substep s).
struct MxFrags {
  v8i a[2][2], b[2][2];
  int sa[2], sb[2];
};

// codes in dwords d, d + 1 of a fragment, times the power of two whose
// exponent field `s` carries, as eight bf16 (exact: the dequantized values)
__device__ __forceinline__ v8bf dequant8(const v8i &f, int d, float s) {
  const v2bf a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(f[d], s, false);
  const v2bf b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(f[d], s, true);
  const v2bf c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(f[d + 1], s, false);
  const v2bf e = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(f[d + 1], s, true);
  v8bf r;
  r[0] = a[0]; r[1] = a[1]; r[2] = b[0]; r[3] = b[1];
  r[4] = c[0]; r[5] = c[1]; r[6] = e[0]; r[7] = e[1];
  return r;
}

// A float whose exponent field is byte i of a scale record, as the scale
// operand of v_cvt_scalef32_pk_bf16_fp8, which reads the exponent field alone
// (its sign and mantissa bits, here parts of the neighbouring bytes, leave
// the result unchanged: every code at every exponent -48 .. 120 measured), so
// one shift places the byte
__device__ __forceinline__ float e8m0_at(int w, int i) {
  return __uint_as_float(i == 3 ? (uint32_t)w >> 1 : (uint32_t)w << (23 - 8 * i));
}

// The fp8 matrix cores with the E8M0 scales applied by the scaled MFMA.
template <int BS>
__global__ __launch_bounds__(kThreads, 1) void gemm_mx_fast_kernel(GemmArgs g, int tiles_m) {
  __shared__ uint4 lds_raw[kSlots * kSlot / 16];
  __shared__ float lds_w[4 * kMaxRank];
  uint8_t *lds = reinterpret_cast<uint8_t *>(lds_raw);
  const uint32_t lds_base = dma::lds_addr(lds_raw);
  const int t = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int lane = t & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int r32 = lane & 31, h = lane >> 5;
  int tm, tn;
  int64_t ro, bt;
  item_of(tiles_m, g.tiles_n, tm, tn, ro, bt);
  const int64_t pm0 = (int64_t)tm * BM, pn0 = (int64_t)tn * BN;
  const uint32_t kp = (uint32_t)g.kp, kblocks = (uint32_t)g.kblocks;
  const int nk = (int)(g.kp / FBK);
  const int total = g.R * nk;
  const int wrow_a = wm * 64, wrow_b = wn * 64;
  if (t == 0) {   // uniform loads of the zero-padded table; read only after the first barrier
#pragma unroll
    for (int i = 0; i < 4 * kMaxRank; ++i) lds_w[i] = g.w[i];
  }

  // Codes and scales arrive tiled (the 128-row x 128-byte tile image and 4
  // scale bytes per tile row and step), so every transfer is a straight copy:
  // lane l moves bytes 16 l .. 16 l + 15 (codes) or 4 l .. 4 l + 3 (scales).
  // Scales: waves 0/1 move A tile rows 64 w .., waves 2/3 B tile rows 64 (w - 2) ..
  const bool scale_is_b = wave >= 2;
  const int64_t kt = g.kp / FBK;                           // 128-byte steps per row tile

  auto issue = [&](int step) {
    const int ri = step / nk, ks = step - ri * nk;
    const int64_t r = ro * g.R + ri;
    const int64_t ta = ((bt * g.T + r) * (g.mp / BM) + tm) * kt + ks;   // tile index, A
    const int64_t tb = ((bt * g.T + r) * (g.np / BN) + tn) * kt + ks;
    const uint8_t *xa = g.xa + ta * (BM * FBK);
    const uint8_t *xb = g.xb + tb * (BN * FBK);
    const uint32_t m0 = lds_base + (uint32_t)(step & (kSlots - 1)) * kSlot;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int region = wave * 4 + j;                     // tile rows 8 region .. + 7
      copy16(16u * (uint32_t)lane, xa + region * 1024, m0 + region * 1024);
      copy16(16u * (uint32_t)lane, xb + region * 1024, m0 + BM * FBK + region * 1024);
    }
    const uint8_t *sbase = scale_is_b ? g.sb + tb * (BN * 4) : g.sa + ta * (BM * 4);
    copy4(4u * (uint32_t)lane + (wave & 1) * 256u, sbase,
          m0 + 2 * BM * FBK + (scale_is_b ? BM * 4 : 0) + (wave & 1) * 256);
  };

  // LDS -> registers for one step (slot step % 4; any step index reads in bounds).
  // Scale record of a row: blocks (0, 2, 1, 3) at block 32, so lane (r, h) reads
  // the 16-bit pair at byte 2h: byte 0 = block h (substep 0), byte 1 = block 2 + h.
  auto load = [&](int step, MxFrags &f) {
    const uint8_t *la = lds + (step & (kSlots - 1)) * kSlot;
    const uint8_t *lb = la + BM * FBK;
    const uint8_t *lsa = la + 2 * BM * FBK;
    const uint8_t *lsb = lsa + BM * 4;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      f.sa[i] = *reinterpret_cast<const uint16_t *>(lsa + 4 * (wrow_a + 32 * i + r32) + 2 * h);
      f.sb[i] = *reinterpret_cast<const uint16_t *>(lsb + 4 * (wrow_b + 32 * i + r32) + 2 * h);
    }
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        f.a[s][i] = frag_mx(la, wrow_a + 32 * i + r32, s, h);
        f.b[s][i] = frag_mx(lb, wrow_b + 32 * i + r32, s, h);
      }
  };

  v16f acc[2][2];
  float quad[4][2][2][16];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      acc[i][j] = (v16f){};
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < 16; ++e) agpr_zero(quad[q][i][j][e]);
    }

  // one step: wait for step + 1, start step + 3, read step + 1 into `nxt`
  // while the MFMAs of `cur` (step) run, and at the end of a term fold P_r
  // into the quadrants.  The scale bytes of `cur` are selected here, a step after
  // their words were read, so no MFMA waits on a scale read.
  auto body = [&](int step, MxFrags &cur, MxFrags &nxt) {
    if (step + 1 < total) {
      if (step + 2 < total) wait_vmcnt<9>(); else wait_vmcnt<0>();
      __syncthreads();
    }
    if (step + 3 < total) issue(step + 3);
    const int ks = step % nk;
    load(step + 1, nxt);
    {
#define FMM_MFMA_SIJ(S, I, J)                                                                      \
  acc[I][J] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(cur.a[S][I], cur.b[S][J], acc[I][J], 0, 0, \
                                                              S, cur.sa[I], S, cur.sb[J])
      FMM_MFMA_SIJ(0, 0, 0); FMM_MFMA_SIJ(0, 0, 1); FMM_MFMA_SIJ(0, 1, 0); FMM_MFMA_SIJ(0, 1, 1);
      FMM_MFMA_SIJ(1, 0, 0); FMM_MFMA_SIJ(1, 0, 1); FMM_MFMA_SIJ(1, 1, 0); FMM_MFMA_SIJ(1, 1, 1);
#undef FMM_MFMA_SIJ
      // MFMA and LDS reads alternate: 1 MFMA, then 3 reads (20 reads over 7 gaps)
#pragma unroll
      for (int k = 0; k < 6; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    }
    if (ks + 1 == nk) {
      const int ri = step / nk;
      // end of term ri: quadrant q += w[ri][q] * P
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float wq = __builtin_bit_cast(
            float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, lds_w[4 * ri + q])));
        if (wq != 0.0f) {
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
              for (int e = 0; e < 16; e += 8) {
                float pv[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) pv[u] = acc[i][j][e + u];
                agpr_fma8(&quad[q][i][j][e], wq, pv);
              }
        }
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = (v16f){};
    }
  };

  // prologue: steps 0, 1, 2 in flight, step 0 read into registers
  issue(0);
  if (total > 1) issue(1);
  if (total > 2) issue(2);
  if (total > 2) wait_vmcnt<18>(); else if (total > 1) wait_vmcnt<9>(); else wait_vmcnt<0>();
  __syncthreads();
  MxFrags f0, f1;
  load(0, f0);
  for (int step = 0; step < total; step += 2) {
    body(step, f0, f1);
    if (step + 1 < total) body(step + 1, f1, f0);
  }

#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        v16f v;
#pragma unroll
        for (int e = 0; e < 16; ++e) v[e] = agpr_read(quad[q][i][j][e]);
        store_tile(g, bt, ro, q, pm0 + wrow_a + 32 * i, pn0 + wrow_b + 32 * j, v);
      }
}

// ---------------------------------------------------------------------------
// Exact-dot fused sub-products on the 128 x 128 tile layout (E8M0 scales,
// blocks 32 and 128), two waves per SIMD.
//
// One persistent workgroup of eight waves per CU walks a list of (tile,
// outer term, batch) items; its (item, term, K step) sequence is a single
// transfer pipeline, so the codes of the next item are in flight while the
// current one ends.  Each wave owns 64 rows x 32 columns of the 128 x 128
// tile (two 32 x 32 MFMA tiles), which leaves room for its four W-combine
// quadrants (128 floats a lane) in the architectural registers beside the
// accumulators: a term-end combine is one multiply-add per nonzero weight and
// element, and while one wave converts codes or combines, the other wave on
// its SIMD keeps the matrix core busy.
//
// The MFMAs take the A fragment as their first operand, so a lane holds one
// column of P and, in each register quadruple, four consecutive rows: one
// store instruction writes 128 contiguous bytes of each of two rows (whole
// cache lines; a lane holding four consecutive columns instead writes 32
// bytes of each of 32 rows per 16-byte store instruction, measured 10% slower
// on the batched 512^3 products).
//
// Transfers and fragments are those of gemm_mx_fast_kernel (the 128 x 128
// tile images through a four-slot ring).  Each 64-byte substep runs as four
// v_mfma_f32_32x32x16_bf16 per tile pair on operands converted by
// v_cvt_scalef32_pk_bf16_fp8 with the block's E8M0 scale as the scale
// operand (the dequantized value, exact for every scale the rules produce),
// so the products of the dequantized operands are summed across the whole
// contracted axis at fp32 grade.  Instruction t of substep s takes, in lane
// half h, bytes 64 s + 32 (t >> 1) + 16 h + 8 (t & 1) .. + 7 of the row on
// both operands, which lie in block 2 s + (t >> 1) at block 32 (record byte
// 2 (t >> 1) + s, the record holding blocks 0, 2, 1, 3).  P_r starts from
// zero at each term, and quadrant q of an item accumulates w[r_i][q] * P_r by
// a fused multiply-add in ascending r_i.
// Requires m', n', k' multiples of 128 (the layout's).
// ---------------------------------------------------------------------------
constexpr int kDqThreads = 512;

// s_barrier after this wave's LDS reads have completed; the transfers a wave
// waits for are tracked by wait_vmcnt, and no global store needs to drain here
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int BS>
__global__ __launch_bounds__(kDqThreads, 1) void gemm_dq8_kernel(GemmArgs g, int tiles_m, int nitems) {
  // scale record per row and step: 4 bytes (blocks 32, 128) or 8 (block 16)
  constexpr int REC = BS == 16 ? 8 : 4;
  constexpr int SLOT = 2 * BM * FBK + 2 * BM * REC;
  __shared__ uint4 lds_raw[kSlots * SLOT / 16];
  __shared__ float lds_w[4 * kMaxRank];
  uint8_t *lds = reinterpret_cast<uint8_t *>(lds_raw);
  const uint32_t lds_base = dma::lds_addr(lds_raw);
  const int t = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int lane = t & 63;
  const int r32 = lane & 31, h = lane >> 5;
  const int wrow_a = (wave >> 2) * 64, wrow_b = (wave & 3) * 32;
  const int tiles_n = g.tiles_n, ntiles = tiles_m * tiles_n;
  const int nk = (int)(g.kp / FBK), R = g.R, To = (int)g.To;
  if (t < 4 * kMaxRank) lds_w[t] = g.w[t];   // read only after the first barrier

  // This workgroup's items.  Workgroups are dispatched round-robin over the
  // eight XCDs, so XCD x = blockIdx.x mod 8 is given a contiguous range of
  // items and its P workgroups take every P-th item of it: at any time the
  // workgroups of one XCD work on neighbouring tiles (eight tile rows by four
  // tile columns of one term) and share their codes in its L2.
  int it0, itstep, nmine;
  {
    const int nwg = gridDim.x, b = blockIdx.x;
    if ((nwg & 7) == 0) {
      const int P = nwg >> 3, x = b & 7, j = b >> 3;
      const int lo = (int)((int64_t)x * nitems / 8), hi = (int)((int64_t)(x + 1) * nitems / 8);
      it0 = lo + j;
      itstep = P;
      nmine = hi > it0 ? (hi - it0 + P - 1) / P : 0;
    } else {
      it0 = b;
      itstep = nwg;
      nmine = nitems > it0 ? (nitems - it0 + nwg - 1) / nwg : 0;
    }
  }
  if (nmine == 0) return;                  // uniform over the workgroup
  const int64_t total = (int64_t)nmine * R * nk;   // K steps of this workgroup

  // item id -> tile (tm, tn) in groups of eight tile rows, outer term, batch
  struct Item {
    int tm, tn, ro, bt;
  };
  auto item_of_id = [&](int id) {
    Item x;
    const int rest = id / ntiles, tile = id - rest * ntiles;
    x.ro = rest % To;
    x.bt = rest / To;
    constexpr int GM = 8;
    const int per_group = GM * tiles_n, group = tile / per_group, first_m = group * GM;
    const int gm = min(tiles_m - first_m, GM), in = tile - group * per_group;
    x.tm = first_m + in % gm;
    x.tn = in / gm;
    return x;
  };

  // Transfers of one step: A and B code regions 2 wave, 2 wave + 1 (tile
  // rows 8 region .. + 7), and 256-byte pieces of the scales (A then B: four
  // pieces at block 16, moved by all eight waves; two at blocks 32 and 128,
  // moved by waves 0-3).  The tile indices ta, tb of the next step to
  // transfer advance by one per step and by (tiles - 1) k'/128 more at a
  // term's end.
  const int64_t tma = g.mp / BM, tna = g.np / BN;
  const int64_t da = (tma - 1) * nk, db = (tna - 1) * nk;
  int ri_i = 0, ks_i = 0, k_i = 0;
  int64_t ta = 0, tb = 0;
  auto start_item = [&](int k) {
    const Item x = item_of_id(it0 + k * itstep);
    const int64_t r0 = (int64_t)x.bt * g.T + (int64_t)x.ro * R;
    ta = (r0 * tma + x.tm) * nk;
    tb = (r0 * tna + x.tn) * nk;
  };
  constexpr int SPIECES = BM * REC / 256;                  // 256-byte pieces per side
  const bool scale_wave = wave < 2 * SPIECES, scale_b = wave >= SPIECES;
  const uint32_t piece = 256u * (uint32_t)(wave % SPIECES);
  const uint32_t lds_sc = 2 * BM * FBK + (scale_b ? BM * REC : 0) + piece;
  auto issue_next = [&](int64_t step) {
    const uint8_t *xa = g.xa + ta * (BM * FBK);
    const uint8_t *xb = g.xb + tb * (BN * FBK);
    const uint32_t m0 = lds_base + (uint32_t)(step & (kSlots - 1)) * SLOT;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int region = 2 * wave + j;
      copy16(16u * (uint32_t)lane, xa + region * 1024, m0 + region * 1024);
      copy16(16u * (uint32_t)lane, xb + region * 1024, m0 + BM * FBK + region * 1024);
    }
    if (scale_wave) {
      const uint8_t *sbase = scale_b ? g.sb + tb * (BN * REC) : g.sa + ta * (BM * REC);
      copy4(4u * (uint32_t)lane + piece, sbase, m0 + lds_sc);
    }
    ++ta;
    ++tb;
    if (++ks_i == nk) {
      ks_i = 0;
      ta += da;
      tb += db;
      if (++ri_i == R) {
        ri_i = 0;
        if (++k_i < nmine) start_item(k_i);
      }
    }
  };

  // fragments of one 64-byte substep: A row tiles i = 0, 1 and the B column
  // tile.  The rows a lane reads (wrow_a + r32, + 32, wrow_b + r32) agree
  // mod 16, so they share the swizzle: chunk 2 k + h (k = 0 .. 3; substep s
  // uses k = 2 s, 2 s + 1) of each sits at one lane offset per k, and the
  // second A tile 4096 bytes further.
  struct Frag {
    v8i a[2], b;
  };
  uint32_t la_k[4], lb_k[4];
  {
    const uint32_t x = (uint32_t)((r32 & 7) ^ ((r32 >> 3) & 1));
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t ch = 16u * (((uint32_t)(2 * k + h)) ^ x);
      la_k[k] = (uint32_t)(wrow_a + r32) * BK + ch;
      lb_k[k] = (uint32_t)(BM * FBK) + (uint32_t)(wrow_b + r32) * BK + ch;
    }
  }
  auto read_frag = [&](int64_t step, auto ssc, Frag &f) {
    constexpr int SS = decltype(ssc)::value;
    const uint8_t *slot = lds + (step & (kSlots - 1)) * SLOT;
    const uint8_t *pa0 = slot + la_k[2 * SS], *pa1 = slot + la_k[2 * SS + 1];
    const uint8_t *pb0 = slot + lb_k[2 * SS], *pb1 = slot + lb_k[2 * SS + 1];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint4 lo = *reinterpret_cast<const uint4 *>(pa0 + i * 32 * BK);
      const uint4 hi = *reinterpret_cast<const uint4 *>(pa1 + i * 32 * BK);
      f.a[i] = (v8i){(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
    }
    const uint4 lo = *reinterpret_cast<const uint4 *>(pb0);
    const uint4 hi = *reinterpret_cast<const uint4 *>(pb1);
    f.b = (v8i){(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
  };
  // scales of one step: at blocks 32 and 128 the rows' whole records
  // (blocks 0, 2, 1, 3 at block 32); at block 16 the word of the lane half,
  // h = 0: blocks 0, 2, 4, 6, h = 1: blocks 1, 3, 5, 7 (instruction t of
  // substep s reads block 4 s + 2 (t >> 1) + h)
  const uint32_t lsa_off = 2 * BM * FBK + REC * (uint32_t)(wrow_a + r32) + (BS == 16 ? 4 * h : 0);
  const uint32_t lsb_off = 2 * BM * FBK + BM * REC + REC * (uint32_t)(wrow_b + r32) + (BS == 16 ? 4 * h : 0);
  auto read_scales = [&](int64_t step, int (&sa)[2], int &sb) {
    const uint8_t *slot = lds + (step & (kSlots - 1)) * SLOT;
    sa[0] = *reinterpret_cast<const int *>(slot + lsa_off);
    sa[1] = *reinterpret_cast<const int *>(slot + lsa_off + 32 * REC);
    sb = *reinterpret_cast<const int *>(slot + lsb_off);
  };

  v16f acc[2];
  float quad[4][2][16];
  acc[0] = (v16f){};
  acc[1] = (v16f){};
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) quad[q][i][e] = 0.0f;

  // the MFMAs of substep SS (the A fragment as the first operand)
  auto mfma_sub = [&](auto ssc, const Frag &f, const int (&sa)[2], int sb) {
    constexpr int SS = decltype(ssc)::value;
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
      const int c = tt >> 1, d = 4 * c + 2 * (tt & 1);
      const int sbyte = BS == 16 ? 2 * SS + c : BS == 32 ? 2 * c + SS : 0;
      const v8bf fb = dequant8(f.b, d, e8m0_at(sb, sbyte));
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const v8bf fa = dequant8(f.a[i], d, e8m0_at(sa[i], sbyte));
        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb, acc[i], 0, 0, 0);
      }
    }
  };

  // output of one item: quadrant q = 2 k + i of the tile; lane (c, h) holds
  // column c of the wave's 32 columns and, in register e of 32-row tile i,
  // row 32 i + 8 (e / 4) + 4 h + e % 4 (any 4-byte-aligned C: scalar stores).
  // The stores are nontemporal: C (or the partials, read once by the outer
  // combine) is not read here again, and dirty lines left in the caches
  // would only displace codes and cost the next pass their write-back
  // (depth-3 products 3.69 -> 3.54 ms and the following encode 2.2 -> 2.1 ms
  // at 16384 x 8192 x 16384, paired runs).
  const int64_t ld = g.depth == 1 ? g.N : (int64_t)To * 4 * g.np;   // one row of C, or of the partials
  const int64_t lane_off = (int64_t)(4 * h) * ld + r32;
  auto store_item = [&](int k) {
    const Item x = item_of_id(it0 + k * itstep);
    const int64_t pm0 = (int64_t)x.tm * BM + wrow_a, pn0 = (int64_t)x.tn * BN + wrow_b;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int iq = q & 1, kq = q >> 1;
      float *base = g.depth == 1
                        ? g.out + x.bt * g.M * g.N + (iq * g.mp + pm0) * g.N + kq * g.np + pn0
                        : g.out + ((((int64_t)x.bt * g.mp + pm0) * To + x.ro) * 4 + q) * g.np + pn0;
      base += lane_off;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          __builtin_nontemporal_store(quad[q][i][e], base + (32 * i + 8 * (e >> 2) + (e & 3)) * ld);
    }
  };

  // prologue: steps 0, 1, 2 in flight, step 0 waited for
  start_item(0);
  issue_next(0);
  if (total > 1) issue_next(1);
  if (total > 2) issue_next(2);
  if (total > 2) {
    if (scale_wave) wait_vmcnt<10>(); else wait_vmcnt<8>();
  } else if (total > 1) {
    if (scale_wave) wait_vmcnt<5>(); else wait_vmcnt<4>();
  } else {
    wait_vmcnt<0>();
  }
  lds_barrier();

  // compute stream: item k_c, term ri_c, step ks_c
  int k_c = 0, ri_c = 0, ks_c = 0;
  Frag f0, f1;
  int sa[2], sb;
  read_frag(0, std::integral_constant<int, 0>(), f0);
  read_scales(0, sa, sb);
  int sa_n[2] = {sa[0], sa[1]}, sb_n = sb;
  for (int64_t step = 0; step < total; ++step) {
    read_frag(step, std::integral_constant<int, 1>(), f1);
    mfma_sub(std::integral_constant<int, 0>(), f0, sa, sb);
    if (step + 1 < total) {
      // step + 1 transferred (step + 2 may still be in flight) and every wave
      // done reading step - 1's slot, which step + 3 then takes
      if (step + 2 < total) {
        if (scale_wave) wait_vmcnt<5>(); else wait_vmcnt<4>();
      } else {
        wait_vmcnt<0>();
      }
      lds_barrier();
      if (step + 3 < total) issue_next(step + 3);
      read_frag(step + 1, std::integral_constant<int, 0>(), f0);
      read_scales(step + 1, sa_n, sb_n);
    }
    mfma_sub(std::integral_constant<int, 1>(), f1, sa, sb);
    sa[0] = sa_n[0];
    sa[1] = sa_n[1];
    sb = sb_n;
    if (++ks_c == nk) {
      ks_c = 0;
      // end of term ri_c: quadrant q += w[ri_c][q] * P
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float wq = __builtin_bit_cast(
            float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, lds_w[4 * ri_c + q])));
        if (wq != 0.0f) {
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) quad[q][i][e] = __fmaf_rn(wq, acc[i][e], quad[q][i][e]);
        }
      }
      acc[0] = (v16f){};
      acc[1] = (v16f){};
      if (++ri_c == R) {
        ri_c = 0;
        store_item(k_c);
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) quad[q][i][e] = 0.0f;
        ++k_c;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Promotion path: fp32 block scales (or block 16)
// ---------------------------------------------------------------------------

constexpr int kMaxKbPerStep = BK / 16;   // block 16 -> 8 blocks per k-step

__global__ __launch_bounds__(kThreads, 1) void gemm_promote_kernel(GemmArgs g, int scale_bytes) {
  __shared__ uint4 lds_raw[2 * 2 * BM * BK / 16];
  __shared__ float lsa[BM * kMaxKbPerStep];
  __shared__ float lsb[BN * kMaxKbPerStep];
  uint8_t *lds = reinterpret_cast<uint8_t *>(lds_raw);
  const int t = threadIdx.x;
  const int wave = t >> 6, lane = t & 63;
  const int wm = wave >> 1, wn = wave & 1;
  const int r32 = lane & 31, h = lane >> 5;
  const int64_t tm = blockIdx.x / g.tiles_n, tn = blockIdx.x % g.tiles_n;
  const int64_t ro = blockIdx.y, bt = blockIdx.z;
  const int64_t pm0 = tm * BM, pn0 = tn * BN;
  const int64_t rowa0 = pm0 + wm * 64, rowb0 = pn0 + wn * 64;
  const int64_t nsteps = (g.kp + BK - 1) / BK;
  const int64_t total = (int64_t)g.R * nsteps;
  const int kb_step = BK / g.block > 0 ? BK / g.block : 1;  // blocks per k-step (block <= 128)
  const int chunks_per_block = g.block / 16;

  v16f acc[2][2], quad[4][2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      acc[i][j] = (v16f){};
#pragma unroll
      for (int q = 0; q < 4; ++q) quad[q][i][j] = (v16f){};
    }

  Stage st;
  load_stage(g, bt, ro * g.R, 0, pm0, pn0, st);
  store_stage(lds, lds + BM * BK, st);

  for (int64_t it = 0; it < total; ++it) {
    const int ri = (int)(it / nsteps);
    const int64_t ks = it % nsteps;
    const int64_t r = ro * g.R + ri;
    const int buf = (int)(it & 1);
    const bool more = it + 1 < total;
    // scales of this step into LDS (fp32 values)
    for (int e = t; e < (BM + BN) * kb_step; e += kThreads) {
      const bool isb = e >= BM * kb_step;
      const int ee = isb ? e - BM * kb_step : e;
      const int row = ee / kb_step, kbl = ee % kb_step;
      const int64_t kb = ks * kb_step + kbl;
      const int64_t p = (isb ? pn0 : pm0) + row;
      const int64_t rows = isb ? g.np : g.mp;
      float v = 0.f;
      if (p < rows && kb < g.kblocks) {
        const int64_t idx = ((bt * g.T + r) * rows + p) * g.kblocks + kb;
        const uint8_t *base = isb ? g.sb : g.sa;
        if (scale_bytes == 4)
          v = reinterpret_cast<const float *>(base)[idx];
        else
          v = __uint_as_float((uint32_t)base[idx] << 23);   // 2^(e8m0 - 127)
      }
      (isb ? lsb : lsa)[row * kMaxKbPerStep + kbl] = v;
    }
    __syncthreads();
    if (more) {
      const int64_t rn = ro * g.R + (it + 1) / nsteps;
      const int64_t kn = ((it + 1) % nsteps) * BK;
      load_stage(g, bt, rn, kn, pm0, pn0, st);
    }
    const uint8_t *la = lds + buf * 2 * BM * BK;
    const uint8_t *lb = la + BM * BK;
    for (int kbl = 0; kbl < kb_step; ++kbl) {
      v16f tmp[2][2];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) tmp[i][j] = (v16f){};
      for (int cc = 0; cc < chunks_per_block; ++cc) {
        const int c = kbl * chunks_per_block + cc;   // 16-byte chunk within the step
        v8bf fa[2], fb[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const int rowa = wm * 64 + 32 * i + r32, rowb = wn * 64 + 32 * i + r32;
          fa[i] = e4m3x8_to_bf16(*reinterpret_cast<const uint2 *>(la + swz(rowa, c) + 8 * h));
          fb[i] = e4m3x8_to_bf16(*reinterpret_cast<const uint2 *>(lb + swz(rowb, c) + 8 * h));
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            tmp[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], tmp[i][j], 0, 0, 0);
      }
      // promote: acc += sA[row] sB[col] tmp
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const float sbv = lsb[(wn * 64 + 32 * j + r32) * kMaxKbPerStep + kbl];
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int row = wm * 64 + 32 * i + 8 * (e >> 2) + 4 * h + (e & 3);
            const float s = lsa[row * kMaxKbPerStep + kbl] * sbv;
            acc[i][j][e] = __fmaf_rn(s, tmp[i][j][e], acc[i][j][e]);
          }
        }
    }
    if (ks == nsteps - 1) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float wq = g.w[4 * ri + q];
        if (wq != 0.0f) {
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
              for (int e = 0; e < 16; ++e) quad[q][i][j][e] = __fmaf_rn(wq, acc[i][j][e], quad[q][i][j][e]);
        }
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = (v16f){};
    }
    __syncthreads();   // everyone is done with this buffer and with lsa/lsb
    if (more) {
      uint8_t *na = lds + (buf ^ 1) * 2 * BM * BK;
      store_stage(na, na + BM * BK, st);
    }
  }

#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        store_tile(g, bt, ro, q, rowa0 + 32 * i, rowb0 + 32 * j, quad[q][i][j]);
}

// ---------------------------------------------------------------------------
// Outer combine (depth >= 2): C block (I, K) with I = 2 I_o + i, K = 2 K_o + k:
//   C = sum_{r_o} w_outer[r_o][K_o 2^(l-1) + I_o] * Q[r_o][2k + i]
// ---------------------------------------------------------------------------
template <int NO>   // NO = 4^(l-1) outer blocks
__global__ __launch_bounds__(256) void outer_combine_kernel(const float *__restrict__ Q,
                                                            const float *__restrict__ wo,
                                                            float *__restrict__ C, Problem pb) {
  constexpr int no = NO == 4 ? 2 : 4;   // 2^(l-1)
  const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // p * n' + q
  const int iq = blockIdx.y;                                           // inner quadrant 2k + i
  const int64_t bt = blockIdx.z;
  if (pos >= pb.mp * pb.np) return;
  const int64_t p = pos / pb.np, q = pos % pb.np;
  float acc[NO];
#pragma unroll
  for (int o = 0; o < NO; ++o) acc[o] = 0.f;
  for (int64_t ro = 0; ro < pb.To; ++ro) {
    const float v = Q[(((bt * pb.mp + p) * pb.To + ro) * 4 + iq) * pb.np + q];
#pragma unroll
    for (int o = 0; o < NO; ++o) acc[o] = __fmaf_rn(wo[ro * NO + o], v, acc[o]);
  }
  const int i = iq & 1, k = iq >> 1;
#pragma unroll
  for (int o = 0; o < NO; ++o) {
    const int Ko = o / no, Io = o % no;       // column index o = K_o 2^(l-1) + I_o
    const int64_t I = 2 * Io + i, K = 2 * Ko + k;
    C[bt * pb.M * pb.N + (I * pb.mp + p) * pb.N + K * pb.np + q] = acc[o];
  }
}

// The same with four consecutive columns per thread (n' a multiple of 4, C
// 16-byte aligned): each Q plane read once as float4, eight outer terms'
// loads issued together ahead of the multiply-adds, each term's NO weights
// as one scalar block.  Same arithmetic and order as above.
template <int NO>
__global__ __launch_bounds__(256) void outer_combine4_kernel(const float *__restrict__ Q,
                                                             const float *__restrict__ wo,
                                                             float *__restrict__ C, Problem pb) {
  typedef float f4v __attribute__((ext_vector_type(4)));
  constexpr int no = NO == 4 ? 2 : 4;   // 2^(l-1)
  const int64_t n4 = pb.np / 4;
  const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // p * n4 + q4
  const int iq = blockIdx.y;                                           // inner quadrant 2k + i
  const int64_t bt = blockIdx.z;
  if (pos >= pb.mp * n4) return;
  const int64_t p = pos / n4, q4 = pos - p * n4;
  const int64_t plane = 4 * pb.np;                                     // outer term r_o at src + r_o plane
  const float *src = Q + ((bt * pb.mp + p) * pb.To * 4 + iq) * pb.np + 4 * q4;
  f4v acc[NO];
#pragma unroll
  for (int o = 0; o < NO; ++o) acc[o] = (f4v){0.f, 0.f, 0.f, 0.f};
  const int To = (int)pb.To;
  for (int r0 = 0; r0 < To; r0 += 8) {
    f4v v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int ro = min(r0 + j, To - 1);     // past the last term: a repeated, unused load
      v[j] = __builtin_nontemporal_load(reinterpret_cast<const f4v *>(src + ro * plane));
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (r0 + j < To) {
        float w[NO];
#pragma unroll
        for (int o = 0; o < NO; ++o) w[o] = wo[(r0 + j) * NO + o];
#pragma unroll
        for (int o = 0; o < NO; ++o) {
          acc[o].x = __fmaf_rn(w[o], v[j].x, acc[o].x);
          acc[o].y = __fmaf_rn(w[o], v[j].y, acc[o].y);
          acc[o].z = __fmaf_rn(w[o], v[j].z, acc[o].z);
          acc[o].w = __fmaf_rn(w[o], v[j].w, acc[o].w);
        }
      }
    }
  }
  const int i = iq & 1, k = iq >> 1;
#pragma unroll
  for (int o = 0; o < NO; ++o) {
    const int Ko = o / no, Io = o % no;
    const int64_t I = 2 * Io + i, K = 2 * Ko + k;
    *reinterpret_cast<f4v *>(C + bt * pb.M * pb.N + (I * pb.mp + p) * pb.N + K * pb.np + 4 * q4) = acc[o];
  }
}

}  // namespace

int launch_products(const Problem &pb, const DeviceTables &tab, const uint8_t *ws,
                    const Workspace &wl, float *C, void *stream) {
  if (pb.batch == 0 || pb.M == 0 || pb.N == 0) return hipSuccess;
  if (pb.split) return launch_products_split(pb, ws, wl, stream);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  GemmArgs g;
  g.xa = ws + wl.a_codes;
  g.xb = ws + wl.b_codes;
  g.sa = ws + wl.a_scales;
  g.sb = ws + wl.b_scales;
  g.out = pb.depth == 1 ? C : reinterpret_cast<float *>(const_cast<uint8_t *>(ws) + wl.partial);
  g.mp = pb.mp; g.np = pb.np; g.kp = pb.kp; g.kblocks = pb.kblocks;
  g.T = pb.T; g.To = pb.To; g.M = pb.M; g.N = pb.N;
  g.R = pb.R; g.block = pb.block; g.depth = pb.depth;
  const int64_t tiles_m = (pb.mp + BM - 1) / BM, tiles_n = (pb.np + BN - 1) / BN;
  g.tiles_n = (int)tiles_n;
  g.w = tab.w_inner;
  const dim3 grid((unsigned)(tiles_m * tiles_n), (unsigned)pb.To, (unsigned)pb.batch);
  const bool mx = !pb.exact_dot && pb.rule != dev::RULE_FP32_AMAX && (pb.block == 32 || pb.block == 128);
  // the 128 x 128 tile layout: E8M0 scales at blocks 32 and 128 (fp8 path, or
  // the exact-dot path with each block's power of two folded into the codes)
  const bool aligned = pb.layout == FMM_LAYOUT_TILE128x128;
  if (aligned && (pb.exact_dot || pb.block == 16)) {
    // one persistent workgroup per CU (its LDS ring and registers fill one)
    const int64_t items = tiles_m * tiles_n * pb.To * pb.batch;
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu <= 0)
      ncu = 256;
    if (items > INT32_MAX) return hipErrorInvalidValue;
    const dim3 pgrid((unsigned)(items < ncu ? items : ncu));
#define FMM_DQ8(BSV) \
  hipLaunchKernelGGL((gemm_dq8_kernel<BSV>), pgrid, dim3(kDqThreads), 0, st, g, (int)tiles_m, (int)items)
    if (pb.block == 16)
      FMM_DQ8(16);
    else if (pb.block == 32)
      FMM_DQ8(32);
    else
      FMM_DQ8(128);
#undef FMM_DQ8
  } else if (aligned && pb.block == 32)
    hipLaunchKernelGGL(gemm_mx_fast_kernel<32>, grid, dim3(kThreads), 0, st, g, (int)tiles_m);
  else if (aligned)
    hipLaunchKernelGGL(gemm_mx_fast_kernel<128>, grid, dim3(kThreads), 0, st, g, (int)tiles_m);
  else if (mx)
    hipLaunchKernelGGL(gemm_mx_kernel, grid, dim3(kThreads), 0, st, g);
  else
    hipLaunchKernelGGL(gemm_promote_kernel, grid, dim3(kThreads), 0, st, g, pb.scale_bytes);
  return hipGetLastError();
}

int launch_combine(const Problem &pb, const DeviceTables &tab, const uint8_t *ws, const Workspace &wl,
                   float *C, void *stream) {
  if (pb.batch == 0 || pb.M == 0 || pb.N == 0) return hipSuccess;
  if (pb.split) return launch_combine_split(pb, tab, ws, wl, C, stream);
  if (pb.depth == 1) return hipSuccess;     // fused into the sub-product kernel
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const float *Q = reinterpret_cast<const float *>(ws + wl.partial);
  if (pb.np % 4 == 0 && (reinterpret_cast<uintptr_t>(C) & 15) == 0) {
    const int64_t npos4 = pb.mp * (pb.np / 4);
    const dim3 g4((unsigned)((npos4 + 255) / 256), 4, (unsigned)pb.batch);
    if (pb.depth == 2)
      hipLaunchKernelGGL(outer_combine4_kernel<4>, g4, dim3(256), 0, st, Q, tab.w_outer, C, pb);
    else
      hipLaunchKernelGGL(outer_combine4_kernel<16>, g4, dim3(256), 0, st, Q, tab.w_outer, C, pb);
    return hipGetLastError();
  }
  const int64_t npos = pb.mp * pb.np;
  const dim3 g2((unsigned)((npos + 255) / 256), 4, (unsigned)pb.batch);
  if (pb.depth == 2)
    hipLaunchKernelGGL(outer_combine_kernel<4>, g2, dim3(256), 0, st, Q, tab.w_outer, C, pb);
  else
    hipLaunchKernelGGL(outer_combine_kernel<16>, g2, dim3(256), 0, st, Q, tab.w_outer, C, pb);
  return hipGetLastError();
}

}  // namespace fmm
