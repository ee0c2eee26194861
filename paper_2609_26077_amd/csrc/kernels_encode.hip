// Fused operand combine + block quantization (the encoder of Assumption 1).
//
// One workgroup owns a tile of TR "rows" x TL contracted positions of the
// sub-block grid (TL = 128, or 64 / 32 for the B side's narrow tiles at
// depths 2 / 3) and produces the codes and scales of every flattened term
// for that tile.  A rows are rows of A's sub-blocks; B rows are columns of
// B's sub-blocks, so both outputs have the contracted axis last.
//
//   1. stage: the tile of all 4^l sub-blocks is read from HBM (coalesced)
//      into LDS as fp32, laid out [block][row][l] with the contracted axis
//      contiguous (the B side transposes on the way in);
//   2. combine: every lane of a wave works on one term (the term's nonzero
//      coefficients sit in scalar registers) and forms x = sum_b c_b a_b over
//      them in ascending b, as separate fp32 multiplies and adds, for a run of
//      consecutive contracted positions of one row: 16 at depths 1 and 2
//      (one 16-byte store of codes), 4 at depth 3 (whose 64 sub-blocks leave
//      no room in LDS for rows enough to fill a wave with 16-position runs);
//   3. quantize: the block maximum over `block` consecutive positions is
//      reduced across the lanes that hold it, the rule gives the scale, and
//      the lane casts its values and stores their codes.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device.h"
#include "internal.h"

namespace fmm {

namespace {

// One operand side's coefficient tables: the nonzero entries of every term in
// ascending block order (offsets, entries; read at depth 1) and the dense
// flattened rows, T x 4^l fp32 with zeros (read at depths 2 and 3).
struct SideTab {
  const int32_t *off;
  const CoefEntry *ent;
  const float *dense;
};
inline SideTab a_tab(const DeviceTables &t) { return {t.a_off, t.a_ent, t.u_dense}; }
inline SideTab b_tab(const DeviceTables &t) { return {t.b_off, t.b_ent, t.v_dense}; }

// The coefficient of block b of a dense row spread one block per lane (b uniform).
__device__ __forceinline__ float lane_coef(float c, int b) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(c), b));
}

// Takes the lowest set bit of a uniform mask (the next nonzero block in
// ascending order) or, once the mask is empty, repeats `prev`.
__device__ __forceinline__ int next_block(uint64_t &mask, int prev) {
  if (mask == 0) return prev;
  const int b = __builtin_ctzll(mask);
  mask &= mask - 1;
  return b;
}

constexpr int kTL = 128;            // contracted positions per tile (>= every block size)
constexpr int kStride = kTL + 4;    // LDS row stride in floats: 33 16-byte slots, odd, so
                                    // 16-byte accesses of 16 lanes in 4 consecutive rows x
                                    // 4 slots, or in 16 consecutive rows, hit 16 distinct
                                    // bank groups

// Tile geometry.  VEC = contracted positions per lane (16 at depths 1-2, 4 at
// depth 3).  At depth 1 the B side takes 32 columns (its rows of B are read as
// 128-byte segments) with eight waves (two terms at once), the A side 8 rows
// with two waves that
// split the terms between them (8-row tiles leave room for more workgroups
// per CU than 16-row ones and measured 5-7% faster).  The
// NARROW form (depth 2, B side, blocks of 16 and 32) takes 16 columns x 64
// positions instead of 8 x 128, so B's rows are read as 64-byte segments
// rather than 32-byte ones and a wave writes whole 64-byte code runs.
constexpr int kA1Rows = 8, kA1Threads = 128;   // depth-1 A-side tile rows and threads
constexpr int kB1Rows = 32, kB1Threads = 512;  // depth-1 B-side tile rows (columns of B) and threads
constexpr int kB1NThreads = 256;                // threads of its narrow (64-position) form
constexpr int kB3Rows = 8;          // depth-3 B-side tile rows (columns of B), 32 positions each, at blocks <= 32

// CAP: a realization of another shape, staged as up to CAP blocks of a grid
// known at run time (0: the 2^l x 2^l grid of <2,2,2> at depth l).
template <int DEPTH, int VEC, int SIDE, bool NARROW = false, int CAP = 0>
struct Tile {
  static constexpr int nblk = CAP ? CAP : 1 << (2 * DEPTH);
  static constexpr int TL = NARROW ? (DEPTH == 3 ? 256 / kB3Rows : 64) : kTL;   // contracted positions per tile
  static constexpr int stride = TL + 4;                   // LDS row stride in floats (an odd number of 16-byte slots)
  static constexpr int TR = NARROW ? (DEPTH == 3 ? kB3Rows : DEPTH == 1 ? kB1Rows : 16) : VEC == 16 ? (DEPTH == 1 ? (SIDE == 1 ? kB1Rows : kA1Rows) : 8) : (DEPTH == 3 ? 2 : 64 / nblk);
  // depth 1: 128 (A) or 512 (B) threads; depths 2 and 3 deal the terms out to
  // sixteen waves, which with two workgroups per CU keeps eight waves per SIMD
  static constexpr int threads = DEPTH == 1 ? (SIDE == 0 ? kA1Threads : NARROW ? kB1NThreads : kB1Threads) : 1024;
  static constexpr int lds_floats = nblk * TR * stride;   // 33.8 (A) / 67.6 (B; 34.8 narrow), 67.6 (69.6 narrow), 67.6 KB
  static_assert(lds_floats * 4 <= 160 * 1024, "the tile fits in LDS");
  static_assert(!NARROW || (DEPTH <= 2 && SIDE == 1 && VEC == 16) || (DEPTH == 3 && SIDE == 1 && VEC == 4),
                "the narrow tiles are B sides'");
};

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
// The same permutation of a 32-bit pattern.  Maxima of non-negative finite
// floats are taken on their bit patterns, which order like the unsigned
// integers: one unsigned maximum with the permutation folded in per step.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

// Read the tile into LDS ([block][row][l], row stride TL + 4 floats).  Every
// load is issued before the first LDS write, so the workgroup waits for HBM
// once, not once per element.  The fp32 operands are read exactly once, so
// the loads are nontemporal (they do not displace the codes, which the
// sub-product kernel reads next, from the caches), except where a tile takes
// only part of each cache line (B tiles narrower than 32 columns).  Positions
// outside the operand read as zero.
// GEN: a realization of another shape, whose A grid is gm x gk and B grid
// gk x gn (at most NB blocks; the others are neither read nor used).
typedef float f4v __attribute__((ext_vector_type(4)));

template <int SIDE, int NB, int TR, int NT, int TL = kTL, bool GEN = false>
__device__ __forceinline__ void stage_tile(float *lds, const float *__restrict__ src, const Problem &pb,
                                           int64_t bt, int64_t row0, int64_t l0, int t) {
  constexpr int nc = NB == 4 ? 2 : NB == 16 ? 4 : 8;
  // blocks per grid row (A: gk columns of A's grid; B: gn) and blocks in all
  const int n = GEN ? (SIDE == 0 ? pb.gk : pb.gn) : nc;
  const int nbr = GEN ? (SIDE == 0 ? pb.gm * pb.gk : pb.gk * pb.gn) : NB;
  constexpr int kStr = TL + 4;
  constexpr int kPer = NB * TR * (TL / 4) / NT;       // float4s per thread
  static_assert(NB * TR * (TL / 4) % NT == 0, "the tile splits evenly over the threads");
  const int64_t rows = SIDE == 0 ? pb.mp : pb.np;
  const int64_t kp = pb.kp;
  float4 stage[kPer];
  if (SIDE == 0) {
    // A (M x K): block b = I n + J holds rows I m' + p, columns J k' + l.
    const float *Ab = src + bt * pb.M * pb.K;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int e = t + NT * k;
      const int b = e / (TR * (TL / 4));
      const int rem = e % (TR * (TL / 4));
      const int64_t p = row0 + rem / (TL / 4), l = l0 + 4 * (rem % (TL / 4));
      stage[k] = make_float4(0.f, 0.f, 0.f, 0.f);
      if ((!GEN || b < nbr) && p < rows && l < kp) {
        const int I = b / n, J = b % n;
        const f4v x = __builtin_nontemporal_load(reinterpret_cast<const f4v *>(Ab + (I * pb.mp + p) * pb.K + J * kp + l));
        stage[k] = make_float4(x.x, x.y, x.z, x.w);
      }
    }
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int e = t + NT * k;
      const int b = e / (TR * (TL / 4));
      const int rem = e % (TR * (TL / 4));
      *reinterpret_cast<float4 *>(lds + (b * TR + rem / (TL / 4)) * kStr + 4 * (rem % (TL / 4))) = stage[k];
    }
  } else {
    // B (K x N): block b = J n + K holds rows J k' + l, columns K n' + q;
    // lanes run along q so each of the four loads is coalesced.
    const float *Bb = src + bt * pb.K * pb.N;
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int e = t + NT * k;
      const int b = e / (TR * (TL / 4));
      const int rem = e % (TR * (TL / 4));
      const int64_t qq = row0 + rem % TR, l = l0 + 4 * (rem / TR);
      stage[k] = make_float4(0.f, 0.f, 0.f, 0.f);
      if ((!GEN || b < nbr) && qq < rows && l < kp) {
        const int J = b / n, Kb = b % n;
        const float *p = Bb + (J * kp + l) * pb.N + Kb * pb.np + qq;
        if constexpr (TR < 32) {
          // tiles narrower than 32 columns read each 128-byte line of B in
          // parts, the rest by the tiles of the neighbouring columns, which
          // run at the same time on the same XCD: keep the lines in L2
          stage[k].x = p[0];
          stage[k].y = p[pb.N];
          stage[k].z = p[2 * pb.N];
          stage[k].w = p[3 * pb.N];
        } else {
          stage[k].x = __builtin_nontemporal_load(p);
          stage[k].y = __builtin_nontemporal_load(p + pb.N);
          stage[k].z = __builtin_nontemporal_load(p + 2 * pb.N);
          stage[k].w = __builtin_nontemporal_load(p + 3 * pb.N);
        }
      }
    }
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
      const int e = t + NT * k;
      const int b = e / (TR * (TL / 4));
      const int rem = e % (TR * (TL / 4));
      *reinterpret_cast<float4 *>(lds + (b * TR + rem % TR) * kStr + 4 * (rem / TR)) = stage[k];
    }
  }
}

// Where the results of a run of positions starting at (p, l) go inside one
// term's plane (the same for every term, so computed once per lane):
//   codes : row-major p k' + l, or (large-tile plans) the 256-row x 64-byte
//           tile image, chunk c of tile row t at c ^ ((t >> 2) & 3)
//   scales: row-major p kblocks + kb, or (large-tile plans) K-block-major,
//           E8M0 bytes with rows permuted inside each 256-row tile (row
//           128 wm + 32 i + r at byte 4 (32 wm + r) + i of the tile), fp32
//           values in row order
//   128 x 128 tiles: codes as the 128-row x 128-byte tile image (chunk c of
//           tile row t at c ^ (t & 7) ^ ((t >> 3) & 1)); scales 4 bytes per
//           tile row and 128-byte step (blocks 0, 2, 1, 3 at block 32; the
//           one block repeated at block 128), 8 at block 16 (blocks 0, 2, 4,
//           6, then 1, 3, 5, 7)
// `lead`: this run starts its block (its lane stores the block's scale).
struct Out {
  int64_t code, scale;
  bool valid, leader;
};
__device__ __forceinline__ Out out_of(const Problem &pb, int64_t rows, int64_t p, int64_t l, bool lead) {
  Out o;
  const int64_t kp = pb.kp;
  o.valid = p < rows && l < kp;
  o.leader = o.valid && lead;
  const int64_t kb = l / pb.block;
  if (pb.layout == FMM_LAYOUT_TILE256x64) {
    const int64_t t = p & 255, c = (l >> 4) & 3;
    o.code = ((((p >> 8) * (kp >> 6) + (l >> 6)) << 14) + t * 64 + 16 * (c ^ ((t >> 2) & 3)) + (l & 15));
    o.scale = kb * rows + (pb.scale_bytes == 4 ? p : ((p & ~int64_t(255)) | ((((p >> 7) & 1) * 32 + (p & 31)) * 4 + ((p >> 5) & 3))));
  } else if (pb.layout == FMM_LAYOUT_TILE128x128) {
    const int64_t t = p & 127, c = (l >> 4) & 7, tile = (p >> 7) * (kp >> 7) + (l >> 7);
    o.code = (tile << 14) + t * 128 + 16 * (c ^ (t & 7) ^ ((t >> 3) & 1)) + (l & 15);
    if (pb.block == 16) {
      const int64_t b = (l >> 4) & 7;                      // block of the step
      o.scale = tile * 1024 + t * 8 + 4 * (b & 1) + (b >> 1);
    } else {
      const int64_t kq = (l >> 5) & 3;                     // block of the step (block 32)
      o.scale = tile * 512 + t * 4 + (pb.block == 32 ? ((kq & 1) << 1) | (kq >> 1) : 0);
    }
  } else {
    o.code = p * kp + l;
    o.scale = p * pb.kblocks + kb;
  }
  return o;
}

// elements of scales per (batch, term) plane (the 128 x 128 layout keeps 4
// bytes per row and step, 8 at block 16)
__device__ __forceinline__ int64_t scale_plane_of(const Problem &pb, int64_t rows) {
  return pb.layout == FMM_LAYOUT_TILE128x128 ? rows * (pb.kp / 128) * (pb.block == 16 ? 8 : 4)
                                              : rows * pb.kblocks;
}

__device__ __forceinline__ void store_scale(const Problem &pb, uint8_t *scales, int64_t at, uint32_t stored) {
  if (pb.scale_bytes == 4)
    reinterpret_cast<uint32_t *>(scales)[at] = stored;
  else if (pb.layout == FMM_LAYOUT_TILE128x128 && pb.block == 128)
    *reinterpret_cast<uint32_t *>(scales + at) = stored * 0x01010101u;
  else
    scales[at] = (uint8_t)stored;
}

// ---------------------------------------------------------------------------
// Depths 1 and 2: 16 positions per lane.
//
// A wave covers 8 rows x 128 positions of one term: lane = 32 h + 4 r + c'
// holds row r, positions 16 (4 h + c') .. +15, so a 16-lane group reads 4
// rows x 4 slots (conflict-free at the odd stride) and a block of 32 is a lane
// pair (lane, lane ^ 1), a block of 128 the quad plus its partner 32 lanes on
// (the narrow tiles: 16 rows x 64 positions, lane = 4 r + c').  The waves that
// cover a tile's rows work on one term and the workgroup's wave groups take
// the terms in turn: depth 1 A 8 rows (one wave per term, two terms at once),
// B 32 rows (four waves per term, two terms at once); depth 2 one wave per
// term, sixteen terms at once.
// ---------------------------------------------------------------------------
// Weight-side deployment granularity (FMM_FLAG_B_BLOCK128 / FMM_FLAG_B_BF16,
// B side at depth 1), in two launches over the same tiles:
//   MODE 1: combine (and round to bfloat16), then the maximum of |y| over the
//           block's positions and the wave's 8 rows, merged into the 2-D
//           block's maximum amax[bt][r][row block][kb] by an integer atomic
//           maximum on the float bits (non-negative, so the order of the
//           merges does not matter); nothing else is stored;
//   MODE 2: combine (and round), take the block maximum from amax (or, with
//           1-row blocks, from the lanes as in MODE 0), scale, cast, store.
// MODE 0 is the plain encoder.
// MODE 3 measures the operand-side rounding energy of an encoding already in
// the workspace (Appendix D, eq. D.1): it forms x_r exactly as the encoder
// does, decodes the stored codes and scales to xhat_r (exact in binary64),
// and writes each wave's sum of (xhat - x)^2 and of x^2 per term to
// aux[((bt * tiles + tile) * waves + wave) * T + r][2] (binary64, lanes summed
// in a fixed butterfly order).
__device__ __forceinline__ float bf16_round(float x) {
  // nearest bfloat16, ties to even (finite x; a carry past the largest
  // finite value gives infinity, as the definition does)
  uint32_t b = __float_as_uint(x);
  b += 0x7fffu + ((b >> 16) & 1u);
  return __uint_as_float(b & 0xffff0000u);
}

// The plain depth-2 B-side encoder at blocks of 16 and 32 takes the narrow tile.
constexpr bool narrow_b(int side, int depth, int bs, int mode) {
  return side == 1 && depth == 2 && bs <= 32 && mode == 0;
}

template <int SIDE, int DEPTH, int BS, bool F32, int MODE, int CAP = 0, bool N1 = false>
__global__ __launch_bounds__((Tile<DEPTH, 16, SIDE, narrow_b(SIDE, DEPTH, BS, MODE) || N1>::threads)) void encode16_kernel(
    const float *__restrict__ src, Problem pb, SideTab cf, uint8_t *__restrict__ codes, uint8_t *__restrict__ scales,
    int64_t tiles_l, void *__restrict__ aux) {
  static_assert(MODE == 0 || MODE == 3 || (SIDE == 1 && DEPTH == 1), "deployment granularity: B side, depth 1");
  static_assert(CAP == 0 || (MODE == 0 && (DEPTH == 1 || CAP == 16)), "other shapes: the plain encoder");
  constexpr bool GEN = CAP != 0;
  uint32_t *amax = reinterpret_cast<uint32_t *>(aux);
  using TT = Tile<DEPTH, 16, SIDE, narrow_b(SIDE, DEPTH, BS, MODE) || N1, CAP>;
  constexpr int TR = TT::TR, NB = TT::nblk, NT = TT::threads, TL = TT::TL, STR = TT::stride;
  constexpr int RPW = 64 * 16 / TL;         // rows per wave: 8, or 16 in the narrow tile
  constexpr int WPT = TR / RPW;             // waves per term (1 (A), 4 (B) or 2 (narrow B) at depth 1, 1 at depth 2)
  constexpr int TSTEP = NT / 64 / WPT;      // terms a workgroup works on at once
  __shared__ float4 lds4[TT::lds_floats / 4];
  float *lds = reinterpret_cast<float *>(lds4);

  const int t = threadIdx.x;
  const int64_t bt = blockIdx.y;
  // depth-1 B side: the column tile varies fastest over the workgroups, so
  // neighbouring workgroups read adjacent 128-byte pieces of the same rows of
  // B at about the same time (the narrower tiles of depths 2 and 3 instead
  // rely on the neighbouring columns' tile running on the same XCD)
  const int64_t tiles_r = gridDim.x / tiles_l;
  constexpr bool qfast = SIDE == 1 && DEPTH == 1 && MODE != 3;
  const int64_t row0 = (qfast ? blockIdx.x % tiles_r : blockIdx.x / tiles_l) * TR;
  const int64_t l0 = (qfast ? blockIdx.x / tiles_r : blockIdx.x % tiles_l) * TL;
  const int64_t rows = SIDE == 0 ? pb.mp : pb.np;
  stage_tile<SIDE, NB, TR, NT, TL, GEN>(lds, src, pb, bt, row0, l0, t);
  __syncthreads();

  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  // 16-position run of the row and the row: lane = 32 h + 4 r + c' (run 4 h + c'),
  // or in the narrow tile lane = 4 r + c' (run c')
  const int ch = TL == 64 ? (lane & 3) : ((lane >> 5) << 2) | (lane & 3);
  const int row = RPW * (wave % WPT) + (TL == 64 ? (lane >> 2) : ((lane >> 2) & 7));
  const float *lrow = lds + row * STR + 16 * ch;
  const bool lead = BS == 16 ? true : BS == 32 ? (ch & 1) == 0 : ch == 0;
  const Out o = out_of(pb, rows, row0 + row, l0 + 16 * ch, lead);
  const int64_t code_plane = rows * pb.kp;
  const int64_t scale_plane = scale_plane_of(pb, rows);
  const int64_t T = pb.T;

  // depth 2: the term's dense coefficient row (block b in lane b) is loaded
  // one term ahead by a vector load, so the term loop never waits on scalar
  // memory; its nonzero blocks come from the wave's ballot in ascending order
  float cnext = 0.0f;
  if constexpr (DEPTH >= 2) {
    const int64_t rf = wave / WPT;
    if (rf < T && lane < NB) cnext = cf.dense[rf * NB + lane];
  }
  for (int64_t r = wave / WPT; r < T; r += TSTEP) {
    // x = sum_b c_b a_b in ascending b: products and sums rounded separately
    float x[16];
    if constexpr (DEPTH >= 2) {
      const float c = cnext;
      if (r + TSTEP < T && lane < NB) cnext = cf.dense[(r + TSTEP) * NB + lane];
      uint64_t mask = __ballot(c != 0.0f);
      if (mask == 0) {
#pragma unroll
        for (int i = 0; i < 16; ++i) x[i] = 0.0f;
      }
      bool first = true;
      while (mask != 0) {
        // two blocks per pass (the second repeats the first when there is none)
        const int b0 = next_block(mask, 0);
        const bool two = mask != 0;
        const int b1 = next_block(mask, b0);
        const float4 *p0 = reinterpret_cast<const float4 *>(lrow + b0 * (TR * STR));
        const float4 *p1 = reinterpret_cast<const float4 *>(lrow + b1 * (TR * STR));
        const float4 v[8] = {p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], p1[2], p1[3]};
        const float c0 = lane_coef(c, b0), c1 = lane_coef(c, b1);
        const float *a = reinterpret_cast<const float *>(v);
        if (first) {
#pragma unroll
          for (int i = 0; i < 16; ++i) x[i] = __fmul_rn(c0, a[i]);
        } else {
#pragma unroll
          for (int i = 0; i < 16; ++i) x[i] = __fadd_rn(x[i], __fmul_rn(c0, a[i]));
        }
        first = false;
        if (two) {
#pragma unroll
          for (int i = 0; i < 16; ++i) x[i] = __fadd_rn(x[i], __fmul_rn(c1, a[16 + i]));
        }
      }
    } else {
      const int beg = __builtin_amdgcn_readfirstlane(cf.off[r]);
      const int nc = __builtin_amdgcn_readfirstlane(cf.off[r + 1]) - beg;
      CoefEntry ce[NB];
#pragma unroll
      for (int e = 0; e < NB; ++e)
        if (e < nc) ce[e] = cf.ent[beg + e];
      if (nc == 0) {
#pragma unroll
        for (int i = 0; i < 16; ++i) x[i] = 0.0f;
      }
#pragma unroll
      for (int e = 0; e < NB; ++e) {
        if (e < nc) {
          const float4 *p = reinterpret_cast<const float4 *>(lrow + ce[e].block * (TR * STR));
          const float4 v0 = p[0], v1 = p[1], v2 = p[2], v3 = p[3];
          const float a[16] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w,
                               v2.x, v2.y, v2.z, v2.w, v3.x, v3.y, v3.z, v3.w};
          const float c = ce[e].coef;
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const float pr = __fmul_rn(c, a[i]);
            x[i] = e == 0 ? pr : __fadd_rn(x[i], pr);
          }
        }
      }
    }
    if constexpr (MODE == 3) {
      double e2 = 0.0, x2 = 0.0;
      if (o.valid) {
        const int64_t plane = bt * T + r;
        const uint4 cw = *reinterpret_cast<const uint4 *>(codes + plane * code_plane + o.code);
        const double sc = pb.scale_bytes == 4
                              ? (double)__uint_as_float(reinterpret_cast<const uint32_t *>(scales)[plane * scale_plane + o.scale])
                              : ldexp(1.0, (int)scales[plane * scale_plane + o.scale] - 127);
        const int cwv[4] = {(int)cw.x, (int)cw.y, (int)cw.z, (int)cw.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float d0 = __builtin_amdgcn_cvt_f32_fp8(cwv[j], 0), d1 = __builtin_amdgcn_cvt_f32_fp8(cwv[j], 1);
          const float d2 = __builtin_amdgcn_cvt_f32_fp8(cwv[j], 2), d3 = __builtin_amdgcn_cvt_f32_fp8(cwv[j], 3);
          const float dec[4] = {d0, d1, d2, d3};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const double xv = (double)x[4 * j + i];
            const double dv = (double)dec[i] * sc - xv;
            e2 += dv * dv;
            x2 += xv * xv;
          }
        }
      }
#pragma unroll
      for (int sh = 32; sh >= 1; sh >>= 1) {
        e2 += __shfl_xor(e2, sh, 64);
        x2 += __shfl_xor(x2, sh, 64);
      }
      if (lane == 0) {
        double *pp = reinterpret_cast<double *>(aux) +
                     ((((int64_t)bt * gridDim.x + blockIdx.x) * (NT / 64) + wave) * T + r) * 2;
        pp[0] = e2;
        pp[1] = x2;
      }
      continue;
    }
    if constexpr (MODE == 1 || MODE == 2) {
      if (pb.b_bf16) {
#pragma unroll
        for (int i = 0; i < 16; ++i) x[i] = bf16_round(x[i]);
      }
    }
    // block maximum: the lane's 16, then across the lanes of its block
    float m = fmaxf(fabsf(x[0]), fabsf(x[1]));
#pragma unroll
    for (int i = 2; i < 16; ++i) m = fmaxf(m, fabsf(x[i]));
    // the 2-D block of this lane: row block (row0 + row) / 128 (a tile's rows
    // lie in one), K block of position l0 + 16 ch
    const int64_t kb = (l0 + 16 * ch) / pb.block;
    const int64_t aidx = (((int64_t)bt * T + r) * ((rows + 127) / 128) + row0 / 128) * pb.kblocks + kb;
    if constexpr (MODE == 1) {
      // over the wave's 8 rows (lane bits 2..4), then the block's lanes
      m = fmaxf(m, __shfl_xor(m, 4, 64));
      m = fmaxf(m, __shfl_xor(m, 8, 64));
      m = fmaxf(m, __shfl_xor(m, 16, 64));
    }
    if (MODE != 2 || pb.b_rows == 1) {
      if (BS >= 32) {
        uint32_t mb = __float_as_uint(m);                       // m >= 0
        mb = max(mb, dpp_u<0xB1>(mb));                          // quad_perm [1, 0, 3, 2]
        if (BS == 128) {
          mb = max(mb, dpp_u<0x4E>(mb));                        // quad_perm [2, 3, 0, 1]
          mb = max(mb, (uint32_t)__shfl_xor((int)mb, 32, 64));
        }
        m = __uint_as_float(mb);
      }
    }
    if constexpr (MODE == 1) {
      if (((lane >> 2) & 7) == 0 && lead && l0 + 16 * ch < pb.kp) atomicMax(amax + aidx, __float_as_uint(m));
      continue;
    }
    if constexpr (MODE == 2) {
      if (pb.b_rows > 1) m = o.valid ? __uint_as_float(amax[aidx]) : 0.0f;
    }
    uint32_t w[4];
    uint32_t stored;
    if constexpr (F32) {
      const dev::Scale sc = dev::block_scale(m, dev::RULE_FP32_AMAX);
      stored = sc.stored;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w[j] = dev::e4m3_pack4(__fdiv_rn(x[4 * j], sc.div), __fdiv_rn(x[4 * j + 1], sc.div),
                               __fdiv_rn(x[4 * j + 2], sc.div), __fdiv_rn(x[4 * j + 3], sc.div));
    } else {
      // a power-of-two rule (the ceiling or the OCP one)
      const dev::Scale sc = dev::block_scale(m, pb.rule == dev::RULE_POW2_CEIL ? dev::RULE_POW2_CEIL
                                                                                : dev::RULE_POW2_OCP);
      stored = sc.stored;
      const float s = __uint_as_float(sc.stored << 23);     // 2^e (stored = e + 127)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w[j] = dev::e4m3_pack4_pow2(x[4 * j], x[4 * j + 1], x[4 * j + 2], x[4 * j + 3], s);
    }
    const int64_t plane = bt * T + r;
    if (o.valid)
      *reinterpret_cast<uint4 *>(codes + plane * code_plane + o.code) = make_uint4(w[0], w[1], w[2], w[3]);
    if (o.leader) store_scale(pb, scales, plane * scale_plane + o.scale, stored);
  }
}

// ---------------------------------------------------------------------------
// Depth 3: 4 positions per lane (2 rows x 128 positions per tile, or on the B
// side at blocks 16 and 32 8 rows x 32 positions; 64 items of one term per
// wave).
// ---------------------------------------------------------------------------
// Maximum over each group of GL aligned lanes (GL = block / 4: 4, 8 or 32),
// every lane receiving its group's maximum: quad permutations (xor 1, xor 2),
// then the half-row and row mirrors, then across the two rows of 32 lanes.
// Taken on the bit patterns of non-negative finite values (equal to the
// floating-point maximum), one unsigned maximum per step.
template <int GL>
__device__ __forceinline__ uint32_t group_max_bits(uint32_t m) {
  m = max(m, dpp_u<0xB1>(m));                         // quad_perm [1, 0, 3, 2]
  m = max(m, dpp_u<0x4E>(m));                         // quad_perm [2, 3, 0, 1]
  if (GL >= 8) m = max(m, dpp_u<0x141>(m));           // row_half_mirror: lane i <- 7 - i within 8
  if (GL >= 16) m = max(m, dpp_u<0x140>(m));          // row_mirror: lane i <- 15 - i within 16
  if (GL >= 32) m = max(m, (uint32_t)__shfl_xor((int)m, 16, 64));
  return m;
}

// Scale and codes of a lane's 4 values of a block whose maximum is m: the
// fp32 rule divides (IEEE), the power-of-two rules scale exactly inside the
// conversion.
template <bool F32>
__device__ __forceinline__ uint32_t quantize4(const Problem &pb, float m, float x0, float x1, float x2, float x3,
                                              uint32_t &stored) {
  if constexpr (F32) {
    const dev::Scale sc = dev::block_scale(m, dev::RULE_FP32_AMAX);
    stored = sc.stored;
    return dev::e4m3_pack4(__fdiv_rn(x0, sc.div), __fdiv_rn(x1, sc.div), __fdiv_rn(x2, sc.div),
                           __fdiv_rn(x3, sc.div));
  } else {
    const dev::Scale sc =
        dev::block_scale(m, pb.rule == dev::RULE_POW2_CEIL ? dev::RULE_POW2_CEIL : dev::RULE_POW2_OCP);
    stored = sc.stored;
    return dev::e4m3_pack4_pow2(x0, x1, x2, x3, __uint_as_float(sc.stored << 23));
  }
}

constexpr bool narrow_b3(int side, int bs) { return side == 1 && bs <= 256 / kB3Rows; }

template <int SIDE, int BS, bool F32, bool GEN = false>
__global__ __launch_bounds__((Tile<3, 4, SIDE, narrow_b3(SIDE, BS)>::threads), 8) void encode4_kernel(
    const float *__restrict__ src, Problem pb, SideTab cf, uint8_t *__restrict__ codes, uint8_t *__restrict__ scales,
    int64_t tiles_l) {
  using TT = Tile<3, 4, SIDE, narrow_b3(SIDE, BS)>;
  constexpr int TR = TT::TR, NT = TT::threads, TL = TT::TL, STR = TT::stride;
  constexpr int P = TR * (TL / 4);           // positions (row, 4 consecutive l) per term
  static_assert(P == 64 && TT::nblk == 64, "a wave's 64 items are one term's tile; lane b holds block b's coefficient");
  __shared__ float4 lds4[TT::lds_floats / 4];
  float *lds = reinterpret_cast<float *>(lds4);

  const int t = threadIdx.x;
  const int64_t bt = blockIdx.y;
  const int64_t row0 = (blockIdx.x / tiles_l) * TR;
  const int64_t l0 = (blockIdx.x % tiles_l) * TL;
  const int64_t rows = SIDE == 0 ? pb.mp : pb.np;
  stage_tile<SIDE, TT::nblk, TR, NT, TL, GEN>(lds, src, pb, bt, row0, l0, t);
  __syncthreads();

  const int64_t T = pb.T;
  constexpr int GL = BS / 4;                 // lanes per block
  const int pos = t % P;
  const int row = pos / (TL / 4), c4 = pos % (TL / 4);
  static_assert(BS <= TL, "a block lies in one row of the tile");
  const Out o = out_of(pb, rows, row0 + row, l0 + 4 * c4, (c4 % GL) == 0);
  // a lane's offsets inside a (batch, term) plane fit in 32 bits
  const uint32_t o_code = (uint32_t)o.code, o_scale = (uint32_t)o.scale;
  const bool o_valid = o.valid, o_leader = o.leader;
  const int64_t code_plane = rows * pb.kp;
  const int64_t scale_plane = scale_plane_of(pb, rows);
  const float *lrow = lds + row * STR + 4 * c4;
  // A wave takes a group of up to kG consecutive terms at once: at depth 3 the
  // R terms that share their two outer digits (T* flattened: 17 nonzero
  // blocks per term on average, 26 in the union of a group of 7), so each
  // block is read from LDS once per group rather than once per term.  Every
  // term's x = sum_b c_b a_b still runs over its own nonzero blocks in
  // ascending b with products and sums rounded separately, its first block
  // giving x = c a.  The terms' dense coefficient rows (block b in lane b)
  // give each term's nonzero blocks by a ballot; their union is walked in
  // ascending order.
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  // Whole rounds of groups (every wave one group per round) go first; the
  // terms left over are taken one per wave, which keeps the waves' loads
  // within one term of each other (343 terms in groups of 7: 48 groups in
  // three rounds, then 7 single terms).
  constexpr int WSTEP = NT / 64;
  constexpr int kG = 8;
  const int G = GEN ? kG : pb.R;             // R <= 8 at <2,2,2>
  const int64_t nfull = ((T + G - 1) / G / WSTEP) * WSTEP;      // groups taken in whole rounds
  const int64_t tail0 = nfull * G < T ? nfull * G : T;          // the first term taken alone
  const int64_t units = nfull + (T - tail0);
  for (int64_t u = wave; u < units; u += WSTEP) {
    const int64_t g0 = u < nfull ? u * G : tail0 + (u - nfull);
    const int gn = u < nfull ? (int)(T - g0 < G ? T - g0 : G) : 1;
    float c[kG];
#pragma unroll
    for (int j = 0; j < kG; ++j) c[j] = j < gn ? cf.dense[(g0 + j) * 64 + lane] : 0.0f;
    uint64_t m[kG];
    uint64_t uni = 0;
#pragma unroll
    for (int j = 0; j < kG; ++j) {
      m[j] = __ballot(c[j] != 0.0f);
      uni |= m[j];
    }
    // accumulators start at -0: -0 + t = t exactly for every t, so a term's
    // first block gives x = c a as the definition does; a term without
    // nonzero blocks ends at +0
    float x[kG][4];
#pragma unroll
    for (int j = 0; j < kG; ++j) x[j][0] = x[j][1] = x[j][2] = x[j][3] = -0.0f;
    if (uni != 0) {
      // the next block's values are read while this block's are used
      int b = __builtin_ctzll(uni);
      uni &= uni - 1;
      float4 v = *reinterpret_cast<const float4 *>(lrow + b * (TR * STR));
      while (true) {
        const bool more = uni != 0;
        const int bn = more ? __builtin_ctzll(uni) : b;
        uni &= uni - 1;
        const float4 vn = *reinterpret_cast<const float4 *>(lrow + bn * (TR * STR));
#pragma unroll
        for (int j = 0; j < kG; ++j) {
          if ((m[j] >> b) & 1) {
            const float cb = lane_coef(c[j], b);
            x[j][0] = __fadd_rn(x[j][0], __fmul_rn(cb, v.x));
            x[j][1] = __fadd_rn(x[j][1], __fmul_rn(cb, v.y));
            x[j][2] = __fadd_rn(x[j][2], __fmul_rn(cb, v.z));
            x[j][3] = __fadd_rn(x[j][3], __fmul_rn(cb, v.w));
          }
        }
        if (!more) break;
        b = bn;
        v = vn;
      }
    }
#pragma unroll
    for (int j = 0; j < kG; ++j)
      if (m[j] == 0) x[j][0] = x[j][1] = x[j][2] = x[j][3] = 0.0f;
#pragma unroll
    for (int j = 0; j < kG; ++j) {
      if (j < gn) {
        const float mx = __uint_as_float(group_max_bits<GL>(__float_as_uint(
            fmaxf(fmaxf(fabsf(x[j][0]), fabsf(x[j][1])), fmaxf(fabsf(x[j][2]), fabsf(x[j][3]))))));
        uint32_t stored;
        const uint32_t w = quantize4<F32>(pb, mx, x[j][0], x[j][1], x[j][2], x[j][3], stored);
        const int64_t plane = bt * T + g0 + j;      // uniform
        if (o_valid) *reinterpret_cast<uint32_t *>(codes + plane * code_plane + o_code) = w;
        if (o_leader) store_scale(pb, scales, plane * scale_plane + o_scale, stored);
      }
    }
  }
}

// N1: the depth-1 B side's narrow tile (32 columns x 64 positions, 256
// threads), taken on the 256 x 64 tile layout at blocks 16 and 32: each lane
// quad writes a whole 64-byte image row, and the half-size tile lets four
// workgroups share a CU (8192^3 T* encode 149 -> 143.5 us, codes identical).
template <int SIDE, int DEPTH, int BS, bool F32, int MODE = 0, int CAP = 0, bool N1 = false>
hipError_t launch16(const Problem &pb, const float *src, const SideTab &cf,
                    uint8_t *codes, uint8_t *scales, hipStream_t st, void *amax = nullptr) {
  if constexpr (SIDE == 1 && DEPTH == 1 && MODE == 0 && CAP == 0 && BS <= 32 && !N1) {
    if (pb.layout == FMM_LAYOUT_TILE256x64)
      return launch16<SIDE, DEPTH, BS, F32, MODE, CAP, true>(pb, src, cf, codes, scales, st, amax);
  }
  using TT = Tile<DEPTH, 16, SIDE, narrow_b(SIDE, DEPTH, BS, MODE) || N1, CAP>;
  const int64_t rows = SIDE == 0 ? pb.mp : pb.np;
  const int64_t tiles_l = (pb.kp + TT::TL - 1) / TT::TL;
  const int64_t tiles_r = (rows + TT::TR - 1) / TT::TR;
  const dim3 grid((unsigned)(tiles_l * tiles_r), (unsigned)pb.batch);
  hipLaunchKernelGGL((encode16_kernel<SIDE, DEPTH, BS, F32, MODE, CAP, N1>), grid, dim3(TT::threads), 0, st, src, pb, cf,
                     codes, scales, tiles_l, amax);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void zero_u32_kernel(uint32_t *p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = 0u;
}

// B side with the weight-side deployment granularity (depth 1): the 2-D
// block maxima (zeroed, then merged by MODE 1) when blocks span 128 rows,
// then the quantizing pass.
template <int BS, bool F32>
hipError_t launch_b_deploy(const Problem &pb, const float *src, const SideTab &cf,
                           uint8_t *codes, uint8_t *scales, uint32_t *amax, hipStream_t st) {
  if (pb.b_rows > 1) {
    const int64_t n = pb.batch * pb.T * ((pb.np + 127) / 128) * pb.kblocks;
    const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL(zero_u32_kernel, dim3((unsigned)blocks), dim3(256), 0, st, amax, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch16<1, 1, BS, F32, 1>(pb, src, cf, codes, scales, st, amax);
    if (e != hipSuccess) return e;
  }
  return launch16<1, 1, BS, F32, 2>(pb, src, cf, codes, scales, st, amax);
}

hipError_t launch_b_deploy_any(const Problem &pb, const float *src, const SideTab &cf,
                               uint8_t *codes, uint8_t *scales, uint32_t *amax, hipStream_t st) {
  const bool f32 = pb.rule == dev::RULE_FP32_AMAX;
  switch (pb.block) {
    case 16: return f32 ? launch_b_deploy<16, true>(pb, src, cf, codes, scales, amax, st)
                        : launch_b_deploy<16, false>(pb, src, cf, codes, scales, amax, st);
    case 32: return f32 ? launch_b_deploy<32, true>(pb, src, cf, codes, scales, amax, st)
                        : launch_b_deploy<32, false>(pb, src, cf, codes, scales, amax, st);
    case 128: return f32 ? launch_b_deploy<128, true>(pb, src, cf, codes, scales, amax, st)
                         : launch_b_deploy<128, false>(pb, src, cf, codes, scales, amax, st);
  }
  return hipErrorInvalidValue;
}

template <int SIDE, int DEPTH, int CAP = 0>
hipError_t launch_wide(const Problem &pb, const float *src, const SideTab &cf,
                       uint8_t *codes, uint8_t *scales, hipStream_t st) {
  const bool f32 = pb.rule == dev::RULE_FP32_AMAX;
  switch (pb.block) {
    case 16: return f32 ? launch16<SIDE, DEPTH, 16, true, 0, CAP>(pb, src, cf, codes, scales, st)
                        : launch16<SIDE, DEPTH, 16, false, 0, CAP>(pb, src, cf, codes, scales, st);
    case 32: return f32 ? launch16<SIDE, DEPTH, 32, true, 0, CAP>(pb, src, cf, codes, scales, st)
                        : launch16<SIDE, DEPTH, 32, false, 0, CAP>(pb, src, cf, codes, scales, st);
    case 128: return f32 ? launch16<SIDE, DEPTH, 128, true, 0, CAP>(pb, src, cf, codes, scales, st)
                         : launch16<SIDE, DEPTH, 128, false, 0, CAP>(pb, src, cf, codes, scales, st);
  }
  return hipErrorInvalidValue;
}

// 4 positions per lane over a grid of up to 64 blocks (depth 3, or GEN)
template <int SIDE, bool GEN = false>
hipError_t launch_narrow4(const Problem &pb, const float *src, const SideTab &cf,
                          uint8_t *codes, uint8_t *scales, hipStream_t st) {
  const int64_t rows = SIDE == 0 ? pb.mp : pb.np;
  // the B side's tile at blocks <= 256 / kB3Rows (its narrow form), else the common one
  const bool nar = SIDE == 1 && pb.block <= 256 / kB3Rows;
  const int TL = nar ? Tile<3, 4, 1, true>::TL : kTL, TR = nar ? Tile<3, 4, 1, true>::TR : Tile<3, 4, SIDE>::TR;
  const int64_t tiles_l = (pb.kp + TL - 1) / TL;
  const int64_t tiles_r = (rows + TR - 1) / TR;
  const dim3 grid((unsigned)(tiles_l * tiles_r), (unsigned)pb.batch);
  const bool f32 = pb.rule == dev::RULE_FP32_AMAX;
  const dim3 blk(Tile<3, 4, SIDE>::threads);
  switch (pb.block) {
    case 16:
      if (f32) hipLaunchKernelGGL((encode4_kernel<SIDE, 16, true, GEN>), grid, blk, 0, st, src, pb, cf, codes, scales, tiles_l);
      else hipLaunchKernelGGL((encode4_kernel<SIDE, 16, false, GEN>), grid, blk, 0, st, src, pb, cf, codes, scales, tiles_l);
      break;
    case 32:
      if (f32) hipLaunchKernelGGL((encode4_kernel<SIDE, 32, true, GEN>), grid, blk, 0, st, src, pb, cf, codes, scales, tiles_l);
      else hipLaunchKernelGGL((encode4_kernel<SIDE, 32, false, GEN>), grid, blk, 0, st, src, pb, cf, codes, scales, tiles_l);
      break;
    case 128:
      if (f32) hipLaunchKernelGGL((encode4_kernel<SIDE, 128, true, GEN>), grid, blk, 0, st, src, pb, cf, codes, scales, tiles_l);
      else hipLaunchKernelGGL((encode4_kernel<SIDE, 128, false, GEN>), grid, blk, 0, st, src, pb, cf, codes, scales, tiles_l);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int SIDE>
hipError_t launch_side(const Problem &pb, const float *src, const SideTab &cf,
                       uint8_t *codes, uint8_t *scales, hipStream_t st) {
  if (pb.shaped) {
    // another shape: the depth-1 tile staging 4 or 8 blocks (the sizes that
    // keep as many bytes in flight per CU as the <2,2,2> encoder), the
    // depth-2 tile (16 positions per lane, 16 waves) over up to 16 blocks,
    // the depth-3 one (4 per lane) over up to 64
    const int nb = SIDE == 0 ? pb.gm * pb.gk : pb.gk * pb.gn;
    if (nb <= 4) return launch_wide<SIDE, 1, 4>(pb, src, cf, codes, scales, st);
    if (nb <= 8) return launch_wide<SIDE, 1, 8>(pb, src, cf, codes, scales, st);
    if (nb <= 16) return launch_wide<SIDE, 2, 16>(pb, src, cf, codes, scales, st);
    return launch_narrow4<SIDE, true>(pb, src, cf, codes, scales, st);
  }
  switch (pb.depth) {
    case 1: return launch_wide<SIDE, 1>(pb, src, cf, codes, scales, st);
    case 2: return launch_wide<SIDE, 2>(pb, src, cf, codes, scales, st);
    case 3: return launch_narrow4<SIDE>(pb, src, cf, codes, scales, st);
  }
  return hipErrorInvalidValue;
}

// ---- operand-side rounding energy (MODE 3) ----------------------------------

template <int SIDE>
int64_t noise_slots(const Problem &pb) {
  const int64_t rows = SIDE == 0 ? pb.mp : pb.np;
  const int64_t tiles = ((pb.kp + kTL - 1) / kTL) * ((rows + (pb.depth == 1 ? Tile<1, 16, SIDE>::TR : Tile<2, 16, SIDE>::TR) - 1) /
                                                    (pb.depth == 1 ? Tile<1, 16, SIDE>::TR : Tile<2, 16, SIDE>::TR));
  const int64_t waves = (pb.depth == 1 ? Tile<1, 16, SIDE>::threads : Tile<2, 16, SIDE>::threads) / 64;
  return pb.batch * tiles * waves * pb.T;
}

template <int SIDE, int DEPTH>
hipError_t launch_noise_side(const Problem &pb, const float *src, const SideTab &cf,
                             const uint8_t *codes, const uint8_t *scales, double *partial, hipStream_t st) {
  uint8_t *c = const_cast<uint8_t *>(codes), *sc = const_cast<uint8_t *>(scales);
  const bool f32 = pb.rule == dev::RULE_FP32_AMAX;
  switch (pb.block) {
    case 16: return f32 ? launch16<SIDE, DEPTH, 16, true, 3>(pb, src, cf, c, sc, st, partial)
                        : launch16<SIDE, DEPTH, 16, false, 3>(pb, src, cf, c, sc, st, partial);
    case 32: return f32 ? launch16<SIDE, DEPTH, 32, true, 3>(pb, src, cf, c, sc, st, partial)
                        : launch16<SIDE, DEPTH, 32, false, 3>(pb, src, cf, c, sc, st, partial);
    case 128: return f32 ? launch16<SIDE, DEPTH, 128, true, 3>(pb, src, cf, c, sc, st, partial)
                         : launch16<SIDE, DEPTH, 128, false, 3>(pb, src, cf, c, sc, st, partial);
  }
  return hipErrorInvalidValue;
}

// out[(bt * 2 + side) * T + r][q] = sum over the side's tiles and waves of
// partial[((bt * tiles + tile) * waves + wave) * T + r][q], in that order.
__global__ __launch_bounds__(256) void noise_reduce_kernel(const double *__restrict__ partial, double *__restrict__ out,
                                                           int64_t batch, int64_t T, int64_t per_bt, int side) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;     // (bt, r, q)
  if (i >= batch * T * 2) return;
  const int64_t q = i & 1, r = (i >> 1) % T, bt = (i >> 1) / T;
  double s = 0.0;
  const double *p = partial + (bt * per_bt * T + r) * 2 + q;
  for (int64_t k = 0; k < per_bt; ++k) s += p[k * T * 2];
  out[((bt * 2 + side) * T + r) * 2 + q] = s;
}

}  // namespace

size_t encode_noise_scratch_bytes(const Problem &pb) {
  if (pb.depth > 2) return 0;
  return (size_t)(noise_slots<0>(pb) + noise_slots<1>(pb)) * 2 * sizeof(double);
}

int launch_encode_noise(const Problem &pb, const DeviceTables &tab, const float *A, const float *B,
                        const uint8_t *ws, const Workspace &wl, double *out, void *scratch, void *stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (pb.batch == 0 || pb.T == 0) return hipSuccess;
  double *pa = reinterpret_cast<double *>(scratch);
  double *pbp = pa + noise_slots<0>(pb) * 2;
  const int64_t n = (noise_slots<0>(pb) + noise_slots<1>(pb)) * 2;
  // slots a wave does not own (depth 2 deals terms out over the waves) must read as zero
  hipLaunchKernelGGL(zero_u32_kernel, dim3((unsigned)std::min<int64_t>((2 * n + 255) / 256, 4096)), dim3(256), 0, st,
                     reinterpret_cast<uint32_t *>(scratch), 2 * n);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (pb.M > 0 && pb.K > 0) {
    e = pb.depth == 1 ? launch_noise_side<0, 1>(pb, A, a_tab(tab), ws + wl.a_codes, ws + wl.a_scales, pa, st)
                      : launch_noise_side<0, 2>(pb, A, a_tab(tab), ws + wl.a_codes, ws + wl.a_scales, pa, st);
    if (e != hipSuccess) return e;
  }
  if (pb.N > 0 && pb.K > 0) {
    e = pb.depth == 1 ? launch_noise_side<1, 1>(pb, B, b_tab(tab), ws + wl.b_codes, ws + wl.b_scales, pbp, st)
                      : launch_noise_side<1, 2>(pb, B, b_tab(tab), ws + wl.b_codes, ws + wl.b_scales, pbp, st);
    if (e != hipSuccess) return e;
  }
  const int64_t tot = pb.batch * pb.T * 2;
  const dim3 g((unsigned)((tot + 255) / 256));
  hipLaunchKernelGGL(noise_reduce_kernel, g, dim3(256), 0, st, pa, out, pb.batch, pb.T, noise_slots<0>(pb) / (pb.batch * pb.T), 0);
  hipLaunchKernelGGL(noise_reduce_kernel, g, dim3(256), 0, st, pbp, out, pb.batch, pb.T, noise_slots<1>(pb) / (pb.batch * pb.T), 1);
  return hipGetLastError();
}


int launch_encode(const Problem &pb, const DeviceTables &tab, const float *A, const float *B,
                  uint8_t *ws, const Workspace &wl, void *stream) {
  if (pb.batch == 0 || pb.M == 0 || pb.N == 0 || pb.K == 0) return hipSuccess;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = launch_side<0>(pb, A, a_tab(tab), ws + wl.a_codes, ws + wl.a_scales, st);
  if (e != hipSuccess) return e;
  if (pb.b_rows > 1 || pb.b_bf16)
    return launch_b_deploy_any(pb, B, b_tab(tab), ws + wl.b_codes, ws + wl.b_scales,
                               reinterpret_cast<uint32_t *>(ws + wl.b_amax), st);
  return launch_side<1>(pb, B, b_tab(tab), ws + wl.b_codes, ws + wl.b_scales, st);
}

}  // namespace fmm
