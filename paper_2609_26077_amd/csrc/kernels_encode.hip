// Fused operand combine + block quantization (the encoder of Assumption 1).
//
// One workgroup owns a tile of TR "rows" x TL contracted positions of the
// sub-block grid and produces the codes and scales of every flattened term
// for that tile.  A rows are rows of A's sub-blocks; B rows are columns of
// B's sub-blocks, so both outputs have the contracted axis last.
//
//   1. stage: the tile of all 4^l sub-blocks is read from HBM (coalesced)
//      into LDS as fp32, laid out [block][row][l] with the contracted axis
//      contiguous (the B side transposes on the way in);
//   2. combine: a wave takes 64 items (row, 4 consecutive l) of one term; each
//      lane forms x = sum_b c_b a_b over the term's nonzero coefficients in
//      ascending b, as separate fp32 multiplies and adds (the coefficients of a
//      term are read once into scalar registers when a tile holds enough
//      positions per term);
//   3. quantize: the block maximum over `block` consecutive l is reduced
//      across the block/4 lanes that hold it, the rule gives the scale, the
//      lane divides and casts its four values and stores one word of codes.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "device.h"
#include "internal.h"

namespace fmm {

namespace {

constexpr int kThreads = 256;
constexpr int kTL = 128;            // contracted positions per tile (>= every block size)
constexpr int kStride = kTL + 4;    // LDS row stride in floats (conflict-free transposed writes)

template <int DEPTH>
struct Tile {
  static constexpr int nblk = 1 << (2 * DEPTH);
  static constexpr int TR = DEPTH == 3 ? 2 : 64 / nblk;   // 16, 4, 2 rows
  static constexpr int lds_floats = nblk * TR * kStride;  // 33.8, 33.8, 67.6 KB
  // a wave's 64 consecutive items must belong to one term
  static_assert((TR * (kTL / 4)) % 64 == 0, "positions per term must fill whole waves");
};

// max over each group of gl aligned lanes (gl = block / 4: 4, 8 or 32), every
// lane receiving its group's maximum: quad permutations (xor 1, xor 2), then
// the half-row and row mirrors, then across the two rows of 32 lanes.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float group_max(float m, int gl) {
  m = fmaxf(m, dpp<0xB1>(m));        // quad_perm [1, 0, 3, 2]
  m = fmaxf(m, dpp<0x4E>(m));        // quad_perm [2, 3, 0, 1]
  if (gl >= 8) m = fmaxf(m, dpp<0x141>(m));   // row_half_mirror: lane i <- 7 - i within 8
  if (gl >= 16) m = fmaxf(m, dpp<0x140>(m));  // row_mirror: lane i <- 15 - i within 16
  if (gl >= 32) m = fmaxf(m, __shfl_xor(m, 16, 64));
  return m;
}

template <int SIDE, int DEPTH>
__global__ __launch_bounds__(kThreads) void encode_kernel(
    const float *__restrict__ src, Problem pb, const int32_t *__restrict__ off,
    const CoefEntry *__restrict__ ent, uint8_t *__restrict__ codes, uint8_t *__restrict__ scales,
    int64_t tiles_l) {
  using TT = Tile<DEPTH>;
  constexpr int TR = TT::TR;
  constexpr int NB = TT::nblk;
  constexpr int n = 1 << DEPTH;
  __shared__ float4 lds4[TT::lds_floats / 4];
  float *lds = reinterpret_cast<float *>(lds4);

  const int t = threadIdx.x;
  const int64_t bt = blockIdx.y;                         // batch element
  const int64_t tile = blockIdx.x;
  const int64_t row0 = (tile / tiles_l) * TR;
  const int64_t l0 = (tile % tiles_l) * kTL;
  const int64_t rows = SIDE == 0 ? pb.mp : pb.np;        // rows of the output
  const int64_t kp = pb.kp;

  // ---- 1. stage the tile ----------------------------------------------------
  // every load of the tile is issued before the first LDS write, so the
  // workgroup waits for HBM once, not once per element
  constexpr int kPerThread = NB * TR * (kTL / 4) / kThreads;   // float4s per thread
  static_assert(NB * TR * (kTL / 4) % kThreads == 0, "the tile splits evenly over the threads");
  float4 stage[kPerThread];
  if (SIDE == 0) {
    // A (M x K): block b = I n + J holds rows I m' + p, columns J k' + l.
    const float *Ab = src + bt * pb.M * pb.K;
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
      const int e = t + kThreads * k;
      const int b = e / (TR * (kTL / 4));
      const int rem = e % (TR * (kTL / 4));
      const int r = rem / (kTL / 4);
      const int c4 = rem % (kTL / 4);
      const int64_t p = row0 + r, l = l0 + 4 * c4;
      stage[k] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (p < rows && l < kp) {
        const int I = b / n, J = b % n;
        stage[k] = *reinterpret_cast<const float4 *>(Ab + (I * pb.mp + p) * pb.K + J * kp + l);
      }
    }
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
      const int e = t + kThreads * k;
      const int b = e / (TR * (kTL / 4));
      const int rem = e % (TR * (kTL / 4));
      *reinterpret_cast<float4 *>(lds + (b * TR + rem / (kTL / 4)) * kStride + 4 * (rem % (kTL / 4))) = stage[k];
    }
  } else {
    // B (K x N): block b = J n + K holds rows J k' + l, columns K n' + q;
    // lanes run along q so each of the four loads is coalesced.
    const float *Bb = src + bt * pb.K * pb.N;
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
      const int e = t + kThreads * k;
      const int b = e / (TR * (kTL / 4));
      const int rem = e % (TR * (kTL / 4));
      const int q = rem % TR;
      const int c4 = rem / TR;
      const int64_t qq = row0 + q, l = l0 + 4 * c4;
      stage[k] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (qq < rows && l < kp) {
        const int J = b / n, Kb = b % n;
        const float *p = Bb + (J * kp + l) * pb.N + Kb * pb.np + qq;
        stage[k].x = p[0];
        stage[k].y = p[pb.N];
        stage[k].z = p[2 * pb.N];
        stage[k].w = p[3 * pb.N];
      }
    }
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
      const int e = t + kThreads * k;
      const int b = e / (TR * (kTL / 4));
      const int rem = e % (TR * (kTL / 4));
      *reinterpret_cast<float4 *>(lds + (b * TR + rem % TR) * kStride + 4 * (rem / TR)) = stage[k];
    }
  }
  __syncthreads();

  // ---- 2./3. combine and quantize ----------------------------------------------
  constexpr int P = TR * (kTL / 4);          // positions (row, 4 consecutive l) per term
  const int64_t T = pb.T;
  const int gl = pb.block / 4;               // lanes per block
  const int64_t kb_count = pb.kblocks;

  // one (term, position) item: combine, block maximum, scale, cast, store.
  // The values of a group of up to four coefficients are all read before any
  // arithmetic, then x += c * tile[b][row][4 c4 .. +3] in ascending b as
  // separate multiplies and adds (the first term is a plain product).
  auto combine = [&](int n, const CoefEntry *ce, int row, int c4, float &x0, float &x1, float &x2,
                     float &x3, auto reg) {
    constexpr int G = decltype(reg)::value ? NB : 4;
    for (int e0 = 0; e0 < n; e0 += G) {
      float4 v[G];
#pragma unroll
      for (int e = 0; e < G; ++e)
        if (e0 + e < n) v[e] = *reinterpret_cast<const float4 *>(lds + (ce[e0 + e].block * TR + row) * kStride + 4 * c4);
#pragma unroll
      for (int e = 0; e < G; ++e) {
        if (e0 + e < n) {
          const float c = ce[e0 + e].coef;
          const float t0 = __fmul_rn(c, v[e].x), t1 = __fmul_rn(c, v[e].y);
          const float t2 = __fmul_rn(c, v[e].z), t3 = __fmul_rn(c, v[e].w);
          if (e0 + e == 0) {
            x0 = t0; x1 = t1; x2 = t2; x3 = t3;
          } else {
            x0 = __fadd_rn(x0, t0); x1 = __fadd_rn(x1, t1);
            x2 = __fadd_rn(x2, t2); x3 = __fadd_rn(x3, t3);
          }
        }
      }
      if (decltype(reg)::value) break;   // NB >= n: one group holds every coefficient
    }
  };

  // Where the results of one position go, inside one term's plane: a thread's
  // positions are the same for every term it handles, so this is computed once.
  //   codes : row-major p k' + l, or (large-tile plans) the 256-row x 64-byte
  //           tile image, chunk c of tile row t at c ^ ((t >> 2) & 3)
  //   scales: row-major p kblocks + kb, or (large-tile plans) K-block-major with
  //           rows permuted inside each 256-row tile: row 128 wm + 32 i + r at
  //           byte 4 (32 wm + r) + i of the tile
  //   128 x 128 tiles: codes as the 128-row x 128-byte tile image (chunk c of
  //           tile row t at c ^ (t & 7) ^ ((t >> 3) & 1)); scales 4 bytes per
  //           tile row and 128-byte step (blocks 0, 2, 1, 3 at block 32; the
  //           one block repeated at block 128)
  struct Out {
    int64_t code, scale;
    bool valid, leader;
  };
  auto out_of = [&](int pos) {
    Out o;
    const int row = pos / (kTL / 4), c4 = pos % (kTL / 4);
    const int64_t p = row0 + row, l = l0 + 4 * c4;
    o.valid = p < rows && l < kp;
    o.leader = o.valid && (c4 % gl) == 0;
    const int64_t kb = l / pb.block;
    if (pb.layout == FMM_LAYOUT_TILE256x64) {
      const int64_t t = p & 255, c = (l >> 4) & 3;
      o.code = ((((p >> 8) * (kp >> 6) + (l >> 6)) << 14) + t * 64 + 16 * (c ^ ((t >> 2) & 3)) + (l & 15));
      o.scale = kb * rows + ((p & ~int64_t(255)) | ((((p >> 7) & 1) * 32 + (p & 31)) * 4 + ((p >> 5) & 3)));
    } else if (pb.layout == FMM_LAYOUT_TILE128x128) {
      const int64_t t = p & 127, c = (l >> 4) & 7, tile = (p >> 7) * (kp >> 7) + (l >> 7);
      o.code = (tile << 14) + t * 128 + 16 * (c ^ (t & 7) ^ ((t >> 3) & 1)) + (l & 15);
      const int64_t kq = (l >> 5) & 3;                       // block of the step (block 32)
      o.scale = tile * 512 + t * 4 + (pb.block == 32 ? ((kq & 1) << 1) | (kq >> 1) : 0);
    } else {
      o.code = p * kp + l;
      o.scale = p * kb_count + kb;
    }
    return o;
  };
  // elements of scales per (batch, term) plane (the 128 x 128 layout keeps 4 bytes per row and step)
  const int64_t code_plane = rows * kp;
  const int64_t scale_plane = pb.layout == FMM_LAYOUT_TILE128x128 ? rows * (kp / 128) * 4 : rows * kb_count;

  // one (term, position) item: combine, block maximum, scale, cast, store.
  // REG: the term's coefficients sit in a register array indexed by compile-time e.
  auto item = [&](int64_t r, int pos, const Out &o, int n, const CoefEntry *ce, auto reg) {
    const int row = pos / (kTL / 4);
    const int c4 = pos % (kTL / 4);
    float x0 = 0.f, x1 = 0.f, x2 = 0.f, x3 = 0.f;
    combine(n, ce, row, c4, x0, x1, x2, x3, reg);
    // block maximum across the gl lanes of this block (all lanes take part)
    const float m = group_max(fmaxf(fmaxf(fabsf(x0), fabsf(x1)), fmaxf(fabsf(x2), fabsf(x3))), gl);
    const dev::Scale sc = dev::block_scale(m, pb.rule);
    const uint32_t w = dev::e4m3_pack4(dev::scaled(x0, sc, pb.rule), dev::scaled(x1, sc, pb.rule),
                                       dev::scaled(x2, sc, pb.rule), dev::scaled(x3, sc, pb.rule));
    const int64_t plane = bt * T + r;
    if (o.valid) *reinterpret_cast<uint32_t *>(codes + plane * code_plane + o.code) = w;
    if (o.leader) {
      if (pb.scale_bytes == 4)
        reinterpret_cast<uint32_t *>(scales)[plane * scale_plane + o.scale] = sc.stored;
      else if (pb.layout == FMM_LAYOUT_TILE128x128 && pb.block == 128)
        *reinterpret_cast<uint32_t *>(scales + plane * scale_plane + o.scale) = sc.stored * 0x01010101u;
      else
        scales[plane * scale_plane + o.scale] = (uint8_t)sc.stored;
    }
  };

  if constexpr (P >= kThreads) {
    // term-outer: the term's nonzero coefficients are read once into SGPRs
    Out outs[P / kThreads];
#pragma unroll
    for (int pp = 0; pp < P / kThreads; ++pp) outs[pp] = out_of(t + kThreads * pp);
    for (int64_t r = 0; r < T; ++r) {
      const int beg = __builtin_amdgcn_readfirstlane(off[r]);
      const int n = __builtin_amdgcn_readfirstlane(off[r + 1]) - beg;
      CoefEntry ce[NB];
#pragma unroll
      for (int e = 0; e < NB; ++e)
        if (e < n) ce[e] = ent[beg + e];
#pragma unroll
      for (int pp = 0; pp < P / kThreads; ++pp) item(r, t + kThreads * pp, outs[pp], n, ce, std::true_type{});
    }
  } else {
    // few positions per term: a wave takes 64 consecutive items (one term);
    // kThreads is a multiple of P, so a thread's position is t % P throughout
    static_assert(kThreads % P == 0, "a thread keeps one position");
    const Out o = out_of(t % P);
    for (int64_t it = t; it < T * P; it += kThreads) {
      const int64_t r = __builtin_amdgcn_readfirstlane((int)(it / P));
      const int beg = __builtin_amdgcn_readfirstlane(off[r]);
      const int n = __builtin_amdgcn_readfirstlane(off[r + 1]) - beg;
      item(r, t % P, o, n, ent + beg, std::false_type{});
    }
  }
}

template <int SIDE, int DEPTH>
hipError_t launch_side(const Problem &pb, const float *src, const int32_t *off,
                       const CoefEntry *ent, uint8_t *codes, uint8_t *scales, hipStream_t st) {
  const int64_t rows = SIDE == 0 ? pb.mp : pb.np;
  const int64_t tiles_l = (pb.kp + kTL - 1) / kTL;
  const int64_t tiles_r = (rows + Tile<DEPTH>::TR - 1) / Tile<DEPTH>::TR;
  const dim3 grid((unsigned)(tiles_l * tiles_r), (unsigned)pb.batch);
  hipLaunchKernelGGL((encode_kernel<SIDE, DEPTH>), grid, dim3(kThreads), 0, st, src, pb, off,
                     ent, codes, scales, tiles_l);
  return hipGetLastError();
}

template <int SIDE>
hipError_t launch_depth(const Problem &pb, const float *src, const int32_t *off,
                        const CoefEntry *ent, uint8_t *codes, uint8_t *scales, hipStream_t st) {
  switch (pb.depth) {
    case 1: return launch_side<SIDE, 1>(pb, src, off, ent, codes, scales, st);
    case 2: return launch_side<SIDE, 2>(pb, src, off, ent, codes, scales, st);
    case 3: return launch_side<SIDE, 3>(pb, src, off, ent, codes, scales, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace

int launch_encode(const Problem &pb, const DeviceTables &tab, const float *A, const float *B,
                  uint8_t *ws, const Workspace &wl, void *stream) {
  if (pb.batch == 0 || pb.M == 0 || pb.N == 0 || pb.K == 0) return hipSuccess;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = launch_depth<0>(pb, A, tab.a_off, tab.a_ent, ws + wl.a_codes, ws + wl.a_scales, st);
  if (e != hipSuccess) return e;
  return launch_depth<1>(pb, B, tab.b_off, tab.b_ent, ws + wl.b_codes, ws + wl.b_scales, st);
}

}  // namespace fmm
