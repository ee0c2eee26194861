// Large-tile sub-products for tile-aligned block-scaled problems at depths 1 and 2.
//
// The sub-products are the dominant cost; each is a plain block-scaled fp8
// GEMM P_r = A_r B_r^T with fp32 accumulation.  Large tiles cut the operand
// bytes per MFMA flop of a 128 x 128 tile, which is what bounds the feed from
// L2 into LDS; the price is that P_r leaves the workgroup, so the W-combine
// becomes its own bandwidth-bound pass:
//
//   1. gemm_tile256x256_kernel: one workgroup per (batch, term r, 256 x 256
//      tile), eight waves of 128 x 64 (4 x 2 MFMA tiles of 32 x 32, 128
//      accumulation registers each), two per SIMD, one workgroup per CU.
//      64-byte K steps run through a four-slot LDS ring filled by
//      global_load_lds two steps ahead, one barrier per step; P_r is stored
//      in fp32 with nontemporal stores.  Against 256 x 128 tiles (two
//      four-wave workgroups per CU) the L2 -> LDS bytes per flop drop by a
//      third: 8192^3 sub-products 0.47 -> 0.40 ms.
//      Exact-dot plans take gemm_dq256x128_kernel (E8M0 scales: each block's
//      power of two folded into the codes' conversion to bf16) or
//      gemm_exact256x128_kernel (fp32 scales: per-block partial sums promoted
//      in fp32) instead, on the same tiles and layouts.
//   2. combine1_kernel: C block (i, k) = sum_r w[r][2k + i] P_r, ascending r,
//      one fused multiply-add per nonzero weight (the order of the fused
//      W-combine of the 128 x 128 path); combine2_kernel the same over the
//      T = R^2 flattened terms and 16 blocks of depth 2.
//
// P is stored [batch][m'][T][n']: the T terms of one output row sit in
// consecutive n'-float rows, so the W-combine, which reads all T values of a
// position, streams one region of HBM instead of T planes far apart (a probe
// of the depth-2 pattern, 49 terms into 16 outputs: 5.1 TB/s from planes,
// 5.9-6.1 TB/s with the terms interleaved in 4-64 KB pieces).
//
// Scales of these plans are stored K-block-major by the encoder: for each
// (term, K block) the E8M0 bytes of all rows, permuted inside every 256-row
// tile so that row 128 wm + 32 i + r sits at byte 4 (32 wm + r) + i.  One
// 32-bit LDS read then gives a lane the scales of its four A row tiles (or,
// shifted by 16 (wn & 1) bits, of its two B row tiles), and the MFMA's op_sel
// picks the byte of each tile.  A 128-row B tile is one half of a 256-row
// tile: the contiguous 8 KB half of each code image and the contiguous 128
// bytes 128 h .. 128 h + 127 of each K block's scales.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "device.h"
#include "internal.h"
#include "lds_dma.h"

namespace fmm {

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float f4v __attribute__((ext_vector_type(4)));

constexpr int TM = kSplitTile;        // tile rows of A_r (and rows of one code image)
constexpr int TN = kSplitTileN;       // tile rows of B_r: half an image
constexpr int SK = 64;                // contracted bytes per step
constexpr int kCodeA = TM * SK;       // 16 KB of A codes per step
constexpr int kImage = TM * SK;       // one (256-row tile, k-step) code image

// the fp8 kernel: 256 A rows x 256 B rows (a whole B code image) per tile
namespace big {
constexpr int TNB = 2 * TN;
constexpr int kThreadsB = 512;
constexpr int kSlotsB = 4;
constexpr int kCodeB = TNB * SK;                     // 16 KB of B codes per step
constexpr int kScaleA = 2 * TM, kScaleB = 2 * TNB;   // two K blocks x 256 rows each side
constexpr int kSlot = kCodeA + kCodeB + kScaleA + kScaleB;   // 33792 B
static_assert(kSlotsB * kSlot <= 160 * 1024, "one workgroup per CU");
}  // namespace big

// the exact-dot kernels: 256 A rows x 128 B rows (half an image) per tile
constexpr int kThreads = 256;
constexpr int kSlots = 3;
constexpr int kCodeB = TN * SK;       // 8 KB of B codes per step

struct SplitArgs {
  const uint8_t *xa, *xb;      // codes [batch][T][rows / 256][kp / 64][256 x 64 tile image]
  const uint8_t *sat, *sbt;    // scales [batch][T][kblocks][rows] (rows permuted per 256-row tile)
  float *P;                    // products [batch][mp][T][np]: the T terms of a row adjacent
  int64_t mp, np, kp, kblocks, T;
  int tiles_m, tiles_n;        // mp / 256, np / 128
};

// LDS image of one operand: rows x 64 bytes; 16-byte chunk c of row r sits
// at chunk c ^ ((r >> 2) & 3), so the 16 rows of a 16-lane fragment read fall
// on 16 distinct bank groups of the 64 banks.  The encoder writes the codes of
// these plans in exactly this image, one contiguous 16 KB block per
// (term, 256-row tile, 64-byte k-step).
__device__ __forceinline__ int swz64(int row, int chunk) {
  return row * SK + 16 * (chunk ^ ((row >> 2) & 3));
}

// 32 rows x 64 bytes of one operand for v_mfma_scale_f32_32x32x64_f8f6f4:
// lane (r, h) holds bytes [16h, 16h+16) and [32+16h, 32+16h+16) of row r.
__device__ __forceinline__ v8i frag64(const uint8_t *lt, int row, int h) {
  const uint4 lo = *reinterpret_cast<const uint4 *>(lt + swz64(row, h));
  const uint4 hi = *reinterpret_cast<const uint4 *>(lt + swz64(row, 2 + h));
  v8i f;
  f[0] = (int)lo.x; f[1] = (int)lo.y; f[2] = (int)lo.z; f[3] = (int)lo.w;
  f[4] = (int)hi.x; f[5] = (int)hi.y; f[6] = (int)hi.z; f[7] = (int)hi.w;
  return f;
}

struct Frags {
  v8i a[4], b[2];
  uint32_t sa, sb;     // scale bytes of the row tiles (byte i = A tile i, byte j = B tile j)
};

// Work order: workgroups are dispatched round-robin over the eight XCDs, so
// the ids of one XCD (bid, bid + 8, ...) are given a contiguous range of work
// items; items run term-major, and the tiles of a term in groups of GM
// tile-rows, so the workgroups resident on an XCD share A and B rows in L2.
template <int GM = 8>
__device__ __forceinline__ void work_of(int bid, int64_t nitems, int64_t T, int tiles_m, int tiles_n,
                                        int64_t &bt, int64_t &r, int &tm, int &tn) {
  int64_t id = bid;
  if ((nitems & 7) == 0) id = (int64_t)(bid & 7) * (nitems >> 3) + (bid >> 3);
  const int64_t ntiles = (int64_t)tiles_m * tiles_n;
  bt = id / (T * ntiles);
  const int64_t rem = id - bt * T * ntiles;
  r = rem / ntiles;
  const int tile = (int)(rem - r * ntiles);
  const int per_group = GM * tiles_n;
  const int group = tile / per_group;
  const int first_m = group * GM;
  const int gm = min(tiles_m - first_m, GM);
  const int in = tile - group * per_group;
  tm = first_m + in % gm;
  tn = in / gm;
}

template <int BS>
__global__ __launch_bounds__(big::kThreadsB, 1) void gemm_tile256x256_kernel(SplitArgs g) {
  __shared__ uint4 lds_raw[big::kSlotsB * big::kSlot / 16];
  const uint8_t *lds = reinterpret_cast<const uint8_t *>(lds_raw);
  const uint32_t lds_base = dma::lds_addr(lds_raw);
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wm = wave >> 2, wn = wave & 3;       // A rows 128 wm.., B rows 64 wn.. of the tile
  const int r32 = lane & 31, h = lane >> 5;
  const int64_t nitems = (int64_t)gridDim.x;
  const int tiles_nb = g.tiles_n / 2;            // 256-row B tiles
  int64_t bt, r;
  int tm, tn;
  work_of<4>(blockIdx.x, nitems, g.T, g.tiles_m, tiles_nb, bt, r, tm, tn);
  const int64_t pm0 = (int64_t)tm * TM, pn0 = (int64_t)tn * big::TNB;
  const int nk = (int)(g.kp / SK);
  // codes arrive tiled: the image of (256-row tile, k-step) is contiguous, so a
  // transfer is a straight 1 KB copy (lane l moves bytes 16 l .. 16 l + 15)
  const uint8_t *xa = g.xa + ((bt * g.T + r) * g.tiles_m + tm) * (int64_t)nk * kImage;
  const uint8_t *xb = g.xb + ((bt * g.T + r) * tiles_nb + tn) * (int64_t)nk * kImage;
  const uint32_t code_off = 16u * (uint32_t)lane;
  // the four 1 KB regions wave w moves each step: 4 w .. 4 w + 3 of the
  // slot's codes, 0..15 from A's image, 16..31 from B's
  const uint8_t *csrc[4];
  uint32_t cdst[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int region = wave * 4 + j;
    csrc[j] = region < 16 ? xa + region * 1024 : xb + (region - 16) * 1024;
    cdst[j] = (uint32_t)(region < 16 ? region * 1024 : kCodeA + (region - 16) * 1024);
  }
  // one scale transfer per wave and step (256 bytes, lane l moves 4): wave w
  // moves side (w >> 1) & 1 (A, B), K block 2 step + (w & 1) (block 32) or
  // step / 2 (block 128), all 256 rows of the tile; waves 4..7 repeat 0..3
  const int sside = (wave >> 1) & 1, sblk = wave & 1;
  const int64_t srows = sside ? g.np : g.mp;
  const uint8_t *ssrc = sside ? g.sbt + (bt * g.T + r) * g.kblocks * g.np + pn0
                              : g.sat + (bt * g.T + r) * g.kblocks * g.mp + pm0;
  const uint32_t s_off = 4u * (uint32_t)lane + (BS == 32 ? (uint32_t)(sblk * srows) : 0u);
  const uint32_t sdst = (uint32_t)(kCodeA + big::kCodeB + (sside ? big::kScaleA : 0) + (BS == 32 ? sblk * TM : 0));

  auto issue = [&](int step) {
    const uint32_t m0 = lds_base + (uint32_t)(step % big::kSlotsB) * big::kSlot;
    const int64_t src = (int64_t)step * kImage;
#pragma unroll
    for (int j = 0; j < 4; ++j) dma::copy16(code_off, csrc[j] + src, m0 + cdst[j]);
    const int64_t kb = BS == 32 ? 2 * (int64_t)step : step / 2;
    dma::copy4(s_off, ssrc + kb * srows, m0 + sdst);
  };

  // LDS -> registers for one step (any step index reads in bounds)
  auto load = [&](int step, Frags &f) {
    const uint8_t *la = lds + (step % big::kSlotsB) * big::kSlot;
    const uint8_t *lb = la + kCodeA;
    const uint8_t *ls = lb + big::kCodeB;
    // block 2 step + h (block 32) or step / 2: tile row 128 H + 32 I + J at byte 4 (32 H + J) + I;
    // A: H = wm, I = i; B row 64 wn + 32 j + r32: H = wn >> 1, I = 2 (wn & 1) + j
    f.sa = *reinterpret_cast<const uint32_t *>(ls + (BS == 32 ? h * TM : 0) + 4 * (wm * 32 + r32));
    f.sb = *reinterpret_cast<const uint32_t *>(ls + big::kScaleA + (BS == 32 ? h * big::TNB : 0) + 4 * (32 * (wn >> 1) + r32))
           >> (16 * (wn & 1));
#pragma unroll
    for (int i = 0; i < 4; ++i) f.a[i] = frag64(la, wm * 128 + 32 * i + r32, h);
#pragma unroll
    for (int j = 0; j < 2; ++j) f.b[j] = frag64(lb, wn * 64 + 32 * j + r32, h);
  };

  v16f acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = (v16f){};

  auto mfma = [&](const Frags &f) {
#define FMM_MFMA_IJ(I, J)                                                                     \
  acc[I][J] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(f.a[I], f.b[J], acc[I][J], 0, 0, \
                                                              I, (int)f.sa, J, (int)f.sb)
    FMM_MFMA_IJ(0, 0); FMM_MFMA_IJ(0, 1); FMM_MFMA_IJ(1, 0); FMM_MFMA_IJ(1, 1);
    FMM_MFMA_IJ(2, 0); FMM_MFMA_IJ(2, 1); FMM_MFMA_IJ(3, 0); FMM_MFMA_IJ(3, 1);
#undef FMM_MFMA_IJ
  };

  // Step s: wait for this wave's own transfers of step s (five a step; those
  // of step s + 1 may stay in flight), barrier (every wave's transfers of s
  // have landed, and every wave has read step s - 1), start step s + 2 into
  // the slot of step s - 2, read step s, multiply.
  issue(0);
  if (nk > 1) issue(1);
  for (int step = 0; step < nk; ++step) {
    if (step + 1 < nk) dma::wait_vmcnt<5>(); else dma::wait_vmcnt<0>();
    __syncthreads();
    if (step + 2 < nk) issue(step + 2);
    Frags f;
    load(step, f);
    mfma(f);
  }

  // P_r tile: lane l, register e of MFMA tile (i, j) holds row 8 (e / 4) + 4 h + e % 4, column l % 32.
  // The stores are nontemporal: P_r is read once, by the W-combine, and
  // caching it only displaces the codes the other workgroups still read.
  const int64_t pstride = g.T * g.np;                     // one row of P: all T terms
  float *out = g.P + ((bt * g.mp + pm0 + wm * 128) * g.T + r) * g.np + pn0 + wn * 64 + r32;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = 32 * i + 8 * (e >> 2) + 4 * h + (e & 3);
        __builtin_nontemporal_store(acc[i][j][e], out + (int64_t)row * pstride + 32 * j);
      }
}

// ---------------------------------------------------------------------------
// Exact-dot large-tile sub-products with power-of-two (E8M0) scales, blocks
// 16, 32 and 128: the dequantized operands themselves on the bf16 matrix
// cores.
//
// v_cvt_scalef32_pk_bf16_fp8 multiplies a code by the power of two its scale
// operand holds while converting it: code 2^e has at most four significant
// bits and, for every scale the rules produce (e in [-48, 120]) and every
// code below 256 2^e at e = 120, lies in the normal bf16 range, so the
// converted value is the dequantized operand exactly.  The product of two
// such values is exact in fp32, and v_mfma_f32_32x32x16_bf16 sums them
// across the whole contracted axis at fp32 grade: the fp32 accumulation of
// the dequantized products, with no per-block promote (each block's scale
// rides in its codes' conversion).
//
// Tiles of 256 x 128 (four waves of 128 x 64, two workgroups per CU: twice
// the matrix-core time per byte of the fp8 kernel, so the half-size B tile
// feeds it); a three-slot LDS ring two steps ahead, one barrier per step; the
// 64-byte K step is four bf16 instructions per 32 x 32 tile.  Instruction t of a step takes, in
// lane half h, bytes 32 (t >> 1) + 16 h + 8 (t & 1) .. + 7 of the lane's row
// on both operands (so the four instructions cover the step's 64 positions
// once each); those 8 bytes always lie in one block.  Scales per step: the
// step's K blocks (4 at block 16, 2 at block 32, the one block of two steps
// at block 128) for the 256 A rows and the 128 B rows.
namespace dq {
constexpr int kMaxBlocks = 4;                              // K blocks per step (block 16)
constexpr int kScaleA = kMaxBlocks * TM;                   // 1 KB of A scale bytes
constexpr int kScaleB = kMaxBlocks * TN;                   // 512 B of B scale bytes
constexpr int kSlot = kCodeA + kCodeB + kScaleA + kScaleB;  // 26112 B
static_assert(2 * kSlots * kSlot <= 160 * 1024, "two workgroups per CU");
}  // namespace dq

typedef __bf16 v8bfq __attribute__((ext_vector_type(8)));
typedef __bf16 v2bfq __attribute__((ext_vector_type(2)));

// eight codes (two little-endian words) -> their values times the power of
// two whose exponent field `s` carries, as bf16 (exact)
__device__ __forceinline__ v8bfq dequant8(uint32_t lo, uint32_t hi, float s) {
  const v2bfq a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)lo, s, false);
  const v2bfq b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)lo, s, true);
  const v2bfq c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)hi, s, false);
  const v2bfq d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)hi, s, true);
  v8bfq r;
  r[0] = a[0]; r[1] = a[1]; r[2] = b[0]; r[3] = b[1];
  r[4] = c[0]; r[5] = c[1]; r[6] = d[0]; r[7] = d[1];
  return r;
}

// A float whose exponent field is E8M0 byte i of word w, as the scale operand
// of v_cvt_scalef32_pk_bf16_fp8, which reads the exponent field alone (the
// neighbouring bytes in its sign and mantissa bits do not change the result)
__device__ __forceinline__ float e8m0_byte(uint32_t w, int i) {
  return __uint_as_float(i == 3 ? w >> 1 : w << (23 - 8 * i));
}

template <int BS>
__global__ __launch_bounds__(kThreads, 2) void gemm_dq256x128_kernel(SplitArgs g) {
  constexpr int NB = BS >= 64 ? 1 : 64 / BS;   // K blocks per step
  __shared__ uint4 lds_raw[kSlots * dq::kSlot / 16];
  const uint8_t *lds = reinterpret_cast<const uint8_t *>(lds_raw);
  const uint32_t lds_base = dma::lds_addr(lds_raw);
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wm = wave >> 1, wn = wave & 1;       // A rows 128 wm.., B rows 64 wn.. of the tile
  const int r32 = lane & 31, h = lane >> 5;
  const int64_t nitems = (int64_t)gridDim.x;
  int64_t bt, r;
  int tm, tn;
  work_of(blockIdx.x, nitems, g.T, g.tiles_m, g.tiles_n, bt, r, tm, tn);
  const int64_t pm0 = (int64_t)tm * TM, pn0 = (int64_t)tn * TN;
  const int hb = tn & 1;
  const int nk = (int)(g.kp / SK);
  const uint8_t *xa = g.xa + ((bt * g.T + r) * g.tiles_m + tm) * (int64_t)nk * kImage;
  const uint8_t *xb = g.xb + ((bt * g.T + r) * (g.tiles_n / 2) + (tn >> 1)) * (int64_t)nk * kImage + hb * kCodeB;
  const uint32_t code_off = 16u * (uint32_t)lane;
  const uint8_t *csrc[6];
  uint32_t cdst[6];
#pragma unroll
  for (int j = 0; j < 6; ++j) {
    const int region = wave * 6 + j;
    csrc[j] = region < 16 ? xa + region * 1024 : xb + (region - 16) * 1024;
    cdst[j] = (uint32_t)(region < 16 ? region * 1024 : kCodeA + (region - 16) * 1024);
  }
  // Two scale transfers per wave and step (4 bytes a lane):
  //   A: wave w moves the 256 bytes of the step's K block w mod NB into
  //      A slot block w mod NB (the extra waves repeat a transfer);
  //   B: lanes 32 k + r32 move the 128 bytes of K block 2 q + k into B slot
  //      block 2 q + k, q = wave mod (NB / 2) (block 128: both lane halves
  //      take the step's one block; block 32: q = 0).
  const int ablk = wave % NB;
  const int bq = NB >= 2 ? wave % (NB / 2) : 0;
  const int bblk = NB >= 2 ? 2 * bq + h : 0;
  const uint8_t *sa_src = g.sat + (bt * g.T + r) * g.kblocks * g.mp + pm0;
  const uint8_t *sb_src = g.sbt + (bt * g.T + r) * g.kblocks * g.np + pn0;   // bytes 128 hb .. of the 256-row tile
  const uint32_t sa_off = 4u * (uint32_t)lane + (uint32_t)(ablk * g.mp);
  const uint32_t sb_off = 4u * (uint32_t)r32 + (uint32_t)(bblk * g.np);
  const uint32_t sa_dst = (uint32_t)(kCodeA + kCodeB + ablk * TM);
  const uint32_t sb_dst = (uint32_t)(kCodeA + kCodeB + dq::kScaleA + 2 * bq * TN);

  auto issue = [&](int step) {
    const uint32_t m0 = lds_base + (uint32_t)(step % kSlots) * dq::kSlot;
    const int64_t src = (int64_t)step * kImage;
#pragma unroll
    for (int j = 0; j < 6; ++j) dma::copy16(code_off, csrc[j] + src, m0 + cdst[j]);
    const int64_t kb0 = BS >= 64 ? step / 2 : (int64_t)NB * step;   // first K block of the step
    dma::copy4(sa_off, sa_src + kb0 * g.mp, m0 + sa_dst);
    dma::copy4(sb_off, sb_src + kb0 * g.np, m0 + sb_dst);
  };

  v16f acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = (v16f){};

  // one step: raw 16-byte chunks c = 0, 1 (bytes 32 c + 16 h ..) of the
  // lane's rows, the scales of the blocks they lie in, four instructions
  auto step_mfma = [&](int step) {
    const uint8_t *la = lds + (step % kSlots) * dq::kSlot;
    const uint8_t *lb = la + kCodeA;
    const uint8_t *ls = lb + kCodeB;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      // K block of chunk c within the slot: block 16: 2 c + h; 32: c; 128: 0
      const int bi = BS == 16 ? 2 * c + h : (BS == 32 ? c : 0);
      const uint32_t wa = *reinterpret_cast<const uint32_t *>(ls + bi * TM + 4 * (wm * 32 + r32));
      const uint32_t wb = *reinterpret_cast<const uint32_t *>(ls + dq::kScaleA + bi * TN + 4 * r32) >> (16 * wn);
      uint4 ra[4], rb[2];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        ra[i] = *reinterpret_cast<const uint4 *>(la + swz64(wm * 128 + 32 * i + r32, 2 * c + h));
#pragma unroll
      for (int j = 0; j < 2; ++j)
        rb[j] = *reinterpret_cast<const uint4 *>(lb + swz64(wn * 64 + 32 * j + r32, 2 * c + h));
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        v8bfq fa[4], fb[2];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          fa[i] = u == 0 ? dequant8(ra[i].x, ra[i].y, e8m0_byte(wa, i)) : dequant8(ra[i].z, ra[i].w, e8m0_byte(wa, i));
#pragma unroll
        for (int j = 0; j < 2; ++j)
          fb[j] = u == 0 ? dequant8(rb[j].x, rb[j].y, e8m0_byte(wb, j)) : dequant8(rb[j].z, rb[j].w, e8m0_byte(wb, j));
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
      }
    }
  };

  // Step s: wait for this wave's own transfers of step s (eight a step;
  // those of step s + 1 may stay in flight), barrier, start step s + 2 into
  // the slot of step s - 1, multiply step s.
  issue(0);
  if (nk > 1) issue(1);
  for (int step = 0; step < nk; ++step) {
    if (step + 1 < nk) dma::wait_vmcnt<8>(); else dma::wait_vmcnt<0>();
    __syncthreads();
    if (step + 2 < nk) issue(step + 2);
    step_mfma(step);
  }

  const int64_t pstride = g.T * g.np;                     // one row of P: all T terms
  float *out = g.P + ((bt * g.mp + pm0 + wm * 128) * g.T + r) * g.np + pn0 + wn * 64 + r32;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = 32 * i + 8 * (e >> 2) + 4 * h + (e & 3);
        __builtin_nontemporal_store(acc[i][j][e], out + (int64_t)row * pstride + 32 * j);
      }
}

// ---------------------------------------------------------------------------
// Exact-dot large-tile sub-products with fp32 amax/448 scales (blocks 16, 32
// and 128).
//
// fp32 scales are arbitrary numbers, which neither the scaled fp8 MFMA nor
// the scaled conversions can apply, and the fp8 matrix cores' dot product is
// narrower than fp32; so each block's partial sum of code products is formed
// exactly on the bf16 matrix cores (e4m3 -> bf16 is exact, products of two
// codes are exact in fp32) and promoted into the fp32 accumulator as
// acc += (sA sB) partial.  Per block and output that is two
// VALU operations against `block` multiply-adds on the matrix cores, so at
// blocks 16 and 32 the promotes, not the matrix cores, bound the kernel.
//
// One workgroup of eight waves per (batch, term, 256 x 128 tile), each wave a
// 64 x 64 quarter-column (2 x 2 tiles of v_mfma_f32_32x32x16_bf16), one
// workgroup per CU.  The codes arrive through a 64-byte-step LDS ring like the
// fp8 kernel's (four slots here, two steps ahead); each slot also holds the
// step's scales: NB = max(1, 64 / block) K blocks of the 256 A rows and
// max(2, NB) of the 128 B rows (block 128: the step's one block, repeated),
// fp32 in row order.
//
// Each instruction's 16 contracted positions lie in one block, the same
// positions on both operands, so every partial sum is over exactly one block.
// Blocks 32 and 128: a lane's 16-byte read of bytes 32 c + 16 h of its row
// (c = 0, 1) feeds two instructions, bytes 32 c + 16 h + 8 t + 0..7 (t = 0, 1)
// in the lane half h, i.e. positions {8 t + 0..7, 16 + 8 t + 0..7} of the
// 32-byte group c.  Block 16: the instruction of block b takes bytes
// 16 b + 8 h + 0..7 (an 8-byte read).
namespace ex {
constexpr int kThreadsX = 512;
constexpr int kSlotsX = 4;                       // two in flight, the current one, the previous one
template <int BS>
struct Geo {
  static constexpr int SB = 4;                            // fp32 scale bytes
  static constexpr int NB = BS >= 64 ? 1 : 64 / BS;       // K blocks per step
  static constexpr int NBB = NB < 2 ? 2 : NB;             // B scale blocks held per slot
  static constexpr int kScaleA = NB * TM * SB;
  static constexpr int kScaleB = NBB * TN * SB;
  static constexpr int kSlot = kCodeA + kCodeB + kScaleA + kScaleB;
  static_assert(kSlotsX * kSlot <= 160 * 1024, "one workgroup per CU");
};
}  // namespace ex

// eight e4m3 codes (little-endian in two words) -> eight bf16, exactly
typedef __bf16 v8bfx __attribute__((ext_vector_type(8)));
typedef __bf16 v2bfx __attribute__((ext_vector_type(2)));
__device__ __forceinline__ v8bfx codes8_to_bf16(uint32_t lo, uint32_t hi) {
  const v2bfx a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)lo, 1.0f, false);
  const v2bfx b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)lo, 1.0f, true);
  const v2bfx c = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)hi, 1.0f, false);
  const v2bfx d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)hi, 1.0f, true);
  v8bfx r;
  r[0] = a[0]; r[1] = a[1]; r[2] = b[0]; r[3] = b[1];
  r[4] = c[0]; r[5] = c[1]; r[6] = d[0]; r[7] = d[1];
  return r;
}

template <int BS>
__global__ __launch_bounds__(ex::kThreadsX, 1) void gemm_exact256x128_kernel(SplitArgs g) {
  using G = ex::Geo<BS>;
  constexpr int SB = G::SB;
  constexpr int NB = G::NB;
  __shared__ uint4 lds_raw[ex::kSlotsX * G::kSlot / 16];
  const uint8_t *lds = reinterpret_cast<const uint8_t *>(lds_raw);
  const uint32_t lds_base = dma::lds_addr(lds_raw);
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wm = wave >> 1, wn = wave & 1;       // A rows 64 wm.., B rows 64 wn.. of the tile
  const int r32 = lane & 31, h = lane >> 5;
  const int64_t nitems = (int64_t)gridDim.x;
  int64_t bt, r;
  int tm, tn;
  work_of(blockIdx.x, nitems, g.T, g.tiles_m, g.tiles_n, bt, r, tm, tn);
  const int64_t pm0 = (int64_t)tm * TM, pn0 = (int64_t)tn * TN;
  const int hb = tn & 1;
  const int nk = (int)(g.kp / SK);
  const uint8_t *xa = g.xa + ((bt * g.T + r) * g.tiles_m + tm) * (int64_t)nk * kImage;
  const uint8_t *xb = g.xb + ((bt * g.T + r) * (g.tiles_n / 2) + (tn >> 1)) * (int64_t)nk * kImage + hb * kCodeB;
  const uint32_t code_off = 16u * (uint32_t)lane;
  // the three 1 KB code regions wave w moves each step: 3 w .. 3 w + 2
  const uint8_t *csrc[3];
  uint32_t cdst[3];
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    const int region = wave * 3 + j;
    csrc[j] = region < 16 ? xa + region * 1024 : xb + (region - 16) * 1024;
    cdst[j] = (uint32_t)(region < 16 ? region * 1024 : kCodeA + (region - 16) * 1024);
  }
  // one scale transfer per wave and step (16 bytes a lane):
  //   waves 0..3: the 256 A rows of K block NB step + (wave mod NB) (block
  //               128: of block step / 2; the extra waves repeat a transfer)
  //   waves 4..7: the 128 B rows of K blocks NB step + 2 p + h into lane half
  //               h, p = (wave - 4) mod (NB / 2) (blocks 32 and 128: p = 0;
  //               block 128: both halves take block step / 2)
  const bool s_is_a = wave < 4;
  const int sblk = s_is_a ? wave % NB : 2 * ((wave - 4) % (G::NBB / 2));
  const int64_t srows = s_is_a ? g.mp : g.np;
  const uint8_t *sbase = (s_is_a ? g.sat + (bt * g.T + r) * g.kblocks * g.mp * SB + pm0 * SB
                                 : g.sbt + (bt * g.T + r) * g.kblocks * g.np * SB + pn0 * SB);
  const int64_t splane = srows * SB;                   // bytes per K block
  const uint32_t s_off = 16u * (uint32_t)(s_is_a ? lane : r32);
  const uint32_t sdst = (uint32_t)(kCodeA + kCodeB + (s_is_a ? sblk * TM * SB : G::kScaleA + sblk * TN * SB));

  auto issue = [&](int step) {
    const uint32_t m0 = lds_base + (uint32_t)(step % ex::kSlotsX) * G::kSlot;
    const int64_t src = (int64_t)step * kImage;
#pragma unroll
    for (int j = 0; j < 3; ++j) dma::copy16(code_off, csrc[j] + src, m0 + cdst[j]);
    const int64_t kb = BS >= 64 ? step / 2 : (int64_t)NB * step + sblk;
    // B lanes of half h read the next block (blocks 16, 32)
    const uint32_t hoff = (!s_is_a && BS < 64) ? (uint32_t)(h * splane) : 0u;
    dma::copy16(s_off + hoff, sbase + kb * splane, m0 + sdst);
  };

  v16f acc[2][2], part[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      acc[i][j] = (v16f){};
      part[i][j] = (v16f){};
    }

  // A block's promote waits until the next block's first instructions, so
  // that its VALU work overlaps their matrix-core work.  Its scales are still
  // in LDS then: the ring has four slots and refills the one of step s - 2
  // during step s, so the previous step's slot stays intact.
  auto promote = [&](const uint8_t *slot, int blk) {
    const uint8_t *sa = slot + kCodeA + kCodeB + blk * TM * SB;
    const uint8_t *sb = slot + kCodeA + kCodeB + G::kScaleA + blk * TN * SB;
    // sB of the lane's column in column tile j
    float sbv[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) sbv[j] = reinterpret_cast<const float *>(sb)[wn * 64 + 32 * j + r32];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        // rows 64 wm + 32 i + 8 q + 4 h + u, u = 0..3: registers 4 q + u
        const float4 sa4 = *reinterpret_cast<const float4 *>(sa + 4 * (wm * 64 + 32 * i + 8 * q + 4 * h));
        const float sav[4] = {sa4.x, sa4.y, sa4.z, sa4.w};
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int u = 0; u < 4; ++u)
            acc[i][j][4 * q + u] = __fmaf_rn(sav[u] * sbv[j], part[i][j][4 * q + u], acc[i][j][4 * q + u]);
      }
    }
  };

  // one K-step.  The first instruction of a block starts from zero (an
  // inline constant: no register clears) and is preceded by the previous
  // block's promote.  FRESH: the step opens a block of 128.  prev: the
  // previous step's slot.
  auto mfma_group = [&](const v8bfx (&a)[2], const v8bfx (&b)[2], bool opens) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        part[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], opens ? (v16f){} : part[i][j], 0, 0, 0);
  };
  auto mfma_step = [&](const uint8_t *la, const uint8_t *prev, auto FRESH) {
    constexpr bool fresh = decltype(FRESH)::value;
    const uint8_t *lb = la + kCodeA;
    if (BS == 16) {
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) {
        v8bfx a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const uint2 w = *reinterpret_cast<const uint2 *>(la + swz64(wm * 64 + 32 * i + r32, blk) + 8 * h);
          a[i] = codes8_to_bf16(w.x, w.y);
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const uint2 w = *reinterpret_cast<const uint2 *>(lb + swz64(wn * 64 + 32 * j + r32, blk) + 8 * h);
          b[j] = codes8_to_bf16(w.x, w.y);
        }
        promote(blk == 0 ? prev : la, blk == 0 ? 3 : blk - 1);
        mfma_group(a, b, true);
      }
    } else {
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        // this half's 16 bytes of each fragment row (bytes 32 half + 16 h ..)
        uint4 fa[2], fb[2];
#pragma unroll
        for (int i = 0; i < 2; ++i)
          fa[i] = *reinterpret_cast<const uint4 *>(la + swz64(wm * 64 + 32 * i + r32, 2 * half + h));
#pragma unroll
        for (int j = 0; j < 2; ++j)
          fb[j] = *reinterpret_cast<const uint4 *>(lb + swz64(wn * 64 + 32 * j + r32, 2 * half + h));
#pragma unroll
        for (int tt = 0; tt < 2; ++tt) {
          const bool opens = BS == 32 ? tt == 0 : (fresh && half == 0 && tt == 0);
          v8bfx a[2], b[2];
#pragma unroll
          for (int i = 0; i < 2; ++i) a[i] = tt == 0 ? codes8_to_bf16(fa[i].x, fa[i].y) : codes8_to_bf16(fa[i].z, fa[i].w);
#pragma unroll
          for (int j = 0; j < 2; ++j) b[j] = tt == 0 ? codes8_to_bf16(fb[j].x, fb[j].y) : codes8_to_bf16(fb[j].z, fb[j].w);
          if (opens) {
            // block 32: the previous block is the other half (this step's, or
            // the previous step's second); block 128: the previous step's
            if (BS == 32) promote(half == 0 ? prev : la, half == 0 ? 1 : 0);
            else promote(prev, 0);
          }
          mfma_group(a, b, opens);
        }
      }
    }
  };

  // Step s: wait for this wave's own transfers of step s (four a step; those
  // of step s + 1 may stay in flight), barrier, start step s + 2 into the
  // slot of step s - 2, multiply step s.
  auto slot_of = [&](int step) { return lds + (step & (ex::kSlotsX - 1)) * G::kSlot; };
  auto begin_step = [&](int step) -> const uint8_t * {
    if (step + 1 < nk) dma::wait_vmcnt<4>(); else dma::wait_vmcnt<0>();
    __syncthreads();
    if (step + 2 < nk) issue(step + 2);
    return slot_of(step);
  };
  // the first block's "previous" promote reads the scales of the last slot,
  // which step 3 fills only after the first two barriers: zero them (and
  // part is zero), so that it adds 0 x 0
  {
    uint32_t *z = reinterpret_cast<uint32_t *>(lds_raw) + ((ex::kSlotsX - 1) * G::kSlot + kCodeA + kCodeB) / 4;
    for (int e = t; e < (G::kScaleA + G::kScaleB) / 4; e += ex::kThreadsX) z[e] = 0u;
  }
  issue(0);
  if (nk > 1) issue(1);
  if (BS < 64) {
    for (int step = 0; step < nk; ++step) mfma_step(begin_step(step), slot_of(step + ex::kSlotsX - 1), std::false_type{});
    promote(slot_of(nk - 1), NB - 1);
  } else {
    // a block of 128 is two steps (k' is a multiple of 128)
    for (int step = 0; step < nk; step += 2) {
      mfma_step(begin_step(step), slot_of(step + ex::kSlotsX - 1), std::true_type{});
      mfma_step(begin_step(step + 1), slot_of(step), std::false_type{});
    }
    promote(slot_of(nk - 1), 0);
  }

  // P_r tile: lane l, register e of MFMA tile (i, j) holds row 8 (e / 4) + 4 h + e % 4, column l % 32.
  const int64_t pstride = g.T * g.np;                     // one row of P: all T terms
  float *out = g.P + ((bt * g.mp + pm0 + wm * 64) * g.T + r) * g.np + pn0 + wn * 64 + r32;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = 32 * i + 8 * (e >> 2) + 4 * h + (e & 3);
        __builtin_nontemporal_store(acc[i][j][e], out + (int64_t)row * pstride + 32 * j);
      }
}

// C block (i, k) of batch element bt, rows i m' + p, columns k n' + 4 q4 .. + 3:
//   sum over r of w[r][2k + i] P_r[p][4 q4 ..], ascending r, fma per nonzero weight.
template <bool VEC>
__global__ __launch_bounds__(256) void combine1_kernel(const float *__restrict__ P, const float *__restrict__ w,
                                                       float *__restrict__ C, Problem pb) {
  const int64_t n4 = pb.np / 4;
  const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // p * n4 + q4
  const int64_t bt = blockIdx.y;
  if (pos >= pb.mp * n4) return;
  const int64_t p = pos / n4, q4 = pos - p * n4;
  float wr[kMaxRank][4];
#pragma unroll
  for (int r = 0; r < kMaxRank; ++r)
#pragma unroll
    for (int q = 0; q < 4; ++q) wr[r][q] = w[4 * r + q];   // zero-padded table
  float4 acc[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) acc[q] = make_float4(0.f, 0.f, 0.f, 0.f);
  // every term's load is issued before the first multiply-add (past the last
  // term the index is clamped and the load unused); P_r is dead after this
  // read: nontemporal, so it does not displace C in the caches
  const int T = (int)pb.T;
  const float *src = P + (bt * pb.mp + p) * pb.T * pb.np + 4 * q4;   // term r at src + r n'
  f4v xs[kMaxRank];
#pragma unroll
  for (int r = 0; r < kMaxRank; ++r)
    xs[r] = __builtin_nontemporal_load(reinterpret_cast<const f4v *>(src + min(r, T - 1) * pb.np));
#pragma unroll
  for (int r = 0; r < kMaxRank; ++r) {
    if (r < T) {
      const float4 v = make_float4(xs[r].x, xs[r].y, xs[r].z, xs[r].w);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float wq = wr[r][q];
        if (wq != 0.0f) {
          acc[q].x = __fmaf_rn(wq, v.x, acc[q].x);
          acc[q].y = __fmaf_rn(wq, v.y, acc[q].y);
          acc[q].z = __fmaf_rn(wq, v.z, acc[q].z);
          acc[q].w = __fmaf_rn(wq, v.w, acc[q].w);
        }
      }
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int i = q & 1, k = q >> 1;
    float *dst = C + bt * pb.M * pb.N + (i * pb.mp + p) * pb.N + k * pb.np + 4 * q4;
    if (VEC) {
      *reinterpret_cast<float4 *>(dst) = acc[q];
    } else {
      dst[0] = acc[q].x; dst[1] = acc[q].y; dst[2] = acc[q].z; dst[3] = acc[q].w;
    }
  }
}

// Depth 2: C block (I, K) of batch element bt, rows I m' + p, columns
// K n' + 4 q4 .. + 3, I, K < 4: sum over the T flattened terms of
// w[r][4K + I] P_r[p][4 q4 ..], ascending r, fma per nonzero weight, with the
// 16 blocks' accumulators in registers so that every P_r is read once.  The
// weights are uniform over the grid (scalar loads).
// GEN: a realization of another shape with gm gn <= 16 C blocks, block (I, L)
// at w index L gm + I of a row padded to 16; K = 0 leaves C zero.
template <bool VEC, bool GEN = false>
__global__ __launch_bounds__(256) void combine2_kernel(const float *__restrict__ P, const float *__restrict__ w,
                                                       float *__restrict__ C, Problem pb) {
  const int64_t n4 = pb.np / 4;
  const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // p * n4 + q4
  const int64_t bt = blockIdx.y;
  if (pos >= pb.mp * n4) return;
  const int64_t p = pos / n4, q4 = pos - p * n4;
  const float *src = P + (bt * pb.mp + p) * pb.T * pb.np + 4 * q4;   // term r at src + r n'
  float4 acc[16];
#pragma unroll
  for (int b = 0; b < 16; ++b) acc[b] = make_float4(0.f, 0.f, 0.f, 0.f);
  const int T = (GEN && pb.kp == 0) ? 0 : (int)pb.T;
  // eight terms' loads are issued together, ahead of the (uniformly branching)
  // multiply-adds; past the last term the index is clamped and the load unused
  for (int r0 = 0; r0 < T; r0 += 8) {
    f4v x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int r = min(r0 + j, T - 1);
      x[j] = __builtin_nontemporal_load(reinterpret_cast<const f4v *>(src + r * pb.np));
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (r0 + j < T) {
        float wr[16];   // one scalar load of the term's 16 weights
#pragma unroll
        for (int b = 0; b < 16; ++b) wr[b] = w[16 * (r0 + j) + b];
#pragma unroll
        for (int b = 0; b < 16; ++b) {
          const float wb = wr[b];
          if (wb != 0.0f) {
            acc[b].x = __fmaf_rn(wb, x[j].x, acc[b].x);
            acc[b].y = __fmaf_rn(wb, x[j].y, acc[b].y);
            acc[b].z = __fmaf_rn(wb, x[j].z, acc[b].z);
            acc[b].w = __fmaf_rn(wb, x[j].w, acc[b].w);
          }
        }
      }
    }
  }
#pragma unroll
  for (int b = 0; b < 16; ++b) {
    if (GEN && b >= pb.gm * pb.gn) continue;     // (uniform; a full unroll keeps acc in registers)
    const int i = GEN ? b % pb.gm : b & 3, k = GEN ? b / pb.gm : b >> 2;
    float *dst = C + bt * pb.M * pb.N + (i * pb.mp + p) * pb.N + k * pb.np + 4 * q4;
    if (VEC) {
      *reinterpret_cast<float4 *>(dst) = acc[b];
    } else {
      dst[0] = acc[b].x; dst[1] = acc[b].y; dst[2] = acc[b].z; dst[3] = acc[b].w;
    }
  }
}

// Another shape with 16 < gm gn <= 64 C blocks: one output column per thread
// (row p, column q of every block), the blocks' 64 accumulators in registers
// so that every P_r is read once; otherwise as combine2_kernel's GEN form.
__global__ __launch_bounds__(256) void combine64_kernel(const float *__restrict__ P, const float *__restrict__ w,
                                                        float *__restrict__ C, Problem pb) {
  const int64_t pos = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // p * np + q
  const int64_t bt = blockIdx.y;
  if (pos >= pb.mp * pb.np) return;
  const int64_t p = pos / pb.np, q = pos - p * pb.np;
  const float *src = P + (bt * pb.mp + p) * pb.T * pb.np + q;       // term r at src + r n'
  float acc[64];
#pragma unroll
  for (int b = 0; b < 64; ++b) acc[b] = 0.0f;
  const int T = pb.kp == 0 ? 0 : (int)pb.T;
  for (int r0 = 0; r0 < T; r0 += 8) {
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int r = min(r0 + j, T - 1);
      x[j] = __builtin_nontemporal_load(src + r * pb.np);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (r0 + j < T) {
#pragma unroll
        for (int b = 0; b < 64; ++b) {
          const float wb = w[64 * (r0 + j) + b];
          if (wb != 0.0f) acc[b] = __fmaf_rn(wb, x[j], acc[b]);
        }
      }
    }
  }
  const int nbc = pb.gm * pb.gn;
#pragma unroll
  for (int b = 0; b < 64; ++b) {
    if (b >= nbc) continue;
    const int i = b % pb.gm, l = b / pb.gm;
    C[bt * pb.M * pb.N + (i * pb.mp + p) * pb.N + l * pb.np + q] = acc[b];
  }
}

}  // namespace

int launch_products_split(const Problem &pb, const uint8_t *ws, const Workspace &wl, void *stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (pb.kp == 0) return hipSuccess;    // plans of other shapes with K = 0: the W-combine writes C = 0
  SplitArgs g;
  g.xa = ws + wl.a_codes;
  g.xb = ws + wl.b_codes;
  g.sat = ws + wl.a_scales;
  g.sbt = ws + wl.b_scales;
  g.P = reinterpret_cast<float *>(const_cast<uint8_t *>(ws) + wl.products);
  g.mp = pb.mp; g.np = pb.np; g.kp = pb.kp; g.kblocks = pb.kblocks; g.T = pb.T;
  g.tiles_m = (int)(pb.mp / TM);
  g.tiles_n = (int)(pb.np / TN);
  const int64_t items = pb.batch * pb.T * g.tiles_m * g.tiles_n;
  if (exact_split(pb)) {
    if (pb.scale_bytes == 4) {
      const dim3 grid((unsigned)items), block(ex::kThreadsX);
      if (pb.block == 16) hipLaunchKernelGGL(gemm_exact256x128_kernel<16>, grid, block, 0, st, g);
      else if (pb.block == 32) hipLaunchKernelGGL(gemm_exact256x128_kernel<32>, grid, block, 0, st, g);
      else hipLaunchKernelGGL(gemm_exact256x128_kernel<128>, grid, block, 0, st, g);
    } else {
      const dim3 grid((unsigned)items), block(kThreads);
      if (pb.block == 16) hipLaunchKernelGGL(gemm_dq256x128_kernel<16>, grid, block, 0, st, g);
      else if (pb.block == 32) hipLaunchKernelGGL(gemm_dq256x128_kernel<32>, grid, block, 0, st, g);
      else hipLaunchKernelGGL(gemm_dq256x128_kernel<128>, grid, block, 0, st, g);
    }
    return hipGetLastError();
  }
  const int64_t items_big = pb.batch * pb.T * g.tiles_m * (g.tiles_n / 2);
  if (pb.block == 32)
    hipLaunchKernelGGL(gemm_tile256x256_kernel<32>, dim3((unsigned)items_big), dim3(big::kThreadsB), 0, st, g);
  else
    hipLaunchKernelGGL(gemm_tile256x256_kernel<128>, dim3((unsigned)items_big), dim3(big::kThreadsB), 0, st, g);
  return hipGetLastError();
}

int launch_combine_split(const Problem &pb, const DeviceTables &tab, const uint8_t *ws, const Workspace &wl,
                         float *C, void *stream) {
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const float *P = reinterpret_cast<const float *>(ws + wl.products);
  const int64_t npos = pb.mp * (pb.np / 4);
  const dim3 g2((unsigned)((npos + 255) / 256), (unsigned)pb.batch);
  const bool vec = (reinterpret_cast<uintptr_t>(C) & 15) == 0;
  if (pb.shaped) {
    if (pb.gm * pb.gn > 16) {
      const dim3 g1((unsigned)((pb.mp * pb.np + 255) / 256), (unsigned)pb.batch);
      hipLaunchKernelGGL(combine64_kernel, g1, dim3(256), 0, st, P, tab.w_full, C, pb);
    } else if (vec) {
      hipLaunchKernelGGL((combine2_kernel<true, true>), g2, dim3(256), 0, st, P, tab.w_full, C, pb);
    } else {
      hipLaunchKernelGGL((combine2_kernel<false, true>), g2, dim3(256), 0, st, P, tab.w_full, C, pb);
    }
    return hipGetLastError();
  }
  if (pb.depth == 2) {
    if (vec)
      hipLaunchKernelGGL(combine2_kernel<true>, g2, dim3(256), 0, st, P, tab.w_full, C, pb);
    else
      hipLaunchKernelGGL(combine2_kernel<false>, g2, dim3(256), 0, st, P, tab.w_full, C, pb);
    return hipGetLastError();
  }
  if (vec)
    hipLaunchKernelGGL(combine1_kernel<true>, g2, dim3(256), 0, st, P, tab.w_inner, C, pb);
  else
    hipLaunchKernelGGL(combine1_kernel<false>, g2, dim3(256), 0, st, P, tab.w_inner, C, pb);
  return hipGetLastError();
}

}  // namespace fmm
